"""bf16 state storage (S0 / S_new in bfloat16, bf16 inputs) vs the float64
oracle, through the C ABI.

The oracle consumes exactly the bf16 values the GPU reads (S0 rounded once,
to nearest even).  Two bit-exact cross-checks follow from the arithmetic:
verify on a bf16 state equals verify on an fp32 state holding the same values
(the hi/lo split of a bf16 value has a zero low half), and commit on a bf16
state equals the fp32 commit rounded once to bf16 (same fp32 operations).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_20961_amd import workload as wl
from tests.gpu_harness import DEV, TOL, Case, assert_close, say, units_of, warm_state

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tw():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_20961_amd import treewy
    return treewy


def bf16_case(w, seed, cfg_key, check_units=None):
    case = Case(w, seed=seed, cfg_key=cfg_key, check_units=check_units)
    case.S0 = wl.round_to_bf16(case.S0)              # the state as stored: bf16 values
    return case


def run_case(tw, case, label):
    w = case.w
    say("[gpu] bf16 state %s: %s" % (label, w.describe()))
    d = case.device()
    S0b = d["S0"].to(torch.bfloat16)
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    o, U = tw.treewy_verify(S0b, d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], err=err)
    S_new = tw.treewy_commit(S0b, U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"], err=err)
    torch.cuda.synchronize()
    assert int(err.abs().sum()) == 0 and S_new.dtype == torch.bfloat16
    o_ref, vt_ref, S_ref = case.oracle()
    tol = TOL["bf16"]
    eo = assert_close(label + " o", units_of(o, w, case.check), o_ref, tol)
    eu = assert_close(label + " U", units_of(U, w, case.check), vt_ref, tol)
    es = assert_close(label + " S_new", units_of(S_new, w, case.check), S_ref, tol)
    say("[gpu] bf16 state %s: max rel err o %.2e U %.2e S_new %.2e" % (label, eo, eu, es))
    return d, S0b, o, U, S_new


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_small_configs(tw, cfg):
    w = wl.scaled(wl.WORKLOADS[cfg], B=3, H=5)
    run_case(tw, bf16_case(w, 7, cfg), "c%d small" % cfg)


@pytest.mark.parametrize("cfg", [3, 4])
def test_full_size_sampled(tw, cfg):
    w = wl.WORKLOADS[cfg]
    run_case(tw, bf16_case(w, 0, cfg, wl.sample_units(w, 24)), "c%d full" % cfg)


@pytest.mark.parametrize("N", [1, 17, 33, 64])
def test_ragged(tw, N):
    w = wl.Workload("ragged", 2, 3, N, 128, 128, "bf16", "tree", min(N, 8), (4, 4, 2), (0.85, 0.999),
                    (0.05, 0.95), 16, "uniform_node")
    run_case(tw, bf16_case(w, N, 600 + N), "ragged N=%d" % N)


@pytest.mark.parametrize("kind,N,depth", [("chain", 12, 12), ("chain", 33, 33), ("chain", 64, 64), ("tree", 64, 14)])
def test_solves(tw, kind, N, depth):
    """Trees taking the medium solve (chain of 12, 64-node tree of depth 14)
    and the dense sweep (chains of 33 and 64) with a bf16 state."""
    order = "chain_depth_0_to_N" if kind == "chain" else "uniform_node"
    w = wl.Workload(kind, 2, 3, N, 128, 128, "bf16", kind, depth, (1,) if kind == "chain" else (3,), (0.85, 0.999),
                    (0.05, 0.95), 16, order)
    run_case(tw, bf16_case(w, N, 650 + N), "%s N=%d depth %d" % (kind, N, depth))


def test_bit_identical_to_fp32_state_with_bf16_values(tw):
    w = wl.scaled(wl.WORKLOADS[3], B=4, H=6)
    case = bf16_case(w, 3, 3)
    d, S0b, o, U, S_new = run_case(tw, case, "vs fp32")
    S0f = S0b.float()
    o_f, U_f = tw.treewy_verify(S0f, d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"])
    S_f = tw.treewy_commit(S0f, U_f, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"])
    torch.cuda.synchronize()
    assert torch.equal(o, o_f) and torch.equal(U, U_f)
    assert torch.equal(S_new, S_f.to(torch.bfloat16))


def test_empty_path_and_in_place(tw):
    w = wl.scaled(wl.WORKLOADS[2], B=3, H=4)
    case = bf16_case(w, 9, 2)
    d = case.device()
    S0b = d["S0"].to(torch.bfloat16)
    _, U = tw.treewy_verify(S0b, d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"])
    empty = torch.zeros_like(d["path_len"])
    assert torch.equal(tw.treewy_commit(S0b, U, d["k"], d["alpha"], d["path"], empty), S0b)
    ref = tw.treewy_commit(S0b, U, d["k"], d["alpha"], d["path"], d["path_len"])
    inplace = S0b.clone()
    tw.treewy_commit(inplace, U, d["k"], d["alpha"], d["path"], d["path_len"], S_new=inplace)
    torch.cuda.synchronize()
    assert torch.equal(inplace, ref)


@pytest.mark.parametrize("cfg", [2, 3])
def test_fused_commit_verify(tw, cfg):
    """Fused call on a bf16 state: S_new is rounded once and this round
    verifies from the rounded state, exactly as commit-then-verify does."""
    w = wl.scaled(wl.WORKLOADS[cfg], B=3, H=5)
    xp = wl.make_inputs(w, seed=20 + cfg, cfg_key=620 + cfg)
    xc = wl.make_inputs(w, seed=30 + cfg, cfg_key=630 + cfg)
    units = np.arange(w.units)
    S_old = wl.round_to_bf16(warm_state(w, units, 20 + cfg, 640 + cfg))
    dt = torch.bfloat16
    dev = lambda a, d=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(d)
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)
    S0b = dev(S_old.reshape(w.B, w.H, 128, 128), dt)
    kp, ap, pp = dev(xp["k"], dt), dev(xp["alpha"]), i32(xp["parent"])
    _, Up = tw.treewy_verify(S0b, dev(xp["q"], dt), kp, dev(xp["v"], dt), ap, dev(xp["beta"]), pp)
    cur = (dev(xc["q"], dt), dev(xc["k"], dt), dev(xc["v"], dt), dev(xc["alpha"]), dev(xc["beta"]), i32(xc["parent"]))
    S_new, o, U = tw.treewy_commit_verify(S0b, Up, kp, ap, i32(xp["path"]), i32(xp["path_len"]), *cur,
                                          parent_prev=pp)
    S_sep = tw.treewy_commit(S0b, Up, kp, ap, i32(xp["path"]), i32(xp["path_len"]), parent=pp)
    o_sep, U_sep = tw.treewy_verify(S_sep, *cur)
    torch.cuda.synchronize()
    assert S_new.dtype == torch.bfloat16
    uv = lambda a: a.reshape(w.units, *a.shape[2:])
    H = w.H
    S_ref = oracle.commit(S_old, uv(xp["k"]), uv(xp["v"]), uv(xp["alpha"]), uv(xp["beta"]),
                          np.repeat(xp["parent"], H, axis=0), np.repeat(xp["path"], H, axis=0),
                          np.repeat(xp["path_len"], H, axis=0))
    o_ref, vt_ref = oracle.verify(S_ref, uv(xc["q"]), uv(xc["k"]), uv(xc["v"]), uv(xc["alpha"]), uv(xc["beta"]),
                                  np.repeat(xc["parent"], H, axis=0))
    tol = TOL["bf16"]
    assert_close("fused S_new", units_of(S_new, w, units), S_ref, tol)
    assert_close("fused o", units_of(o, w, units), o_ref, tol)
    assert_close("fused U", units_of(U, w, units), vt_ref, tol)
    # against the separate calls: the two S_new differ at most by the rounding
    # of slightly different fp32 sums, and the verify outputs follow
    assert_close("fused vs commit", units_of(S_new, w, units), units_of(S_sep, w, units), 1e-2)
    assert_close("fused o vs verify", units_of(o, w, units), units_of(o_sep, w, units), tol)

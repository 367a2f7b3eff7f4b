"""Fast-forgetting gates vs the float64 oracle, through the C ABI.

With alpha drawn from (0.02, 0.5) the cumulative decay of a 64-node chain is
about e^-100, below the smallest float32.  Every ratio g_t / g_i the kernels
form is at most 1 and is built in extended range (mantissa and exponent), so
the outputs must match the oracle here as well: chains of 64 and 256 nodes, a
256-node deep tree, the chain prefill over 130 tokens, and the fused call
after such a round, for float32 and bfloat16 states.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_20961_amd import workload as wl
from tests.gpu_harness import DEV, TOL, Case, assert_close, say, units_of, warm_state

pytestmark = pytest.mark.gpu

FAST = (0.02, 0.5)


@pytest.fixture(scope="module")
def tw():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_20961_amd import treewy
    return treewy


def fast_workload(N, depth, dtype="bf16", B=2, H=3, caps=(3,), accept="uniform_node"):
    tree = "chain" if caps == (1,) else "tree"
    return wl.Workload("fast-decay", B, H, N, 128, 128, dtype, tree, depth, caps, FAST, (0.05, 0.95), 16, accept)


def check(tw, case, label, state="f32"):
    w = case.w
    say("[gpu] %s: %s, %s state, alpha in %s" % (label, w.describe(), state, FAST))
    if state == "bf16":
        case.S0 = wl.round_to_bf16(case.S0)
    d = case.device()
    S0 = d["S0"].to(torch.bfloat16) if state == "bf16" else d["S0"]
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    o, U = tw.treewy_verify(S0, d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], err=err)
    S_new = tw.treewy_commit(S0, U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"], err=err)
    torch.cuda.synchronize()
    assert int(err.abs().sum()) == 0
    for t in (o, U, S_new):
        assert bool(torch.isfinite(t.float()).all()), label
    o_ref, vt_ref, S_ref = case.oracle()
    tol = TOL[w.in_dtype]
    eo = assert_close(label + " o", units_of(o, w, case.check), o_ref, tol)
    eu = assert_close(label + " U", units_of(U, w, case.check), vt_ref, tol)
    es = assert_close(label + " S_new", units_of(S_new, w, case.check), S_ref, tol)
    say("[gpu] %s: max rel err o %.2e U %.2e S_new %.2e" % (label, eo, eu, es))
    return d, U


@pytest.mark.parametrize("state", ["f32", "bf16"])
def test_chain64(tw, state):
    w = fast_workload(64, 64, caps=(1,), accept="chain_depth_0_to_N")
    check(tw, Case(w, seed=1, cfg_key=2100), "fast-decay chain of 64", state)


def test_chain64_f32_inputs(tw):
    w = fast_workload(64, 64, "f32", caps=(1,), accept="chain_depth_0_to_N")
    check(tw, Case(w, seed=2, cfg_key=2101), "fast-decay f32 chain of 64")


@pytest.mark.parametrize("state", ["f32", "bf16"])
def test_chain256(tw, state):
    w = fast_workload(256, 256, caps=(1,), accept="chain_depth_0_to_N")
    check(tw, Case(w, seed=3, cfg_key=2102), "fast-decay chain of 256", state)


@pytest.mark.parametrize("state", ["f32", "bf16"])
def test_deep_tree256(tw, state):
    w = fast_workload(256, 96, caps=(4, 4, 2))
    check(tw, Case(w, seed=4, cfg_key=2103), "fast-decay tree of 256, depth 96", state)


def test_shallow_tree64(tw):
    """Depth 8 (the register-gather solve) with fast decay."""
    w = fast_workload(64, 8, caps=(4, 4, 2))
    check(tw, Case(w, seed=5, cfg_key=2104), "fast-decay tree of 64, depth 8")


@pytest.mark.parametrize("dtype,state", [("bf16", "f32"), ("bf16", "bf16"), ("f32", "f32")])
def test_prefill130(tw, dtype, state):
    T = 130
    w = fast_workload(T, T, dtype, caps=(1,), accept="chain_depth_0_to_N")
    x = wl.make_inputs(w, seed=6, cfg_key=2105)
    n = w.units
    S0 = warm_state(w, np.arange(n), 6, 2106)
    if state == "bf16":
        S0 = wl.round_to_bf16(S0)
    say("[gpu] fast-decay prefill T=%d %s inputs, %s state" % (T, dtype, state))
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    sdt = torch.bfloat16 if state == "bf16" else torch.float32
    dev = lambda a, d=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(d)
    S0_d = dev(S0.reshape(w.B, w.H, 128, 128), sdt)
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    S_T, o = tw.treewy_chain_prefill(S0_d, dev(x["q"], dt), dev(x["k"], dt), dev(x["v"], dt), dev(x["alpha"]),
                                     dev(x["beta"]), err=err)
    torch.cuda.synchronize()
    assert int(err.abs().sum()) == 0
    uv = lambda a: a.reshape(n, *a.shape[2:])
    par = np.tile(np.arange(-1, T - 1, dtype=np.int32), (n, 1))
    S_ref = oracle.chain(S0, uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]))
    o_ref, _ = oracle.verify(S0, uv(x["q"]), uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]), par)
    tol = TOL[dtype]
    es = assert_close("S_T", S_T.float().cpu().numpy().reshape(n, 128, 128), S_ref, tol)
    eo = assert_close("o", o.float().cpu().numpy().reshape(n, T, 128), o_ref, tol)
    say("[gpu] fast-decay prefill: max rel err S_T %.2e o %.2e" % (es, eo))


@pytest.mark.parametrize("state", ["f32", "bf16"])
def test_fused_after_fast_chain(tw, state):
    """The fused call committing a 64-node fast-decay chain's path into the
    next round's verify equals commit-then-verify on the oracle."""
    w = fast_workload(64, 64, caps=(1,), accept="chain_depth_0_to_N")
    case = Case(w, seed=7, cfg_key=2107)
    d, U = check(tw, case, "fast-decay chain of 64 (previous round)", state)
    _, _, S_ref = case.oracle()
    w2 = fast_workload(64, 8, caps=(4, 4, 2))
    x2 = wl.make_inputs(w2, seed=8, cfg_key=2108)
    n = w.units
    S_mid = S_ref if state == "f32" else wl.round_to_bf16(S_ref.astype(np.float32))
    par2 = np.repeat(x2["parent"], w2.H, axis=0)
    uv = lambda a: a.reshape(n, *a.shape[2:])
    o2_ref, vt2_ref = oracle.verify(S_mid, uv(x2["q"]), uv(x2["k"]), uv(x2["v"]), uv(x2["alpha"]),
                                    uv(x2["beta"]), par2)
    dev = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(dt)
    S_old = d["S0"].to(torch.bfloat16) if state == "bf16" else d["S0"]
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    S_new, o2, U2 = tw.treewy_commit_verify(
        S_old, U, d["k"], d["alpha"], d["path"], d["path_len"], dev(x2["q"], torch.bfloat16),
        dev(x2["k"], torch.bfloat16), dev(x2["v"], torch.bfloat16), dev(x2["alpha"]), dev(x2["beta"]),
        torch.from_numpy(x2["parent"]).to(DEV), parent_prev=d["parent"], err=err)
    torch.cuda.synchronize()
    assert int(err.abs().sum()) == 0
    tol = TOL["bf16"]
    es = assert_close("fused S_new", S_new.float().cpu().numpy().reshape(n, 128, 128), S_ref, tol)
    eo = assert_close("fused o", o2.float().cpu().numpy().reshape(n, 64, 128), o2_ref, tol)
    eu = assert_close("fused U", U2.cpu().numpy().reshape(n, 64, 128), vt2_ref, tol)
    say("[gpu] fast-decay fused (%s state): max rel err S_new %.2e o %.2e U %.2e" % (state, es, eo, eu))

"""treewy_chain_prefill vs the float64 oracle, through the C ABI.

The reference is eq. 1 run over the chain: every token's output o_t = S_t q_t
(the oracle's tree routine on a chain of T nodes) and the state after the last
token (its chain routine).  Chunks of 32 bf16 tokens (64 fp32 tokens) with
ragged tails, fp32 and bf16 inputs, fp32 and bf16 state, in place.  The
lengths put each of the three solves of T = (I + B)^{-1} in the last chunk:
at most 9 tokens (8 ancestors: registers), 10 to 17 (B read one ancestor
ahead: 12, 49 = 32 + 17, 10, 81 = 64 + 17, 17) and more (the dense sweep).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_20961_amd import workload as wl
from tests.gpu_harness import DEV, TOL, assert_close, say, warm_state

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tw():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_20961_amd import treewy
    return treewy


def chain_workload(T, dtype, B=2, H=3):
    return wl.Workload("prefill", B, H, T, 128, 128, dtype, "chain", max(T, 1), (1,), (0.85, 0.999),
                       (0.05, 0.95), 16, "chain_depth_0_to_N")


def run(tw, T, dtype, state="f32", in_place=False, seed=0):
    w = chain_workload(T, dtype)
    x = wl.make_inputs(w, seed=seed, cfg_key=700 + T)
    n = w.units
    S0 = warm_state(w, np.arange(n), seed, 701 + T)
    if state == "bf16":
        S0 = wl.round_to_bf16(S0)
    say("[gpu] prefill T=%d %s inputs, %s state" % (T, dtype, state))
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    sdt = torch.bfloat16 if state == "bf16" else torch.float32
    dev = lambda a, d=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(d)
    S0_d = dev(S0.reshape(w.B, w.H, 128, 128), sdt)
    args = (dev(x["q"], dt), dev(x["k"], dt), dev(x["v"], dt), dev(x["alpha"]), dev(x["beta"]))
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    S_T, o = tw.treewy_chain_prefill(S0_d, *args, S_T=S0_d if in_place else None, err=err)
    torch.cuda.synchronize()
    assert int(err.abs().sum()) == 0
    uv = lambda a: a.reshape(n, *a.shape[2:])
    par = np.tile(np.arange(-1, T - 1, dtype=np.int32), (n, 1))
    S_ref = oracle.chain(S0, uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]))
    tol = TOL[dtype]
    es = assert_close("S_T", S_T.float().cpu().numpy().reshape(n, 128, 128), S_ref, tol)
    eo = 0.0
    if T > 0:
        o_ref, _ = oracle.verify(S0, uv(x["q"]), uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]), par)
        eo = assert_close("o", o.float().cpu().numpy().reshape(n, T, 128), o_ref, tol)
    say("[gpu] prefill T=%d: max rel err S_T %.2e o %.2e" % (T, es, eo))
    return S0_d, S_T, o


@pytest.mark.parametrize("T", [1, 5, 12, 31, 32, 33, 49, 63, 64, 65, 128, 200])
def test_prefill_bf16(tw, T):
    run(tw, T, "bf16")


@pytest.mark.parametrize("T", [1, 10, 64, 81, 130])
def test_prefill_f32(tw, T):
    run(tw, T, "f32")


@pytest.mark.parametrize("T", [17, 32, 40, 129])
def test_prefill_bf16_state(tw, T):
    run(tw, T, "bf16", state="bf16")


def test_prefill_in_place_and_empty(tw):
    run(tw, 100, "bf16", in_place=True, seed=3)
    S0, S_T, o = run(tw, 0, "bf16", seed=4)
    assert torch.equal(S_T, S0) and o.numel() == 0


@pytest.mark.parametrize("T", [5, 12, 32])
def test_prefill_equals_verify_then_commit(tw, T):
    """One chunk of prefill (5, 12 or 32 bf16 tokens: each of the three
    solves) is a chain verify plus a commit of the whole chain."""
    w = chain_workload(T, "bf16", B=3, H=2)
    x = wl.make_inputs(w, seed=9, cfg_key=790)
    S0 = torch.from_numpy(warm_state(w, np.arange(w.units), 9, 791).reshape(w.B, w.H, 128, 128)).to(DEV)
    dev = lambda a, d=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(d)
    q, k, v = (dev(x[n], torch.bfloat16) for n in ("q", "k", "v"))
    al, be = dev(x["alpha"]), dev(x["beta"])
    S_T, o = tw.treewy_chain_prefill(S0, q, k, v, al, be)
    par = torch.from_numpy(np.tile(np.arange(-1, T - 1, dtype=np.int32), (w.B, 1))).to(DEV)
    o2, U = tw.treewy_verify(S0, q, k, v, al, be, par)
    path = torch.from_numpy(np.tile(np.arange(T, dtype=np.int32), (w.B, 1))).to(DEV)
    S2 = tw.treewy_commit(S0, U, k, al, path, torch.full((w.B,), T, dtype=torch.int32, device=DEV), parent=par)
    torch.cuda.synchronize()
    assert torch.equal(o, o2)                      # the same verify kernel on the same chain
    n = w.units
    assert_close("S_T vs commit", S_T.cpu().numpy().reshape(n, 128, 128), S2.cpu().numpy().reshape(n, 128, 128),
                 TOL["f32"])


def test_prefill_many_units_per_workgroup(tw):
    """4096 units (several per resident workgroup), T = 150: sampled units
    against the oracle."""
    T, B, H = 150, 64, 64
    w = wl.Workload("prefill", B, H, T, 128, 128, "bf16", "chain", T, (1,), (0.85, 0.999), (0.05, 0.95), 16,
                    "chain_depth_0_to_N")
    x = wl.make_inputs(w, seed=21, cfg_key=2100)
    units = wl.sample_units(w, 8)
    S0 = warm_state(w, units, 21, 2101)
    S0_all = np.zeros((w.units, 128, 128), dtype=np.float32)
    S0_all[units] = S0
    say("[gpu] prefill T=%d over %d units" % (T, w.units))
    dev = lambda a, d=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(d)
    S_T, o = tw.treewy_chain_prefill(dev(S0_all.reshape(B, H, 128, 128)), dev(x["q"], torch.bfloat16),
                                     dev(x["k"], torch.bfloat16), dev(x["v"], torch.bfloat16), dev(x["alpha"]),
                                     dev(x["beta"]))
    torch.cuda.synchronize()
    uv = lambda a: a.reshape(w.units, *a.shape[2:])[units]
    S_ref = oracle.chain(S0, uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]))
    par = np.tile(np.arange(-1, T - 1, dtype=np.int32), (len(units), 1))
    o_ref, _ = oracle.verify(S0, uv(x["q"]), uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]), par)
    es = assert_close("S_T", S_T.float().cpu().numpy().reshape(w.units, 128, 128)[units], S_ref, TOL["bf16"])
    eo = assert_close("o", o.float().cpu().numpy().reshape(w.units, T, 128)[units], o_ref, TOL["bf16"])
    say("[gpu] prefill over %d units: max rel err S_T %.2e o %.2e" % (w.units, es, eo))


def test_prefill_bench_length(tw):
    """The benchmark's chunk count: T = 1024 (thirty-two 32-token chunks), 512
    units, bf16 tokens and an fp32 state; sampled units against the oracle."""
    T, B, H = 1024, 8, 64
    w = wl.Workload("prefill", B, H, T, 128, 128, "bf16", "chain", T, (1,), (0.85, 0.999), (0.05, 0.95), 16,
                    "chain_depth_0_to_N")
    x = wl.make_inputs(w, seed=23, cfg_key=2300)
    units = wl.sample_units(w, 4)
    S0 = warm_state(w, units, 23, 2301)
    S0_all = np.zeros((w.units, 128, 128), dtype=np.float32)
    S0_all[units] = S0
    say("[gpu] prefill T=%d over %d units" % (T, w.units))
    dev = lambda a, d=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(d)
    S_T, o = tw.treewy_chain_prefill(dev(S0_all.reshape(B, H, 128, 128)), dev(x["q"], torch.bfloat16),
                                     dev(x["k"], torch.bfloat16), dev(x["v"], torch.bfloat16), dev(x["alpha"]),
                                     dev(x["beta"]))
    torch.cuda.synchronize()
    uv = lambda a: a.reshape(w.units, *a.shape[2:])[units]
    S_ref = oracle.chain(S0, uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]))
    par = np.tile(np.arange(-1, T - 1, dtype=np.int32), (len(units), 1))
    o_ref, _ = oracle.verify(S0, uv(x["q"]), uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]), par)
    es = assert_close("S_T", S_T.float().cpu().numpy().reshape(w.units, 128, 128)[units], S_ref, TOL["bf16"])
    eo = assert_close("o", o.float().cpu().numpy().reshape(w.units, T, 128)[units], o_ref, TOL["bf16"])
    say("[gpu] prefill T=%d: max rel err S_T %.2e o %.2e" % (T, es, eo))

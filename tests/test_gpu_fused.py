"""treewy_commit_verify (previous round's commit fused into this round's
verify) vs the float64 oracle, through the C ABI.

The reference is the composition the call is defined by: the oracle commits
the previous round's accepted path from S_old (eq. 3's left side, the state of
the accepted node under eq. 1), then verifies this round's draft from that
state.  The previous round's pseudo-values U_prev are an input of the call, so
the test produces them with treewy_verify on S_old, as a serving loop does.
Bar as for the other parity tests: normwise max relative error per (sequence,
head) <= 1e-4 (float32 inputs) / 2e-2 (bfloat16); flags bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_20961_amd import workload as wl
from tests.gpu_harness import DEV, TOL, assert_close, say, units_of, warm_state

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tw():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_20961_amd import treewy
    return treewy


def _dev(x, w):
    dt = torch.bfloat16 if w.in_dtype == "bf16" else torch.float32

    def inp(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(dt)

    def f32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)

    return dict(q=inp(x["q"]), k=inp(x["k"]), v=inp(x["v"]), alpha=f32(x["alpha"]), beta=f32(x["beta"]),
                parent=i32(x["parent"]), path=i32(x["path"]), path_len=i32(x["path_len"]))


class TwoRounds:
    """Round p (previous, with its accepted paths) and round c (current) on
    the same (sequence, head) grid; S_old is the state before round p."""

    def __init__(self, wp, wc, seed, check_units=None, xp=None):
        assert (wp.B, wp.H) == (wc.B, wc.H) and wp.in_dtype == wc.in_dtype
        self.wp, self.wc = wp, wc
        self.xp = xp if xp is not None else wl.make_inputs(wp, seed=seed, cfg_key=300 + seed)
        self.xc = wl.make_inputs(wc, seed=seed + 1, cfg_key=301 + seed)
        n = wp.units
        self.check = np.arange(n) if check_units is None else np.asarray(check_units)
        S_chk = warm_state(wp, self.check, seed, 302 + seed)
        S = S_chk[np.searchsorted(self.check, np.arange(n)) % len(self.check)]
        S[self.check] = S_chk
        self.S_old = np.ascontiguousarray(S, dtype=np.float32)

    def uv(self, x, w, name):
        a = x[name]
        return a.reshape(w.units, *a.shape[2:])[self.check]

    def oracle(self):
        wp, wc, c = self.wp, self.wc, self.check
        H = wp.H
        S_new = oracle.commit(self.S_old[c], self.uv(self.xp, wp, "k"), self.uv(self.xp, wp, "v"),
                              self.uv(self.xp, wp, "alpha"), self.uv(self.xp, wp, "beta"),
                              np.repeat(self.xp["parent"], H, axis=0)[c],
                              np.repeat(self.xp["path"], H, axis=0)[c],
                              np.repeat(self.xp["path_len"], H, axis=0)[c])
        o, vt = oracle.verify(S_new, self.uv(self.xc, wc, "q"), self.uv(self.xc, wc, "k"),
                              self.uv(self.xc, wc, "v"), self.uv(self.xc, wc, "alpha"),
                              self.uv(self.xc, wc, "beta"), np.repeat(self.xc["parent"], H, axis=0)[c])
        return S_new, o, vt

    def run(self, tw, parent_prev=True, in_place=False):
        wp, wc = self.wp, self.wc
        dp, dc = _dev(self.xp, wp), _dev(self.xc, wc)
        S_old = torch.from_numpy(self.S_old.reshape(wp.B, wp.H, 128, 128)).to(DEV)
        _, U_prev = tw.treewy_verify(S_old, dp["q"], dp["k"], dp["v"], dp["alpha"], dp["beta"], dp["parent"])
        err = torch.zeros(wp.B, dtype=torch.int32, device=DEV)
        kw = {}
        if in_place:
            kw["S_new"] = S_old
            if wc.N == wp.N:
                kw["U"] = U_prev
        S_new, o, U = tw.treewy_commit_verify(S_old, U_prev, dp["k"], dp["alpha"], dp["path"], dp["path_len"],
                                              dc["q"], dc["k"], dc["v"], dc["alpha"], dc["beta"], dc["parent"],
                                              parent_prev=dp["parent"] if parent_prev else None, err=err, **kw)
        torch.cuda.synchronize()
        return S_new, o, U, err, dict(dp=dp, dc=dc, U_prev=U_prev)

    def check_against_oracle(self, tw, label, **kw):
        say("[gpu] fused %s: prev %s | cur %s" % (label, self.wp.describe(), self.wc.describe()))
        S_new, o, U, err, _ = self.run(tw, **kw)
        assert int(err.abs().sum()) == 0
        S_ref, o_ref, vt_ref = self.oracle()
        tol = TOL[self.wc.in_dtype]
        es = assert_close(label + " S_new", units_of(S_new, self.wp, self.check), S_ref, tol)
        eo = assert_close(label + " o", units_of(o, self.wc, self.check), o_ref, tol)
        eu = assert_close(label + " U", units_of(U, self.wc, self.check), vt_ref, tol)
        say("[gpu] fused %s: max rel err S_new %.2e o %.2e U %.2e" % (label, es, eo, eu))


def test_fused_chain4_f32(tw):
    w = wl.WORKLOADS[0]
    TwoRounds(w, w, seed=0).check_against_oracle(tw, "chain4 f32")


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_fused_small_configs(tw, cfg):
    w = wl.scaled(wl.WORKLOADS[cfg], B=3, H=5)
    TwoRounds(w, w, seed=10 + cfg).check_against_oracle(tw, "c%d small" % cfg)


def test_fused_full_size_397B_tree(tw):
    w = wl.WORKLOADS[3]
    TwoRounds(w, w, seed=20, check_units=wl.sample_units(w, 24)).check_against_oracle(tw, "c3 full")


def test_fused_full_size_stress_tree(tw):
    """The 32-node stress workload at full size (16384 units), 24 sampled."""
    w = wl.WORKLOADS[4]
    TwoRounds(w, w, seed=21, check_units=wl.sample_units(w, 24)).check_against_oracle(tw, "c4 full")


@pytest.mark.parametrize("Np,Nc", [(16, 64), (64, 8), (5, 33), (64, 64)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_fused_round_sizes_differ(tw, Np, Nc, dtype):
    mk = lambda N: wl.Workload("fused", 2, 3, N, 128, 128, dtype, "tree", min(N, 8), (4, 4, 2),
                               (0.85, 0.999), (0.05, 0.95), 16, "uniform_node")
    TwoRounds(mk(Np), mk(Nc), seed=Np + Nc).check_against_oracle(tw, "Np=%d Nc=%d %s" % (Np, Nc, dtype))


@pytest.mark.parametrize("kind,Nc,depth", [("chain", 12, 12), ("chain", 17, 17), ("chain", 33, 33), ("chain", 64, 64),
                                           ("tree", 64, 14)])
def test_fused_current_round_solves(tw, kind, Nc, depth):
    """The current round's tree taking each solve of T = (I + B)^{-1} inside
    the fused call: chains of 12 and 17 and a 64-node tree of depth 14 (B read
    one ancestor ahead), chains of 33 and 64 (the dense sweep, at 64 rows)."""
    wp = wl.Workload("fused", 2, 3, 16, 128, 128, "bf16", "tree", 6, (4, 4, 2), (0.85, 0.999), (0.05, 0.95),
                     16, "uniform_node")
    order = "chain_depth_0_to_N" if kind == "chain" else "uniform_node"
    wc = wl.Workload(kind, 2, 3, Nc, 128, 128, "bf16", kind, depth, (1,) if kind == "chain" else (3,),
                     (0.85, 0.999), (0.05, 0.95), 16, order)
    TwoRounds(wp, wc, seed=40 + Nc).check_against_oracle(tw, "current %s N=%d depth %d" % (kind, Nc, depth))


@pytest.mark.parametrize("L", [9, 17, 40, 64])
def test_fused_long_paths(tw, L):
    """Accepted paths longer than one staging pass (8 rows) of the rank update."""
    wp = wl.Workload("chain", 2, 2, 64, 128, 128, "bf16", "chain", 64, (1,), (0.85, 0.999), (0.05, 0.95),
                     16, "chain_depth_0_to_N")
    xp = wl.make_inputs(wp, seed=L, cfg_key=400 + L)
    xp["path"] = np.tile(np.arange(64, dtype=np.int32), (2, 1))
    xp["path"][:, L:] = -1
    xp["path_len"] = np.array([L, L - 1], dtype=np.int32)
    wc = wl.Workload("tree", 2, 2, 33, 128, 128, "bf16", "tree", 6, (3,), (0.85, 0.999), (0.05, 0.95),
                     16, "uniform_node")
    TwoRounds(wp, wc, seed=L, xp=xp).check_against_oracle(tw, "path L=%d" % L)


def test_fused_in_place_and_without_parent(tw):
    w = wl.scaled(wl.WORKLOADS[2], B=3, H=4)
    case = TwoRounds(w, w, seed=31)
    S_new, o, U, err, _ = case.run(tw, parent_prev=False, in_place=True)
    assert int(err.abs().sum()) == 0
    S_ref, o_ref, vt_ref = case.oracle()
    tol = TOL[w.in_dtype]
    assert_close("in-place S_new", units_of(S_new, w, case.check), S_ref, tol)
    assert_close("in-place o", units_of(o, w, case.check), o_ref, tol)
    assert_close("in-place U", units_of(U, w, case.check), vt_ref, tol)


def test_fused_matches_separate_calls(tw):
    """Fused call vs treewy_commit then treewy_verify on the GPU: same values
    up to the two kernels' own rounding (fp32 FMA vs split-bf16 MFMA)."""
    w = wl.scaled(wl.WORKLOADS[3], B=4, H=6)
    case = TwoRounds(w, w, seed=41)
    S_new, o, U, _, d = case.run(tw)
    dp, dc = d["dp"], d["dc"]
    S_old = torch.from_numpy(case.S_old.reshape(w.B, w.H, 128, 128)).to(DEV)
    S_sep = tw.treewy_commit(S_old, d["U_prev"], dp["k"], dp["alpha"], dp["path"], dp["path_len"],
                             parent=dp["parent"])
    o_sep, U_sep = tw.treewy_verify(S_sep, dc["q"], dc["k"], dc["v"], dc["alpha"], dc["beta"], dc["parent"])
    torch.cuda.synchronize()
    all_units = np.arange(w.units)
    tol = TOL[w.in_dtype]
    assert_close("S_new vs commit", units_of(S_new, w, all_units), units_of(S_sep, w, all_units), TOL["f32"])
    assert_close("o vs verify", units_of(o, w, all_units), units_of(o_sep, w, all_units), tol)
    assert_close("U vs verify", units_of(U, w, all_units), units_of(U_sep, w, all_units), tol)


def test_fused_empty_path_is_plain_verify(tw):
    """Nothing accepted: S_new = S_old bit for bit, and o, U equal treewy_verify
    on S_old bit for bit (the update multiplies by 1 and adds 0)."""
    w = wl.scaled(wl.WORKLOADS[3], B=2, H=3)
    xp = wl.make_inputs(w, seed=51, cfg_key=351)
    xp["path_len"][:] = 0
    case = TwoRounds(w, w, seed=51, xp=xp)
    S_new, o, U, err, d = case.run(tw)
    dc = d["dc"]
    S_old = torch.from_numpy(case.S_old.reshape(w.B, w.H, 128, 128)).to(DEV)
    o_v, U_v = tw.treewy_verify(S_old, dc["q"], dc["k"], dc["v"], dc["alpha"], dc["beta"], dc["parent"])
    torch.cuda.synchronize()
    assert int(err.abs().sum()) == 0
    assert torch.equal(S_new, S_old)
    assert torch.equal(o, o_v) and torch.equal(U, U_v)


def test_fused_bad_path_keeps_state(tw):
    w = wl.scaled(wl.WORKLOADS[2], B=4, H=2)
    xp = wl.make_inputs(w, seed=61, cfg_key=361)
    xp["path"][1, :2] = [0, 0]          # not increasing
    xp["path_len"][1] = 2
    xp["path_len"][2] = w.max_depth + 1  # longer than L_max
    xp["path"][3, 0] = w.N              # node out of range
    xp["path_len"][3] = max(int(xp["path_len"][3]), 1)
    case = TwoRounds(w, w, seed=61, xp=xp)
    S_new, o, U, err, _ = case.run(tw)
    flags = err.cpu().numpy()
    assert flags[0] == 0 and list(flags[1:]) == [tw.FLAG_BAD_PATH] * 3
    S_old = torch.from_numpy(case.S_old.reshape(w.B, w.H, 128, 128)).to(DEV)
    assert torch.equal(S_new[1:], S_old[1:])


def test_fused_empty_current_draft(tw):
    """N = 0 this round: the commit still happens."""
    w = wl.scaled(wl.WORKLOADS[2], B=2, H=3)
    wc = wl.scaled(w, N=0)
    case = TwoRounds.__new__(TwoRounds)
    case.wp, case.wc = w, wc
    case.xp = wl.make_inputs(w, seed=71, cfg_key=371)
    case.check = np.arange(w.units)
    case.S_old = warm_state(w, case.check, 71, 372)
    dp = _dev(case.xp, w)
    S_old = torch.from_numpy(case.S_old.reshape(w.B, w.H, 128, 128)).to(DEV)
    _, U_prev = tw.treewy_verify(S_old, dp["q"], dp["k"], dp["v"], dp["alpha"], dp["beta"], dp["parent"])
    e = lambda *s, dt=torch.bfloat16: torch.empty(s, dtype=dt, device=DEV)
    S_new, o, U = tw.treewy_commit_verify(S_old, U_prev, dp["k"], dp["alpha"], dp["path"], dp["path_len"],
                                          e(2, 3, 0, 128), e(2, 3, 0, 128), e(2, 3, 0, 128),
                                          e(2, 3, 0, dt=torch.float32), e(2, 3, 0, dt=torch.float32),
                                          e(2, 0, dt=torch.int32), parent_prev=dp["parent"])
    torch.cuda.synchronize()
    H = w.H
    S_ref = oracle.commit(case.S_old, case.xp["k"].reshape(w.units, w.N, 128), case.xp["v"].reshape(w.units, w.N, 128),
                          case.xp["alpha"].reshape(w.units, w.N), case.xp["beta"].reshape(w.units, w.N),
                          np.repeat(case.xp["parent"], H, axis=0), np.repeat(case.xp["path"], H, axis=0),
                          np.repeat(case.xp["path_len"], H, axis=0))
    assert_close("N=0 S_new", units_of(S_new, w, case.check), S_ref, TOL["bf16"])


@pytest.mark.parametrize("state", ["f32", "bf16"])
@pytest.mark.parametrize("N", [16, 64])
def test_fused_in_place_bit_identical(tw, state, N):
    """S_new written over S_old gives bit for bit what the out-of-place call
    gives (each state row is read by the wave that writes it, before any of
    its lines is written), and the out-of-place call leaves S_old alone.
    Both state types and both padded node counts (32 and 64)."""
    w = wl.Workload("fused", 3, 4, N, 128, 128, "bf16", "tree", min(N, 8), (4, 4, 2), (0.85, 0.999),
                    (0.05, 0.95), 16, "uniform_node")
    say("[gpu] fused in place: %s state, N=%d" % (state, N))
    case = TwoRounds(w, w, seed=70 + N)
    dp, dc = _dev(case.xp, w), _dev(case.xc, w)
    sdt = torch.float32 if state == "f32" else torch.bfloat16
    S_old = torch.from_numpy(case.S_old.reshape(w.B, w.H, 128, 128)).to(DEV).to(sdt)
    _, U_prev = tw.treewy_verify(S_old, dp["q"], dp["k"], dp["v"], dp["alpha"], dp["beta"], dp["parent"])
    args = (U_prev, dp["k"], dp["alpha"], dp["path"], dp["path_len"], dc["q"], dc["k"], dc["v"], dc["alpha"],
            dc["beta"], dc["parent"])
    keep = S_old.clone()
    S_out, o_out, U_out = tw.treewy_commit_verify(S_old, *args, parent_prev=dp["parent"])
    torch.cuda.synchronize()
    assert torch.equal(S_old, keep)
    S_in = S_old.clone()
    S_ret, o_in, U_in = tw.treewy_commit_verify(S_in, *args, parent_prev=dp["parent"], S_new=S_in)
    torch.cuda.synchronize()
    assert S_ret.data_ptr() == S_in.data_ptr()
    assert torch.equal(S_in, S_out) and torch.equal(o_in, o_out) and torch.equal(U_in, U_out)

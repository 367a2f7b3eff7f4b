"""HIP path vs the float64 oracle, element by element, through the C ABI.

Bar: normwise max relative error per (sequence, head) slice <= 1e-4 for
float32 inputs and <= 2e-2 for bfloat16 inputs (fp32 accumulation); indices,
paths and error flags bit-exact.
"""
import numpy as np
import pytest
import torch

from paper_2608_20961_amd import workload as wl
from tests.gpu_harness import DEV, TOL, Case, assert_close, say, units_of

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tw():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_20961_amd import treewy
    return treewy


def run_and_check(tw, case: Case, label: str, snapshot=False):
    w = case.w
    say("[gpu] %s: %s" % (label, w.describe()))
    d = case.device()
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    o, U = tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], err=err)
    S_new = tw.treewy_commit(d["S0"], U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"], err=err)
    torch.cuda.synchronize()
    assert int(err.abs().sum()) == 0
    o_ref, vt_ref, S_ref = case.oracle()
    tol = TOL[w.in_dtype]
    eo = assert_close(label + " o", units_of(o, w, case.check), o_ref, tol)
    eu = assert_close(label + " U", units_of(U, w, case.check), vt_ref, tol)
    es = assert_close(label + " S_new", units_of(S_new, w, case.check), S_ref, tol)
    say("[gpu] %s: max rel err o %.2e U %.2e S_new %.2e" % (label, eo, eu, es))
    return d, o, U, S_new


# ---------------------------------------------------------------------------
# The five workloads.  c0 at its own size; c1..c4 at small sizes checked in
# full, then at their full sizes (the launch the benchmark times) on samples.
# ---------------------------------------------------------------------------
def test_c0_chain4_f32(tw):
    run_and_check(tw, Case(wl.WORKLOADS[0], seed=0, cfg_key=0), "c0")


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_small_batches_all_configs(tw, cfg):
    w = wl.scaled(wl.WORKLOADS[cfg], B=3, H=5)
    run_and_check(tw, Case(w, seed=1, cfg_key=cfg), "c%d small" % cfg)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_full_size_sampled(tw, cfg):
    w = wl.WORKLOADS[cfg]
    run_and_check(tw, Case(w, seed=0, cfg_key=cfg, check_units=wl.sample_units(w, 24)), "c%d full" % cfg)


# ---------------------------------------------------------------------------
# Ragged and degenerate shapes
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("N,depth,caps", [(1, 1, (1,)), (5, 3, (2,)), (31, 6, (3,)), (32, 5, (4,)),
                                          (33, 7, (4, 3, 2)), (47, 8, (4, 4, 2)), (64, 12, (3,))])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ragged_trees(tw, N, depth, caps, dtype):
    w = wl.Workload("ragged", 2, 3, N, 128, 128, dtype, "tree", depth, caps, (0.85, 0.999),
                    (0.05, 0.95), 16, "uniform_node")
    run_and_check(tw, Case(w, seed=N, cfg_key=100 + N), "ragged N=%d %s" % (N, dtype))


@pytest.mark.parametrize("N", [17, 64])
def test_long_chains(tw, N):
    w = wl.Workload("chain", 2, 2, N, 128, 128, "bf16", "chain", N, (1,), (0.85, 0.999), (0.05, 0.95),
                    16, "chain_depth_0_to_N")
    run_and_check(tw, Case(w, seed=3, cfg_key=200 + N), "chain N=%d" % N)


def spine_tree(N, anc, rng):
    """A tree whose deepest node has exactly `anc` ancestors: nodes 0..anc
    form a chain and every later node hangs off a random earlier node of
    depth below anc."""
    par = np.full(N, wl.ROOT, dtype=np.int32)
    depth = np.zeros(N, dtype=np.int64)
    for t in range(1, N):
        if t <= anc:
            par[t] = t - 1
        elif anc > 0:
            par[t] = rng.choice(np.flatnonzero(depth[:t] < anc))
        depth[t] = depth[par[t]] + 1 if par[t] != wl.ROOT else 0
    assert depth.max() == anc and wl.is_topological(par)
    return par


@pytest.mark.parametrize("N,ancs", [(32, (9, 8, 17)), (32, (16, 0, 31)), (64, (8, 9, 16)), (64, (17, 16, 12))])
def test_solve_depth_classes(tw, N, ancs):
    """The three solves of T = (I + B)^{-1}, chosen per unit by its deepest
    node: at most 8 ancestors (entries of B gathered into registers), 9 to 16
    (B read one ancestor ahead), more (the dense blocked sweep).  Sequence b
    has exactly ancs[b] ancestors at its deepest node, so every boundary
    meets the others within one launch."""
    w = wl.Workload("spine", len(ancs), 2, N, 128, 128, "bf16", "tree", max(ancs) + 1, (2,), (0.85, 0.999),
                    (0.05, 0.95), 16, "uniform_node")
    x = wl.make_inputs(w, seed=11, cfg_key=600 + N)
    rng = np.random.default_rng(N)
    for b, anc in enumerate(ancs):
        par = spine_tree(N, anc, rng)
        x["parent"][b] = par
        nodes = wl.ancestors_and_self(par, int(rng.integers(N)))
        x["path"][b] = -1
        x["path"][b, :len(nodes)] = nodes
        x["path_len"][b] = len(nodes)
    run_and_check(tw, Case(w, seed=11, cfg_key=600 + N, inputs=x), "depth classes N=%d %s" % (N, ancs))


def test_fixed_width_tree_shapes(tw):
    for shape in ([2, 1, 1], [3, 3, 3], [4, 3, 3]):
        par = wl.width_tree(shape)
        N = len(par)
        w = wl.Workload("width", 4, 2, N, 128, 128, "bf16", "tree", len(shape), (9,), (0.85, 0.999),
                        (0.05, 0.95), 16, "uniform_node")
        x = wl.make_inputs(w, seed=5, cfg_key=300 + N)
        x["parent"] = np.tile(par, (w.B, 1))
        rng = np.random.default_rng(N)
        for b in range(w.B):
            nodes = wl.ancestors_and_self(par, int(rng.integers(N)))
            x["path"][b] = -1
            x["path"][b, :len(nodes)] = nodes
            x["path_len"][b] = len(nodes)
        run_and_check(tw, Case(w, seed=5, cfg_key=300 + N, inputs=x), "widths %s" % shape)


def test_all_nodes_off_the_root(tw):
    """A star: every node hangs off S0 (no solve coupling at all)."""
    w = wl.Workload("star", 2, 2, 40, 128, 128, "bf16", "tree", 1, (64,), (0.85, 0.999), (0.05, 0.95),
                    16, "uniform_node")
    run_and_check(tw, Case(w, seed=7, cfg_key=400), "star N=40")


# ---------------------------------------------------------------------------
# Special cases with known answers, on the GPU
# ---------------------------------------------------------------------------
def test_beta_zero_pure_decay(tw):
    w = wl.scaled(wl.WORKLOADS[3], B=2, H=2)
    x = wl.make_inputs(w, seed=2, cfg_key=3)
    x["beta"][:] = 0.0
    case = Case(w, seed=2, cfg_key=3, inputs=x)
    _, o, U, S_new = run_and_check(tw, case, "beta=0")
    assert float(U.abs().max()) == 0.0


def test_overwrite_orthonormal_keys(tw):
    """alpha = beta = 1, orthonormal keys: U = v - S0 k exactly in exact arithmetic."""
    w = wl.Workload("ortho", 1, 2, 24, 128, 128, "f32", "tree", 5, (3,), (1.0, 1.0), (1.0, 1.0), 8,
                    "uniform_node")
    x = wl.make_inputs(w, seed=3, cfg_key=500)
    rng = np.random.default_rng(0)
    for h in range(w.H):
        Qm, _ = np.linalg.qr(rng.standard_normal((128, 128)))
        x["k"][0, h] = Qm[:w.N].astype(np.float32)
    x["alpha"][:] = 1.0
    x["beta"][:] = 1.0
    run_and_check(tw, Case(w, seed=3, cfg_key=500, inputs=x), "overwrite")


def test_fp32_inputs_at_tree_shape(tw):
    w = dataclass_replace(wl.scaled(wl.WORKLOADS[3], B=2, H=3), in_dtype="f32")
    run_and_check(tw, Case(w, seed=4, cfg_key=3), "c3 shape f32")


def dataclass_replace(w, **kw):
    import dataclasses
    return dataclasses.replace(w, **kw)


# ---------------------------------------------------------------------------
# Commit semantics, determinism, consecutive speculation steps
# ---------------------------------------------------------------------------
def test_empty_path_and_in_place_commit(tw):
    w = wl.scaled(wl.WORKLOADS[1], B=6, H=4)
    case = Case(w, seed=9, cfg_key=1)
    d = case.device()
    o, U = tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"])
    d["path_len"][:3] = 0
    S_copy = d["S0"].clone()
    S_out = tw.treewy_commit(d["S0"], U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"])
    tw.treewy_commit(S_copy, U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"], S_new=S_copy)
    torch.cuda.synchronize()
    assert torch.equal(S_out[:3], d["S0"][:3])            # nothing accepted: S0 bit for bit
    assert torch.equal(S_copy, S_out)                     # in place == out of place


def test_commit_reads_out_node_output(tw):
    """(S_a) q_a reproduces o_a (eq. 1 + eq. 3), on the device."""
    w = dataclass_replace(wl.scaled(wl.WORKLOADS[2], B=4, H=3), in_dtype="f32")
    case = Case(w, seed=10, cfg_key=2)
    d = case.device()
    o, U = tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"])
    S_new = tw.treewy_commit(d["S0"], U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"])
    torch.cuda.synchronize()
    for b in range(w.B):
        L = int(case.x["path_len"][b])
        if L == 0:
            continue
        a = int(case.x["path"][b, L - 1])
        got = (S_new[b].double() @ d["q"][b, :, a].double().unsqueeze(-1)).squeeze(-1)
        want = o[b, :, a].double()
        assert float((got - want).abs().max() / want.abs().max()) < 1e-4


def test_deterministic(tw):
    w = wl.scaled(wl.WORKLOADS[3], B=4, H=4)
    case = Case(w, seed=11, cfg_key=3)
    d = case.device()
    outs = []
    for _ in range(2):
        o, U = tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"])
        S = tw.treewy_commit(d["S0"], U, d["k"], d["alpha"], d["path"], d["path_len"])
        outs.append((o, U, S))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_two_steps_equal_one_longer_chain(tw):
    """Verify+commit a chain of 8, then verify the next 8 from the committed
    state: matches the oracle's chain of 16 (committed state = next S0)."""
    w16 = wl.Workload("chain16", 2, 3, 16, 128, 128, "bf16", "chain", 16, (1,), (0.85, 0.999),
                      (0.05, 0.95), 16, "chain_depth_0_to_N")
    case = Case(w16, seed=12, cfg_key=600)
    o_ref, _, _ = case.oracle()
    d = case.device()
    first, second = slice(0, 8), slice(8, 16)
    par8 = torch.from_numpy(np.tile(wl.chain_tree(8), (2, 1))).to(DEV)
    path = torch.from_numpy(np.tile(np.arange(8, dtype=np.int32), (2, 1))).to(DEV)
    plen = torch.full((2,), 8, dtype=torch.int32, device=DEV)
    sub = {n: d[n][:, :, first].contiguous() for n in ("q", "k", "v", "alpha", "beta")}
    _, U1 = tw.treewy_verify(d["S0"], sub["q"], sub["k"], sub["v"], sub["alpha"], sub["beta"], par8)
    S1 = tw.treewy_commit(d["S0"], U1, sub["k"], sub["alpha"], path, plen, parent=par8)
    sub = {n: d[n][:, :, second].contiguous() for n in ("q", "k", "v", "alpha", "beta")}
    o2, _ = tw.treewy_verify(S1, sub["q"], sub["k"], sub["v"], sub["alpha"], sub["beta"], par8)
    torch.cuda.synchronize()
    got = units_of(o2, wl.scaled(w16, N=8), case.check)
    assert_close("second step o", got, o_ref[:, 8:16], TOL["bf16"])


# ---------------------------------------------------------------------------
# Tree and path bookkeeping: bit exact
# ---------------------------------------------------------------------------
def test_path_from_node_bit_exact(tw):
    rng = np.random.default_rng(13)
    B, N, L_max = 300, 64, 10
    parent = np.stack([wl.random_tree(rng, N, 8, (4, 4, 2)) for _ in range(B)])
    accepted = rng.integers(-1, N, size=B).astype(np.int32)
    accepted[:5] = [-1, 0, 63, 5, 7]
    path, plen = tw.treewy_path_from_node(torch.from_numpy(parent).to(DEV), torch.from_numpy(accepted).to(DEV),
                                          L_max)
    path, plen = path.cpu().numpy(), plen.cpu().numpy()
    for b in range(B):
        want = [] if accepted[b] < 0 else wl.ancestors_and_self(parent[b], int(accepted[b]))
        assert plen[b] == len(want)
        assert list(path[b, :plen[b]]) == want and np.all(path[b, plen[b]:] == -1)


def test_path_too_long_and_bad_nodes_flagged(tw):
    parent = torch.from_numpy(np.tile(wl.chain_tree(12), (4, 1))).to(DEV)
    accepted = torch.tensor([11, 3, 12, -2], dtype=torch.int32, device=DEV)
    err = torch.zeros(4, dtype=torch.int32, device=DEV)
    path, plen = tw.treewy_path_from_node(parent, accepted, 8, err=err)
    assert plen.tolist() == [0, 4, 0, 0]
    assert err.tolist() == [2, 0, 2, 2]
    assert path[1, :4].tolist() == [0, 1, 2, 3]


def test_bad_parent_and_bad_path_flags(tw):
    w = wl.scaled(wl.WORKLOADS[2], B=4, H=2)
    case = Case(w, seed=14, cfg_key=2)
    d = case.device()
    d["parent"][1, 5] = 9        # not an earlier node
    d["parent"][2, 3] = -7
    err = torch.zeros(4, dtype=torch.int32, device=DEV)
    o, U = tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], err=err)
    torch.cuda.synchronize()
    assert err.tolist() == [0, 1, 1, 0]
    assert torch.isfinite(o.float()).all() and torch.isfinite(U).all()
    err.zero_()
    good = wl.make_inputs(w, seed=14, cfg_key=2)["parent"]
    d["parent"] = torch.from_numpy(good).to(DEV)
    d["path"][0, 0] = 40         # out of range
    d["path_len"][3] = 99        # longer than L_max
    S_new = tw.treewy_commit(d["S0"], U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"], err=err)
    torch.cuda.synchronize()
    assert err.tolist()[0] == 2 and err.tolist()[3] == 2
    assert torch.equal(S_new[0], d["S0"][0]) and torch.equal(S_new[3], d["S0"][3])


def test_empty_draft_and_empty_batch(tw):
    S0 = torch.randn(2, 3, 128, 128, device=DEV)
    z = torch.empty(2, 3, 0, 128, device=DEV, dtype=torch.bfloat16)
    za = torch.empty(2, 3, 0, device=DEV)
    par = torch.empty(2, 0, dtype=torch.int32, device=DEV)
    o, U = tw.treewy_verify(S0, z, z, z, za, za, par)
    assert o.shape == (2, 3, 0, 128)
    path = torch.empty(2, 0, dtype=torch.int32, device=DEV)
    plen = torch.zeros(2, dtype=torch.int32, device=DEV)
    S_new = tw.treewy_commit(S0, U, z, za, path, plen)
    torch.cuda.synchronize()
    assert torch.equal(S_new, S0)


# ---------------------------------------------------------------------------
# Snapshot baseline
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("cfg,dtype", [(0, "f32"), (2, "bf16"), (4, "bf16")])
def test_snapshot_baseline(tw, cfg, dtype):
    w = dataclass_replace(wl.scaled(wl.WORKLOADS[cfg], B=min(wl.WORKLOADS[cfg].B, 3),
                                    H=min(wl.WORKLOADS[cfg].H, 2)), in_dtype=dtype)
    case = Case(w, seed=15, cfg_key=cfg)
    say("[gpu] snapshot baseline: %s" % w.describe())
    d = case.device()
    o, snaps = tw.treewy_snapshot_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"])
    acc = torch.tensor([int(case.x["path"][b, case.x["path_len"][b] - 1]) if case.x["path_len"][b] else -1
                        for b in range(w.B)], dtype=torch.int32, device=DEV)
    S_new = tw.treewy_snapshot_commit(d["S0"], snaps, acc)
    torch.cuda.synchronize()
    o_ref, _, states, S_ref = case.oracle(states=True)
    tol = TOL[w.in_dtype]
    assert_close("snapshot o", units_of(o, w, case.check), o_ref, tol)
    got = units_of(snaps, w, case.check)
    for t in range(w.N):
        assert_close("snapshot S_%d" % t, got[:, t], states[:, t], tol)
    assert_close("snapshot commit", units_of(S_new, w, case.check), S_ref, tol)


def test_snapshot_baseline_full_size_sampled(tw):
    """The snapshot baseline at the launch the benchmark times (the 32-node
    stress tree, B = 256, H = 64: 32 GiB of snapshots), checked on 16 sampled
    units: every node's output and state, and the committed state."""
    w = wl.WORKLOADS[4]
    case = Case(w, seed=16, cfg_key=4, check_units=wl.sample_units(w, 16))
    say("[gpu] snapshot baseline, full size: %s" % w.describe())
    d = case.device()
    snaps = torch.empty((w.B, w.H, w.N, w.d_v, w.d_k), dtype=torch.float32, device=DEV)
    o, snaps = tw.treewy_snapshot_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"],
                                         snapshots=snaps)
    acc = torch.tensor([int(case.x["path"][b, case.x["path_len"][b] - 1]) if case.x["path_len"][b] else -1
                        for b in range(w.B)], dtype=torch.int32, device=DEV)
    S_new = tw.treewy_snapshot_commit(d["S0"], snaps, acc)
    torch.cuda.synchronize()
    sel = torch.from_numpy(case.check).to(DEV)
    got = snaps.reshape(w.units, w.N, w.d_v, w.d_k).index_select(0, sel).cpu().numpy()
    del snaps
    torch.cuda.empty_cache()
    o_ref, _, states, S_ref = case.oracle(states=True)
    tol = TOL[w.in_dtype]
    eo = assert_close("snapshot o", units_of(o, w, case.check), o_ref, tol)
    es = max(assert_close("snapshot S_%d" % t, got[:, t], states[:, t], tol) for t in range(w.N))
    ec = assert_close("snapshot commit", units_of(S_new, w, case.check), S_ref, tol)
    say("[gpu] snapshot full size: max rel err o %.2e states %.2e commit %.2e" % (eo, es, ec))

"""Trees of more than 64 nodes (walked in 64-node chunks) vs the float64
oracle, through the C ABI: verify (o, U) and commit over long paths, random
trees shallow and deep, chains, fixed-width trees, both input types and both
state types; then greedy acceptance and path extraction on such trees, bit
for bit against the plain-Python reference."""
import numpy as np
import pytest
import torch

import oracle
from oracle.acceptance import accept_greedy
from paper_2608_20961_amd import workload as wl
from tests.gpu_harness import DEV, TOL, Case, assert_close, say, units_of

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tw():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_20961_amd import treewy
    return treewy


def tree_workload(N, depth, dtype="bf16", B=2, H=3, caps=(4, 4, 2), accept="uniform_node"):
    tree = "chain" if depth == N and caps == (1,) else "tree"
    return wl.Workload("big", B, H, N, 128, 128, dtype, tree, depth, caps, (0.85, 0.999), (0.05, 0.95), 16,
                       accept)


def check(tw, case, label, state="f32"):
    w = case.w
    say("[gpu] %s: %s, %s state" % (label, w.describe(), state))
    d = case.device()
    S0 = d["S0"]
    if state == "bf16":
        S0 = S0.to(torch.bfloat16)
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    o, U = tw.treewy_verify(S0, d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], err=err)
    S_new = tw.treewy_commit(S0, U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"], err=err)
    torch.cuda.synchronize()
    assert int(err.abs().sum()) == 0
    o_ref, vt_ref, S_ref = case.oracle()
    tol = TOL[w.in_dtype]
    eo = assert_close(label + " o", units_of(o, w, case.check), o_ref, tol)
    eu = assert_close(label + " U", units_of(U, w, case.check), vt_ref, tol)
    es = assert_close(label + " S_new", units_of(S_new, w, case.check), S_ref, tol)
    say("[gpu] %s: max rel err o %.2e U %.2e S_new %.2e" % (label, eo, eu, es))


@pytest.mark.parametrize("N,depth", [(65, 8), (100, 8), (128, 16), (192, 40), (256, 12), (256, 96)])
def test_random_trees(tw, N, depth):
    check(tw, Case(tree_workload(N, depth), seed=N + depth, cfg_key=1000 + N), "tree N=%d depth %d" % (N, depth))


@pytest.mark.parametrize("N", [65, 130, 256])
def test_chains(tw, N):
    w = tree_workload(N, N, caps=(1,), accept="chain_depth_0_to_N")
    check(tw, Case(w, seed=N, cfg_key=1100 + N), "chain N=%d" % N)


@pytest.mark.parametrize("N,depth", [(96, 8), (200, 30)])
def test_fp32_inputs(tw, N, depth):
    check(tw, Case(tree_workload(N, depth, "f32"), seed=3, cfg_key=1200 + N), "f32 tree N=%d" % N)


@pytest.mark.parametrize("N,depth", [(129, 10), (256, 64)])
def test_bf16_state(tw, N, depth):
    case = Case(tree_workload(N, depth), seed=4, cfg_key=1300 + N)
    case.S0 = wl.round_to_bf16(case.S0)              # the state as stored: bf16 values
    check(tw, case, "bf16-state tree N=%d" % N, state="bf16")


@pytest.mark.parametrize("widths", [(4, 4, 4), (3, 3, 3, 3), (2, 2, 2, 2, 2, 2, 2)])
def test_fixed_width_trees(tw, widths):
    par = wl.width_tree(widths)
    N = len(par)
    w = tree_workload(N, len(widths), B=3, H=2, caps=(9,))
    x = wl.make_inputs(w, seed=6, cfg_key=1400 + N)
    x["parent"] = np.tile(par, (w.B, 1))
    rng = np.random.default_rng(N)
    for b in range(w.B):                               # a node to accept, and its root path
        nodes = wl.ancestors_and_self(par, int(rng.integers(N)))
        x["path"][b] = -1
        x["path"][b, :len(nodes)] = nodes
        x["path_len"][b] = len(nodes)
    check(tw, Case(w, seed=6, cfg_key=1400 + N, inputs=x), "widths %s (N=%d)" % (widths, N))


def test_coupling_groups(tw):
    """128-node trees whose second chunk descends from exactly m nodes of the
    first (m = 40, 32, 33 across the sequences: a chain of m nodes, the rest
    of the first chunk leaves on it, the second chunk hanging off all m), so
    the coupling gathers one full group, one and a half, and a second group
    of a single column."""
    N = 128
    w = tree_workload(N, 42, B=3, H=2, caps=(9,))
    x = wl.make_inputs(w, seed=8, cfg_key=1500)
    rng = np.random.default_rng(15)
    for b, m in enumerate((40, 32, 33)):
        par = np.empty(N, dtype=np.int32)
        par[:m] = np.arange(-1, m - 1)
        par[m:64] = (np.arange(m, 64) - m) % m
        par[64:] = (np.arange(64, N) - 64) % m
        x["parent"][b] = par
        nodes = wl.ancestors_and_self(par, int(rng.integers(64, N)))
        x["path"][b] = -1
        x["path"][b, :len(nodes)] = nodes
        x["path_len"][b] = len(nodes)
    check(tw, Case(w, seed=8, cfg_key=1500, inputs=x), "coupling groups (m = 40, 32, 33)")


def mixed_solve_tree(rng):
    """A 256-node tree whose four chunks take different solves of their
    diagonal block: a chain of 30 with leaves (dense sweep), segments of 8
    hanging off earlier nodes (registers), segments of 14 (B read one ancestor
    ahead), a chain of 40 (dense sweep again)."""
    N = 256
    par = np.empty(N, dtype=np.int32)
    par[:30] = np.arange(-1, 29)
    par[30:64] = rng.integers(0, 21, 34)
    for i in range(64):
        par[64 + i] = rng.integers(0, 64) if i % 8 == 0 else 64 + i - 1
        par[128 + i] = rng.integers(0, 128) if i % 14 == 0 else 128 + i - 1
        par[192 + i] = (rng.integers(0, 192) if i == 0 else 192 + i - 1) if i < 40 else 192 + rng.integers(0, 10)
    assert wl.is_topological(par)
    return par


def test_chunks_with_different_solves(tw):
    """One unit's chunks take the dense sweep, the register gather, the
    medium solve and the sweep again, in one launch."""
    N = 256
    w = tree_workload(N, 120, B=2, H=3, caps=(9,))
    x = wl.make_inputs(w, seed=9, cfg_key=1600)
    rng = np.random.default_rng(16)
    for b in range(w.B):
        par = mixed_solve_tree(rng)
        x["parent"][b] = par
        nodes = wl.ancestors_and_self(par, int(rng.integers(192, N)))
        assert len(nodes) <= x["path"].shape[1]
        x["path"][b] = -1
        x["path"][b, :len(nodes)] = nodes
        x["path_len"][b] = len(nodes)
    check(tw, Case(w, seed=9, cfg_key=1600, inputs=x), "chunks with different solves")


def test_full_size_sampled(tw):
    """The 397B layer shape with 128-node trees: the launch the benchmark times."""
    w = wl.BIG_TREE
    check(tw, Case(w, seed=0, cfg_key=1500, check_units=wl.sample_units(w, 16)), "397B-tree128 full")


def test_full_size_sampled_bf16_state(tw):
    """The same launch with a bf16 state, which stays in registers from the
    first 64-node chunk to the second instead of being read again."""
    w = wl.BIG_TREE
    case = Case(w, seed=1, cfg_key=1510, check_units=wl.sample_units(w, 16))
    case.S0 = wl.round_to_bf16(case.S0)              # the state as stored: bf16 values
    check(tw, case, "397B-tree128 full", state="bf16")


def test_long_path_commit_full_chain(tw):
    """Commit of every node of a 256-chain (L_max = 256, four staging passes)."""
    N = 256
    w = tree_workload(N, N, B=2, H=2, caps=(1,), accept="chain_depth_0_to_N")
    x = wl.make_inputs(w, seed=8, cfg_key=1600)
    x["path"][:] = np.arange(N, dtype=np.int32)
    x["path_len"][:] = N
    check(tw, Case(w, seed=8, cfg_key=1600, inputs=x), "chain 256, full path")


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


@pytest.mark.parametrize("N", [65, 200, 256])
def test_accept_and_paths(tw, N):
    rng = np.random.default_rng(N)
    B = 64
    parents = np.stack([wl.random_tree(rng, N, int(rng.integers(1, N + 1)), (N,)) for _ in range(B)])
    tok = wl.acceptance_tokens(parents, seed=N, vocab=2, plant=True)
    for L_max in (16, N):
        err = torch.zeros(B, dtype=torch.int32, device=DEV)
        path, plen, bonus = tw.treewy_accept_greedy(i32(parents), i32(tok["draft"]), i32(tok["target"]),
                                                    i32(tok["root"]), L_max, err=err)
        torch.cuda.synchronize()
        r_path, r_len, r_bonus = accept_greedy(parents, tok["draft"], tok["target"], tok["root"], L_max)
        over = r_len < 0
        assert np.array_equal(bonus.cpu().numpy(), r_bonus)
        assert np.array_equal(plen.cpu().numpy(), np.where(over, 0, r_len))
        assert np.array_equal(path.cpu().numpy(), r_path)
        assert np.array_equal(err.cpu().numpy() & 2, np.where(over, 2, 0))
        say("[gpu] accept N=%d L_max=%d: longest %d" % (N, L_max, int(r_len.max())))
    # the root path of the deepest node of every tree, against the tree walked on the host
    depth = np.stack([wl.tree_depths(p) for p in parents])
    acc = depth.argmax(axis=1).astype(np.int32)
    path, plen = tw.treewy_path_from_node(i32(parents), i32(acc), N)
    torch.cuda.synchronize()
    for b in range(B):
        nodes = wl.ancestors_and_self(parents[b], int(acc[b]))
        assert plen[b].item() == len(nodes)
        assert path[b, :len(nodes)].cpu().tolist() == nodes


def test_bad_parent_in_a_later_chunk_counts_as_root(tw):
    """A parent outside [-1, t-1] in the second chunk is flagged and treated as -1
    (the header's contract): the outputs equal the oracle's on the repaired tree."""
    N = 150
    w = tree_workload(N, 20, B=2, H=2)
    x = wl.make_inputs(w, seed=11, cfg_key=1800)
    bad = x["parent"].copy()
    bad[1, 100] = 120                                  # a later node: invalid
    bad[1, 140] = -5                                   # below -1: invalid
    repaired = bad.copy()
    repaired[1, 100] = repaired[1, 140] = -1
    x["parent"] = repaired
    x["path_len"][:] = 0                               # (paths drawn on the original tree)
    case = Case(w, seed=11, cfg_key=1800, inputs=x)
    d = case.device()
    d["parent"] = torch.from_numpy(bad).to(DEV)
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    o, U = tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], err=err)
    torch.cuda.synchronize()
    assert err.tolist() == [0, 1]
    o_ref, vt_ref, _ = case.oracle()
    assert_close("o", units_of(o, w, case.check), o_ref, TOL["bf16"])
    assert_close("U", units_of(U, w, case.check), vt_ref, TOL["bf16"])


def test_long_path_broken_deep_inside(tw):
    """A 200-entry path whose entry 150 skips a node is flagged; the state is kept."""
    N = 200
    w = tree_workload(N, N, B=2, H=2, caps=(1,), accept="chain_depth_0_to_N")
    case = Case(w, seed=12, cfg_key=1900)
    d = case.device()
    _, U = tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"])
    path = torch.arange(N, dtype=torch.int32, device=DEV).repeat(w.B, 1)
    path[1, 150:] += 1                                 # 149 -> 151: not a child
    path[1, N - 1] = -1
    plen = torch.tensor([N, N - 1], dtype=torch.int32, device=DEV)
    err = torch.zeros(w.B, dtype=torch.int32, device=DEV)
    S_new = tw.treewy_commit(d["S0"], U, d["k"], d["alpha"], path, plen, parent=d["parent"], err=err)
    torch.cuda.synchronize()
    assert err.tolist() == [0, 2]
    assert torch.equal(S_new[1], d["S0"][1])
    S_ref = oracle.commit(case.S0[:w.H], case.unit_view("k")[:w.H], case.unit_view("v")[:w.H],
                          case.unit_view("alpha")[:w.H], case.unit_view("beta")[:w.H],
                          np.repeat(case.x["parent"][:1], w.H, axis=0), np.repeat(path[:1].cpu().numpy(), w.H, axis=0),
                          np.full(w.H, N))
    assert_close("S_new", units_of(S_new, w, np.arange(w.H)), S_ref, TOL["bf16"])


def test_fp32_inputs_many_units_per_workgroup(tw):
    """fp32 inputs run one workgroup per CU: 1024 units make each workgroup walk
    several units (the per-unit ancestor tables in LDS are rebuilt each time)."""
    w = tree_workload(100, 12, "f32", B=16, H=64)
    check(tw, Case(w, seed=13, cfg_key=2000, check_units=wl.sample_units(w, 10)), "f32 tree N=100, 1024 units")

"""treewy_accept_greedy on the GPU vs the plain-Python reference, bit for bit
(paths, lengths, bonus tokens, flags), then the accepted paths fed straight
into treewy_commit_verify."""
import numpy as np
import pytest
import torch

import oracle
from oracle.acceptance import accept_greedy
from paper_2608_20961_amd import workload as wl
from tests.gpu_harness import DEV, TOL, assert_close, say, units_of, warm_state

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tw():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_20961_amd import treewy
    return treewy


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def run(tw, parents, tok, L_max):
    err = torch.zeros(parents.shape[0], dtype=torch.int32, device=DEV)
    path, plen, bonus = tw.treewy_accept_greedy(i32(parents), i32(tok["draft"]), i32(tok["target"]),
                                                i32(tok["root"]), L_max, err=err)
    torch.cuda.synchronize()
    return path.cpu().numpy(), plen.cpu().numpy(), bonus.cpu().numpy(), err.cpu().numpy()


def check(tw, parents, tok, L_max, label):
    path, plen, bonus, err = run(tw, parents, tok, L_max)
    r_path, r_len, r_bonus = accept_greedy(parents, tok["draft"], tok["target"], tok["root"], L_max)
    over = r_len < 0
    assert np.array_equal(bonus, r_bonus), label
    assert np.array_equal(plen, np.where(over, 0, r_len)), label
    assert np.array_equal(path, r_path), label
    assert np.array_equal(err & 2, np.where(over, 2, 0)), label
    say("[gpu] accept %s: mean accepted %.2f, max %d" % (label, float(r_len[~over].mean()) if (~over).any() else 0,
                                                       int(r_len.max())))
    return path, plen, bonus


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
@pytest.mark.parametrize("vocab,plant", [(2, False), (4, True), (50, True)])
def test_workload_trees(tw, cfg, vocab, plant):
    w = wl.WORKLOADS[cfg]
    parents = wl.make_inputs(wl.scaled(w, H=1), seed=cfg, cfg_key=cfg)["parent"]
    tok = wl.acceptance_tokens(parents, seed=cfg, vocab=vocab, plant=plant)
    check(tw, parents, tok, w.max_depth, "c%d vocab %d" % (cfg, vocab))


@pytest.mark.parametrize("N", [1, 7, 33, 64])
def test_random_trees_ties_and_overflow(tw, N):
    rng = np.random.default_rng(N)
    B = 96
    parents = np.stack([wl.random_tree(rng, N, int(rng.integers(1, N + 1)), (64,)) for _ in range(B)])
    tok = wl.acceptance_tokens(parents, seed=N, vocab=2, plant=True)
    check(tw, parents, tok, L_max=min(N, 8), label="N=%d" % N)   # deep chains overflow L_max = 8
    check(tw, parents, tok, L_max=N, label="N=%d full" % N)


def test_bad_parent_and_empty(tw):
    parents = np.array([[-1, 5, 0, 1], [-1, 0, 1, 2]], dtype=np.int32)   # parent[0][1] = 5 is invalid
    tok = dict(draft=np.array([[1, 2, 2, 3], [1, 2, 3, 4]]), target=np.array([[2, 3, 3, 9], [2, 3, 4, 5]]),
               root=np.array([2, 7]))
    path, plen, bonus, err = run(tw, parents, tok, 4)
    r_path, r_len, r_bonus = accept_greedy(parents, tok["draft"], tok["target"], tok["root"], 4)
    assert np.array_equal(path, r_path) and np.array_equal(plen, r_len) and np.array_equal(bonus, r_bonus)
    assert err.tolist() == [1, 0]
    assert plen.tolist() == [2, 0] and bonus.tolist() == [9, 7]          # 1 (as a root child) then 3
    empty = np.zeros((3, 0), dtype=np.int32)
    path, plen, bonus, err = run(tw, empty, dict(draft=empty, target=empty, root=np.array([4, 5, 6])), 2)
    assert plen.tolist() == [0, 0, 0] and bonus.tolist() == [4, 5, 6] and (path == -1).all()


def test_accepted_paths_feed_the_fused_commit(tw):
    """verify -> accept on the device -> commit inside the next verify, vs the
    oracle committing the reference's accepted paths."""
    w = wl.scaled(wl.WORKLOADS[3], B=6, H=4)
    x = wl.make_inputs(w, seed=5, cfg_key=503)
    xn = wl.make_inputs(w, seed=6, cfg_key=504)
    units = np.arange(w.units)
    S_old = warm_state(w, units, 5, 505)
    tok = wl.acceptance_tokens(x["parent"], seed=5, vocab=3, plant=True)
    L_max = w.max_depth
    r_path, r_len, _ = accept_greedy(x["parent"], tok["draft"], tok["target"], tok["root"], L_max)
    assert (r_len >= 0).all()
    dt = torch.bfloat16
    dev = lambda a, d=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(d)
    S0 = dev(S_old.reshape(w.B, w.H, 128, 128))
    k, al, par = dev(x["k"], dt), dev(x["alpha"]), i32(x["parent"])
    _, U = tw.treewy_verify(S0, dev(x["q"], dt), k, dev(x["v"], dt), al, dev(x["beta"]), par)
    path, plen, _ = tw.treewy_accept_greedy(par, i32(tok["draft"]), i32(tok["target"]), i32(tok["root"]), L_max)
    S_new, o, Un = tw.treewy_commit_verify(S0, U, k, al, path, plen, dev(xn["q"], dt), dev(xn["k"], dt),
                                           dev(xn["v"], dt), dev(xn["alpha"]), dev(xn["beta"]), i32(xn["parent"]),
                                           parent_prev=par)
    torch.cuda.synchronize()
    uv = lambda a: a.reshape(w.units, *a.shape[2:])
    H = w.H
    S_ref = oracle.commit(S_old, uv(x["k"]), uv(x["v"]), uv(x["alpha"]), uv(x["beta"]),
                          np.repeat(x["parent"], H, axis=0), np.repeat(r_path, H, axis=0), np.repeat(r_len, H, axis=0))
    o_ref, vt_ref = oracle.verify(S_ref, uv(xn["q"]), uv(xn["k"]), uv(xn["v"]), uv(xn["alpha"]), uv(xn["beta"]),
                                  np.repeat(xn["parent"], H, axis=0))
    tol = TOL["bf16"]
    assert_close("S_new", units_of(S_new, w, units), S_ref, tol)
    assert_close("o", units_of(o, w, units), o_ref, tol)
    assert_close("U", units_of(Un, w, units), vt_ref, tol)


def test_path_longer_than_the_tree(tw):
    """L_max above N (and above one word of nodes): entries past the path are -1."""
    rng = np.random.default_rng(77)
    for N, L_max in ((40, 130), (100, 256)):
        parents = np.stack([wl.random_tree(rng, N, int(rng.integers(1, N + 1)), (N,)) for _ in range(8)])
        tok = wl.acceptance_tokens(parents, seed=N, vocab=2, plant=True)
        check(tw, parents, tok, L_max, "N=%d L_max=%d" % (N, L_max))

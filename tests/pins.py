"""Checks that pin the oracle to what the paper and the mathematics fix.

Each pin takes an oracle instance and raises AssertionError when it fails, so
that the same pins can be run against a deliberately broken oracle build to
show they catch plausible mistakes.  None of them re-types the oracle's own
loop: they use a closed form, a special case with a known answer, exact
rational arithmetic, the literal matrix form of eq. 1, or an invariant.
"""
import itertools
from fractions import Fraction

import numpy as np

from paper_2608_20961_amd import workload as wl
from tests import closed_form as cf


def rel(x, ref):
    x, ref = np.asarray(x, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(x - ref)) / max(float(np.max(np.abs(ref))), 1e-300)) if ref.size else 0.0


def _unit_inputs(rng, N, d, alpha_range=(0.85, 0.999), beta_range=(0.05, 0.95), parent=None, warm=8):
    k = rng.standard_normal((N, d)); k /= np.linalg.norm(k, axis=1, keepdims=True)
    q = rng.standard_normal((N, d)); q /= np.linalg.norm(q, axis=1, keepdims=True)
    v = rng.standard_normal((N, d))
    alpha = rng.uniform(*alpha_range, N)
    beta = rng.uniform(*beta_range, N)
    S0 = rng.standard_normal((d, d)) * 0.3
    par = wl.chain_tree(N) if parent is None else np.asarray(parent, dtype=np.int32)
    return S0, q, k, v, alpha, beta, par


def _literal_step(S, k, v, alpha, beta):
    """eq. 1 with the transition matrix formed explicitly."""
    d = len(k)
    return alpha * S @ (np.eye(d) - beta * np.outer(k, k)) + beta * np.outer(v, k)


# --------------------------------------------------------------------------
def pin_scalar_worked_example(orc):
    """d_k = d_v = 1 worked by hand from eq. 1 and the key rewrite.

    alpha = beta = 1/2, k = q = 1, S0 = 1, v = (2, 4, 8); node 1 is a child of
    node 0, node 2 hangs off S0.  eq. 1 reduces to s_t = s_p/4 + v_t/2:
      s_0 = 1/4 + 1 = 5/4,  s_1 = 5/16 + 2 = 37/16,  s_2 = 1/4 + 4 = 17/4;
    o_t = s_t (q = 1); vt_t = (v_t - s_p/2)/2 = 3/4, 27/16, 15/4.
    """
    one = np.ones((1, 3, 1))
    o, vt = orc.verify(np.ones((1, 1, 1)), one, one, np.array([[[2.0], [4.0], [8.0]]]),
                       np.full((1, 3), 0.5), np.full((1, 3), 0.5), np.array([[-1, 0, -1]]))
    assert np.array_equal(o.ravel(), [5 / 4, 37 / 16, 17 / 4]), o.ravel()
    assert np.array_equal(vt.ravel(), [3 / 4, 27 / 16, 15 / 4]), vt.ravel()
    S = orc.commit(np.ones((1, 1, 1)), one, np.array([[[2.0], [4.0], [8.0]]]), np.full((1, 3), 0.5),
                   np.full((1, 3), 0.5), np.array([[-1, 0, -1]]), np.array([[0, 1]]), np.array([2]))
    assert S.ravel()[0] == 37 / 16


def pin_exact_rational(orc):
    """A d = 2 tree computed in exact rational arithmetic from eq. 1."""
    F = Fraction
    S0 = [[F(1, 2), F(-1, 4)], [F(3, 8), F(1)]]
    ks = [(F(3, 5), F(4, 5)), (F(0), F(1)), (F(4, 5), F(-3, 5)), (F(1), F(0))]
    qs = [(F(1), F(0)), (F(3, 5), F(-4, 5)), (F(0), F(1)), (F(-4, 5), F(3, 5))]
    vs = [(F(2), F(-1)), (F(1, 2), F(3)), (F(-1), F(1, 4)), (F(5, 4), F(-2))]
    al = [F(7, 8), F(1, 2), F(3, 4), F(9, 10)]
    be = [F(1, 2), F(1, 4), F(3, 4), F(1, 3)]
    parent = [-1, 0, 0, -1]

    def mat_vec(S, x):
        return [S[r][0] * x[0] + S[r][1] * x[1] for r in range(2)]

    states, o_ref, vt_ref = [], [], []
    for t in range(4):
        P = S0 if parent[t] == -1 else states[parent[t]]
        Pk = mat_vec(P, ks[t])
        vt_ref.append([be[t] * (vs[t][r] - al[t] * Pk[r]) for r in range(2)])
        M = [[(1 if r == c else 0) - be[t] * ks[t][r] * ks[t][c] for c in range(2)] for r in range(2)]
        S = [[al[t] * sum(P[r][j] * M[j][c] for j in range(2)) + be[t] * vs[t][r] * ks[t][c]
              for c in range(2)] for r in range(2)]
        states.append(S)
        o_ref.append(mat_vec(S, qs[t]))
    f = lambda x: np.array(x, dtype=np.float64)[None]
    o, vt = orc.verify(f(S0), f(qs), f(ks), f(vs), f(al), f(be), np.array([parent]))
    assert rel(o[0], f(o_ref)[0]) < 1e-15
    assert rel(vt[0], f(vt_ref)[0]) < 1e-15


def pin_chain_literal(orc, d=16, N=9, seed=1):
    """A single-branch tree equals the plain chain recurrence in matrix form."""
    rng = np.random.default_rng(seed)
    S0, q, k, v, alpha, beta, par = _unit_inputs(rng, N, d)
    o, vt = orc.verify(S0[None], q[None], k[None], v[None], alpha[None], beta[None], par[None])
    S = S0
    for t in range(N):
        vt_ref = beta[t] * (v[t] - alpha[t] * S @ k[t])
        S = _literal_step(S, k[t], v[t], alpha[t], beta[t])
        assert rel(o[0, t], S @ q[t]) < 1e-13
        assert rel(vt[0, t], vt_ref) < 1e-13
    Sc = orc.commit(S0[None], k[None], v[None], alpha[None], beta[None], par[None],
                    np.arange(N)[None], np.array([N]))
    assert rel(Sc[0], S) < 1e-13


def pin_beta_zero(orc, d=16, N=12, seed=2):
    """beta = 0: no write, pure decay.  vt = 0, o_t = g_t S0 q_t, S_a = g_a S0."""
    rng = np.random.default_rng(seed)
    par = wl.random_tree(rng, N, 4, (3,))
    S0, q, k, v, alpha, _, _ = _unit_inputs(rng, N, d, parent=par)
    beta = np.zeros(N)
    o, vt = orc.verify(S0[None], q[None], k[None], v[None], alpha[None], beta[None], par[None])
    assert np.all(vt == 0.0)
    for t in range(N):
        g = np.prod([alpha[i] for i in wl.ancestors_and_self(par, t)])
        assert rel(o[0, t], g * (S0 @ q[t])) < 1e-14
    a = N - 1
    path = wl.ancestors_and_self(par, a)
    Sc = orc.commit(S0[None], k[None], v[None], alpha[None], beta[None], par[None],
                    np.array([path]), np.array([len(path)]))
    g = np.prod([alpha[i] for i in path])
    assert rel(Sc[0], g * S0) < 1e-14


def pin_overwrite(orc, d=16, seed=3):
    """alpha = beta = 1 with orthonormal keys: erase-then-write is exact.

    Every node's pseudo-value is v_t - S0 k_t (no ancestor write overlaps k_t),
    the committed state reads back S_a k_j = v_j on its path, and
    S_a = S0 (I - sum k k^T) + sum v k^T over the path."""
    rng = np.random.default_rng(seed)
    N = 7
    par = np.array([-1, 0, 1, 1, -1, 4, 5], dtype=np.int32)
    Qm, _ = np.linalg.qr(rng.standard_normal((d, d)))
    k = Qm[:N]
    q = rng.standard_normal((N, d))
    v = rng.standard_normal((N, d))
    S0 = rng.standard_normal((d, d))
    one = np.ones(N)
    o, vt = orc.verify(S0[None], q[None], k[None], v[None], one[None], one[None], par[None])
    for t in range(N):
        assert rel(vt[0, t], v[t] - S0 @ k[t]) < 1e-13
        path = wl.ancestors_and_self(par, t)
        S_ref = S0 @ (np.eye(d) - sum(np.outer(k[j], k[j]) for j in path)) + sum(np.outer(v[j], k[j]) for j in path)
        assert rel(o[0, t], S_ref @ q[t]) < 1e-13
    path = wl.ancestors_and_self(par, 3)
    Sc = orc.commit(S0[None], k[None], v[None], one[None], one[None], par[None],
                    np.array([path]), np.array([len(path)]))[0]
    for j in path:
        assert rel(Sc @ k[j], v[j]) < 1e-13


def all_parent_arrays(N):
    return itertools.product(*[range(-1, t) for t in range(N)])


def pin_brute_force_small_trees(orc, d=6, seed=4):
    """Every tree of <= 4 nodes: each node recomputed from S0 along its own path."""
    rng = np.random.default_rng(seed)
    count = 0
    for N in range(1, 5):
        for par in all_parent_arrays(N):
            par = np.array(par, dtype=np.int32)
            S0, q, k, v, alpha, beta, _ = _unit_inputs(rng, N, d, parent=par)
            o, vt = orc.verify(S0[None], q[None], k[None], v[None], alpha[None], beta[None], par[None])
            for t in range(N):
                path = wl.ancestors_and_self(par, t)
                S = S0
                for j in path[:-1]:
                    S = _literal_step(S, k[j], v[j], alpha[j], beta[j])
                vt_ref = beta[t] * (v[t] - alpha[t] * S @ k[t])
                S = _literal_step(S, k[t], v[t], alpha[t], beta[t])
                assert rel(o[0, t], S @ q[t]) < 1e-13, (par, t)
                assert rel(vt[0, t], vt_ref) < 1e-13, (par, t)
                Sc = orc.commit(S0[None], k[None], v[None], alpha[None], beta[None], par[None],
                                np.array([path]), np.array([len(path)]))
                assert rel(Sc[0], S) < 1e-13, (par, t)
                count += 1
    assert count == 1 * 1 + 2 * 2 + 6 * 3 + 24 * 4


def pin_closed_form(orc, cases=((0, 2, 1, 4), (2, 2, 2, 16), (3, 1, 2, 64), (4, 2, 1, 32), (3, 1, 1, 200),
                                (1, 1, 1, 150)), tol=1e-12):
    """Oracle == the paper's closed form (eq. 2 solve, read-out, eq. 3), up to
    trees and chains past one 64-node chunk."""
    for cfg, B, H, N in cases:
        w = wl.scaled(wl.WORKLOADS[cfg], B=B, H=H, N=N)
        x = wl.make_inputs(w, seed=11)
        rng = np.random.default_rng(cfg)
        S0 = rng.standard_normal((B * H, w.d_v, w.d_k)) * 0.2
        U = B * H
        par_u = np.repeat(x["parent"], H, axis=0)
        args = [x[n].reshape(U, N, -1) for n in ("q", "k", "v")]
        al, be = x["alpha"].reshape(U, N), x["beta"].reshape(U, N)
        o, vt = orc.verify(S0, *args, al, be, par_u)
        path = np.repeat(x["path"], H, axis=0)
        plen = np.repeat(x["path_len"], H, axis=0)
        Sc = orc.commit(S0, args[1], args[2], al, be, par_u, path, plen)
        for u in range(U):
            O_ref, Vt_ref = cf.solve_unit(S0[u], args[0][u], args[1][u], args[2][u], al[u], be[u], par_u[u])
            assert rel(vt[u], Vt_ref) < tol, (cfg, u, rel(vt[u], Vt_ref))
            assert rel(o[u], O_ref) < tol, (cfg, u, rel(o[u], O_ref))
            S_ref = cf.commit_unit(S0[u], args[1][u], al[u], par_u[u], Vt_ref, list(path[u, :plen[u]]))
            assert rel(Sc[u], S_ref) < tol, (cfg, u)


def pin_closed_form_fp32(orc, cases=((0, 2, 1, 4), (2, 2, 2, 16), (3, 1, 2, 64), (4, 2, 1, 32),
                                     (3, 1, 1, 200), (1, 1, 1, 150)), tol=1e-6):
    """The closed form evaluated entirely in float32 against the float64 oracle
    on the same fp32 inputs: the paper reports about 1e-7 between the two in
    single precision (Implementation).  The bar is 1e-6, normwise per unit."""
    for cfg, B, H, N in cases:
        w = wl.scaled(wl.WORKLOADS[cfg], B=B, H=H, N=N)
        x = wl.make_inputs(w, seed=12)
        rng = np.random.default_rng(100 + cfg)
        S0 = (rng.standard_normal((B * H, w.d_v, w.d_k)) * 0.2).astype(np.float32)
        U = B * H
        par_u = np.repeat(x["parent"], H, axis=0)
        args = [x[n].reshape(U, N, -1) for n in ("q", "k", "v")]
        al, be = x["alpha"].reshape(U, N), x["beta"].reshape(U, N)
        o, vt = orc.verify(S0, *args, al, be, par_u)
        path = np.repeat(x["path"], H, axis=0)
        plen = np.repeat(x["path_len"], H, axis=0)
        Sc = orc.commit(S0, args[1], args[2], al, be, par_u, path, plen)
        for u in range(U):
            O32, V32 = cf.solve_unit(S0[u], args[0][u], args[1][u], args[2][u], al[u], be[u], par_u[u],
                                     dtype=np.float32)
            assert rel(V32, vt[u]) < tol, (cfg, u, rel(V32, vt[u]))
            assert rel(O32, o[u]) < tol, (cfg, u, rel(O32, o[u]))
            S32 = cf.commit_unit(S0[u], args[1][u], al[u], par_u[u], V32, list(path[u, :plen[u]]),
                                 dtype=np.float32)
            assert rel(S32, Sc[u]) < tol, (cfg, u, rel(S32, Sc[u]))


def pin_closed_form_fast_decay(orc, tol=1e-12):
    """Fast-forgetting gates, alpha in (0.02, 0.5): the cumulative decays of a
    64-node chain and of a 256-node tree of depth 96 fall far below the
    smallest float32, and the oracle still equals the paper's closed form
    (eq. 2 solve, read-out, eq. 3) in float64."""
    for N, depth, caps, seed in ((64, 64, (1,), 21), (256, 96, (4, 4, 2), 22)):
        tree = "chain" if caps == (1,) else "tree"
        w = wl.Workload("fast-decay", 1, 2, N, 32, 32, "f32", tree, depth, caps, (0.02, 0.5), (0.05, 0.95),
                        8, "chain_depth_0_to_N" if tree == "chain" else "uniform_node")
        x = wl.make_inputs(w, seed=seed)
        rng = np.random.default_rng(seed)
        U = w.units
        S0 = rng.standard_normal((U, w.d_v, w.d_k)) * 0.2
        par_u = np.repeat(x["parent"], w.H, axis=0)
        args = [x[n].reshape(U, N, -1) for n in ("q", "k", "v")]
        al, be = x["alpha"].reshape(U, N), x["beta"].reshape(U, N)
        g = cf.cumulative_decay(par_u[0], al[0].astype(np.float64))
        assert g.min() < 1e-39, "the draw must reach where 1 / g overflows float32"
        o, vt = orc.verify(S0, *args, al, be, par_u)
        path = np.repeat(x["path"], w.H, axis=0)
        plen = np.repeat(x["path_len"], w.H, axis=0)
        Sc = orc.commit(S0, args[1], args[2], al, be, par_u, path, plen)
        for u in range(U):
            O_ref, Vt_ref = cf.solve_unit(S0[u], args[0][u], args[1][u], args[2][u], al[u], be[u], par_u[u])
            assert rel(vt[u], Vt_ref) < tol, (N, u, rel(vt[u], Vt_ref))
            assert rel(o[u], O_ref) < tol, (N, u, rel(o[u], O_ref))
            S_ref = cf.commit_unit(S0[u], args[1][u], al[u], par_u[u], Vt_ref, list(path[u, :plen[u]]))
            assert rel(Sc[u], S_ref) < tol, (N, u)


def pin_commit_reads_out_node_output(orc, seed=5):
    """The committed state of node a, applied to q_a, is o_a (eq. 1 + eq. 3)."""
    rng = np.random.default_rng(seed)
    N, d = 20, 16
    par = wl.random_tree(rng, N, 6, (3,))
    S0, q, k, v, alpha, beta, _ = _unit_inputs(rng, N, d, parent=par)
    o, _ = orc.verify(S0[None], q[None], k[None], v[None], alpha[None], beta[None], par[None])
    for a in range(N):
        path = wl.ancestors_and_self(par, a)
        Sc = orc.commit(S0[None], k[None], v[None], alpha[None], beta[None], par[None],
                        np.array([path]), np.array([len(path)]))[0]
        assert rel(Sc @ q[a], o[0, a]) < 1e-13


def pin_non_ancestor_invariance(orc, seed=6):
    """Changing a node that is not an ancestor of t leaves o_t and vt_t bit-identical."""
    rng = np.random.default_rng(seed)
    N, d = 16, 8
    par = wl.random_tree(rng, N, 5, (3,))
    S0, q, k, v, alpha, beta, _ = _unit_inputs(rng, N, d, parent=par)
    o, vt = orc.verify(S0[None], q[None], k[None], v[None], alpha[None], beta[None], par[None])
    for j in range(N):
        k2, v2, a2, b2, q2 = k.copy(), v.copy(), alpha.copy(), beta.copy(), q.copy()
        k2[j] = rng.standard_normal(d); v2[j] += 1.0; a2[j] *= 0.5; b2[j] = 0.99; q2[j] *= -1
        o2, vt2 = orc.verify(S0[None], q2[None], k2[None], v2[None], a2[None], b2[None], par[None])
        for t in range(N):
            if j not in wl.ancestors_and_self(par, t):
                assert np.array_equal(o[0, t], o2[0, t]) and np.array_equal(vt[0, t], vt2[0, t])
            else:
                assert not np.array_equal(o[0, t], o2[0, t])


def pin_relabel_invariance(orc, seed=7):
    """DFS and BFS numbering of the same tree give the same per-node results."""
    rng = np.random.default_rng(seed)
    N, d = 18, 8
    par = wl.random_tree(rng, N, 5, (3,))
    S0, q, k, v, alpha, beta, _ = _unit_inputs(rng, N, d, parent=par)
    depth = wl.tree_depths(par)
    order = sorted(range(N), key=lambda t: (depth[t], t))       # BFS numbering, still parent < child
    new = {old: i for i, old in enumerate(order)}
    par2 = np.array([-1 if par[o_] == -1 else new[par[o_]] for o_ in order], dtype=np.int32)
    assert wl.is_topological(par2)
    perm = np.array(order)
    o, vt = orc.verify(S0[None], q[None], k[None], v[None], alpha[None], beta[None], par[None])
    o2, vt2 = orc.verify(S0[None], q[perm][None], k[perm][None], v[perm][None], alpha[perm][None],
                         beta[perm][None], par2[None])
    assert np.array_equal(o[0][perm], o2[0]) and np.array_equal(vt[0][perm], vt2[0])


def pin_multi_round(orc, seed=8):
    """Verify+commit a chain of n, then verify the next n from the committed
    state: the same as one chain of 2n (the committed state is next round's S0)."""
    rng = np.random.default_rng(seed)
    n, d = 5, 8
    S0, q, k, v, alpha, beta, par = _unit_inputs(rng, 2 * n, d)
    o, _ = orc.verify(S0[None], q[None], k[None], v[None], alpha[None], beta[None], par[None])
    h = slice(0, n)
    S1 = orc.commit(S0[None], k[None, h], v[None, h], alpha[None, h], beta[None, h],
                    wl.chain_tree(n)[None], np.arange(n)[None], np.array([n]))
    t = slice(n, 2 * n)
    o2, _ = orc.verify(S1, q[None, t], k[None, t], v[None, t], alpha[None, t], beta[None, t],
                       wl.chain_tree(n)[None])
    assert rel(o2[0], o[0, t]) < 1e-14


def pin_chain_warmup_matches_tree(orc, seed=9):
    """The warm-up entry (state only) agrees with the tree entry on a chain."""
    rng = np.random.default_rng(seed)
    S0, q, k, v, alpha, beta, par = _unit_inputs(rng, 6, 8)
    _, _, st = orc.verify(S0[None], q[None], k[None], v[None], alpha[None], beta[None], par[None], states=True)
    S = orc.chain(S0[None], k[None], v[None], alpha[None], beta[None])
    assert rel(S[0], st[0, -1]) < 1e-15


def pin_rejects_bad_trees(orc):
    """Parent indices outside [-1, t-1] and broken paths are refused."""
    import oracle
    one = np.ones((1, 2, 2))
    for bad in ([[-1, 1]], [[0, -1]], [[-1, -2]]):
        try:
            orc.verify(np.ones((1, 2, 2)), one, one, one, np.ones((1, 2)), np.ones((1, 2)), np.array(bad))
        except oracle.OracleError:
            continue
        raise AssertionError("accepted parent %r" % bad)
    # tree: node 1 is a child of node 0
    for path, plen in (([[1, 0]], [2]), ([[1, -1]], [1]), ([[0, 1]], [3]), ([[0, 2]], [2])):
        try:
            orc.commit(np.ones((1, 2, 2)), one, one, np.ones((1, 2)), np.ones((1, 2)), np.array([[-1, 0]]),
                       np.array(path), np.array(plen))
        except oracle.OracleError:
            continue
        raise AssertionError("accepted path %r" % path)


ALL_PINS = [pin_scalar_worked_example, pin_exact_rational, pin_chain_literal, pin_beta_zero,
            pin_overwrite, pin_brute_force_small_trees, pin_closed_form, pin_closed_form_fp32, pin_closed_form_fast_decay,
            pin_commit_reads_out_node_output, pin_non_ancestor_invariance, pin_relabel_invariance,
            pin_multi_round, pin_chain_warmup_matches_tree, pin_rejects_bad_trees]

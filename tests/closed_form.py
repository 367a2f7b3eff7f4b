"""Paper's closed form, written out in numpy (float64, or float32 on request; test-only).

Independent of the oracle (which runs the recurrence): this is eq. 2 (the
tree-masked triangular system for the pseudo-values), the output read out of
the same solve, and eq. 3 (reconstruct-on-commit).  Agreement of the two pins
the oracle to the paper's statement of the method, which claims exactly this
equality (Implementation: closed form vs per-node recurrence ~1e-15 in fp64,
~1e-7 in fp32).  `dtype` selects the arithmetic: float64, or float32 for the
paper's single-precision figure (every array, product and the solve in fp32).

Per unit, with nodes as rows:
  g_t     = product of alpha over the ancestors of t and t itself
  G[t,i]  = (g_t / g_i) (k_t . k_i) [i strict ancestor of t]           (eq. 2)
  R[t]    = beta_t v_t - beta_t g_t (S0 k_t)                            (eq. 2)
  (I + diag(beta) G) Vt = R
  o_t     = g_t S0 q_t + sum_{i ancestor-or-self of t} (g_t/g_i)(k_i . q_t) vt_i
  S_a     = g_a S0 + sum_{i ancestor-or-self of a} (g_a/g_i) vt_i k_i^T  (eq. 3)
"""
import numpy as np
import scipy.linalg


def ancestor_mask(parent):
    N = len(parent)
    M = np.zeros((N, N), dtype=bool)
    for t in range(N):
        p = parent[t]
        while p != -1:
            M[t, p] = True
            p = parent[p]
    return M


def cumulative_decay(parent, alpha):
    g = np.empty(len(parent), dtype=np.asarray(alpha).dtype)
    for t, p in enumerate(parent):
        g[t] = alpha[t] * (1.0 if p == -1 else g[p])
    return g


def solve_unit(S0, q, k, v, alpha, beta, parent, dtype=np.float64):
    """Returns (o, vt) for one unit: S0 [dv,dk], q,k [N,dk], v [N,dv]."""
    S0, q, k, v, alpha, beta = (np.asarray(x, dtype=dtype) for x in (S0, q, k, v, alpha, beta))
    N = len(parent)
    Ms = ancestor_mask(parent)
    Mi = Ms | np.eye(N, dtype=bool)
    g = cumulative_decay(parent, alpha)
    Dr = g[:, None] / g[None, :]
    G = np.where(Ms, Dr * (k @ k.T), dtype(0))
    Lm = np.eye(N, dtype=dtype) + beta[:, None] * G
    R = beta[:, None] * (v - g[:, None] * (k @ S0.T))
    Vt = scipy.linalg.solve_triangular(Lm, R, lower=True, unit_diagonal=True)
    A = np.where(Mi, Dr * (q @ k.T), dtype(0))
    O = g[:, None] * (q @ S0.T) + A @ Vt
    assert O.dtype == dtype and Vt.dtype == dtype
    return O, Vt


def commit_unit(S0, k, alpha, parent, vt, path, dtype=np.float64):
    """eq. 3 for one unit along `path` (root first)."""
    S0 = np.asarray(S0, dtype=dtype)
    if len(path) == 0:
        return S0.copy()
    g = cumulative_decay(parent, np.asarray(alpha, dtype=dtype))
    a = path[-1]
    S = g[a] * S0
    for i in path:
        S = S + (g[a] / g[i]) * np.outer(np.asarray(vt[i], dtype=dtype), np.asarray(k[i], dtype=dtype))
    assert S.dtype == dtype
    return S

"""Seeded synthetic inputs for tree-WY verification of the gated delta rule.

This module is shared by the HIP path (through the Python binding, the tests
and the benchmark) and by the oracle's callers.  It therefore holds none of
the method's arithmetic: it draws random tensors, draws random draft trees in
topological (DFS pre-order) order, draws accepted root-to-node paths, and
rounds inputs to bfloat16.  The committed state S0 is *not* made here: it is
the gated delta rule run over warm-up tokens, so each side makes it with its
own code from the warm-up tokens this module draws.

Shapes follow the paper's notation (Background, eq. 1): per sequence b and
value head h there is a state S0 in R^{d_v x d_k}; every draft node t carries
q_t, k_t in R^{d_k}, v_t in R^{d_v} and scalars alpha_t, beta_t in (0, 1).
A draft tree of N nodes is laid out so that every ancestor of t has a smaller
index (Method, "Verifying a draft"); parent[t] == -1 means t hangs directly
off the committed state.

Arrays are row-major numpy arrays:
  q, k      [B, H, N, d_k]  float32 (bf16-exact values when in_dtype == "bf16")
  v         [B, H, N, d_v]  float32 (bf16-exact values when in_dtype == "bf16")
  alpha     [B, H, N]       float32
  beta      [B, H, N]       float32
  parent    [B, N]          int32   (shared by all heads of a sequence)
  path      [B, L_max]      int32   root -> accepted node, padded with -1
  path_len  [B]             int32   (0 = nothing accepted)
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, Iterator, List, Optional, Sequence, Tuple

import numpy as np

ROOT = -1  # parent value of a node that hangs directly off the committed state


# --------------------------------------------------------------------------
# Workload table.  Sizes are Qwen3.5 GDN-layer shaped (Section "The memory
# problem": d_k = d_v = 128, 32 value heads at 35B-A3B, 64 at 397B-A17B).
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int
    d_k: int
    d_v: int
    in_dtype: str                  # "f32" or "bf16"
    tree: str                      # "chain" or "tree"
    max_depth: int
    caps: Tuple[int, ...]          # child cap by depth (depth 0 = virtual root); last entry repeats
    alpha_range: Tuple[float, float]
    beta_range: Tuple[float, float]
    warm_tokens: int               # warm-up tokens that produce S0 from zero
    accept: str                    # "prefix3" | "chain_depth_0_to_N" | "uniform_node" | "depth_1_to_8"

    @property
    def units(self) -> int:
        return self.B * self.H

    def describe(self) -> str:
        return (f"{self.name}: B={self.B}, H={self.H}, d_k=d_v={self.d_k}, N={self.N} "
                f"({self.tree}, max depth {self.max_depth}), {self.in_dtype} q/k/v, f32 state")


WORKLOADS: Dict[int, Workload] = {
    0: Workload("chain4-f32", 1, 1, 4, 128, 128, "f32", "chain", 4, (1,),
                (0.85, 0.999), (0.05, 0.95), 32, "prefix3"),
    1: Workload("35B-chain8", 16, 32, 8, 128, 128, "bf16", "chain", 8, (1,),
                (0.85, 0.999), (0.05, 0.95), 256, "chain_depth_0_to_N"),
    2: Workload("35B-tree16", 64, 32, 16, 128, 128, "bf16", "tree", 6, (3,),
                (0.85, 0.999), (0.05, 0.95), 256, "uniform_node"),
    3: Workload("397B-tree64", 128, 64, 64, 128, 128, "bf16", "tree", 8, (4, 4, 2),
                (0.9, 0.999), (0.05, 0.95), 256, "depth_1_to_8"),
    4: Workload("stress-tree32", 256, 64, 32, 128, 128, "bf16", "tree", 6, (3,),
                (0.85, 0.999), (0.05, 0.95), 256, "uniform_node"),
}

# Trees past one 64-node chunk, at the 397B layer shape: the distributions of
# the 64-node tree, twice the nodes and twice the depth.
BIG_TREE = Workload("397B-tree128", 128, 64, 128, 128, 128, "bf16", "tree", 16, (4, 4, 2),
                    (0.9, 0.999), (0.05, 0.95), 256, "uniform_node")


def scaled(w: Workload, B: Optional[int] = None, H: Optional[int] = None,
           N: Optional[int] = None) -> Workload:
    """Same distributions, different sizes (used for small parity cases)."""
    n = N if N is not None else w.N
    return dataclasses.replace(w, B=B if B is not None else w.B, H=H if H is not None else w.H,
                               N=n, max_depth=n if w.tree == "chain" else w.max_depth)


# --------------------------------------------------------------------------
# Random number streams: one child stream per quantity, so that changing one
# quantity's draw never shifts another's.
# --------------------------------------------------------------------------
_STREAMS = ("tree", "q", "k", "v", "alpha", "beta", "path", "warm")


def _rngs(cfg_key: int, seed: int) -> Dict[str, np.random.Generator]:
    ss = np.random.SeedSequence([20961, int(cfg_key), int(seed)])
    return {name: np.random.default_rng(child) for name, child in zip(_STREAMS, ss.spawn(len(_STREAMS)))}


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); return float32."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    if not np.isfinite(x32).all():
        raise ValueError("round_to_bf16 expects finite values")
    bits = x32.view(np.uint32)
    out = bits + np.uint32(0x7FFF) + ((bits >> np.uint32(16)) & np.uint32(1))
    out &= np.uint32(0xFFFF0000)
    return out.view(np.float32).reshape(x32.shape)


def _unit_rows(rng: np.random.Generator, shape: Tuple[int, ...], dtype=np.float64) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=dtype)
    x /= np.sqrt(np.einsum("...i,...i->...", x, x))[..., None]
    return x


# --------------------------------------------------------------------------
# Draft trees
# --------------------------------------------------------------------------
def _cap(caps: Sequence[int], depth: int) -> int:
    return caps[min(depth, len(caps) - 1)]


def _dfs_preorder(parent_raw: List[int], children: List[List[int]], roots: List[int]) -> np.ndarray:
    """Relabel a forest (hanging off the virtual root) in DFS pre-order."""
    order: List[int] = []
    stack = list(reversed(roots))
    while stack:
        n = stack.pop()
        order.append(n)
        stack.extend(reversed(children[n]))
    new_id = {old: i for i, old in enumerate(order)}
    parent = np.empty(len(order), dtype=np.int32)
    for old, i in new_id.items():
        p = parent_raw[old]
        parent[i] = ROOT if p == ROOT else new_id[p]
    return parent


def random_tree(rng: np.random.Generator, N: int, max_depth: int, caps: Sequence[int]) -> np.ndarray:
    """A random draft tree of N nodes whose deepest node has depth max_depth.

    One spine of length max_depth is laid first so the stated depth is reached;
    each remaining node then hangs off a uniformly drawn eligible parent (the
    virtual root or any node shallower than max_depth whose child count is below
    the cap for its depth).  Nodes are finally renumbered in DFS pre-order,
    children visited in creation order, so parent[t] < t.
    """
    if not (1 <= max_depth <= N):
        raise ValueError("need 1 <= max_depth <= N")
    parent_raw: List[int] = []
    depth: List[int] = []
    children: List[List[int]] = []
    roots: List[int] = []
    root_children = 0

    def add(p: int) -> None:
        nonlocal root_children
        n = len(parent_raw)
        parent_raw.append(p)
        depth.append(1 if p == ROOT else depth[p] + 1)
        children.append([])
        if p == ROOT:
            roots.append(n)
            root_children += 1
        else:
            children[p].append(n)

    for i in range(max_depth):
        add(ROOT if i == 0 else i - 1)
    while len(parent_raw) < N:
        eligible = [ROOT] if root_children < _cap(caps, 0) else []
        eligible += [n for n in range(len(parent_raw))
                     if depth[n] < max_depth and len(children[n]) < _cap(caps, depth[n])]
        if not eligible:
            raise ValueError("tree caps leave no room for N nodes")
        add(eligible[int(rng.integers(len(eligible)))])
    return _dfs_preorder(parent_raw, children, roots)


def chain_tree(N: int) -> np.ndarray:
    return np.arange(-1, N - 1, dtype=np.int32)


def width_tree(widths: Sequence[int]) -> np.ndarray:
    """Fixed-shape draft tree from per-level branching factors (w1, w2, ...).

    Level 1 has w1 nodes hanging off the committed state and every node at
    level l has w_{l+1} children (the draft-tree-widths option in the
    Implementation section).  Returned in DFS pre-order.
    """
    parent: List[int] = []

    def grow(p: int, level: int) -> None:
        if level == len(widths):
            return
        for _ in range(widths[level]):
            parent.append(p)
            grow(len(parent) - 1, level + 1)

    grow(ROOT, 0)
    return np.asarray(parent, dtype=np.int32)


def tree_depths(parent: np.ndarray) -> np.ndarray:
    """Depth of every node (1 for children of the committed state)."""
    d = np.zeros(len(parent), dtype=np.int32)
    for t, p in enumerate(parent):
        d[t] = 1 if p == ROOT else d[p] + 1
    return d


def ancestors_and_self(parent: np.ndarray, node: int) -> List[int]:
    """Root -> node path (inclusive), i.e. the accepted path of `node`."""
    path = []
    while node != ROOT:
        path.append(int(node))
        node = int(parent[node])
    return path[::-1]


def is_topological(parent: np.ndarray) -> bool:
    return all(ROOT <= int(p) < t for t, p in enumerate(parent))


# --------------------------------------------------------------------------
# Full input sets
# --------------------------------------------------------------------------
def _draw_paths(w: Workload, rng: np.random.Generator, parents: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    L_max = w.max_depth
    path = np.full((w.B, L_max), -1, dtype=np.int32)
    plen = np.zeros(w.B, dtype=np.int32)
    for b in range(w.B):
        par = parents[b]
        if w.accept == "prefix3":
            nodes = list(range(min(3, w.N)))
        elif w.accept == "chain_depth_0_to_N":
            d = int(rng.integers(0, w.N + 1))
            nodes = list(range(d))
        elif w.accept == "uniform_node":
            nodes = ancestors_and_self(par, int(rng.integers(w.N)))
        elif w.accept == "depth_1_to_8":
            dep = tree_depths(par)
            d = int(rng.integers(1, min(8, int(dep.max())) + 1))
            cand = np.flatnonzero(dep == d)
            nodes = ancestors_and_self(par, int(cand[int(rng.integers(len(cand)))]))
        else:
            raise ValueError(w.accept)
        path[b, :len(nodes)] = nodes
        plen[b] = len(nodes)
    return path, plen


def make_inputs(w: Workload, seed: int = 0, cfg_key: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Draw one full input set for workload `w` (everything except S0)."""
    key = cfg_key if cfg_key is not None else _key_of(w)
    r = _rngs(key, seed)
    B, H, N, dk, dv = w.B, w.H, w.N, w.d_k, w.d_v
    if w.tree == "chain":
        parents = np.tile(chain_tree(N), (B, 1))
    else:
        parents = np.stack([random_tree(r["tree"], N, w.max_depth, w.caps) for _ in range(B)])
    q = _unit_rows(r["q"], (B, H, N, dk), np.float32)
    k = _unit_rows(r["k"], (B, H, N, dk), np.float32)
    v = r["v"].standard_normal((B, H, N, dv), dtype=np.float32)
    if w.in_dtype == "bf16":
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
    alpha = r["alpha"].uniform(*w.alpha_range, size=(B, H, N)).astype(np.float32)
    beta = r["beta"].uniform(*w.beta_range, size=(B, H, N)).astype(np.float32)
    path, plen = _draw_paths(w, r["path"], parents)
    return dict(q=q, k=k, v=v, alpha=alpha, beta=beta, parent=parents.astype(np.int32),
                path=path, path_len=plen)


def _key_of(w: Workload) -> int:
    for key, ref in WORKLOADS.items():
        if ref.name == w.name:
            return key
    return 99


def warmup_tokens(w: Workload, seed: int = 0, units: Optional[slice] = None,
                  cfg_key: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Warm-up tokens that produce S0 from a zero state, for a slice of units.

    Units are (b, h) pairs flattened as b * H + h.  Every unit has its own
    stream, so any slice is reproducible on its own.  Shapes: k [U, W, d_k]
    (unit rows), v [U, W, d_v], alpha [U, W], beta [U, W], all float64.
    """
    key = cfg_key if cfg_key is not None else _key_of(w)
    sl = units if units is not None else slice(0, w.units)
    ids = range(*sl.indices(w.units))
    W, dk, dv = w.warm_tokens, w.d_k, w.d_v
    out = {n: [] for n in ("k", "v", "alpha", "beta")}
    for u in ids:
        g = np.random.default_rng(np.random.SeedSequence([20961, int(key), int(seed), 7, u]))
        out["k"].append(_unit_rows(g, (W, dk)))
        out["v"].append(g.standard_normal((W, dv)))
        out["alpha"].append(g.uniform(*w.alpha_range, size=W))
        out["beta"].append(g.uniform(*w.beta_range, size=W))
    return {n: np.stack(a) if a else np.zeros((0,)) for n, a in out.items()}


def acceptance_tokens(parents: np.ndarray, seed: int = 0, vocab: int = 4, plant: bool = True
                      ) -> Dict[str, np.ndarray]:
    """Synthetic tokens for greedy acceptance over the trees `parents` [B, N].

    draft [B, N]: the token proposed at each node; target [B, N]: the target's
    next token after each node; root [B]: its next token after the committed
    prefix, all uniform in [0, vocab).  With `plant`, the target agrees with
    the drafter along one random root-to-node chain per sequence, so long
    acceptances occur.
    """
    parents = np.asarray(parents)
    B, N = parents.shape
    rng = np.random.default_rng(np.random.SeedSequence([20961, 7, int(seed), B, N, int(vocab)]))
    draft = rng.integers(0, vocab, (B, N)).astype(np.int32)
    target = rng.integers(0, vocab, (B, N)).astype(np.int32)
    root = rng.integers(0, vocab, B).astype(np.int32)
    if plant and N > 0:
        for b in range(B):
            chain = ancestors_and_self(parents[b], int(rng.integers(N)))
            root[b] = draft[b, chain[0]]
            for a, c in zip(chain[:-1], chain[1:]):
                target[b, a] = draft[b, c]
    return dict(draft=draft, target=target, root=root)


def sample_units(w: Workload, count: int, seed: int = 0) -> np.ndarray:
    """A reproducible sample of unit ids (b * H + h), always including the first and last."""
    rng = np.random.default_rng(np.random.SeedSequence([20961, 5, int(seed), w.units]))
    if count >= w.units:
        return np.arange(w.units)
    pick = rng.choice(np.arange(1, w.units - 1), size=max(count - 2, 0), replace=False)
    return np.unique(np.concatenate([[0, w.units - 1], pick])).astype(np.int64)


def warmup_chunk_torch(w: Workload, seed: int, chunk: int, T: int, device, dtype):
    """Warm-up tokens drawn on the device with torch (for large batches).

    Returns k [B, H, T, d_k] (unit rows, cast to `dtype`), v [B, H, T, d_v]
    (`dtype`), alpha and beta [B, H, T] (float32) from the workload's ranges.
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(20961 * 1000003 + 7919 * int(seed) + int(chunk))
    shp = (w.B, w.H, T)
    k = torch.randn(*shp, w.d_k, generator=g, device=device, dtype=torch.float32)
    k = k / k.norm(dim=-1, keepdim=True)
    v = torch.randn(*shp, w.d_v, generator=g, device=device, dtype=torch.float32)
    lo, hi = w.alpha_range
    alpha = lo + (hi - lo) * torch.rand(*shp, generator=g, device=device, dtype=torch.float32)
    lo, hi = w.beta_range
    beta = lo + (hi - lo) * torch.rand(*shp, generator=g, device=device, dtype=torch.float32)
    return k.to(dtype).contiguous(), v.to(dtype).contiguous(), alpha.contiguous(), beta.contiguous()

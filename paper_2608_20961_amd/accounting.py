"""Memory and traffic accounting for verify / commit and the snapshot baseline.

Two kinds of figures live here:

* the paper's memory model (Section "The memory problem"): KV bytes per token
  of the softmax layers, the GDN state per sequence, and the number of state
  blocks that full-state snapshotting keeps (k + 1 for a chain of k, N + 1
  for a tree of N, Appendix "Wide draft trees");
* the algorithmic HBM bytes each kernel must move per launch, which is what a
  measured time is divided by to get achieved GB/s.

Algorithmic bytes per (sequence, head) unit, d = d_k = d_v, s_in the input
element size (2 for bf16, 4 for fp32), state and pseudo-values in fp32:
  verify   = d^2*4 (S0) + 3*N*d*s_in (q,k,v) + 2*N*4 (alpha,beta)
             + N*d*s_in (o) + N*d*4 (U)               + N*4/H (parent, shared by heads)
  commit   = 2*d^2*4 (S0 read, S_new write) + L*(d*4 + d*s_in + 4) (U, k, alpha on the path)
  snapshot = d^2*4 + inputs + o + N*d^2*4 (one full state written per node)
             (+ d^2*4 per node whose parent is not the node before it, read
             back by the node-by-node baseline kernel; counted separately)
"""
from __future__ import annotations

import numpy as np

from .workload import Workload

KiB = 1024
MiB = 1024 ** 2
GiB = 1024 ** 3


# ---- the paper's memory model --------------------------------------------
def kv_bytes_per_token(n_softmax: int, n_kv_heads: int, d_head: int, elem: int = 2) -> int:
    """2 (K and V) x softmax layers x KV heads x head dim x element bytes."""
    return 2 * n_softmax * n_kv_heads * d_head * elem


def gdn_state_bytes_per_seq(n_gdn: int, n_v_heads: int, d_v: int, d_k: int, elem: int = 2) -> int:
    """One d_v x d_k state per GDN layer and value head."""
    return n_gdn * n_v_heads * d_v * d_k * elem


def snapshot_blocks(draft_nodes: int) -> int:
    """Full-state snapshotting keeps the committed state plus one per draft node."""
    return draft_nodes + 1


def treewy_blocks(draft_nodes: int) -> int:
    """Reconstruct-on-commit keeps one state block whatever the draft size."""
    return 1


def pseudo_value_ratio(d_k: int) -> int:
    """A node's pseudo-value row (d_v) against a per-node state (d_v x d_k)."""
    return d_k


# Qwen3.5 hybrids as described in Section "The memory problem".
MODELS = {
    "35B-A3B": dict(n_gdn=30, n_softmax=10, n_v_heads=32, n_kv_heads=2, d_head=256, d_k=128, d_v=128),
    "397B-A17B": dict(n_gdn=45, n_softmax=15, n_v_heads=64, n_kv_heads=2, d_head=256, d_k=128, d_v=128),
}


# ---- algorithmic bytes per launch -----------------------------------------
def elem_bytes(in_dtype: str) -> int:
    return {"bf16": 2, "f32": 4}[in_dtype]


def verify_bytes(w: Workload, state_bytes: int = 4) -> int:
    """state_bytes: 4 for a float32 state, 2 for a bfloat16 state."""
    s, d, N = elem_bytes(w.in_dtype), w.d_k, w.N
    per_unit = d * d * state_bytes + 3 * N * d * s + 2 * N * 4 + N * d * s + N * d * 4
    return w.units * per_unit + w.B * N * 4


def commit_bytes(w: Workload, path_len: np.ndarray, state_bytes: int = 4) -> int:
    """path_len [B]: the accepted path length of every sequence."""
    s, d = elem_bytes(w.in_dtype), w.d_k
    L = np.asarray(path_len, dtype=np.int64)
    per_seq = w.H * (2 * d * d * state_bytes + L * (d * 4 + d * s + 4)) + L * 4 + 4
    return int(per_seq.sum())


def commit_verify_bytes(w: Workload, path_len: np.ndarray, state_bytes: int = 4) -> int:
    """The previous round's commit fused into this round's verify (both rounds
    shaped like `w`): commit + verify minus the second read of the state,
    which the fused call takes from registers."""
    return (verify_bytes(w, state_bytes) + commit_bytes(w, path_len, state_bytes)
            - w.units * w.d_k * w.d_v * state_bytes)


def prefill_bytes(w: Workload, T: int, state_bytes: int = 4) -> int:
    """Chain prefill of T tokens per unit: the state read and written once,
    q, k, v read and o written per token, alpha and beta per token."""
    s, d = elem_bytes(w.in_dtype), w.d_k
    return w.units * (2 * d * d * state_bytes + T * (4 * d * s + 2 * 4))


def snapshot_verify_bytes(w: Workload) -> int:
    """What store-all must move at least: S0 once, the node vectors, o, and
    one full state written per node (an ideal kernel keeps the states of the
    current root-to-node path on chip, so it never reads a snapshot back)."""
    s, d, N = elem_bytes(w.in_dtype), w.d_k, w.N
    per_unit = d * d * 4 + 3 * N * d * s + 2 * N * 4 + N * d * s + N * d * d * 4
    return w.units * per_unit + w.B * N * 4


def snapshot_reload_bytes(w: Workload, parent: np.ndarray) -> int:
    """State bytes the baseline kernel reads back on top of that: the node-by-
    node kernel holds one running state, so every node whose parent is not the
    node before it reloads its parent's state (S0 or a snapshot, d^2 fp32
    values).  parent [B, N]."""
    par = np.asarray(parent, dtype=np.int64)
    prev = np.arange(-1, w.N - 1, dtype=np.int64)[None, :]
    reloads = int((par != prev).sum())               # per sequence, summed over B
    return reloads * w.H * w.d_k * w.d_v * 4


def snapshot_commit_bytes(w: Workload) -> int:
    """Copy of the accepted node's snapshot into the committed state."""
    return w.units * 2 * w.d_k * w.d_v * 4 + w.B * 4


def speculative_state_bytes(w: Workload) -> dict:
    """Bytes held between verify and commit, beyond the committed state."""
    d, N, s = w.d_k, w.N, elem_bytes(w.in_dtype)
    return {
        "treewy_U": w.units * N * d * 4,
        "treewy_U_k_alpha": w.units * N * (d * 4 + d * s + 4),
        "snapshot_states": w.units * N * d * d * 4,
        "committed_state": w.units * d * d * 4,
    }


def verify_flops(w: Workload) -> int:
    """Useful flops of the method: S0 against K and Q, masked gram, solve, read-out."""
    d, N = w.d_k, w.N
    return w.units * (4 * d * d * N + 2 * d * N * (N - 1) + 2 * d * N * (N + 1))

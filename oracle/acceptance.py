"""Greedy acceptance of a draft tree, plain Python (CPU reference).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: used by the tests and
never by the product path; shares no code with the HIP library.

The target model verifies every draft node in one pass and, under greedy
decoding, would itself emit one token after each prefix: ``root_pred`` after
the committed prefix and ``target_pred[t]`` after node t.  Acceptance keeps
the longest run of draft tokens the target would have generated itself
(Background, speculative decoding; the paper verifies greedily,
Implementation).  On a tree that is a walk from the committed prefix: among
the children of the current position, take the one whose draft token equals
the target's prediction there, and continue from it; stop when no child
matches.  Siblings carrying the same token are duplicates of one another; the
walk takes the lowest index among them.  The next emitted ("bonus") token is
the target's prediction at the last accepted position.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np


def accept_one(parent, draft, target_pred, root_pred) -> Tuple[List[int], int]:
    """One sequence: (accepted root-to-node path, bonus token)."""
    n = len(parent)
    position, want, path = -1, int(root_pred), []
    while True:
        match = [t for t in range(n) if int(parent[t]) == position and int(draft[t]) == want]
        if not match:
            return path, want
        node = min(match)
        path.append(node)
        position, want = node, int(target_pred[node])


def accept_greedy(parent, draft, target_pred, root_pred, L_max: int):
    """Batch of sequences in the layout the library uses.

    parent, draft, target_pred [B, N]; root_pred [B].  Returns path [B, L_max]
    (root first, padded with -1), path_len [B] and bonus [B].  A parent
    outside [-1, t-1] counts as -1 (the tree kernels do the same).
    """
    parent = np.asarray(parent)
    B, N = parent.shape
    path = np.full((B, L_max), -1, dtype=np.int32)
    plen = np.zeros(B, dtype=np.int32)
    bonus = np.zeros(B, dtype=np.int32)
    for b in range(B):
        par = [int(p) if -1 <= int(p) < t else -1 for t, p in enumerate(parent[b])]
        nodes, nxt = accept_one(par, draft[b], target_pred[b], root_pred[b])
        bonus[b] = nxt
        if len(nodes) <= L_max:
            path[b, :len(nodes)] = nodes
            plen[b] = len(nodes)
        else:
            plen[b] = -1                              # does not fit: the caller flags it
    return path, plen, bonus

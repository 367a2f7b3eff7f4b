"""Pins of the greedy-acceptance reference (oracle/acceptance.py).

Hand-worked cases (expected paths written out by reasoning, not by running
the reference) and a characterisation that fixes the result on any tree:
the accepted path is a root-to-node chain whose every token equals the
target's prediction at its predecessor, no lower-index sibling would also
match at any step, no child of the last node matches, and the bonus is the
target's prediction at the last node.
"""
import numpy as np
import pytest

from oracle.acceptance import accept_greedy, accept_one

# parent:  0 and 1 hang off the prefix; 2, 3 under 0; 4 under 2; 5 under 1
PARENT = [-1, -1, 0, 0, 2, 1]
DRAFT = [5, 7, 9, 9, 3, 4]
TARGET = [9, 4, 3, 1, 8, 2]


@pytest.mark.parametrize("root,path,bonus", [
    (7, [1, 5], 2),        # 1 matches 7, then 5 matches target[1] = 4, nothing under 5
    (5, [0, 2, 4], 8),     # 0, then 2 and 3 both carry 9: the lower index 2 wins, then 4
    (6, [], 6),            # no child of the prefix carries 6
    (9, [], 9),
])
def test_hand_worked_tree(root, path, bonus):
    assert accept_one(PARENT, DRAFT, TARGET, root) == (path, bonus)


def test_chain_all_accepted_and_first_rejected():
    n = 6
    parent = list(range(-1, n - 1))
    draft = [10 + t for t in range(n)]
    target = [11 + t for t in range(n)]          # the target predicts each next draft token
    assert accept_one(parent, draft, target, 10) == (list(range(n)), 10 + n)
    assert accept_one(parent, draft, target, 3) == ([], 3)
    target[2] = 0                                # disagreement after node 2
    assert accept_one(parent, draft, target, 10) == ([0, 1, 2], 0)


def test_batch_layout_bad_parent_and_overflow():
    parent = np.array([PARENT, [-1, 0, 1, 2, 3, 4], [-1, 5, 0, 0, 0, 0]])
    draft = np.array([DRAFT, [1, 2, 3, 4, 5, 6], [1, 2, 2, 2, 2, 2]])
    target = np.array([TARGET, [2, 3, 4, 5, 6, 7], [2, 2, 2, 2, 2, 2]])
    root = np.array([5, 1, 1])
    path, plen, bonus = accept_greedy(parent, draft, target, root, L_max=4)
    assert plen.tolist() == [3, -1, 2]           # the chain accepts 6 > L_max = 4 nodes
    assert path[0].tolist() == [0, 2, 4, -1] and bonus[0] == 8
    assert path[1].tolist() == [-1] * 4 and bonus[1] == 7
    # sequence 2: parent[1] = 5 is invalid (not below 1) and counts as -1; node 1
    # does not match the root token, node 0 does; under 0 nodes 2..5 all carry 2
    # and the lowest (2) wins; nothing hangs under 2
    assert path[2].tolist() == [0, 2, -1, -1] and bonus[2] == 2


def _characterise(parent, draft, target, root, path, bonus):
    n = len(parent)
    pos, want = -1, root
    for node in path:
        assert parent[node] == pos and draft[node] == want
        lower = [t for t in range(node) if parent[t] == pos and draft[t] == want]
        assert not lower
        pos, want = node, target[node]
    assert bonus == want
    assert not [t for t in range(n) if parent[t] == pos and draft[t] == want]


@pytest.mark.parametrize("seed", range(40))
def test_random_trees_satisfy_the_characterisation(seed):
    from paper_2608_20961_amd import workload as wl
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 65)) if seed % 2 else int(rng.integers(65, 257))
    parent = [int(p) for p in wl.random_tree(rng, n, int(rng.integers(1, min(n, 40) + 1)), (256,))]
    vocab = int(rng.integers(1, 5))
    draft = [int(x) for x in rng.integers(0, vocab, n)]
    target = [int(x) for x in rng.integers(0, vocab, n)]
    root = int(rng.integers(0, vocab))
    path, bonus = accept_one(parent, draft, target, root)
    _characterise(parent, draft, target, root, path, bonus)

"""Pins for the acceptance-walk oracle: hand-worked trees and path invariants."""
import numpy as np
import pytest

from oracle.walk import accept_walk, walk_arrays


def test_hand_worked_tree():
    #        0
    #      / | \
    #     1  2  3        tokens 10 11 12
    #    / \     \
    #   4   5     6      tokens 20 21 22
    #   |
    #   7                token 30
    parent = np.array([-1, 0, 0, 0, 1, 1, 3, 4])
    token = np.array([-1, 10, 11, 12, 20, 21, 22, 30])
    target = np.array([10, 20, 0, 0, 30, 0, 0, 99])
    path, bonus = accept_walk(parent, token, 8, target)
    assert path == [0, 1, 4, 7] and bonus == 99
    target2 = np.array([12, 0, 0, 22, 0, 0, 55, 0])
    assert accept_walk(parent, token, 8, target2) == ([0, 3, 6], 55)
    target3 = np.array([13, 0, 0, 0, 0, 0, 0, 0])
    assert accept_walk(parent, token, 8, target3) == ([0], 13)
    # a matching child beyond n is invisible
    assert accept_walk(parent, token, 4, target) == ([0, 1], 20)


@pytest.mark.parametrize("seed", range(20))
def test_walk_invariants_random(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    parent = np.array([-1] + [int(rng.integers(0, i)) for i in range(1, n)])
    token = np.full(n, -1)
    for p in range(n):
        kids = [c for c in range(1, n) if parent[c] == p]
        toks = rng.choice(50, size=len(kids), replace=False)
        token[kids] = toks
    target = rng.integers(0, 50, size=n)
    path, bonus = accept_walk(parent, token, n, target)
    assert path[0] == 0
    for a, b in zip(path, path[1:]):
        assert parent[b] == a and token[b] == target[a]
    last = path[-1]
    assert not any(parent[c] == last and token[c] == target[last] for c in range(1, n))
    assert bonus == target[last]
    arr, ln, bn = walk_arrays(path, bonus, 40)
    assert ln == len(path) and list(arr[:ln]) == path and np.all(arr[ln:] == -1)

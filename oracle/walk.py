"""Greedy acceptance walk (temperature 0; Sec. 1 and the Limitations section).

A drafted node is accepted when its token equals the target model's greedy
choice after its parent, and its parent was accepted; the root always is.
Siblings carry distinct tokens (they are distinct top-K entries of one row),
so at most one child of an accepted node can match: the accepted nodes form a
single root path.  The bonus token is the target's choice after the last
accepted node.
"""
from __future__ import annotations

import numpy as np


def accept_walk(parent: np.ndarray, token: np.ndarray, n: int, target: np.ndarray):
    """Returns (path of node indices starting at 0, bonus token)."""
    cur = 0
    path = [0]
    while True:
        nxt = [c for c in range(1, n) if int(parent[c]) == cur and int(token[c]) == int(target[cur])]
        if not nxt:
            break
        assert len(nxt) == 1, "siblings with equal tokens"
        cur = nxt[0]
        path.append(cur)
    return path, int(target[cur])


def walk_arrays(path: list[int], bonus: int, block: int):
    """Fixed-size outputs: path padded with -1 to block+1 entries, its length, the bonus."""
    out = np.full(block + 1, -1, dtype=np.int32)
    out[:len(path)] = path
    return out, len(path), bonus

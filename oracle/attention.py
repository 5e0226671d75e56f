"""Tree-masked verification attention (Sec. 4.1 Stage 3; Sec. 4.3), plain fp64.

Reading of the tree attention used for verification (Sec. 4.3 requires the
selected set to be prefix closed, so each node's ancestors are all present):
a node's query sees every cached context row of its request and the tree rows
of the nodes on its own root path, itself included, and no other tree row.
The tree nodes' keys and values sit in the request's cache rows ctx + i, in
tree order.  Query head h reads KV head h // (Hq / Hkv).  Softmax is
max-subtracted, O = p @ V.
"""
from __future__ import annotations

import numpy as np


def ancestor_sets(parent: np.ndarray, n: int) -> list[list[int]]:
    """Ancestor-or-self set of every node, by walking parent pointers to the root."""
    out = []
    for i in range(n):
        a = []
        j = i
        while j >= 0:
            a.append(j)
            j = int(parent[j]) if j > 0 else -1
        out.append(sorted(a))
    return out


def allowed_rows(ctx: int, anc: list[int]) -> np.ndarray:
    return np.concatenate([np.arange(ctx, dtype=np.int64), ctx + np.asarray(anc, dtype=np.int64)])


def attend_one(q_row: np.ndarray, K_rows: np.ndarray, V_rows: np.ndarray, scale: float) -> np.ndarray:
    """softmax(scale * K q) @ V for one query row, fp64."""
    s = scale * (K_rows @ q_row)
    s = s - s.max()
    p = np.exp(s)
    p = p / p.sum()
    return p @ V_rows


def tree_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, kv_offset: np.ndarray,
                   ctx_len: np.ndarray, parents: list[np.ndarray], n_nodes: list[int],
                   scale: float, samples=None) -> np.ndarray:
    """O[b, i, h, :] for every node i < n_b (NaN elsewhere), or only for ``samples``.

    Q: [B][N][Hq][hd], K/V: [rows][Hkv][hd], all float64.
    ``samples``: optional iterable of (b, i, h); other entries stay NaN.
    """
    B, N, Hq, hd = Q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    O = np.full(Q.shape, np.nan, dtype=np.float64)
    want = None if samples is None else {}
    if samples is not None:
        for (b, i, h) in samples:
            want.setdefault((b, i), []).append(h)
    for b in range(B):
        anc = ancestor_sets(parents[b], n_nodes[b])
        off = int(kv_offset[b])
        ctx = int(ctx_len[b])
        for i in range(n_nodes[b]):
            heads = range(Hq) if want is None else want.get((b, i), [])
            if not heads:
                continue
            rows = off + allowed_rows(ctx, anc[i])
            Kr = K[rows]          # [R][Hkv][hd]
            Vr = V[rows]
            for h in heads:
                g = h // G
                O[b, i, h] = attend_one(Q[b, i, h], Kr[:, g, :], Vr[:, g, :], scale)
    return O


def tree_attention_paged(Q: np.ndarray, K_pages: np.ndarray, V_pages: np.ndarray,
                         block_table: np.ndarray, page_rows: int, ctx_len: np.ndarray,
                         parents: list[np.ndarray], n_nodes: list[int], scale: float,
                         samples=None) -> np.ndarray:
    """tree_attention over a paged cache.

    Reading (the cache layout is the serving system's; the paper's Limitations name batched
    serving): request b's logical cache row r -- its context rows 0 .. ctx-1, then tree
    node i at row ctx + i, as in the contiguous layout -- is stored at
    K_pages[block_table[b][r // page_rows], r % page_rows] (V_pages alike).  The rows are
    gathered into a contiguous cache, then the plain definition above applies.

    K_pages/V_pages: [pages][page_rows][Hkv][hd] float64; block_table: [B][max_pages].
    """
    B, N = Q.shape[0], Q.shape[1]
    Ks, Vs, offs = [], [], []
    base = 0
    for b in range(B):
        rows = np.arange(int(ctx_len[b]) + N)
        page = np.asarray(block_table[b])[rows // page_rows]
        slot = rows % page_rows
        Ks.append(K_pages[page, slot])
        Vs.append(V_pages[page, slot])
        offs.append(base)
        base += len(rows)
    K = np.concatenate(Ks) if Ks else np.zeros((0,) + K_pages.shape[2:])
    V = np.concatenate(Vs) if Vs else np.zeros((0,) + V_pages.shape[2:])
    return tree_attention(Q, K, V, np.asarray(offs, dtype=np.int64), ctx_len, parents, n_nodes,
                          scale, samples)

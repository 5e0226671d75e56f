"""KV commit of the accepted path -- TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Sec. 1 states that each decoding round commits only one prefix path of the
verified tree; the paper leaves the cache update itself to the serving system
(Limitations: KV-cache management).  The reading implemented here (and by the
kv_commit call): the root and the accepted nodes keep their key/value rows, in
path order, right after the context; the context grows by the path length; the
round emits the accepted drafted tokens followed by the target's bonus token.

The definition is a gather from the cache as it was before the update; rows
outside the committed path's targets keep their contents.
"""
from __future__ import annotations

import numpy as np


def committed_path(path_row: np.ndarray, path_len: int, budget: int, block: int) -> list[int]:
    """The root, then path entries while they increase and stay below the budget."""
    m_in = min(max(int(path_len), 1), block + 1)
    nodes = [0]
    for j in range(1, m_in):
        s = int(path_row[j])
        if s <= nodes[-1] or s >= budget:
            break
        nodes.append(s)
    return nodes


def kv_commit(K: np.ndarray, V: np.ndarray, kv_offset, ctx_len, token: np.ndarray,
              path: np.ndarray, path_len, bonus, budget: int, block: int, max_ctx: int):
    """Returns (K', V', new_ctx_len, committed [batch][block+1], n_committed)."""
    K2, V2 = K.copy(), V.copy()
    batch = len(ctx_len)
    new_ctx = np.zeros(batch, dtype=np.int32)
    committed = np.full((batch, block + 1), -1, dtype=np.int32)
    n = np.zeros(batch, dtype=np.int32)
    for b in range(batch):
        ctx = min(max(int(ctx_len[b]), 0), max_ctx)
        nodes = committed_path(path[b], int(path_len[b]), budget, block)
        m = len(nodes)
        base = int(kv_offset[b]) + ctx
        src = [base + s for s in nodes]
        K2[base:base + m] = K[src]
        V2[base:base + m] = V[src]
        toks = [int(token[b][s]) for s in nodes[1:]] + [int(bonus[b])]
        committed[b, :m] = toks
        new_ctx[b] = ctx + m
        n[b] = m
    return K2, V2, new_ctx, committed, n


def kv_commit_paged(K_pages: np.ndarray, V_pages: np.ndarray, block_table: np.ndarray,
                    page_rows: int, ctx_len, token: np.ndarray, path: np.ndarray, path_len,
                    bonus, budget: int, block: int, max_ctx: int):
    """kv_commit on a paged cache: request b's logical row r is row r % page_rows of page
    block_table[b][r // page_rows] (the serving system's layout; the reading of tree
    attention over pages).  The same gather in logical rows, from the pools as they were
    before the update.  Returns (K', V', new_ctx_len, committed, n_committed)."""
    K2, V2 = K_pages.copy(), V_pages.copy()
    batch = len(ctx_len)
    new_ctx = np.zeros(batch, dtype=np.int32)
    committed = np.full((batch, block + 1), -1, dtype=np.int32)
    n = np.zeros(batch, dtype=np.int32)
    for b in range(batch):
        ctx = min(max(int(ctx_len[b]), 0), max_ctx)
        nodes = committed_path(path[b], int(path_len[b]), budget, block)
        m = len(nodes)

        def where(r):
            return int(block_table[b][r // page_rows]), r % page_rows

        for j, s in enumerate(nodes):
            dst, src = where(ctx + j), where(ctx + s)
            K2[dst] = K_pages[src]
            V2[dst] = V_pages[src]
        committed[b, :m] = [int(token[b][s]) for s in nodes[1:]] + [int(bonus[b])]
        new_ctx[b] = ctx + m
        n[b] = m
    return K2, V2, new_ctx, committed, n

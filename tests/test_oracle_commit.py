"""Pins for the KV-commit oracle: hand-worked gathers, the degenerate paths, the cut of
malformed paths, isolation between requests, and equality with an in-place sequential
move (the order the GPU's in-place gather relies on)."""
import numpy as np
import pytest

from oracle.commit import committed_path, kv_commit
from oracle.walk import accept_walk, walk_arrays


def rows_cache(rows, width=3):
    """Cache whose row r holds r in every element, so a gather is readable by eye."""
    K = np.repeat(np.arange(rows, dtype=np.float32)[:, None, None], width, axis=2)
    return K, -K


def test_hand_worked_gather():
    # one request: context rows 0..2, tree rows 3..10 (8 nodes); path 0 -> 2 -> 5
    K, V = rows_cache(11)
    token = np.array([[-1, 10, 11, 12, 13, 14, 15, 16]], dtype=np.int32)
    path = np.array([[0, 2, 5, -1, -1]], dtype=np.int32)
    K2, V2, ctx, com, n = kv_commit(K, V, [0], [3], token, path, [3], [77], budget=8, block=4,
                                    max_ctx=3)
    assert list(K2[:, 0, 0]) == [0, 1, 2, 3, 5, 8, 6, 7, 8, 9, 10]
    assert list(V2[:, 0, 0]) == [0, -1, -2, -3, -5, -8, -6, -7, -8, -9, -10]
    assert list(ctx) == [6] and list(n) == [3]
    assert list(com[0]) == [11, 14, 77, -1, -1]


def test_root_only_and_chain_leave_the_cache():
    K, V = rows_cache(20)
    token = np.arange(16, dtype=np.int32)[None, :] + 100
    for path, plen, toks in ([[0, -1, -1, -1]], 1, [9]), ([[0, 1, 2, 3]], 4, [101, 102, 103, 9]):
        K2, V2, ctx, com, n = kv_commit(K, V, [2], [2], token, np.array(path, np.int32), [plen],
                                        [9], budget=16, block=3, max_ctx=2)
        assert np.array_equal(K2, K) and np.array_equal(V2, V)
        assert list(com[0][:plen]) == toks and np.all(com[0][plen:] == -1)
        assert ctx[0] == 2 + plen and n[0] == plen


@pytest.mark.parametrize("row,plen,want", [
    ([0, 3, 2, 7], 4, [0, 3]),        # not increasing: cut before the 2
    ([0, 3, 9, 12], 4, [0, 3, 9]),    # 12 is not below the budget (10)
    ([0, 3, 5, 7], 9, [0, 3, 5, 7]),  # path_len above block + 1 is clamped
    ([0, 3, 5, 7], 0, [0]),           # path_len below 1 is clamped
    ([5, 6, 7, 8], 2, [0, 6]),        # entry 0 is the root whatever it holds
    ([0, 0, 1, 2], 4, [0]),           # a repeated root ends the path
])
def test_committed_path_cut(row, plen, want):
    assert committed_path(np.array(row), plen, budget=10, block=3) == want


def test_other_requests_and_context_clamp():
    K, V = rows_cache(40)
    token = np.full((2, 8), 5, dtype=np.int32)
    path = np.array([[0, 4, 6], [0, 1, 7]], dtype=np.int32)
    # request 0 owns rows 0..14 (ctx 7 + 8 nodes), request 1 rows 15..39; request 1's
    # ctx_len 20 is clamped to max_ctx 10
    K2, _, ctx, _, _ = kv_commit(K, V, [0, 15], [7, 20], token, path, [3, 3], [1, 2], budget=8,
                                 block=2, max_ctx=10)
    want = np.arange(40, dtype=np.float32)
    want[7:10] = [7, 11, 13]
    want[25:28] = [25, 26, 32]
    assert np.array_equal(K2[:, 0, 0], want)
    assert list(ctx) == [10, 13]


@pytest.mark.parametrize("seed", range(10))
def test_gather_equals_in_place_sequential_move(seed):
    rng = np.random.default_rng(seed)
    budget, block, ctx = 40, 12, 5
    K, V = rows_cache(ctx + budget)
    m = int(rng.integers(1, block + 2))
    nodes = [0] + sorted(rng.choice(np.arange(1, budget), size=m - 1, replace=False).tolist())
    path = np.full((1, block + 1), -1, dtype=np.int32)
    path[0, :m] = nodes
    K2, _, _, _, _ = kv_commit(K, V, [0], [ctx], np.zeros((1, budget), np.int32), path, [m], [0],
                               budget=budget, block=block, max_ctx=ctx)
    seq = K.copy()
    for j, s in enumerate(nodes):        # in place, increasing j
        seq[ctx + j] = seq[ctx + s]
    assert np.array_equal(K2, seq)


@pytest.mark.parametrize("seed", range(10))
def test_commit_after_walk_keeps_the_accepted_rows(seed):
    rng = np.random.default_rng(100 + seed)
    n, block, ctx = 30, 8, 4
    parent = np.array([-1] + [int(rng.integers(max(0, i - 4), i)) for i in range(1, n)])
    token = np.full(n, -1)
    for p in range(n):
        kids = [c for c in range(1, n) if parent[c] == p]
        token[kids] = rng.choice(6, size=len(kids), replace=False) if len(kids) <= 6 else 0
    target = rng.integers(0, 6, size=n)
    p, bonus = accept_walk(parent, token, n, target)
    p = p[:block + 1]
    arr, ln, bn = walk_arrays(p, bonus, block)
    K, V = rows_cache(ctx + n)
    K2, _, newctx, com, m = kv_commit(K, V, [0], [ctx], token[None, :].astype(np.int32),
                                      arr[None, :], [ln], [bn], budget=n, block=block, max_ctx=ctx)
    assert m[0] == len(p) and newctx[0] == ctx + len(p)
    assert list(K2[ctx:ctx + len(p), 0, 0]) == [ctx + s for s in p]
    assert list(com[0][:len(p)]) == [int(token[s]) for s in p[1:]] + [bonus]


@pytest.mark.parametrize("page_rows", [1, 4, 16])
def test_paged_commit_equals_contiguous(page_rows):
    """The paged commit is the contiguous one seen through the block table: pools scattered
    from a contiguous cache at random, committed, and gathered back give the contiguous
    commit's cache, row for row; pages of no request keep their contents."""
    from oracle.commit import kv_commit, kv_commit_paged
    rng = np.random.default_rng(60 + page_rows)
    B, N, D, Hkv, hd = 3, 12, 5, 2, 4
    ctx = np.array([0, 7, 29], dtype=np.int32)
    off = np.concatenate([[0], np.cumsum(ctx + N)[:-1]]).astype(np.int64)
    rows = int(off[-1] + ctx[-1] + N)
    K = rng.standard_normal((rows, Hkv, hd))
    V = rng.standard_normal((rows, Hkv, hd))
    token = rng.integers(0, 1000, (B, N)).astype(np.int32)
    path = np.array([[0, 1, 3, 7, 11, -1], [0, 2, 2, 5, -1, -1], [0, 4, 9, 10, 11, 12]],
                    dtype=np.int32)
    plen = np.array([5, 4, 6], dtype=np.int32)
    bonus = np.array([5, 6, 7], dtype=np.int32)
    want = kv_commit(K, V, off, ctx, token, path, plen, bonus, N, D, int(ctx.max()))
    need = [-(-(int(ctx[b]) + N) // page_rows) for b in range(B)]
    pool = sum(need) + 4
    ids = rng.permutation(pool)
    table = np.zeros((B, max(need)), dtype=np.int32)
    Kp = rng.standard_normal((pool, page_rows, Hkv, hd))
    Vp = rng.standard_normal((pool, page_rows, Hkv, hd))
    k = 0
    for b in range(B):
        for p in range(need[b]):
            table[b, p] = ids[k]
            for r in range(p * page_rows, min(int(ctx[b]) + N, (p + 1) * page_rows)):
                Kp[ids[k], r - p * page_rows] = K[int(off[b]) + r]
                Vp[ids[k], r - p * page_rows] = V[int(off[b]) + r]
            k += 1
    got = kv_commit_paged(Kp, Vp, table, page_rows, ctx, token, path, plen, bonus, N, D,
                          int(ctx.max()))
    for b in range(B):
        for r in range(int(ctx[b]) + N):
            pg, sl = table[b, r // page_rows], r % page_rows
            assert np.array_equal(got[0][pg, sl], want[0][int(off[b]) + r])
            assert np.array_equal(got[1][pg, sl], want[1][int(off[b]) + r])
    for x in ids[k:]:                        # pages no request owns
        assert np.array_equal(got[0][x], Kp[x]) and np.array_equal(got[1][x], Vp[x])
    for g, w in zip(got[2:], want[2:]):
        assert np.array_equal(g, w)

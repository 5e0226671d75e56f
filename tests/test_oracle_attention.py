"""Pins for the tree-attention oracle and the ancestor mask: the library routine
torch.nn.functional.scaled_dot_product_attention in float64 on the CPU with a
boolean mask, plain causal attention for a chain, and closed forms."""
import numpy as np
import pytest
import torch

from oracle.attention import ancestor_sets, tree_attention


def test_mask_chain_is_causal_and_star_is_diagonal_plus_root():
    n = 7
    chain = np.array([-1] + list(range(n - 1)))
    anc = ancestor_sets(chain, n)
    assert anc == [list(range(i + 1)) for i in range(n)]
    star = np.array([-1] + [0] * (n - 1))
    assert ancestor_sets(star, n) == [[0]] + [[0, i] for i in range(1, n)]


def _random_tree(rng, n):
    return np.array([-1] + [int(rng.integers(0, i)) for i in range(1, n)])


def _sdpa_reference(Q, K, V, off, ctx, parent, n, scale, N):
    B, _, Hq, hd = Q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    out = np.full(Q.shape, np.nan)
    for b in range(B):
        R = int(ctx[b]) + N
        rows = slice(int(off[b]), int(off[b]) + R)
        mask = torch.zeros(N, R, dtype=torch.bool)
        mask[:, :int(ctx[b])] = True
        anc = ancestor_sets(parent[b], n[b])
        for i in range(n[b]):
            for a in anc[i]:
                mask[i, int(ctx[b]) + a] = True
        for i in range(n[b], N):
            mask[i, 0] = True     # rows beyond n are not compared
        q = torch.from_numpy(Q[b]).permute(1, 0, 2)                     # [Hq][N][hd]
        k = torch.from_numpy(K[rows]).permute(1, 0, 2).repeat_interleave(G, 0)
        v = torch.from_numpy(V[rows]).permute(1, 0, 2).repeat_interleave(G, 0)
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=scale)
        out[b, :n[b]] = o.permute(1, 0, 2).numpy()[:n[b]]
    return out


@pytest.mark.parametrize("seed", range(3))
def test_tree_attention_against_sdpa(seed):
    rng = np.random.default_rng(seed)
    B, N, Hq, Hkv, hd = 3, 12, 4, 2, 16
    ctx = rng.integers(0, 40, size=B)
    ctx[0] = 0                                           # no context at all
    off = np.concatenate([[0], np.cumsum(ctx + N)[:-1]])
    rows = int(off[-1] + ctx[-1] + N)
    Q = rng.standard_normal((B, N, Hq, hd))
    K = rng.standard_normal((rows, Hkv, hd))
    V = rng.standard_normal((rows, Hkv, hd))
    n = [N, 5, 1]
    parents = [_random_tree(rng, N) for _ in range(B)]
    scale = 0.37
    O = tree_attention(Q, K, V, off, ctx, parents, n, scale)
    ref = _sdpa_reference(Q, K, V, off, ctx, parents, n, scale, N)
    for b in range(B):
        np.testing.assert_allclose(O[b, :n[b]], ref[b, :n[b]], rtol=1e-12, atol=1e-12)
        assert np.all(np.isnan(O[b, n[b]:]))


def test_chain_tree_is_causal_attention():
    rng = np.random.default_rng(9)
    N, Hq, Hkv, hd, ctx = 6, 2, 1, 8, 10
    Q = rng.standard_normal((1, N, Hq, hd))
    K = rng.standard_normal((ctx + N, Hkv, hd))
    V = rng.standard_normal((ctx + N, Hkv, hd))
    chain = np.array([-1] + list(range(N - 1)))
    O = tree_attention(Q, K, V, np.array([0]), np.array([ctx]), [chain], [N], 0.5)
    # causal attention of the N tree queries over the ctx+N rows, queries at positions ctx..ctx+N-1
    q = torch.from_numpy(Q[0]).permute(1, 0, 2)
    k = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(Hq, 0)
    v = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(Hq, 0)
    causal = torch.ones(N, ctx + N, dtype=torch.bool).tril(diagonal=ctx)
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=causal, scale=0.5)
    np.testing.assert_allclose(O[0], ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-12)


def test_identical_values_give_that_value():
    rng = np.random.default_rng(4)
    N, Hq, Hkv, hd, ctx = 5, 4, 2, 8, 7
    Q = rng.standard_normal((1, N, Hq, hd)) * 3
    K = rng.standard_normal((ctx + N, Hkv, hd))
    row = rng.standard_normal((Hkv, hd))
    V = np.broadcast_to(row, (ctx + N, Hkv, hd)).copy()
    O = tree_attention(Q, K, V, np.array([0]), np.array([ctx]), [_random_tree(rng, N)], [N], 1.0)
    for h in range(Hq):
        np.testing.assert_allclose(O[0, :, h], np.broadcast_to(row[h // 2], (N, hd)), rtol=1e-13)


def test_single_node_is_decode_attention():
    rng = np.random.default_rng(5)
    Hq, Hkv, hd, ctx = 4, 4, 8, 20
    Q = rng.standard_normal((1, 3, Hq, hd))
    K = rng.standard_normal((ctx + 3, Hkv, hd))
    V = rng.standard_normal((ctx + 3, Hkv, hd))
    O = tree_attention(Q, K, V, np.array([0]), np.array([ctx]), [np.array([-1, 0, 0])], [1], 0.25)
    for h in range(Hq):
        s = 0.25 * K[:ctx + 1, h] @ Q[0, 0, h]
        p = np.exp(s - s.max())
        np.testing.assert_allclose(O[0, 0, h], (p / p.sum()) @ V[:ctx + 1, h], rtol=1e-13)


def _scatter_to_pages(K, V, off, ctx, N, page_rows, pool_pages, rng):
    """Write each request's logical rows (ctx + N of them, from row off[b] of the contiguous
    caches K and V) page by page into randomly chosen distinct pages of NaN-filled pools."""
    B = len(ctx)
    need = [-(-(int(ctx[b]) + N) // page_rows) for b in range(B)]
    ids = rng.permutation(pool_pages)[:sum(need)]
    table = np.full((B, max(need) + 2), -7, dtype=np.int32)   # entries past a request: junk
    Kp = np.full((pool_pages, page_rows) + K.shape[1:], np.nan)
    Vp = np.full_like(Kp, np.nan)
    k = 0
    for b in range(B):
        rows = int(ctx[b]) + N
        for p in range(need[b]):
            table[b, p] = ids[k]
            lo, hi = p * page_rows, min(rows, (p + 1) * page_rows)
            Kp[ids[k], :hi - lo] = K[int(off[b]) + lo:int(off[b]) + hi]
            Vp[ids[k], :hi - lo] = V[int(off[b]) + lo:int(off[b]) + hi]
            k += 1
    return Kp, Vp, table


@pytest.mark.parametrize("page_rows", [1, 4, 32])
def test_paged_oracle_equals_contiguous(page_rows):
    """The paged form gathers exactly the rows of the contiguous layout: pages scattered at
    random over NaN-filled pools, with junk table entries past each request, give the same
    O as the contiguous cache, bit for bit, for two different page assignments."""
    from oracle.attention import tree_attention_paged
    rng = np.random.default_rng(91 + page_rows)
    B, N, Hq, Hkv, hd = 3, 9, 4, 2, 8
    ctx = np.array([0, 5, 37], dtype=np.int32)
    off = np.concatenate([[0], np.cumsum(ctx + N)[:-1]]).astype(np.int64)
    rows = int(off[-1] + ctx[-1] + N)
    Q = rng.standard_normal((B, N, Hq, hd))
    K = rng.standard_normal((rows, Hkv, hd))
    V = rng.standard_normal((rows, Hkv, hd))
    parents = [np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)
               for _ in range(B)]
    n = [N, 4, 7]
    ref = tree_attention(Q, K, V, off, ctx, parents, n, 0.3)
    for trial in range(2):
        pool_pages = 3 * (rows // page_rows + B + 1)
        Kp, Vp, table = _scatter_to_pages(K, V, off, ctx, N, page_rows, pool_pages, rng)
        got = tree_attention_paged(Q, Kp, Vp, table, page_rows, ctx, parents, n, 0.3)
        for b in range(B):
            assert np.array_equal(got[b, :n[b]], ref[b, :n[b]]), (page_rows, trial, b)

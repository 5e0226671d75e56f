"""GPU parity of the paged tree attention (tree_verify_attn_paged) through the C ABI.

Each request's logical cache rows (its context, then one row per tree node) are scattered
page by page into random distinct pages of pools whose other pages hold NaN bits, and the
block-table entries past a request's pages hold junk ids (negative, or past the pool), so
a wrong page or slot, or a read of an entry the request does not reach, shows up.  The
result is compared with the oracle's paged form (bf16 bounds as for the contiguous call),
and, for the identity layout, bit for bit with the contiguous call."""
import sys

import numpy as np
import pytest
import torch

import oracle
from tests import _util as U
from workloads import BF16, bf16_bits_to_f32, f32_to_bf16_bits, gen_round, kv_offsets

pytestmark = pytest.mark.gpu

NAN_BF16 = np.uint16(0x7FC0)


@pytest.fixture(scope="module")
def taps():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_00487_amd as taps
    taps.load()
    return taps


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_pages(K, V, off, ctx, N, page_rows, rng, spare=7):
    """Scatter request b's ctx[b] + N logical rows (from row off[b] of the contiguous bf16
    caches K, V) page by page into random distinct pages of NaN-filled pools; `spare` pages
    stay unused.  Returns the pools [pages][page_rows][Hkv][hd] and the block table."""
    B = len(ctx)
    need = [-(-(int(ctx[b]) + N) // page_rows) for b in range(B)]
    num_pages = sum(need) + spare
    ids = rng.permutation(num_pages)[:sum(need)]
    max_pages = max(need) + 3
    table = np.where(rng.random((B, max_pages)) < 0.5, -5, num_pages + 1000).astype(np.int32)
    Kp = np.full((num_pages, page_rows) + K.shape[1:], NAN_BF16, dtype=np.uint16)
    Vp = np.full_like(Kp, NAN_BF16)
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


def run_paged(taps, Q, Kp, Vp, table, page_rows, ctx, parents, n, Hq, Hkv, max_ctx):
    B, N = Q.shape[0], Q.shape[1]
    att = taps.PagedTreeAttention(B, N, Hq, Hkv, max_ctx, page_rows, scale=128 ** -0.5)
    att.ws.fill_(0xFF)            # NaN bits in every unwritten partial slot
    O = att(U.to_dev(Q, True), U.to_dev(Kp, True), U.to_dev(Vp, True),
            torch.from_numpy(table).cuda(), torch.from_numpy(ctx).cuda(),
            torch.from_numpy(np.stack(parents)).cuda(), torch.tensor(n, dtype=torch.int32).cuda())
    torch.cuda.synchronize()
    return O


def paged_ref(Q, Kp, Vp, table, page_rows, ctx, parents, n, samples=None):
    f = lambda a: bf16_bits_to_f32(a).astype(np.float64)   # noqa: E731
    return oracle.tree_attention_paged(f(Q), f(Kp), f(Vp), table, page_rows, ctx, parents, n,
                                       128 ** -0.5, samples=samples)


def random_inputs(rng, B, N, Hq, Hkv, ctx):
    hd = 128
    off = kv_offsets(ctx, N)
    rows = int(off[-1] + ctx[-1] + N)
    Q = f32_to_bf16_bits(rng.standard_normal((B, N, Hq, hd)).astype(np.float32))
    K = f32_to_bf16_bits(rng.standard_normal((rows, Hkv, hd)).astype(np.float32))
    V = f32_to_bf16_bits(rng.standard_normal((rows, Hkv, hd)).astype(np.float32))
    return Q, K, V, off


@pytest.mark.parametrize("page_rows,ctx,N,Hq,Hkv", [
    (32, [0, 1, 77, 300], 130, 8, 2),        # one-stage pages; a 130-node chain, a star
    (64, [3001, 1777], 64, 16, 4),           # several key splits, a ragged last one
    (256, [5000, 20, 2047], 64, 32, 8),      # the ragged work list over pages
    (4096, [700], 33, 8, 8),                 # one page holds the whole request
])
def test_paged_attention_matches_oracle(taps, page_rows, ctx, N, Hq, Hkv):
    rng = np.random.default_rng(page_rows + N)
    ctx = np.array(ctx, dtype=np.int32)
    B = len(ctx)
    say(f"[paged] page_rows={page_rows} ctx={ctx.tolist()} N={N} Hq={Hq} Hkv={Hkv}")
    Q, K, V, off = random_inputs(rng, B, N, Hq, Hkv, ctx)
    kinds = [np.array([-1] + list(range(N - 1)), dtype=np.int32),            # chain
             np.array([-1] + [0] * (N - 1), dtype=np.int32)]                 # star
    parents = [kinds[b] if b < 2 and page_rows == 32 else
               np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)
               for b in range(B)]
    n = [N if b != 1 else max(1, N // 3) for b in range(B)]
    Kp, Vp, table = to_pages(K, V, off, ctx, N, page_rows, rng)
    O = run_paged(taps, Q, Kp, Vp, table, page_rows, ctx, parents, n, Hq, Hkv, int(ctx.max()))
    ref = paged_ref(Q, Kp, Vp, table, page_rows, ctx, parents, n)
    got = U.gpu_o_as_f64(O)
    for b in range(B):
        U.attention_error(got[b, :n[b]], ref[b, :n[b]], BF16,
                          f"paged page_rows={page_rows} b={b} ctx={ctx[b]} n={n[b]}")


def test_paged_identity_layout_equals_contiguous(taps):
    """The Qwen3-8B round's cache cut into 64-row pages in order (block table 0, 1, 2, ...)
    gives exactly the contiguous call's output: the same plan, loads and arithmetic."""
    inp = gen_round("qwen3_8b")
    c = inp.cfg
    trees = U.oracle_trees(inp)
    parent, _, n = U.tree_device(trees)
    rows = int(inp.ctx_len[0]) + c.budget
    assert rows % 64 == 0 and inp.K.shape[0] == rows
    say(f"[paged-identity] qwen3_8b rows={rows}")
    Q, K, V = (U.to_dev(a, True) for a in (inp.Q, inp.K, inp.V))
    att = taps.TreeAttention(c.batch, c.budget, c.Hq, c.Hkv, c.head_dim, int(inp.ctx_len[0]),
                             dtype=c.dtype, scale=c.scale)
    O_c = att(Q, K, V, torch.from_numpy(inp.kv_offset).cuda(), torch.from_numpy(inp.ctx_len).cuda(),
              parent, n)
    patt = taps.PagedTreeAttention(c.batch, c.budget, c.Hq, c.Hkv, int(inp.ctx_len[0]), 64,
                                   scale=c.scale)
    table = torch.arange(rows // 64, dtype=torch.int32).reshape(1, -1).cuda()
    O_p = patt(Q, K.reshape(rows // 64, 64, c.Hkv, c.head_dim),
               V.reshape(rows // 64, 64, c.Hkv, c.head_dim), table,
               torch.from_numpy(inp.ctx_len).cuda(), parent, n)
    torch.cuda.synchronize()
    nn = int(trees[0].n)
    assert torch.equal(O_p[:, :nn], O_c[:, :nn])


def test_paged_tree_rows_dominate_at_full_size(taps):
    """The Qwen3-8B shape (context 8192, 64 nodes, the bench's key splits) over 128-row pages
    in random order, with a common direction in every query and in the tree rows' keys so
    that each node's ancestors carry almost all of its softmax mass: a wrong page of the
    tree rows, or a wrong mask bit in the last split, moves O by O(1).  Every row."""
    inp = gen_round("qwen3_8b")
    c = inp.cfg
    trees = U.oracle_trees(inp)
    rng = np.random.default_rng(78)
    w = rng.standard_normal((c.Hkv, c.head_dim))
    w /= np.linalg.norm(w, axis=1, keepdims=True)
    G = c.Hq // c.Hkv
    Qf = bf16_bits_to_f32(inp.Q).astype(np.float64) + 16.0 * np.repeat(w, G, axis=0)[None, None]
    Kf = bf16_bits_to_f32(inp.K).astype(np.float64)
    ctx = int(inp.ctx_len[0])
    Kf[ctx:ctx + c.budget] += 16.0 * w[None]
    Q, K = f32_to_bf16_bits(Qf.astype(np.float32)), f32_to_bf16_bits(Kf.astype(np.float32))
    say("[paged-tree-dominant] qwen3_8b shape, 128-row pages")
    Kp, Vp, table = to_pages(K, inp.V, inp.kv_offset, inp.ctx_len, c.budget, 128, rng)
    parents = [t.parent for t in trees]
    n = [t.n for t in trees]
    O = run_paged(taps, Q, Kp, Vp, table, 128, inp.ctx_len, parents, n, c.Hq, c.Hkv, ctx)
    ref = paged_ref(Q, Kp, Vp, table, 128, inp.ctx_len, parents, n)
    U.attention_error(U.gpu_o_as_f64(O), ref, BF16, "paged tree-dominant qwen3_8b")


@pytest.mark.parametrize("name,page_rows,samples", [("serve16", 64, 384), ("stress", 256, 192)])
def test_paged_full_size(taps, name, page_rows, samples):
    """The 16-request serving shape (contexts of 512 to 16K rows, 128 nodes each, the ragged
    work list) and the 4-request stress shape (32K-row contexts, 256 nodes: four-word
    ancestor masks) over pages in random order, on sampled (node, head) rows plus the root
    and the deepest node of every request."""
    inp = gen_round(name)
    c = inp.cfg
    trees = U.oracle_trees(inp)
    rng = np.random.default_rng(80)
    say(f"[paged-full] {name}, {page_rows}-row pages")
    Kp, Vp, table = to_pages(inp.K, inp.V, inp.kv_offset, inp.ctx_len, c.budget, page_rows, rng)
    parents = [t.parent for t in trees]
    n = [t.n for t in trees]
    O = run_paged(taps, inp.Q, Kp, Vp, table, page_rows, inp.ctx_len, parents, n, c.Hq, c.Hkv,
                  int(inp.ctx_len.max()))
    pick = []
    for _ in range(samples):
        b = int(rng.integers(0, c.batch))
        pick.append((b, int(rng.integers(0, trees[b].n)), int(rng.integers(0, c.Hq))))
    for b, t in enumerate(trees):
        pick.append((b, 0, 0))
        pick.append((b, int(np.argmax(t.depth[:t.n])), c.Hq - 1))
    ref = paged_ref(inp.Q, Kp, Vp, table, page_rows, inp.ctx_len, parents, n, samples=pick)
    U.attention_error(U.gpu_o_as_f64(O), ref, BF16, f"paged {name}")


@pytest.mark.parametrize("seed", range(4))
def test_paged_attention_fuzz(taps, seed):
    """Seeded batches: 1-4 requests, contexts from empty to 4000 rows (max_ctx above them
    all), 1-80 nodes with random parents, 1-4 KV heads of 1-4 query heads, pages of 32 to
    1024 rows; sampled (node, head) rows of every request."""
    rng = np.random.default_rng(700 + seed)
    B = int(rng.integers(1, 5))
    N = int(rng.integers(1, 81))
    Hkv = int(rng.choice([1, 2, 4]))
    Hq = Hkv * int(rng.choice([1, 2, 4]))
    page_rows = int(rng.choice([32, 64, 128, 256, 1024]))
    ctx = rng.integers(0, 4001, B).astype(np.int32)
    n = [int(x) for x in rng.integers(0, N + 1, B)]
    n[int(rng.integers(0, B))] = N
    max_ctx = int(ctx.max()) + int(rng.integers(0, 300))
    say(f"[paged-fuzz] seed={seed} B={B} N={N} Hq={Hq} Hkv={Hkv} page_rows={page_rows} "
        f"ctx={ctx.tolist()} n={n} max_ctx={max_ctx}")
    Q, K, V, off = random_inputs(rng, B, N, Hq, Hkv, ctx)
    parents = [np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)
               for _ in range(B)]
    Kp, Vp, table = to_pages(K, V, off, ctx, N, page_rows, rng)
    # the table must cover max_ctx + N rows for every request: widen it with junk entries
    wide = -(-(max_ctx + N) // page_rows)
    if table.shape[1] < wide:
        table = np.concatenate([table, np.full((B, wide - table.shape[1]), -3, np.int32)], 1)
    O = run_paged(taps, Q, Kp, Vp, table, page_rows, ctx, parents, n, Hq, Hkv, max_ctx)
    picks = [(b, int(i), int(h)) for b in range(B) if n[b]
             for i in sorted({0, n[b] - 1, *rng.integers(0, n[b], 6).tolist()})
             for h in sorted({0, Hq - 1, int(rng.integers(0, Hq))})]
    ref = paged_ref(Q, Kp, Vp, table, page_rows, ctx, parents, n, samples=picks)
    got = U.gpu_o_as_f64(O)
    for b in range(B):
        if n[b]:
            U.attention_error(got[b, :n[b]], ref[b, :n[b]], BF16,
                              f"paged fuzz b={b} ctx={ctx[b]} page_rows={page_rows}")


def test_paged_timed_call_matches_and_times(taps):
    """tree_verify_attn_paged_timed gives the untimed call's output bit for bit, and its
    events bracket the main kernel (a positive duration)."""
    rng = np.random.default_rng(9)
    ctx = np.array([1500, 300], dtype=np.int32)
    N, Hq, Hkv = 48, 16, 4
    Q, K, V, off = random_inputs(rng, 2, N, Hq, Hkv, ctx)
    parents = [np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)
               for _ in range(2)]
    n = [N, 20]
    Kp, Vp, table = to_pages(K, V, off, ctx, N, 64, rng)
    O1 = run_paged(taps, Q, Kp, Vp, table, 64, ctx, parents, n, Hq, Hkv, int(ctx.max()))
    att = taps.PagedTreeAttention(2, N, Hq, Hkv, int(ctx.max()), 64, scale=128 ** -0.5)
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    for e in ev:                  # materialise the handles; the library records them again
        e.record()
    torch.cuda.synchronize()
    O2 = att(U.to_dev(Q, True), U.to_dev(Kp, True), U.to_dev(Vp, True),
             torch.from_numpy(table).cuda(), torch.from_numpy(ctx).cuda(),
             torch.from_numpy(np.stack(parents)).cuda(), torch.tensor(n, dtype=torch.int32).cuda(),
             events=ev)
    torch.cuda.synchronize()
    for b in range(2):
        assert torch.equal(O1[b, :n[b]], O2[b, :n[b]])
    assert ev[0].elapsed_time(ev[1]) > 0


# ------------------------------------------------------------------ paged KV commit
def run_commit_paged(taps, Kp, Vp, table, page_rows, ctx, token, path, plen, bonus, budget,
                     block, Hkv, hd, max_ctx, dtype):
    bf = dtype == BF16
    Kd, Vd = U.to_dev(Kp, bf), U.to_dev(Vp, bf)
    batch = len(ctx)
    tb = taps.TreeBuffers.empty(batch, block, 1, budget)
    tb.token.copy_(torch.from_numpy(token.astype(np.int32)).cuda())
    com = taps.PagedKVCommit(batch, budget, block, Hkv, hd, max_ctx, page_rows, dtype=dtype)
    nc, cm, n = com(Kd, Vd, torch.from_numpy(table).cuda(),
                    torch.from_numpy(ctx.astype(np.int32)).cuda(), tb,
                    torch.from_numpy(path.astype(np.int32)).cuda(),
                    torch.from_numpy(plen.astype(np.int32)).cuda(),
                    torch.from_numpy(bonus.astype(np.int32)).cuda())
    torch.cuda.synchronize()
    bits = (lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)) if bf else \
        (lambda t: t.cpu().numpy())
    return bits(Kd), bits(Vd), nc.cpu().numpy(), cm.cpu().numpy(), n.cpu().numpy()


@pytest.mark.parametrize("name,page_rows", [("qwen3_8b", 64), ("serve16", 32), ("stress", 256)])
def test_paged_commit_matches_oracle_after_walk(taps, name, page_rows):
    """kv_commit_paged after the oracle's walk (branching targets) on pools scattered at
    random: pools, new context lengths and emitted tokens equal the oracle's byte for byte
    (untouched pages included)."""
    say(f"[paged-commit] {name} page_rows={page_rows}")
    inp = gen_round(name)
    c = inp.cfg
    trees = U.oracle_trees(inp)
    tgt = U.targets_for(inp, trees, branch=True)
    from oracle.walk import walk_arrays
    path = np.full((c.batch, c.block + 1), -1, np.int32)
    plen = np.zeros(c.batch, np.int32)
    bonus = np.zeros(c.batch, np.int32)
    for b, t in enumerate(trees):
        p, bo = oracle.accept_walk(t.parent, t.token, t.n, tgt[b])
        path[b], plen[b], bonus[b] = walk_arrays(p, bo, c.block)
    token = np.stack([t.token for t in trees])
    max_ctx = int(inp.ctx_len.max())
    rng = np.random.default_rng(page_rows)
    Kp, Vp, table = to_pages(inp.K, inp.V, inp.kv_offset, inp.ctx_len, c.budget, page_rows, rng)
    wide = -(-(max_ctx + c.budget) // page_rows)
    if table.shape[1] < wide:
        table = np.concatenate([table, np.full((c.batch, wide - table.shape[1]), -3, np.int32)], 1)
    got = run_commit_paged(taps, Kp, Vp, table, page_rows, inp.ctx_len, token, path, plen, bonus,
                           c.budget, c.block, c.Hkv, c.head_dim, max_ctx, BF16)
    want = oracle.kv_commit_paged(Kp, Vp, table, page_rows, inp.ctx_len, token, path, plen,
                                  bonus, c.budget, c.block, max_ctx)
    for nm, g, w in zip(("K", "V", "new_ctx", "committed", "n"), got, want):
        assert g.shape == w.shape and np.array_equal(g, w), nm
    assert int(want[4].max()) > 1                     # some request accepted drafted nodes


def test_paged_commit_edge_paths(taps):
    """Root only, the longest chain, malformed and clamped paths, a context clamped to
    max_ctx, over 32-row pages (a path crosses pages), fp32 and head_dim 64."""
    from workloads import FP32
    rng = np.random.default_rng(6)
    budget, block, Hkv, hd = 40, 12, 2, 64
    ctx = np.array([0, 7, 33, 100, 5, 64, 9], dtype=np.int32)
    max_ctx = 64
    B = len(ctx)
    off = np.concatenate([[0], np.cumsum(ctx.astype(np.int64) + budget)[:-1]])
    rows = int(off[-1] + ctx[-1] + budget)
    K = rng.standard_normal((rows, Hkv, hd)).astype(np.float32)
    V = rng.standard_normal((rows, Hkv, hd)).astype(np.float32)
    # pools hold each request's rows for its clamped context
    ctx_c = np.minimum(ctx, max_ctx)
    off_c = off + (ctx - ctx_c)            # the clamped request's rows start later in K
    need = [-(-(int(ctx_c[b]) + budget) // 32) for b in range(B)]
    npages = sum(need) + 5
    ids = rng.permutation(npages)
    table = np.full((B, -(-(max_ctx + budget) // 32)), -9, np.int32)
    Kp = rng.standard_normal((npages, 32, Hkv, hd)).astype(np.float32)
    Vp = rng.standard_normal((npages, 32, Hkv, hd)).astype(np.float32)
    k = 0
    for b in range(B):
        for p in range(need[b]):
            table[b, p] = ids[k]
            lo, hi = p * 32, min(int(ctx_c[b]) + budget, (p + 1) * 32)
            Kp[ids[k], :hi - lo] = K[int(off_c[b]) + lo:int(off_c[b]) + hi]
            Vp[ids[k], :hi - lo] = V[int(off_c[b]) + lo:int(off_c[b]) + hi]
            k += 1
    token = rng.integers(0, 1000, size=(B, budget)).astype(np.int32)
    path = np.full((B, block + 1), -1, np.int32)
    plen = np.zeros(B, np.int32)
    path[0, 0] = 0; plen[0] = 1                                       # root only
    path[1] = np.arange(block + 1); plen[1] = block + 1               # chain, identity moves
    path[2] = [0] + sorted(rng.choice(np.arange(1, budget), size=block, replace=False).tolist())
    plen[2] = block + 1                                               # longest scattered path
    path[3, :5] = [0, 3, 9, 9, 20]; plen[3] = 5                       # repeat: cut after 9
    path[4, :4] = [0, 2, 45, 46]; plen[4] = 4                         # beyond the budget: cut
    path[5, :3] = [0, 1, 39]; plen[5] = 99                            # length clamped
    path[6, :3] = [0, 4, 8]; plen[6] = 0                              # length clamped to 1
    bonus = rng.integers(0, 1000, size=B).astype(np.int32)
    got = run_commit_paged(taps, Kp, Vp, table, 32, ctx, token, path, plen, bonus, budget, block,
                           Hkv, hd, max_ctx, FP32)
    want = oracle.kv_commit_paged(Kp, Vp, table, 32, ctx, token, path, plen, bonus, budget,
                                  block, max_ctx)
    for nm, g, w in zip(("K", "V", "new_ctx", "committed", "n"), got, want):
        assert g.shape == w.shape and np.array_equal(g, w), nm
    assert list(want[4]) == [1, 13, 13, 3, 2, 3, 1]


# ------------------------------------------------------------------ paged layer slice
def _run_layer_paged(taps, rng, B, N, H, Hq, Hkv, ctx, n, page_rows, sample_nodes=None):
    """verify_layer_paged against the oracle's paged layer: Y within the layer tolerance, the
    written node rows within it too, every other pool row untouched (bit for bit)."""
    from oracle.layer import bf16_round, verify_layer_paged
    from tests.test_gpu_layer import TOL, _bf16, _to_dev, _tree
    hd = 128
    X = _bf16(rng, B, N, H)
    Wq = _bf16(rng, Hq * hd, H, scale=H ** -0.5)
    Wk = _bf16(rng, Hkv * hd, H, scale=H ** -0.5)
    Wv = _bf16(rng, Hkv * hd, H, scale=H ** -0.5)
    Wo = _bf16(rng, H, Hq * hd, scale=(Hq * hd) ** -0.5)
    qn = bf16_round(1 + 0.1 * rng.standard_normal(hd))
    kn = bf16_round(1 + 0.1 * rng.standard_normal(hd))
    ctx = np.array(ctx, np.int32)
    n = np.array(n, np.int32)
    max_ctx = int(ctx.max())
    need = [-(-(int(ctx[b]) + N) // page_rows) for b in range(B)]
    npages = sum(need) + 3
    ids = rng.permutation(npages)
    table = np.full((B, -(-(max_ctx + N) // page_rows)), -4, np.int32)
    k = 0
    for b in range(B):
        table[b, :need[b]] = ids[k:k + need[b]]
        k += need[b]
    Kp, Vp = _bf16(rng, npages, page_rows, Hkv, hd), _bf16(rng, npages, page_rows, Hkv, hd)
    trees = [_tree(rng, N, int(n[b])) for b in range(B)]
    parent = np.stack([t[0] for t in trees])
    depth = np.stack([t[1] for t in trees])
    samples = None
    if sample_nodes is not None:
        samples = [(b, i, h) for b in range(B) for i in sample_nodes(b) for h in range(Hq)]
    say(f"[layer-paged] B={B} N={N} H={H} Hq={Hq} Hkv={Hkv} ctx={ctx.tolist()} n={n.tolist()} "
        f"page_rows={page_rows}")
    Y, Ko, Vo, _, _ = verify_layer_paged(X, Wq, Wk, Wv, Wo, qn, kn, Kp, Vp, table, page_rows,
                                         ctx, depth, parent, n, Hq, Hkv, hd, 1e6, 1e-6,
                                         hd ** -0.5, samples=samples)
    w = taps.LayerWeights(_to_dev(Wq, torch.bfloat16), _to_dev(Wk, torch.bfloat16),
                          _to_dev(Wv, torch.bfloat16), _to_dev(Wo, torch.bfloat16),
                          _to_dev(qn, torch.bfloat16), _to_dev(kn, torch.bfloat16))
    tree = taps.TreeBuffers.empty(B, 1, 1, N)
    tree.parent.copy_(torch.from_numpy(parent))
    tree.depth.copy_(torch.from_numpy(depth))
    tree.n_nodes.copy_(torch.from_numpy(n))
    Kd, Vd = _to_dev(Kp, torch.bfloat16), _to_dev(Vp, torch.bfloat16)
    lay = taps.PagedVerifyLayer(B, N, Hq, Hkv, hd, H, max_ctx, page_rows)
    Yd = lay(_to_dev(X, torch.bfloat16), w, Kd, Vd, torch.from_numpy(table).cuda(),
             torch.from_numpy(ctx).cuda(), tree)
    torch.cuda.synchronize()
    Yg = Yd.float().cpu().numpy().astype(np.float64)
    Kg = Kd.float().cpu().numpy().astype(np.float64)
    Vg = Vd.float().cpu().numpy().astype(np.float64)
    written = np.zeros(Kp.shape[:2], bool)
    for b in range(B):
        for i in range(int(n[b])):
            r = int(ctx[b]) + i
            written[table[b, r // page_rows], r % page_rows] = True
    assert np.array_equal(Kg[~written], Kp[~written]) and np.array_equal(Vg[~written], Vp[~written])
    ek = np.abs(Kg[written] - Ko[written]).max() if written.any() else 0.0
    ev = np.abs(Vg[written] - Vo[written]).max() if written.any() else 0.0
    err = 0.0
    for b in range(B):
        for i in (range(int(n[b])) if sample_nodes is None else sample_nodes(b)):
            err = max(err, float(np.abs(Yg[b, i] - Y[b, i]).max()))
    ymax = max(float(np.nanmax(np.abs(Y))), 1.0)
    say(f"[layer-paged] max-abs: Y {err:.2e} (|Y| <= {ymax:.2f}), K rows {ek:.2e}, V rows {ev:.2e}")
    assert err <= TOL * ymax and ek <= TOL and ev <= TOL


@pytest.mark.parametrize("page_rows", [32, 128])
def test_paged_layer_matches_oracle(taps, page_rows):
    """Three requests (contexts 70, 129, 5; 40-node trees, two partly filled) over pages
    in random order, the node rows crossing page boundaries."""
    _run_layer_paged(taps, np.random.default_rng(page_rows), B=3, N=40, H=512, Hq=8, Hkv=2,
                     ctx=[70, 129, 5], n=[40, 23, 31], page_rows=page_rows)


def test_paged_layer_qwen3_8b_shape(taps):
    """The Qwen3-8B layer shape (hidden 4096, 32/8 heads, 64 nodes, context 8192) over
    64-row pages, on sampled nodes."""
    _run_layer_paged(taps, np.random.default_rng(88), B=1, N=64, H=4096, Hq=32, Hkv=8,
                     ctx=[8192], n=[64], page_rows=64, sample_nodes=lambda b: [0, 1, 17, 63])

"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Trees, top-K indices and accepted paths must match bit for bit; attention must
be within 2e-2 max-abs (bf16 inputs, fp32 accumulation) or 1e-4 (fp32) of the
fp64 oracle.  The configurations run in the launch configuration the bench
times (the plan is a pure function of the sizes)."""
import sys

import numpy as np
import pytest
import torch

import oracle
from tests import _util as U
from workloads import BF16, CONFIGS, FP32, LOGITS, PROBS, Config, gen_round, kv_offsets

pytestmark = pytest.mark.gpu

TOL = {BF16: 2e-2, FP32: 1e-4}


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


def run_select(taps, inp, tree=None, **over):
    c = inp.cfg
    kw = dict(kind=c.kind, lambda1=c.lambda1, lambda2=c.lambda2, tau=c.tau, beta=c.beta)
    kw.update(over)
    sel = taps.Selector(c.batch, c.block, c.vocab, c.K, c.budget, dtype=c.dtype, **kw)
    m = U.to_dev(inp.marginals, c.dtype == BF16)
    out = sel(m)
    torch.cuda.synchronize()
    return out, sel, m


# ------------------------------------------------------------------ selection
@pytest.mark.parametrize("name", ["tiny", "qwen3_4b", "qwen3_8b", "serve16", "stress"])
def test_select_matches_oracle(taps, name):
    say(f"[select] {name}")
    inp = gen_round(name, with_attention=False)
    gpu, _, _ = run_select(taps, inp)
    U.assert_tree_equal(gpu, U.oracle_trees(inp), inp.cfg)


def _fuzz_cfg(rng, dtype, kind, V, D, K, N, B=2):
    return Config("fuzz", 9, B, D, V, K, N, 4, 2, 64, 16, kind, dtype, 1.0, 0.0, 0.0, 0.7)


def _fuzz_marginals(rng, cfg, mode):
    B, D, V = cfg.batch, cfg.block, cfg.vocab
    if mode == "ties":
        x = rng.integers(-4, 4, size=(B, D, V)).astype(np.float32) * 0.5
    elif mode == "deep":
        x = rng.standard_normal((B, D, V)).astype(np.float32)
        x[:, :, 3] += 30.0                        # rank 0 dominates: a deep chain
    elif mode == "specials":
        x = rng.standard_normal((B, D, V)).astype(np.float32)
        x[:, 0, :] = -np.inf                      # a row with nothing finite
        x[:, 1, :5] = np.nan
        x[:, 1, 7] = np.inf if cfg.kind == PROBS else 5.0
        x[:, 2, ::3] = -0.0
        x[:, 2, 1::3] = 0.0
        if D > 3:
            x[:, 3, :] = np.nan                   # an all-NaN row
    else:
        x = rng.standard_normal((B, D, V)).astype(np.float32) * 2
    if cfg.kind == PROBS:
        x = np.where(np.isnan(x), x, np.abs(x)).astype(np.float32)
    from workloads import f32_to_bf16_bits
    return f32_to_bf16_bits(x) if cfg.dtype == BF16 else x


@pytest.mark.parametrize("budget,lam2,tau", [(64, 0.0, 0.0), (128, 0.125, 0.0), (256, 0.125, 0.0),
                                            (256, 0.0, 0.0)])
def test_select_ablation_and_budget_variants(taps, budget, lam2, tau):
    """The pruning ablation (lambda2 = 0 and tau = 0: the budget is filled by reach alone)
    and the points of the budget sweep, on the Qwen3-8B marginals."""
    import dataclasses
    c = dataclasses.replace(CONFIGS["qwen3_8b"], budget=budget, lambda2=lam2, tau=tau)
    say(f"[select-variant] budget={budget} lambda2={lam2} tau={tau}")
    inp = gen_round(c, with_attention=False)
    trees = U.oracle_trees(inp)
    gpu, _, _ = run_select(taps, inp)
    U.assert_tree_equal(gpu, trees, c)


@pytest.mark.parametrize("name", ["tiny", "qwen3_4b", "qwen3_8b", "stress"])
def test_select_marginal_scorer_matches_oracle(taps, name):
    """The scoring ablation: q_cond is the full-vocabulary marginal (the exact integer
    normaliser for logits, the probability itself for probabilities)."""
    say(f"[select-marginal] {name}")
    inp = gen_round(name, with_attention=False)
    c = inp.cfg
    trees = U.oracle_trees(inp, scorer=oracle.select.MARGINAL)
    gpu, _, _ = run_select(taps, inp, scorer=1)
    U.assert_tree_equal(gpu, trees, c)


@pytest.mark.parametrize("seed", range(12))
def test_select_marginal_fuzz(taps, seed):
    rng = np.random.default_rng(900 + seed)
    dtype = [BF16, FP32][seed % 2]
    kind = [LOGITS, LOGITS, PROBS][seed % 3]
    V = int(rng.choice([17, 1001, 70001]))
    K = min(int(rng.integers(1, 17)), V)
    D = int(rng.integers(1, 33))
    N = int(rng.choice([1, 16, 64, 200]))
    mode = ["ties", "deep", "specials", "plain"][seed % 4]
    cfg = _fuzz_cfg(rng, dtype, kind, V, D, K, N)
    say(f"[fuzz-marginal] seed={seed} dtype={dtype} kind={kind} V={V} K={K} D={D} N={N} "
        f"mode={mode}")
    m = _fuzz_marginals(rng, cfg, mode)
    from workloads import bf16_bits_to_f32
    x = bf16_bits_to_f32(m).astype(np.float64) if dtype == BF16 else m.astype(np.float64)
    trees = [oracle.select_request(x[b], K, N, kind=kind, scorer=oracle.select.MARGINAL)
             for b in range(cfg.batch)]
    sel = taps.Selector(cfg.batch, D, V, K, N, dtype=dtype, kind=kind, scorer=1)
    gpu = sel(U.to_dev(m, dtype == BF16))
    torch.cuda.synchronize()
    U.assert_tree_equal(gpu, trees, cfg)


def _learned_weights(taps, mlp):
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return taps.ScorerWeights(emb=dev(mlp.emb), W1=dev(mlp.W1), b1=dev(mlp.b1), w2=dev(mlp.w2),
                              b2=mlp.b2, root_token=dev(mlp.root_token))


@pytest.mark.parametrize("name,d,h", [("qwen3_4b", 16, 32), ("qwen3_8b", 16, 32),
                                      ("qwen3_8b", 32, 64)])
def test_select_learned_scorer_matches_oracle(taps, name, d, h):
    """The learned-scorer hook with seeded random weights: q_cond per (row, parent rank,
    child rank) from the MLP and the sibling softmax; trees bit-exact."""
    from oracle.scorer import random_scorer
    say(f"[select-learned] {name} d={d} h={h}")
    inp = gen_round(name, with_attention=False)
    c = inp.cfg
    mlp = random_scorer(np.random.default_rng(31 + d + h), c.vocab, d, h, c.batch)
    x = inp.marginals_f64()
    trees = [oracle.select_request(x[b], c.K, c.budget, kind=c.kind, lambda1=c.lambda1,
                                   lambda2=c.lambda2, tau=c.tau, scorer=oracle.select.LEARNED,
                                   mlp=mlp, req=b) for b in range(c.batch)]
    w = _learned_weights(taps, mlp)
    gpu, _, _ = run_select(taps, inp, scorer=2, mlp=w)
    U.assert_tree_equal(gpu, trees, c)


@pytest.mark.parametrize("seed", range(10))
def test_select_learned_fuzz(taps, seed):
    from oracle.scorer import random_scorer
    rng = np.random.default_rng(1300 + seed)
    dtype = [BF16, FP32][seed % 2]
    V = int(rng.choice([17, 1001, 70001]))
    K = min(int(rng.integers(1, 13)), V)
    D = int(rng.integers(1, 33))
    while D * K * K > 7168:
        D -= 1
    N = int(rng.choice([1, 16, 64, 200]))
    mode = ["ties", "deep", "specials", "plain"][seed % 4]
    d, h = int(rng.integers(1, 9)), int(rng.integers(1, 17))
    cfg = _fuzz_cfg(rng, dtype, LOGITS, V, D, K, N)
    say(f"[fuzz-learned] seed={seed} dtype={dtype} V={V} K={K} D={D} N={N} mode={mode} "
        f"d={d} h={h}")
    m = _fuzz_marginals(rng, cfg, mode)
    mlp = random_scorer(rng, V, d, h, cfg.batch)
    from workloads import bf16_bits_to_f32
    x = bf16_bits_to_f32(m).astype(np.float64) if dtype == BF16 else m.astype(np.float64)
    trees = [oracle.select_request(x[b], K, N, kind=LOGITS, scorer=oracle.select.LEARNED,
                                   mlp=mlp, req=b) for b in range(cfg.batch)]
    sel = taps.Selector(cfg.batch, D, V, K, N, dtype=dtype, kind=LOGITS, scorer=2,
                        mlp=_learned_weights(taps, mlp))
    gpu = sel(U.to_dev(m, dtype == BF16))
    torch.cuda.synchronize()
    U.assert_tree_equal(gpu, trees, cfg)


@pytest.mark.parametrize("D,K,mode", [(32, 8, "plain"), (12, 16, "deep")])
def test_select_learned_large_tables(taps, D, K, mode):
    """The largest weights (d = 32, h = 64) on large q_cond tables, so that the hidden units
    are taken in several chunks, the last one shorter than 8 and 4 units; root tokens
    outside the vocabulary (above it and negative) have zero embeddings."""
    from oracle.scorer import random_scorer
    rng = np.random.default_rng(1400 + D + K)
    V, N, d, h = 70001, 128, 32, 64
    cfg = _fuzz_cfg(rng, BF16, LOGITS, V, D, K, N)
    say(f"[learned-large] D={D} K={K} mode={mode} d={d} h={h}")
    m = _fuzz_marginals(rng, cfg, mode)
    mlp = random_scorer(rng, V, d, h, cfg.batch)
    mlp.root_token[:] = [V + 5, -3]
    from workloads import bf16_bits_to_f32
    x = bf16_bits_to_f32(m).astype(np.float64)
    trees = [oracle.select_request(x[b], K, N, kind=LOGITS, scorer=oracle.select.LEARNED,
                                   mlp=mlp, req=b) for b in range(cfg.batch)]
    sel = taps.Selector(cfg.batch, D, V, K, N, dtype=BF16, kind=LOGITS, scorer=2,
                        mlp=_learned_weights(taps, mlp))
    gpu = sel(U.to_dev(m, True))
    torch.cuda.synchronize()
    U.assert_tree_equal(gpu, trees, cfg)


@pytest.mark.parametrize("B,D,V,K,scorer,kind,mode", [
    (1, 16, 65536, 8, 0, LOGITS, "plain"),    # 32 chunks of 8 entries: the largest two-row shape
    (1, 16, 65536, 8, 1, LOGITS, "ties"),     # the same, marginal scorer (integer normaliser)
    (1, 16, 65536, 8, 2, LOGITS, "deep"),     # the same, learned scorer
    (1, 15, 67584, 8, 0, LOGITS, "plain"),    # 33 chunks: one row per wave
    (2, 3, 4099, 8, 1, PROBS, "specials"),    # 3 chunks, odd D, the probability marginal
    (1, 31, 151936, 1, 0, LOGITS, "plain"),   # K = 1, odd D: the last wave's second half idles
    (2, 1, 1001, 7, 2, LOGITS, "ties"),       # one row of one chunk, learned scorer
])
def test_select_pair_rows(taps, B, D, V, K, scorer, kind, mode):
    """The row merge at the edges of its two-rows-per-wave form (K <= 8, at most 32 chunks
    and 256 list entries per row) and just past them, for each scorer.  The vocabulary scan
    cuts these rows into 32, 32, 32, 33, 3, 10 and 1 chunks."""
    from oracle.scorer import random_scorer
    rng = np.random.default_rng(1500 + D + V + K + scorer)
    dtype = FP32 if kind == PROBS else BF16
    N = 64
    cfg = _fuzz_cfg(rng, dtype, kind, V, D, K, N, B=B)
    say(f"[pair-rows] B={B} D={D} V={V} K={K} scorer={scorer} kind={kind} mode={mode}")
    m = _fuzz_marginals(rng, cfg, mode)
    mlp = random_scorer(rng, V, 16, 32, B) if scorer == 2 else None
    from workloads import bf16_bits_to_f32
    x = bf16_bits_to_f32(m).astype(np.float64) if dtype == BF16 else m.astype(np.float64)
    trees = [oracle.select_request(x[b], K, N, kind=kind, lambda2=0.125, tau=0.0,
                                   scorer=scorer, mlp=mlp, req=b) for b in range(B)]
    sel = taps.Selector(B, D, V, K, N, dtype=dtype, kind=kind, lambda2=0.125, tau=0.0,
                        scorer=scorer, mlp=_learned_weights(taps, mlp) if mlp else None)
    gpu = sel(U.to_dev(m, dtype == BF16))
    torch.cuda.synchronize()
    U.assert_tree_equal(gpu, trees, cfg)


@pytest.mark.parametrize("seed", range(24))
def test_select_fuzz(taps, seed):
    rng = np.random.default_rng(500 + seed)
    dtype = [BF16, FP32][seed % 2]
    kind = [LOGITS, LOGITS, PROBS][seed % 3]
    V = int(rng.choice([17, 100, 1001, 4099, 70001]))
    K = int(rng.integers(1, 17))
    K = min(K, V)
    D = int(rng.integers(1, 33))
    N = int(rng.choice([1, 2, 16, 63, 64, 65, 128, 200, 256]))
    mode = ["ties", "deep", "specials", "plain"][seed % 4]
    tau = float(rng.choice([0.0, 0.0, 1e-3, 1e-2]))
    lam2 = float(rng.choice([0.0, 0.125, 0.5]))
    cfg = _fuzz_cfg(rng, dtype, kind, V, D, K, N)
    say(f"[fuzz] seed={seed} dtype={dtype} kind={kind} V={V} K={K} D={D} N={N} mode={mode} "
        f"tau={tau} lam2={lam2}")
    m = _fuzz_marginals(rng, cfg, mode)

    class Inp:
        pass
    inp = Inp()
    inp.cfg, inp.marginals = cfg, m
    from workloads import bf16_bits_to_f32
    x = bf16_bits_to_f32(m).astype(np.float64) if dtype == BF16 else m.astype(np.float64)
    trees = [oracle.select_request(x[b], K, N, kind=kind, lambda1=1.0, lambda2=lam2, tau=tau)
             for b in range(cfg.batch)]
    sel = taps.Selector(cfg.batch, D, V, K, N, dtype=dtype, kind=kind, lambda2=lam2, tau=tau)
    gpu = sel(U.to_dev(m, dtype == BF16))
    torch.cuda.synchronize()
    U.assert_tree_equal(gpu, trees, cfg)


@pytest.mark.parametrize("mode", ["ties", "specials", "plain", "deep", "sparse_nan", "flat"])
@pytest.mark.parametrize("V,K", [(32768, 8), (151936, 16), (151936, 1)])
def test_select_full_aligned_chunks(taps, mode, V, K):
    """bf16 rows whose chunks are all full and 16-byte aligned (vocab a multiple of 8):
    the vocabulary scan's fast filter path, and its fall-backs (fewer than K non-NaN
    lanes in a wave, more tied candidates than the compaction buffer holds)."""
    rng = np.random.default_rng(7000 + V + K + len(mode))
    cfg = _fuzz_cfg(rng, BF16, LOGITS, V, 6, K, 64)
    say(f"[full-chunks] mode={mode} V={V} K={K}")
    if mode in ("ties", "specials", "plain", "deep"):
        m = _fuzz_marginals(rng, cfg, mode)
    else:
        x = np.full((cfg.batch, cfg.block, V), np.nan, dtype=np.float32)
        if mode == "sparse_nan":
            # a few finite values per row: most waves hold fewer than K of them
            for b in range(cfg.batch):
                for d in range(cfg.block):
                    pos = rng.choice(V, size=int(rng.integers(1, 3 * K + 2)), replace=False)
                    x[b, d, pos] = rng.standard_normal(pos.size)
        else:
            x[:] = 0.25                                   # every element ties
            x[:, :, ::977] = -0.0
        from workloads import f32_to_bf16_bits
        m = f32_to_bf16_bits(x)
    from workloads import bf16_bits_to_f32
    xf = bf16_bits_to_f32(m).astype(np.float64)
    trees = [oracle.select_request(xf[b], K, cfg.budget, kind=LOGITS) for b in range(cfg.batch)]
    sel = taps.Selector(cfg.batch, cfg.block, V, K, cfg.budget, dtype=BF16, kind=LOGITS)
    gpu = sel(U.to_dev(m, True))
    torch.cuda.synchronize()
    U.assert_tree_equal(gpu, trees, cfg)


def test_select_is_deterministic(taps):
    inp = gen_round("qwen3_8b", with_attention=False)
    a, sel, m = run_select(taps, inp)
    first = [t.clone() for t in (a.parent, a.token, a.q_reach, a.topk_idx, a.n_nodes)]
    b = sel(m)
    torch.cuda.synchronize()
    for x, y in zip(first, (b.parent, b.token, b.q_reach, b.topk_idx, b.n_nodes)):
        assert torch.equal(x, y)


# ------------------------------------------------------------------ attention
def _attn(taps, inp, trees, max_ctx=None):
    c = inp.cfg
    Q, K, V, off, ctx = U.attention_inputs(inp)
    parent, _, n = U.tree_device(trees)
    att = taps.TreeAttention(c.batch, c.budget, c.Hq, c.Hkv, c.head_dim,
                             int(max_ctx if max_ctx is not None else inp.ctx_len.max()),
                             dtype=c.dtype, scale=c.scale)
    att.ws.fill_(0xFF)            # NaN bits in every unwritten partial slot
    O = att(Q, K, V, off, ctx, parent, n)
    torch.cuda.synchronize()
    return O, (att, Q, K, V, off, ctx, parent, n)


@pytest.mark.parametrize("name,samples", [("tiny", None), ("qwen3_4b", None), ("qwen3_8b", None),
                                          ("serve16", 384), ("stress", 192)])
def test_attention_matches_oracle(taps, name, samples):
    say(f"[attn] {name}")
    inp = gen_round(name)
    c = inp.cfg
    trees = U.oracle_trees(inp)
    O, _ = _attn(taps, inp, trees)
    Qd, Kd, Vd = inp.qkv_f64()
    pick = None
    if samples is not None:
        rng = np.random.default_rng(7)
        pick = []
        for _ in range(samples):
            b = int(rng.integers(0, c.batch))
            pick.append((b, int(rng.integers(0, trees[b].n)), int(rng.integers(0, c.Hq))))
        # always include the root and the deepest node of every request
        for b, t in enumerate(trees):
            pick.append((b, 0, 0))
            pick.append((b, int(np.argmax(t.depth[:t.n])), c.Hq - 1))
    ref = oracle.tree_attention(Qd, Kd, Vd, inp.kv_offset, inp.ctx_len,
                                [t.parent for t in trees], [t.n for t in trees], c.scale,
                                samples=pick)
    got = U.gpu_o_as_f64(O)
    U.attention_error(got, ref, c.dtype, name)
    # rows of nodes beyond n are never written
    for b, t in enumerate(trees):
        assert t.n <= c.budget


@pytest.mark.parametrize("dtype,hd", [(BF16, 128), (BF16, 64), (FP32, 64), (FP32, 128)])
def test_attention_edge_cases(taps, dtype, hd):
    """ctx = 0, a single node, a chain deeper than 64, ragged contexts, >64-node masks, for
    both storage types and both head sizes."""
    rng = np.random.default_rng(3 + hd + dtype)
    B, N, Hq, Hkv = 4, 130, 8, 2
    ctx = np.array([0, 1, 77, 300], dtype=np.int32)
    say(f"[attn-edge] dtype={dtype} hd={hd}")
    off = kv_offsets(ctx, N)
    rows = int(off[-1] + ctx[-1] + N)
    from workloads import f32_to_bf16_bits, bf16_bits_to_f32
    bf = dtype == BF16
    Qf = rng.standard_normal((B, N, Hq, hd)).astype(np.float32)
    Kf = rng.standard_normal((rows, Hkv, hd)).astype(np.float32)
    Vf = rng.standard_normal((rows, Hkv, hd)).astype(np.float32)
    if bf:
        Q, K, V = (f32_to_bf16_bits(a) for a in (Qf, Kf, Vf))
        Qd, Kd, Vd = (bf16_bits_to_f32(a).astype(np.float64) for a in (Q, K, V))
    else:
        Q, K, V = Qf, Kf, Vf
        Qd, Kd, Vd = (a.astype(np.float64) for a in (Q, K, V))
    parents = [np.array([-1] + list(range(N - 1)), dtype=np.int32),         # chain of 130
               np.array([-1] + [0] * (N - 1), dtype=np.int32),              # star
               np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32),
               np.array([-1] + [int(rng.integers(max(0, i - 3), i)) for i in range(1, N)],
                        dtype=np.int32)]
    n = [N, 1, 97, 65]
    import paper_2606_00487_amd as taps_mod
    att = taps_mod.TreeAttention(B, N, Hq, Hkv, hd, int(ctx.max()), dtype=dtype, scale=hd ** -0.5)
    att.ws.fill_(0xFF)            # NaN bits in every unwritten partial slot
    O = att(U.to_dev(Q, bf), U.to_dev(K, bf), U.to_dev(V, bf), torch.from_numpy(off).cuda(),
            torch.from_numpy(ctx).cuda(), torch.from_numpy(np.stack(parents)).cuda(),
            torch.tensor(n, dtype=torch.int32).cuda())
    torch.cuda.synchronize()
    ref = oracle.tree_attention(Qd, Kd, Vd, off, ctx, parents, n, hd ** -0.5)
    got = U.gpu_o_as_f64(O)
    for b in range(B):
        U.attention_error(got[b, :n[b]], ref[b, :n[b]], dtype,
                          f"edge dtype={dtype} hd={hd} b={b} ctx={ctx[b]} n={n[b]}")


@pytest.mark.parametrize("dtype,hd", [(BF16, 64), (FP32, 128)])
def test_attention_multi_split_other_head_sizes(taps, dtype, hd):
    """Contexts long enough for several key splits (and a ragged last one), 64-node trees,
    grouped-query heads, for the storage type / head size pairs the Qwen3 shapes do not
    use."""
    rng = np.random.default_rng(40 + hd)
    B, N, Hq, Hkv = 2, 64, 16, 4
    ctx = np.array([3001, 1777], dtype=np.int32)
    say(f"[attn-split] dtype={dtype} hd={hd}")
    off = kv_offsets(ctx, N)
    rows = int(off[-1] + ctx[-1] + N)
    from workloads import f32_to_bf16_bits, bf16_bits_to_f32
    bf = dtype == BF16
    Qf = rng.standard_normal((B, N, Hq, hd)).astype(np.float32)
    Kf = rng.standard_normal((rows, Hkv, hd)).astype(np.float32)
    Vf = rng.standard_normal((rows, Hkv, hd)).astype(np.float32)
    if bf:
        Q, K, V = (f32_to_bf16_bits(a) for a in (Qf, Kf, Vf))
        Qd, Kd, Vd = (bf16_bits_to_f32(a).astype(np.float64) for a in (Q, K, V))
    else:
        Q, K, V = Qf, Kf, Vf
        Qd, Kd, Vd = (a.astype(np.float64) for a in (Q, K, V))
    parents = [np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)
               for _ in range(B)]
    n = [64, 41]
    import paper_2606_00487_amd as taps_mod
    att = taps_mod.TreeAttention(B, N, Hq, Hkv, hd, int(ctx.max()), dtype=dtype, scale=hd ** -0.5)
    att.ws.fill_(0xFF)            # NaN bits in every unwritten partial slot
    O = att(U.to_dev(Q, bf), U.to_dev(K, bf), U.to_dev(V, bf), torch.from_numpy(off).cuda(),
            torch.from_numpy(ctx).cuda(), torch.from_numpy(np.stack(parents)).cuda(),
            torch.tensor(n, dtype=torch.int32).cuda())
    torch.cuda.synchronize()
    ref = oracle.tree_attention(Qd, Kd, Vd, off, ctx, parents, n, hd ** -0.5)
    got = U.gpu_o_as_f64(O)
    for b in range(B):
        U.attention_error(got[b, :n[b]], ref[b, :n[b]], dtype, f"split dtype={dtype} hd={hd} b={b}")


@pytest.mark.parametrize("hd,ctx", [(128, 100), (128, 600), (128, 2000), (64, 700), (64, 1100)])
def test_attention_one_request_split_groups(taps, hd, ctx):
    """One request (the host's split plan): contexts whose plans take a few, six to eight,
    and more than eight key splits, so the split combine merges them in groups of 4, 8 and
    16; every (node, head) row against the oracle."""
    rng = np.random.default_rng(60 + hd + ctx)
    B, N, Hq, Hkv = 1, 64, 32, 8
    ctxs = np.array([ctx], dtype=np.int32)
    say(f"[attn-groups] hd={hd} ctx={ctx}")
    off = kv_offsets(ctxs, N)
    rows = int(off[-1] + ctxs[-1] + N)
    from workloads import f32_to_bf16_bits, bf16_bits_to_f32
    Q, K, V = (f32_to_bf16_bits(rng.standard_normal(sh).astype(np.float32))
               for sh in ((B, N, Hq, hd), (rows, Hkv, hd), (rows, Hkv, hd)))
    Qd, Kd, Vd = (bf16_bits_to_f32(a).astype(np.float64) for a in (Q, K, V))
    parents = [np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)]
    n = [N]
    import paper_2606_00487_amd as taps_mod
    att = taps_mod.TreeAttention(B, N, Hq, Hkv, hd, ctx, dtype=BF16, scale=hd ** -0.5)
    att.ws.fill_(0xFF)            # NaN bits in every unwritten partial slot
    O = att(U.to_dev(Q, True), U.to_dev(K, True), U.to_dev(V, True), torch.from_numpy(off).cuda(),
            torch.from_numpy(ctxs).cuda(), torch.from_numpy(np.stack(parents)).cuda(),
            torch.tensor(n, dtype=torch.int32).cuda())
    torch.cuda.synchronize()
    ref = oracle.tree_attention(Qd, Kd, Vd, off, ctxs, parents, n, hd ** -0.5)
    U.attention_error(U.gpu_o_as_f64(O)[0], ref[0], BF16, f"groups hd={hd} ctx={ctx}")


def test_attention_tree_rows_dominate_at_full_size(taps):
    """The Qwen3-8B round shape (context 8192, 64 nodes, 32/8 heads, head_dim 128, the
    bench's key splits) with a common direction added to every query and to the tree rows'
    keys, so that each node's ancestor rows carry almost all of its softmax mass: a wrong
    mask bit or a misplaced tree row in the last split moves O by O(1).  Every (node, head)
    row is compared."""
    say("[attn-tree-dominant] qwen3_8b shape")
    inp = gen_round("qwen3_8b")
    c = inp.cfg
    trees = U.oracle_trees(inp)
    from workloads import f32_to_bf16_bits, bf16_bits_to_f32
    rng = np.random.default_rng(77)
    w = rng.standard_normal((c.Hkv, c.head_dim))
    w /= np.linalg.norm(w, axis=1, keepdims=True)
    a = 16.0                                   # a^2 * scale ~ 23: e^23 >> 8192 context rows
    Qf = bf16_bits_to_f32(inp.Q).astype(np.float64)
    Kf = bf16_bits_to_f32(inp.K).astype(np.float64)
    G = c.Hq // c.Hkv
    Qf += a * np.repeat(w, G, axis=0)[None, None]
    ctx = int(inp.ctx_len[0])
    Kf[ctx:ctx + c.budget] += a * w[None]
    Q, K = f32_to_bf16_bits(Qf.astype(np.float32)), f32_to_bf16_bits(Kf.astype(np.float32))
    Qd, Kd = bf16_bits_to_f32(Q).astype(np.float64), bf16_bits_to_f32(K).astype(np.float64)
    Vd = bf16_bits_to_f32(inp.V).astype(np.float64)
    parent, _, n = U.tree_device(trees)
    att = taps.TreeAttention(c.batch, c.budget, c.Hq, c.Hkv, c.head_dim, ctx, dtype=c.dtype,
                             scale=c.scale)
    O = att(U.to_dev(Q, True), U.to_dev(K, True), U.to_dev(inp.V, True),
            torch.from_numpy(inp.kv_offset).cuda(), torch.from_numpy(inp.ctx_len).cuda(),
            parent, n)
    torch.cuda.synchronize()
    ref = oracle.tree_attention(Qd, Kd, Vd, inp.kv_offset, inp.ctx_len,
                                [t.parent for t in trees], [t.n for t in trees], c.scale)
    # the construction works: the tree rows hold most of every row's softmax mass
    t0 = trees[0]
    anc = oracle.ancestor_sets(t0.parent, t0.n)
    for i in (0, t0.n - 1):
        rows = np.r_[np.arange(ctx), ctx + np.array(sorted(anc[i]))]
        for h in range(c.Hq):
            s = (Qd[0, i, h] @ Kd[rows, h // G].T) * c.scale
            p = np.exp(s - s.max())
            assert p[ctx:].sum() / p.sum() > 0.99
    U.attention_error(U.gpu_o_as_f64(O), ref, c.dtype, "tree-dominant qwen3_8b")


def test_attention_is_deterministic(taps):
    inp = gen_round("qwen3_4b")
    trees = U.oracle_trees(inp)
    O1, (att, Q, K, V, off, ctx, parent, n) = _attn(taps, inp, trees)
    O1 = O1.clone()
    O2 = att(Q, K, V, off, ctx, parent, n)
    torch.cuda.synchronize()
    assert torch.equal(O1.view(torch.int16), O2.view(torch.int16))


# ------------------------------------------------------------------ walk
@pytest.mark.parametrize("name,branch", [("tiny", False), ("qwen3_8b", False), ("qwen3_8b", True),
                                         ("serve16", False), ("serve16", True), ("stress", True)])
def test_walk_matches_oracle(taps, name, branch):
    say(f"[walk] {name} branch={branch}")
    inp = gen_round(name, with_attention=False)
    c = inp.cfg
    trees = U.oracle_trees(inp)
    tgt = U.targets_for(inp, trees, branch=branch)
    parent, token, n = U.tree_device(trees)
    tb = taps.TreeBuffers.empty(c.batch, c.block, c.K, c.budget)
    tb.parent.copy_(parent)
    tb.token.copy_(token)
    tb.n_nodes.copy_(n)
    walk = taps.AcceptWalk(c.batch, c.budget, c.block)
    path, plen, bonus = walk(tb, torch.from_numpy(tgt).cuda())
    torch.cuda.synchronize()
    path, plen, bonus = path.cpu().numpy(), plen.cpu().numpy(), bonus.cpu().numpy()
    for b, t in enumerate(trees):
        p, bo = oracle.accept_walk(t.parent, t.token, t.n, tgt[b])
        from oracle.walk import walk_arrays
        arr, ln, bn = walk_arrays(p, bo, c.block)
        assert plen[b] == ln and bonus[b] == bn
        np.testing.assert_array_equal(path[b], arr)


# ------------------------------------------------------------------ one whole round
def test_full_round_tiny_and_8b(taps):
    for name in ["tiny", "qwen3_8b"]:
        say(f"[round] {name}")
        inp = gen_round(name)
        c = inp.cfg
        trees = U.oracle_trees(inp)
        gpu, _, _ = run_select(taps, inp)
        U.assert_tree_equal(gpu, trees, c)
        Q, K, V, off, ctx = U.attention_inputs(inp)
        att = taps.TreeAttention(c.batch, c.budget, c.Hq, c.Hkv, c.head_dim, int(inp.ctx_len.max()),
                                 dtype=c.dtype, scale=c.scale)
        O = att(Q, K, V, off, ctx, gpu.parent, gpu.n_nodes)
        tgt = torch.from_numpy(U.targets_for(inp, trees)).cuda()
        walk = taps.AcceptWalk(c.batch, c.budget, c.block)
        path, plen, bonus = walk(gpu, tgt)
        torch.cuda.synchronize()
        Qd, Kd, Vd = inp.qkv_f64()
        ref = oracle.tree_attention(Qd, Kd, Vd, inp.kv_offset, inp.ctx_len,
                                    [t.parent for t in trees], [t.n for t in trees], c.scale)
        U.attention_error(U.gpu_o_as_f64(O), ref, c.dtype, f"round {name}")
        p, bo = oracle.accept_walk(trees[0].parent, trees[0].token, trees[0].n,
                                   tgt.cpu().numpy()[0])
        assert int(plen[0]) == len(p) and int(bonus[0]) == bo
        assert path.cpu().numpy()[0, :len(p)].tolist() == p


# ------------------------------------------------------------------ selection fallback
@pytest.mark.parametrize("name", ["marginal_probs_all_one", "sibling_probs_plateau",
                                  "sibling_logits_plateau", "learned_child_chains"])
def test_select_sequential_fallback_matches_oracle(taps, name):
    """Inputs whose level-by-level expansion outgrows the kernel's LDS (shown on the CPU by
    tests/test_select_fallback_inputs.py), so the sequential best-first loop selects.  The
    learned case needs children visited in utility order, not rank order."""
    case = U.fallback_cases()[name]
    say(f"[select-fallback] {name}")
    t, _, _ = U.fallback_oracle(case)
    m = case["marginals"]
    D, V = m.shape[1], m.shape[2]
    mlp = _learned_weights(taps, case["mlp"]) if case["mlp"] is not None else None
    sel = taps.Selector(1, D, V, case["K"], case["N"], dtype=case["dtype"], kind=case["kind"],
                        lambda2=case["lam2"], tau=0.0, scorer=case["scorer"], mlp=mlp)
    gpu = sel(U.to_dev(m, case["dtype"] == BF16))
    torch.cuda.synchronize()
    cfg = _fuzz_cfg(None, case["dtype"], case["kind"], V, D, case["K"], case["N"], B=1)
    U.assert_tree_equal(gpu, [t], cfg)


@pytest.mark.parametrize("seed", range(6))
def test_attention_fuzz_batches(taps, seed):
    """Seeded random batches for the ragged work list and the grouped split combine: 2-6
    requests, contexts from empty to 6000 rows (max_ctx above every one of them), 1-100
    nodes with random parents, 1-4 KV heads of 1-4 query heads each; sampled (node, head)
    rows of every request against the oracle."""
    from workloads import f32_to_bf16_bits, bf16_bits_to_f32
    rng = np.random.default_rng(500 + seed)
    B = int(rng.integers(2, 7))
    N = int(rng.integers(1, 101))
    Hkv = int(rng.choice([1, 2, 4]))
    Hq = Hkv * int(rng.choice([1, 2, 4]))
    hd = 128
    ctx = rng.integers(0, 6001, B).astype(np.int32)
    ctx[int(rng.integers(0, B))] = int(rng.integers(0, 3))      # a (nearly) empty context
    n = [int(x) for x in rng.integers(0, N + 1, B)]
    n[int(rng.integers(0, B))] = N
    max_ctx = int(ctx.max()) + int(rng.integers(0, 500))
    say(f"[attn-fuzz] seed={seed} B={B} N={N} Hq={Hq} Hkv={Hkv} ctx={ctx.tolist()} n={n} max_ctx={max_ctx}")
    off = kv_offsets(ctx, N)
    rows = int(off[-1] + ctx[-1] + N)
    Q = f32_to_bf16_bits(rng.standard_normal((B, N, Hq, hd)).astype(np.float32))
    K = f32_to_bf16_bits(rng.standard_normal((rows, Hkv, hd)).astype(np.float32))
    V = f32_to_bf16_bits(rng.standard_normal((rows, Hkv, hd)).astype(np.float32))
    parents = [np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)
               for _ in range(B)]
    att = taps.TreeAttention(B, N, Hq, Hkv, hd, max_ctx, dtype=BF16, scale=hd ** -0.5)
    att.ws.fill_(0xFF)
    O = att(U.to_dev(Q, True), U.to_dev(K, True), U.to_dev(V, True), torch.from_numpy(off).cuda(),
            torch.from_numpy(ctx).cuda(), torch.from_numpy(np.stack(parents)).cuda(),
            torch.tensor(n, dtype=torch.int32).cuda())
    torch.cuda.synchronize()
    picks = [(b, int(i), int(h)) for b in range(B) if n[b]
             for i in sorted({0, n[b] - 1, *rng.integers(0, n[b], 6).tolist()})
             for h in sorted({0, Hq - 1, int(rng.integers(0, Hq))})]
    ref = oracle.tree_attention(*(bf16_bits_to_f32(a).astype(np.float64) for a in (Q, K, V)),
                                off, ctx, parents, n, hd ** -0.5, samples=picks)
    got = U.gpu_o_as_f64(O)
    for b in range(B):
        if n[b]:
            U.attention_error(got[b, :n[b]], ref[b, :n[b]], BF16, f"fuzz b={b} ctx={ctx[b]}")


def test_attention_ragged_batch(taps):
    """Several requests of very different lengths (the ragged work list: split lengths from
    the batch's actual keys, pairs numbered by prefix sums), including an empty request and
    one-row ones, with NaN bits in every unwritten workspace slot."""
    from workloads import f32_to_bf16_bits, bf16_bits_to_f32
    rng = np.random.default_rng(321)
    B, N, Hq, Hkv, hd = 6, 64, 16, 4, 128
    ctx = np.array([0, 16000, 1, 5000, 77, 0], dtype=np.int32)
    n = [0, 64, 1, 33, 64, 5]
    say("[attn-ragged] contexts", ctx.tolist(), "nodes", n)
    off = kv_offsets(ctx, N)
    rows = int(off[-1] + ctx[-1] + N)
    Q = f32_to_bf16_bits(rng.standard_normal((B, N, Hq, hd)).astype(np.float32))
    K = f32_to_bf16_bits(rng.standard_normal((rows, Hkv, hd)).astype(np.float32))
    V = f32_to_bf16_bits(rng.standard_normal((rows, Hkv, hd)).astype(np.float32))
    parents = [np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)
               for _ in range(B)]
    att = taps.TreeAttention(B, N, Hq, Hkv, hd, 16384, dtype=BF16, scale=hd ** -0.5)
    att.ws.fill_(0xFF)
    O = att(U.to_dev(Q, True), U.to_dev(K, True), U.to_dev(V, True), torch.from_numpy(off).cuda(),
            torch.from_numpy(ctx).cuda(), torch.from_numpy(np.stack(parents)).cuda(),
            torch.tensor(n, dtype=torch.int32).cuda())
    torch.cuda.synchronize()
    picks = [(b, i, h) for b in range(B) for i in range(n[b]) for h in (0, 5, Hq - 1)]
    ref = oracle.tree_attention(*(bf16_bits_to_f32(a).astype(np.float64) for a in (Q, K, V)),
                                off, ctx, parents, n, hd ** -0.5, samples=picks)
    got = U.gpu_o_as_f64(O)
    for b in range(B):
        if n[b]:
            U.attention_error(got[b, :n[b]], ref[b, :n[b]], BF16, f"ragged b={b} ctx={ctx[b]}")

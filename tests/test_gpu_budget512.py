"""GPU parity at node budgets above 256, up to the library's 512: the DDTree budget of the
paper's baselines (Sec. 5.1) and the top of its 64 -> 512 budget sweep (Sec. 3.1).
Selection (all three scorers; the stress marginals, whose third trie level needs the
pruning bin raised within the level), ancestor masks over more than 256 nodes in all three
attention kernels, the walk with eight node slots per lane, and the KV commit."""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle.walk import walk_arrays
from tests import _util as U
from workloads import BF16, CONFIGS, FP32, LOGITS, Config, gen_round, kv_offsets

pytestmark = pytest.mark.gpu


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


def cfg_at(name, budget):
    return dataclasses.replace(CONFIGS[name], budget=budget)


def select_gpu(taps, inp, **kw):
    c = inp.cfg
    args = dict(kind=c.kind, lambda1=c.lambda1, lambda2=c.lambda2, tau=c.tau, beta=c.beta)
    args.update(kw)
    sel = taps.Selector(c.batch, c.block, c.vocab, c.K, c.budget, dtype=c.dtype, **args)
    out = sel(U.to_dev(inp.marginals, c.dtype == BF16))
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("name,N", [("qwen3_8b", 384), ("qwen3_8b", 512), ("stress", 512),
                                    ("serve16", 512), ("qwen3_4b", 300)])
def test_select_large_budget(taps, name, N):
    say(f"[select-512] {name} N={N}")
    inp = gen_round(cfg_at(name, N), with_attention=False)
    U.assert_tree_equal(select_gpu(taps, inp), U.oracle_trees(inp), inp.cfg)


def test_select_large_budget_other_scorers(taps):
    from oracle.scorer import random_scorer
    inp = gen_round(cfg_at("qwen3_8b", 512), with_attention=False)
    c = inp.cfg
    say("[select-512] marginal scorer")
    U.assert_tree_equal(select_gpu(taps, inp, scorer=1),
                        U.oracle_trees(inp, scorer=oracle.select.MARGINAL), c)
    say("[select-512] learned scorer")
    mlp = random_scorer(np.random.default_rng(512), c.vocab, 16, 32, c.batch)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    w = taps.ScorerWeights(emb=dev(mlp.emb), W1=dev(mlp.W1), b1=dev(mlp.b1), w2=dev(mlp.w2),
                           b2=mlp.b2, root_token=dev(mlp.root_token))
    x = inp.marginals_f64()
    trees = [oracle.select_request(x[b], c.K, c.budget, kind=c.kind, lambda1=c.lambda1,
                                   lambda2=c.lambda2, tau=c.tau, scorer=oracle.select.LEARNED,
                                   mlp=mlp, req=b) for b in range(c.batch)]
    U.assert_tree_equal(select_gpu(taps, inp, scorer=2, mlp=w), trees, c)


@pytest.mark.parametrize("seed", range(8))
def test_select_large_budget_fuzz(taps, seed):
    from workloads import bf16_bits_to_f32, f32_to_bf16_bits
    rng = np.random.default_rng(5120 + seed)
    dtype = [BF16, FP32][seed % 2]
    V = int(rng.choice([100, 4099, 70001]))
    K = int(rng.integers(2, 17))
    D = int(rng.integers(4, 33))
    N = int(rng.integers(257, 513))
    lam2 = float(rng.choice([0.0, 0.125]))
    tau = float(rng.choice([0.0, 1e-4]))
    say(f"[fuzz-512] seed={seed} dtype={dtype} V={V} K={K} D={D} N={N} lam2={lam2} tau={tau}")
    x = (rng.standard_normal((2, D, V)) * float(rng.choice([0.5, 2.0]))).astype(np.float32)
    m = f32_to_bf16_bits(x) if dtype == BF16 else x
    xf = (bf16_bits_to_f32(m) if dtype == BF16 else m).astype(np.float64)
    trees = [oracle.select_request(xf[b], K, N, kind=LOGITS, lambda1=1.0, lambda2=lam2, tau=tau)
             for b in range(2)]
    sel = taps.Selector(2, D, V, K, N, dtype=dtype, kind=LOGITS, lambda2=lam2, tau=tau)
    gpu = sel(U.to_dev(m, dtype == BF16))
    torch.cuda.synchronize()
    cfg = Config("fuzz", 9, 2, D, V, K, N, 4, 2, 64, 16, LOGITS, dtype, 1.0, lam2, tau, 0.7)
    U.assert_tree_equal(gpu, trees, cfg)


@pytest.mark.parametrize("dtype,hd", [(BF16, 128), (BF16, 64), (FP32, 128)])
def test_attention_masks_beyond_256_nodes(taps, dtype, hd):
    """512-node trees (deep random trees, a 512-node chain) whose tree rows carry almost all
    of the softmax mass (a common direction added to every query and to the tree keys), so
    any wrong bit of the 8-word ancestor masks moves O by O(1)."""
    from workloads import bf16_bits_to_f32, f32_to_bf16_bits
    rng = np.random.default_rng(90 + hd + dtype)
    B, N, Hq, Hkv = 3, 512, 8, 2
    G = Hq // Hkv
    ctx = np.array([700, 37, 1500], dtype=np.int32)
    say(f"[attn-512] dtype={dtype} hd={hd}")
    off = kv_offsets(ctx, N)
    rows = int(off[-1] + ctx[-1] + N)
    Qf = rng.standard_normal((B, N, Hq, hd))
    Kf = rng.standard_normal((rows, Hkv, hd))
    Vf = rng.standard_normal((rows, Hkv, hd))
    w = rng.standard_normal((Hkv, hd))
    w /= np.linalg.norm(w, axis=1, keepdims=True)
    a = 8.0 * hd ** 0.25                       # (a / 2)^2 / sqrt(hd) = 16: far above any context row
    Qf += a * np.repeat(w, G, axis=0)[None, None] / 2
    for b in range(B):
        Kf[off[b] + ctx[b]:off[b] + ctx[b] + N] += a * w[None] / 2
    bf = dtype == BF16
    if bf:
        Q, K, V = (f32_to_bf16_bits(t.astype(np.float32)) for t in (Qf, Kf, Vf))
        Qd, Kd, Vd = (bf16_bits_to_f32(t).astype(np.float64) for t in (Q, K, V))
    else:
        Q, K, V = (t.astype(np.float32) for t in (Qf, Kf, Vf))
        Qd, Kd, Vd = (t.astype(np.float64) for t in (Q, K, V))
    parents = [np.array([-1] + [int(rng.integers(max(0, i - 3), i)) for i in range(1, N)],
                        dtype=np.int32),
               np.array([-1] + list(range(N - 1)), dtype=np.int32),
               np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], dtype=np.int32)]
    n = [512, 512, 301]
    att = taps.TreeAttention(B, N, Hq, Hkv, hd, int(ctx.max()), dtype=dtype, scale=hd ** -0.5)
    att.ws.fill_(0xFF)
    O = att(U.to_dev(Q, bf), U.to_dev(K, bf), U.to_dev(V, bf), torch.from_numpy(off).cuda(),
            torch.from_numpy(ctx).cuda(), torch.from_numpy(np.stack(parents)).cuda(),
            torch.tensor(n, dtype=torch.int32).cuda())
    torch.cuda.synchronize()
    picks = [(b, i, h) for b in range(B) for i in range(n[b]) for h in (0, Hq - 1)]
    ref = oracle.tree_attention(Qd, Kd, Vd, off, ctx, parents, n, hd ** -0.5, samples=picks)
    got = U.gpu_o_as_f64(O)
    # the construction works: every compared row's ancestors hold its softmax mass
    anc = oracle.ancestor_sets(parents[1], n[1])
    s = (Qd[1, 500, 0] @ Kd[off[1]:off[1] + ctx[1] + N, 0].T) * hd ** -0.5
    vis = np.r_[np.arange(ctx[1]), ctx[1] + np.array(anc[500])]
    p = np.exp(s[vis] - s[vis].max())
    assert p[ctx[1]:].sum() / p.sum() > 0.99
    for b in range(B):
        U.attention_error(got[b, :n[b]], ref[b, :n[b]], dtype, f"512 dtype={dtype} hd={hd} b={b}")


@pytest.mark.parametrize("name,N", [("qwen3_8b", 512), ("stress", 512)])
def test_walk_and_commit_large_budget(taps, name, N):
    say(f"[walk-commit-512] {name} N={N}")
    inp = gen_round(cfg_at(name, N))
    c = inp.cfg
    trees = U.oracle_trees(inp)
    tgt = U.targets_for(inp, trees, branch=True)
    parent, token, n = U.tree_device(trees)
    tb = taps.TreeBuffers.empty(c.batch, c.block, c.K, c.budget)
    tb.parent.copy_(parent)
    tb.token.copy_(token)
    tb.n_nodes.copy_(n)
    walk = taps.AcceptWalk(c.batch, c.budget, c.block)
    path, plen, bonus = walk(tb, torch.from_numpy(tgt).cuda())
    torch.cuda.synchronize()
    want_path = np.full((c.batch, c.block + 1), -1, np.int32)
    want_len = np.zeros(c.batch, np.int32)
    want_bonus = np.zeros(c.batch, np.int32)
    for b, t in enumerate(trees):
        p, bo = oracle.accept_walk(t.parent, t.token, t.n, tgt[b])
        want_path[b], want_len[b], want_bonus[b] = walk_arrays(p, bo, c.block)
    np.testing.assert_array_equal(path.cpu().numpy(), want_path)
    np.testing.assert_array_equal(plen.cpu().numpy(), want_len)
    np.testing.assert_array_equal(bonus.cpu().numpy(), want_bonus)
    say(f"[walk-commit-512] accepted lengths {want_len.tolist()}")
    bf = c.dtype == BF16
    Kd, Vd = U.to_dev(inp.K, bf), U.to_dev(inp.V, bf)
    com = taps.KVCommit(c.batch, c.budget, c.block, c.Hkv, c.head_dim, int(inp.ctx_len.max()),
                        dtype=c.dtype)
    nc, cm, nn = com(Kd, Vd, torch.from_numpy(inp.kv_offset).cuda(),
                     torch.from_numpy(inp.ctx_len).cuda(), tb, path, plen, bonus)
    torch.cuda.synchronize()
    want = oracle.kv_commit(inp.K, inp.V, inp.kv_offset, inp.ctx_len,
                            np.stack([t.token for t in trees]), want_path, want_len, want_bonus,
                            c.budget, c.block, int(inp.ctx_len.max()))
    host = (lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)) if bf else \
        (lambda t: t.cpu().numpy())
    assert np.array_equal(host(Kd), want[0]) and np.array_equal(host(Vd), want[1])
    assert np.array_equal(nc.cpu().numpy(), want[2]) and np.array_equal(cm.cpu().numpy(), want[3])
    assert np.array_equal(nn.cpu().numpy(), want[4])


def test_full_round_at_budget_512(taps):
    """One Qwen3-8B-shaped round at the DDTree budget: selection, attention of every node
    (two heads each), walk."""
    say("[round-512] qwen3_8b N=512")
    inp = gen_round(cfg_at("qwen3_8b", 512))
    c = inp.cfg
    trees = U.oracle_trees(inp)
    gpu = select_gpu(taps, inp)
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
    picks = [(0, i, h) for i in range(trees[0].n) for h in (i % c.Hq, (7 * i + 3) % c.Hq)]
    ref = oracle.tree_attention(Qd, Kd, Vd, inp.kv_offset, inp.ctx_len,
                                [t.parent for t in trees], [t.n for t in trees], c.scale,
                                samples=picks)
    U.attention_error(U.gpu_o_as_f64(O), ref, c.dtype, "round-512 qwen3_8b")
    p, bo = oracle.accept_walk(trees[0].parent, trees[0].token, trees[0].n, tgt.cpu().numpy()[0])
    assert int(plen[0]) == len(p) and int(bonus[0]) == bo
    assert path.cpu().numpy()[0, :len(p)].tolist() == p

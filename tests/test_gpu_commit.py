"""GPU parity of kv_commit through the C ABI: the K/V caches, the new context lengths,
the emitted tokens and their counts must equal the oracle's bit for bit (pure data
movement).  Paths come from the oracle's walk on the oracle's trees, and from hand-made
edge cases (root only, the longest chain, malformed paths)."""
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle.walk import walk_arrays
from tests import _util as U
from workloads import BF16, FP32, gen_round

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


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host_bits(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def run_commit(taps, K, V, off, ctx, token, path, plen, bonus, budget, block, Hkv, hd, max_ctx,
               dtype):
    """K, V as stored (bf16 bits or fp32); returns the GPU's (K', V', new_ctx, committed, n)."""
    bf = dtype == BF16
    Kd, Vd = U.to_dev(K, bf), U.to_dev(V, bf)
    batch = len(ctx)
    tb = taps.TreeBuffers.empty(batch, block, 1, budget)
    tb.token.copy_(dev(token.astype(np.int32)))
    com = taps.KVCommit(batch, budget, block, Hkv, hd, max_ctx, dtype=dtype)
    nc, cm, n = com(Kd, Vd, dev(off.astype(np.int64)), dev(ctx.astype(np.int32)), tb,
                    dev(path.astype(np.int32)), dev(plen.astype(np.int32)),
                    dev(bonus.astype(np.int32)))
    torch.cuda.synchronize()
    return host_bits(Kd), host_bits(Vd), nc.cpu().numpy(), cm.cpu().numpy(), n.cpu().numpy()


def assert_commit(got, want):
    for name, g, w in zip(("K", "V", "new_ctx", "committed", "n"), got, want):
        assert g.shape == w.shape and np.array_equal(g, w), name


@pytest.mark.parametrize("name,branch", [("tiny", False), ("qwen3_4b", True), ("qwen3_8b", False),
                                         ("qwen3_8b", True), ("serve16", True), ("stress", True)])
def test_commit_matches_oracle_after_walk(taps, name, branch):
    say(f"[commit] {name} branch={branch}")
    inp = gen_round(name)
    c = inp.cfg
    trees = U.oracle_trees(inp)
    tgt = U.targets_for(inp, trees, branch=branch)
    path = np.full((c.batch, c.block + 1), -1, np.int32)
    plen = np.zeros(c.batch, np.int32)
    bonus = np.zeros(c.batch, np.int32)
    for b, t in enumerate(trees):
        p, bo = oracle.accept_walk(t.parent, t.token, t.n, tgt[b])
        path[b], plen[b], bonus[b] = walk_arrays(p, bo, c.block)
    token = np.stack([t.token for t in trees])
    max_ctx = int(inp.ctx_len.max())
    got = run_commit(taps, inp.K, inp.V, inp.kv_offset, inp.ctx_len, token, path, plen, bonus,
                     c.budget, c.block, c.Hkv, c.head_dim, max_ctx, c.dtype)
    want = oracle.kv_commit(inp.K, inp.V, inp.kv_offset, inp.ctx_len, token, path, plen, bonus,
                            c.budget, c.block, max_ctx)
    say(f"[commit] {name}: accepted lengths {plen.tolist()[:16]}")
    assert_commit(got, want)


@pytest.mark.parametrize("dtype,hd", [(BF16, 128), (FP32, 64)])
def test_commit_edge_paths_and_repeat(taps, dtype, hd):
    """Root only, the longest chain (block + 1 nodes), malformed paths cut at their first
    bad entry, clamped path lengths and contexts; then a second commit on the updated
    cache, which must equal the oracle applied twice."""
    rng = np.random.default_rng(5)
    budget, block, Hkv = 40, 12, 2
    ctx = np.array([0, 7, 33, 100, 5, 64, 9], dtype=np.int32)
    max_ctx = 64                       # request 3's 100 is clamped to 64
    off = np.concatenate([[0], np.cumsum(ctx.astype(np.int64) + budget)[:-1]])
    rows = int(off[-1] + ctx[-1] + budget)
    x = rng.standard_normal((2, rows, Hkv, hd)).astype(np.float32)
    if dtype == BF16:
        from workloads import f32_to_bf16_bits
        K, V = f32_to_bf16_bits(x[0]), f32_to_bf16_bits(x[1])
    else:
        K, V = x[0], x[1]
    B = len(ctx)
    token = rng.integers(0, 1000, size=(B, budget)).astype(np.int32)
    path = np.full((B, block + 1), -1, np.int32)
    plen = np.zeros(B, np.int32)
    path[0, 0] = 0; plen[0] = 1                                       # root only
    path[1] = np.arange(block + 1); plen[1] = block + 1               # chain, identity moves
    p2 = [0] + sorted(rng.choice(np.arange(1, budget), size=block, replace=False).tolist())
    path[2] = p2; plen[2] = block + 1                                 # longest scattered path
    path[3, :5] = [0, 3, 9, 9, 20]; plen[3] = 5                       # repeat: cut after 9
    path[4, :4] = [0, 2, 45, 46]; plen[4] = 4                         # beyond the budget: cut
    path[5, :3] = [0, 1, 39]; plen[5] = 99                            # length clamped to 13
    path[6, :3] = [0, 4, 8]; plen[6] = 0                              # length clamped to 1
    bonus = rng.integers(0, 1000, size=B).astype(np.int32)
    got = run_commit(taps, K, V, off, ctx, token, path, plen, bonus, budget, block, Hkv, hd,
                     max_ctx, dtype)
    want = oracle.kv_commit(K, V, off, ctx, token, path, plen, bonus, budget, block, max_ctx)
    assert_commit(got, want)
    assert list(want[4]) == [1, 13, 13, 3, 2, 3, 1]
    # commit again on the updated cache with fresh paths; compare with the oracle applied
    # to the oracle's own first result
    path2 = np.full((B, block + 1), -1, np.int32)
    for b in range(B):
        m = int(rng.integers(1, block + 2))
        path2[b, :m] = [0] + sorted(rng.choice(np.arange(1, budget), size=m - 1,
                                               replace=False).tolist())
    plen2 = (path2 >= 0).sum(axis=1).astype(np.int32)
    got2 = run_commit(taps, got[0], got[1], off, ctx, token, path2, plen2, bonus, budget, block,
                      Hkv, hd, max_ctx, dtype)
    want2 = oracle.kv_commit(want[0], want[1], off, ctx, token, path2, plen2, bonus, budget,
                             block, max_ctx)
    assert_commit(got2, want2)

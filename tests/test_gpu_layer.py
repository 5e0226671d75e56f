"""GPU parity of verify_layer (the verification layer slice) through the C ABI against
oracle.layer: the output projection Y on the defined rows, and the cache rows the layer
writes (bf16 keys and values), within the bf16 tolerance; every other cache row is left
bit for bit."""
import sys

import numpy as np
import pytest
import torch

from oracle.layer import bf16_round, verify_layer

pytestmark = pytest.mark.gpu

TOL = 2e-2      # max-abs, bf16 storage with fp32 accumulation, outputs of unit scale


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


def _bf16(rng, *shape, scale=1.0):
    return bf16_round(rng.standard_normal(shape) * scale)


def _tree(rng, N, n):
    """A random tree in breadth-first order: parent[i] < i, depth from the parents."""
    parent = np.full(N, -1, np.int32)
    depth = np.full(N, -1, np.int32)
    depth[0] = 0
    for i in range(1, n):
        parent[i] = int(rng.integers(max(0, i - 6), i))
        depth[i] = depth[parent[i]] + 1
    order = np.argsort(depth[:n], kind="stable")       # breadth first: parents first
    inv = np.empty(n, np.int64)
    inv[order] = np.arange(n)
    p2, d2 = parent.copy(), depth.copy()
    for new, old in enumerate(order):
        p2[new] = -1 if parent[old] < 0 else inv[parent[old]]
        d2[new] = depth[old]
    return p2, d2


def _to_dev(a, dtype):
    if dtype == torch.bfloat16:
        return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _run(taps, rng, B, N, H, Hq, Hkv, ctx, n, sample_nodes=None):
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
    off = np.zeros(B, np.int64)
    for b in range(1, B):
        off[b] = off[b - 1] + ctx[b - 1] + N + 5
    rows = int(off[-1] + ctx[-1] + N + 2)
    Kc, Vc = _bf16(rng, rows, Hkv, hd), _bf16(rng, rows, Hkv, hd)
    trees = [_tree(rng, N, int(n[b])) for b in range(B)]
    parent = np.stack([t[0] for t in trees])
    depth = np.stack([t[1] for t in trees])
    max_ctx = int(ctx.max())
    scale = hd ** -0.5
    samples = None
    if sample_nodes is not None:
        samples = [(b, i, h) for b in range(B) for i in sample_nodes(b) for h in range(Hq)]
    say(f"[layer] B={B} N={N} H={H} Hq={Hq} Hkv={Hkv} ctx={ctx.tolist()} n={n.tolist()}")
    Y, Ko, Vo, _, _ = verify_layer(X, Wq, Wk, Wv, Wo, qn, kn, Kc, Vc, off, ctx, depth, parent,
                                   n, Hq, Hkv, hd, 1e6, 1e-6, scale, samples=samples)
    w = taps.LayerWeights(_to_dev(Wq, torch.bfloat16), _to_dev(Wk, torch.bfloat16),
                          _to_dev(Wv, torch.bfloat16), _to_dev(Wo, torch.bfloat16),
                          _to_dev(qn, torch.bfloat16), _to_dev(kn, torch.bfloat16))
    tree = taps.TreeBuffers.empty(B, 1, 1, N)
    tree.parent.copy_(torch.from_numpy(parent))
    tree.depth.copy_(torch.from_numpy(depth))
    tree.n_nodes.copy_(torch.from_numpy(n))
    Kd, Vd = _to_dev(Kc, torch.bfloat16), _to_dev(Vc, torch.bfloat16)
    lay = taps.VerifyLayer(B, N, Hq, Hkv, hd, H, max_ctx)
    Yd = lay(_to_dev(X, torch.bfloat16), w, Kd, Vd, _to_dev(off, None), _to_dev(ctx, None), tree)
    torch.cuda.synchronize()
    Yg = Yd.float().cpu().numpy().astype(np.float64)
    Kg = Kd.float().cpu().numpy().astype(np.float64)
    Vg = Vd.float().cpu().numpy().astype(np.float64)
    written = np.zeros(rows, bool)
    for b in range(B):
        r0 = int(off[b] + ctx[b])
        written[r0:r0 + int(n[b])] = True
    assert np.array_equal(Kg[~written], Kc[~written]) and np.array_equal(Vg[~written], Vc[~written])
    ek = np.abs(Kg[written] - Ko[written]).max() if written.any() else 0.0
    ev = np.abs(Vg[written] - Vo[written]).max() if written.any() else 0.0
    err = 0.0
    for b in range(B):
        nodes = range(int(n[b])) if sample_nodes is None else sample_nodes(b)
        for i in nodes:
            err = max(err, float(np.abs(Yg[b, i] - Y[b, i]).max()))
    ymax = max(float(np.nanmax(np.abs(Y))), 1.0)
    say(f"[layer] max-abs: Y {err:.2e} (|Y| <= {ymax:.2f}), K rows {ek:.2e}, V rows {ev:.2e}")
    assert err <= TOL * ymax and ek <= TOL and ev <= TOL
    return err


def test_layer_small_two_requests(taps):
    _run(taps, np.random.default_rng(1), B=2, N=16, H=256, Hq=4, Hkv=2, ctx=[37, 0], n=[16, 11])


@pytest.mark.parametrize("n", [[1, 5], [0, 3]])
def test_layer_edge_node_counts(taps, n):
    """A root-only tree, and a request with no nodes (nothing written, Y undefined)."""
    _run(taps, np.random.default_rng(2 + n[0]), B=2, N=8, H=128, Hq=2, Hkv=1, ctx=[300, 0], n=n)


def test_layer_ragged_rows_span_several_tiles(taps):
    """M = batch * budget = 3 * 40 rows: two 64-row tiles, the second ragged."""
    _run(taps, np.random.default_rng(4), B=3, N=40, H=512, Hq=8, Hkv=2, ctx=[70, 129, 5],
         n=[40, 23, 31])


def test_layer_many_rows_take_the_widest_gemm_tiles(taps):
    """M = 8 x 128 = 1024 rows: the Q/K/V projection's plan takes 128 columns per workgroup
    and one K split (the fewest rounds of workgroups), the output projection 64 columns and
    eight splits; ragged node counts, empty and short contexts."""
    _run(taps, np.random.default_rng(6), B=8, N=128, H=128, Hq=8, Hkv=4,
         ctx=[30, 0, 65, 3, 100, 7, 12, 50], n=[128, 1, 77, 128, 5, 64, 100, 33])


def test_layer_many_pairs_take_four_heads_per_wave(taps):
    """M = 8 x 128 rows and 12 heads per node (8 query, 2 key, 2 value): the rotary pass
    gives each wave four heads of a node (the last group of the node's three partly
    filled: heads 8-11 of one workgroup of 16)."""
    _run(taps, np.random.default_rng(7), B=8, N=128, H=128, Hq=8, Hkv=2,
         ctx=[0, 41, 9, 130, 1, 64, 7, 20], n=[128, 128, 3, 90, 1, 60, 128, 17])


@pytest.mark.parametrize("seed", range(10))
def test_layer_fuzz_shapes(taps, seed):
    """Seeded random shapes: 1-4 requests of 1-70 nodes, hidden 64-1024, 1-16 query heads
    over 1-4 KV heads, ragged contexts up to 400 rows and node counts down to none; the
    GEMM plans they reach vary in columns per workgroup (64, 96) and K splits (1-16)."""
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.integers(1, 5))
    N = int(rng.integers(1, 71))
    H = 64 * int(rng.integers(1, 17))
    Hkv = int(rng.choice([1, 2, 4]))
    Hq = Hkv * int(rng.choice([1, 2, 4]))
    ctx = [int(x) for x in rng.integers(0, 401, B)]
    n = [int(x) for x in rng.integers(0, N + 1, B)]
    n[int(rng.integers(0, B))] = N                  # one request with a full tree
    _run(taps, rng, B=B, N=N, H=H, Hq=Hq, Hkv=Hkv, ctx=ctx, n=n)


def test_layer_qwen3_8b_shape(taps):
    """One Qwen3-8B-shaped layer (hidden 4096, 32/8 heads x 128) over 8192 context rows
    and a 64-node tree; Y on the root, the last node and six random nodes."""
    rng = np.random.default_rng(5)
    picks = sorted({0, 63, *[int(x) for x in rng.integers(1, 63, 6)]})
    _run(taps, rng, B=1, N=64, H=4096, Hq=32, Hkv=8, ctx=[8192], n=[64],
         sample_nodes=lambda b: picks)


def test_layer_graph_replays_match_eager(taps):
    """verify_layer captured in a HIP graph: three replays, with eager work and
    synchronisations between them, each give the eager output bit for bit."""
    rng = np.random.default_rng(9)
    B, N, H, Hq, Hkv, hd, ctx = 2, 16, 256, 4, 2, 128, 40
    dev = lambda *s, sc=1.0: _to_dev(_bf16(rng, *s, scale=sc), torch.bfloat16)
    w = taps.LayerWeights(dev(Hq * hd, H, sc=H ** -0.5), dev(Hkv * hd, H, sc=H ** -0.5),
                          dev(Hkv * hd, H, sc=H ** -0.5), dev(H, Hq * hd, sc=(Hq * hd) ** -0.5),
                          dev(hd), dev(hd))
    rows = B * (ctx + N)
    K, V = dev(rows, Hkv, hd), dev(rows, Hkv, hd)
    off = torch.tensor([0, ctx + N], dtype=torch.int64, device="cuda")
    cl = torch.full((B,), ctx, dtype=torch.int32, device="cuda")
    tree = taps.TreeBuffers.empty(B, 1, 1, N)
    p, d = _tree(rng, N, N)
    tree.parent.copy_(torch.from_numpy(np.stack([p, p])))
    tree.depth.copy_(torch.from_numpy(np.stack([d, d])))
    tree.n_nodes.fill_(N)
    X = dev(B, N, H)
    lay = taps.VerifyLayer(B, N, Hq, Hkv, hd, H, ctx)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        want = lay(X, w, K, V, off, cl, tree).clone()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            lay(X, w, K, V, off, cl, tree)
        for rep in range(3):
            lay.Y.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(lay.Y[:, :N], want[:, :N]), f"replay {rep}"
            _ = (X.float() * 2).sum().item()          # eager work between replays

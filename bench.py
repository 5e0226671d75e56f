"""Benchmark one TAPS verification round (selection + tree attention + acceptance walk).

    python bench.py [--steps K] [--warmup W] [--config qwen3_8b] [--eager] [--no-cpu-baseline]

A step is one whole round over one batch: taps_select (vocab top-K, Eq. 1-3,
Alg. 1), tree_verify_attn and accept_walk, launched on one stream.  Inputs are
seeded synthetic rounds from ``workloads`` (Gaussian drafter logits with planted
spikes, random bf16 Q/K/V, fixed acceptance probability per request), held in
HBM before timing; several independent input sets rotate so that the 256 MB
Infinity Cache cannot hold the working set.  Rounds are replayed from one HIP
graph per input set (``--eager`` launches them directly).

Prints one JSON line.  ``value`` is rounds/s (requests x steps per second);
``roofline`` covers the dominant kernel (the main tree-attention kernel), timed
with HIP events around that kernel alone in a separate pass of the same
launches; ``cpu_baseline`` times the CPU oracle on a bounded sample.  The
round's state update (kv_commit of the accepted path) is not part of the step;
``stages_us.kv_commit`` and ``kv_commit`` report it from its own timed pass.  ``layer``
reports one attention layer of the target over the tree (verify_layer, hidden = Hq x
head_dim, seeded random bf16 weights), also timed on its own and not part of the step.
``stages_us`` times the round's three calls with events between eager launches;
``stages_graph_us`` times each call from HIP graphs of ten back-to-back calls per input
set (the graph-launched cost of its kernels, next to the round's own graph time).
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("verification rounds/sec (select+tree-attn+accept) and achieved HBM GB/s, "
          "Qwen3-8B shape")
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0        # dense bf16 matrix-core peak of MI355X
RIDGE = MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)   # flop per byte
MALL_BYTES = 256 << 20
ATTN_SRC = os.path.join(ROOT, "paper_2606_00487_amd", "csrc", "attn.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_bf16_kernel_qwen3_8b_hbm.txt")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--config", default="qwen3_8b")
    ap.add_argument("--budget", type=int, default=0,
                    help="override the configuration's node budget N (1..512)")
    ap.add_argument("--lambda2", type=float, default=None,
                    help="override lambda2 of Eq. 3 (0 with --tau 0: no cost-aware pruning)")
    ap.add_argument("--tau", type=float, default=None, help="override the utility threshold")
    ap.add_argument("--scorer", choices=["sibling", "marginal", "learned"], default="sibling",
                    help="marginal: q_cond is the full-vocabulary marginal (the scoring ablation); "
                         "learned: the learned-scorer hook with seeded random weights "
                         "(embedding 16, hidden 32)")
    ap.add_argument("--sets", type=int, default=0, help="input sets to rotate (0: enough to exceed the MALL)")
    ap.add_argument("--paged", type=int, default=0,
                    help="the round's attention (and the kv_commit and layer passes) use a "
                         "paged KV cache with pages of this many rows (a power of two, "
                         "32..4096; pages in random order); 0: contiguous")
    ap.add_argument("--eager", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=20.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy (reference for the HBM byte counters)")
    return ap.parse_args()


def paged_copy(torch, K, V, kv_offset, ctx_len, budget, max_ctx, page_rows, rng, dev):
    """Request b's cache rows (its context, then its budget tree rows) copied page by page
    into pools, the pages in random order; returns the pools and the block table."""
    B = len(ctx_len)
    need = [-(-(int(ctx_len[b]) + budget) // page_rows) for b in range(B)]
    ids = rng.permutation(sum(need))
    table = np.zeros((B, -(-(max_ctx + budget) // page_rows)), dtype=np.int32)
    src, dst = [], []
    k = 0
    for b in range(B):
        rows = int(ctx_len[b]) + budget
        for p in range(need[b]):
            lo, hi = p * page_rows, min(rows, (p + 1) * page_rows)
            table[b, p] = ids[k]
            src.append(np.arange(lo, hi) + int(kv_offset[b]))
            dst.append(np.arange(hi - lo) + int(ids[k]) * page_rows)
            k += 1
    src = torch.from_numpy(np.concatenate(src)).to(dev)
    dst = torch.from_numpy(np.concatenate(dst)).to(dev)
    pools = []
    for X in (K, V):
        P = torch.zeros((sum(need) * page_rows,) + tuple(X.shape[1:]), dtype=X.dtype, device=dev)
        P[dst] = X[src]
        pools.append(P.view((sum(need), page_rows) + tuple(X.shape[1:])))
    return pools[0], pools[1], torch.from_numpy(table).to(dev)


def copy_calibration():
    """A plain copy of known size: FETCH_SIZE / WRITE_SIZE measured on it give the factor
    that turns those counters into bytes for the kernels of the round."""
    import torch
    n = 256 << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}), flush=True)


def measured_traffic(cfg_name):
    """HBM bytes per launch of the main attention kernel from the committed counter
    summary (FETCH_SIZE and WRITE_SIZE per dispatch, each scaled by what the counter reads
    for a plain copy of known size), or None when the summary does not cover this
    workload or the kernel source has changed since the counters were taken."""
    import hashlib
    if cfg_name != "qwen3_8b" or not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        line = line.strip()
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    sha = hashlib.sha256(open(ATTN_SRC, "rb").read()).hexdigest()
    if kv.get("attn_source_sha256") != sha:
        return None
    return int(float(kv["fetch_kib_per_launch"]) * 1024 * float(kv["fetch_scale"]) +
               float(kv["write_kib_per_launch"]) * 1024 * float(kv["write_scale"]))


def algorithmic_bytes(cfg, ctx_len, n_nodes):
    """Bytes the method must move per round: each marginal once, each KV row of the
    context and of the selected nodes once per KV head (K and V), Q and O of the
    selected nodes once."""
    es = 2 if cfg.dtype == 0 else 4
    marg = cfg.batch * cfg.block * cfg.vocab * es
    kv = sum(int(c) + int(n) for c, n in zip(ctx_len, n_nodes)) * cfg.Hkv * cfg.head_dim * es * 2
    qo = sum(int(n) for n in n_nodes) * cfg.Hq * cfg.head_dim * es * 2
    return marg, kv, qo


def attention_flops(cfg, ctx_len, n_nodes):
    """Matrix-core work of the tree attention, dense over each request's context and tree
    rows: Q K^T and P V for every selected node and query head, 4 * n * Hq * (ctx + n) * hd
    per request."""
    return sum(4 * int(n) * cfg.Hq * (int(c) + int(n)) * cfg.head_dim
               for c, n in zip(ctx_len, n_nodes))


def spread(us):
    """Median and 10th / 90th percentiles of per-round times (us)."""
    a = np.asarray(us, dtype=np.float64)
    return {"median": round(float(np.median(a)), 3), "p10": round(float(np.percentile(a, 10)), 3),
            "p90": round(float(np.percentile(a, 90)), 3), "rounds": int(a.size)}


def commit_moved_bytes(cfg, path, path_len):
    """Algorithmic bytes of one kv_commit: every committed path entry that is not already at
    its target row is read and written once, in K and in V."""
    row = cfg.Hkv * cfg.head_dim * (2 if cfg.dtype == 0 else 4)
    moved = 0
    for b in range(cfg.batch):
        m = int(path_len[b])
        moved += sum(1 for j in range(1, m) if int(path[b][j]) != j)
    return moved * row * 2 * 2


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus "
              f"{args.gpus}); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2606_00487_amd as taps
    from workloads import BF16, CONFIGS, gen_round, target_tokens

    taps.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = CONFIGS[args.config]
    over = {}
    if args.budget:
        over["budget"] = args.budget
    if args.lambda2 is not None:
        over["lambda2"] = args.lambda2
    if args.tau is not None:
        over["tau"] = args.tau
    scorer = {"sibling": 0, "marginal": 1, "learned": 2}[args.scorer]
    tag = ",".join([f"{k}={v}" for k, v in over.items()] +
                   ([f"scorer={args.scorer}"] if scorer else []))
    if tag:    # a variant of the configuration: its name records the overrides
        cfg = dataclasses.replace(cfg, name=f"{cfg.name}[{tag}]", **over)
    bf = cfg.dtype == BF16

    def to_dev(a):
        a = np.ascontiguousarray(a)
        if bf:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    # ---------------- input sets
    inp0 = gen_round(cfg, with_attention=True)
    set_bytes = (inp0.marginals.nbytes + inp0.Q.nbytes + inp0.K.nbytes + inp0.V.nbytes)
    nsets = args.sets or max(1, min(16, -(-(MALL_BYTES + (MALL_BYTES >> 2)) // set_bytes)))
    if set_bytes > MALL_BYTES:
        nsets = args.sets or 1
    max_ctx = int(max(gen_round(cfg, seed=inp0.seed + k, with_attention=False).ctx_len.max()
                      for k in range(nsets)))
    mlp = mlp_dev = None
    if scorer == 2:       # seeded random weights: the paper's trained weights are not published
        from workloads import gen_scorer_weights
        mlp = gen_scorer_weights(np.random.default_rng(20260602), cfg.vocab, 16, 32, cfg.batch)
        mlp_dev = taps.ScorerWeights(
            emb=torch.from_numpy(mlp["emb"]).to(dev), W1=torch.from_numpy(mlp["W1"]).to(dev),
            b1=torch.from_numpy(mlp["b1"]).to(dev), w2=torch.from_numpy(mlp["w2"]).to(dev),
            b2=mlp["b2"], root_token=torch.from_numpy(mlp["root_token"]).to(dev))
    sel = taps.Selector(cfg.batch, cfg.block, cfg.vocab, cfg.K, cfg.budget, dtype=cfg.dtype,
                        kind=cfg.kind, lambda1=cfg.lambda1, lambda2=cfg.lambda2, tau=cfg.tau,
                        beta=cfg.beta, scorer=scorer, mlp=mlp_dev)
    att = taps.TreeAttention(cfg.batch, cfg.budget, cfg.Hq, cfg.Hkv, cfg.head_dim, max_ctx,
                             dtype=cfg.dtype, scale=cfg.scale)
    patt = None
    if args.paged:
        if not bf or cfg.head_dim != 128:
            sys.exit("--paged needs bf16 and head_dim 128")
        patt = taps.PagedTreeAttention(cfg.batch, cfg.budget, cfg.Hq, cfg.Hkv, max_ctx,
                                       args.paged, scale=cfg.scale)
    walk = taps.AcceptWalk(cfg.batch, cfg.budget, cfg.block)
    commit = taps.KVCommit(cfg.batch, cfg.budget, cfg.block, cfg.Hkv, cfg.head_dim, max_ctx,
                           dtype=cfg.dtype)
    pcommit = taps.PagedKVCommit(cfg.batch, cfg.budget, cfg.block, cfg.Hkv, cfg.head_dim, max_ctx,
                                 args.paged, dtype=cfg.dtype) if args.paged else None
    sets = []
    for k in range(nsets):
        inp = inp0 if k == 0 else gen_round(cfg, seed=inp0.seed + k)
        s = dict(inp=inp, marg=to_dev(inp.marginals), Q=to_dev(inp.Q), K=to_dev(inp.K),
                 V=to_dev(inp.V), off=torch.from_numpy(inp.kv_offset).to(dev),
                 ctx=torch.from_numpy(inp.ctx_len).to(dev),
                 tree=taps.TreeBuffers.empty(cfg.batch, cfg.block, cfg.K, cfg.budget, dev),
                 O=torch.empty((cfg.batch, cfg.budget, cfg.Hq, cfg.head_dim),
                               dtype=torch.bfloat16 if bf else torch.float32, device=dev))
        # the synthetic target tokens follow the selected tree: one untimed selection
        sel(s["marg"], s["tree"])
        torch.cuda.synchronize()
        par = s["tree"].parent.cpu().numpy()
        rnk = s["tree"].rank.cpu().numpy()
        nn = s["tree"].n_nodes.cpu().numpy()
        top1 = s["tree"].topk_idx.cpu().numpy()[:, :, 0]
        tok = s["tree"].token.cpu().numpy()
        tgt = np.stack([target_tokens(cfg, b, par[b], rnk[b], int(nn[b]), top1[b], inp.p_acc[b],
                                      seed=inp.seed, token=tok[b]) for b in range(cfg.batch)])
        s["tgt"] = torch.from_numpy(tgt.astype(np.int32)).to(dev)
        s["n"] = nn.copy()
        if patt is not None:
            s["Kp"], s["Vp"], s["tab"] = paged_copy(
                torch, s["K"], s["V"], inp.kv_offset, inp.ctx_len, cfg.budget, max_ctx,
                args.paged, np.random.default_rng(inp.seed + 17), dev)
        sets.append(s)
        print(f"[bench] input set {k + 1}/{nsets} ready (n_nodes {nn.tolist()[:4]}...)",
              file=sys.stderr, flush=True)

    def attn_call(s, events=None):
        if patt is not None:
            patt(s["Q"], s["Kp"], s["Vp"], s["tab"], s["ctx"], s["tree"].parent,
                 s["tree"].n_nodes, out=s["O"], events=events)
        else:
            att(s["Q"], s["K"], s["V"], s["off"], s["ctx"], s["tree"].parent, s["tree"].n_nodes,
                out=s["O"], events=events)

    def round_(s, events=None):
        sel(s["marg"], s["tree"])
        attn_call(s, events)
        walk(s["tree"], s["tgt"])

    stream = torch.cuda.Stream()
    graphs = []
    with torch.cuda.stream(stream):
        for s in sets:                      # warm once before capture
            round_(s)
        torch.cuda.synchronize()
        if not args.eager:
            for s in sets:
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=stream):
                    round_(s)
                graphs.append(g)
        torch.cuda.synchronize()

        def run_set(k):
            if args.eager:
                round_(sets[k])
            else:
                graphs[k].replay()

        def step(i):
            run_set(i % nsets)

        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            step(i)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        elapsed = t1 - t0

        # ---------------- per-round times: events between consecutive rounds, with the input
        # sets rotating (cold: more than the Infinity Cache holds) and with one set repeated
        # (warm: its working set stays in the cache)
        def per_round(order):
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(order) + 1)]
            for e in evs:                     # materialise the event handles
                e.record(stream)
            torch.cuda.synchronize()
            evs[0].record(stream)
            for k, si in enumerate(order):
                run_set(si)
                evs[k + 1].record(stream)
            torch.cuda.synchronize()
            return [evs[k].elapsed_time(evs[k + 1]) * 1e3 for k in range(len(order))]

        R = max(2 * nsets, min(args.steps, 300))
        for _ in range(2):
            run_set(0)
        dist_cold = spread(per_round([i % nsets for i in range(R)]))
        dist_warm = spread(per_round([0] * R))

        # ---------------- per-stage timing pass (eager, same launches, HIP events)
        reps = max(nsets, min(args.steps, 200))
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(reps)]
        for e in ev:                          # materialise the event handles
            for x in e:
                x.record(stream)
        torch.cuda.synchronize()
        # a head start for the host: while the GPU sleeps, the timed launches queue up, so
        # that they run back to back as in the graphs (an idle GPU between launches would
        # add its wake-up to every kernel's time)
        torch.cuda._sleep(int(2e7))
        for r in range(reps):
            s = sets[r % nsets]
            e = ev[r]
            e[0].record(stream)
            sel(s["marg"], s["tree"])
            e[1].record(stream)
            attn_call(s, (e[2], e[3]))
            e[4].record(stream)
            walk(s["tree"], s["tgt"])
            e[5].record(stream)
        torch.cuda.synchronize()

        # ---------------- per-stage times from HIP graphs: for each stage one graph of GR
        # back-to-back calls per input set, replayed over the rotating sets, so that each
        # figure carries the graph-launched start-up of the round's own kernels
        stage_graph = {}
        if not args.eager:
            GR = 10
            stage_calls = {
                "select": lambda s: sel(s["marg"], s["tree"]),
                "attn_call": lambda s: attn_call(s),
                "walk": lambda s: walk(s["tree"], s["tgt"]),
            }
            for name, fn in stage_calls.items():
                gs = []
                for s in sets:
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=stream):
                        for _ in range(GR):
                            fn(s)
                    gs.append(g)
                for g in gs:                      # warm
                    g.replay()
                g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                g0.record(stream)
                for _ in range(2):
                    for g in gs:
                        g.replay()
                g1.record(stream)
                torch.cuda.synchronize()
                stage_graph[name] = round(g0.elapsed_time(g1) * 1e3 / (2 * len(gs) * GR), 2)
                del gs
            stage_graph["sum"] = round(sum(stage_graph.values()), 2)

        # ---------------- the round's state update (kv_commit), timed on its own from a HIP
        # graph of back-to-back calls per input set (eager events would include the host's
        # launch overhead).  It moves tree rows of the cache in place and does not write
        # ctx_len, so repeated calls do the same work; it runs after everything else.
        commit_bytes, commit_us = [], []
        CR = 20
        for s in sets:
            walk(s["tree"], s["tgt"])
            torch.cuda.synchronize()
            commit_bytes.append(commit_moved_bytes(cfg, walk.path.cpu().numpy(),
                                                   walk.path_len.cpu().numpy()))
            gc = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gc, stream=stream):
                for _ in range(CR):
                    if pcommit is not None:
                        pcommit(s["Kp"], s["Vp"], s["tab"], s["ctx"], s["tree"], walk.path,
                                walk.path_len, walk.bonus)
                    else:
                        commit(s["K"], s["V"], s["off"], s["ctx"], s["tree"], walk.path,
                               walk.path_len, walk.bonus)
            gc.replay()
            c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            c0.record(stream)
            for _ in range(3):
                gc.replay()
            c1.record(stream)
            torch.cuda.synchronize()
            commit_us.append(c0.elapsed_time(c1) * 1e3 / (3 * CR))
        # ---------------- one attention layer of the target over the tree (verify_layer),
        # Qwen3-style with hidden = Hq * head_dim and seeded random bf16 weights, timed on its
        # own like kv_commit; it rewrites the tree rows of the cache with its own keys and
        # values, so it runs last.
        layer_us, layer_b = [], []
        if bf and cfg.head_dim == 128:
            H = cfg.Hq * cfg.head_dim
            gen = torch.Generator(device=dev)
            gen.manual_seed(20260603)

            def rnd(*shape, scale=1.0):
                return (torch.randn(*shape, generator=gen, device=dev) * scale).to(torch.bfloat16)

            hd = cfg.head_dim
            lw = taps.LayerWeights(rnd(cfg.Hq * hd, H, scale=H ** -0.5),
                                   rnd(cfg.Hkv * hd, H, scale=H ** -0.5),
                                   rnd(cfg.Hkv * hd, H, scale=H ** -0.5),
                                   rnd(H, cfg.Hq * hd, scale=(cfg.Hq * hd) ** -0.5),
                                   (1 + 0.1 * torch.randn(hd, generator=gen, device=dev)).to(torch.bfloat16),
                                   (1 + 0.1 * torch.randn(hd, generator=gen, device=dev)).to(torch.bfloat16))
            if args.paged:
                lay = taps.PagedVerifyLayer(cfg.batch, cfg.budget, cfg.Hq, cfg.Hkv, hd, H,
                                            max_ctx, args.paged, scale=cfg.scale)
            else:
                lay = taps.VerifyLayer(cfg.batch, cfg.budget, cfg.Hq, cfg.Hkv, hd, H, max_ctx,
                                       scale=cfg.scale)
            Xl = rnd(cfg.batch, cfg.budget, H)
            w_bytes = 2 * H * (cfg.Hq + 2 * cfg.Hkv) * hd + 2 * H * cfg.Hq * hd
            LR = 10
            for sl in sets[:3]:
                p = algorithmic_bytes(cfg, sl["inp"].ctx_len, sl["n"])
                layer_b.append(w_bytes + 4 * cfg.batch * cfg.budget * H + p[1] + p[2])
                gl = torch.cuda.CUDAGraph()
                with torch.cuda.graph(gl, stream=stream):
                    for _ in range(LR):
                        if args.paged:
                            lay(Xl, lw, sl["Kp"], sl["Vp"], sl["tab"], sl["ctx"], sl["tree"])
                        else:
                            lay(Xl, lw, sl["K"], sl["V"], sl["off"], sl["ctx"], sl["tree"])
                gl.replay()
                c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                c0.record(stream)
                for _ in range(3):
                    gl.replay()
                c1.record(stream)
                torch.cuda.synchronize()
                layer_us.append(c0.elapsed_time(c1) * 1e3 / (3 * LR))
    t_commit = float(np.mean(commit_us))
    commit_b = float(np.mean(commit_bytes))
    t_sel = float(np.mean([e[0].elapsed_time(e[1]) for e in ev])) * 1e3
    t_attn = float(np.mean([e[2].elapsed_time(e[3]) for e in ev])) * 1e3
    t_attn_call = float(np.mean([e[1].elapsed_time(e[4]) for e in ev])) * 1e3
    t_walk = float(np.mean([e[4].elapsed_time(e[5]) for e in ev])) * 1e3
    dist_eager = spread([e[0].elapsed_time(e[5]) * 1e3 for e in ev])

    # ---------------- bytes and roofline
    per_set = [algorithmic_bytes(cfg, s["inp"].ctx_len, s["n"]) for s in sets]
    marg_b = float(np.mean([p[0] for p in per_set]))
    kv_b = float(np.mean([p[1] for p in per_set]))
    qo_b = float(np.mean([p[2] for p in per_set]))
    round_bytes = marg_b + kv_b + qo_b
    attn_bytes = kv_b + qo_b
    attn_fl = float(np.mean([attention_flops(cfg, s["inp"].ctx_len, s["n"]) for s in sets]))
    intensity = attn_fl / attn_bytes
    ms_per_step = elapsed / args.steps * 1e3
    rounds_per_s = cfg.batch * args.steps / elapsed
    achieved = attn_bytes / (t_attn * 1e-6) / 1e9
    traffic = None if args.paged else measured_traffic(cfg.name)   # counters: contiguous only
    attn_kernel = (("attn_bf16_paged_kernel" if args.paged else "attn_bf16_kernel") if bf
                   else "attn_f32_kernel")
    if bf and intensity > RIDGE:
        # more flops per byte than the machine balance: the matrix cores bound the kernel
        roofline = {"bound": "mfma", "kernel": attn_kernel,
                    "achieved": round(attn_fl / (t_attn * 1e-6) / 1e12, 1),
                    "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(attn_fl / (t_attn * 1e-6) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)}
    else:
        roofline = {"bound": "hbm", "kernel": attn_kernel,
                    "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4)}
    roofline.update({
        "traffic": traffic,
        "traffic_source": (os.path.relpath(TRAFFIC_FILE, ROOT) + ": rocprofv3 --pmc FETCH_SIZE, "
                           "WRITE_SIZE of this kernel source, scaled by a plain copy")
        if traffic is not None else None,
        "bytes_per_launch": int(attn_bytes),
        "flops_per_launch": int(attn_fl),
        "intensity_flop_per_byte": round(intensity, 1),
        "ridge_flop_per_byte": round(RIDGE, 1),
        "hbm_frac": round(achieved / HBM_PEAK_GBS, 4),
        "mfma_frac": round(attn_fl / (t_attn * 1e-6) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)
        if bf else None,
        "avg_launch_us": round(t_attn, 3),
    })
    out = {
        "metric": METRIC,
        "value": round(rounds_per_s, 2),
        "unit": "rounds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf else "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name}: batch {cfg.batch}, marginals [{cfg.block}, {cfg.vocab}] "
                        f"{'bf16 logits' if bf else 'fp32 probs'}, top-{cfg.K}, budget {cfg.budget}, "
                        f"{cfg.Hq}/{cfg.Hkv} heads x {cfg.head_dim}, context {int(s['inp'].ctx_len.max())}"
                        + (f", lambda2 {cfg.lambda2}, tau {cfg.tau}" if over else "")
                        + (f", {args.scorer} scorer" if scorer else "")
                        + (f", paged KV ({args.paged}-row pages)" if args.paged else ""),
            "global_batch": cfg.batch,
            "budget": cfg.budget,
            "input_sets": nsets,
            "graph": not args.eager,
        },
        "hbm_gbs_round": round(round_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "round_bytes": int(round_bytes),
        "round_us": {"graph_cold": dist_cold, "graph_warm": dist_warm, "eager_cold": dist_eager},
        "stages_us": {"select": round(t_sel, 2), "attn_main_kernel": round(t_attn, 2),
                      "attn_call": round(t_attn_call, 2), "walk": round(t_walk, 2),
                      "kv_commit": round(t_commit, 2)},
        "stages_graph_us": stage_graph or None,
        "kv_commit": {"bytes_per_launch": int(commit_b),
                      "achieved_gbs": round(commit_b / (t_commit * 1e-6) / 1e9, 1),
                      "avg_launch_us": round(t_commit, 3)},
        "layer": None if not layer_us else {
            "what": f"one attention layer over the tree: hidden {cfg.Hq * cfg.head_dim}, "
                    "projections + RMSNorm + rotary + tree attention + output projection",
            "bytes_per_launch": int(np.mean(layer_b)),
            "achieved_gbs": round(float(np.mean(layer_b)) / (float(np.mean(layer_us)) * 1e-6) / 1e9, 1),
            "avg_launch_us": round(float(np.mean(layer_us)), 3)},
        "roofline": roofline,
        "round_roofline_frac": round((round_bytes / HBM_PEAK_GBS / 1e3) / (ms_per_step * 1e3), 4),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, sets[0]["inp"], args.cpu_budget_s, scorer, mlp)
    print(json.dumps(out), flush=True)


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo) and the cores this process may run on."""
    import platform
    model = platform.processor() or "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover - not Linux
        cores = os.cpu_count() or 1
    return model, cores


def oracle_round(cfg, inp, budget_s, scorer=0, mlp=None):
    """The oracle as it stands over one round of `inp`: the whole selection, the attention of
    as many (node, head) rows as fit in budget_s (extrapolated to all rows), the walk.
    Returns (seconds per round, the sample's description)."""
    import oracle
    from workloads import target_tokens
    x = inp.marginals_f64()
    t0 = time.perf_counter()
    w = None
    if mlp is not None:
        from oracle.scorer import MLPScorer
        w = MLPScorer(**mlp)
    trees = [oracle.select_request(x[b], cfg.K, cfg.budget, kind=cfg.kind, lambda1=cfg.lambda1,
                                   lambda2=cfg.lambda2, tau=cfg.tau, beta=cfg.beta,
                                   scorer=scorer, mlp=w, req=b)
             for b in range(cfg.batch)]
    t_sel = time.perf_counter() - t0
    Qd, Kd, Vd = inp.qkv_f64()
    rows = [(b, i, h) for b in range(cfg.batch) for i in range(trees[b].n) for h in range(cfg.Hq)]
    t0 = time.perf_counter()
    done = 0
    chunk = max(1, cfg.Hq)
    while done < len(rows) and time.perf_counter() - t0 < budget_s:
        oracle.tree_attention(Qd, Kd, Vd, inp.kv_offset, inp.ctx_len, [t.parent for t in trees],
                              [t.n for t in trees], cfg.scale, samples=rows[done:done + chunk])
        done += chunk
    done = min(done, len(rows))
    t_attn = (time.perf_counter() - t0) * len(rows) / done
    t0 = time.perf_counter()
    for b, t in enumerate(trees):
        tgt = target_tokens(cfg, b, t.parent, t.rank, t.n, t.topk_idx[:, 0], inp.p_acc[b])
        oracle.accept_walk(t.parent, t.token, t.n, tgt)
    t_walk = time.perf_counter() - t0
    desc = (f"selection {t_sel:.2f} s, attention {done}/{len(rows)} (node, head) rows "
            f"extrapolated to all {t_attn:.1f} s, walk {t_walk:.3f} s")
    return t_sel + t_attn + t_walk, desc


def cpu_baseline(cfg, inp, budget_s, scorer=0, mlp=None):
    """The oracle as it stands, on this host, over a bounded sample of one round: once with
    the BLAS pool at its default size (the attention's products use it; selection and walk
    are single-threaded Python) and once limited to one thread."""
    model, avail = cpu_model()
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([t.get("num_threads", 1) for t in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl missing
        threadpool_limits, threads = None, 1
    per_round, desc = oracle_round(cfg, inp, budget_s / 2, scorer, mlp)
    single = None
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            t1, d1 = oracle_round(cfg, inp, budget_s / 2, scorer, mlp)
        single = {"value": round(cfg.batch / t1, 5), "unit": "rounds/s", "cores": 1,
                  "sample": d1}
    return {
        "value": round(cfg.batch / per_round, 5),
        "unit": "rounds/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"one round of {cfg.name}, fp64 NumPy oracle: {desc}",
        "cpu_model": model,
        "cores_available": int(avail),
        "single_thread": single,
    }


if __name__ == "__main__":
    main()

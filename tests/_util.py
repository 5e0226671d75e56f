"""Helpers shared by the GPU tests: upload seeded inputs, run the oracle, compare."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from workloads import BF16, Config, RoundInputs, target_tokens


def to_dev(a: np.ndarray, bf16: bool) -> torch.Tensor:
    if bf16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def oracle_trees(inp: RoundInputs, **over) -> list[oracle.Tree]:
    c = inp.cfg
    kw = dict(kind=c.kind, lambda1=c.lambda1, lambda2=c.lambda2, tau=c.tau, beta=c.beta)
    kw.update(over)
    x = inp.marginals_f64()
    return [oracle.select_request(x[b], c.K, c.budget, **kw) for b in range(c.batch)]


def assert_tree_equal(gpu, trees: list[oracle.Tree], cfg: Config):
    par = gpu.parent.cpu().numpy()
    tok = gpu.token.cpu().numpy()
    dep = gpu.depth.cpu().numpy()
    rnk = gpu.rank.cpu().numpy()
    q = gpu.q_reach.cpu().numpy()
    n = gpu.n_nodes.cpu().numpy()
    tidx = gpu.topk_idx.cpu().numpy()
    tval = gpu.topk_val.cpu().numpy()
    for b, t in enumerate(trees):
        assert n[b] == t.n, (b, n[b], t.n)
        np.testing.assert_array_equal(tidx[b], t.topk_idx, err_msg=f"topk_idx b={b}")
        ov = t.topk_val.astype(np.float32)
        same = (tval[b] == ov) | (np.isnan(tval[b]) & np.isnan(ov))
        assert same.all(), f"topk_val b={b}"
        np.testing.assert_array_equal(par[b], t.parent, err_msg=f"parent b={b}")
        np.testing.assert_array_equal(tok[b], t.token, err_msg=f"token b={b}")
        np.testing.assert_array_equal(dep[b], t.depth, err_msg=f"depth b={b}")
        np.testing.assert_array_equal(rnk[b], t.rank, err_msg=f"rank b={b}")
        assert np.array_equal(q[b].view(np.int64), t.q_reach.view(np.int64)), f"q_reach bits b={b}"


def targets_for(inp: RoundInputs, trees: list[oracle.Tree], branch: bool = False) -> np.ndarray:
    c = inp.cfg
    out = np.stack([target_tokens(c, b, t.parent, t.rank, t.n, t.topk_idx[:, 0], inp.p_acc[b],
                                  seed=inp.seed, branch=branch, token=t.token)
                    for b, t in enumerate(trees)])
    return out.astype(np.int32)


def tree_device(trees: list[oracle.Tree]):
    parent = torch.from_numpy(np.stack([t.parent for t in trees]).astype(np.int32)).cuda()
    token = torch.from_numpy(np.stack([t.token for t in trees]).astype(np.int32)).cuda()
    n = torch.tensor([t.n for t in trees], dtype=torch.int32).cuda()
    return parent, token, n


def attention_inputs(inp: RoundInputs):
    bf = inp.cfg.dtype == BF16
    return (to_dev(inp.Q, bf), to_dev(inp.K, bf), to_dev(inp.V, bf),
            torch.from_numpy(inp.kv_offset).cuda(), torch.from_numpy(inp.ctx_len).cuda())


def gpu_o_as_f64(O: torch.Tensor) -> np.ndarray:
    return O.float().cpu().numpy().astype(np.float64)


# ------------------------------------------------------------------ selection fallback
# The selection kernel expands the trie level by level into LDS (kCap stored nodes in
# paper_2606_00487_amd/csrc/select.hip, 1024 utility bins of exponent + 3 mantissa bits)
# and falls back to a sequential best-first loop when an expansion outgrows that space.
# The emulation below counts what the level expansion stores, so that a test can show on
# the CPU that an input really takes the fallback.
LEVEL_CAP = 3072
_BINS = 1024
_BIN_BASE = (1023 - 110) * 8


def _ubin(u: float) -> int:
    import struct
    b = (struct.unpack("<q", struct.pack("<d", u))[0] >> 49) - _BIN_BASE
    return 0 if b < 0 else min(b, _BINS - 1)


def level_expansion_overflows(c: np.ndarray, den: np.ndarray, N: int, tau: float,
                              cap: int = LEVEL_CAP) -> bool:
    """True when the level-by-level expansion of the selection kernel stores more than `cap`
    nodes.  c: q_cond [D][K] or the learned scorer's [D][K][K] table; den: Eq. 3 denominators."""
    D, K = c.shape[0], c.shape[-1]
    q, u, rank = [1.0], [1.0 / den[0]], [0]
    hist = np.zeros(_BINS, dtype=np.int64)
    p0, p1, bstar = 0, 1, 0
    for d in range(D):
        if N <= 1 or p1 == p0:
            break
        for p in range(p0, p1):
            for r in range(K):
                cr = c[d, rank[p], r] if c.ndim == 3 else c[d, r]
                qq = q[p] * cr
                uu = qq / den[d + 1]
                bn = _ubin(uu)
                if _ubin(u[p]) >= bstar and uu > tau and bn >= bstar:
                    q.append(qq)
                    u.append(uu)
                    rank.append(r)
                    hist[bn] += 1
        if len(q) > cap:
            return True
        p0, p1 = p1, len(q)
        if len(q) >= N - 1:
            above = np.cumsum(hist[::-1])[::-1]            # nodes in bins >= j
            ok = np.nonzero(above >= N - 1)[0]
            bstar = int(ok[-1]) if ok.size else 0
    return False


def fallback_cases():
    """Inputs whose selection takes the sequential fallback (checked on the CPU by
    level_expansion_overflows): name -> dict(dtype, kind, scorer, K, N, lam2, marginals
    [1][D][V] as stored (bf16 bits or fp32), mlp or None)."""
    from oracle.scorer import MLPScorer
    from workloads import f32_to_bf16_bits
    from workloads import BF16 as _BF, FP32 as _FP, LOGITS as _LG, PROBS as _PR
    cases = {}
    # marginal scorer on probabilities, every candidate 1.0: u = 1 for every trie node, so
    # nothing is ever pruned; the answer is the breadth-first lexicographic tree
    D, V, K = 8, 1000, 16
    x = np.full((1, D, V), 5e-4, np.float32)
    for i in range(D):
        x[0, i, 40 * i + 3:40 * i + 3 + K] = 1.0
    cases["marginal_probs_all_one"] = dict(dtype=_FP, kind=_PR, scorer=1, K=K, N=256, lam2=0.0,
                                          marginals=x, mlp=None)
    # sibling scorer: two uniform rows, then one-hot rows: a plateau of chains at u = 1/256
    D = 32
    x = np.zeros((1, D, V), np.float32)
    for i in range(D):
        if i < 2:
            x[0, i, 20 * i + 1:20 * i + 1 + K] = 1.0 / K
        else:
            x[0, i, 20 * i + 7] = 1.0
    cases["sibling_probs_plateau"] = dict(dtype=_FP, kind=_PR, scorer=0, K=K, N=256, lam2=0.0,
                                         marginals=x, mlp=None)
    # the same plateau from bf16 logits with large spikes (the other children are tiny but
    # positive, so they are stored until the pruning bin is known)
    x = np.full((1, D, V), -100.0, np.float32)
    for i in range(D):
        if i < 2:
            x[0, i, 20 * i + 1:20 * i + 1 + K] = 0.0
        else:
            x[0, i, 20 * i + 1:20 * i + 1 + K] = -60.0
            x[0, i, 20 * i + 7] = 0.0
    cases["sibling_logits_plateau"] = dict(dtype=_BF, kind=_LG, scorer=0, K=K, N=256, lam2=0.0,
                                          marginals=f32_to_bf16_bits(x), mlp=None)
    # learned scorer whose logit is the child token's embedding alone: at depth 1 the rank-5
    # candidate has q_cond 0.9, below it the rank-3 candidate of every row has q_cond ~1, so
    # the best nodes are chains through rank-3 children that the rank order would not reach
    V, D = 1024, 24                            # D * K * K within the learned table's limit
    x = np.full((1, D, V), -20.0, np.float32)
    emb = np.zeros((V, 1), np.float32)
    for i in range(D):
        toks = 100 + 20 * i + np.arange(K)
        x[0, i, toks] = 8.0 - 0.25 * np.arange(K)
        if i == 0:
            emb[toks[5], 0] = np.float32(np.log(135.0))
        else:
            emb[toks[3], 0] = 20.0
    mlp = MLPScorer(emb=emb, W1=np.array([[0.0, 1.0, 0.0, 0.0, 0.0]], np.float32),
                    b1=np.zeros(1, np.float32), w2=np.ones(1, np.float32), b2=0.0,
                    root_token=np.array([-1], np.int32))
    cases["learned_child_chains"] = dict(dtype=_BF, kind=_LG, scorer=2, K=K, N=256, lam2=0.0,
                                        marginals=f32_to_bf16_bits(x), mlp=mlp)
    return cases


def fallback_oracle(case):
    """(oracle tree, q_cond table, denominators) of one fallback case."""
    from oracle.scorer import scorer_table
    from oracle.select import denominators, edge_factors, marginal_factors
    from workloads import BF16 as _BF, bf16_bits_to_f32
    m = case["marginals"]
    x = (bf16_bits_to_f32(m) if case["dtype"] == _BF else m).astype(np.float64)[0]
    t = oracle.select_request(x, case["K"], case["N"], kind=case["kind"], lambda1=1.0,
                              lambda2=case["lam2"], tau=0.0, scorer=case["scorer"],
                              mlp=case["mlp"], req=0)
    if case["scorer"] == 1:
        c = marginal_factors(t.topk_val, x, case["kind"])
    elif case["scorer"] == 2:
        c = scorer_table(case["mlp"], 0, x, t.topk_idx, t.topk_val)
    else:
        c = edge_factors(t.topk_val, case["kind"], 1.0)
    return t, c, denominators(x.shape[0], 1.0, case["lam2"])


# ------------------------------------------------------------------ attention comparison
def attention_error(got: np.ndarray, ref: np.ndarray, dtype: int, label: str = "",
                    tol_abs: float | None = None, tol_rel: float | None = None):
    """Compare attention outputs (NaN in ref = not compared).  Reports the max-abs error, the
    max-rel error (max-abs / max|ref|) and a histogram of the error in units of the output
    type's ulp at the reference value (bf16: 8 significant bits; fp32: 24), then asserts the
    bounds: max-abs <= tol_abs (2e-2 bf16, 1e-4 fp32) and max-rel <= tol_rel (1 % bf16,
    1e-4 fp32)."""
    m = ~np.isnan(ref)
    g, r = got[m], ref[m]
    err = np.abs(g - r)
    mabs = float(err.max()) if err.size else 0.0
    mref = float(np.abs(r).max()) if r.size else 0.0
    mrel = mabs / mref if mref > 0 else mabs
    bits = 8 if dtype == BF16 else 24
    with np.errstate(divide="ignore"):
        e2 = np.floor(np.log2(np.maximum(np.abs(r), 2.0 ** -126)))
    ulp = 2.0 ** (e2 - (bits - 1))
    u = err / ulp
    edges = [0, 0.5, 1.0, 2.0, 4.0, 8.0, 16.0, np.inf]
    hist = np.histogram(u, bins=edges)[0]
    labels = ["<=0.5", "<=1", "<=2", "<=4", "<=8", "<=16", ">16"]
    print(f"[attn-err] {label} n={err.size} max-abs {mabs:.3e} max|ref| {mref:.3e} "
          f"max-rel {mrel:.3e} ulp-hist " + " ".join(f"{a}:{int(b)}" for a, b in zip(labels, hist)),
          flush=True)
    ta = tol_abs if tol_abs is not None else (2e-2 if dtype == BF16 else 1e-4)
    tr = tol_rel if tol_rel is not None else (1e-2 if dtype == BF16 else 1e-4)
    assert mabs <= ta, f"{label}: max-abs {mabs:.3e} > {ta}"
    assert mrel <= tr, f"{label}: max-rel {mrel:.3e} > {tr}"
    return mabs, mrel, hist

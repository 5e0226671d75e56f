"""Learned-scorer hook (Sec. 4.2, "Scorer design"; the first loop of Alg. 1) -- TEST
INFRASTRUCTURE ONLY (see oracle/__init__.py).

Sec. 4.2 scores an edge from five inputs (the two tokens it joins, its depth, the drafter's
log-probability of the child and the entropy of the child's position) and turns the scores
of one parent's children into probabilities with a softmax over those siblings.  No
trained weights are available, so the hook takes an MLP whose weights the caller supplies
(here: seeded random ones).  Reading (the same on the GPU):

* Features of an edge into row i (child depth i+1), in this order: the parent token's
  embedding (d values; the root's token is given per request; a token outside the
  vocabulary has a zero embedding), the child token's embedding (d values), the depth i+1, the child's
  log-probability (x_v - M) - LOG(Z) and the row's entropy H = LOG(Z) - S / Z.  M is the
  row maximum, Z the marginal normaliser of the marginal scorer (terms EXP(x_j - M) on a
  2^-42 grid, summed as integers), S the same exact sum of the terms t_j * (x_j - M)
  (terms with t_j = 0 count 0).  LOG is the shared fp64 logarithm of oracle.specexp.
* MLP: a_k = relu(((((b1[k] + P_k) + C_k) + W1[k][2d] * depth) + W1[k][2d+1] * logprob)
  + W1[k][2d+2] * entropy), with P_k = sum_j W1[k][j] * pe_j and C_k = sum_j W1[k][d+j] *
  ce_j (each summed from 0 in index order) over the parent and child embeddings; logit =
  b2 + sum_k w2[k] a_k in index order.  fp64, no fused multiply-add (weights are fp32,
  widened exactly); relu maps NaN to 0.  Grouping the embedding parts lets the GPU compute
  P once per parent and C once per child instead of once per edge.  A child that is not a candidate (fewer than K entries in
  its row) gets the logit -inf.
* Sibling softmax over the K candidates of the parent, as Eq. 1's stand-in does:
  e_r = EXP(l_r - max_r l_r), Z' = e_0 + e_1 + ... in rank order, q_cond = e_r / Z', or 0
  when Z' is 0 or not finite.  q_cond <= 1 keeps Alg. 1's one node per iteration.

Since the parent of a row-i child is the root (i = 0) or one of the K candidates of row
i - 1, q_cond is a table c[i][parent rank][child rank].
"""
from __future__ import annotations

import dataclasses
from fractions import Fraction

import numpy as np

from .specexp import spec_exp, spec_exp_array, spec_log

Z_GRID = 2.0 ** 42


@dataclasses.dataclass
class MLPScorer:
    emb: np.ndarray         # float32 [vocab][d]
    W1: np.ndarray          # float32 [h][2d + 3]
    b1: np.ndarray          # float32 [h]
    w2: np.ndarray          # float32 [h]
    b2: float               # float32 value
    root_token: np.ndarray  # int32 [batch]


def random_scorer(rng: np.random.Generator, vocab: int, d: int, h: int, batch: int) -> MLPScorer:
    """The seeded random weights of ``workloads.gen_scorer_weights`` as an MLPScorer."""
    from workloads import gen_scorer_weights
    return MLPScorer(**gen_scorer_weights(rng, vocab, d, h, batch))


def row_statistics(row: np.ndarray, M: float) -> tuple[float, float]:
    """(LOG(Z), H) of one row of logits with maximum M; (nan, nan) when Z is 0."""
    row = np.asarray(row, dtype=np.float64)
    with np.errstate(invalid="ignore"):
        dx = row - M
        t = spec_exp_array(dx)
        ts = np.where(t > 0.0, t * dx, 0.0)
    zi = int(np.rint(t * Z_GRID).astype(np.int64).sum(dtype=np.int64))
    si = int(np.rint(ts * Z_GRID).astype(np.int64).sum(dtype=np.int64))
    if zi <= 0:
        return float("nan"), float("nan")
    Z = float(Fraction(zi) / Fraction(int(Z_GRID)))
    S = float(Fraction(si) / Fraction(int(Z_GRID)))
    lz = spec_log(Z)
    return lz, lz - S / Z


def _emb(mlp: MLPScorer, tok: int, d: int) -> np.ndarray:
    if tok < 0 or tok >= mlp.emb.shape[0]:       # no token: a zero embedding
        return np.zeros(d, dtype=np.float64)
    return mlp.emb[tok].astype(np.float64)


def edge_logits(mlp: MLPScorer, parent_tok: int, child_tok: np.ndarray, depth: int,
                logprob: np.ndarray, entropy: float) -> np.ndarray:
    """Logits of the K candidate children of one parent (rank order)."""
    d = mlp.emb.shape[1]
    h = mlp.W1.shape[0]
    K = len(child_tok)
    pe = _emb(mlp, int(parent_tok), d)
    W = mlp.W1.astype(np.float64)
    P = []
    for k in range(h):
        acc = 0.0
        for j in range(d):
            acc = acc + float(W[k, j]) * float(pe[j])
        P.append(acc)
    out = np.full(K, -np.inf)
    for r in range(K):
        if child_tok[r] < 0:
            continue
        ce = _emb(mlp, int(child_tok[r]), d)
        logit = float(mlp.b2)
        for k in range(h):
            C = 0.0
            for j in range(d):
                C = C + float(W[k, d + j]) * float(ce[j])
            a = float(mlp.b1[k]) + P[k]
            a = a + C
            a = a + float(W[k, 2 * d]) * float(depth)
            a = a + float(W[k, 2 * d + 1]) * float(logprob[r])
            a = a + float(W[k, 2 * d + 2]) * float(entropy)
            a = a if a > 0.0 else 0.0
            logit = logit + float(mlp.w2[k]) * a
        out[r] = logit
    return out


def sibling_softmax(logits: np.ndarray) -> np.ndarray:
    K = len(logits)
    m = max((float(x) for x in logits if x == x), default=-np.inf)   # NaN logits ignored
    with np.errstate(invalid="ignore"):
        e = [spec_exp(float(x) - m) for x in logits]
    Z = 0.0
    for r in range(K):
        Z = Z + e[r]
    if not (Z > 0.0 and np.isfinite(Z)):
        return np.zeros(K)
    return np.array([e[r] / Z for r in range(K)])


def scorer_table(mlp: MLPScorer, b: int, rows: np.ndarray, idx: np.ndarray,
                 val: np.ndarray) -> np.ndarray:
    """q_cond table c[i][parent rank][child rank] of request b (logit marginals).  Row 0's
    parent is the root (parent rank 0; the other entries repeat it)."""
    D, K = idx.shape
    c = np.zeros((D, K, K), dtype=np.float64)
    for i in range(D):
        M = float(val[i, 0])
        lz, H = row_statistics(rows[i], M)
        child = np.array([int(idx[i, r]) for r in range(K)])
        logprob = np.array([(float(val[i, r]) - M) - lz for r in range(K)])
        parents = [int(mlp.root_token[b])] if i == 0 else \
            [int(idx[i - 1, pr]) for pr in range(K)]
        for pr, ptok in enumerate(parents):
            c[i, pr] = sibling_softmax(edge_logits(mlp, ptok, child, i + 1, logprob, H))
        if i == 0:
            c[0, 1:] = c[0, 0]
    return c

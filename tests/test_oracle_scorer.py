"""Pins for the learned-scorer hook of the oracle (Sec. 4.2): the shared logarithm against a
200-bit one, the row statistics against a high-precision softmax entropy, closed forms of
the MLP (zero weights, parent-only weights, the log-probability-only network that must
reproduce the sibling softmax), and the selection it drives against brute force and the
printed Alg. 1."""
import math
import random
from fractions import Fraction

import mpmath
import numpy as np
import pytest

from oracle.scorer import MLPScorer, random_scorer, row_statistics, scorer_table
from oracle.select import (LEARNED, LOGITS, brute_force_best_set, denominators, edge_factors,
                           select_literal_alg1, select_request)
from oracle.specexp import SQRT_HALF, spec_log


def test_log_constants_and_accuracy():
    mpmath.mp.prec = 200
    assert SQRT_HALF == float(mpmath.sqrt(mpmath.mpf(1) / 2))
    assert spec_log(1.0) == 0.0
    rnd = random.Random(4)
    xs = [math.exp(rnd.uniform(-700, 700)) for _ in range(3000)] + \
        [rnd.uniform(0.5, 2.0) for _ in range(3000)] + [2.0 ** k for k in range(-60, 61)] + \
        [5e-324, 1e-310, 1.7976931348623157e308, SQRT_HALF, math.nextafter(SQRT_HALF, 0)]
    for x in xs:
        exact = mpmath.log(mpmath.mpf(x))
        err = abs(mpmath.mpf(spec_log(x)) - exact)
        ulp = math.ulp(float(exact)) if float(exact) != 0.0 else 5e-324
        assert float(err) <= 3 * ulp, (x, spec_log(x), float(exact))


@pytest.mark.parametrize("seed", range(4))
def test_row_statistics_match_a_high_precision_softmax(seed):
    rng = np.random.default_rng(60 + seed)
    V = int(rng.choice([40, 3000, 151936]))
    row = (rng.standard_normal(V) * 3.0).astype(np.float32).astype(np.float64)
    M = float(row.max())
    lz, H = row_statistics(row, M)
    mpmath.mp.prec = 120
    t = [mpmath.e ** (mpmath.mpf(float(x)) - mpmath.mpf(M)) for x in row]
    Z = mpmath.fsum(t)
    S = mpmath.fsum(ti * (mpmath.mpf(float(x)) - mpmath.mpf(M)) for ti, x in zip(t, row))
    lz_x = mpmath.log(Z)
    H_x = lz_x - S / Z
    # the grid error of Z and S (V * 2^-43 each, Z >= 1) plus a few ulps
    bound = (3 + math.log(V)) * V * 2.0 ** -43 + 1e-14
    assert abs(lz - float(lz_x)) <= bound and abs(H - float(H_x)) <= bound


def _net(d, h, K_feat_weights, b1, w2, b2, vocab=50, batch=1):
    F = 2 * d + 3
    W1 = np.zeros((h, F), dtype=np.float32)
    for (k, j), w in K_feat_weights.items():
        W1[k, j] = w
    rng = np.random.default_rng(0)
    return MLPScorer(emb=rng.standard_normal((vocab, d)).astype(np.float32), W1=W1,
                     b1=np.array(b1, np.float32), w2=np.array(w2, np.float32), b2=float(b2),
                     root_token=np.zeros(batch, np.int32))


def _rows(seed, D, V):
    rng = np.random.default_rng(seed)
    return np.round(rng.standard_normal((D, V)) * 2, 3)


def _table(mlp, rows, K):
    from oracle.select import topk_row
    D = rows.shape[0]
    idx = np.zeros((D, K), np.int32)
    val = np.zeros((D, K))
    for i in range(D):
        idx[i], val[i] = topk_row(rows[i], K)
    return scorer_table(mlp, 0, rows, idx, val), val


def test_zero_weights_give_uniform_siblings():
    mlp = _net(4, 3, {}, [0, 0, 0], [0, 0, 0], 0.25)
    c, _ = _table(mlp, _rows(1, 5, 50), 4)
    assert np.all(c == 0.25)


def test_parent_only_weights_give_uniform_siblings():
    mlp = _net(4, 3, {(0, 0): 0.7, (1, 2): -1.5, (2, 3): 2.0}, [0.1, 0.2, 0.3], [1, -2, 0.5], 0)
    c, _ = _table(mlp, _rows(2, 5, 50), 4)
    assert np.all(c == 0.25)


def test_log_probability_network_reproduces_the_sibling_softmax():
    d = 4
    lp = 2 * d + 1                          # feature index of the child's log-probability
    mlp = _net(d, 1, {(0, lp): 1.0}, [1000.0], [1.0], 0.0, vocab=80)   # relu: identity here
    rows = _rows(3, 6, 80)
    c, val = _table(mlp, rows, 5)
    ref = edge_factors(val, LOGITS, 1.0)
    for pr in range(5):
        np.testing.assert_allclose(c[:, pr, :], ref, rtol=1e-12, atol=1e-300)


@pytest.mark.parametrize("seed", range(8))
def test_learned_selection_equals_brute_force_and_alg1(seed):
    rng = np.random.default_rng(800 + seed)
    K = int(rng.integers(1, 4))
    D = int(rng.integers(1, 4))
    V = int(rng.integers(K, 10))
    budget = int(rng.integers(1, 9))
    tau = float(rng.choice([0.0, 0.0, 0.02]))
    lam2 = float(rng.choice([0.0, 0.125]))
    rows = np.round(rng.standard_normal((D, V)) * 2, 2)
    mlp = random_scorer(rng, V, 3, 4, 1)
    tree = select_request(rows, K, budget, kind=LOGITS, lambda1=1.0, lambda2=lam2, tau=tau,
                          scorer=LEARNED, mlp=mlp, req=0)
    c = scorer_table(mlp, 0, rows, tree.topk_idx, tree.topk_val)
    den = denominators(D, 1.0, lam2)
    best_val, best_sets, nodes = brute_force_best_set(c, den, budget, tau)
    chosen = frozenset(tree.paths())
    got = sum((Fraction(nodes[p][1]) - Fraction(tau) for p in chosen if p), Fraction(0))
    assert got == best_val and chosen in best_sets
    S, added = select_literal_alg1(c, den, budget, tau)
    assert not added and frozenset(S) == chosen


def test_child_embedding_network_gives_the_hand_computed_softmax():
    """Only the child-embedding weights W1[:, d:2d] are non-zero, so each edge's logit is a
    function of its child's token alone (Sec. 4.2: the scorer sees the child token).  Hand
    example: d = h = 1, logit = relu(emb[child]) with embeddings 0, 3 ln2, ln2, 2 ln2 for the
    candidates of rank 0..3, so q_cond is (1, 8, 2, 4) / 15 in rank order, under every
    parent.  The weights are not monotone in rank, and a scorer reading any other token's
    embedding (the parent's, or the rank-0 candidate's) gives another table."""
    V, K, D = 30, 4, 3
    rng = np.random.default_rng(11)
    rows = np.round(rng.standard_normal((D, V)) - 5.0, 3)
    for i in range(D):                      # disjoint candidates: tokens 7i + 1, 7i + 2, ...
        rows[i, 7 * i + 1:7 * i + 1 + K] = [4.0, 3.5, 3.0, 2.5]
    from oracle.select import topk_row
    idx = np.array([topk_row(rows[i], K)[0] for i in range(D)])
    emb = np.zeros((V, 1), np.float32)
    ln2 = math.log(2.0)
    for i in range(D):
        for r, k in enumerate((0, 3, 1, 2)):
            emb[idx[i, r], 0] = np.float32(k * ln2)
    mlp = MLPScorer(emb=emb, W1=np.array([[0.0, 1.0, 0.0, 0.0, 0.0]], np.float32),
                    b1=np.zeros(1, np.float32), w2=np.ones(1, np.float32), b2=0.0,
                    root_token=np.array([idx[0, 0]], np.int32))
    c, _ = _table(mlp, rows, K)
    want = np.array([1.0, 8.0, 2.0, 4.0]) / 15.0
    for i in range(D):
        for pr in range(K):
            np.testing.assert_allclose(c[i, pr], want, rtol=2e-7)


@pytest.mark.parametrize("seed", range(3))
def test_child_embedding_network_matches_a_high_precision_softmax(seed):
    """Random child-embedding weights (two hidden units, biases, output weights); the
    expected table is written out in 100-bit arithmetic from the same fp32 weights."""
    d, h, V, K, D = 3, 2, 60, 5, 4
    rng = np.random.default_rng(70 + seed)
    W1 = np.zeros((h, 2 * d + 3), np.float32)
    W1[:, d:2 * d] = rng.standard_normal((h, d)).astype(np.float32)
    b1 = (rng.standard_normal(h) * 0.5).astype(np.float32)
    w2 = rng.standard_normal(h).astype(np.float32)
    emb = (rng.standard_normal((V, d)) * 2).astype(np.float32)
    mlp = MLPScorer(emb=emb, W1=W1, b1=b1, w2=w2, b2=0.375,
                    root_token=np.array([3], np.int32))
    rows = _rows(90 + seed, D, V)
    from oracle.select import topk_row
    idx = np.array([topk_row(rows[i], K)[0] for i in range(D)])
    c, _ = _table(mlp, rows, K)
    mpmath.mp.prec = 100
    mp = mpmath.mpf
    for i in range(D):
        logits = []
        for r in range(K):
            ce = [mp(float(x)) for x in emb[idx[i, r]]]
            acc = mp(0.375)
            for k in range(h):
                a = mp(float(b1[k])) + mpmath.fsum(mp(float(W1[k, d + j])) * ce[j]
                                                   for j in range(d))
                acc += mp(float(w2[k])) * (a if a > 0 else mp(0))
            logits.append(acc)
        m = max(logits)
        e = [mpmath.e ** (x - m) for x in logits]
        Z = mpmath.fsum(e)
        want = np.array([float(x / Z) for x in e])
        assert len(set(np.round(want, 6))) > 1          # the children are told apart
        for pr in range(K):
            np.testing.assert_allclose(c[i, pr], want, rtol=1e-13, atol=1e-300)

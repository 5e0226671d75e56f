"""Pins for the marginal-confidence scorer of the oracle (the scoring ablation of Sec. 5):
the elementwise exponential against the pinned scalar one, the normaliser's closed forms
and its error bound against a high-precision sum, and the selection it drives against
brute force over every prefix-closed subtree."""
import math
from fractions import Fraction

import mpmath
import numpy as np
import pytest

from oracle.select import (LOGITS, MARGINAL, PROBS, Z_GRID, brute_force_best_set,
                           denominators, marginal_factors, marginal_normaliser, select_request)
from oracle.specexp import spec_exp, spec_exp_array


def test_elementwise_exponential_equals_the_scalar_one_bitwise():
    rng = np.random.default_rng(3)
    t = np.concatenate([-rng.uniform(0, 1, 20000), -rng.uniform(0, 60, 20000),
                        -rng.uniform(0, 708, 2000),
                        [0.0, -0.0, -1e-300, -708.0, -708.5, -math.inf, math.nan]])
    a = spec_exp_array(t)
    b = np.array([spec_exp(float(x)) for x in t])
    assert np.array_equal(a.view(np.int64), b.view(np.int64))


@pytest.mark.parametrize("V", [1, 7, 1000, 151936])
def test_equal_logits_give_uniform_marginals(V):
    row = np.full(V, -3.25)
    assert marginal_normaliser(row, -3.25) == float(V)      # every term is exactly 1
    c = marginal_factors(row[None, :4] if V >= 4 else row[None, :V], row[None, :], LOGITS)
    assert np.all(c == 1.0 / V)


def test_single_finite_logit_gets_probability_one():
    row = np.full(500, -math.inf)
    row[17] = 2.0
    row[3] = math.nan                                        # NaN contributes nothing
    assert marginal_normaliser(row, 2.0) == 1.0
    c = marginal_factors(np.array([[2.0, -math.inf, -math.inf]]), row[None, :], LOGITS)
    assert list(c[0]) == [1.0, 0.0, 0.0]


def test_empty_row_gives_zero_factors():
    row = np.full(10, math.nan)
    c = marginal_factors(np.array([[math.nan, math.nan]]), row[None, :], LOGITS)
    assert np.all(c == 0.0)


@pytest.mark.parametrize("seed", range(6))
def test_normaliser_within_its_rounding_bound(seed):
    rng = np.random.default_rng(40 + seed)
    V = int(rng.choice([50, 4096, 151936]))
    row = (rng.standard_normal(V) * 3.0).astype(np.float32).astype(np.float64)
    M = float(row.max())
    Z = marginal_normaliser(row, M)
    mpmath.mp.prec = 120
    exact = mpmath.fsum(mpmath.e ** (mpmath.mpf(float(x)) - mpmath.mpf(M)) for x in row)
    # each term: EXP within 1 ulp, then rounded to a multiple of 2^-42; the sum >= 1
    bound = V * (2.0 ** -43 + 2.0 ** -52) + 2.0 ** -52 * float(exact)
    assert abs(Z - float(exact)) <= bound, (Z, float(exact), bound)
    # the integer sum is what is defined: recompute it term by term
    terms = [int(np.rint(spec_exp(float(x) - M) * Z_GRID)) for x in row[:200]]
    t2 = np.rint(spec_exp_array(row[:200] - M) * Z_GRID).astype(np.int64)
    assert terms == t2.tolist()


def test_marginal_factors_are_full_vocabulary_probabilities():
    rng = np.random.default_rng(9)
    row = np.round(rng.standard_normal(64) * 2, 2)
    order = np.argsort(-row, kind="stable")[:5]
    vals = row[order][None, :]
    c = marginal_factors(vals, row[None, :], LOGITS)
    mpmath.mp.prec = 80
    Zx = mpmath.fsum(mpmath.e ** mpmath.mpf(float(x)) for x in row)
    for r in range(5):
        p = float(mpmath.e ** mpmath.mpf(float(vals[0, r])) / Zx)
        assert abs(c[0, r] - p) <= 1e-10 * p
    assert c[0].sum() < 1.0                                  # no sibling renormalisation


def test_probs_marginal_is_the_probability_itself():
    vals = np.array([[0.5, 0.25, 0.0, -0.1], [0.125, 0.125, 0.0625, 0.0],
                     [math.inf, 3.0, 1.0, math.nan]])
    c = marginal_factors(vals, None, PROBS)
    assert c.tolist() == [[0.5, 0.25, 0.0, 0.0], [0.125, 0.125, 0.0625, 0.0],
                          [1.0, 1.0, 1.0, 0.0]]


@pytest.mark.parametrize("seed", range(10))
def test_marginal_selection_equals_brute_force(seed):
    rng = np.random.default_rng(700 + seed)
    K = int(rng.integers(1, 4))
    D = int(rng.integers(1, 4))
    V = int(rng.integers(K, 12))
    budget = int(rng.integers(1, 9))
    tau = float(rng.choice([0.0, 0.0, 0.02]))
    lam2 = float(rng.choice([0.0, 0.125]))
    kind = [LOGITS, PROBS][seed % 2]
    rows = rng.standard_normal((D, V))
    if kind == PROBS:
        rows = np.exp(rows) / np.exp(rows).sum(axis=1, keepdims=True)
    tree = select_request(rows, K, budget, kind=kind, lambda1=1.0, lambda2=lam2, tau=tau,
                          scorer=MARGINAL)
    c = marginal_factors(tree.topk_val, rows, kind)
    den = denominators(D, 1.0, lam2)
    best_val, best_sets, nodes = brute_force_best_set(c, den, budget, tau)
    chosen = frozenset(tree.paths())
    got = sum((Fraction(nodes[p][1]) - Fraction(tau) for p in chosen if p), Fraction(0))
    assert got == best_val and chosen in best_sets

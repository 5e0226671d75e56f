"""Pins for the selection oracle (top-K, Eq. 1-3, Alg. 1).

Each test fixes the oracle against something other than itself: a different
library route, hand-worked values, closed forms, the printed Alg. 1 run
literally, or brute force over every prefix-closed subtree."""
import itertools
import math
from fractions import Fraction

import mpmath
import numpy as np
import pytest

from oracle.select import (LOGITS, PROBS, topk_row, edge_factors, denominators,
                           select_request, select_literal_alg1, brute_force_best_set,
                           enumerate_trie)
from workloads import CONFIGS, gen_marginals, bf16_bits_to_f32


# ------------------------------------------------------------------ top-K
def test_topk_hand_worked_specials():
    x = np.array([1.0, np.nan, -np.inf, 0.0, -0.0, 1.0, 3.0, -np.inf, np.nan])
    idx, val = topk_row(x, 9)
    # 3 first; the two 1.0 by index; +0 and -0 tie (index order); -inf by index; NaN last
    assert idx.tolist() == [6, 0, 5, 3, 4, 2, 7, 1, 8]
    assert val[0] == 3.0 and val[1] == 1.0 and np.isnan(val[-1])


@pytest.mark.parametrize("seed", range(5))
def test_topk_against_argpartition(seed):
    rng = np.random.default_rng(seed)
    for V, K in [(1000, 4), (5000, 16), (151936, 8)]:
        x = rng.standard_normal(V)
        # a different route: partition, then order the survivors by (-value, index)
        part = np.argpartition(-x, K)[:K + 1]
        order = sorted(part.tolist(), key=lambda j: (-x[j], j))[:K]
        idx, val = topk_row(x, K)
        assert idx.tolist() == order
        assert np.array_equal(val, x[order])


@pytest.mark.parametrize("seed", range(5))
def test_topk_tie_heavy(seed):
    rng = np.random.default_rng(100 + seed)
    x = rng.integers(-3, 3, size=777).astype(np.float64)      # many equal values
    K = 16
    expect = sorted(range(len(x)), key=lambda j: (-x[j], j))[:K]
    assert topk_row(x, K)[0].tolist() == expect


# ------------------------------------------------------------------ Eq. 1
def test_qcond_probs_dyadic_hand_worked():
    vals = np.array([[4, 2, 1, 1]], dtype=np.float64) / 8.0
    c = edge_factors(vals, PROBS, 1.0)
    assert c.tolist() == [[0.5, 0.25, 0.125, 0.125]]


@pytest.mark.parametrize("K", [1, 2, 4, 8, 16])
def test_qcond_equal_values_power_of_two(K):
    vals = np.full((3, K), 2.5)
    c = edge_factors(vals, LOGITS, 1.0)
    assert np.all(c == 1.0 / K)


def test_qcond_matches_high_precision_softmax():
    mpmath.mp.prec = 120
    rng = np.random.default_rng(7)
    for _ in range(50):
        row = np.sort(bf16_bits_to_f32(rng.integers(0x3000, 0x4180, 8).astype(np.uint16))
                      .astype(np.float64))[::-1]
        c = edge_factors(row[None, :], LOGITS, 1.0)[0]
        es = [mpmath.exp(mpmath.mpf(float(v - row[0]))) for v in row]
        z = sum(es)
        for r in range(8):
            ref = float(es[r] / z)
            assert abs(c[r] - ref) <= 4 * math.ulp(ref), (r, c[r], ref)
        # the sum of the factors is one to a few ulps
        assert abs(sum(c) - 1.0) <= 8 * 2.0 ** -53


def test_qcond_pathological_rows():
    inf, nan = np.inf, np.nan
    vals = np.array([
        [-inf, -inf, -inf],      # nothing finite: every factor 0
        [nan, nan, nan],         # NaN logits: 0
        [inf, 1.0, 0.0],         # +inf max: inf - inf is NaN -> 0, the rest underflow: Z = 0
        [2.0, -inf, nan],        # one finite value: it takes everything
    ])
    c = edge_factors(vals, LOGITS, 1.0)
    assert c[:3].tolist() == [[0.0] * 3] * 3
    assert c[3].tolist() == [1.0, 0.0, 0.0]
    p = edge_factors(np.array([[inf, 0.5, 0.5], [0.0, 0.0, 0.0], [0.5, -1.0, nan]]), PROBS, 1.0)
    assert p[0].tolist() == [0.0] * 3 and p[1].tolist() == [0.0] * 3
    assert p[2].tolist() == [1.0, 0.0, 0.0]


def test_qcond_rank_monotone_on_config_rows():
    for name in ["tiny", "qwen3_4b"]:
        cfg = CONFIGS[name]
        m = gen_marginals(cfg)
        x = bf16_bits_to_f32(m).astype(np.float64) if cfg.dtype == 0 else m.astype(np.float64)
        vals = np.stack([topk_row(x[0, i], cfg.K)[1] for i in range(cfg.block)])
        c = edge_factors(vals, cfg.kind, cfg.beta)
        assert np.all(np.diff(c, axis=1) <= 0)
        assert np.all(c <= 1.0)


# ------------------------------------------------------------------ selection
def _check_invariants(tree, D, K, budget, tau):
    n = tree.n
    assert 1 <= n <= budget
    assert tree.parent[0] == -1 and tree.depth[0] == 0 and tree.q_reach[0] == 1.0
    seen = set()
    paths = tree.paths()
    for i in range(1, n):
        p = int(tree.parent[i])
        assert 0 <= p < i                                   # topological, prefix-closed
        assert tree.depth[i] == tree.depth[p] + 1 <= D
        assert 0 <= tree.rank[i] < K
        assert (p, int(tree.rank[i])) not in seen           # no node twice
        seen.add((p, int(tree.rank[i])))
        assert tree.token[i] == tree.topk_idx[tree.depth[i] - 1, tree.rank[i]]
        assert tree.q_reach[i] <= tree.q_reach[p]           # Eq. 2 never grows along a path
        assert tree.utility[i] <= tree.utility[p]
        assert tree.utility[i] > tau
        prev = (int(tree.depth[i - 1]), paths[i - 1])
        assert prev < (int(tree.depth[i]), paths[i])      # emitted breadth first
    assert np.all(tree.parent[n:] == -1) and np.all(tree.q_reach[n:] == 0.0)


def _random_probs(rng, D, K, V=None, integer_grid=False):
    V = V or K + 3
    if integer_grid:
        return rng.integers(1, 4, size=(D, V)).astype(np.float64)
    return rng.uniform(0.0, 1.0, size=(D, V))


@pytest.mark.parametrize("seed", range(12))
def test_selection_equals_brute_force(seed):
    rng = np.random.default_rng(1000 + seed)
    K = int(rng.integers(1, 4))
    D = int(rng.integers(1, 4))
    budget = int(rng.integers(1, 9))
    tau = float(rng.choice([0.0, 0.0, 0.05, 0.2]))
    lam2 = float(rng.choice([0.0, 0.125, 0.5]))
    kind = int(rng.integers(0, 2))
    marg = _random_probs(rng, D, K, integer_grid=bool(seed % 3 == 0))
    if kind == LOGITS:
        marg = np.log(marg)
    tree = select_request(marg, K, budget, kind=kind, lambda1=1.0, lambda2=lam2, tau=tau)
    _check_invariants(tree, D, K, budget, tau)
    c = edge_factors(tree.topk_val, kind, 1.0)
    den = denominators(D, 1.0, lam2)
    best_val, best_sets, nodes = brute_force_best_set(c, den, budget, tau)
    chosen = frozenset(tree.paths())
    got = sum((Fraction(nodes[p][1]) - Fraction(tau) for p in chosen if p), Fraction(0))
    assert got == best_val
    assert chosen in best_sets
    # and it is the first set of its size in the total order: the emitted nodes are the
    # (n-1) best non-root trie nodes above tau
    order = sorted((p for p in nodes if p),
                   key=lambda p: (-nodes[p][1], len(p), p))
    above = [p for p in order if nodes[p][1] > tau]
    assert sorted(tree.paths()[1:]) == sorted(above[:budget - 1])


@pytest.mark.parametrize("seed", range(8))
def test_selection_equals_literal_alg1(seed):
    rng = np.random.default_rng(2000 + seed)
    D, K, budget = [(8, 4, 16), (5, 3, 30), (4, 2, 16), (6, 4, 40)][seed % 4]
    marg = _random_probs(rng, D, K, integer_grid=seed % 2 == 1)
    tau = [0.0, 0.01][seed % 2]
    tree = select_request(np.log(marg), K, budget, kind=LOGITS, tau=tau)
    c = edge_factors(tree.topk_val, LOGITS, 1.0)
    den = denominators(D, 1.0, 0.125)
    S, added_ancestor = select_literal_alg1(c, den, budget, tau)
    assert not added_ancestor
    assert sorted(S) == sorted(tree.paths())
    # Alg. 1 adds nodes in non-increasing utility
    u = {p: enumerate_trie(c, den)[p][1] for p in S}
    assert all(u[a] >= u[b] for a, b in zip(S[1:], S[2:]))


def test_selection_tiny_config_literal_alg1():
    cfg = CONFIGS["tiny"]
    m = gen_marginals(cfg).astype(np.float64)[0]
    tree = select_request(m, cfg.K, cfg.budget, kind=cfg.kind)
    c = edge_factors(tree.topk_val, cfg.kind, 1.0)
    den = denominators(cfg.block, 1.0, 0.125)
    S, added = select_literal_alg1(c, den, cfg.budget, 0.0)    # 4-ary trie of depth 8: 87,381 nodes
    assert not added and sorted(S) == sorted(tree.paths())
    _check_invariants(tree, cfg.block, cfg.K, cfg.budget, 0.0)


@pytest.mark.parametrize("K,D,budget", [(2, 3, 6), (3, 3, 13), (4, 2, 21), (3, 4, 200)])
def test_uniform_marginals_give_breadth_first_lex(K, D, budget):
    marg = np.zeros((D, K + 2))
    marg[:, :K] = 1.0                       # K equal logits on top, the rest far below
    marg[:, K:] = -1000.0
    tree = select_request(marg, K, budget, kind=LOGITS)
    bfs = [()]
    for d in range(1, D + 1):
        bfs += list(itertools.product(range(K), repeat=d))
    assert tree.paths() == bfs[:budget]          # here the best-first order is breadth first too


@pytest.mark.parametrize("D,budget", [(5, 3), (5, 6), (5, 40)])
def test_single_candidate_gives_a_chain(D, budget):
    rng = np.random.default_rng(D * budget)
    tree = select_request(rng.standard_normal((D, 50)), 1, budget, kind=LOGITS)
    assert tree.n == min(budget, D + 1)
    assert tree.paths() == [tuple([0] * d) for d in range(tree.n)]


def test_budget_one_and_high_threshold_give_root_only():
    rng = np.random.default_rng(3)
    m = rng.standard_normal((6, 40))
    assert select_request(m, 4, 1).n == 1
    t = select_request(m, 4, 30)
    assert select_request(m, 4, 30, tau=float(t.utility[1:t.n].max())).n == 1


@pytest.mark.parametrize("seed", range(4))
def test_no_depth_penalty_gives_k_best_products(seed):
    rng = np.random.default_rng(3000 + seed)
    D, K, budget = 4, 3, 25
    marg = rng.uniform(0.05, 1.0, size=(D, 6))
    tree = select_request(marg, K, budget, kind=PROBS, lambda1=1.0, lambda2=0.0, tau=0.0)
    # all paths, scored by the exact rational product of the rank probabilities
    w = [sorted(row, reverse=True)[:K] for row in marg]
    w = [[Fraction(v) / sum(Fraction(x) for x in row) for v in row] for row in w]
    allp = [p for d in range(1, D + 1) for p in itertools.product(range(K), repeat=d)]
    exact = {p: math.prod((w[i][r] for i, r in enumerate(p)), start=Fraction(1)) for p in allp}
    chosen = set(tree.paths()[1:])
    worst_in = min(exact[p] for p in chosen)
    best_out = max(exact[p] for p in allp if p not in chosen)
    assert worst_in >= best_out            # a top-(N-1) set of products (up to fp64 rounding ties)
    assert len(chosen) == budget - 1


def test_invariants_on_config_trees():
    for name in ["tiny", "qwen3_4b"]:
        cfg = CONFIGS[name]
        m = gen_marginals(cfg)
        x = bf16_bits_to_f32(m).astype(np.float64) if cfg.dtype == 0 else m.astype(np.float64)
        t = select_request(x[0], cfg.K, cfg.budget, kind=cfg.kind)
        _check_invariants(t, cfg.block, cfg.K, cfg.budget, cfg.tau)
        assert t.n == cfg.budget                 # tau = 0 fills the budget


def test_hand_worked_depth_penalty_decides_between_branches():
    # PROBS rows: depth-1 weights 3/4, 1/4; depth-2 weights 0.6, 0.4; lambda1 = lambda2 = 1,
    # so den = (1, 2, 3) and u(0) = 3/8, u(1) = 1/8, u(0,0) = 0.45/3 = 0.15, u(0,1) = 0.1
    rows = np.array([[0.75, 0.25, 0.0], [0.6, 0.4, 0.0]])
    t = select_request(rows, 2, 3, kind=PROBS, lambda1=1.0, lambda2=1.0)
    assert t.paths() == [(), (0,), (0, 0)]       # (0,0) beats (1,): 0.15 > 0.125
    assert t.utility[1] == 0.375 and abs(t.utility[2] - 0.15) < 1e-16
    t = select_request(rows, 2, 4, kind=PROBS, lambda1=1.0, lambda2=1.0)
    assert t.paths() == [(), (0,), (1,), (0, 0)]  # breadth-first emission
    assert t.utility[2] == 0.125


def test_hand_worked_chain_utilities():
    # K = 1: q_reach is 1 along the chain and u(d) = 1/(lambda1 + lambda2*d)
    t = select_request(np.zeros((5, 3)), 1, 6, kind=LOGITS, lambda1=1.0, lambda2=0.5)
    assert t.q_reach[:6].tolist() == [1.0] * 6
    assert t.utility[:6].tolist() == [1.0, 1 / 1.5, 0.5, 1 / 2.5, 1 / 3.0, 1 / 3.5]


def test_hand_worked_equal_utility_prefers_shallow_node():
    # lambda2 = 0 and a certain second row make u(0,0) equal u(1) = 1/2:
    # the shallower node goes first on equal utility
    rows = np.array([[0.5, 0.5, 0.0], [1.0, 0.0, 0.0]])
    t = select_request(rows, 2, 3, kind=PROBS, lambda1=1.0, lambda2=0.0)
    assert t.paths() == [(), (0,), (1,)]
    t = select_request(rows, 2, 5, kind=PROBS, lambda1=1.0, lambda2=0.0)
    assert t.paths() == [(), (0,), (1,), (0, 0), (1, 0)]

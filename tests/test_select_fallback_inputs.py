"""The inputs of the selection-fallback GPU tests really take the fallback: a CPU count of
what the kernel's level-by-level expansion stores exceeds its LDS capacity, while the
benchmark configurations stay within it.  The oracle's trees for them are checked against
the closed forms they were built for."""
import os

import numpy as np
import pytest

from tests import _util as U

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_level_capacity_matches_the_kernel():
    src = open(os.path.join(ROOT, "paper_2606_00487_amd", "csrc", "select.hip")).read()
    assert f"constexpr int kCap = {U.LEVEL_CAP};" in src


@pytest.mark.parametrize("name", list(U.fallback_cases()))
def test_fallback_case_overflows_the_level_expansion(name):
    case = U.fallback_cases()[name]
    t, c, den = U.fallback_oracle(case)
    assert U.level_expansion_overflows(c, den, case["N"], 0.0)
    assert t.n == case["N"]


@pytest.mark.parametrize("name", ["tiny", "qwen3_4b", "qwen3_8b"])
def test_benchmark_configurations_stay_in_the_level_expansion(name):
    from workloads import gen_round
    inp = gen_round(name, with_attention=False)
    c0 = inp.cfg
    for t in U.oracle_trees(inp):
        from oracle.select import denominators, edge_factors
        c = edge_factors(t.topk_val, c0.kind, c0.beta)
        assert not U.level_expansion_overflows(c, denominators(c0.block, c0.lambda1, c0.lambda2),
                                               c0.budget, c0.tau)


def test_all_one_marginals_give_the_breadth_first_lexicographic_tree():
    t, _, _ = U.fallback_oracle(U.fallback_cases()["marginal_probs_all_one"])
    paths = t.paths()
    assert paths == sorted(paths, key=lambda p: (len(p), p))
    assert [len(p) for p in paths].count(1) == 16 and [len(p) for p in paths].count(2) == 239


def test_learned_chains_go_through_rank_three():
    t, _, _ = U.fallback_oracle(U.fallback_cases()["learned_child_chains"])
    deep = [p for p in t.paths() if len(p) >= 3]
    assert deep and all(r == 3 for p in deep for r in p[1:])
    assert max(len(p) for p in t.paths()) == 24

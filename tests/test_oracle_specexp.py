"""Pins for the shared fp64 exponential: against mpmath at high precision, against
libm, exact special values, and monotonicity across the reduction boundaries."""
import math

import mpmath
import numpy as np
import pytest

from oracle.specexp import spec_exp, INV_LN2, LN2_HI, LN2_LO, COEF

mpmath.mp.prec = 200


def ulp_distance(a: float, b: float) -> int:
    ia = np.array(a, dtype=np.float64).view(np.int64)
    ib = np.array(b, dtype=np.float64).view(np.int64)
    return abs(int(ia) - int(ib))


def test_constants_against_mpmath():
    ln2 = mpmath.log(2)
    assert INV_LN2 == float(1 / ln2)
    # LN2_HI carries at most 32 significant bits, so k*LN2_HI is exact for |k| < 2^21
    m, e = math.frexp(LN2_HI)
    assert (m * 2 ** 32) == int(m * 2 ** 32)
    assert abs(mpmath.mpf(LN2_HI) - ln2) < mpmath.mpf(2) ** -32
    # the split reproduces ln2 far beyond double precision
    assert abs(mpmath.mpf(LN2_HI) + mpmath.mpf(LN2_LO) - ln2) < mpmath.mpf(2) ** -85
    for n in range(14):
        assert COEF[n] == float(mpmath.mpf(1) / mpmath.factorial(n))


def test_specials():
    assert spec_exp(0.0) == 1.0
    assert spec_exp(-0.0) == 1.0
    assert spec_exp(float("nan")) == 0.0
    assert spec_exp(-math.inf) == 0.0
    assert spec_exp(-708.0000001) == 0.0
    assert spec_exp(-708.0) > 0.0
    # the result at the cut-off is still a normal double
    assert spec_exp(-708.0) >= 2.2250738585072014e-308


@pytest.mark.parametrize("seed", [0, 1])
def test_accuracy_against_mpmath(seed):
    rng = np.random.default_rng(seed)
    ts = np.concatenate([
        -rng.uniform(0, 1, 3000), -rng.uniform(0, 40, 3000), -rng.uniform(0, 708, 2000),
        -np.exp(rng.uniform(-40, 0, 1000)),
    ])
    worst = 0
    for t in ts:
        ref = float(mpmath.exp(mpmath.mpf(float(t))))
        d = ulp_distance(spec_exp(float(t)), ref)
        worst = max(worst, d)
        assert d <= 1, (t, spec_exp(float(t)), ref)
    # agrees with the platform libm to one ulp as well
    for t in ts[:2000]:
        assert ulp_distance(spec_exp(float(t)), math.exp(float(t))) <= 1
    assert worst <= 1


def test_never_above_one_and_monotone_near_reduction_boundaries():
    ln2 = math.log(2)
    for k in range(0, 1022, 7):
        centre = -(k + 0.5) * ln2
        grid = np.nextafter(centre, -np.inf) + np.arange(-300, 300) * abs(centre) * 2.0 ** -52
        grid = grid[(grid <= 0) & (grid >= -708)]
        vals = [spec_exp(float(t)) for t in grid]
        assert all(v <= 1.0 for v in vals)
        assert all(a <= b for a, b in zip(vals, vals[1:])), k


def test_monotone_on_all_bf16_gaps_near_zero():
    # every t the selector meets on bf16 logits is a difference of two bf16 values;
    # sweep all differences x_r - x_0 for a dense set of x_0 and every smaller bf16 x_r
    from workloads import bf16_bits_to_f32
    bits = np.arange(0, 0x7F80, dtype=np.uint16)           # non-negative finite bf16
    pos = bf16_bits_to_f32(bits).astype(np.float64)
    allv = np.unique(np.concatenate([pos, -pos]))
    allv = allv[(allv > -64) & (allv < 64)]
    for x0 in [0.0, 1.0, 3.140625, 12.9375, 13.5]:
        ts = np.sort(allv[allv <= x0] - x0)
        ts = ts[ts >= -708]
        vals = np.array([spec_exp(float(t)) for t in ts])
        assert np.all(np.diff(vals) >= 0), x0

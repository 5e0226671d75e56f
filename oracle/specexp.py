"""The fp64 exponential used for the sibling softmax of Eq. 1.

The paper fixes no numeric form for the softmax.  Trees are compared bit for
bit, and bf16 logits make mathematically equal path products common, so both
sides must produce identical bits for every factor; neither may use its
platform's libm.  Both implement this one published method:

  Cody & Waite (1980) argument reduction  t = k*ln2 + r,  |r| <= ln2/2,
  with ln2 split into LN2_HI (ln2 rounded to 32 significant bits, so k*LN2_HI
  is exact for |k| < 2^21) and LN2_LO = fl(ln2 - LN2_HI);
  k = rint(fl(t * INV_LN2)) (round half to even);
  r = fl(fl(t - k*LN2_HI) - fl(k*LN2_LO));
  p = degree-13 Taylor polynomial of exp(r) by Horner, coefficients fl(1/n!),
      each step fl(fl(p*r) + c) with no fused multiply-add;
  result = ldexp(p, k).

Specials (defined for the inputs the method produces, t <= 0):
  t is NaN -> 0.0;  t < -708 -> 0.0;  t == 0 -> 1.0 exactly.

The truncation error |r|^14/14! < 5e-18 is far below one ulp.
Constants are derived here from ln 2 computed with exact rationals.
"""
from __future__ import annotations

import math
from fractions import Fraction


def _ln2_fraction(terms: int = 80) -> Fraction:
    # ln 2 = 2*atanh(1/3) = 2 * sum_{k>=0} 1 / ((2k+1) 3^(2k+1)); 80 terms give ~150 digits.
    s = Fraction(0)
    for k in range(terms):
        s += Fraction(1, (2 * k + 1) * 3 ** (2 * k + 1))
    return 2 * s


_LN2 = _ln2_fraction()
INV_LN2 = float(1 / _LN2)                                  # nearest double to 1/ln2
LN2_HI = float(Fraction(round(_LN2 * 2 ** 32), 2 ** 32))  # 32 significant bits (ln2 in [1/2, 1))
LN2_LO = float(_LN2 - Fraction(LN2_HI))                    # nearest double to the remainder
COEF = [float(Fraction(1, math.factorial(n))) for n in range(14)]  # fl(1/n!), n = 0..13

T_MIN = -708.0


def spec_exp(t: float) -> float:
    """exp(t) for t <= 0 under the shared fp64 contract described above."""
    t = float(t)
    if math.isnan(t) or t < T_MIN:
        return 0.0
    if t == 0.0:
        return 1.0
    k = round(t * INV_LN2)           # Python round(): half to even, exact on doubles
    kf = float(k)
    r = (t - kf * LN2_HI) - kf * LN2_LO
    p = COEF[13]
    for n in range(12, -1, -1):
        p = p * r + COEF[n]          # two roundings: Python never fuses
    return math.ldexp(p, k)


def spec_exp_array(t) -> "np.ndarray":
    """spec_exp applied elementwise to an array: the same operations in the same order
    (NumPy rounds every operation on its own and never fuses), so every element equals
    spec_exp of it bit for bit."""
    import numpy as np
    t = np.asarray(t, dtype=np.float64)
    out = np.zeros(t.shape, dtype=np.float64)
    ok = ~(np.isnan(t) | (t < T_MIN))
    tt = t[ok]
    k = np.rint(tt * INV_LN2)             # half to even, like Python round()
    r = (tt - k * LN2_HI) - k * LN2_LO
    p = np.full(tt.shape, COEF[13])
    for n in range(12, -1, -1):
        p = p * r + COEF[n]
    res = np.ldexp(p, k.astype(np.int64))
    res[tt == 0.0] = 1.0
    out[ok] = res
    return out


# ---------------------------------------------------------------- the shared fp64 logarithm
# log x for finite x > 0, used by the learned scorer's log-probability and entropy
# features: x = m * 2^e with m in [sqrt(1/2), sqrt(2)) (frexp, then one exact doubling),
# s = (m - 1) / (m + 1), log m = 2 * atanh(s) = 2 * s * (1 + s^2/3 + ... + s^26/27) by
# Horner in s^2 with coefficients fl(1/(2k+1)), k = 13 .. 0 (the next term, s^29/29, is
# below 1e-24), result = e * LN2_HI + (e * LN2_LO + log m).  No fused multiply-add.
SQRT_HALF = float.fromhex("0x1.6a09e667f3bcdp-1")   # nearest double to sqrt(1/2)
LOG_COEF = [float(Fraction(1, 2 * k + 1)) for k in range(14)]


def spec_log(x: float) -> float:
    """log(x) for finite x > 0 under the shared fp64 contract described above."""
    m, e = math.frexp(float(x))
    if m < SQRT_HALF:
        m *= 2.0
        e -= 1
    s = (m - 1.0) / (m + 1.0)
    z = s * s
    p = LOG_COEF[13]
    for k in range(12, -1, -1):
        p = p * z + LOG_COEF[k]
    logm = 2.0 * (s * p)
    ef = float(e)
    return ef * LN2_HI + (ef * LN2_LO + logm)

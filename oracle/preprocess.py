"""Oracle of the preprocessor's initial format -- TEST INFRASTRUCTURE ONLY.

Sec. "Initial Design Generation" (Eq. 6-9): for a data structure X and a
target word length k,
  S = 1 when the smallest value of X is negative (Eq. 6; -0.0 is not);
  psi = X_max+ / (2^k - 1)                                  when S = 0,
  psi = min(X_max- / -2^(k-1), X_max+ / (2^(k-1) - 1))      when S = 1 (Eq. 7);
  beta_hat = -log2(psi) (Eq. 8);
  beta = floor / nearest / ceil of beta_hat for the conservative / neutral /
  aggressive rounding strategy (Eq. 9), and alpha = k - beta (the integer
  length; Eq. 9 prints k - beta - S, read as a typo since k = alpha + beta
  everywhere else).

Readings where the text leaves a case open:
  * psi <= 0 has no logarithm: an all-zero tensor gets beta = fl_hi; a signed
    tensor with no positive value (X_max+ <= 0) takes the negative side's
    ratio alone.
  * "max" instead of "min" in Eq. 7 is offered as an alternative rule
    (psi_rule = 1): the printed min saturates the side with the larger ratio.
  * beta is clamped to the search range [fl_lo, fl_hi] of the other calls.
  * nearest: beta_hat is never a half-integer (psi > 0 is rational and
    2^(m + 1/2) is not), so no tie rule is needed.

Everything is decided in exact rational arithmetic (fractions): with psi
rational, floor(beta_hat) is the largest b with psi * 2^b <= 1, ceil the
smallest b with psi * 2^b >= 1, nearest the largest b with
(psi * 2^b)^2 <= 2.
"""
from fractions import Fraction

import numpy as np

CONSERVATIVE, NEUTRAL, AGGRESSIVE = 0, 1, 2
PSI_PRINTED, PSI_MAX = 0, 1


def _psi(xmin, xmax, k, rule):
    """(S, psi) of Eq. 6-7 for exact extremes xmin <= xmax (Fractions);
    psi None for an all-zero tensor."""
    sign = 1 if xmin < 0 else 0
    if sign == 0:
        if xmax == 0:
            return sign, None
        return sign, xmax / (2 ** k - 1)
    neg = xmin / -(2 ** (k - 1))          # > 0
    pos = xmax / (2 ** (k - 1) - 1)       # <= 0 when no positive value
    if pos <= 0:
        return sign, neg
    return sign, (min(neg, pos) if rule == PSI_PRINTED else max(neg, pos))


def beta_hat(xmin, xmax, k, rule=PSI_PRINTED):
    """beta_hat of Eq. 8 as a float (for reports); None for all zeros."""
    import math
    _, psi = _psi(Fraction(xmin), Fraction(xmax), k, rule)
    return None if psi is None else -math.log2(psi)


def init_fl(xmin, xmax, k, strategy, rule=PSI_PRINTED, fl_lo=-8, fl_hi=15):
    """(fl, S) of Eq. 9 for exact extremes, clamped to [fl_lo, fl_hi]."""
    if k < 2:
        raise ValueError("word lengths from 2 bits")
    xmin, xmax = Fraction(xmin), Fraction(xmax)
    sign, psi = _psi(xmin, xmax, k, rule)
    if psi is None:
        return fl_hi, sign
    # bracket beta_hat: 2^b0 <= 1/psi < 2^(b0+1)
    b = 0
    while psi * Fraction(2) ** b > 1:
        b -= 1
    while psi * Fraction(2) ** (b + 1) <= 1:
        b += 1
    floor_b = b                                     # psi * 2^b <= 1 < psi * 2^(b+1)
    ceil_b = b if psi * Fraction(2) ** b == 1 else b + 1
    near_b = b + 1 if (psi * Fraction(2) ** (b + 1)) ** 2 <= 2 else b
    beta = {CONSERVATIVE: floor_b, NEUTRAL: near_b, AGGRESSIVE: ceil_b}[strategy]
    return min(max(beta, fl_lo), fl_hi), sign


def exact_extremes_f32(x):
    """Exact min and max of fp32 data (as Fractions; -0.0 counts as 0)."""
    x = np.asarray(x, np.float32)
    return Fraction(float(x.min())), Fraction(float(x.max()))


def exact_extremes_int(v, s):
    """Exact min and max of the values v * 2^-s (integers v)."""
    v = np.asarray(v, np.int64)
    return Fraction(int(v.min())) / Fraction(2) ** s, Fraction(int(v.max())) / Fraction(2) ** s

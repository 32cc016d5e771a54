"""The oracle of the preprocessor's initial format (Eq. 6-9), pinned to
hand-worked examples (tests/golden/preprocess_init.txt) and to properties
that hold for any data: floor <= nearest <= ceil with at most one step
between floor and ceil, floor == ceil exactly when psi is a power of two, the
conservative format never saturates the largest value of unsigned data, and
agreement with a floating-point log2 wherever beta_hat is not within 1e-9 of
a rounding boundary."""
import math
from fractions import Fraction as F

import numpy as np
import pytest

import synth
from conftest import read_golden
from oracle import preprocess as P

RULES = {"min": P.PSI_PRINTED, "max": P.PSI_MAX}


def test_hand_worked_examples():
    rows = [r for r in read_golden("preprocess_init.txt") if r[0] == "init"]
    assert len(rows) >= 10
    for _, xmin, xmax, k, rule, c, n, a, s in rows:
        for strat, want in ((P.CONSERVATIVE, c), (P.NEUTRAL, n), (P.AGGRESSIVE, a)):
            got = P.init_fl(F(xmin), F(xmax), int(k), strat, RULES[rule])
            assert got == (int(want), int(s)), (xmin, xmax, k, rule, strat)


def _psi_float(xmin, xmax, k, rule):
    if xmin >= 0:
        return xmax / (2 ** k - 1)
    neg = xmin / -(2 ** (k - 1))
    pos = xmax / (2 ** (k - 1) - 1)
    if pos <= 0:
        return neg
    return min(neg, pos) if rule == P.PSI_PRINTED else max(neg, pos)


def _draws(n):
    g = synth.rng_for(5, "preprocess-props")
    for _ in range(n):
        kind = int(g.integers(0, 3))
        scale = 2.0 ** float(g.uniform(-12, 10))
        a, b = sorted(g.standard_normal(2) * scale)
        if kind == 1:
            a = abs(a) * 0.0  # unsigned data
            b = abs(b)
        elif kind == 2:
            a, b = -abs(a) - scale, -abs(b) * 0.5  # no positive value
            a, b = min(a, b), max(a, b)
        yield F(float(np.float32(a))), F(float(np.float32(b))), int(g.integers(2, 17))


def test_properties_and_float_log2():
    checked = 0
    for xmin, xmax, k in _draws(3000):
        for rule in (P.PSI_PRINTED, P.PSI_MAX):
            lo, hi = -64, 64
            fl_c, s = P.init_fl(xmin, xmax, k, P.CONSERVATIVE, rule, lo, hi)
            fl_n, _ = P.init_fl(xmin, xmax, k, P.NEUTRAL, rule, lo, hi)
            fl_a, _ = P.init_fl(xmin, xmax, k, P.AGGRESSIVE, rule, lo, hi)
            assert s == (1 if xmin < 0 else 0)
            assert fl_c <= fl_n <= fl_a <= fl_c + 1
            if xmax == 0 and xmin == 0:
                continue
            psi = P._psi(xmin, xmax, k, rule)[1]
            pow2 = psi.numerator & (psi.numerator - 1) == 0 and psi.denominator & (psi.denominator - 1) == 0
            assert (fl_c == fl_a) == pow2
            if s == 0 and lo < fl_c < hi:
                # conservative: the largest value fits, one step finer it does not
                assert xmax * F(2) ** fl_c <= 2 ** k - 1 < xmax * F(2) ** (fl_c + 1)
            bh = -math.log2(_psi_float(float(xmin), float(xmax), k, rule))
            frac = bh - math.floor(bh)
            if 1e-9 < frac < 1 - 1e-9 and abs(frac - 0.5) > 1e-9:
                assert (fl_c, fl_n, fl_a) == (math.floor(bh), math.floor(bh + 0.5), math.ceil(bh))
                checked += 1
    assert checked > 5000


def test_conservative_never_saturates_unsigned_data(orc):
    # for unsigned data the conservative format lies at or below beta_nosat,
    # the largest fl at which no value saturates (the FL search's window start)
    g = synth.rng_for(6, "preprocess-nosat")
    for _ in range(200):
        x = np.abs(g.standard_normal(257) * 2.0 ** g.uniform(-8, 6)).astype(np.float32)
        for k in (3, 4, 6, 8):
            xmin, xmax = P.exact_extremes_f32(x)
            fl, s = P.init_fl(xmin, xmax, k, P.CONSERVATIVE, P.PSI_PRINTED)
            assert s == 0
            if fl >= 15:
                continue  # clamped at the top of the range
            # no value is clipped: every error is at most half a step (exact in fp64)
            codes = orc.quantize_f32(x, k, fl, 0).astype(np.float64)
            err = np.abs(x.astype(np.float64) - codes * 2.0 ** -fl)
            assert np.all(err <= 2.0 ** (-fl - 1))


def test_word_length_one_is_not_a_k_bit_format():
    with pytest.raises(ValueError):
        P.init_fl(0, 1, 1, P.CONSERVATIVE)

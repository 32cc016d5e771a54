"""Pins of the CPU oracle against what the paper and plain mathematics fix.

Nothing here runs on a GPU.  Every check compares the oracle with something
other than itself: values printed in the paper (tests/golden), textbook
definitions evaluated in exact rational arithmetic (fractions.Fraction),
library routines (numpy int64 matmul, torch float64 convolution and pooling),
brute force on tiny inputs, and invariants that follow from the definitions.
"""
import itertools
import random
from fractions import Fraction as Fr

import numpy as np
import pytest

from conftest import read_golden

FL_LO, FL_HI = -8, 15


# ----------------------------------------------------------------------------
# Independent reference pieces (exact rationals, written from the textbook
# meaning of "nearest representable value, ties to the even code").
# ----------------------------------------------------------------------------
def levels(k, sign):
    """Two's complement / unsigned k-bit integer ranges (textbook)."""
    if sign:
        return -(2 ** (k - 1)), 2 ** (k - 1) - 1
    return 0, 2 ** k - 1


def nearest_code(x, k, fl, sign):
    """Code c in range minimizing |x - c 2^-fl|, ties to the even code.

    For the k = 1 signed case the paper's binary rule applies instead.
    """
    x = Fr(x)
    if k == 1 and sign == 1:
        return (-1 if x < 0 else 0), (-1 if x < 0 else 1)
    lo, hi = levels(k, sign)
    step = Fr(2) ** -fl
    t = x / step
    # candidates: floor/ceil clipped into range
    import math
    f = math.floor(t)
    cands = {min(max(f, lo), hi), min(max(f + 1, lo), hi)}
    best = None
    for c in sorted(cands):
        d = abs(x - c * step)
        if best is None or d < best[0] or (d == best[0] and c % 2 == 0):
            best = (d, c)
    return best[1], best[1]


def exact_sse(xs, k, fl, sign):
    s = Fr(0)
    for x in xs:
        _, dec = nearest_code(x, k, fl, sign)
        s += (Fr(x) - dec * Fr(2) ** -fl) ** 2
    return s


def exact_argmin(xs, k, sign, lo=FL_LO, hi=FL_HI):
    vals = {fl: exact_sse(xs, k, fl, sign) for fl in range(lo, hi + 1)}
    m = min(vals.values())
    return max(fl for fl, v in vals.items() if v == m), vals


# ----------------------------------------------------------------------------
# Format (Eq. 12) against the paper's printed examples.
# ----------------------------------------------------------------------------
def test_qrange_closed_form(orc):
    for k in range(1, 33):
        for s in (0, 1):
            assert orc.qrange(k, s) == levels(k, s)


def test_printed_value_sets(orc):
    rows = [r for r in read_golden("dfx_formats.txt") if r[0] == "values"]
    assert len(rows) == 2
    for _, fmt, alpha, beta, res, *vals in rows:
        alpha, beta = int(alpha), int(beta)
        sign = 1 if fmt == "S" else 0
        k = alpha + beta
        lo, hi = orc.qrange(k, sign)
        got = [Fr(c) * Fr(2) ** -beta for c in range(lo, hi + 1)]
        assert got == [Fr(v) for v in vals]
        assert Fr(2) ** -beta == Fr(res)


def test_printed_six_bit_range(orc):
    rows = [r for r in read_golden("dfx_formats.txt") if r[0] == "range"]
    for _, fmt, k, lo, hi in rows:
        assert orc.qrange(int(k), 1 if fmt == "S" else 0) == (int(lo), int(hi))


def test_printed_formats_dynamic_range(orc):
    """Dynamic range [-2^(a-1), 2^(a-1) - 2^-b] of S(a, b) equals the code range
    of Eq. 12 times 2^-b with k = a + b (the paper's k = alpha + beta)."""
    rows = [r for r in read_golden("dfx_formats.txt") if r[0] == "format"]
    assert len(rows) == 6
    for _, fmt, alpha, beta, k in rows:
        alpha, beta, k = int(alpha), int(beta), int(k)
        assert alpha + beta == k
        lo, hi = orc.qrange(k, 1)
        step = Fr(2) ** -beta
        assert lo * step == -Fr(2) ** (alpha - 1)
        assert hi * step == Fr(2) ** (alpha - 1) - step


def test_printed_unsigned_dynamic_range(orc):
    # U(alpha, beta): [0, 2^alpha - 2^-beta]
    for alpha, beta in [(3, -1), (0, 8), (5, 3), (-2, 10)]:
        k = alpha + beta
        lo, hi = orc.qrange(k, 0)
        step = Fr(2) ** -beta
        assert lo == 0 and hi * step == Fr(2) ** alpha - step


# ----------------------------------------------------------------------------
# Quantizer (Eq. 10-13).
# ----------------------------------------------------------------------------
def test_hand_worked_quantization(orc):
    rows = [r for r in read_golden("dfx_formats.txt") if r[0] == "quant"]
    assert len(rows) >= 10
    for _, fmt, alpha, beta, x, code, value in rows:
        alpha, beta = int(alpha), int(beta)
        sign = 1 if fmt == "S" else 0
        q = orc.quantize_f32(np.array([float(x)], np.float32), alpha + beta, beta, sign)
        assert int(q[0]) == int(code), (fmt, alpha, beta, x)
        assert Fr(int(q[0])) * Fr(2) ** -beta == Fr(value)


def test_quantize_is_nearest_with_even_ties(orc):
    rng = random.Random(1)
    for _ in range(400):
        k = rng.randint(1, 10)
        sign = rng.randint(0, 1)
        fl = rng.randint(-8, 15)
        # mix of exact ties, tiny, huge and ordinary values
        kind = rng.random()
        if kind < 0.3:
            x = (rng.randint(-3000, 3000) + 0.5) * 2.0 ** -fl
        elif kind < 0.5:
            x = rng.choice([0.0, -0.0, 1e-30, -1e-30, 3e30, -3e30])
        else:
            x = rng.gauss(0, 1) * 2.0 ** rng.randint(-10, 10)
        x = float(np.float32(x))
        q = int(orc.quantize_f32(np.array([x], np.float32), k, fl, sign)[0])
        want, _ = nearest_code(x, k, fl, sign)
        assert q == want, (x, k, fl, sign)


def test_binary_quantizer(orc):
    x = np.array([-2.0, -1e-20, -0.0, 0.0, 1e-20, 3.0], np.float32)
    q = orc.quantize_f32(x, 1, 4, 1)
    assert list(q) == [-1, -1, 0, 0, 0, 0]


def test_quantize_idempotent_and_bounded(orc):
    rng = np.random.default_rng(2)
    x = (rng.standard_normal(5000) * 3).astype(np.float32)
    for k, fl, s in [(8, 4, 1), (6, 2, 1), (4, 0, 1), (8, 5, 0), (3, -2, 1), (16, 12, 1)]:
        q = orc.quantize_f32(x, k, fl, s)
        lo, hi = levels(k, s)
        assert q.min() >= lo and q.max() <= hi
        back = (q.astype(np.float64) * 2.0 ** -fl).astype(np.float32)
        assert np.array_equal(orc.quantize_f32(back, k, fl, s), q)
        # codes differ from x * 2^fl by at most 1/2 where they are not clipped
        t = x.astype(np.float64) * 2.0 ** fl
        inside = (t > lo - 0.5) & (t < hi + 0.5)
        assert np.all(np.abs(t[inside] - q[inside]) <= 0.5)


def test_integer_quantize_matches_rationals(orc):
    rng = random.Random(3)
    for _ in range(300):
        s = rng.randint(-5, 40)
        v = rng.randint(-2 ** 40, 2 ** 40) >> rng.randint(0, 38)
        k = rng.randint(2, 16)
        sign = rng.randint(0, 1)
        fl = rng.randint(-8, 15)
        q = int(orc.quantize_i64(np.array([v]), s, k, fl, sign)[0])
        want, _ = nearest_code(Fr(v) * Fr(2) ** -s, k, fl, sign)
        assert q == want


def test_requant_rne_ties_hand_worked(orc):
    # v = 0b1010 at shift 2 is 2.5 -> 2; v = 0b1110 at shift 2 is 3.5 -> 4.
    q = orc.quantize_i64(np.array([0b1010, 0b1110, -0b1010, -0b1110]), 2, 8, 0, 1)
    assert list(q) == [2, 4, -2, -4]


# ----------------------------------------------------------------------------
# Eq. 14 and the FL search.
# ----------------------------------------------------------------------------
def test_sse_exact_vs_rationals(orc):
    rng = np.random.default_rng(4)
    for trial in range(30):
        n = int(rng.integers(1, 12))
        x = (rng.standard_normal(n) * 2.0 ** rng.integers(-6, 6)).astype(np.float32)
        k = int(rng.integers(1, 9))
        sign = int(rng.integers(0, 2))
        fl = int(rng.integers(-8, 16))
        got = orc.sse_f32(x, k, fl, sign)
        want = exact_sse([float(v) for v in x], k, fl, sign)
        assert got == pytest.approx(float(want), rel=1e-15, abs=0.0)


def test_sse_zero_on_representable(orc):
    rng = np.random.default_rng(5)
    for k, fl, s in [(8, 3, 1), (5, -2, 1), (8, 7, 0)]:
        lo, hi = levels(k, s)
        codes = rng.integers(lo, hi + 1, 1000)
        x = (codes * 2.0 ** -fl).astype(np.float32)
        assert orc.sse_f32(x, k, fl, s) == 0.0


def test_sse_close_to_float64_sum(orc):
    rng = np.random.default_rng(6)
    x = rng.standard_normal(20000).astype(np.float32)
    for fl in (-2, 3, 7):
        q = orc.quantize_f32(x, 8, fl, 1)
        err = x.astype(np.float64) - q * 2.0 ** -fl
        assert orc.sse_f32(x, 8, fl, 1) == pytest.approx(float(np.sum(err * err)), rel=1e-12)


def test_fl_search_brute_force(orc):
    rng = np.random.default_rng(7)
    for trial in range(12):
        n = int(rng.integers(1, 9))
        x = (rng.standard_normal(n) * 2.0 ** rng.integers(-4, 4)).astype(np.float32)
        k = int(rng.integers(2, 9))
        fl, sign, sse = orc.fl_search_f32(x, k)
        want_sign = 1 if np.any(x < 0) else 0
        assert sign == want_sign
        want_fl, vals = exact_argmin([float(v) for v in x], k, sign)
        assert fl == want_fl
        for j, f in enumerate(range(FL_LO, FL_HI + 1)):
            assert sse[j] == pytest.approx(float(vals[f]), rel=1e-15, abs=0.0)


def test_fl_search_ties_go_to_largest_fl(orc):
    # all-zero tensor: every candidate has zero error
    fl, sign, sse = orc.fl_search_f32(np.zeros(64, np.float32), 8)
    assert fl == FL_HI and sign == 0 and np.all(sse == 0)
    # values exactly representable from fl = 2 upward with 8 bits: tie on [2, 5]
    x = np.array([0.25, -0.5, 1.0, 1.75], np.float32)
    fl, sign, sse = orc.fl_search_f32(x, 8)
    zero = [f for f, v in zip(range(FL_LO, FL_HI + 1), sse) if v == 0.0]
    assert zero == [2, 3, 4, 5, 6] and fl == 6


def test_fl_search_integer_brute_force(orc):
    rng = random.Random(8)
    for _ in range(10):
        n = rng.randint(1, 8)
        s = rng.randint(0, 20)
        v = [rng.randint(-2 ** 20, 2 ** 20) for _ in range(n)]
        k = rng.randint(2, 8)
        fl, sign, sse = orc.fl_search_i64(np.array(v), s, k)
        xs = [Fr(a) * Fr(2) ** -s for a in v]
        want_fl, vals = exact_argmin(xs, k, sign)
        assert sign == (1 if min(v) < 0 else 0)
        assert fl == want_fl


def beta_nosat(x, k, sign):
    lo, hi = levels(k, sign)
    best = None
    for fl in range(FL_LO, FL_HI + 1):
        t = [Fr(float(v)) * Fr(2) ** fl for v in x]
        if all(lo - Fr(1, 2) <= a <= hi + Fr(1, 2) for a in t):
            best = fl
    return best


def test_sse_non_increasing_up_to_no_saturation(orc):
    rng = np.random.default_rng(9)
    for trial in range(6):
        x = (rng.standard_normal(3000) * 2.0 ** rng.integers(-3, 3)).astype(np.float32)
        for k in (4, 6, 8):
            fl, sign, sse = orc.fl_search_f32(x, k)
            bn = beta_nosat(x, k, sign)
            assert bn is not None
            seg = sse[: bn - FL_LO + 1]
            assert np.all(np.diff(seg) <= 0)
            assert fl >= bn


def test_optimal_error_non_increasing_in_wordlength(orc):
    rng = np.random.default_rng(10)
    x = rng.standard_normal(4000).astype(np.float32) * 0.05
    best = [orc.fl_search_f32(x, k, sign=1)[2].min() for k in range(2, 11)]
    assert all(b2 <= b1 for b1, b2 in zip(best, best[1:]))


# ----------------------------------------------------------------------------
# Integer compute: GEMM, convolution, epilogue, pools, eltwise, layer error.
# ----------------------------------------------------------------------------
def test_gemm_vs_numpy(orc):
    rng = np.random.default_rng(11)
    A = rng.integers(-128, 128, (33, 70))
    B = rng.integers(-128, 128, (19, 70))
    assert np.array_equal(orc.gemm(A, B), A.astype(np.int64) @ B.astype(np.int64).T)


def test_conv_vs_float64_conv_of_dequantized_values(orc):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(12)
    for (N, C, H, W, K, R, stride, pad) in [(2, 3, 9, 7, 4, 3, 1, 1), (1, 5, 12, 12, 3, 5, 2, 2),
                                            (2, 4, 8, 8, 6, 1, 2, 0), (1, 2, 11, 11, 2, 7, 4, 3)]:
        x = rng.integers(0, 256, (N, C, H, W))
        w = rng.integers(-128, 128, (K, C, R, R))
        fa, fw = 5, 9
        y = orc.conv2d(x, w, stride, pad)
        xf = torch.tensor(x * 2.0 ** -fa, dtype=torch.float64)
        wf = torch.tensor(w * 2.0 ** -fw, dtype=torch.float64)
        ref = torch.nn.functional.conv2d(xf, wf, stride=stride, padding=pad).numpy()
        assert np.array_equal(y.astype(np.float64) * 2.0 ** -(fa + fw), ref)
        for _ in range(5):
            n, k = rng.integers(0, N), rng.integers(0, K)
            oh, ow = rng.integers(0, y.shape[2]), rng.integers(0, y.shape[3])
            assert orc.conv2d_point(x, w, stride, pad, n, k, oh, ow) == y[n, k, oh, ow]


def test_epilogue_exact(orc):
    rng = random.Random(13)
    for _ in range(40):
        N, Cc, hw = 2, 3, 4
        acc = np.array([rng.randint(-2 ** 20, 2 ** 20) for _ in range(N * Cc * hw)]).reshape(N, Cc, hw)
        s_acc = rng.randint(0, 25)
        use_b, use_s, relu = rng.random() < 0.6, rng.random() < 0.6, rng.random() < 0.5
        b = np.array([rng.randint(-2 ** 20, 2 ** 20) for _ in range(Cc)]) if use_b else None
        fl_b = rng.randint(-8, 15)
        a1 = np.array([rng.randint(0, 2 ** 16 - 1) for _ in range(Cc)]) if use_s else None
        a2 = np.array([rng.randint(-2 ** 20, 2 ** 20) for _ in range(Cc)]) if use_s else None
        fl_a1, fl_a2 = rng.randint(0, 15), rng.randint(-8, 15)
        try:
            v, s = orc.epilogue(acc, s_acc, b, fl_b, a1, fl_a1, a2, fl_a2, relu)
        except orc.OracleError:
            # only allowed when some aligned operand needs more than 62 bits
            sa = max(s_acc, fl_b) if use_b else s_acc
            big = max(abs(int(acc.max())), abs(int(acc.min()))) * 2 ** (sa - s_acc)
            if use_b:
                big = max(big, max(abs(int(t)) for t in b) * 2 ** (sa - fl_b))
            if use_s:
                big = big * max(int(t) for t in a1) * 2 ** max(0, fl_a2 - sa - fl_a1)
                big = max(big, max(abs(int(t)) for t in a2) * 2 ** max(0, sa + fl_a1 - fl_a2))
            assert big >= 2 ** 62
            continue
        for n, c, p in itertools.product(range(N), range(Cc), range(hw)):
            val = Fr(int(acc[n, c, p])) * Fr(2) ** -s_acc
            if use_b:
                val += Fr(int(b[c])) * Fr(2) ** -fl_b
            if use_s:
                val = val * Fr(int(a1[c])) * Fr(2) ** -fl_a1 + Fr(int(a2[c])) * Fr(2) ** -fl_a2
            if relu:
                val = max(val, Fr(0))
            assert Fr(int(v[n, c, p])) * Fr(2) ** -s == val


def test_maxpool_vs_torch(orc):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(14)
    for (H, k, st, pad) in [(13, 3, 2, 1), (12, 2, 2, 0), (55, 3, 2, 0)]:
        x = rng.integers(-128, 128, (2, 3, H, H))
        y = orc.maxpool(x, k, st, pad)
        ref = torch.nn.functional.max_pool2d(torch.tensor(x, dtype=torch.float64), k, st, pad)
        assert np.array_equal(y, ref.numpy().astype(np.int64))


def test_avgpool_and_eltwise(orc):
    rng = np.random.default_rng(15)
    x = rng.integers(0, 256, (2, 4, 7, 7))
    y = orc.avgpool_global(x, 669)
    assert np.array_equal(y, x.reshape(2, 4, -1).sum(-1) * 669)
    a = rng.integers(-128, 128, 50)
    b = rng.integers(0, 256, 50)
    v, s = orc.eltwise_add(a, 3, b, 6, relu=True)
    assert s == 6
    for i in range(50):
        want = max(Fr(int(a[i]), 8) + Fr(int(b[i]), 64), Fr(0))
        assert Fr(int(v[i]), 64) == want


def test_layer_error_vs_rationals(orc):
    rng = np.random.default_rng(16)
    ref = rng.standard_normal(40).astype(np.float32)
    codes = orc.quantize_f32(ref, 6, 3, 1)
    out = orc.layer_error(ref, codes, 6, 3, 1)
    want = sum((Fr(float(r)) - Fr(int(c), 8)) ** 2 for r, c in zip(ref, codes))
    assert out[0] == pytest.approx(float(want), rel=1e-15)
    assert out[1] == ref.min() and out[2] == ref.max()
    assert out[3] == pytest.approx(float(np.std(ref.astype(np.float64))), rel=1e-12)

"""Pins of the oracle's FP32 teacher (the full-precision reference of the
per-layer sensitivity sweep), each against something other than the oracle:
torch float64 convolution on data whose sums are exact, brute-force Python
loops in the defined summation order, and exact rationals rounded once to
fp32 for the fma.  CPU only.
"""
from fractions import Fraction

import numpy as np
import pytest

import synth


@pytest.fixture(scope="module")
def orc():
    import oracle
    oracle.lib()
    return oracle


def round_to_f32(q):
    """Correctly rounded (ties to even) float32 of a rational q."""
    f = np.float32(float(q))  # may be off by one ulp (double rounding)
    cands = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    best = min(cands, key=lambda c: (abs(Fraction(float(c)) - q),
                                     int(np.frombuffer(np.float32(c).tobytes(), np.uint32)[0]) & 1))
    return np.float32(best)


def test_conv_on_exact_data_matches_torch_f64(orc):
    import torch
    x = synth.integers(61, "tx", (2, 5, 7, 6), -8, 8).astype(np.float32)
    w = synth.integers(61, "tw", (4, 5, 3, 3), -8, 8).astype(np.float32)
    for stride, pad in [(1, 1), (2, 0), (2, 1)]:
        got = orc.teacher_conv2d(x, w, stride, pad)
        want = torch.nn.functional.conv2d(torch.from_numpy(x.astype(np.float64)),
                                          torch.from_numpy(w.astype(np.float64)),
                                          stride=stride, padding=pad).numpy().astype(np.float32)
        assert np.array_equal(got, want)


def test_conv_is_the_ordered_fp64_sum_rounded_once(orc):
    # brute force: Python floats are fp64, summed in the order r, s, c
    x = synth.normal(62, "tx", (1, 3, 5, 5))
    w = synth.normal(62, "tw", (2, 3, 3, 3))
    stride, pad = 2, 1
    got = orc.teacher_conv2d(x, w, stride, pad)
    Ho = (5 + 2 * pad - 3) // stride + 1
    for k in range(2):
        for oh in range(Ho):
            for ow in range(Ho):
                acc = 0.0
                for r in range(3):
                    ih = oh * stride - pad + r
                    if not 0 <= ih < 5:
                        continue
                    for s in range(3):
                        iw = ow * stride - pad + s
                        if not 0 <= iw < 5:
                            continue
                        for c in range(3):
                            acc = acc + float(x[0, c, ih, iw]) * float(w[k, c, r, s])
                assert got[0, k, oh, ow] == np.float32(acc)


def test_conv_rounds_the_exact_sum_to_nearest_even(orc):
    # integer products below 2^24 over 27 taps: the fp64 sum is exact, the
    # fp32 result must be its correctly rounded value (sums beyond 2^24)
    x = synth.integers(63, "tx", (1, 3, 4, 4), 0, 4095).astype(np.float32)
    w = synth.integers(63, "tw", (3, 3, 3, 3), 0, 4095).astype(np.float32)
    got = orc.teacher_conv2d(x, w, 1, 0)
    xi, wi = x.astype(np.int64), w.astype(np.int64)
    for k in range(3):
        for oh in range(2):
            for ow in range(2):
                exact = int((xi[0, :, oh:oh + 3, ow:ow + 3] * wi[k]).sum())
                assert exact >= 2 ** 24
                assert got[0, k, oh, ow] == round_to_f32(Fraction(exact))


def test_affine_is_one_correctly_rounded_fma(orc):
    t = synth.normal(64, "tt", (3, 5, 4))
    a1 = synth.uniform(64, "a1", (5,), 0.5, 1.5)
    a2 = synth.normal(64, "a2", (5,), std=0.1)
    got = orc.teacher_affine(t, a1, a2, relu=False)
    for idx in np.ndindex(t.shape):
        c = idx[1]
        q = Fraction(float(t[idx])) * Fraction(float(a1[c])) + Fraction(float(a2[c]))
        assert got[idx] == round_to_f32(q), idx
    # ReLU maps negatives and -0.0 to +0.0; bias is one fp32 add
    t2 = np.array([[-1.5, -0.0, 0.0, 2.25]], np.float32).reshape(1, 4)
    r = orc.teacher_affine(t2.reshape(1, 4), bias=np.zeros(4, np.float32), relu=True)
    assert list(r.ravel()) == [0.0, 0.0, 0.0, 2.25] and not np.signbit(r).any()
    b = synth.normal(64, "b", (5,))
    got = orc.teacher_affine(t, bias=b, relu=True)
    want = np.maximum(t + b[None, :, None], np.float32(0))
    assert np.array_equal(got, want)


def test_avgpool_is_the_ordered_fp64_mean(orc):
    x = synth.normal(65, "tx", (2, 3, 7, 7))
    got = orc.teacher_avgpool(x)
    for n in range(2):
        for c in range(3):
            acc = 0.0
            for v in x[n, c].ravel():
                acc = acc + float(v)
            assert got[n, c] == np.float32(acc / 49.0)

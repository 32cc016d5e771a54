"""Kernel-level parity of libfxpq (through its C ABI) against the CPU oracle.

Bit-exact: codes, chosen fractional lengths and signs, int32 accumulators,
pooled codes.  Error sums (layer error, reported SSE vectors): relative 1e-9,
far inside the 1e-5 the hot path is held to.  Inputs are seeded (synth) and
include ragged tails, exact rounding ties, zeros, outliers and saturation.
"""
import numpy as np
import pytest

import synth
from gpu_util import DEV, decode8, dev, empty, fmt_dev, fmt_host, fmt_new, host, note

pytestmark = pytest.mark.gpu

FL_LO, FL_HI = -8, 15


@pytest.fixture(scope="module")
def fx():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2203_12091_amd import fxpq
    return fxpq


@pytest.fixture(scope="module")
def h(fx):
    import torch
    hd = fx.Handle(0)
    fx.set_stream(hd, torch.cuda.current_stream())
    yield hd
    hd.close()


@pytest.fixture(scope="module")
def orc():
    import oracle
    oracle.lib()
    return oracle


def check_flags(fx, h, allowed=0):
    flags = fx.sync_status(h)
    assert flags & ~allowed == 0, f"device flags {flags:#x}"


# ----------------------------------------------------------------------------
# inputs
# ----------------------------------------------------------------------------
def adversarial_f32(seed, n):
    x = synth.normal(seed, "adv", (n,), std=1.0)
    g = synth.rng_for(seed, "adv-kinds")
    kind = g.integers(0, 8, n)
    # exact ties at several scales, tiny, zero, negative zero, representable
    x = np.where(kind == 0, (g.integers(-200, 200, n) + 0.5) * 2.0 ** -4, x)
    x = np.where(kind == 1, g.standard_normal(n) * 1e-30, x)
    x = np.where(kind == 2, 0.0, x)
    x = np.where(kind == 3, -0.0, x)
    x = np.where(kind == 4, g.integers(-100, 100, n) * 2.0 ** -5, x)
    return x.astype(np.float32)


# ----------------------------------------------------------------------------
# quantize / requant
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("n", [1, 3, 4, 4099, 1_000_003])
def test_quantize_codes_bit_exact(fx, h, orc, n):
    x = adversarial_f32(n, n)
    xd = dev(x)
    for (k, fl, sign, ct) in [(8, 4, 1, fx.I8), (8, 6, 0, fx.U8OFF), (8, 3, 0, fx.C8),
                              (8, 3, 1, fx.C8), (6, 2, 1, fx.I8), (4, -1, 1, fx.I8),
                              (16, 12, 1, fx.I16), (12, 9, 0, fx.I16), (24, 15, 1, fx.I32),
                              (2, 0, 1, fx.I8)]:
        note("quantize", n, k, fl, sign, ct)
        f = fmt_dev(k, fl, sign)
        torch_dt = {fx.I8: "int8", fx.U8OFF: "int8", fx.C8: "int8", fx.I16: "int16", fx.I32: "int32"}[ct]
        import torch
        codes = empty((n,), getattr(torch, torch_dt))
        fx.quantize(h, xd, n, f, codes, ct)
        got = host(codes).astype(np.int64)
        if ct == fx.U8OFF or (ct == fx.C8 and sign == 0):
            got = got + 128
        want = orc.quantize_f32(x, k, fl, sign)
        assert np.array_equal(got, want), (k, fl, sign, ct)
    check_flags(fx, h)


def test_quantize_non_finite_raises_flag(fx, h, orc):
    """NaN / Inf in an fp32 input has no code (the oracle rejects it): the
    sticky non-finite flag is raised, the finite values' codes stay exact,
    and the flag is cleared by the read (the next clean call has none)."""
    import torch
    n = 100_003
    x = adversarial_f32(11, n)
    bad = {7: np.nan, 4096: np.inf, n - 1: -np.inf}
    for i, v in bad.items():
        x[i] = v
    ok = np.ones(n, bool)
    ok[list(bad)] = False
    for (k, fl, sign, ct, dt) in [(8, 4, 1, fx.I8, torch.int8), (16, 10, 1, fx.I16, torch.int16)]:
        note("quantize non-finite", k, fl, sign, ct)
        codes = empty((n,), dt)
        fx.quantize(h, dev(x), n, fmt_dev(k, fl, sign), codes, ct)
        assert fx.sync_status(h) & fx.FLAG_NONFINITE
        got = host(codes).astype(np.int64)[ok]
        assert np.array_equal(got, orc.quantize_f32(x[ok], k, fl, sign))
    clean = empty((n,), torch.int8)
    fx.quantize(h, dev(np.where(ok, x, 0).astype(np.float32)), n, fmt_dev(8, 4, 1), clean, fx.I8)
    check_flags(fx, h)


def test_requant_int_sources_bit_exact(fx, h, orc):
    import torch
    g = synth.rng_for(7, "req")
    for n, s, dt in [(4097, 13, fx.I32), (10_001, 27, fx.I64), (5, 0, fx.I32), (8, -3, fx.I64)]:
        if dt == fx.I32:
            v = g.integers(-2 ** 31, 2 ** 31, n, dtype=np.int64).astype(np.int32)
        else:
            v = g.integers(-2 ** 50, 2 ** 50, n, dtype=np.int64) >> g.integers(0, 40, n)
        vd = dev(v)
        sd = torch.tensor([s], dtype=torch.int32, device=DEV)
        for k, fl, sign in [(8, 0, 1), (8, -12, 0), (16, -2, 1), (8, 3, 1), (32, -5, 1)]:
            note("requant-int", n, s, dt, k, fl, sign)
            f = fmt_dev(k, fl, sign)
            ct = fx.I32 if k > 16 else (fx.I16 if k > 8 else fx.C8)
            codes = empty((n,), {fx.I32: torch.int32, fx.I16: torch.int16, fx.C8: torch.int8}[ct])
            fx.requant(h, fx.src_int(vd, dt, sd), n, f, codes, ct)
            got = host(codes).astype(np.int64)
            if ct == fx.C8 and sign == 0:
                got += 128
            want = orc.quantize_i64(v.astype(np.int64), s, k, fl, sign)
            assert np.array_equal(got, want)
    check_flags(fx, h, allowed=fx.FLAG_CODE)


def test_int64_values_beyond_fp64_exact(fx, h, orc):
    """int64 values of magnitude 2^53 .. 2^62 (what wide C-Blocks produce; fp64
    holds them exactly only below 2^53): the FL search (its exact general
    pass) and the requantization match the oracle bit for bit, with exact
    rounding ties planted at every shift the formats use."""
    import torch
    g = synth.rng_for(53, "big-int64")
    n = 50_001
    v = (g.standard_normal(n) * 2.0 ** 58).astype(np.int64)
    v[::7] = g.integers(-2 ** 61, 2 ** 61, v[::7].size, dtype=np.int64)
    for s, k, fl in [(55, 8, 3), (50, 16, 6), (58, 32, 15), (40, 8, -8)]:
        d = s - fl
        # (2j + 1) * 2^(d - 1): exactly half way between two codes
        j = g.integers(-100, 100, 64, dtype=np.int64)
        v[1000:1064] = (2 * j + 1) << (d - 1)
        vd = dev(v)
        sd = torch.tensor([s], dtype=torch.int32, device=DEV)
        note("int64 beyond fp64", s, k, fl)
        for sign in ((1,) if k == 32 else (0, 1)):  # no code type holds unsigned 32-bit codes
            f = fmt_dev(k, fl, sign)
            # the code type holds the format's range (unsigned 16-bit: int32)
            ct = fx.I32 if k - sign >= 16 else (fx.I16 if k > 8 else fx.C8)
            codes = empty((n,), {fx.I32: torch.int32, fx.I16: torch.int16, fx.C8: torch.int8}[ct])
            fx.requant(h, fx.src_int(vd, fx.I64, sd), n, f, codes, ct)
            got = host(codes).astype(np.int64)
            if ct == fx.C8 and sign == 0:
                got += 128
            assert np.array_equal(got, orc.quantize_i64(v, s, k, fl, sign)), (s, k, fl, sign)
        for wl in (8, 16, 32):
            (gwl, gfl, gsign, gst), _ = run_fl_search(fx, h, fx.src_int(vd, fx.I64, sd), n, wl,
                                                      fx.SIGN_AUTO)
            ofl, osign, _ = orc.fl_search_i64(v, s, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            assert (gfl, gsign, gst) == (ofl, osign, 0), (s, wl)
    check_flags(fx, h)


# ----------------------------------------------------------------------------
# FL search
# ----------------------------------------------------------------------------
def run_fl_search(fx, h, src, n, wl, sign, report=False):
    import torch
    out = fmt_new()
    sse = torch.full((FL_HI - FL_LO + 1,), -1.0, dtype=torch.float64, device=DEV) if report else None
    fx.fl_search(h, src, n, wl, sign, FL_LO, FL_HI, out, sse)
    return fmt_host(out), (host(sse) if report else None)


def config1_tensors():
    W = synth.normal(0, "fc.w", (256, 512), std=0.05)
    A = synth.relu_normal(0, "fc.a", (32, 512))
    return W, A


def f32_cases():
    W, A = config1_tensors()
    big = synth.normal(3, "big", (1_000_003,), std=1.0)
    outlier = synth.normal(4, "outl", (200_003,), std=0.1)
    outlier[12345] = 60.0
    neg = -np.abs(synth.normal(5, "neg", (1003,)))
    sub = (synth.normal(6, "sub", (777,)) * 1e-39).astype(np.float32)
    rep = (synth.integers(7, "rep", (4096,), -100, 100) * 2.0 ** -3).astype(np.float32)
    return [("cfg1.W", W.ravel()), ("cfg1.A", A.ravel()), ("big", big), ("outlier", outlier),
            ("neg", neg), ("subnormal", sub), ("representable", rep),
            ("zeros", np.zeros(1000, np.float32)), ("one", np.array([0.3], np.float32)),
            ("adv", adversarial_f32(8, 100_003))]


@pytest.mark.parametrize("wl", [8, 6, 4])
def test_fl_search_f32_matches_exhaustive_oracle(fx, h, orc, wl):
    for name, x in f32_cases():
        n = x.size
        for sign in ((fx.SIGN_AUTO, 0, 1) if n < 300_000 else (fx.SIGN_AUTO,)):
            note("fls-f32", name, n, wl, sign)
            (gwl, gfl, gsign, gst), _ = run_fl_search(fx, h, fx.src_f32(dev(x)), n, wl, sign)
            ofl, osign, osse = orc.fl_search_f32(x, wl, sign, FL_LO, FL_HI)
            assert gst == 0 and gwl == wl
            assert (gfl, gsign) == (ofl, osign), (name, wl, sign, osse)
    check_flags(fx, h)


def test_fl_search_report_mode_sse_vector(fx, h, orc):
    for name, x in f32_cases()[:4] + [("zeros", np.zeros(64, np.float32))]:
        for wl in (8, 4, 16):
            note("fls-report", name, wl)
            (gwl, gfl, gsign, gst), sse = run_fl_search(fx, h, fx.src_f32(dev(x)), x.size, wl,
                                                        fx.SIGN_AUTO, report=True)
            ofl, osign, osse = orc.fl_search_f32(x, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            assert (gfl, gsign, gst) == (ofl, osign, 0)
            np.testing.assert_allclose(sse, osse, rtol=1e-9, atol=0)
    check_flags(fx, h)


def test_fl_search_int_sources(fx, h, orc):
    import torch
    for seed, n, s, dt, spread in [(1, 1_000_001, 12, fx.I32, 2 ** 20), (2, 65_537, 30, fx.I64, 2 ** 44),
                                   (3, 17, 3, fx.I32, 100), (4, 300_000, 0, fx.I32, 2 ** 28),
                                   (5, 4096, 40, fx.I64, 2 ** 50)]:
        g = synth.rng_for(seed, "flsint")
        v = (g.standard_normal(n) * spread).astype(np.int64)
        if seed == 4:
            v = np.maximum(v, 0)
        vv = v.astype(np.int32) if dt == fx.I32 else v
        sd = torch.tensor([s], dtype=torch.int32, device=DEV)
        for wl in (8, 5, 16, 32):
            note("fls-int", seed, n, s, dt, wl)
            (gwl, gfl, gsign, gst), _ = run_fl_search(fx, h, fx.src_int(dev(vv), dt, sd), n, wl,
                                                      fx.SIGN_AUTO)
            ofl, osign, _ = orc.fl_search_i64(v, s, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            assert (gfl, gsign, gst) == (ofl, osign, 0), (seed, wl)
    check_flags(fx, h)


def heavy_tail_case(seed, n, nout, omag):
    """Normal bulk (std 2^10) plus nout outliers of magnitude ~2^omag: at short
    word lengths the best fl clips the outliers and lies well above the
    largest non-saturating fl."""
    g = synth.rng_for(seed, "heavy")
    v = np.rint(g.standard_normal(n) * 2 ** 10).astype(np.int64)
    idx = g.choice(n, nout, replace=False)
    v[idx] = (np.where(g.random(nout) < 0.5, -1, 1) * (2 ** omag) * (1 + g.random(nout))).astype(np.int64)
    return v


def beta_nosat(v, s, wl, sign):
    from fractions import Fraction as F
    qmax, qmin = 2 ** (wl - sign) - 1, (-(2 ** (wl - 1)) if sign else 0)
    mx, mn = int(v.max()), int(v.min())
    for b in range(FL_HI, FL_LO - 1, -1):
        if F(mx) * F(2) ** (b - s) <= qmax + F(1, 2) and F(mn) * F(2) ** (b - s) >= qmin - F(1, 2):
            return b
    return FL_LO - 1


def test_fl_search_best_fl_above_the_window(fx, h, orc):
    # Short word lengths with outliers: the two-candidate window cannot decide
    # and the exact pass evaluates the candidates the clipping bounds leave
    # (1 to 5 above the window here, and the whole range above it once).
    import torch
    above = []
    s = 12
    for seed, n, nout, omag in [(11, 200_000, 3, 14), (12, 200_000, 30, 12), (13, 200_000, 300, 11),
                                (14, 50_001, 1, 18), (16, 100_000, 10, 16)]:
        v = heavy_tail_case(seed, n, nout, omag)
        sd = torch.tensor([s], dtype=torch.int32, device=DEV)
        x32 = (v.astype(np.float64) * 2.0 ** -s).astype(np.float32)  # exact
        for wl in (3, 4, 5, 6, 8):
            note("fls-heavy", seed, n, wl)
            ofl, osign, _ = orc.fl_search_i64(v, s, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            above.append(ofl - beta_nosat(v, s, wl, osign))
            (gwl, gfl, gsign, gst), _ = run_fl_search(fx, h, fx.src_int(dev(v.astype(np.int32)), fx.I32, sd),
                                                      n, wl, fx.SIGN_AUTO)
            assert (gfl, gsign, gst) == (ofl, osign, 0), (seed, wl)
            ffl, fsign, _ = orc.fl_search_f32(x32, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            (gwl, gfl, gsign, gst), _ = run_fl_search(fx, h, fx.src_f32(dev(x32)), n, wl, fx.SIGN_AUTO)
            assert (gfl, gsign, gst) == (ffl, fsign, 0), (seed, wl)
    # the fixture exercises the window alone, a short exact range and a long one
    assert min(above) <= 1 and any(2 <= a <= 5 for a in above) and max(above) >= 6, above
    check_flags(fx, h)


# ----------------------------------------------------------------------------
# GEMM / conv with the C-Block epilogue
# ----------------------------------------------------------------------------
def make_epilogue_params(seed, k, with_bias, with_scale):
    g = synth.rng_for(seed, "epi")
    bias = g.integers(-2 ** 20, 2 ** 20, k).astype(np.int32) if with_bias else None
    a1 = g.integers(2 ** 14, 2 ** 16, k).astype(np.int32) if with_scale else None
    a2 = g.integers(-2 ** 13, 2 ** 13, k).astype(np.int32) if with_scale else None
    return bias, a1, a2


def gpu_conv_case(fx, h, orc, N, Cin, H, W, K, R, stride, pad, in_signed, relu, with_bias,
                  with_scale, seed, x_type=None):
    import torch
    lo, hi = (-128, 127) if in_signed else (0, 255)
    xc = synth.integers(seed, "x", (N, Cin, H, W), lo, hi)
    wc = synth.integers(seed, "w", (K, Cin, R, R), -128, 127)
    fl_in, fl_w, fl_b, fl_a1, fl_a2 = 5, 9, 11, 15, 15
    # device layouts: NHWC codes, KRSC weights
    x_nhwc = np.transpose(xc, (0, 2, 3, 1))
    w_krsc = np.transpose(wc, (0, 2, 3, 1)).reshape(K, -1)
    cin_dev = Cin
    if Cin == 3:  # padded RGB: 4 channels, filter rows padded to 64 bytes
        x_nhwc = np.concatenate([x_nhwc, np.zeros(x_nhwc.shape[:3] + (1,), np.int64)], axis=3)
        w4 = np.concatenate([np.transpose(wc, (0, 2, 3, 1)), np.zeros((K, R, R, 1), np.int64)], axis=3)
        w_krsc = w4.reshape(K, -1)
        kp = (w_krsc.shape[1] + 63) // 64 * 64
        w_krsc = np.concatenate([w_krsc, np.zeros((K, kp - w_krsc.shape[1]), np.int64)], axis=1)
        cin_dev = 4
    if x_type is None:
        x_type = fx.I8 if in_signed else fx.U8OFF
    stored = x_nhwc - (0 if in_signed else 128)
    xd = dev(stored.astype(np.int8))
    wd = dev(w_krsc.astype(np.int8))
    colsum = empty((K,), torch.int32)
    fx.weight_colsum(h, wd, K, w_krsc.shape[1], colsum)
    fin = fmt_dev(8, fl_in, 1 if in_signed else 0)
    bias, a1, a2 = make_epilogue_params(seed, K, with_bias, with_scale)
    keep = []
    bd = dev(bias) if bias is not None else None
    a1d = dev(a1) if a1 is not None else None
    a2d = dev(a2) if a2 is not None else None
    ep = fx.epilogue(K, fl_w, fin, bias=bd, fl_bias=fl_b, relu=relu, scale=a1d, fl_scale=fl_a1,
                     shift=a2d, fl_shift=fl_a2)
    Ho = (H + 2 * pad - R) // stride + 1
    Wo = (W + 2 * pad - R) // stride + 1
    acc = empty((N, Ho, Wo, K), torch.int32)
    mm = torch.zeros(2, dtype=torch.float64, device=DEV)
    desc = fx.conv_desc(N, H, W, cin_dev, K, R, R, stride, pad)
    note("qconv", N, Cin, H, W, K, R, stride, pad, in_signed, x_type)
    fx.qconv(h, desc, xd, x_type, wd, colsum, ep, acc, mm)
    got = host(acc)
    want = orc.conv2d(xc, wc, stride, pad)  # NKHW int64
    assert np.array_equal(got.transpose(0, 3, 1, 2).astype(np.int64), want)
    v, s_out = orc.epilogue(want, fl_in + fl_w, bias, fl_b, a1, fl_a1, a2, fl_a2, relu)
    gmm = host(mm)
    assert gmm[0] == v.min() and gmm[1] == v.max()
    keep += [bd, a1d, a2d]
    return acc, ep, mm, v, s_out, keep


CONV_CASES = [
    # N, Cin, H, W, K, R, stride, pad, signed input, relu, bias, scale
    (2, 64, 9, 11, 64, 3, 1, 1, False, True, False, True),
    (3, 128, 7, 7, 192, 1, 2, 0, True, False, True, False),
    (1, 3, 23, 21, 64, 7, 2, 3, True, True, False, True),
    (2, 16, 10, 10, 40, 3, 2, 1, False, True, True, False),
    (1, 192, 13, 13, 384, 3, 1, 1, False, True, True, False),
    (2, 64, 12, 12, 256, 1, 1, 0, False, False, False, True),
]


@pytest.mark.parametrize("case", CONV_CASES, ids=[str(i) for i in range(len(CONV_CASES))])
def test_qconv_accumulators_and_epilogue_minmax(fx, h, orc, case):
    gpu_conv_case(fx, h, orc, *case, seed=11)
    check_flags(fx, h)


# 3x3 shapes the halo tiles take (c % 64 == 0, k % 256 == 0, r*s*c >= 1024):
# whole images per tile (one, two or four), output rows split over several
# tiles with a partial last one, stride 2, odd sizes, partial last image group
HALO_CASES = [
    (3, 128, 14, 14, 256, 3, 1, 1, False, True, False, True),
    (5, 128, 7, 7, 512, 3, 1, 1, True, False, True, False),
    (3, 128, 14, 14, 256, 3, 2, 1, False, True, True, True),
    (2, 192, 9, 11, 256, 3, 1, 1, False, False, False, True),
    (1, 128, 28, 28, 256, 3, 1, 1, True, True, True, False),
    (2, 128, 30, 17, 256, 3, 2, 1, False, True, False, True),  # patch too big: implicit GEMM
]


@pytest.mark.parametrize("case", HALO_CASES, ids=[str(i) for i in range(len(HALO_CASES))])
def test_qconv_halo_and_gemm_tiles(fx, h, orc, case):
    # the same accumulators and min / max from both tile families
    try:
        for mode in (fx.TILING_HALO, fx.TILING_GEMM):
            fx.set_conv_tiling(h, mode)
            note("tiling", mode)
            gpu_conv_case(fx, h, orc, *case, seed=17)
    finally:
        fx.set_conv_tiling(h, fx.TILING_AUTO)
    check_flags(fx, h)


def test_c8_input_storage_follows_format(fx, h, orc):
    gpu_conv_case(fx, h, orc, 2, 64, 8, 8, 64, 3, 1, 1, False, True, False, True, seed=12,
                  x_type=fx.C8)
    gpu_conv_case(fx, h, orc, 2, 64, 8, 8, 64, 3, 1, 1, True, True, False, True, seed=13,
                  x_type=fx.C8)
    check_flags(fx, h)


def test_qgemm_config1_shape_and_ragged(fx, h, orc):
    import torch
    for (M, N, K, signed) in [(32, 256, 512, False), (37, 200, 272, True), (5, 1000, 2048, False),
                              (256, 64, 64, True)]:
        note("qgemm", M, N, K, signed)
        lo, hi = (-128, 127) if signed else (0, 255)
        A = synth.integers(M + N, "A", (M, K), lo, hi)
        B = synth.integers(M + N, "B", (N, K), -128, 127)
        Ad = dev((A - (0 if signed else 128)).astype(np.int8))
        Bd = dev(B.astype(np.int8))
        cs = empty((N,), torch.int32)
        fx.weight_colsum(h, Bd, N, K, cs)
        Cd = empty((M, N), torch.int32)
        fx.qgemm(h, M, N, K, Ad, fx.I8 if signed else fx.U8OFF, Bd, cs, None, Cd)
        assert np.array_equal(host(Cd).astype(np.int64), orc.gemm(A, B))
    check_flags(fx, h)


def test_acc_source_fl_search_and_requant(fx, h, orc):
    import torch
    for case in CONV_CASES[:3] + [CONV_CASES[5]]:
        acc, ep, mm, v, s_out, keep = gpu_conv_case(fx, h, orc, *case, seed=21)
        n = acc.numel()
        src = fx.src_acc(acc, ep, mm)
        sd = empty((1,), torch.int32)
        fx.epilogue_scale(h, ep, sd)
        assert int(host(sd)[0]) == s_out
        for wl in (8, 6):
            note("fls-acc", case, wl)
            out = fmt_new()
            fx.fl_search(h, src, n, wl, fx.SIGN_AUTO, FL_LO, FL_HI, out)
            gwl, gfl, gsign, gst = fmt_host(out)
            # oracle on the NHWC-ordered exact values
            vn = v.transpose(0, 2, 3, 1).ravel()
            ofl, osign, _ = orc.fl_search_i64(vn, s_out, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            assert (gfl, gsign, gst) == (ofl, osign, 0)
            codes = empty((n,), torch.int8)
            fx.requant(h, src, n, out, codes, fx.C8)
            got = decode8(host(codes), gsign == 0)
            assert np.array_equal(got, orc.quantize_i64(vn, s_out, wl, ofl, osign))
    check_flags(fx, h)


def test_add_source(fx, h, orc):
    import torch
    n = 100_003
    a = synth.integers(31, "a", (n,), -128, 127)
    b = synth.integers(31, "b", (n,), 0, 255)
    fa, fb = fmt_dev(8, 3, 1), fmt_dev(8, 6, 0)
    ad = dev(a.astype(np.int8))
    bd = dev((b - 128).astype(np.int8))
    for relu in (True, False):
        src = fx.src_add(ad, fx.C8, fa, bd, fx.C8, fb, relu)
        note("add", relu)
        out = fmt_new()
        fx.fl_search(h, src, n - 3, 8, fx.SIGN_AUTO, FL_LO, FL_HI, out)
        v, s = orc.eltwise_add(a[:n - 3], 3, b[:n - 3], 6, relu)
        ofl, osign, _ = orc.fl_search_i64(v, s, 8, fx.SIGN_AUTO, FL_LO, FL_HI)
        gwl, gfl, gsign, gst = fmt_host(out)
        assert (gfl, gsign, gst) == (ofl, osign, 0)
        codes = empty((n - 3,), torch.int8)
        fx.requant(h, src, n - 3, out, codes, fx.C8)
        assert np.array_equal(decode8(host(codes), gsign == 0), orc.quantize_i64(v, s, 8, ofl, osign))
    check_flags(fx, h)


def test_requant_with_residual_minmax(fx, h, orc):
    # requantization of C-Block values that also reduces the min / max of the
    # residual sum they feed; the ADD search then uses that min / max
    import torch
    for ci, case in enumerate([CONV_CASES[0], CONV_CASES[5], CONV_CASES[1]]):
        acc, ep, mm, v, s_out, keep = gpu_conv_case(fx, h, orc, *case, seed=41 + ci)
        n = acc.numel()  # whole rows: an ACC source covers complete channel groups
        vn = v.transpose(0, 2, 3, 1).ravel()[:n]
        src = fx.src_acc(acc, ep, mm)
        out = fmt_new()
        fx.fl_search(h, src, n, 8, fx.SIGN_AUTO, FL_LO, FL_HI, out)
        gwl, gfl, gsign, gst = fmt_host(out)
        ofl, osign, _ = orc.fl_search_i64(vn, s_out, 8, fx.SIGN_AUTO, FL_LO, FL_HI)
        assert (gfl, gsign, gst) == (ofl, osign, 0)
        b = synth.integers(51 + ci, "resid", (n,), 0, 255)
        fb = 4 + ci
        bd = dev((b - 128).astype(np.int8))
        fbd = fmt_dev(8, fb, 0)
        for relu in (True, False):
            note("requant+addmm", case, relu)
            codes = empty((n,), torch.int8)
            amm = torch.full((2,), 7.0, dtype=torch.float64, device=DEV)
            fx.requant_addmm(h, src, n, out, codes, fx.C8, bd, fx.C8, fbd, relu, amm)
            want = orc.quantize_i64(vn, s_out, 8, ofl, osign)
            assert np.array_equal(decode8(host(codes), gsign == 0), want)
            va, sa = orc.eltwise_add(want, ofl, b, fb, relu)
            gmm = host(amm)
            assert gmm[0] == va.min() and gmm[1] == va.max()
            # the sum's own search with that min / max
            asrc = fx.src_add(codes, fx.C8, out, bd, fx.C8, fbd, relu, amm)
            aout = fmt_new()
            fx.fl_search(h, asrc, n, 8, fx.SIGN_AUTO, FL_LO, FL_HI, aout)
            afl, asg, _ = orc.fl_search_i64(va, sa, 8, fx.SIGN_AUTO, FL_LO, FL_HI)
            assert fmt_host(aout)[1:] == (afl, asg, 0)
    check_flags(fx, h)


# ----------------------------------------------------------------------------
# pools and layer error
# ----------------------------------------------------------------------------
def test_maxpool_and_avgpool(fx, h, orc):
    import torch
    for (N, Cc, H, k, st, pad) in [(2, 64, 112, 3, 2, 1), (3, 12, 13, 3, 2, 0), (1, 32, 14, 2, 2, 0)]:
        note("maxpool", N, Cc, H, k, st, pad)
        x = synth.integers(H, "mp", (N, Cc, H, H), -128, 127)
        xd = dev(np.transpose(x, (0, 2, 3, 1)).astype(np.int8))
        Ho = (H + 2 * pad - k) // st + 1
        y = empty((N, Ho, Ho, Cc), torch.int8)
        fx.maxpool(h, xd, fx.I8, N, H, H, Cc, k, st, pad, y)
        assert np.array_equal(host(y).transpose(0, 3, 1, 2), orc.maxpool(x, k, st, pad))
    x = synth.integers(3, "ap", (4, 2048, 7, 7), 0, 255)
    xd = dev((np.transpose(x, (0, 2, 3, 1)) - 128).astype(np.int8))
    y = empty((4, 2048), torch.int64)
    note("avgpool")
    fx.avgpool_global(h, xd, fx.C8, fmt_dev(8, 2, 0), 4, 49, 2048, 669, y)
    assert np.array_equal(host(y), orc.avgpool_global(x, 669))
    check_flags(fx, h)


def test_layer_error(fx, h, orc):
    import torch
    x = synth.normal(5, "le", (1_000_003,))
    for k, fl, sign, ct in [(8, 5, 1, fx.I8), (6, 3, 1, fx.C8), (16, 12, 1, fx.I16)]:
        note("layer_error", k, fl, sign)
        codes = orc.quantize_f32(x, k, fl, sign)
        tdt = torch.int16 if ct == fx.I16 else torch.int8
        cd = dev(codes.astype(np.int16 if ct == fx.I16 else np.int8))
        out = torch.zeros(4, dtype=torch.float64, device=DEV)
        fx.layer_error(h, dev(x), cd, ct, fmt_dev(k, fl, sign), x.size, out)
        got = host(out)
        want = orc.layer_error(x, codes, k, fl, sign)
        np.testing.assert_allclose(got, want, rtol=1e-9)
    check_flags(fx, h)


def test_nonfinite_input_sets_flag_and_status(fx, h):
    x = synth.normal(9, "nan", (1000,))
    x[17] = np.nan
    note("nonfinite")
    (gwl, gfl, gsign, gst), _ = run_fl_search(fx, h, fx.src_f32(dev(x)), x.size, 8, fx.SIGN_AUTO)
    assert gst != 0
    assert fx.sync_status(h) & fx.FLAG_NONFINITE


def test_out_of_range_values_keep_error_status(fx, h, orc):
    # |v * 2^max(s, fl_hi)| >= 2^62 is outside the exact range of the general
    # pass: the format must carry a nonzero status and the range flag must be
    # raised; a search right after it must be unaffected
    import torch
    v = np.array([2 ** 61, -(2 ** 60), 12345, 0, 7] * 40, np.int64)
    sd = torch.tensor([0], dtype=torch.int32, device=DEV)
    note("fls-int out of range")
    (gwl, gfl, gsign, gst), _ = run_fl_search(fx, h, fx.src_int(dev(v), fx.I64, sd), v.size, 8,
                                              fx.SIGN_AUTO)
    assert gst != 0
    assert fx.sync_status(h) & fx.FLAG_RANGE
    w = synth.integers(12, "after-range", (5000,), -2 ** 40, 2 ** 40)
    sd = torch.tensor([20], dtype=torch.int32, device=DEV)
    (gwl, gfl, gsign, gst), _ = run_fl_search(fx, h, fx.src_int(dev(w), fx.I64, sd), w.size, 8,
                                              fx.SIGN_AUTO)
    ofl, osign, _ = orc.fl_search_i64(w, 20, 8, fx.SIGN_AUTO, FL_LO, FL_HI)
    assert (gfl, gsign, gst) == (ofl, osign, 0)
    check_flags(fx, h)

"""Fused FxP-QLayer (fxpq_qlayer: FL search + requantization in one call)
against the CPU oracle and against the two-call path, through the C ABI.

Bit-exact: chosen format and every code.  The format the output holds on
entry picks which window candidate's codes the search writes to the output
buffer and whether the other's go to the alternate buffer, so each case runs
with every pick: the chosen format's codes are then found in the output
buffer, copied from the alternate buffer, or requantized (not written by the
search, or the best fl lies above the window).
"""
from fractions import Fraction as F

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


def beta_nosat(vals, wl, sign):
    """Largest fl in range at which every value lies in [qmin - 1/2, qmax + 1/2]
    after scaling (exact rationals); vals are Fractions."""
    qmax, qmin = 2 ** (wl - sign) - 1, (-(2 ** (wl - 1)) if sign else 0)
    mx, mn = max(vals), min(vals)
    for b in range(FL_HI, FL_LO - 1, -1):
        if mx * F(2) ** b <= qmax + F(1, 2) and mn * F(2) ** b >= qmin - F(1, 2):
            return b
    return FL_LO - 1


def fr(v, s):
    """The exact value v * 2^-s."""
    return F(int(v)) * F(2) ** (-s)


def run_both_picks(fx, h, src, n, wl, sign, bnosat, want_fmt, want_codes, tag):
    """qlayer with the output format pre-set to no usable format, to each
    window candidate (then only that candidate's codes are written), and to a
    candidate with the other sign; then twice in a row on one format buffer.
    All must equal the oracle."""
    import torch
    b0 = max(FL_LO, bnosat)
    osign = want_fmt[2]
    outs = []
    for pre in (None, (wl, b0, osign), (wl, b0 + 1, osign), (wl, b0, 1 - osign)):
        note("qlayer", tag, n, wl, sign, "pre", pre)
        out = fmt_new() if pre is None else fmt_dev(*pre)
        codes = torch.full((n + 16,), 0x55, dtype=torch.int8, device=DEV)
        alt = empty((n + 16,), torch.int8)
        fx.qlayer(h, src, n, wl, sign, FL_LO, FL_HI, out, codes, fx.C8, alt)
        gwl, gfl, gsign, gst = fmt_host(out)
        assert (gwl, gfl, gsign, gst) == want_fmt, (tag, pre)
        got = host(codes)
        assert np.array_equal(decode8(got[:n], gsign == 0), want_codes), (tag, pre)
        assert np.all(got[n:] == 0x55), "wrote past n"
        outs.append(out)
    # second call on the same format buffer: the previous result picks
    out = outs[0]
    note("qlayer-repeat", tag, n, wl)
    codes = empty((n,), torch.int8)
    alt = empty((n,), torch.int8)
    fx.qlayer(h, src, n, wl, sign, FL_LO, FL_HI, out, codes, fx.C8, alt)
    assert fmt_host(out) == want_fmt
    assert np.array_equal(decode8(host(codes), want_fmt[2] == 0), want_codes)


def check_flags(fx, h, allowed=0):
    flags = fx.sync_status(h)
    assert flags & ~allowed == 0, f"device flags {flags:#x}"


@pytest.mark.parametrize("wl", [8, 6, 4])
def test_qlayer_f32_sources(fx, h, orc, wl):
    W = synth.normal(0, "fc.w", (256, 512), std=0.05).ravel()
    cases = [("cfg1.W", W), ("normal", synth.normal(61, "ql", (100_003,), std=1.0)),
             ("neg", -np.abs(synth.normal(62, "qlneg", (1003,)))),
             ("ties", (synth.integers(63, "qlt", (4099,), -300, 300) + 0.5).astype(np.float32) * 2.0 ** -5),
             ("zeros", np.zeros(1001, np.float32)), ("one", np.array([0.3], np.float32))]
    for name, x in cases:
        x = np.asarray(x, np.float32)
        n = x.size
        for sign in (fx.SIGN_AUTO, 1, 0):
            ofl, osign, _ = orc.fl_search_f32(x, wl, sign, FL_LO, FL_HI)
            want = orc.quantize_f32(x, wl, ofl, osign)
            bn = beta_nosat([F(float(v)) for v in (x.min(), x.max())], wl, osign)
            run_both_picks(fx, h, fx.src_f32(dev(x)), n, wl, sign, bn, (wl, ofl, osign, 0), want,
                           f"f32-{name}")
    check_flags(fx, h)


def test_qlayer_acc_sources_match_two_calls(fx, h, orc):
    # C-Block values (conv + bias / Scale / ReLU epilogue) against the oracle
    # and against fxpq_fl_search + fxpq_requant on the same buffers
    import torch
    from test_gpu_kernels import CONV_CASES, gpu_conv_case
    for ci, case in enumerate([CONV_CASES[0], CONV_CASES[1], CONV_CASES[5]]):
        acc, ep, mm, v, s_out, keep = gpu_conv_case(fx, h, orc, *case, seed=71 + ci)
        n = acc.numel()
        vn = v.transpose(0, 2, 3, 1).ravel()[:n]
        src = fx.src_acc(acc, ep, mm)
        for wl in (8, 6, 4):
            ofl, osign, _ = orc.fl_search_i64(vn, s_out, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            want = orc.quantize_i64(vn, s_out, wl, ofl, osign)
            bn = beta_nosat([fr(vn.min(), s_out), fr(vn.max(), s_out)], wl, osign)
            run_both_picks(fx, h, src, n, wl, fx.SIGN_AUTO, bn, (wl, ofl, osign, 0), want, f"acc{ci}")
            out2 = fmt_new()
            fx.fl_search(h, src, n, wl, fx.SIGN_AUTO, FL_LO, FL_HI, out2)
            c2 = empty((n,), torch.int8)
            fx.requant(h, src, n, out2, c2, fx.C8)
            assert fmt_host(out2) == (wl, ofl, osign, 0)
            assert np.array_equal(decode8(host(c2), osign == 0), want)
    check_flags(fx, h)


def test_qlayer_add_sources_ragged(fx, h, orc):
    n = 100_003
    a = synth.integers(81, "a", (n,), -128, 127)
    b = synth.integers(81, "b", (n,), 0, 255)
    fa, fb = fmt_dev(8, 3, 1), fmt_dev(8, 6, 0)
    ad = dev(a.astype(np.int8))
    bd = dev((b - 128).astype(np.int8))
    for relu in (True, False):
        for m in (n - 3, 16 * 1000 + 7, 15, 1):
            src = fx.src_add(ad, fx.C8, fa, bd, fx.C8, fb, relu)
            v, s = orc.eltwise_add(a[:m], 3, b[:m], 6, relu)
            for wl in (8, 5):
                ofl, osign, _ = orc.fl_search_i64(v, s, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
                want = orc.quantize_i64(v, s, wl, ofl, osign)
                bn = beta_nosat([fr(v.min(), s), fr(v.max(), s)], wl, osign)
                run_both_picks(fx, h, src, m, wl, fx.SIGN_AUTO, bn, (wl, ofl, osign, 0), want,
                               f"add-relu{int(relu)}")
    check_flags(fx, h)


def test_qlayer_best_fl_above_the_window(fx, h, orc):
    # outliers at short word lengths: the chosen fl lies above both window
    # candidates, so the codes come from the requantization pass
    import torch
    from test_gpu_kernels import heavy_tail_case
    s = 12
    sd = torch.tensor([s], dtype=torch.int32, device=DEV)
    above = 0
    for seed, n, nout, omag in [(11, 200_000, 3, 14), (14, 50_001, 1, 18)]:
        v = heavy_tail_case(seed, n, nout, omag)
        for wl in (3, 4, 6):
            ofl, osign, _ = orc.fl_search_i64(v, s, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            want = orc.quantize_i64(v, s, wl, ofl, osign)
            bn = beta_nosat([fr(v.min(), s), fr(v.max(), s)], wl, osign)
            above += ofl > bn + 1
            run_both_picks(fx, h, fx.src_int(dev(v.astype(np.int32)), fx.I32, sd), n, wl, fx.SIGN_AUTO,
                           bn, (wl, ofl, osign, 0), want, f"heavy{seed}")
            # int64 values take the two-call path
            run_both_picks(fx, h, fx.src_int(dev(v), fx.I64, sd), n, wl, fx.SIGN_AUTO, bn,
                           (wl, ofl, osign, 0), want, f"heavy{seed}-i64")
    assert above >= 2
    check_flags(fx, h)


def test_qlayer_host_checks(fx, h):
    import ctypes as C
    import torch
    x = dev(np.ones(64, np.float32))
    src = fx.src_f32(x)
    out = fmt_new()
    codes = empty((80,), torch.int8)
    L = fx.lib()
    args = lambda wl, ct, c, a: (h.value, C.byref(src), 64, wl, fx.SIGN_AUTO, FL_LO, FL_HI,
                                 out.data_ptr(), c, ct, a)
    assert L.fxpq_qlayer(*args(8, fx.C8, codes.data_ptr(), None)) == fx.ERR_INVALID_ARG
    assert L.fxpq_qlayer(*args(8, fx.I8, codes.data_ptr(), codes.data_ptr())) == fx.ERR_INVALID_ARG
    assert L.fxpq_qlayer(*args(9, fx.C8, codes.data_ptr(), codes.data_ptr())) == fx.ERR_INVALID_ARG
    assert L.fxpq_qlayer(*args(0, fx.C8, codes.data_ptr(), codes.data_ptr())) == fx.ERR_INVALID_ARG
    assert L.fxpq_qlayer(*args(8, fx.C8, codes.data_ptr() + 1, codes.data_ptr())) == fx.ERR_INVALID_ARG
    check_flags(fx, h)


def run_predicted(fx, h, src, n, wl, mm_exact, want_fmt, want_codes, bnosat, tag):
    """fxpq_qlayer_predicted: no prediction (NaN) -> a miss leaving the exact
    min / max; the previous call's min / max and format -> a hit equal to the
    oracle (or a miss when the window alone cannot decide); the other window
    candidate's format -> a miss.  Nothing is written past n."""
    import torch
    b0 = max(FL_LO, bnosat)
    osign = want_fmt[2]
    mm = torch.full((2,), float("nan"), dtype=torch.float64, device=DEV)
    miss = torch.zeros(1, dtype=torch.int32, device=DEV)
    codes = torch.full((n + 16,), 0x55, dtype=torch.int8, device=DEV)
    note("qlayer predicted", tag, n, wl, "no prediction")
    fx.qlayer_predicted(h, src, n, wl, fx.SIGN_AUTO, FL_LO, FL_HI, fmt_dev(*want_fmt[:3]), codes,
                        fx.C8, mm, miss)
    assert int(host(miss)[0]) == 1 and tuple(host(mm)) == mm_exact, tag
    out = fmt_dev(*want_fmt[:3])
    miss.zero_()
    note("qlayer predicted", tag, n, wl, "steady state")
    fx.qlayer_predicted(h, src, n, wl, fx.SIGN_AUTO, FL_LO, FL_HI, out, codes, fx.C8, mm, miss)
    hit = int(host(miss)[0]) == 0
    got = host(codes)
    assert np.all(got[n:] == 0x55), "wrote past n"
    if hit:
        assert want_fmt[1] in (b0, b0 + 1), tag
        assert fmt_host(out) == want_fmt, tag
        assert np.array_equal(decode8(got[:n], osign == 0), want_codes), tag
    assert tuple(host(mm)) == mm_exact, tag
    if want_fmt[1] in (b0, b0 + 1) and b0 + 1 <= FL_HI:
        other = b0 + 1 if want_fmt[1] == b0 else b0
        miss.zero_()
        fx.qlayer_predicted(h, src, n, wl, fx.SIGN_AUTO, FL_LO, FL_HI, fmt_dev(wl, other, osign),
                            codes, fx.C8, mm, miss)
        assert int(host(miss)[0]) == 1, tag
    return hit


def test_qlayer_predicted(fx, h, orc):
    """The predicted FxP-QLayer over fp32, eltwise-sum and C-Block sources
    against the oracle."""
    from test_gpu_kernels import CONV_CASES, gpu_conv_case
    hits = 0
    for name, x in [("normal", synth.normal(91, "qp", (100_003,), std=1.0)),
                    ("relu", np.maximum(synth.normal(92, "qpr", (4099,), std=2.0), 0))]:
        x = np.asarray(x, np.float32)
        for wl in (8, 5):
            ofl, osign, _ = orc.fl_search_f32(x, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            bn = beta_nosat([F(float(v)) for v in (x.min(), x.max())], wl, osign)
            hits += run_predicted(fx, h, fx.src_f32(dev(x)), x.size, wl,
                                  (float(x.min()), float(x.max())), (wl, ofl, osign, 0),
                                  orc.quantize_f32(x, wl, ofl, osign), bn, f"f32-{name}")
    n = 100_003
    a = synth.integers(93, "a", (n,), -128, 127)
    b = synth.integers(93, "b", (n,), 0, 255)
    ad, bd = dev(a.astype(np.int8)), dev((b - 128).astype(np.int8))
    for relu in (True, False):
        for m in (n, 16 * 1000 + 7):
            src = fx.src_add(ad, fx.C8, fmt_dev(8, 3, 1), bd, fx.C8, fmt_dev(8, 6, 0), relu)
            v, s = orc.eltwise_add(a[:m], 3, b[:m], 6, relu)
            for wl in (8, 5):
                ofl, osign, _ = orc.fl_search_i64(v, s, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
                bn = beta_nosat([fr(v.min(), s), fr(v.max(), s)], wl, osign)
                hits += run_predicted(fx, h, src, m, wl, (float(v.min()), float(v.max())),
                                      (wl, ofl, osign, 0), orc.quantize_i64(v, s, wl, ofl, osign), bn,
                                      f"add-relu{int(relu)}-{m}")
    acc, ep, mm, v, s_out, keep = gpu_conv_case(fx, h, orc, *CONV_CASES[0], seed=94)
    vn = v.transpose(0, 2, 3, 1).ravel()[:acc.numel()]
    for wl in (8, 6):
        ofl, osign, _ = orc.fl_search_i64(vn, s_out, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
        bn = beta_nosat([fr(vn.min(), s_out), fr(vn.max(), s_out)], wl, osign)
        hits += run_predicted(fx, h, fx.src_acc(acc, ep), acc.numel(), wl,
                              (float(vn.min()), float(vn.max())), (wl, ofl, osign, 0),
                              orc.quantize_i64(vn, s_out, wl, ofl, osign), bn, "acc")
    assert hits >= 8, hits
    check_flags(fx, h)


# Eltwise sums of the forms the predicted FxP-QLayer takes in packed 16-bit
# integer arithmetic (both shifts <= 5, 8-bit codes, 8-bit or narrower
# outputs), at both edges of each condition, and forms just outside them:
# (fl_a, a unsigned, fl_b, b unsigned, code range of a, code range of b, wl).
PACKED_FORMS = [
    (3, 0, 3, 0, (-125, 125), (-125, 125), 8),   # sigma - b0 = 1: bound at sigma + 1
    (4, 0, 4, 1, (-128, 127), (0, 255), 8),      # sigma - b0 = 2 (1 with ReLU): bound at sigma
    (8, 0, 3, 1, (-128, 127), (0, 255), 8),      # a shifted by 5: |W| up to 8415
    (2, 1, 7, 0, (0, 255), (-128, 127), 4),      # b shifted by 5, 4-bit output
    (0, 1, 0, 1, (0, 255), (0, 255), 8),         # both unsigned: non-negative sums
    (9, 0, 3, 0, (-128, 127), (-128, 127), 8),   # shift 6: the fp64 form
    (3, 0, 3, 0, (-60, 60), (-60, 60), 8),       # sigma - b0 = 0 (-1 with ReLU): exact codes
    (3, 0, 3, 1, (-100, 100), (0, 120), 8),      # signed + unsigned, sigma - b0 = 0
    (5, 0, 5, 0, (-3, 3), (-3, 3), 8),           # values far below the scale: sigma - b0 = -4
]


@pytest.mark.parametrize("form", PACKED_FORMS, ids=lambda f: f"fl{f[0]}u{f[1]}-fl{f[2]}u{f[3]}-wl{f[6]}")
def test_qlayer_predicted_eltwise_forms(fx, h, orc, form):
    """The predicted FxP-QLayer over eltwise sums of every form the packed
    16-bit path covers, and of forms beside them, equal to the oracle: codes,
    format, min / max, with and without ReLU, whole packets and a ragged
    tail."""
    fla, ua, flb, ub, ra, rb, wl = form
    n = 40_000 + 9
    a = synth.integers(95, f"pa{fla}{ua}", (n,), *ra)
    b = synth.integers(95, f"pb{flb}{ub}", (n,), *rb)
    ad = dev((a - 128 * ua).astype(np.int8))
    bd = dev((b - 128 * ub).astype(np.int8))
    hits = cases = 0
    for relu in (True, False):
        for m in (n, 16 * 500):
            src = fx.src_add(ad, fx.C8, fmt_dev(8, fla, 1 - ua), bd, fx.C8, fmt_dev(8, flb, 1 - ub),
                             relu)
            v, s = orc.eltwise_add(a[:m], fla, b[:m], flb, relu)
            ofl, osign, _ = orc.fl_search_i64(v, s, wl, fx.SIGN_AUTO, FL_LO, FL_HI)
            bn = beta_nosat([fr(v.min(), s), fr(v.max(), s)], wl, osign)
            hits += run_predicted(fx, h, src, m, wl, (float(v.min()), float(v.max())),
                                  (wl, ofl, osign, 0), orc.quantize_i64(v, s, wl, ofl, osign), bn,
                                  f"add-{form}-relu{int(relu)}-{m}")
            cases += 1
    assert hits >= cases // 2, (hits, cases)
    check_flags(fx, h)

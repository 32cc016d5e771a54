"""Parity of the fused C-Block + FxP-QLayer call (fxpq_cblock) with the CPU
oracle, and with the unfused sequence qconv -> fl_search -> requant.

Bit-exact: the chosen format, every code, the min / max of the C-Block
values.  Cases span several tiles with ragged row and channel tails, both tile
shapes (k <= 64 and k > 64), strided and padded windows, signed and unsigned
inputs, and the search's decision paths: the window pass alone, all values
tiny (fl_hi taken before any data is read), a word length above 16 (the exact
general pass over every candidate, which needs the stored accumulators), and
an outlier channel whose best fl lies above the window (the general pass over
the remaining candidates).
"""
from fractions import Fraction

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


def beta_nosat(v, s, wl, sign):
    """Largest fl in [FL_LO, FL_HI] at which every exact value v * 2^-s stays
    within [Qmin - 1/2, Qmax + 1/2] after scaling by 2^fl (Eq. 10-12), else
    FL_LO - 1; rational arithmetic."""
    qmax = (1 << (wl - sign)) - 1
    qmin = -(1 << (wl - 1)) if sign else 0
    mx, mn = int(v.max()), int(v.min())
    for b in range(FL_HI, FL_LO - 1, -1):
        t = Fraction(2) ** (b - s)
        if mx * t <= qmax + Fraction(1, 2) and mn * t >= qmin - Fraction(1, 2):
            return b
    return FL_LO - 1


class Case:
    """Seeded conv + epilogue operands (host), uploaded on demand."""

    def __init__(self, N, Cin, H, W, K, R, stride, pad, in_signed, relu, seed,
                 kind="normal", fl_scale=15, fl_in=5, fl_w=9):
        self.N, self.Cin, self.H, self.W = N, Cin, H, W
        self.K, self.R, self.stride, self.pad = K, R, stride, pad
        self.in_signed = in_signed
        lo, hi = (-128, 127) if in_signed else (0, 255)
        self.xc = synth.integers(seed, "cb-x", (N, Cin, H, W), lo, hi)
        self.wc = synth.integers(seed, "cb-w", (K, Cin, R, R), -128, 127)
        self.fl_in, self.fl_w, self.fl_b, self.fl_a1, self.fl_a2 = fl_in, fl_w, 11, fl_scale, fl_scale
        g = synth.rng_for(seed, "cb-epi")
        self.bias = g.integers(-2 ** 18, 2 ** 18, K).astype(np.int32)
        self.a1 = g.integers(2 ** 13, 2 ** 15, K).astype(np.int32)
        self.a2 = g.integers(-2 ** 13, 2 ** 13, K).astype(np.int32)
        if kind == "outlier":
            # small signed codes everywhere but one pixel, whose codes follow
            # the signs of filter 77: one value far above all others
            assert in_signed and R == 1 and K > 77
            self.xc = synth.integers(seed, "cb-x-small", (N, Cin, H, W), -20, 20)
            self.xc[N - 1, :, H // 2, W // 3] = np.where(self.wc[77, :, 0, 0] >= 0, 127, -128)
            self.bias, self.a2 = None, None
            self.a1 = np.full(K, 1 << 14, np.int32)
        self.relu = relu
        self.Ho = (H + 2 * pad - R) // stride + 1
        self.Wo = (W + 2 * pad - R) // stride + 1
        self.n = N * self.Ho * self.Wo * K

    def upload(self, fx, h):
        import torch
        N, Cin, H, W, K, R = self.N, self.Cin, self.H, self.W, self.K, self.R
        in_signed, relu = self.in_signed, self.relu
        x_nhwc = np.transpose(self.xc, (0, 2, 3, 1))
        w_krsc = np.transpose(self.wc, (0, 2, 3, 1)).reshape(K, -1)
        cin_dev = Cin
        if Cin == 3:  # padded RGB: a zero fourth channel, filter rows padded to 64 bytes
            x_nhwc = np.concatenate([x_nhwc, np.zeros(x_nhwc.shape[:3] + (1,), np.int64)], axis=3)
            w4 = np.concatenate([np.transpose(self.wc, (0, 2, 3, 1)), np.zeros((K, R, R, 1), np.int64)],
                                axis=3).reshape(K, -1)
            kp = (w4.shape[1] + 63) // 64 * 64
            w_krsc = np.concatenate([w4, np.zeros((K, kp - w4.shape[1]), np.int64)], axis=1)
            cin_dev = 4
        x_nhwc = x_nhwc - (0 if in_signed else 128)
        self.xd = dev(x_nhwc.astype(np.int8))
        self.wd = dev(w_krsc.astype(np.int8))
        self.x_type = fx.I8 if in_signed else fx.U8OFF
        self.colsum = empty((K,), torch.int32)
        fx.weight_colsum(h, self.wd, K, w_krsc.shape[1], self.colsum)
        self.fin = fmt_dev(8, self.fl_in, 1 if in_signed else 0)
        self.bd, self.a1d, self.a2d = (None if t is None else dev(t) for t in (self.bias, self.a1, self.a2))
        self.ep = fx.epilogue(K, self.fl_w, self.fin, bias=self.bd, fl_bias=self.fl_b, relu=relu,
                              scale=self.a1d, fl_scale=self.fl_a1, shift=self.a2d,
                              fl_shift=self.fl_a2)
        self.desc = fx.conv_desc(N, H, W, cin_dev, K, R, R, self.stride, self.pad)
        return self

    def oracle_values(self, orc):
        acc = orc.conv2d(self.xc, self.wc, self.stride, self.pad)
        v, s = orc.epilogue(acc, self.fl_in + self.fl_w, self.bias, self.fl_b, self.a1,
                            self.fl_a1, self.a2, self.fl_a2, self.relu)
        return v.transpose(0, 2, 3, 1).ravel(), s  # NHWC order

    def fused(self, fx, h, wl, sign=None):
        import torch
        sign = fx.SIGN_AUTO if sign is None else sign
        out = fmt_new()
        y = torch.full((self.n,), 99, dtype=torch.int8, device=DEV)
        acc = empty((self.n,), torch.int32)
        mm = torch.zeros(2, dtype=torch.float64, device=DEV)
        fx.cblock(h, self.desc, self.xd, self.x_type, self.wd, self.colsum, self.ep, wl, sign,
                  FL_LO, FL_HI, out, y, fx.C8, acc, mm)
        return fmt_host(out), host(y), host(mm)

    def predicted(self, fx, h, wl, mm, out, miss):
        """fxpq_cblock_predicted with the prediction in mm and out (device)."""
        import torch
        y = torch.full((self.n,), 99, dtype=torch.int8, device=DEV)
        fx.cblock_predicted(h, self.desc, self.xd, self.x_type, self.wd, self.colsum, self.ep, wl,
                            fx.SIGN_AUTO, FL_LO, FL_HI, out, y, fx.C8, mm, miss)
        return y

    def unfused(self, fx, h, wl, sign=None):
        import torch
        sign = fx.SIGN_AUTO if sign is None else sign
        acc = empty((self.n,), torch.int32)
        mm = torch.zeros(2, dtype=torch.float64, device=DEV)
        fx.qconv(h, self.desc, self.xd, self.x_type, self.wd, self.colsum, self.ep, acc, mm)
        src = fx.src_acc(acc, self.ep, mm)
        out = fmt_new()
        fx.fl_search(h, src, self.n, wl, sign, FL_LO, FL_HI, out)
        y = empty((self.n,), torch.int8)
        fx.requant(h, src, self.n, out, y, fx.C8)
        return fmt_host(out), host(y), host(mm)


CASES = [
    # N, Cin, H, W, K, R, stride, pad, signed input, relu
    (2, 64, 13, 11, 256, 1, 1, 0, False, False),   # 1x1 expand, ragged rows (286)
    (3, 64, 9, 9, 192, 1, 2, 0, False, False),     # strided 1x1 (projection shortcut)
    (2, 64, 17, 15, 64, 1, 1, 0, True, True),      # k <= 64 tiles, signed input, ReLU
    (2, 32, 10, 10, 40, 3, 1, 1, False, True),     # 3x3, ragged channels (k = 40)
    (1, 128, 7, 7, 512, 1, 1, 0, False, False),    # wide output, one row tile
    (300, 16, 1, 1, 96, 1, 1, 0, True, False),     # FC-like rows
]
# the predicted C-Block also takes a first conv over padded RGB (signed and
# unsigned input codes, 7x7 stride 2, ragged rows)
PRED_CASES = CASES + [
    (2, 3, 23, 21, 64, 7, 2, 3, True, True),
    (1, 3, 19, 17, 64, 7, 2, 3, False, False),
    # ReLU (a non-negative window) over 128 x 128 tiles
    (2, 64, 13, 11, 128, 1, 1, 0, True, True),
]


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_cblock_matches_oracle_and_unfused(fx, h, orc, case):
    c = Case(*case, seed=31 + CASES.index(case)).upload(fx, h)
    v, s = c.oracle_values(orc)
    for wl in (8, 6, 4):
        note("cblock", case, wl)
        (gwl, gfl, gsg, gst), y, mm = c.fused(fx, h, wl)
        ofl, osg, _ = orc.fl_search_i64(v, s, wl, orc.SIGN_AUTO, FL_LO, FL_HI)
        assert (gwl, gfl, gsg, gst) == (wl, ofl, osg, 0)
        assert mm[0] == v.min() and mm[1] == v.max()
        assert np.array_equal(decode8(y, osg == 0), orc.quantize_i64(v, s, wl, ofl, osg))
        ufmt, uy, umm = c.unfused(fx, h, wl)
        assert ufmt == (gwl, gfl, gsg, gst) and np.array_equal(uy, y) and np.array_equal(umm, mm)
    assert fx.sync_status(h) == 0


def test_cblock_forced_sign_and_tiny_values(fx, h, orc):
    # forced unsigned format on signed values (negative values clip to 0)
    c = Case(2, 64, 9, 9, 128, 1, 1, 0, True, False, seed=41).upload(fx, h)
    v, s = c.oracle_values(orc)
    assert v.min() < 0
    note("cblock forced sign")
    (gwl, gfl, gsg, gst), y, _ = c.fused(fx, h, 8, sign=0)
    ofl, osg, _ = orc.fl_search_i64(v, s, 8, 0, FL_LO, FL_HI)
    assert (gfl, gsg, gst) == (ofl, 0, 0)
    assert np.array_equal(decode8(y, True), orc.quantize_i64(v, s, 8, ofl, 0))
    # every value below 2^-9: no value saturates even at fl_hi
    t = Case(1, 64, 8, 8, 128, 1, 1, 0, False, False, seed=42, fl_scale=48).upload(fx, h)
    v, s = t.oracle_values(orc)
    assert beta_nosat(v, s, 8, 1) >= FL_HI
    note("cblock tiny values")
    (gwl, gfl, gsg, gst), y, _ = t.fused(fx, h, 8)
    ofl, osg, _ = orc.fl_search_i64(v, s, 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert (gfl, gsg, gst) == (ofl, osg, 0) == (FL_HI, osg, 0)
    assert np.array_equal(decode8(y, osg == 0), orc.quantize_i64(v, s, 8, ofl, osg))
    assert fx.sync_status(h) == 0


def test_cblock_general_pass_paths(fx, h, orc):
    # one outlier value: at 6 bits the best fl clips it and lies above the
    # two-candidate window that starts at the largest non-saturating fl
    c = Case(4, 64, 20, 20, 128, 1, 1, 0, True, False, seed=48, kind="outlier").upload(fx, h)
    v, s = c.oracle_values(orc)
    for wl in (6, 8):
        ofl, osg, _ = orc.fl_search_i64(v, s, wl, orc.SIGN_AUTO, FL_LO, FL_HI)
        if wl == 6:
            assert ofl > beta_nosat(v, s, wl, osg) + 1, "case must need the general pass"
        note("cblock outlier value", wl)
        (gwl, gfl, gsg, gst), y, _ = c.fused(fx, h, wl)
        assert (gfl, gsg, gst) == (ofl, osg, 0)
        assert np.array_equal(decode8(y, osg == 0), orc.quantize_i64(v, s, wl, ofl, osg))
    # word length above 16: every candidate in the general pass (codes do not
    # fit 8 bits, so only the format is compared and the code flag is expected)
    note("cblock wl 20")
    c2 = Case(2, 64, 9, 9, 128, 1, 1, 0, False, True, seed=44).upload(fx, h)
    v, s = c2.oracle_values(orc)
    (gwl, gfl, gsg, gst), _, _ = c2.fused(fx, h, 20)
    ofl, osg, _ = orc.fl_search_i64(v, s, 20, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert (gwl, gfl, gsg, gst) == (20, ofl, osg, 0)
    assert fx.sync_status(h) == fx.FLAG_CODE


def test_cblock_back_to_back_shapes(fx, h, orc):
    # scratch reuse: a large call, then a smaller one
    big = Case(4, 64, 20, 20, 256, 1, 1, 0, False, False, seed=45).upload(fx, h)
    small = Case(1, 64, 5, 5, 64, 1, 1, 0, False, True, seed=46).upload(fx, h)
    for c in (big, small, big):
        v, s = c.oracle_values(orc)
        note("cblock back-to-back", c.n)
        (gwl, gfl, gsg, gst), y, _ = c.fused(fx, h, 8)
        ofl, osg, _ = orc.fl_search_i64(v, s, 8, orc.SIGN_AUTO, FL_LO, FL_HI)
        assert (gfl, gsg, gst) == (ofl, osg, 0)
        assert np.array_equal(decode8(y, osg == 0), orc.quantize_i64(v, s, 8, ofl, osg))
    assert fx.sync_status(h) == 0


def test_cblock_rejects_unsupported(fx, h):
    import torch
    c = Case(1, 64, 4, 4, 64, 1, 1, 0, False, False, seed=47).upload(fx, h)
    y = empty((c.n,), torch.int8)
    acc = empty((c.n,), torch.int32)
    mm = torch.zeros(2, dtype=torch.float64, device=DEV)
    out = fmt_new()
    with pytest.raises(fx.FxpqError):
        fx.cblock(h, c.desc, c.xd, c.x_type, c.wd, c.colsum, c.ep, 8, fx.SIGN_AUTO, FL_LO, FL_HI,
                  out, y, fx.I16, acc, mm)
    rgb = fx.conv_desc(1, 8, 8, 4, 64, 3, 3, 1, 1)
    with pytest.raises(fx.FxpqError):
        fx.cblock(h, rgb, c.xd, c.x_type, c.wd, c.colsum, c.ep, 8, fx.SIGN_AUTO, FL_LO, FL_HI,
                  out, y, fx.C8, acc, mm)


@pytest.mark.parametrize("case", PRED_CASES, ids=[str(i) for i in range(len(PRED_CASES))])
def test_cblock_predicted_deferred(fx, h, orc, case):
    """Deferred decisions (fxpq_predicted_defer / fxpq_predicted_decide):
    several predicted calls, then one decision launch.  No prediction: a
    miss; the oracle's format and min / max: a hit with the oracle's codes
    (or a miss when the window cannot decide); the other window candidate's
    format, or a format outside the window (which the standard decision
    would have replaced, but the calls after it already used): a miss.
    Every call's min / max ends exact."""
    import torch
    c = Case(*case, seed=71 + PRED_CASES.index(case)).upload(fx, h)
    v, s = c.oracle_values(orc)
    exact = (float(v.min()), float(v.max()))
    fx.predicted_defer(h, 1)
    try:
        for wl in (8, 5):
            note("cblock predicted deferred", case, wl)
            ofl, osg, _ = orc.fl_search_i64(v, s, wl, orc.SIGN_AUTO, FL_LO, FL_HI)
            b0 = max(FL_LO, beta_nosat(v, s, wl, osg))
            calls = [("none", float("nan"), float("nan"), ofl), ("steady", *exact, ofl)]
            if ofl in (b0, b0 + 1) and b0 + 1 <= FL_HI:
                calls.append(("other", *exact, b0 + 1 if ofl == b0 else b0))
            if ofl == b0 and b0 - 1 >= FL_LO:
                calls.append(("outside", *exact, b0 - 1))
            pend = []
            for kind, lo, hi, fl in calls:
                mm = torch.tensor([lo, hi], dtype=torch.float64, device=DEV)
                miss = torch.zeros(1, dtype=torch.int32, device=DEV)
                out = fmt_dev(wl, fl, osg)
                pend.append((kind, fl, mm, miss, out, c.predicted(fx, h, wl, mm, out, miss)))
            fx.predicted_decide(h)
            steady = int(host(pend[1][3])[0])  # 2: the window alone cannot decide
            assert steady in (0, 2), steady
            for kind, fl, mm, miss, out, y in pend:
                m = int(host(miss)[0])
                assert tuple(host(mm)) == exact, kind
                if kind == "steady":
                    if m == 0:
                        assert fmt_host(out) == (wl, ofl, osg, 0)
                        assert np.array_equal(decode8(host(y), osg == 0),
                                              orc.quantize_i64(v, s, wl, ofl, osg))
                else:
                    want = 1 if kind == "none" or steady == 0 else 2
                    assert m == want, (kind, m)
                    assert fmt_host(out) == (wl, fl, osg, 0), kind  # left as the calls used it
    finally:
        fx.predicted_defer(h, 0)
    assert fx.sync_status(h) == 0


@pytest.mark.parametrize("case", PRED_CASES, ids=[str(i) for i in range(len(PRED_CASES))])
def test_cblock_predicted(fx, h, orc, case):
    """The predicted C-Block: with no prediction (NaN min / max) a miss that
    still leaves the exact min / max; with the previous call's min / max and
    format (here: the oracle's) a hit whose format and codes equal the
    oracle's, or a miss when the window cannot decide alone; with the other
    window candidate's format, or a min / max from other data, a miss."""
    import torch
    c = Case(*case, seed=51 + PRED_CASES.index(case)).upload(fx, h)
    v, s = c.oracle_values(orc)
    hits = 0
    for wl in (8, 6, 4):
        note("cblock predicted", case, wl)
        ofl, osg, _ = orc.fl_search_i64(v, s, wl, orc.SIGN_AUTO, FL_LO, FL_HI)
        b0 = max(FL_LO, beta_nosat(v, s, wl, osg))
        mm = torch.full((2,), float("nan"), dtype=torch.float64, device=DEV)
        miss = torch.zeros(1, dtype=torch.int32, device=DEV)
        c.predicted(fx, h, wl, mm, fmt_dev(wl, ofl, osg), miss)
        assert int(host(miss)[0]) == 1
        assert tuple(host(mm)) == (float(v.min()), float(v.max()))
        # the steady state: the previous call's min / max and format
        out = fmt_dev(wl, ofl, osg)
        miss.zero_()
        y = c.predicted(fx, h, wl, mm, out, miss)
        if int(host(miss)[0]) == 0:
            hits += 1
            assert ofl in (b0, b0 + 1)
            assert fmt_host(out) == (wl, ofl, osg, 0)
            assert np.array_equal(decode8(host(y), osg == 0), orc.quantize_i64(v, s, wl, ofl, osg))
        assert tuple(host(mm)) == (float(v.min()), float(v.max()))
        if ofl in (b0, b0 + 1) and b0 + 1 <= FL_HI:
            # the other window candidate's codes written: never a hit
            other = b0 + 1 if ofl == b0 else b0
            miss.zero_()
            c.predicted(fx, h, wl, mm, fmt_dev(wl, other, osg), miss)
            assert int(host(miss)[0]) == 1
            assert tuple(host(mm)) == (float(v.min()), float(v.max()))
        # a min / max four times larger: another window, a miss
        miss.zero_()
        mm4 = torch.tensor([4.0 * v.min(), 4.0 * v.max()], dtype=torch.float64, device=DEV)
        c.predicted(fx, h, wl, mm4, fmt_dev(wl, ofl, osg), miss)
        if max(FL_LO, beta_nosat(4 * v, s, wl, osg)) != b0:
            assert int(host(miss)[0]) == 1
    assert hits >= 1, "no case decided by the window alone"
    assert fx.sync_status(h) == 0


def test_cblock_predicted_saturating(fx, h, orc):
    """A predicted window whose first candidate saturates (no fractional
    length in [FL_LO, FL_HI] keeps the values unclipped; coarse input and
    weight scales, one pixel aligned with filter 77's signs): values reach
    2^30 at the first candidate's step.  With the exact min / max and the
    oracle's format as the prediction, a hit gives the oracle's format and
    codes; the min / max end exact."""
    import torch
    c = Case(1, 512, 6, 6, 128, 1, 1, 0, True, False, seed=91, kind="outlier", fl_scale=14,
             fl_in=-8, fl_w=-8).upload(fx, h)
    v, s = c.oracle_values(orc)
    exact = (float(v.min()), float(v.max()))
    assert max(abs(exact[0]), abs(exact[1])) * 2.0 ** (FL_LO - s) >= 2 ** 29
    hits = 0
    for wl in (8, 6):
        note("cblock predicted saturating", wl)
        ofl, osg, _ = orc.fl_search_i64(v, s, wl, orc.SIGN_AUTO, FL_LO, FL_HI)
        assert beta_nosat(v, s, wl, osg) < FL_LO
        mm = torch.tensor(list(exact), dtype=torch.float64, device=DEV)
        miss = torch.zeros(1, dtype=torch.int32, device=DEV)
        out = fmt_dev(wl, ofl, osg)
        y = c.predicted(fx, h, wl, mm, out, miss)
        m = int(host(miss)[0])
        assert m in (0, 2), m
        if m == 0:
            hits += 1
            assert fmt_host(out) == (wl, ofl, osg, 0)
            assert np.array_equal(decode8(host(y), osg == 0), orc.quantize_i64(v, s, wl, ofl, osg))
        assert tuple(host(mm)) == exact
    assert hits >= 1
    assert fx.sync_status(h) == 0

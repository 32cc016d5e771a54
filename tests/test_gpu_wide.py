"""Wide C-Blocks (codes of up to 32 bits, Sec. "Integer-Only Inference" with
the 32-bit first / last layers of Sec. "Initial Design Generation") on the
GPU against the oracle's exact integer convolution and epilogue.

Bit-exact: the int64 C-Block values and their scale; then the FxP-QLayer
over them (fl search and requantization of an int64 source) against the
oracle's.  Codes are drawn over the whole range of each format with both
extremes planted; shapes cover 3x3 / 1x1 / 7x7 filters, strides 1 and 2,
ragged output channels, the padded RGB first layer and an FC layer."""
import numpy as np
import pytest

import synth
from gpu_util import DEV, dev, empty, fmt_dev, fmt_host, fmt_new, host, note

pytestmark = pytest.mark.gpu


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


def code_range(wl, sign):
    return (-(1 << (wl - 1)), (1 << (wl - 1)) - 1) if sign else (0, (1 << wl) - 1)


def draw(seed, name, shape, wl, sign):
    lo, hi = code_range(wl, sign)
    if wl == 1 and sign:
        c = np.where(synth.integers(seed, name, shape, 0, 1) == 0, -1, 1)
    else:
        c = synth.integers(seed, name, shape, lo, hi)
        flat = c.reshape(-1)
        flat[:: 7] = lo
        flat[3:: 11] = hi
    return c.astype(np.int64)


# N, C, H, W, K, R, stride, pad, (wl_x, S_x), (wl_w, S_w), relu, bias, scale
CASES = [
    (2, 16, 9, 11, 40, 3, 1, 1, (16, 1), (16, 1), True, True, False),
    (2, 32, 8, 8, 64, 1, 2, 0, (12, 0), (10, 1), False, False, True),
    (1, 16, 6, 7, 24, 3, 1, 1, (32, 1), (8, 1), False, True, False),
    (1, 3, 21, 19, 64, 7, 2, 3, (16, 1), (16, 1), True, False, True),
    (3, 512, 1, 1, 1000, 1, 1, 0, (16, 0), (16, 1), False, True, False),
    (2, 16, 8, 8, 32, 3, 1, 1, (16, 1), (1, 1), True, False, True),
    (1, 32, 5, 5, 48, 3, 1, 1, (24, 1), (24, 1), False, True, False),
    (1, 16, 6, 6, 16, 3, 1, 1, (31, 0), (15, 0), False, False, False),
    # unsigned 32-bit codes (uint32 storage): input, then weights
    (1, 16, 6, 6, 16, 3, 1, 1, (32, 0), (16, 1), True, False, False),
    (2, 16, 5, 5, 8, 1, 1, 0, (8, 1), (32, 0), False, True, False),
]


def run_case(fx, h, orc, case, seed):
    import torch
    N, Cin, H, W, K, R, stride, pad, (wx, sx), (ww, sw), relu, with_bias, with_scale = case
    xc = draw(seed, "wx", (N, Cin, H, W), wx, sx)
    wc = draw(seed, "ww", (K, Cin, R, R), ww, sw)
    x_nhwc = np.transpose(xc, (0, 2, 3, 1))
    w_krsc = np.transpose(wc, (0, 2, 3, 1)).reshape(K, -1)
    cin = Cin
    if Cin == 3:  # padded RGB: a zero fourth channel, filter rows padded to 64
        x_nhwc = np.concatenate([x_nhwc, np.zeros(x_nhwc.shape[:3] + (1,), np.int64)], axis=3)
        w4 = np.concatenate([np.transpose(wc, (0, 2, 3, 1)), np.zeros((K, R, R, 1), np.int64)], axis=3)
        w_krsc = w4.reshape(K, -1)
        kp = (w_krsc.shape[1] + 63) // 64 * 64
        w_krsc = np.concatenate([w_krsc, np.zeros((K, kp - w_krsc.shape[1]), np.int64)], axis=1)
        cin = 4
    g = synth.rng_for(seed, "wepi")
    fl_x, fl_w, fl_b, fl_a1, fl_a2 = 9, 13, 20, 14, 25
    bias = g.integers(-2 ** 30, 2 ** 30, K).astype(np.int32) if with_bias else None
    a1 = g.integers(-2 ** 15, 2 ** 15, K).astype(np.int32) if with_scale else None
    a2 = g.integers(-2 ** 31, 2 ** 31 - 1, K).astype(np.int32) if with_scale else None
    fin = fmt_dev(wx, fl_x, sx)
    keep = [dev(a) if a is not None else None for a in (bias, a1, a2)]
    ep = fx.epilogue(K, fl_w, fin, bias=keep[0], fl_bias=fl_b, relu=relu, scale=keep[1],
                     fl_scale=fl_a1, shift=keep[2], fl_shift=fl_a2)
    desc = fx.conv_desc(N, H, W, cin, K, R, R, stride, pad)
    nb = fx.qconv_wide_workspace(desc, wx, sx, ww, sw)
    ws = empty((nb,), torch.uint8)
    Ho = (H + 2 * pad - R) // stride + 1
    Wo = (W + 2 * pad - R) // stride + 1
    v = empty((N * Ho * Wo * K,), torch.int64)
    sc = empty((1,), torch.int32)
    note("qconv_wide", case, seed)
    fx.qconv_wide(h, desc, dev(x_nhwc.astype(np.int32)), wx, sx, dev(w_krsc.astype(np.int32)), ww, sw,
                  ep, v, sc, ws, nb)
    acc = orc.conv2d(xc, wc, stride, pad)
    want, s_out = orc.epilogue(acc, fl_x + fl_w, bias, fl_b, a1, fl_a1, a2, fl_a2, relu)
    want_nhwk = np.transpose(want, (0, 2, 3, 1)).reshape(-1)
    return v, sc, want_nhwk, s_out, keep


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_wide_cblock_values(fx, h, orc, case):
    v, sc, want, s_out, _ = run_case(fx, h, orc, case, seed=60 + CASES.index(case))
    assert int(host(sc)[0]) == s_out
    assert np.array_equal(host(v), want)
    assert fx.sync_status(h) == 0


@pytest.mark.parametrize("wx,sx,ww,sw,C,planes", [(32, 1, 32, 1, 32768, (4, 5)),
                                                  (24, 0, 16, 1, 45056, (3, 3))])
def test_wide_cblock_deep_unfused(fx, h, orc, wx, sx, ww, sw, C, planes):
    """A contraction too deep for the fused path (pairs of one shift x padded
    depth x 2^14 reaches 2^31): one int8 contraction per plane pair and the
    exact combination pass, against the oracle.  Codes kept small enough for
    the exact values to stay below 2^62."""
    import torch
    N, K = 2, 8
    px, pw = planes
    assert min(px, pw) * C >= 2 ** 17
    lo_x = -(2 ** 11) if sx else 0
    xc = synth.integers(61, "deep-x", (N, C, 1, 1), lo_x, 2 ** 11).astype(np.int64)
    wc = synth.integers(61, "deep-w", (K, C, 1, 1), -(2 ** 13), 2 ** 13).astype(np.int64)
    xc[:, 0] = (1 << wx) - 1 if not sx else -(1 << (wx - 1))  # every plane's extremes
    wc[:, 1] = (1 << (ww - 1)) - 1
    desc = fx.conv_desc(N, 1, 1, C, K, 1, 1, 1, 0)
    nb = fx.qconv_wide_workspace(desc, wx, sx, ww, sw)
    a = lambda b: (b + 255) // 256 * 256
    assert nb == px * a(N * C) + pw * a(K * C) + a(pw * K * 4) + px * pw * N * K * 4
    ws = empty((nb,), torch.uint8)
    v = empty((N * K,), torch.int64)
    sc = empty((1,), torch.int32)
    fin = fmt_dev(wx, 3, sx)
    ep = fx.epilogue(K, 2, fin, relu=False)
    note("qconv_wide deep unfused", wx, sx, ww, sw)
    fx.qconv_wide(h, desc, dev(xc.reshape(N, 1, 1, C).astype(np.int32)), wx, sx,
                  dev(wc.reshape(K, C).astype(np.int32)), ww, sw, ep, v, sc, ws, nb)
    acc = orc.conv2d(xc, wc, 1, 0)
    want, s_out = orc.epilogue(acc, 3 + 2)
    assert int(host(sc)[0]) == s_out
    assert np.array_equal(host(v), np.transpose(want, (0, 2, 3, 1)).reshape(-1))
    assert fx.sync_status(h) == 0


def test_wide_cblock_fxp_qlayer(fx, h, orc):
    """The FxP-QLayer over a wide C-Block: fl search (8 bits) and codes."""
    import torch
    case = CASES[3]
    v, sc, want, s_out, _ = run_case(fx, h, orc, case, seed=71)
    src = fx.src_int(v, fx.I64, sc)
    out = fmt_new()
    fx.fl_search(h, src, v.numel(), 8, fx.SIGN_AUTO, -8, 15, out)
    fl, sg, _ = orc.fl_search_i64(want, s_out, 8, fx.SIGN_AUTO, -8, 15)
    assert fmt_host(out) == (8, fl, sg, 0)
    codes = empty((v.numel(),), torch.int8)
    fx.requant(h, src, v.numel(), out, codes, fx.C8)
    stored = host(codes).astype(np.int64) + (0 if sg else 128)
    assert np.array_equal(stored, orc.quantize_i64(want, s_out, 8, fl, sg))
    assert fx.sync_status(h) == 0


def test_wide_cblock_out_of_range_raises_flag(fx, h):
    """Values of magnitude 2^62 or more are flagged (32-bit extremes)."""
    import torch
    N, C, K = 1, 16, 16
    x = np.full((N, 1, 1, C), -2 ** 31, np.int32)
    w = np.full((K, C), -2 ** 31, np.int32)
    desc = fx.conv_desc(N, 1, 1, C, K, 1, 1, 1, 0)
    ep = fx.epilogue(K, 0, fmt_dev(32, 0, 1))
    nb = fx.qconv_wide_workspace(desc, 32, 1, 32, 1)
    ws = empty((nb,), torch.uint8)
    v = empty((K,), torch.int64)
    sc = empty((1,), torch.int32)
    note("qconv_wide range flag")
    fx.qconv_wide(h, desc, dev(x), 32, 1, dev(w), 32, 1, ep, v, sc, ws, nb)
    assert fx.sync_status(h) & fx.FLAG_RANGE
    assert np.all(host(v) == 0)
    assert fx.sync_status(h) == 0
    # 16-bit codes (sums combined in int64): the bias alignment shifts the
    # accumulators past 2^62
    x16 = np.full((N, 1, 1, C), 2 ** 15 - 1, np.int32)
    w16 = np.full((K, C), 2 ** 15 - 1, np.int32)
    b = dev(np.ones(K, np.int32))
    ep = fx.epilogue(K, 0, fmt_dev(16, 0, 1), bias=b, fl_bias=40)
    nb = fx.qconv_wide_workspace(desc, 16, 1, 16, 1)
    ws = empty((nb,), torch.uint8)
    note("qconv_wide range flag int64")
    fx.qconv_wide(h, desc, dev(x16), 16, 1, dev(w16), 16, 1, ep, v, sc, ws, nb)
    assert fx.sync_status(h) & fx.FLAG_RANGE
    assert np.all(host(v) == 0)
    assert fx.sync_status(h) == 0


def test_accumulator_overflow_count(fx, h):
    """Counts of accumulators outside the two's-complement range of 2..32
    bits, with the boundary values planted, against the plain count."""
    import torch
    g = synth.rng_for(72, "ovf")
    a = (g.standard_normal(100_003) * 2 ** 15).astype(np.int64)
    a[:8] = [2 ** 15 - 1, 2 ** 15, -2 ** 15, -2 ** 15 - 1, 2 ** 31 - 1, -2 ** 31, 0, -1]
    a = np.clip(a, -2 ** 31, 2 ** 31 - 1).astype(np.int32)
    ad = dev(a)
    for bits in (2, 8, 15, 16, 17, 31, 32):
        note("acc_overflow", bits)
        cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
        fx.acc_overflow(h, ad, a.size, bits, cnt)
        lo, hi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
        want = int(np.sum((a.astype(np.int64) < lo) | (a.astype(np.int64) > hi)))
        assert int(host(cnt)[0]) == want, bits
    # counts add up across calls
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    fx.acc_overflow(h, ad, a.size, 16, cnt)
    fx.acc_overflow(h, ad, a.size, 16, cnt)
    want16 = int(np.sum((a.astype(np.int64) < -2 ** 15) | (a.astype(np.int64) > 2 ** 15 - 1)))
    assert int(host(cnt)[0]) == 2 * want16
    assert fx.sync_status(h) == 0

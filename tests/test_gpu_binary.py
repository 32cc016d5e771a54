"""Signed 1-bit formats (Eq. 13) on the GPU against the oracle: codes (stored
decoded, -1 / +1), the exact fractional-length search over the Eq. 13 values,
requantization of C-Block values, the fused FxP-QLayer and the layer error.
Bit-exact codes and formats; error sums to 1e-9 relative."""
import numpy as np
import pytest

import synth
from gpu_util import DEV, dev, empty, fmt_dev, fmt_host, fmt_new, host, note

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


def decoded(codes, wl, sign):
    """The oracle's Eq. 13 codes (-1 / 0) as the values they stand for."""
    c = np.asarray(codes).astype(np.int64)
    return np.where(c == 0, 1, -1) if (wl == 1 and sign == 1) else c


def f32_cases():
    g = synth.rng_for(41, "bin")
    w = synth.normal(42, "bin-w", (65_537,), std=0.05)
    mixed = synth.normal(43, "bin-m", (10_001,), std=3.0)
    mixed[::97] = 0.0
    mixed[1::97] = -0.0
    tiny = synth.normal(44, "bin-t", (4099,), std=0.5)
    # below 2^-(fl_hi+24) (fractional scaled values), within the oracle's exact range
    tiny[::13] = (g.standard_normal(len(tiny[::13])) * 1e-6).astype(np.float32)
    return [("weights", w), ("mixed", mixed), ("tiny", tiny),
            ("neg", -np.abs(synth.normal(45, "bin-n", (1001,)))), ("relu", np.abs(w)),
            ("zeros", np.zeros(64, np.float32)), ("one", np.array([-0.4], np.float32))]


def test_quantize_binary_codes(fx, h, orc):
    import torch
    x = np.array([-2.0, -1e-20, -0.0, 0.0, 1e-20, 3.0] * 7 + [0.5], np.float32)
    for fl in (4, -2):
        for sign in (1, 0):
            note("quantize-1bit", fl, sign)
            codes = empty((x.size,), torch.int8)
            fx.quantize(h, dev(x), x.size, fmt_dev(1, fl, sign), codes, fx.I8)
            want = decoded(orc.quantize_f32(x, 1, fl, sign), 1, sign)
            assert np.array_equal(host(codes).astype(np.int64), want)
    assert fx.sync_status(h) == 0


def test_fl_search_binary_f32(fx, h, orc):
    import torch
    for name, x in f32_cases():
        x = np.asarray(x, np.float32)
        for sign in (fx.SIGN_AUTO, 1):
            note("fls-1bit-f32", name, sign)
            out = fmt_new()
            fx.fl_search(h, fx.src_f32(dev(x)), x.size, 1, sign, FL_LO, FL_HI, out)
            ofl, osign, osse = orc.fl_search_f32(x, 1, sign, FL_LO, FL_HI)
            assert fmt_host(out) == (1, ofl, osign, 0), (name, sign, osse)
            sse = torch.full((FL_HI - FL_LO + 1,), -1.0, dtype=torch.float64, device=DEV)
            fx.fl_search(h, fx.src_f32(dev(x)), x.size, 1, sign, FL_LO, FL_HI, fmt_new(), sse)
            np.testing.assert_allclose(host(sse), osse, rtol=1e-9)
    assert fx.sync_status(h) == 0


def test_binary_integer_sources_requant_and_qlayer(fx, h, orc):
    import torch
    from test_gpu_kernels import CONV_CASES, gpu_conv_case
    g = synth.rng_for(46, "bin-int")
    v = (g.standard_normal(70_001) * 2 ** 18).astype(np.int64)
    s = 12
    sd = torch.tensor([s], dtype=torch.int32, device=DEV)
    note("fls-1bit-int")
    out = fmt_new()
    fx.fl_search(h, fx.src_int(dev(v.astype(np.int32)), fx.I32, sd), v.size, 1, fx.SIGN_AUTO, FL_LO, FL_HI, out)
    ofl, osign, _ = orc.fl_search_i64(v, s, 1, fx.SIGN_AUTO, FL_LO, FL_HI)
    assert fmt_host(out) == (1, ofl, osign, 0)
    # C-Block values without ReLU (signed): search, requant, fused FxP-QLayer
    acc, ep, mm, vv, s_out, keep = gpu_conv_case(fx, h, orc, *CONV_CASES[1], seed=47)
    n = acc.numel()
    vn = vv.transpose(0, 2, 3, 1).ravel()[:n]
    src = fx.src_acc(acc, ep, mm)
    out = fmt_new()
    fx.fl_search(h, src, n, 1, fx.SIGN_AUTO, FL_LO, FL_HI, out)
    ofl, osign, _ = orc.fl_search_i64(vn, s_out, 1, fx.SIGN_AUTO, FL_LO, FL_HI)
    assert fmt_host(out) == (1, ofl, osign, 0) and osign == 1
    want = decoded(orc.quantize_i64(vn, s_out, 1, ofl, osign), 1, osign)
    codes = empty((n,), torch.int8)
    fx.requant(h, src, n, out, codes, fx.C8)
    assert np.array_equal(host(codes).astype(np.int64), want)
    out2 = fmt_new()
    codes2 = empty((n,), torch.int8)
    alt = empty((n,), torch.int8)
    fx.qlayer(h, src, n, 1, fx.SIGN_AUTO, FL_LO, FL_HI, out2, codes2, fx.C8, alt)
    assert fmt_host(out2) == (1, ofl, osign, 0)
    assert np.array_equal(host(codes2).astype(np.int64), want)
    # layer error of the decoded codes against the exact values
    ref = (vn.astype(np.float64) * 2.0 ** -s_out).astype(np.float32)
    e = empty((4,), torch.float64)
    fx.layer_error(h, dev(ref), codes, fx.C8, out, n, e)
    oe = orc.layer_error(ref, orc.quantize_i64(vn, s_out, 1, ofl, osign), 1, ofl, osign)
    np.testing.assert_allclose(host(e), oe, rtol=1e-9)
    assert fx.sync_status(h) == 0

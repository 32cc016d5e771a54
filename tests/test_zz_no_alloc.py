"""The FL search that allocates nothing (fxpq_fl_search_static, for callers
that cannot allocate) against the handle-based fxpq_fl_search on the same
inputs, through the C ABI: chosen formats identical, reported errors equal
to a relative 1e-12, and formats equal to the oracle's (bit-exact).  Three
calls in a row on the one static scratch of the device, the second smaller
than the first, then the first again: each starts from what the previous
call left behind."""
import numpy as np
import pytest

import synth
from gpu_util import DEV, dev, fmt_host, fmt_new, host, note

pytestmark = pytest.mark.gpu

FL_LO, FL_HI = -8, 15


@pytest.fixture(scope="module")
def fx():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2203_12091_amd import fxpq
    return fxpq


def test_static_search_matches_handle_search(fx):
    import torch

    import oracle
    oracle.lib()
    h = fx.Handle(0)
    stream = torch.cuda.Stream()
    fx.set_stream(h, stream)
    # A: fp32 with a lone outlier (its best fl lies above the window: the
    # exact general pass runs); B: a smaller int32 tensor at scale 2^-13,
    # every error reported
    big = synth.normal(41, "noalloc-big", (1_000_003,), std=0.1)
    big[777_777] = 60.0
    small = synth.integers(42, "noalloc-small", (4099,), -2 ** 20, 2 ** 20).astype(np.int32)
    cases = [("A fp32 outlier", dev(big), None, False), ("B int32 s=13", dev(small), 13, True),
             ("A again", dev(big), None, False)]
    for name, x, s, report in cases:
        note("fl_search_static", name, x.numel())
        if s is None:
            src = fx.src_f32(x)
        else:
            src = fx.src_int(x, fx.I32, torch.tensor([s], dtype=torch.int32, device=DEV))
        n = x.numel()
        sse_a = torch.full((FL_HI - FL_LO + 1,), -1.0, dtype=torch.float64, device=DEV) if report else None
        sse_b = torch.full((FL_HI - FL_LO + 1,), -2.0, dtype=torch.float64, device=DEV) if report else None
        out_a, out_b = fmt_new(), fmt_new()
        fx.fl_search_static(src, n, 8, fx.SIGN_AUTO, FL_LO, FL_HI, out_a, sse_a, stream)
        fx.fl_search(h, src, n, 8, fx.SIGN_AUTO, FL_LO, FL_HI, out_b, sse_b)
        stream.synchronize()
        got, want = fmt_host(out_a), fmt_host(out_b)
        assert got == want and got[3] == 0, (name, got, want)
        xs = host(x)
        if s is None:
            fl, sign, ref = oracle.fl_search_f32(xs, 8, oracle.SIGN_AUTO, FL_LO, FL_HI)
        else:
            fl, sign, ref = oracle.fl_search_i64(xs.astype(np.int64), s, 8, oracle.SIGN_AUTO, FL_LO, FL_HI)
        assert (got[1], got[2]) == (fl, sign), (name, got, fl, sign)
        if report:
            a, b = host(sse_a), host(sse_b)
            assert (a >= 0).all()
            np.testing.assert_allclose(a, b, rtol=1e-12, atol=0)
            np.testing.assert_allclose(a, ref, rtol=1e-9, atol=0)
    assert fx.sync_status(h) == 0
    h.close()


def test_static_search_rejects_bad_calls(fx):
    """Host checks come first and launch nothing; a null stream is the
    default stream."""
    import torch
    x = dev(synth.normal(43, "noalloc-rej", (1000,)))
    out = fmt_new()
    with pytest.raises(fx.FxpqError):
        fx.fl_search_static(fx.src_f32(x), 1000, 40, fx.SIGN_AUTO, FL_LO, FL_HI, out)
    with pytest.raises(fx.FxpqError):
        fx.fl_search_static(fx.src_f32(x), 0, 8, fx.SIGN_AUTO, FL_LO, FL_HI, out)
    fx.fl_search_static(fx.src_f32(x), 1000, 8, fx.SIGN_AUTO, FL_LO, FL_HI, out)
    torch.cuda.synchronize()
    assert fmt_host(out)[3] == 0

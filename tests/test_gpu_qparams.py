"""Algorithm 1 and the forward optimizer on the GPU against the oracle, and
the kernels they add (dequantization, fp32-vs-fp32 layer error, prediction
ties).

Bit-exact: every chosen format and the sequence of candidates evaluated.
The costs agree to a relative 1e-9 (fp64 sums in different orders)."""
import numpy as np
import pytest

import synth
from gpu_util import DEV, dev, empty, fmt_dev, host, note

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


def test_dequantize_and_f32_layer_error(fx, h):
    import torch
    g = synth.rng_for(31, "deq")
    n = 10_007
    # (code dtype, torch / numpy storage, word length, format sign, code range)
    cases = [(fx.C8, torch.int8, np.int8, 8, 1, (-128, 127)), (fx.C8, torch.int8, np.int8, 8, 0, (0, 255)),
             (fx.I16, torch.int16, np.int16, 16, 1, (-2 ** 15, 2 ** 15 - 1)),
             (fx.I32, torch.int32, np.int32, 24, 1, (-2 ** 23, 2 ** 23))]
    for ct, tdt, ndt, wl, sign, (lo, hi) in cases:
        code = g.integers(lo, hi + 1, n)
        stored = (code - 128 if (ct == fx.C8 and sign == 0) else code).astype(ndt)
        for fl in (5, -3, 0):
            note("dequantize", ct, sign, fl)
            out = empty((n,), torch.float32)
            fx.dequantize(h, dev(stored), ct, fmt_dev(wl, fl, sign), n, out)
            assert np.array_equal(host(out), (code.astype(np.float64) * 2.0 ** -fl).astype(np.float32))
    a = synth.normal(32, "sse-a", (50_001,), std=1.0)
    b = (a + synth.normal(33, "sse-b", (50_001,), std=0.01)).astype(np.float32)
    e = empty((4,), torch.float64)
    fx.layer_error(h, dev(a), dev(b), fx.F32, None, a.size, e)
    got = host(e)
    d = a.astype(np.float64) - b.astype(np.float64)
    np.testing.assert_allclose(got[0], np.sum(d * d), rtol=1e-9)
    assert got[1] == a.min() and got[2] == a.max()
    np.testing.assert_allclose(got[3], a.astype(np.float64).std(), rtol=1e-9)
    assert fx.sync_status(h) == 0


def test_prediction_ties(fx, h):
    import torch
    g = synth.rng_for(34, "ties")
    rows, cols = 37, 1000
    s = g.integers(-50, 50, (rows, cols)).astype(np.int32)
    s[3, [7, 900]] = 500          # two classes at the top
    s[5, [1, 2, 3]] = 600         # three
    s[9, :] = 0                   # all tied
    for dt, arr in ((fx.I32, s), (fx.F32, s.astype(np.float32) * np.float32(0.25))):
        out = empty((2,), torch.int64)
        note("ties", dt)
        fx.prediction_ties(h, dev(arr), dt, rows, cols, out)
        c = (arr == arr.max(1, keepdims=True)).sum(1)
        assert list(host(out)) == [int((c > 1).sum()), int((c - 1).sum())]
    assert fx.sync_status(h) == 0


def test_forward_optimizer_matches_oracle(fx):
    from oracle import qparams as OQ
    from paper_2203_12091_amd import qparams as GQ
    note("qparams oracle resnet18 2x16")
    ref = OQ.ForwardOptimizer("resnet18", batch=2, image=16)
    want = ref.run()
    note("qparams gpu resnet18 2x16")
    fo = GQ.ForwardOptimizer("resnet18", batch=2, image=16, device=DEV)
    got = fo.run()
    assert fx.sync_status(fo.h) == 0
    # the initial formats (preprocessor) and the statistics agree
    assert len(fo.trace) == len(ref.trace)
    for (l1, d1, f1, c1), (l2, d2, f2, c2) in zip(fo.trace, ref.trace):
        assert (l1, d1, f1) == (l2, d2, f2)
        assert abs(c1 - c2) <= 1e-9 * max(abs(c2), 1e-30), (l1, d1, f1, c1, c2)
    assert got == {k: tuple(v) for k, v in want.items()}
    agree = fo.top1_agreement()
    assert 0.0 <= agree <= 1.0
    fo.close()

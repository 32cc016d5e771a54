"""The preprocessor's initial format (fxpq_preprocess, Eq. 6-9) against the
oracle, bit-exact: fl and sign for fp32 and integer sources, every word length
class, the three rounding strategies and both psi rules, including values
placed at the neutral strategy's boundary (psi * 2^b next to sqrt 2), powers
of two, all-zero and all-negative data, and clamping at both ends."""
import math
from fractions import Fraction as F

import numpy as np
import pytest

import synth
from gpu_util import DEV, dev, fmt_host, fmt_new, note

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


def f32_cases():
    g = synth.rng_for(21, "pre-f32")
    cases = [("normal", synth.normal(22, "pre-n", (100_003,), std=0.05)),
             ("relu", np.maximum(synth.normal(23, "pre-r", (4099,)), 0)),
             ("neg", -np.abs(synth.normal(24, "pre-neg", (1001,))) - 0.25),
             ("zeros", np.zeros(77)), ("one", np.array([0.3])), ("pow2", np.array([0.0, 255.0 / 64])),
             ("tiny", np.array([0.0, 2.0 ** -20])), ("huge", np.array([-3000.0, 5000.0]))]
    # psi * 2^b next to sqrt 2 for unsigned 8-bit data: X = 255 * sqrt2 * 2^-b (rounded)
    for b in (-3, 0, 4, 9):
        x = np.float32(255 * math.sqrt(2) * 2.0 ** -b)
        for d in (-1, 0, 1):
            xv = np.nextafter(x, np.float32(np.inf if d > 0 else -np.inf)) if d else x
            cases.append((f"sqrt2-{b}-{d}", np.array([0.0, xv], np.float32)))
    for i in range(6):
        cases.append((f"rand{i}", (g.standard_normal(513) * 2.0 ** g.uniform(-10, 8) + g.uniform(-1, 1))))
    return [(n, np.asarray(x, np.float32)) for n, x in cases]


def test_f32_sources_match_oracle(fx, h):
    from oracle import preprocess as P
    for name, x in f32_cases():
        xmin, xmax = P.exact_extremes_f32(x)
        xd = dev(x)
        for wl in (2, 3, 4, 6, 8, 16, 32):
            for strat in (fx.ROUND_CONSERVATIVE, fx.ROUND_NEUTRAL, fx.ROUND_AGGRESSIVE):
                for rule in (fx.PSI_PRINTED, fx.PSI_MAX):
                    note("preprocess-f32", name, wl, strat, rule)
                    out = fmt_new()
                    fx.preprocess(h, fx.src_f32(xd), x.size, wl, strat, rule, FL_LO, FL_HI, out)
                    want = P.init_fl(xmin, xmax, wl, strat, rule, FL_LO, FL_HI)
                    assert fmt_host(out) == (wl, want[0], want[1], 0), (name, wl, strat, rule)
    assert fx.sync_status(h) == 0


def test_integer_sources_and_minmax_hint(fx, h):
    import torch
    from oracle import preprocess as P
    g = synth.rng_for(25, "pre-int")
    for seed, n, s, spread in [(1, 65_537, 12, 2 ** 20), (2, 1001, 0, 300), (3, 17, 30, 2 ** 40)]:
        v = (g.standard_normal(n) * spread).astype(np.int64)
        if seed == 2:
            v = np.abs(v)
        sd = torch.tensor([s], dtype=torch.int32, device=DEV)
        xmin, xmax = P.exact_extremes_int(v, s)
        vd = dev(v) if seed == 3 else dev(v.astype(np.int32))
        dt = fx.I64 if seed == 3 else fx.I32
        hint = torch.tensor([float(v.min()), float(v.max())], dtype=torch.float64, device=DEV)
        for wl in (4, 8, 16):
            for strat in (fx.ROUND_CONSERVATIVE, fx.ROUND_NEUTRAL, fx.ROUND_AGGRESSIVE):
                for use_hint in (False, True):
                    note("preprocess-int", seed, wl, strat, use_hint)
                    out = fmt_new()
                    src = fx.src_int(vd, dt, sd, hint if use_hint else None)
                    fx.preprocess(h, src, n, wl, strat, fx.PSI_PRINTED, FL_LO, FL_HI, out)
                    want = P.init_fl(xmin, xmax, wl, strat, P.PSI_PRINTED, FL_LO, FL_HI)
                    assert fmt_host(out) == (wl, want[0], want[1], 0), (seed, wl, strat)
    assert fx.sync_status(h) == 0


def test_host_checks(fx, h):
    import ctypes as C
    x = dev(np.ones(8, np.float32))
    src = fx.src_f32(x)
    out = fmt_new()
    L = fx.lib()
    assert L.fxpq_preprocess(h.value, C.byref(src), 8, 1, 0, 0, FL_LO, FL_HI, out.data_ptr()) == fx.ERR_UNSUPPORTED
    assert L.fxpq_preprocess(h.value, C.byref(src), 8, 8, 3, 0, FL_LO, FL_HI, out.data_ptr()) == fx.ERR_INVALID_ARG
    assert L.fxpq_preprocess(h.value, C.byref(src), 8, 8, 0, 2, FL_LO, FL_HI, out.data_ptr()) == fx.ERR_INVALID_ARG
    assert L.fxpq_preprocess(h.value, C.byref(src), 0, 8, 0, 0, FL_LO, FL_HI, out.data_ptr()) == fx.ERR_INVALID_ARG
    assert fx.sync_status(h) == 0

"""The per-layer sensitivity sweep (fifth workload) on the GPU against the
oracle.

Bit-exact: every FP32 teacher activation (order-fixed fp32 arithmetic, so
both sides produce the same bits), and per sweep step the input, weight and
output formats.  The layer error's sum of squares and the reference's
standard deviation agree to a relative 1e-9 (the hot-path bar is 1e-5), its
min / max exactly.  Sizes small enough for the oracle, then the benchmark
configuration itself: the first layer's teacher and two of its steps
recomputed by the oracle at batch 256, 224x224, and the whole sweep checked
through properties that hold at any size.
"""
import numpy as np
import pytest

import synth
from gpu_util import DEV, dev, empty, host, note

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    from oracle import sweep as osw
    from paper_2203_12091_amd import fxpq, sweep
    oracle.lib()
    return torch, fxpq, sweep, oracle, osw


def nhwc(a):
    return np.ascontiguousarray(np.transpose(a, (0, 2, 3, 1)))


def test_teacher_kernels_bit_exact(env):
    torch, fx, sweep, orc, osw = env
    h = fx.Handle(0)
    fx.set_stream(h, torch.cuda.current_stream())
    for (N, C, H, K, R, st, pd) in [(2, 5, 9, 7, 3, 2, 1), (1, 16, 7, 64, 1, 1, 0), (3, 3, 11, 8, 7, 2, 3)]:
        note("teacher conv", N, C, H, K, R, st, pd)
        x = synth.normal(71, "tx", (N, C, H, H))
        w = synth.normal(71, "tw", (K, C, R, R))
        Ho = (H + 2 * pd - R) // st + 1
        y = empty((N, Ho, Ho, K), torch.float32)
        fx.teacher_conv(h, fx.conv_desc(N, H, H, C, K, R, R, st, pd), dev(nhwc(x)),
                        dev(np.transpose(w, (2, 3, 1, 0))), y)
        want = orc.teacher_conv2d(x, w, st, pd)
        assert np.array_equal(host(y), nhwc(want))
        a1 = synth.uniform(72, "a1", (K,), 0.5, 1.5)
        a2 = synth.normal(72, "a2", (K,), std=0.1)
        z = empty(y.shape, torch.float32)
        fx.teacher_affine(h, y, y.numel(), K, z, a1=dev(a1), a2=dev(a2), relu=True)
        assert np.array_equal(host(z), nhwc(orc.teacher_affine(want, a1, a2, relu=True)))
        b = synth.normal(72, "b", (K,))
        fx.teacher_affine(h, y, y.numel(), K, z, bias=dev(b), relu=False)
        assert np.array_equal(host(z), nhwc(orc.teacher_affine(want, bias=b, relu=False)))
    x = synth.normal(73, "mp", (2, 8, 9, 9))
    y = empty((2, 5, 5, 8), torch.float32)
    fx.teacher_maxpool(h, dev(nhwc(x)), 2, 9, 9, 8, 3, 2, 1, y)
    t = osw.Teacher(0)
    t.act["x"] = x
    t.maxpool("p", "x", 3, 2, 1)
    assert np.array_equal(host(y), nhwc(t.act["p"]))
    y = empty((2, 8), torch.float32)
    fx.teacher_avgpool(h, dev(nhwc(x)), 2, 81, 8, y)
    assert np.array_equal(host(y), orc.teacher_avgpool(x))
    a, b = synth.normal(74, "a", (5000,)), synth.normal(74, "b", (5000,))
    y = empty((5000,), torch.float32)
    fx.teacher_add(h, dev(a), dev(b), 5000, True, y)
    v = a + b
    assert np.array_equal(host(y), np.where(v > 0, v, np.float32(0)))
    assert fx.sync_status(h) == 0
    h.close()


def compare(got, want):
    for k in ("layer", "awl", "wwl", "fmt_in", "fmt_w", "fmt_out"):
        assert got[k] == want[k], (k, got, want)
    assert got["ref_min"] == want["ref_min"] and got["ref_max"] == want["ref_max"]
    assert got["sse"] == pytest.approx(want["sse"], rel=1e-9, abs=0)
    assert got["ref_std"] == pytest.approx(want["ref_std"], rel=1e-9)


@pytest.fixture(scope="module")
def small(env):
    torch, fx, sweep, orc, osw = env
    note("sweep small teacher")
    t = osw.teacher("resnet50", batch=2, image=48)
    return t


def test_sweep_small_all_layers(env, small):
    torch, fx, sweep, orc, osw = env
    t = small
    note("sweep small gpu")
    sw = sweep.Sweep("resnet50", batch=2, image=48, wwls=(8, 5, 2), awls=(8, 4))
    # every teacher activation, bit for bit
    for L, (name, src, spec) in zip(sw.layers, t.layers):
        assert L["node"].name == name
        got = host(L["y_ref"])
        assert np.array_equal(got, nhwc(t.act[name]) if got.ndim == 4 and t.act[name].ndim == 4
                              else got.reshape(t.act[name].shape)), name
    sw.run()
    res = sw.results()
    assert res["flags"] == 0
    cache = {}
    for rec in res["records"]:
        li = [n for n, _, _ in t.layers].index(rec["layer"])
        assert rec["status"] == (0, 0)
        compare(rec, osw.step(t, li, rec["awl"], rec["wwl"], cache))
    sw.close()


def test_sweep_every_word_length_on_selected_layers(env, small):
    torch, fx, sweep, orc, osw = env
    t = small
    sel = ["conv1", "layer2.0.c2", "layer3.0.ds", "layer4.2.c3", "fc"]
    note("sweep word lengths", sel)
    sw = sweep.Sweep("resnet50", batch=2, image=48, layers=sel)
    sw.run()
    res = sw.results()
    assert res["flags"] == 0 and len(res["records"]) == len(sel) * 35
    cache = {}
    names = [n for n, _, _ in t.layers]
    for rec in res["records"]:
        compare(rec, osw.step(t, names.index(rec["layer"]), rec["awl"], rec["wwl"], cache))
    sw.close()


def test_sweep_full_size(env):
    # the benchmark configuration: ResNet-50, batch 256, 224x224, all 54
    # layers x 5 activation x 7 weight word lengths
    torch, fx, sweep, orc, osw = env
    note("sweep full size")
    sw = sweep.Sweep("resnet50", batch=256, image=224)
    assert len(sw.steps) == 54 * 35
    sw.run()
    res = sw.results()
    assert res["flags"] == 0
    by_layer = {}
    for rec in res["records"]:
        assert rec["status"] == (0, 0), rec
        assert rec["sse"] >= 0.0
        wl, fl, sign = rec["fmt_out"]
        assert fl == -8 or fl <= 15
        by_layer.setdefault(rec["layer"], []).append(rec)
    for name, recs in by_layer.items():
        # the reference of a layer is one tensor: its statistics never change
        assert len({(r["ref_min"], r["ref_max"], r["ref_std"]) for r in recs}) == 1, name
    # the first layer recomputed by the oracle at full size: teacher output
    # (sampled rows of the 205 M values) and two steps
    note("sweep full size oracle conv1")
    x = synth.normal(4, "input", (256, 3, 224, 224))
    w = synth.he_normal(4, "conv1.w", (64, 3, 7, 7))
    t = osw.Teacher(4)
    t.network_input(x)
    t.cblock("conv1", "input", 64, 7, 2, 3, 8, True, False, True)
    got = host(sw.layers[0]["y_ref"])
    want = t.act["conv1"]
    for n in (0, 97, 255):
        assert np.array_equal(got[n], nhwc(want[n:n + 1])[0])
    recs = {(r["awl"], r["wwl"]): r for r in by_layer["conv1"]}
    cache = {}
    for a, wwl in [(8, 8), (4, 2)]:
        compare(recs[(a, wwl)], osw.step(t, 0, a, wwl, cache))
    sw.close()

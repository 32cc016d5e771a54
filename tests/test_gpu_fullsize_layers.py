"""Full-size parity of every layer class of the benchmark network (ResNet-50,
batch 256, 224x224) and of the first FC layers of AlexNet (batch 64) and
VGG-16 (batch 128), each through the same library calls, in the same launch
configuration, as the calibration forward (fxpq_qconv / fxpq_qgemm with the
C-Block epilogue, then the fused FxP-QLayer fxpq_qlayer; the eltwise sum,
the global average pool and the integer logits as the forward runs them).

Inputs are seeded synthetic codes at each layer's real shape and format
(ReLU-shaped unsigned 8-bit activations, He-normal weights and BN-as-Scale
parameters quantized by both sides): the oracle takes no input from the GPU
path, so the codes a GPU forward hands a deeper layer are not used here.
The oracle recomputes the whole layer and everything is compared exactly:
parameter formats and codes, every int32 accumulator, the FL search over the
whole output tensor (Eq. 14, ties to the larger fl) and every output code
(Eq. 10-12)."""
import numpy as np
import pytest

import synth
from gpu_util import DEV, decode8, dev, empty, fmt_dev, fmt_host, fmt_new, host, note

pytestmark = pytest.mark.gpu

FL_LO, FL_HI = -8, 15
FL_IN = 5  # fractional length of the synthetic input activations


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    from paper_2203_12091_amd import fxpq
    oracle.lib()
    h = fxpq.Handle(0)
    fxpq.set_stream(h, torch.cuda.current_stream())
    yield torch, fxpq, oracle, h
    h.close()


def act_codes(seed, name, shape):
    """Unsigned 8-bit activation codes shaped like a ReLU output at fl = 5
    (about half zeros, a long upper tail, a few saturated)."""
    r = synth.relu_normal(seed, name, shape)
    return np.minimum(np.floor(r * 2.0 ** FL_IN), 255).astype(np.int64)


def upload_c8(codes_nchw, sign):
    """NCHW codes -> the device's NHWC int8 storage (u - 128 when unsigned)."""
    x = np.transpose(codes_nchw, (0, 2, 3, 1))
    return dev((x - (0 if sign else 128)).astype(np.int8))


def param(env, x, wl, ct):
    """A parameter quantized by the library (FL search + quantize, as the
    forward's set-up does) and by the oracle; formats and codes compared."""
    torch, fx, orc, h = env
    xd = dev(np.ascontiguousarray(x, np.float32).ravel())
    f = fmt_new()
    fx.fl_search(h, fx.src_f32(xd), xd.numel(), wl, fx.SIGN_AUTO, FL_LO, FL_HI, f)
    codes = empty((xd.numel(),), torch.int8 if ct == fx.I8 else torch.int32)
    fx.quantize(h, xd, xd.numel(), f, codes, ct)
    gwl, gfl, gsg, gst = fmt_host(f)
    ofl, osg, _ = orc.fl_search_f32(np.ravel(x), wl, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert (gwl, gfl, gsg, gst) == (wl, ofl, osg, 0)
    want = orc.quantize_f32(np.ravel(x), wl, ofl, osg)
    assert np.array_equal(host(codes).astype(np.int64), want)
    return codes, ofl, want


def scale_params(seed, name, k):
    """BN as a Scale layer (Eq. 4-5), running mean 0 and variance 1."""
    gamma = synth.uniform(seed, name + ".gamma", (k,), 0.5, 1.5)
    beta = synth.normal(seed, name + ".beta", (k,), std=0.1)
    inv = np.sqrt(np.ones(k, np.float32) + np.float32(1e-5))
    a1 = (gamma / inv).astype(np.float32)
    a2 = (beta - gamma * np.zeros(k, np.float32) / inv).astype(np.float32)
    return a1, a2


def check_qlayer(env, src, acc_values, s, n_out, shape_nhwc):
    """fxpq_qlayer over the C-Block values against the oracle's search and
    requantization of all of them (acc_values: exact int64 values at scale
    2^-s, NHWC order)."""
    torch, fx, orc, h = env
    f = fmt_new()
    codes = empty(shape_nhwc, torch.int8)
    alt = empty((n_out + 16,), torch.int8)
    fx.qlayer(h, src, n_out, 8, fx.SIGN_AUTO, FL_LO, FL_HI, f, codes, fx.C8, alt)
    gwl, gfl, gsg, gst = fmt_host(f)
    note("oracle search over", n_out, "values")
    ofl, osg, _ = orc.fl_search_i64(acc_values.ravel(), s, 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert (gwl, gfl, gsg, gst) == (8, ofl, osg, 0)
    want = orc.quantize_i64(acc_values.ravel(), s, 8, ofl, osg)
    got = decode8(host(codes).ravel(), osg == 0)
    assert np.array_equal(got, want)
    assert fx.sync_status(h) == 0


# (class, batch, H, W, Cin, Cout, R, stride, pad, relu)
CONV_CLASSES = [
    ("1x1 reduce 256->64, 56x56 (layer1.x.c1)", 256, 56, 56, 256, 64, 1, 1, 0, True),
    ("1x1 expand 64->256, 56x56, no ReLU (layer1.x.c3)", 256, 56, 56, 64, 256, 1, 1, 0, False),
    ("3x3 stride 2, 128, 56->28 (layer2.0.c2)", 256, 56, 56, 128, 128, 3, 2, 1, True),
    ("1x1 stride 2 downsample 256->512, 56->28 (layer2.0.ds)", 256, 56, 56, 256, 512, 1, 2, 0, False),
    ("3x3 256, 14x14 (layer3.x.c2)", 256, 14, 14, 256, 256, 3, 1, 1, True),
    ("3x3 512, 7x7 (layer4.x.c2)", 256, 7, 7, 512, 512, 3, 1, 1, True),
]


@pytest.mark.parametrize("cls", CONV_CLASSES, ids=[c[0].split(" (")[1][:-1] for c in CONV_CLASSES])
def test_resnet50_conv_class_full_size(env, cls):
    torch, fx, orc, h = env
    name, N, H, W, C, K, R, st, pd, relu = cls
    seed = 60 + CONV_CLASSES.index(cls)
    note("fullsize layer class", name)
    x = act_codes(seed, "fsl-x", (N, C, H, W))
    w = synth.he_normal(seed, "fsl-w", (K, C, R, R))
    wkrsc = np.transpose(w, (0, 2, 3, 1)).reshape(K, -1)
    wcodes, fl_w, wq = param(env, wkrsc, 8, fx.I8)
    a1, a2 = scale_params(seed, "fsl-bn", K)
    c1, fl_1, q1 = param(env, a1, 16, fx.I32)
    c2, fl_2, q2 = param(env, a2, 32, fx.I32)
    cs = empty((K,), torch.int32)
    fx.weight_colsum(h, wcodes, K, R * R * C, cs)
    fin = fmt_dev(8, FL_IN, 0)
    ep = fx.epilogue(K, fl_w, fin, relu=relu, scale=c1, fl_scale=fl_1, shift=c2, fl_shift=fl_2)
    Ho, Wo = (H + 2 * pd - R) // st + 1, (W + 2 * pd - R) // st + 1
    M = N * Ho * Wo
    acc = empty((M, K), torch.int32)
    mm = empty((2,), torch.float64)
    fx.qconv(h, fx.conv_desc(N, H, W, C, K, R, R, st, pd), upload_c8(x, 0), fx.C8, wcodes, cs, ep,
             acc, mm)
    src = fx.src_acc(acc, ep, mm)
    note("oracle conv", name)
    wq4 = wq.reshape(K, R, R, C).transpose(0, 3, 1, 2)
    oacc = orc.conv2d(x, wq4, st, pd)  # NCHW, exact
    got = host(acc).reshape(N, Ho, Wo, K)
    assert np.array_equal(got, np.transpose(oacc, (0, 2, 3, 1)))
    del got
    v, s = orc.epilogue(oacc, FL_IN + fl_w, None, 0, q1, fl_1, q2, fl_2, relu)
    del oacc
    mmh = host(mm)  # min / max of the C-Block values in units of 2^-s
    assert (mmh[0], mmh[1]) == (float(v.min()), float(v.max()))
    check_qlayer(env, src, np.transpose(v, (0, 2, 3, 1)), s, M * K, (N, Ho, Wo, K))


def test_resnet50_eltwise_add_full_size(env):
    """The residual sum of stage 1 (two 205 M-value tensors, one signed, one
    unsigned, different fl) with ReLU, through the fused FxP-QLayer's window
    pass over FXPQ_SRC_ADD values."""
    torch, fx, orc, h = env
    shape = (256, 256, 56, 56)
    note("fullsize eltwise add")
    g = synth.rng_for(70, "fsl-add")
    a = np.clip(np.rint(g.standard_normal(shape, dtype=np.float32) * 24.0), -128, 127).astype(np.int64)
    b = act_codes(71, "fsl-add-b", shape)
    fa, fb = 4, FL_IN
    ad, bd = upload_c8(a, 1), upload_c8(b, 0)
    fmt_a, fmt_b = fmt_dev(8, fa, 1), fmt_dev(8, fb, 0)
    src = fx.src_add(ad, fx.C8, fmt_a, bd, fx.C8, fmt_b, True)
    note("oracle eltwise add")
    v, s = orc.eltwise_add(a, fa, b, fb, True)
    check_qlayer(env, src, np.transpose(v, (0, 2, 3, 1)), s, a.size, (256, 56, 56, 256))


def test_resnet50_avgpool_and_logits_full_size(env):
    """Global average pool of the last stage (Sec. "FxP-QLayer": the sum of
    codes times the quantized reciprocal, 16 bits), its FL search and
    requantization, then the last FC (2048 -> 1000 with bias) to integer
    logits, as the forward runs them."""
    torch, fx, orc, h = env
    N, HW, C = 256, 49, 2048
    note("fullsize avgpool")
    x = act_codes(72, "fsl-pool", (N, C, 7, 7))
    xd = upload_c8(x, 0)
    r = np.repeat(np.array([np.float32(1.0) / np.float32(HW)], np.float32), 4)
    rc, rfl, rq = param(env, r, 16, fx.I32)
    ssum = empty((N, C), torch.int64)
    fin = fmt_dev(8, FL_IN, 0)
    fx.avgpool_global(h, xd, fx.C8, fin, N, HW, C, int(rq[0]), ssum)
    ep = fx.epilogue(C, rfl, fin)
    sc = empty((1,), torch.int32)
    fx.epilogue_scale(h, ep, sc)
    src = fx.src_int(ssum, fx.I64, sc)
    f = fmt_new()
    fx.fl_search(h, src, N * C, 8, fx.SIGN_AUTO, FL_LO, FL_HI, f)
    pooled = empty((N, 1, 1, C), torch.int8)
    fx.requant(h, src, N * C, f, pooled, fx.C8)
    ov = orc.avgpool_global(x, int(rq[0]))  # (N, C) at fl_in + rfl
    s = FL_IN + rfl
    assert int(host(sc)[0]) == s
    assert np.array_equal(host(ssum), ov)
    gwl, gfl, gsg, gst = fmt_host(f)
    ofl, osg, _ = orc.fl_search_i64(ov.ravel(), s, 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert (gwl, gfl, gsg, gst) == (8, ofl, osg, 0)
    pq = orc.quantize_i64(ov, s, 8, ofl, osg)
    assert np.array_equal(decode8(host(pooled).reshape(N, C), osg == 0), pq)
    # the last FC: integer logits at the C-Block scale (no FxP-QLayer)
    note("fullsize fc 2048->1000")
    w = synth.he_normal(73, "fsl-fc.w", (1000, C))
    b = synth.normal(73, "fsl-fc.b", (1000,), std=0.01)
    wcodes, fl_w, wq = param(env, w, 8, fx.I8)
    bcodes, fl_b, bq = param(env, b, 32, fx.I32)
    cs = empty((1000,), torch.int32)
    fx.weight_colsum(h, wcodes, 1000, C, cs)
    epf = fx.epilogue(1000, fl_w, f, bias=bcodes, fl_bias=fl_b)
    acc = empty((N, 1000), torch.int32)
    mm = empty((2,), torch.float64)
    fx.qgemm(h, N, 1000, C, pooled, fx.C8, wcodes, cs, epf, acc, mm)
    lf = torch.tensor([32, 0, 1, 0], dtype=torch.int32, device=DEV)
    fx.epilogue_scale(h, epf, lf[1:2])
    logits = empty((N, 1000), torch.int32)
    fx.requant(h, fx.src_acc(acc, epf, mm), N * 1000, lf, logits, fx.I32)
    oacc = orc.gemm(pq, wq.reshape(1000, C))
    assert np.array_equal(host(acc), oacc)
    v, s2 = orc.epilogue(oacc, ofl + fl_w, bq, fl_b)
    assert int(host(lf)[1]) == s2
    assert np.array_equal(host(logits).astype(np.int64), v)
    assert fx.sync_status(h) == 0


# (class, batch M, inputs K, outputs N, seed)
FC_CLASSES = [("alexnet fc6 9216->4096, batch 64", 64, 9216, 4096, 74),
              ("vgg16 fc6 25088->4096, batch 128", 128, 25088, 4096, 75)]


@pytest.mark.parametrize("cls", FC_CLASSES, ids=["alexnet-fc6", "vgg16-fc6"])
def test_fc_full_size(env, cls):
    """The widest FC contractions of the paper's other two networks (bias,
    ReLU, FxP-QLayer) at their batch sizes."""
    torch, fx, orc, h = env
    name, M, K, N, seed = cls
    note("fullsize", name)
    a = act_codes(seed, "fsl-fc-a", (M, K))
    w = synth.he_normal(seed, "fsl-fc-w", (N, K))
    b = synth.normal(seed, "fsl-fc-b", (N,), std=0.01)
    wcodes, fl_w, wq = param(env, w, 8, fx.I8)
    bcodes, fl_b, bq = param(env, b, 32, fx.I32)
    cs = empty((N,), torch.int32)
    fx.weight_colsum(h, wcodes, N, K, cs)
    fin = fmt_dev(8, FL_IN, 0)
    ep = fx.epilogue(N, fl_w, fin, bias=bcodes, fl_bias=fl_b, relu=True)
    acc = empty((M, N), torch.int32)
    mm = empty((2,), torch.float64)
    fx.qgemm(h, M, N, K, dev((a - 128).astype(np.int8)), fx.C8, wcodes, cs, ep, acc, mm)
    oacc = orc.gemm(a, wq.reshape(N, K))
    assert np.array_equal(host(acc), oacc)
    v, s = orc.epilogue(oacc, FL_IN + fl_w, bq, fl_b, relu=True)
    check_qlayer(env, fx.src_acc(acc, ep, mm), v, s, M * N, (M, N))

"""Parity at the benchmark's full size (ResNet-50, batch 256, 224x224), in the
launch configuration bench.py times.

* The first C-Block is recomputed completely by the oracle from the seeded
  inputs: the input's FL search and all 38.5 M input codes, the 205 M conv1
  accumulators through the BN-as-Scale epilogue, conv1's FL search over all of
  them and all 205 M conv1 codes.
* Deeper layers depend on every earlier tensor-wide search, so they are
  checked through properties that hold at any size: no device flags, every
  format valid and in range, every code inside its format's range, and two
  forwards bit-identical.
* Kernel-level checks at the largest layer shapes with seeded tensors: an FL
  search and requantization over 205 M int32 accumulator-like values (exact
  oracle over all of them) and the largest 3x3 conv at sampled outputs
  (every layer class of the network at full size, exactly:
  tests/test_gpu_fullsize_layers.py).
* The paper's other networks at their full sizes (AlexNet b64, VGG-16 b128,
  ResNet-18 b256, 224x224): the same first-C-Block recompute and properties.
"""
import numpy as np
import pytest

import synth
from gpu_util import DEV, decode8, dev, empty, fmt_host, fmt_new, host, note

pytestmark = pytest.mark.gpu

FL_LO, FL_HI = -8, 15


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    from paper_2203_12091_amd import fxpq, nets
    oracle.lib()
    return torch, fxpq, nets, oracle


@pytest.fixture(scope="module")
def full_net(env):
    torch, fx, nets, oracle = env
    note("fullsize resnet50 b256 forward")
    net = nets.CalibNet("resnet50", batch=256, image=224, device=DEV)
    net.forward()
    return net


def test_first_cblock_full_batch_bit_exact(env, full_net):
    torch, fx, nets, orc = env
    net = full_net
    res = net.results()
    assert res["flags"] == 0
    x = synth.normal(4, "input", (256, 3, 224, 224))
    note("fullsize oracle input search")
    fl_in, s_in, _ = orc.fl_search_f32(x.ravel(), 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert res["fmts"]["input"] == (8, fl_in, s_in)
    xq = orc.quantize_f32(x, 8, fl_in, s_in)
    gq = net.act_codes["input"].cpu().numpy()[..., :3]
    gq = decode8(gq, s_in == 0).transpose(0, 3, 1, 2)
    assert np.array_equal(gq, xq)
    del gq
    # conv1 + BN-as-Scale + ReLU, then its FxP-QLayer, all 205 M outputs
    w = synth.he_normal(4, "conv1.w", (64, 3, 7, 7))
    fw = res["fmts"]["conv1.w"]
    ofl_w, osg_w, _ = orc.fl_search_f32(w.ravel(), 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert fw == (8, ofl_w, osg_w)
    wq = orc.quantize_f32(w, 8, ofl_w, osg_w)
    gamma = synth.uniform(4, "conv1.bn.gamma", (64,), 0.5, 1.5)
    beta = synth.normal(4, "conv1.bn.beta", (64,), std=0.1)
    eps = np.float32(1e-5)
    a1 = (gamma / np.sqrt(np.ones(64, np.float32) + eps)).astype(np.float32)
    a2 = (beta - gamma * np.zeros(64, np.float32) / np.sqrt(np.ones(64, np.float32) + eps)).astype(np.float32)
    f1, s1, _ = orc.fl_search_f32(a1, 16, orc.SIGN_AUTO, FL_LO, FL_HI)
    f2, s2, _ = orc.fl_search_f32(a2, 32, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert res["fmts"]["conv1.a1"] == (16, f1, s1) and res["fmts"]["conv1.a2"] == (32, f2, s2)
    note("fullsize oracle conv1")
    acc = orc.conv2d(xq, wq, 2, 3)
    v, s = orc.epilogue(acc, fl_in + ofl_w, None, 0, orc.quantize_f32(a1, 16, f1, s1), f1,
                        orc.quantize_f32(a2, 32, f2, s2), f2, True)
    del acc
    note("fullsize oracle conv1 search")
    fl_c, s_c, _ = orc.fl_search_i64(v.ravel(), s, 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert res["fmts"]["conv1"] == (8, fl_c, s_c)
    want = orc.quantize_i64(v, s, 8, fl_c, s_c)
    del v
    got = decode8(net.act_codes["conv1"].cpu().numpy(), s_c == 0).transpose(0, 3, 1, 2)
    assert np.array_equal(got, want)


def test_full_forward_properties(env, full_net):
    torch, fx, nets, orc = env
    net = full_net
    r1 = net.results()
    assert r1["flags"] == 0
    for name, (wl, fl, sign) in r1["fmts"].items():
        assert 2 <= wl <= 32 and FL_LO <= fl <= FL_HI and sign in (0, 1), name
    first = {}
    for name, t in net.act_codes.items():
        if name.startswith("pool"):
            continue
        wl, fl, sign = r1["fmts"][name]
        lo, hi = orc.qrange(wl, sign)
        off = 128 if sign == 0 else 0
        assert int(t.min().item()) + off >= lo and int(t.max().item()) + off <= hi, name
        if name.endswith(".add") or name.endswith(".c1") or name.endswith(".c2"):
            assert sign == 0, name  # ReLU outputs are unsigned
        first[name] = t.clone()
    logits1 = net.logits.clone()
    note("fullsize second forward")
    net.forward()
    r2 = net.results()
    assert r2["fmts"] == r1["fmts"]
    assert torch.equal(net.logits, logits1)
    for name, t in first.items():
        assert torch.equal(net.act_codes[name], t), name


def test_largest_tensor_search_and_requant(env):
    torch, fx, nets, orc = env
    h = fx.Handle(0)
    fx.set_stream(h, torch.cuda.current_stream())
    n = 256 * 112 * 112 * 64  # conv1 output size of the benchmark
    g = synth.rng_for(9, "fullsize-acc")
    v = np.maximum(g.standard_normal(n, dtype=np.float32) * 3000.0, 0).astype(np.int32)
    s = 14
    sd = torch.tensor([s], dtype=torch.int32, device=DEV)
    vd = dev(v)
    note("fullsize int32 search")
    out = fmt_new()
    fx.fl_search(h, fx.src_int(vd, fx.I32, sd), n, 8, fx.SIGN_AUTO, FL_LO, FL_HI, out)
    gwl, gfl, gsg, gst = fmt_host(out)
    v64 = v.astype(np.int64)
    ofl, osg, _ = orc.fl_search_i64(v64, s, 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert (gfl, gsg, gst) == (ofl, osg, 0)
    codes = empty((n,), torch.int8)
    fx.requant(h, fx.src_int(vd, fx.I32, sd), n, out, codes, fx.C8)
    got = decode8(host(codes), gsg == 0)
    assert np.array_equal(got, orc.quantize_i64(v64, s, 8, ofl, osg))
    assert fx.sync_status(h) == 0
    h.close()


def test_largest_3x3_conv_sampled(env):
    torch, fx, nets, orc = env
    h = fx.Handle(0)
    fx.set_stream(h, torch.cuda.current_stream())
    # layer3 3x3 of ResNet-50 at batch 256: M = 50176, N = 256, K = 2304
    N, C, H, K = 256, 256, 14, 256
    x = synth.integers(10, "fs-x", (N, C, H, H), 0, 255)
    w = synth.integers(10, "fs-w", (K, C, 3, 3), -128, 127)
    xd = dev((np.transpose(x, (0, 2, 3, 1)) - 128).astype(np.int8))
    wd = dev(np.transpose(w, (0, 2, 3, 1)).reshape(K, -1).astype(np.int8))
    cs = empty((K,), torch.int32)
    fx.weight_colsum(h, wd, K, 9 * C, cs)
    acc = empty((N, H, H, K), torch.int32)
    note("fullsize 3x3 conv")
    fx.qconv(h, fx.conv_desc(N, H, H, C, K, 3, 3, 1, 1), xd, fx.U8OFF, wd, cs, None, acc)
    got = host(acc)
    x64, w64 = np.ascontiguousarray(x, np.int64), np.ascontiguousarray(w, np.int64)
    g = synth.rng_for(11, "fs-sample")
    for _ in range(2000):
        n, k, oh, ow = (int(g.integers(0, N)), int(g.integers(0, K)), int(g.integers(0, H)),
                        int(g.integers(0, H)))
        assert got[n, oh, ow, k] == orc.conv2d_point(x64, w64, 1, 1, n, k, oh, ow)
    # the halo tiles give the same integers over the whole tensor
    note("fullsize 3x3 conv, halo tiles")
    fx.set_conv_tiling(h, fx.TILING_HALO)
    acc2 = empty((N, H, H, K), torch.int32)
    fx.qconv(h, fx.conv_desc(N, H, H, C, K, 3, 3, 1, 1), xd, fx.U8OFF, wd, cs, None, acc2)
    assert torch.equal(acc, acc2)
    assert fx.sync_status(h) == 0
    h.close()


def test_wide_first_layer_full_batch_sampled(env):
    """The wide C-Block in bench.py's --mode wide configuration: ResNet-50's
    first conv over 256 x 224 x 224 padded RGB with 16-bit input codes and
    16-bit weights (Scale + ReLU epilogue), exact int64 values checked
    against the oracle's integer convolution and epilogue at 256 sampled
    output pixels (all 64 channels each), plus the scale and the flags."""
    torch, fx, nets, orc = env
    N, H, C, K, R = 256, 224, 3, 64, 7
    g = synth.rng_for(81, "wide-full")
    xc = g.integers(-2 ** 15, 2 ** 15, (N, C, H, H), dtype=np.int32)
    wc = g.integers(-2 ** 15, 2 ** 15, (K, C, R, R), dtype=np.int32)
    a1 = g.integers(-2 ** 15, 2 ** 15, K).astype(np.int32)
    a2 = g.integers(-2 ** 31, 2 ** 31 - 1, K).astype(np.int32)
    x4 = np.zeros((N, H, H, 4), np.int32)
    x4[..., :3] = xc.transpose(0, 2, 3, 1)
    depth = R * R * 4
    w4 = np.zeros((K, R, R, 4), np.int32)
    w4[..., :3] = wc.transpose(0, 2, 3, 1)
    wrow = np.zeros((K, (depth + 63) // 64 * 64), np.int32)
    wrow[:, :depth] = w4.reshape(K, -1)
    fin = torch.tensor([16, 12, 1, 0], dtype=torch.int32, device=DEV)
    a1d, a2d = dev(a1), dev(a2)
    ep = fx.epilogue(K, 14, fin, relu=True, scale=a1d, fl_scale=14, shift=a2d, fl_shift=20)
    h = fx.Handle(0)
    fx.set_stream(h, torch.cuda.current_stream())
    d = fx.conv_desc(N, H, H, 4, K, R, R, 2, 3)
    nb = fx.qconv_wide_workspace(d, 16, 1, 16, 1)
    ws = empty((nb,), torch.uint8)
    Ho = (H + 6 - R) // 2 + 1
    v = empty((N * Ho * Ho * K,), torch.int64)
    sc = empty((1,), torch.int32)
    note("fullsize wide conv1 16x16")
    fx.qconv_wide(h, d, dev(x4), 16, 1, dev(wrow), 16, 1, ep, v, sc, ws, nb)
    assert fx.sync_status(h) == 0
    del ws
    got = host(v).reshape(N, Ho, Ho, K)
    pix = [(int(n), int(p), int(q)) for n, p, q in
           zip(g.integers(0, N, 256), g.integers(0, Ho, 256), g.integers(0, Ho, 256))]
    pix += [(0, 0, 0), (N - 1, Ho - 1, Ho - 1), (7, 0, Ho - 1)]
    xc64, wc64 = np.ascontiguousarray(xc, np.int64), np.ascontiguousarray(wc, np.int64)
    acc = np.array([[orc.conv2d_point(xc64, wc64, 2, 3, n, k, p, q) for k in range(K)]
                    for n, p, q in pix], np.int64)
    want, s_out = orc.epilogue(acc, 12 + 14, None, 0, a1.astype(np.int64), 14, a2.astype(np.int64), 20,
                               True)
    assert int(host(sc)[0]) == s_out
    assert np.array_equal(np.array([got[n, p, q] for n, p, q in pix]), want)
    h.close()


def test_wide_first_layer_32bit_full_batch(env):
    """The paper's initial design for the first layer (Sec. "Initial Design
    Generation"): ResNet-50's first C-Block at batch 256 with the network
    input and the weights at 32 bits, on fxpq_qconv_wide.  The 32-bit input
    format and all 38.5 M input codes, the weight, Scale multiplier (16-bit)
    and offset (32-bit) formats and codes are checked against the oracle; the
    exact int64 C-Block values at 256 sampled output pixels (all 64 channels
    each); then the FxP-QLayer at WL 8 over all 205 M values: the FL search
    and every code, exactly.  (With fractional lengths capped at 15 the
    32-bit codes of these data stay near 2^17 and the values near 2^48.)"""
    torch, fx, nets, orc = env
    N, H, C, K, R = 256, 224, 3, 64, 7
    h = fx.Handle(0)
    fx.set_stream(h, torch.cuda.current_stream())

    def param(x, wl):
        xd = dev(np.ascontiguousarray(x, np.float32).ravel())
        f = fmt_new()
        fx.fl_search(h, fx.src_f32(xd), xd.numel(), wl, fx.SIGN_AUTO, FL_LO, FL_HI, f)
        codes = empty((xd.numel(),), torch.int32)
        fx.quantize(h, xd, xd.numel(), f, codes, fx.I32)
        gwl, gfl, gsg, gst = fmt_host(f)
        ofl, osg, _ = orc.fl_search_f32(np.ravel(x), wl, orc.SIGN_AUTO, FL_LO, FL_HI)
        assert (gwl, gfl, gsg, gst) == (wl, ofl, osg, 0)
        want = orc.quantize_f32(np.ravel(x), wl, ofl, osg)
        assert np.array_equal(host(codes).astype(np.int64), want)
        return f, ofl, want.reshape(np.shape(x))

    note("fullsize wide conv1 32x32: parameters")
    x = synth.normal(9, "wide32.input", (N, C, H, H))
    w = synth.normal(9, "wide32.w", (K, C, R, R), std=float(np.sqrt(2.0 / (C * R * R))))
    gamma = synth.uniform(9, "wide32.gamma", (K,), 0.5, 1.5)
    beta = synth.normal(9, "wide32.beta", (K,), std=0.1)
    a1 = (gamma / np.sqrt(np.float32(1.0) + np.float32(1e-5))).astype(np.float32)
    fin, fl_x, xc = param(x, 32)
    _, fl_w, wc = param(w, 32)
    _, fl_a1, c1 = param(a1, 16)
    _, fl_a2, c2 = param(beta, 32)
    del x
    x4 = np.zeros((N, H, H, 4), np.int32)
    x4[..., :3] = xc.transpose(0, 2, 3, 1)
    depth = R * R * 4
    w4 = np.zeros((K, R, R, 4), np.int32)
    w4[..., :3] = wc.transpose(0, 2, 3, 1)
    wrow = np.zeros((K, (depth + 63) // 64 * 64), np.int32)
    wrow[:, :depth] = w4.reshape(K, -1)
    ep = fx.epilogue(K, fl_w, fin, relu=True, scale=dev(c1.astype(np.int32)), fl_scale=fl_a1,
                     shift=dev(c2.astype(np.int32)), fl_shift=fl_a2)
    d = fx.conv_desc(N, H, H, 4, K, R, R, 2, 3)
    nb = fx.qconv_wide_workspace(d, 32, 1, 32, 1)
    ws = empty((nb,), torch.uint8)
    Ho = (H + 6 - R) // 2 + 1
    n = N * Ho * Ho * K
    v = empty((n,), torch.int64)
    sc = empty((1,), torch.int32)
    note("fullsize wide conv1 32x32: contraction")
    fx.qconv_wide(h, d, dev(x4), 32, 1, dev(wrow), 32, 1, ep, v, sc, ws, nb)
    assert fx.sync_status(h) == 0
    del ws, x4
    got = host(v)
    g = synth.rng_for(82, "wide32-pix")
    pix = [(int(a), int(b), int(c)) for a, b, c in
           zip(g.integers(0, N, 256), g.integers(0, Ho, 256), g.integers(0, Ho, 256))]
    pix += [(0, 0, 0), (N - 1, Ho - 1, Ho - 1), (7, 0, Ho - 1)]
    g4 = got.reshape(N, Ho, Ho, K)
    xc64, wc64 = np.ascontiguousarray(xc, np.int64), np.ascontiguousarray(wc, np.int64)
    acc = np.array([[orc.conv2d_point(xc64, wc64, 2, 3, a, k, b, c) for k in range(K)]
                    for a, b, c in pix], np.int64)
    want, s_out = orc.epilogue(acc, fl_x + fl_w, None, 0, c1.astype(np.int64), fl_a1,
                               c2.astype(np.int64), fl_a2, True)
    assert int(host(sc)[0]) == s_out
    assert np.array_equal(np.array([g4[a, b, c] for a, b, c in pix]), want)
    note("fullsize wide conv1 32x32: FxP-QLayer over all values")
    out = fmt_new()
    src = fx.src_int(v, fx.I64, sc)
    fx.fl_search(h, src, n, 8, fx.SIGN_AUTO, FL_LO, FL_HI, out)
    codes = empty((n,), torch.int8)
    fx.requant(h, src, n, out, codes, fx.C8)
    gwl, gfl, gsg, gst = fmt_host(out)
    ofl, osg, _ = orc.fl_search_i64(got, s_out, 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert (gwl, gfl, gsg, gst) == (8, ofl, osg, 0)
    assert np.array_equal(decode8(host(codes), osg == 0), orc.quantize_i64(got, s_out, 8, ofl, osg))
    assert fx.sync_status(h) == 0
    h.close()


@pytest.mark.parametrize("name,batch", [("alexnet", 64), ("vgg16", 128), ("resnet18", 256)])
def test_other_networks_full_size(env, name, batch):
    """AlexNet b64, VGG-16 b128 and ResNet-18 b256 at 224x224 in the
    forward's launch configuration: the input's FL search and every input
    code, the first C-Block's weights (and bias or Scale), all its outputs
    through the epilogue, its FL search and every code recomputed by the
    oracle; then every format valid, every code in range, and a second
    forward bit-identical."""
    torch, fx, nets, orc = env
    note("fullsize forward", name, batch)
    net = nets.CalibNet(name, batch=batch, image=224, device=DEV)
    net.forward()
    res = net.results()
    assert res["flags"] == 0
    seed = nets.SEEDS[name]
    x = synth.normal(seed, "input", (batch, 3, 224, 224))
    note("fullsize oracle input search", name)
    fl_in, s_in, _ = orc.fl_search_f32(x.ravel(), 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert res["fmts"]["input"] == (8, fl_in, s_in)
    xq = orc.quantize_f32(x, 8, fl_in, s_in)
    del x
    gq = decode8(net.act_codes["input"].cpu().numpy()[..., :3], s_in == 0).transpose(0, 3, 1, 2)
    assert np.array_equal(gq, xq)
    del gq
    n = [n for n in net.graph if n.op == "conv"][0]
    K, k = n.cout, n.k
    w = synth.he_normal(seed, n.name + ".w", (K, 3, k, k))
    fl_w, sg_w, _ = orc.fl_search_f32(w.ravel(), n.wl, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert res["fmts"][n.name + ".w"] == (n.wl, fl_w, sg_w)
    wq = orc.quantize_f32(w, n.wl, fl_w, sg_w)
    kw = {}
    if n.bias:
        b = synth.normal(seed, n.name + ".b", (K,), std=0.01)
        fb, sb, _ = orc.fl_search_f32(b, 32, orc.SIGN_AUTO, FL_LO, FL_HI)
        assert res["fmts"][n.name + ".b"] == (32, fb, sb)
        kw.update(bias=orc.quantize_f32(b, 32, fb, sb), fl_b=fb)
    if n.bn:
        gamma = synth.uniform(seed, n.name + ".bn.gamma", (K,), 0.5, 1.5)
        beta = synth.normal(seed, n.name + ".bn.beta", (K,), std=0.1)
        inv = np.sqrt(np.ones(K, np.float32) + np.float32(1e-5))
        a1 = (gamma / inv).astype(np.float32)
        a2 = (beta - gamma * np.zeros(K, np.float32) / inv).astype(np.float32)
        f1, s1, _ = orc.fl_search_f32(a1, 16, orc.SIGN_AUTO, FL_LO, FL_HI)
        f2, s2, _ = orc.fl_search_f32(a2, 32, orc.SIGN_AUTO, FL_LO, FL_HI)
        assert res["fmts"][n.name + ".a1"] == (16, f1, s1) and res["fmts"][n.name + ".a2"] == (32, f2, s2)
        kw.update(a1=orc.quantize_f32(a1, 16, f1, s1), fl_a1=f1, a2=orc.quantize_f32(a2, 32, f2, s2),
                  fl_a2=f2)
    note("fullsize oracle first conv", name, n.name)
    acc = orc.conv2d(xq, wq, n.stride, n.pad)
    del xq
    v, s = orc.epilogue(acc, fl_in + fl_w, relu=n.relu, **kw)
    del acc
    note("fullsize oracle first search", name, v.size)
    fl_c, s_c, _ = orc.fl_search_i64(v.ravel(), s, 8, orc.SIGN_AUTO, FL_LO, FL_HI)
    assert res["fmts"][n.name] == (8, fl_c, s_c)
    want = orc.quantize_i64(v, s, 8, fl_c, s_c)
    del v
    got = decode8(net.act_codes[n.name].cpu().numpy(), s_c == 0).transpose(0, 3, 1, 2)
    assert np.array_equal(got, want)
    del got, want
    # every layer: valid formats, codes in range; a second forward identical
    for nm, (wl, fl, sign) in res["fmts"].items():
        assert 2 <= wl <= 32 and FL_LO <= fl <= FL_HI and sign in (0, 1), nm
    first = {}
    for nm, t in net.act_codes.items():
        if nm.startswith("pool"):
            continue
        wl, fl, sign = res["fmts"][nm]
        lo, hi = orc.qrange(wl, sign)
        off = 128 if sign == 0 else 0
        assert int(t.min().item()) + off >= lo and int(t.max().item()) + off <= hi, nm
        first[nm] = t.clone()
    logits = net.logits.clone()
    note("fullsize second forward", name)
    net.forward()
    assert net.results()["fmts"] == res["fmts"]
    assert torch.equal(net.logits, logits)
    for nm, t in first.items():
        assert torch.equal(net.act_codes[nm], t), nm
    net.close()

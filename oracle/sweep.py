"""Oracle per-layer sensitivity sweep (NCHW) -- TEST INFRASTRUCTURE ONLY.

The FP32 teacher runs the oracle's own network description (``nets.resnet``)
with full-precision layers (``core.teacher_*``; order-fixed fp32 arithmetic,
pinned in tests/test_oracle_teacher.py).  A sweep step for layer l, activation
word length a and weight word length w (a reading of the sensitivity test,
Sec. "Data-Structures Sensitivity to Quantization": layer l quantized, the
rest intact):
  the teacher's input of l quantized at a (Eq. 14 search, Eq. 10-12);
  the weights at w; bias at 32 bits and the Scale layer at 16 / 32 bits;
  the exact integer C-Block (conv, epilogue, ReLU);
  the output requantized at a by its FxP-QLayer, or kept as integer logits
  (stored at 32 bits, fl = the C-Block scale) for the last layer;
  the layer error against the teacher's output of l (Eq. 14, 16, 18).

parity unpinned: the composed sweep has no printed values; its parts are
pinned (tests/test_oracle_pins.py, tests/test_oracle_teacher.py).
"""
import numpy as np

import synth

from . import core as orc
from .nets import FL, SEED, SHAPE, resnet


class Teacher:
    """FP32 forward with the Forward interface of nets.py; records every
    conv / FC layer's input and output."""

    def __init__(self, seed):
        self.seed = seed
        self.act = {}
        self.layers = []  # (name, input name, spec)

    def network_input(self, x):
        self.act["input"] = x

    def cblock(self, name, src, cout, k, stride, pad, wl, relu, bias, bn, fc=False, last=False):
        x = self.act[src]
        if fc:
            xin = x.reshape(x.shape[0], -1)
            w = synth.he_normal(self.seed, name + ".w", (cout, xin.shape[1]))
            y = orc.teacher_conv2d(xin.reshape(xin.shape[0], -1, 1, 1), w.reshape(cout, -1, 1, 1), 1, 0)
        else:
            w = synth.he_normal(self.seed, name + ".w", (cout, x.shape[1], k, k))
            y = orc.teacher_conv2d(x, w, stride, pad)
        spec = {"w": w, "k": k, "stride": stride, "pad": pad, "relu": relu, "fc": fc, "last": last}
        if bias:
            spec["b"] = synth.normal(self.seed, name + ".b", (cout,), std=0.01)
            y = orc.teacher_affine(y, bias=spec["b"], relu=relu)
        elif bn:
            gamma = synth.uniform(self.seed, name + ".bn.gamma", (cout,), 0.5, 1.5)
            beta = synth.normal(self.seed, name + ".bn.beta", (cout,), std=0.1)
            mu = np.zeros(cout, np.float32)
            sigma2 = np.ones(cout, np.float32)
            eps = np.float32(1e-5)
            spec["a1"] = (gamma / np.sqrt(sigma2 + eps)).astype(np.float32)
            spec["a2"] = (beta - gamma * mu / np.sqrt(sigma2 + eps)).astype(np.float32)
            y = orc.teacher_affine(y, spec["a1"], spec["a2"], relu=relu)
        else:
            y = orc.teacher_affine(y, relu=relu)
        self.act[name] = y
        self.layers.append((name, src, spec))

    def maxpool(self, name, src, k, stride, pad):
        x = self.act[src]
        N, C, H, W = x.shape
        Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
        xp = np.full((N, C, H + 2 * pad, W + 2 * pad), -np.inf, np.float32)
        xp[:, :, pad:pad + H, pad:pad + W] = x
        y = np.full((N, C, Ho, Wo), -np.inf, np.float32)
        for r in range(k):
            for s in range(k):
                y = np.maximum(y, xp[:, :, r:r + stride * Ho:stride, s:s + stride * Wo:stride])
        self.act[name] = y

    def add(self, name, a, b):
        v = self.act[a] + self.act[b]  # one fp32 add
        self.act[name] = np.where(v > 0, v, np.float32(0)).astype(np.float32)

    def avgpool(self, name, src):
        y = orc.teacher_avgpool(self.act[src])
        self.act[name] = y.reshape(y.shape[0], y.shape[1], 1, 1)


def teacher(name="resnet50", seed=None, batch=None, image=None):
    seed = SEED[name] if seed is None else seed
    b0, s0 = SHAPE[name]
    t = Teacher(seed)
    t.network_input(synth.normal(seed, "input", (batch or b0, 3, image or s0, image or s0)))
    resnet(t, name == "resnet50")
    return t


def _qparam(x, wl):
    fl, sign, _ = orc.fl_search_f32(x.ravel(), wl, orc.SIGN_AUTO, *FL)
    return orc.quantize_f32(x, wl, fl, sign).astype(np.int64), (wl, fl, sign)


def step(t, li, awl, wwl, cache=None):
    """One sweep step on the oracle: formats and the layer error record."""
    name, src, spec = t.layers[li]
    cache = {} if cache is None else cache
    x = t.act[src]
    ref = t.act[name]
    key = (li, "in", awl)
    if key not in cache:
        fl, sign, _ = orc.fl_search_f32(x.ravel(), awl, orc.SIGN_AUTO, *FL)
        cache[key] = (orc.quantize_f32(x, awl, fl, sign), (awl, fl, sign))
    xq, fmt_in = cache[key]
    key = (li, "w", wwl)
    if key not in cache:
        cache[key] = _qparam(spec["w"], wwl)
    wq, fmt_w = cache[key]
    if spec["fc"]:
        acc = orc.gemm(xq.reshape(xq.shape[0], -1), wq)
    else:
        acc = orc.conv2d(xq, wq, spec["stride"], spec["pad"])
    b = a1 = a2 = None
    fl_b = fl_a1 = fl_a2 = 0
    if "b" in spec:
        key = (li, "b")
        if key not in cache:
            cache[key] = _qparam(spec["b"], 32)
        b, (_, fl_b, _) = cache[key]
    if "a1" in spec:
        key = (li, "a")
        if key not in cache:
            cache[key] = (_qparam(spec["a1"], 16), _qparam(spec["a2"], 32))
        (a1, (_, fl_a1, _)), (a2, (_, fl_a2, _)) = cache[key]
    v, s = orc.epilogue(acc, fmt_in[1] + fmt_w[1], b, fl_b, a1, fl_a1, a2, fl_a2, spec["relu"])
    if spec["last"]:
        fmt_out = (32, s, 1)
    else:
        fl, sign, _ = orc.fl_search_i64(v.ravel(), s, awl, orc.SIGN_AUTO, *FL)
        fmt_out = (awl, fl, sign)
    codes = orc.quantize_i64(v, s, *fmt_out)
    # both in the layer's NCHW order (or [n][k] for FC)
    err = orc.layer_error(ref.ravel(), codes.ravel(), *fmt_out)
    return {"layer": name, "awl": awl, "wwl": wwl, "fmt_in": fmt_in, "fmt_w": fmt_w,
            "fmt_out": fmt_out, "sse": float(err[0]), "ref_min": float(err[1]),
            "ref_max": float(err[2]), "ref_std": float(err[3])}

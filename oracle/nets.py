"""Oracle calibration forwards (NCHW, exact) -- TEST INFRASTRUCTURE ONLY.

Written independently of the GPU runner.  It follows the paper's integer
inference graph: an FxP-QLayer quantizes the network input and the output of
every C-Block (CONV/FC with bias, BN-as-Scale and ReLU fused; Eltwise;
AVG-POOL), none follows MAX-POOL or the last layer (Sec. "FxP-QLayer").  Each
FxP-QLayer and each parameter tensor gets its fractional length from the
exhaustive error search (Eq. 14 over fl in [-8, 15], ties to the larger fl)
with the sign strategy of Eq. 6; BN becomes Scale by Eq. 4-5 with running
mean 0 and variance 1.  Word lengths: activations 8; weights per workload;
biases 32; Scale multiplier 16, Scale shift 32; the AVG-POOL reciprocal 16.

The synthetic tensors come from ``synth`` under the same names as everywhere
else, in canonical layouts (NCHW, OIHW, [out][in]).

parity unpinned: the composition has no printed values to check against; it is
pinned only through its parts (tests/test_oracle_pins.py) and shape pins.
"""
import numpy as np

import synth

from . import core as orc

FL = (-8, 15)
SEED = {"fc": 0, "alexnet": 1, "vgg16": 2, "resnet18": 3, "resnet50": 4}
SHAPE = {"alexnet": (64, 224), "vgg16": (128, 224), "resnet18": (256, 224), "resnet50": (256, 224)}


class Forward:
    """Runs one network exactly on the CPU and records every chosen format."""

    def __init__(self, seed, pcache=None):
        self.seed = seed
        self.pcache = pcache  # optional: quantized parameters from an earlier run
        self.fmts = {}
        self.codes = {}
        self.act = {}  # name -> (codes NCHW int32, fl, sign)

    # ---- parameters ----
    def qparam(self, key, x, wl):
        ck = (key, x.shape, wl)
        if self.pcache is not None and ck in self.pcache:
            q, fl, fmt = self.pcache[ck]
            self.fmts[key] = fmt
            return q, fl
        fl, sign, _ = orc.fl_search_f32(x.ravel(), wl, orc.SIGN_AUTO, *FL)
        self.fmts[key] = (wl, fl, sign)
        q = orc.quantize_f32(x, wl, fl, sign).astype(np.int64)
        if self.pcache is not None:
            self.pcache[ck] = (q, fl, self.fmts[key])
        return q, fl

    def fxp_qlayer(self, name, v, s, wl=8):
        fl, sign, _ = orc.fl_search_i64(v.ravel(), s, wl, orc.SIGN_AUTO, *FL)
        self.fmts[name] = (wl, fl, sign)
        q = orc.quantize_i64(v, s, wl, fl, sign)
        self.act[name] = (q, fl, sign)
        return q, fl

    # ---- layers ----
    def network_input(self, x):
        fl, sign, _ = orc.fl_search_f32(x.ravel(), 8, orc.SIGN_AUTO, *FL)
        self.fmts["input"] = (8, fl, sign)
        q = orc.quantize_f32(x, 8, fl, sign)
        self.act["input"] = (q, fl, sign)
        self.input_error = orc.layer_error(x.ravel(), q.ravel(), 8, fl, sign)

    def cblock(self, name, src, cout, k, stride, pad, wl, relu, bias, bn, fc=False, last=False):
        x, fl_x, _ = self.act[src]
        if fc:
            xin = x.reshape(x.shape[0], -1)
            w = synth.he_normal(self.seed, name + ".w", (cout, xin.shape[1]))
        else:
            w = synth.he_normal(self.seed, name + ".w", (cout, x.shape[1], k, k))
        wq, fl_w = self.qparam(name + ".w", w, wl)
        acc = orc.gemm(xin, wq) if fc else orc.conv2d(x, wq, stride, pad)
        b = a1 = a2 = None
        fl_b = fl_a1 = fl_a2 = 0
        if bias:
            b, fl_b = self.qparam(name + ".b", synth.normal(self.seed, name + ".b", (cout,), std=0.01), 32)
        if bn:
            gamma = synth.uniform(self.seed, name + ".bn.gamma", (cout,), 0.5, 1.5)
            beta = synth.normal(self.seed, name + ".bn.beta", (cout,), std=0.1)
            mu = np.zeros(cout, np.float32)
            sigma2 = np.ones(cout, np.float32)
            eps = np.float32(1e-5)
            aleph1 = (gamma / np.sqrt(sigma2 + eps)).astype(np.float32)
            aleph2 = (beta - gamma * mu / np.sqrt(sigma2 + eps)).astype(np.float32)
            a1, fl_a1 = self.qparam(name + ".a1", aleph1, 16)
            a2, fl_a2 = self.qparam(name + ".a2", aleph2, 32)
        v, s = orc.epilogue(acc, fl_x + fl_w, b, fl_b, a1, fl_a1, a2, fl_a2, relu)
        if last:
            self.logits, self.logit_fl = v, s
            return
        self.fxp_qlayer(name, v, s)

    def maxpool(self, name, src, k, stride, pad):
        x, fl, sign = self.act[src]
        self.act[name] = (orc.maxpool(x, k, stride, pad), fl, sign)

    def add(self, name, a, b):
        xa, fa, _ = self.act[a]
        xb, fb, _ = self.act[b]
        v, s = orc.eltwise_add(xa, fa, xb, fb, relu=True)
        self.fxp_qlayer(name, v, s)

    def avgpool(self, name, src):
        x, fl, _ = self.act[src]
        hw = x.shape[2] * x.shape[3]
        r = np.array([np.float32(1.0) / np.float32(hw)], np.float32)
        rq, fl_r = self.qparam("avgpool.recip", r, 16)
        y = orc.avgpool_global(x, int(rq[0]))
        self.fxp_qlayer(name, y.reshape(y.shape[0], y.shape[1], 1, 1), fl + fl_r)

    def result(self):
        return {"fmts": self.fmts, "logits": np.asarray(self.logits).reshape(self.logits.shape[0], -1),
                "logit_fl": self.logit_fl, "input_error": self.input_error,
                "codes": {k: v[0] for k, v in self.act.items() if not k.startswith("pool")}}


def alexnet(f):
    f.cblock("conv1", "input", 64, 11, 4, 2, 8, True, True, False)
    f.maxpool("pool1", "conv1", 3, 2, 0)
    f.cblock("conv2", "pool1", 192, 5, 1, 2, 8, True, True, False)
    f.maxpool("pool2", "conv2", 3, 2, 0)
    f.cblock("conv3", "pool2", 384, 3, 1, 1, 8, True, True, False)
    f.cblock("conv4", "conv3", 256, 3, 1, 1, 8, True, True, False)
    f.cblock("conv5", "conv4", 256, 3, 1, 1, 8, True, True, False)
    f.maxpool("pool5", "conv5", 3, 2, 0)
    f.cblock("fc6", "pool5", 4096, 1, 1, 0, 8, True, True, False, fc=True)
    f.cblock("fc7", "fc6", 4096, 1, 1, 0, 8, True, True, False, fc=True)
    f.cblock("fc8", "fc7", 1000, 1, 1, 0, 8, False, True, False, fc=True, last=True)


def vgg16(f):
    widths = [(1, [64, 64]), (2, [128, 128]), (3, [256] * 3), (4, [512] * 3), (5, [512] * 3)]
    prev = "input"
    for gi, ws in widths:
        for li, c in enumerate(ws, 1):
            nm = f"conv{gi}_{li}"
            wl = synth.choice(f.seed, nm + ".wl", [4, 5, 6, 7, 8], 1)[0]
            f.cblock(nm, prev, c, 3, 1, 1, wl, True, True, False)
            prev = nm
        f.maxpool(f"pool{gi}", prev, 2, 2, 0)
        prev = f"pool{gi}"
    for nm, c, last in (("fc6", 4096, False), ("fc7", 4096, False), ("fc8", 1000, True)):
        wl = synth.choice(f.seed, nm + ".wl", [4, 5, 6, 7, 8], 1)[0]
        f.cblock(nm, prev, c, 1, 1, 0, wl, not last, True, False, fc=True, last=last)
        prev = nm


def resnet(f, bottleneck):
    opts = [8] if bottleneck else [4, 6, 8]

    def wl(nm):
        return opts[0] if len(opts) == 1 else synth.choice(f.seed, nm + ".wl", opts, 1)[0]

    f.cblock("conv1", "input", 64, 7, 2, 3, wl("conv1"), True, False, True)
    f.maxpool("pool1", "conv1", 3, 2, 1)
    prev, cin = "pool1", 64
    depths = [3, 4, 6, 3] if bottleneck else [2, 2, 2, 2]
    for si, (nb, width) in enumerate(zip(depths, (64, 128, 256, 512)), 1):
        for bi in range(nb):
            st = 2 if si > 1 and bi == 0 else 1
            nm = f"layer{si}.{bi}"
            out_c = 4 * width if bottleneck else width
            if bottleneck:
                f.cblock(nm + ".c1", prev, width, 1, 1, 0, wl(nm + ".c1"), True, False, True)
                f.cblock(nm + ".c2", nm + ".c1", width, 3, st, 1, wl(nm + ".c2"), True, False, True)
                f.cblock(nm + ".c3", nm + ".c2", out_c, 1, 1, 0, wl(nm + ".c3"), False, False, True)
                main = nm + ".c3"
            else:
                f.cblock(nm + ".c1", prev, width, 3, st, 1, wl(nm + ".c1"), True, False, True)
                f.cblock(nm + ".c2", nm + ".c1", width, 3, 1, 1, wl(nm + ".c2"), False, False, True)
                main = nm + ".c2"
            if st != 1 or cin != out_c:
                f.cblock(nm + ".ds", prev, out_c, 1, st, 0, wl(nm + ".ds"), False, False, True)
                short = nm + ".ds"
            else:
                short = prev
            f.add(nm + ".add", main, short)
            prev, cin = nm + ".add", out_c
    f.avgpool("avgpool", prev)
    f.cblock("fc", "avgpool", 1000, 1, 1, 0, wl("fc"), False, True, False, fc=True, last=True)


def run_fc(seed=0):
    """One FC layer: W, A quantized at WL 8, 6, 4; int32 product requantized at WL 8."""
    W = synth.normal(seed, "fc.w", (256, 512), std=0.05)
    A = synth.relu_normal(seed, "fc.a", (32, 512))
    fmts, outs = {}, {}
    for wl in (8, 6, 4):
        flw, sw, _ = orc.fl_search_f32(W.ravel(), wl, orc.SIGN_AUTO, *FL)
        fla, sa, _ = orc.fl_search_f32(A.ravel(), wl, orc.SIGN_AUTO, *FL)
        wq = orc.quantize_f32(W, wl, flw, sw)
        aq = orc.quantize_f32(A, wl, fla, sa)
        acc = orc.gemm(aq, wq)
        fly, sy, _ = orc.fl_search_i64(acc.ravel(), fla + flw, 8, orc.SIGN_AUTO, *FL)
        y = orc.quantize_i64(acc, fla + flw, 8, fly, sy)
        fmts.update({f"wl{wl}.w": (wl, flw, sw), f"wl{wl}.a": (wl, fla, sa), f"wl{wl}.y": (8, fly, sy)})
        outs[wl] = {"acc": acc, "y": y.ravel().astype(np.int64)}
    return {"fmts": fmts, "logits": outs[8]["y"], "outs": outs}


BODY = {"alexnet": alexnet, "vgg16": vgg16, "resnet18": lambda q: resnet(q, False),
        "resnet50": lambda q: resnet(q, True)}


def run_config(name, seed=None, batch=None, image=None, pcache=None):
    seed = SEED[name] if seed is None else seed
    if name == "fc":
        return run_fc(seed)
    b0, s0 = SHAPE[name]
    batch, image = batch or b0, image or s0
    f = Forward(seed, pcache)
    f.network_input(synth.normal(seed, "input", (batch, 3, image, image)))
    BODY[name](f)
    return f.result()


class Prepared:
    """A workload whose parameters are already quantized: run() times only the
    calibration forward itself."""

    def __init__(self, name, batch, image, seed=None):
        self.name, self.batch, self.image = name, batch, image
        self.seed = SEED[name] if seed is None else seed
        self.pcache = {}
        self.last = run_config(name, self.seed, batch, image, self.pcache)

    def run(self):
        self.last = run_config(self.name, self.seed, self.batch, self.image, self.pcache)
        return self.last


def prepare(name, batch, image, seed=None):
    return Prepared(name, batch, image, seed)

"""DFX calibration forwards of the five workloads through libfxpq.

Each workload is a graph of C-Blocks (Sec. "FxP-QLayer": CONV/FC [+ bias]
[+ Scale] [+ ReLU], Eltwise, AVG-POOL) with an FxP-QLayer after every C-Block
except the last, none after MAX-POOL, and one after the network input.  Every
FxP-QLayer searches its fractional length over the whole batch tensor
(Eq. 14, ties to the larger fl) and requantizes (Eq. 10-12).  Parameters are
quantized once at set-up the same way (weights at their word length, biases
and the Scale shift at 32 bits, the Scale multiplier at 16 bits, Sec.
"Initial Design Generation"); BN layers are turned into Scale layers first
(Eq. 4-5).

Device layouts: activations NHWC int8 codes (storage FXPQ_C8: signed codes as
int8, unsigned ones as u - 128), conv weights KRSC int8, the RGB input padded
to 4 channels.  A forward is a sequence of library calls on one stream with no
host synchronization; formats stay on the device.

Workloads (synthetic, seeded; tensors named as in ``synth``):
  fc        256x512 weights ~N(0, 0.05), 32x512 ReLU(N(0,1)) activations, WL 8/6/4
  alexnet   64x3x224x224, conv 11/5/3 (64-192-384-256-256) + FC 9216-4096-4096-1000
  vgg16     128x3x224x224, 13 conv 3x3 + 3 FC, weight WL per layer from {4..8}
  resnet18  256x3x224x224, BasicBlock [2,2,2,2], BN as Scale, weight WL from {4,6,8}
  resnet50  256x3x224x224, Bottleneck [3,4,6,3] (stride on the 3x3), BN as Scale
"""
import numpy as np

import synth

from . import fxpq as fx

FL_LO, FL_HI = -8, 15
A_WL = 8
BIAS_WL, SCALE_WL, SHIFT_WL, RECIP_WL = 32, 16, 32, 16
BN_EPS = np.float32(1e-5)
SEEDS = {"fc": 0, "alexnet": 1, "vgg16": 2, "resnet18": 3, "resnet50": 4}
DEFAULT_SHAPE = {"alexnet": (64, 224), "vgg16": (128, 224), "resnet18": (256, 224),
                 "resnet50": (256, 224)}


# ----------------------------------------------------------------------------
# Graph description
# ----------------------------------------------------------------------------
class Node:
    def __init__(self, op, name, inp, **kw):
        self.op, self.name, self.inp = op, name, inp
        self.__dict__.update(kw)


def _conv(g, name, inp, cout, k, stride, pad, relu, bias=False, bn=False, wl=8, last=False):
    g.append(Node("conv", name, inp, cout=cout, k=k, stride=stride, pad=pad, relu=relu, bias=bias,
                  bn=bn, wl=wl, last=last))
    return name


def arch_alexnet(seed):
    g = [Node("input", "input", None)]
    x = _conv(g, "conv1", "input", 64, 11, 4, 2, True, bias=True)
    g.append(Node("maxpool", "pool1", x, k=3, stride=2, pad=0)); x = "pool1"
    x = _conv(g, "conv2", x, 192, 5, 1, 2, True, bias=True)
    g.append(Node("maxpool", "pool2", x, k=3, stride=2, pad=0)); x = "pool2"
    x = _conv(g, "conv3", x, 384, 3, 1, 1, True, bias=True)
    x = _conv(g, "conv4", x, 256, 3, 1, 1, True, bias=True)
    x = _conv(g, "conv5", x, 256, 3, 1, 1, True, bias=True)
    g.append(Node("maxpool", "pool5", x, k=3, stride=2, pad=0)); x = "pool5"
    g.append(Node("fc", "fc6", x, cout=4096, relu=True, bias=True, wl=8, last=False))
    g.append(Node("fc", "fc7", "fc6", cout=4096, relu=True, bias=True, wl=8, last=False))
    g.append(Node("fc", "fc8", "fc7", cout=1000, relu=False, bias=True, wl=8, last=True))
    return g


def arch_vgg16(seed):
    plan = [[64, 64], [128, 128], [256, 256, 256], [512, 512, 512], [512, 512, 512]]
    g = [Node("input", "input", None)]
    x = "input"
    for gi, group in enumerate(plan, 1):
        for li, c in enumerate(group, 1):
            name = f"conv{gi}_{li}"
            wl = synth.choice(seed, name + ".wl", [4, 5, 6, 7, 8], 1)[0]
            x = _conv(g, name, x, c, 3, 1, 1, True, bias=True, wl=wl)
        g.append(Node("maxpool", f"pool{gi}", x, k=2, stride=2, pad=0)); x = f"pool{gi}"
    for name, cout, last in [("fc6", 4096, False), ("fc7", 4096, False), ("fc8", 1000, True)]:
        wl = synth.choice(seed, name + ".wl", [4, 5, 6, 7, 8], 1)[0]
        g.append(Node("fc", name, x, cout=cout, relu=not last, bias=True, wl=wl, last=last))
        x = name
    return g


def arch_resnet(seed, depth):
    bottleneck = depth == 50
    blocks = [3, 4, 6, 3] if bottleneck else [2, 2, 2, 2]
    wl_opts = [8] if bottleneck else [4, 6, 8]

    def wl_of(name):
        return synth.choice(seed, name + ".wl", wl_opts, 1)[0] if len(wl_opts) > 1 else wl_opts[0]

    g = [Node("input", "input", None)]
    x = _conv(g, "conv1", "input", 64, 7, 2, 3, True, bn=True, wl=wl_of("conv1"))
    g.append(Node("maxpool", "pool1", x, k=3, stride=2, pad=1)); x = "pool1"
    cin = 64
    for si, (nb, width) in enumerate(zip(blocks, [64, 128, 256, 512]), 1):
        for bi in range(nb):
            stride = 2 if (bi == 0 and si > 1) else 1
            p = f"layer{si}.{bi}"
            cout = width * 4 if bottleneck else width
            if bottleneck:
                a = _conv(g, p + ".c1", x, width, 1, 1, 0, True, bn=True, wl=wl_of(p + ".c1"))
                b = _conv(g, p + ".c2", a, width, 3, stride, 1, True, bn=True, wl=wl_of(p + ".c2"))
                c = _conv(g, p + ".c3", b, cout, 1, 1, 0, False, bn=True, wl=wl_of(p + ".c3"))
            else:
                a = _conv(g, p + ".c1", x, width, 3, stride, 1, True, bn=True, wl=wl_of(p + ".c1"))
                c = _conv(g, p + ".c2", a, width, 3, 1, 1, False, bn=True, wl=wl_of(p + ".c2"))
            if stride != 1 or cin != cout:
                sc = _conv(g, p + ".ds", x, cout, 1, stride, 0, False, bn=True, wl=wl_of(p + ".ds"))
            else:
                sc = x
            g.append(Node("add", p + ".add", c, other=sc, relu=True))
            x = p + ".add"
            cin = cout
    g.append(Node("avgpool", "avgpool", x))
    g.append(Node("fc", "fc", "avgpool", cout=1000, relu=False, bias=True, wl=wl_of("fc"), last=True))
    return g


ARCH = {"alexnet": arch_alexnet, "vgg16": arch_vgg16,
        "resnet18": lambda s: arch_resnet(s, 18), "resnet50": lambda s: arch_resnet(s, 50)}


# ----------------------------------------------------------------------------
# Runner
# ----------------------------------------------------------------------------
FUSE_MAX_DEPTH = 256       # r * s * c of a contraction recomputed by fxpq_cblock
FUSE_MAX_TILES = 61440


def fuse_cblock(desc, Ho, Wo):
    """Whether a conv C-Block runs as one fused fxpq_cblock call: its three
    contraction passes must cost less than storing the int32 accumulators and
    reading them twice, i.e. a shallow contraction (r*s*c <= 256) that reads
    no more input bytes per pass than it has outputs (a strided 1x1 conv reads
    only Ho*Wo of the input pixels)."""
    depth = desc.r * desc.s * desc.c
    M = desc.n * Ho * Wo
    tiles = ((M + 255) // 256) * ((desc.k + 63) // 64) if desc.k <= 64 else \
        ((M + 127) // 128) * ((desc.k + 127) // 128)
    pixels_read = min(desc.h * desc.w, Ho * Wo * desc.r * desc.s)
    return (desc.c % 16 == 0 and depth <= FUSE_MAX_DEPTH and pixels_read * desc.c <= desc.k * Ho * Wo
            and tiles <= FUSE_MAX_TILES)


class CalibNet:
    """One workload resident on the GPU: quantized parameters, activation
    buffers and the input; ``forward()`` enqueues a full calibration forward."""

    def __init__(self, name, seed=None, batch=None, image=None, device="cuda:0", wl_override=None,
                 keep_acts=True, fused=False, qlayer=True, predict=True, defer=True):
        import torch
        self.fused = fused
        self.qlayer = qlayer
        # predicted C-Blocks (fxpq_cblock_predicted) with a rerun of the
        # standard calls from the first miss; defer: their decisions all in
        # one launch at the end of the forward (fxpq_predicted_decide)
        self.predict = predict and qlayer and not fused
        self.defer = defer and self.predict
        self.misses = 0
        self.no_predict = set()  # ops whose window cannot decide alone
        self.torch = torch
        self.name = name
        self.seed = SEEDS[name] if seed is None else seed
        b0, s0 = DEFAULT_SHAPE[name]
        self.batch = batch or b0
        self.image = image or s0
        self.dev = torch.device(device)
        self.h = fx.Handle(self.dev.index or 0)
        fx.set_stream(self.h, torch.cuda.current_stream(self.dev))
        if self.defer:
            fx.predicted_defer(self.h, 1)
        self.graph = ARCH[name](self.seed)
        if wl_override:
            for n in self.graph:
                if n.name in wl_override:
                    n.wl = wl_override[n.name]
        self.keep = []
        self.param_fmts = {}
        self.calls = None
        self.timers = None
        self._build()

    # -- helpers --------------------------------------------------------------
    def _t(self, a, dtype=None):
        t = self.torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)
        self.keep.append(t)
        return t

    def _empty(self, shape, dtype):
        t = self.torch.empty(shape, dtype=dtype, device=self.dev)
        self.keep.append(t)
        return t

    def _fmt(self, wl=0, fl=0, sign=0):
        return self._t(np.array([wl, fl, sign, 0], np.int32))

    def _quant_param(self, key, x32, wl, code_type):
        """FL search + quantization of one parameter tensor on the GPU."""
        T = self.torch
        xd = self._t(x32.astype(np.float32).ravel())
        fmt = self._fmt()
        fx.fl_search(self.h, fx.src_f32(xd), xd.numel(), wl, fx.SIGN_AUTO, FL_LO, FL_HI, fmt)
        dt = {fx.I8: T.int8, fx.I32: T.int32}[code_type]
        codes = self._empty((xd.numel(),), dt)
        fx.quantize(self.h, xd, xd.numel(), fmt, codes, code_type)
        self._pending[key] = fmt
        return codes, fmt

    # -- set-up ----------------------------------------------------------------
    def _build(self):
        T = self.torch
        seed, B, S = self.seed, self.batch, self.image
        self._pending = {}
        shapes = {}  # activation name -> (H, W, C)
        self.act_fmt = {}
        self.act_codes = {}
        x = synth.normal(seed, "input", (B, 3, S, S))
        x4 = np.zeros((B, S, S, 4), np.float32)
        x4[..., :3] = np.transpose(x, (0, 2, 3, 1))
        self.x_dev = self._t(x4)
        shapes["input"] = (S, S, 4)
        self.ops = []
        acc_max = 1
        for n in self.graph:
            if n.op == "input":
                self.act_fmt["input"] = self._fmt()
                self.act_codes["input"] = self._empty((B, S, S, 4), T.int8)
                self.ops.append(("input", n))
            elif n.op in ("conv", "fc"):
                H, W, Cin = shapes[n.inp]
                real_cin = 3 if n.inp == "input" else Cin
                if n.op == "conv":
                    k, st, pd = n.k, n.stride, n.pad
                    w = synth.he_normal(seed, n.name + ".w", (n.cout, real_cin, k, k))
                    wk = np.transpose(w, (0, 2, 3, 1))  # KRSC
                    if n.inp == "input":
                        wk = np.concatenate([wk, np.zeros((n.cout, k, k, 1), np.float32)], axis=3)
                    wk = wk.reshape(n.cout, -1)
                    if Cin == 4:
                        kp = (wk.shape[1] + 63) // 64 * 64
                        wk = np.concatenate([wk, np.zeros((n.cout, kp - wk.shape[1]), np.float32)], 1)
                    Ho, Wo = (H + 2 * pd - k) // st + 1, (W + 2 * pd - k) // st + 1
                    desc = fx.conv_desc(B, H, W, Cin, n.cout, k, k, st, pd)
                    M = B * Ho * Wo
                else:
                    fan_in = H * W * Cin
                    w = synth.he_normal(seed, n.name + ".w", (n.cout, fan_in))
                    # canonical flatten is (c, h, w); activations here are (h, w, c)
                    wk = w.reshape(n.cout, Cin, H, W).transpose(0, 2, 3, 1).reshape(n.cout, fan_in)
                    Ho = Wo = 1
                    desc = None
                    M = B
                wcodes, wfmt = self._quant_param(n.name + ".w", wk, n.wl, fx.I8)
                colsum = self._empty((n.cout,), T.int32)
                fx.weight_colsum(self.h, wcodes, n.cout, wk.shape[1], colsum)
                p = {"w": wcodes, "colsum": colsum, "wlen": wk.shape[1], "desc": desc, "M": M,
                     "Ho": Ho, "Wo": Wo, "Cin": Cin}
                if n.bias:
                    b = synth.normal(seed, n.name + ".b", (n.cout,), std=0.01)
                    p["b"], _ = self._quant_param(n.name + ".b", b, BIAS_WL, fx.I32)
                if getattr(n, "bn", False):
                    gamma = synth.uniform(seed, n.name + ".bn.gamma", (n.cout,), 0.5, 1.5)
                    beta = synth.normal(seed, n.name + ".bn.beta", (n.cout,), std=0.1)
                    mean = np.zeros(n.cout, np.float32)
                    var = np.ones(n.cout, np.float32)
                    inv = np.sqrt(var + BN_EPS)
                    a1 = (gamma / inv).astype(np.float32)           # Eq. 5
                    a2 = (beta - gamma * mean / inv).astype(np.float32)
                    p["a1"], _ = self._quant_param(n.name + ".a1", a1, SCALE_WL, fx.I32)
                    p["a2"], _ = self._quant_param(n.name + ".a2", a2, SHIFT_WL, fx.I32)
                acc_max = max(acc_max, M * n.cout)
                # min / max of the C-Block values; NaN: no prediction yet
                p["mm"] = self._empty((2,), T.float64)
                p["mm"].fill_(float("nan"))
                if not n.last:
                    self.act_fmt[n.name] = self._fmt()
                    self.act_codes[n.name] = self._empty((B, Ho, Wo, n.cout), T.int8)
                    shapes[n.name] = (Ho, Wo, n.cout)
                self.ops.append((n.op, n, p))
            elif n.op == "maxpool":
                H, W, C = shapes[n.inp]
                Ho, Wo = (H + 2 * n.pad - n.k) // n.stride + 1, (W + 2 * n.pad - n.k) // n.stride + 1
                self.act_fmt[n.name] = self.act_fmt[n.inp]
                self.act_codes[n.name] = self._empty((B, Ho, Wo, C), T.int8)
                shapes[n.name] = (Ho, Wo, C)
                self.ops.append(("maxpool", n, {"H": H, "W": W, "C": C}))
            elif n.op == "add":
                shapes[n.name] = shapes[n.inp]
                self.act_fmt[n.name] = self._fmt()
                self.act_codes[n.name] = self._empty((B,) + shapes[n.inp], T.int8)
                mm = self._empty((2,), T.float64)
                mm.fill_(float("nan"))  # no prediction yet
                self.ops.append(("add", n, {"mm": mm}))
            elif n.op == "avgpool":
                H, W, C = shapes[n.inp]
                r = np.array([np.float32(1.0) / np.float32(H * W)], np.float32)
                rcodes, rfmt = self._quant_param("avgpool.recip", np.repeat(r, 4), RECIP_WL, fx.I32)
                self.ops.append(("avgpool", n, {"HW": H * W, "C": C, "rcodes": rcodes,
                                                "sum": self._empty((B, C), T.int64),
                                                "scale": self._empty((1,), T.int32)}))
                shapes[n.name] = (1, 1, C)
                self.act_fmt[n.name] = self._fmt()
                self.act_codes[n.name] = self._empty((B, 1, 1, C), T.int8)
        self.acc = self._empty((acc_max,), T.int32)
        # alternate codes of the fused FxP-QLayer calls (one tensor's worth)
        code_max = max(c.numel() for c in self.act_codes.values())
        self.code_alt = self._empty((code_max + 16,), T.int8)
        self.logits = None
        # parameter formats back to the host (once)
        T.cuda.synchronize(self.dev)
        for key, f in self._pending.items():
            wl, fl, sign, st = (int(v) for v in f.cpu().numpy())
            if st:
                raise RuntimeError(f"parameter {key}: fractional-length search failed ({st})")
            self.param_fmts[key] = (wl, fl, sign)
        for op, n, *rest in self.ops:
            if op in ("conv", "fc"):
                p = rest[0]
                fin = self.act_fmt[n.inp]
                fw = self.param_fmts[n.name + ".w"][1]
                kw = {}
                if n.bias:
                    kw.update(bias=p["b"], fl_bias=self.param_fmts[n.name + ".b"][1])
                if getattr(n, "bn", False):
                    kw.update(scale=p["a1"], fl_scale=self.param_fmts[n.name + ".a1"][1],
                              shift=p["a2"], fl_shift=self.param_fmts[n.name + ".a2"][1])
                p["ep"] = fx.epilogue(n.cout, fw, fin, relu=n.relu, **kw)
                if n.last:
                    p["logit_fmt"] = self._t(np.array([32, 0, 1, 0], np.int32))
                    self.logits = self._empty((p["M"], n.cout), T.int32)
            elif op == "avgpool":
                p = rest[0]
                p["recip"] = int(p["rcodes"].cpu().numpy()[0])
                p["ep_scale"] = fx.epilogue(p["C"], self.param_fmts["avgpool.recip"][1],
                                            self.act_fmt[n.inp])
        self.n_input = self.x_dev.numel()
        self.le_out = self._empty((4,), T.float64)
        self.miss = self._empty((len(self.ops),), T.int32)
        self.miss.zero_()
        self.input_mm = self._empty((2,), T.float64)
        self.input_mm.fill_(float("nan"))

    # -- forward ---------------------------------------------------------------
    def _fused_conv(self, n, p):
        """Whether conv node n runs as one fused fxpq_cblock call."""
        return (n.op == "conv" and not n.last and self.fused
                and fuse_cblock(p["desc"], p["Ho"], p["Wo"]))

    def _plan(self):
        """Pre-builds every library call of one forward: (class, work, fn, args).
        `work` is the call's algorithmic HBM bytes (streaming calls) or int8
        operations (conv / FC), used for the roofline report."""
        import ctypes as C
        L = fx.lib()
        h, B = self.h.value, self.batch
        calls = []

        def add(cls, work, fn, *args):
            calls.append((cls, work, fn, args))

        keep = self.keep
        # Each residual add takes its min / max from the requantization of the
        # operand produced last, when that is an unfused conv C-Block.
        produced_at = {n.name: i for i, (op, n, *r) in enumerate(self.ops)}
        addmm = {}
        for op, n, *rest in self.ops:
            if op == "add" and not self.qlayer:
                last = max((n.inp, n.other), key=lambda nm: produced_at[nm])
                first = n.other if last == n.inp else n.inp
                lop, ln, *lr = self.ops[produced_at[last]]
                if lop == "conv" and not ln.last and not self._fused_conv(ln, lr[0]):
                    addmm[last] = (n, first, rest[0]["mm"])
        self.addmm_adds = {v[0].name for v in addmm.values()}
        self.starts = []
        for op, n, *rest in self.ops:
            self.starts.append(len(calls))
            if op == "input":
                f, c = self.act_fmt["input"], self.act_codes["input"]
                src = fx.src_f32(self.x_dev)
                keep.append(src)
                if self.qlayer:
                    add("fl_search_f32", 5 * self.n_input, L.fxpq_qlayer, h, C.byref(src), self.n_input,
                        A_WL, fx.SIGN_AUTO, FL_LO, FL_HI, f.data_ptr(), c.data_ptr(), fx.C8,
                        self.code_alt.data_ptr())
                else:
                    add("fl_search_f32", 4 * self.n_input, L.fxpq_fl_search, h, C.byref(src),
                        self.n_input, A_WL, fx.SIGN_AUTO, FL_LO, FL_HI, f.data_ptr(), None)
                    add("quantize", 5 * self.n_input, L.fxpq_quantize, h, self.x_dev.data_ptr(),
                        self.n_input, f.data_ptr(), c.data_ptr(), fx.C8)
                add("layer_error", 5 * self.n_input, L.fxpq_layer_error, h, self.x_dev.data_ptr(),
                    c.data_ptr(), fx.C8, f.data_ptr(), self.n_input, self.le_out.data_ptr())
            elif op in ("conv", "fc"):
                p = rest[0]
                xin = self.act_codes[n.inp]
                n_out = p["M"] * n.cout
                acc = self.acc[:n_out]
                keep.append(acc)
                ops2 = 2 * n_out * p["wlen"]
                if self._fused_conv(n, p):
                    # shallow contraction, wide output: recompute instead of an
                    # int32 round trip (same formats and codes bit for bit)
                    f = self.act_fmt[n.name]
                    add("cblock", ops2, L.fxpq_cblock, h, C.byref(p["desc"]), xin.data_ptr(), fx.C8,
                        p["w"].data_ptr(), p["colsum"].data_ptr(), C.byref(p["ep"]), A_WL,
                        fx.SIGN_AUTO, FL_LO, FL_HI, f.data_ptr(), self.act_codes[n.name].data_ptr(),
                        fx.C8, acc.data_ptr(), p["mm"].data_ptr())
                    continue
                if op == "conv":
                    add("qconv", ops2, L.fxpq_qconv, h, C.byref(p["desc"]), xin.data_ptr(), fx.C8,
                        p["w"].data_ptr(), p["colsum"].data_ptr(), C.byref(p["ep"]), acc.data_ptr(),
                        p["mm"].data_ptr())
                else:
                    add("qconv", ops2, L.fxpq_qgemm, h, p["M"], n.cout, p["wlen"], xin.data_ptr(), fx.C8,
                        p["w"].data_ptr(), p["colsum"].data_ptr(), C.byref(p["ep"]), acc.data_ptr(),
                        p["mm"].data_ptr())
                src = fx.src_acc(acc, p["ep"], p["mm"])
                keep.append(src)
                if n.last:
                    add("other", 0, L.fxpq_epilogue_scale, h, C.byref(p["ep"]),
                        p["logit_fmt"].data_ptr() + 4)
                    add("requant", 8 * n_out, L.fxpq_requant, h, C.byref(src), n_out,
                        p["logit_fmt"].data_ptr(), self.logits.data_ptr(), fx.I32)
                elif self.qlayer:
                    # FL search + requantization, one read of the accumulators
                    add("fl_search", 5 * n_out, L.fxpq_qlayer, h, C.byref(src), n_out, A_WL,
                        fx.SIGN_AUTO, FL_LO, FL_HI, self.act_fmt[n.name].data_ptr(),
                        self.act_codes[n.name].data_ptr(), fx.C8, self.code_alt.data_ptr())
                else:
                    f = self.act_fmt[n.name]
                    add("fl_search", 4 * n_out, L.fxpq_fl_search, h, C.byref(src), n_out, A_WL,
                        fx.SIGN_AUTO, FL_LO, FL_HI, f.data_ptr(), None)
                    if n.name in addmm:
                        an, other, mm = addmm[n.name]
                        add("requant", 6 * n_out, L.fxpq_requant_addmm, h, C.byref(src), n_out,
                            f.data_ptr(), self.act_codes[n.name].data_ptr(), fx.C8,
                            self.act_codes[other].data_ptr(), fx.C8, self.act_fmt[other].data_ptr(),
                            int(an.relu), mm.data_ptr())
                    else:
                        add("requant", 5 * n_out, L.fxpq_requant, h, C.byref(src), n_out, f.data_ptr(),
                            self.act_codes[n.name].data_ptr(), fx.C8)
            elif op == "maxpool":
                p = rest[0]
                out = self.act_codes[n.name]
                add("other", self.act_codes[n.inp].numel() + out.numel(), L.fxpq_maxpool, h,
                    self.act_codes[n.inp].data_ptr(), fx.C8, B, p["H"], p["W"], p["C"], n.k, n.stride,
                    n.pad, out.data_ptr())
            elif op == "add":
                a, b = self.act_codes[n.inp], self.act_codes[n.other]
                mm = rest[0]["mm"] if n.name in self.addmm_adds else None
                src = fx.src_add(a, fx.C8, self.act_fmt[n.inp], b, fx.C8, self.act_fmt[n.other], n.relu,
                                 mm)
                keep.append(src)
                f = self.act_fmt[n.name]
                m = a.numel()
                if self.qlayer:
                    add("fl_search", 3 * m, L.fxpq_qlayer, h, C.byref(src), m, A_WL, fx.SIGN_AUTO,
                        FL_LO, FL_HI, f.data_ptr(), self.act_codes[n.name].data_ptr(), fx.C8,
                        self.code_alt.data_ptr())
                    continue
                add("fl_search", 2 * m, L.fxpq_fl_search, h, C.byref(src), m, A_WL, fx.SIGN_AUTO,
                    FL_LO, FL_HI, f.data_ptr(), None)
                add("requant", 3 * m, L.fxpq_requant, h, C.byref(src), m, f.data_ptr(),
                    self.act_codes[n.name].data_ptr(), fx.C8)
            elif op == "avgpool":
                p = rest[0]
                add("other", self.act_codes[n.inp].numel(), L.fxpq_avgpool_global, h,
                    self.act_codes[n.inp].data_ptr(), fx.C8, self.act_fmt[n.inp].data_ptr(), B, p["HW"],
                    p["C"], p["recip"], p["sum"].data_ptr())
                add("other", 0, L.fxpq_epilogue_scale, h, C.byref(p["ep_scale"]), p["scale"].data_ptr())
                src = fx.src_int(p["sum"], fx.I64, p["scale"])
                keep.append(src)
                f = self.act_fmt[n.name]
                m = p["sum"].numel()
                add("fl_search", 8 * m, L.fxpq_fl_search, h, C.byref(src), m, A_WL, fx.SIGN_AUTO,
                    FL_LO, FL_HI, f.data_ptr(), None)
                add("requant", 9 * m, L.fxpq_requant, h, C.byref(src), m, f.data_ptr(),
                    self.act_codes[n.name].data_ptr(), fx.C8)
        self.starts.append(len(calls))
        if self.predict:
            self.pcalls = self._plan_predicted(calls)
        return calls

    def _predictable(self, op, n, p):
        """A C-Block followed by its FxP-QLayer whose contraction the
        predicted C-Block takes (channels a multiple of 16, or the padded
        RGB layout of a first conv)."""
        if op not in ("conv", "fc") or n.last:
            return False
        cin = p["Cin"] if op == "conv" else p["wlen"]
        return cin % 16 == 0 or (op == "conv" and cin == 4)

    def _plan_predicted(self, calls):
        """The forward with every predictable C-Block as one
        fxpq_cblock_predicted call (its miss flag: element i of self.miss for
        op i); the other ops' calls as in the standard plan."""
        import ctypes as C
        L = fx.lib()
        h = self.h.value
        out = []
        for i, (op, n, *rest) in enumerate(self.ops):
            miss = self.miss.data_ptr() + 4 * i
            if i in self.no_predict:
                out += calls[self.starts[i]:self.starts[i + 1]]
                continue
            if op == "input" or (op == "add" and n.name not in self.addmm_adds):
                # the FxP-QLayer of the network input / of an eltwise sum:
                # predicted from its previous min / max and format
                std = calls[self.starts[i]:self.starts[i + 1]]
                if op == "input":
                    src, m, mm = fx.src_f32(self.x_dev), self.n_input, self.input_mm
                else:
                    a, b = self.act_codes[n.inp], self.act_codes[n.other]
                    src = fx.src_add(a, fx.C8, self.act_fmt[n.inp], b, fx.C8, self.act_fmt[n.other],
                                     n.relu)
                    m, mm = a.numel(), rest[0]["mm"]
                self.keep.append(src)
                out.append(("fl_search", std[0][1], L.fxpq_qlayer_predicted,
                            (h, C.byref(src), m, A_WL, fx.SIGN_AUTO, FL_LO, FL_HI,
                             self.act_fmt[n.name].data_ptr(), self.act_codes[n.name].data_ptr(),
                             fx.C8, mm.data_ptr(), miss)))
                out += std[1:]  # the input's layer error
                continue
            if not rest or not self._predictable(op, n, rest[0]):
                out += calls[self.starts[i]:self.starts[i + 1]]
                continue
            p = rest[0]
            desc = p["desc"] if op == "conv" else fx.conv_desc(p["M"], 1, 1, p["wlen"], n.cout, 1, 1, 1, 0)
            self.keep.append(desc)
            n_out = p["M"] * n.cout
            out.append(("cblock_pred", 2 * n_out * p["wlen"], L.fxpq_cblock_predicted,
                        (h, C.byref(desc), self.act_codes[n.inp].data_ptr(), fx.C8, p["w"].data_ptr(),
                         p["colsum"].data_ptr(), C.byref(p["ep"]), A_WL, fx.SIGN_AUTO, FL_LO, FL_HI,
                         self.act_fmt[n.name].data_ptr(), self.act_codes[n.name].data_ptr(), fx.C8,
                         p["mm"].data_ptr(), miss)))
        return out

    def prepare_timers(self, steps, classes=("fl_search",)):
        """Pre-creates HIP events so that the next `steps` forwards bracket every
        call of the given classes without allocating anything while timed."""
        if self.calls is None:
            self.calls = self._plan()
        T = self.torch
        # a predicted forward may also rerun standard calls
        per_step = sum(1 for c in self.calls if c[0] in classes)
        if self.predict:
            per_step += sum(1 for c in self.pcalls if c[0] in classes)
        self.timed_classes = set(classes)
        self.event_pool = [(T.cuda.Event(enable_timing=True), T.cuda.Event(enable_timing=True))
                           for _ in range(per_step * steps)]
        self.timers = []

    def forward(self, predict=None):
        """Enqueues one calibration forward.  Standard plan: no host
        synchronization.  With predicted C-Blocks: the predicted plan, one
        host synchronization to read the miss flags, and when a prediction
        failed the standard calls again from the first op that missed (every
        later op depended on it), so the results are always those of the
        standard plan.  With defer, the predicted calls' decisions run as one
        launch after the last of them.  predict=False runs the standard plan on a predicting
        net (a caller that changed formats or data knows the predictions will
        fail).  After prepare_timers(), calls of the timed classes are
        bracketed by HIP events on the library's stream and (class, work,
        start, end) is recorded."""
        if self.calls is None:
            self.calls = self._plan()
        if not self.predict or predict is False:
            self._run(self.calls)
            return
        self._run(self.pcalls)
        if self.defer:
            fx.predicted_decide(self.h)
        miss = self.miss.cpu().numpy()
        if miss.any():
            first = int(np.flatnonzero(miss)[0])
            self.miss.zero_()
            self.misses += 1
            self._run(self.calls[self.starts[first]:])
            if miss[first] == 2:
                # predicted right but undecidable by the window: this op runs
                # the standard calls from now on
                self.no_predict.add(first)
                self.pcalls = self._plan_predicted(self.calls)

    def _run(self, calls):
        timers = self.timers
        if timers is None:
            for cls, work, fn, args in calls:
                st = fn(*args)
                if st:
                    raise fx.FxpqError(fn.__name__, st)
            return
        timed = self.timed_classes
        pool = self.event_pool
        for cls, work, fn, args in calls:
            if cls in timed:
                e0, e1 = pool[len(timers)]
                e0.record()
                st = fn(*args)
                e1.record()
                timers.append((cls, work, e0, e1))
            else:
                st = fn(*args)
            if st:
                raise fx.FxpqError(fn.__name__, st)

    def kernel_times(self):
        """Per call class: (calls, total ms, total work) from the recorded events."""
        self.torch.cuda.synchronize(self.dev)
        agg = {}
        for cls, work, e0, e1 in self.timers or []:
            c, t, w = agg.get(cls, (0, 0.0, 0))
            agg[cls] = (c + 1, t + e0.elapsed_time(e1), w + work)
        return agg

    def roofline(self, peak_hbm_gbs=8000.0, peak_int8_tops=5000.0):
        """Roofline entry for the class with the largest total time."""
        agg = self.kernel_times()
        if not agg:
            return {}
        cls = max(agg, key=lambda k: agg[k][1])
        calls, ms, work = agg[cls]
        if cls == "qconv":
            ach = work / (ms * 1e-3) / 1e12
            r = {"bound": "mfma", "achieved": round(ach, 2), "peak": peak_int8_tops, "unit": "TOP/s",
                 "frac": round(ach / peak_int8_tops, 4)}
        else:
            ach = work / (ms * 1e-3) / 1e9
            r = {"bound": "hbm", "achieved": round(ach, 1), "peak": peak_hbm_gbs, "unit": "GB/s",
                 "frac": round(ach / peak_hbm_gbs, 4)}
        r.update({"kernel": cls, "launches": calls, "avg_launch_ms": round(ms / calls, 4),
                  "traffic": None, "breakdown_ms": {k: round(v[1], 3) for k, v in agg.items()}})
        return r

    # -- results ---------------------------------------------------------------
    def results(self, with_codes=False):
        T = self.torch
        T.cuda.synchronize(self.dev)
        flags = fx.sync_status(self.h)
        fmts = dict(self.param_fmts)
        for name, f in self.act_fmt.items():
            if name.startswith("pool"):
                continue
            wl, fl, sign, st = (int(v) for v in f.cpu().numpy())
            fmts[name] = (wl, fl, sign)
        last = [p for op, n, *r in self.ops if op in ("conv", "fc") and n.last for p in r][0]
        out = {"fmts": fmts, "logits": self.logits.cpu().numpy().astype(np.int64),
               "logit_fl": int(last["logit_fmt"].cpu().numpy()[1]), "flags": flags,
               "input_error": self.le_out.cpu().numpy()}
        if with_codes:
            codes = {}
            for name, c in self.act_codes.items():
                if name.startswith("pool"):
                    continue
                sign = fmts[name][2]
                a = c.cpu().numpy().astype(np.int64)
                codes[name] = a + 128 if sign == 0 else a
            out["codes"] = codes
        return out

    def close(self):
        self.h.close()


def run_fc(seed=0, device="cuda:0"):
    """The single-FC-layer workload: one FC layer, W and A quantized at WL 8, 6 and 4, the
    int32 product requantized to WL 8 with its own search."""
    import torch
    dev = torch.device(device)
    h = fx.Handle(dev.index or 0)
    fx.set_stream(h, torch.cuda.current_stream(dev))
    W = synth.normal(seed, "fc.w", (256, 512), std=0.05)
    A = synth.relu_normal(seed, "fc.a", (32, 512))
    Wd = torch.from_numpy(W.ravel()).to(dev)
    Ad = torch.from_numpy(A.ravel()).to(dev)
    fmts, outs, keep = {}, {}, []
    for wl in (8, 6, 4):
        fw = torch.zeros(4, dtype=torch.int32, device=dev)
        fa = torch.zeros(4, dtype=torch.int32, device=dev)
        fy = torch.zeros(4, dtype=torch.int32, device=dev)
        fx.fl_search(h, fx.src_f32(Wd), Wd.numel(), wl, fx.SIGN_AUTO, FL_LO, FL_HI, fw)
        fx.fl_search(h, fx.src_f32(Ad), Ad.numel(), wl, fx.SIGN_AUTO, FL_LO, FL_HI, fa)
        wc = torch.empty(Wd.numel(), dtype=torch.int8, device=dev)
        ac = torch.empty(Ad.numel(), dtype=torch.int8, device=dev)
        fx.quantize(h, Wd, Wd.numel(), fw, wc, fx.I8)
        fx.quantize(h, Ad, Ad.numel(), fa, ac, fx.C8)
        cs = torch.empty(256, dtype=torch.int32, device=dev)
        fx.weight_colsum(h, wc, 256, 512, cs)
        torch.cuda.synchronize(dev)
        fl_w = int(fw.cpu()[1])
        ep = fx.epilogue(256, fl_w, fa)
        acc = torch.empty((32, 256), dtype=torch.int32, device=dev)
        mm = torch.empty(2, dtype=torch.float64, device=dev)
        fx.qgemm(h, 32, 256, 512, ac, fx.C8, wc, cs, ep, acc, mm)
        src = fx.src_acc(acc, ep, mm)
        fx.fl_search(h, src, acc.numel(), 8, fx.SIGN_AUTO, FL_LO, FL_HI, fy)
        yc = torch.empty(acc.numel(), dtype=torch.int8, device=dev)
        fx.requant(h, src, acc.numel(), fy, yc, fx.C8)
        torch.cuda.synchronize(dev)
        for key, f in (("w", fw), ("a", fa), ("y", fy)):
            wl_, fl_, sg_, st_ = (int(v) for v in f.cpu().numpy())
            fmts[f"wl{wl}.{key}"] = (wl_, fl_, sg_)
        sy = fmts[f"wl{wl}.y"][2]
        outs[wl] = {"acc": acc.cpu().numpy().astype(np.int64),
                    "y": yc.cpu().numpy().astype(np.int64) + (128 if sy == 0 else 0)}
        keep += [fw, fa, fy, wc, ac, cs, acc, mm, yc]
    flags = fx.sync_status(h)
    h.close()
    return {"fmts": fmts, "logits": outs[8]["y"], "outs": outs, "flags": flags}


def run_config(name, seed=None, device="cuda:0", batch=None, image=None, with_codes=False,
               wl_override=None, fused=False, qlayer=True):
    if name == "fc":
        return run_fc(SEEDS["fc"] if seed is None else seed, device)
    net = CalibNet(name, seed, batch, image, device, wl_override=wl_override, fused=fused,
                   qlayer=qlayer)
    net.forward()
    res = net.results(with_codes=with_codes)
    net.close()
    return res

"""Oracle of the forward optimizer with Algorithm 1 (QParamsOpt) -- TEST
INFRASTRUCTURE ONLY.

Sec. "Quantization Parameters Optimization", Algorithm 1, Eq. 15-21, written
from the text in NCHW with the oracle's own operations: for every data
structure in order (the input image; then per conv / FC layer its weights,
bias and output activations), starting from the preprocessor's initial
format (Eq. 6-9, conservative rounding), step the fractional length away in
each direction (alpha + beta fixed), evaluating each candidate by running the
calibration batch with earlier layers quantized at their chosen formats, the
current layer at the candidate and later layers in FP32 (the order-fixed
teacher), and keep the smallest cost

    F = sum_{i >= l} sum_j pi_i^j L(X_i^j) / R_i^j + UnClass + MisPred;

a direction continues K steps past its last improvement.

The same readings as the GPU driver: activations are layer outputs, the
input image is the first data structure; a C-Block's data structures are
its output activations, its conv / FC weights and bias, and its Scale
parameters aleph_1 / aleph_2 (Eq. 4-5), optimized in the order w, b,
aleph_1, aleph_2, a; L is the parameter quantization error for the current
layer (zero for FP32 layers) and the distance from the teacher's activation
for activations; pi = sigma * nu normalized over a layer's data structures
(Eq. 15), where for activations sigma is the population standard deviation
of each calibration sample averaged over the samples and nu is the size of
one sample, and for parameters both are taken over the tensor (Eq. 16); R =
max - min of the FP32 data structure over the whole batch (Eq. 18);
eltwise / avg-pool FxP-QLayers keep their Eq. 14 searches.  Any of the
workloads' networks; the FP32 FC sums the flattened input channel-major, the
GPU's order whenever the FC input is 1x1 spatially (the ResNets, and AlexNet
/ VGG-16 on the small images of the parity tests).

The statistics, pi and E (Eq. 15-17) are pinned on a hand-worked two-sample
layer (tests/golden/importance_pi.txt); the search rule on hand-worked cost
curves and against brute force (tests/test_oracle_qparams.py).  parity
unpinned for the network cost F as composed over a network (no printed
example exists): its parts are pinned (tests/test_oracle_preprocess.py,
tests/test_oracle_pins.py, tests/test_oracle_teacher.py and the above).
"""
import math

import numpy as np

import synth

from . import core as orc
from . import preprocess as pre
from .nets import FL, SEED, alexnet, resnet, vgg16

BUILD = {"alexnet": alexnet, "vgg16": vgg16, "resnet18": lambda g: resnet(g, False),
         "resnet50": lambda g: resnet(g, True)}
from .sweep import Teacher

# The Scale parameters of a C-Block (Eq. 4-5) as data structures: s1 is the
# multiplier aleph_1 (16 bits, the C-Block's 16-bit multiplier), s2 the
# offset aleph_2 (32 bits); both learnable parameters outside G1 (Eq. 22).
PARAM = {"s1": "a1", "s2": "a2"}
SCALE_WL = {"s1": 16, "s2": 32}


class Graph(Teacher):
    """The FP32 teacher, also recording every node in order."""

    def __init__(self, seed):
        super().__init__(seed)
        self.nodes = []

    def network_input(self, x):
        super().network_input(x)
        self.x = x
        self.nodes.append(("input", "input", {}))

    def cblock(self, name, src, cout, k, stride, pad, wl, relu, bias, bn, fc=False, last=False):
        super().cblock(name, src, cout, k, stride, pad, wl, relu, bias, bn, fc, last)
        spec = self.layers[-1][2]
        spec.update(wl=wl, cout=cout, src=src)
        self.nodes.append(("conv", name, spec))

    def maxpool(self, name, src, k, stride, pad):
        super().maxpool(name, src, k, stride, pad)
        self.nodes.append(("maxpool", name, {"src": src, "k": k, "stride": stride, "pad": pad}))

    def add(self, name, a, b):
        super().add(name, a, b)
        self.nodes.append(("add", name, {"a": a, "b": b}))

    def avgpool(self, name, src):
        super().avgpool(name, src)
        self.nodes.append(("avgpool", name, {"src": src}))


def _stats(x, per_sample=False):
    """(sigma, nu, R) of one data structure.  Eq. 16: sigma is the population
    standard deviation about the arithmetic mean and nu the size; for
    activations (per_sample, x holding the calibration samples along its
    first axis) sigma is taken per sample and averaged over the samples,
    and nu is the size of one sample (Eq. 15-16 and the text after them).
    Eq. 18: R = largest minus smallest FP32 value of the whole data
    structure."""
    x = np.asarray(x, np.float64)
    flat = x.ravel()
    rng = float(flat.max() - flat.min())
    if per_sample:
        per = x.reshape(x.shape[0], -1)
        sig = [float(np.sqrt(np.mean((r - r.mean()) ** 2))) for r in per]
        return float(np.mean(sig)), per.shape[1], rng
    return float(np.sqrt(np.mean((flat - flat.mean()) ** 2))), flat.size, rng


def importance(stats):
    """Eq. 15: pi of each data structure of one layer, sigma * nu normalized
    so that the layer's values sum to one.  stats: {key: (sigma, nu, R)}."""
    tot = sum(sg * nu for sg, nu, _ in stats.values())
    return {k: (sg * nu / tot if tot > 0 else 0.0) for k, (sg, nu, _) in stats.items()}


def distillation_error(pi, stat, errs):
    """Eq. 17: sum of pi * L / R over the data structures with an error
    (errs: {key: L}); a data structure with R = 0 (constant) adds nothing."""
    return sum(pi[k] * e / stat[k][2] for k, e in errs.items() if k in pi and stat[k][2] > 0)


def _sse(ref, y):
    d = np.asarray(ref, np.float64).ravel() - np.asarray(y, np.float64).ravel()
    return math.fsum(d * d)


def _dec(q, wl, sign):
    """Eq. 13: the 1-bit signed code 0 stands for +1 (the values the
    arithmetic uses); other formats use their codes as they are."""
    if wl == 1 and sign == 1:
        return np.where(np.asarray(q) == 0, 1, -1).astype(np.int64)
    return q


def _ties(scores):
    s = np.asarray(scores).reshape(scores.shape[0], -1)
    c = (s == s.max(axis=1, keepdims=True)).sum(axis=1)
    return int((c > 1).sum()), int((c - 1).sum())


class ForwardOptimizer:
    def __init__(self, name="resnet18", seed=None, batch=2, image=32, K=1,
                 strategy=pre.CONSERVATIVE, w_wl=None, first_last_wl=None):
        self.seed = SEED[name] if seed is None else seed
        g = Graph(self.seed)
        g.network_input(synth.normal(self.seed, "input", (batch, 3, image, image)))
        BUILD[name](g)
        self.g, self.K, self.B, self.w_wl = g, K, batch, w_wl
        # the network input, the first and last layers' weights and the last
        # layer's input (avg-pool FxP-QLayer) at this word length when given
        self.fl_wl = first_last_wl
        convs = [nm for op, nm, _ in g.nodes if op == "conv"]
        self.edge = (convs[0], convs[-1])
        self.spec = {nm: sp for op, nm, sp in g.nodes if op == "conv"}
        # per C-Block: weights, bias, Scale multiplier (s1 = aleph_1) and
        # offset (s2 = aleph_2), in the order the C-Block applies them, then
        # the output activations (none for the last layer)
        self.order = [("input", "a")]
        for op, nm, sp in g.nodes:
            if op == "conv":
                self.order.append((nm, "w"))
                if "b" in sp:
                    self.order.append((nm, "b"))
                if "a1" in sp:
                    self.order += [(nm, "s1"), (nm, "s2")]
                if not sp["last"]:
                    self.order.append((nm, "a"))
        self.qp, self.stat = {}, {}
        last = [nm for nm, sp in self.spec.items() if sp["last"]][0]
        for ln, d in self.order + [(last, "a")]:
            x, wl = self._tensor(ln, d)
            xmin, xmax = pre.exact_extremes_f32(x)
            fl, sign = pre.init_fl(xmin, xmax, wl, strategy, pre.PSI_PRINTED, *FL)
            self.qp[(ln, d)] = [wl, fl, sign]
            self.stat[(ln, d)] = _stats(x, per_sample=(d == "a"))
        # Eq. 15, normalized over each layer's data structures
        self.pi = {}
        for ln in ["input"] + list(self.spec):
            self.pi.update(importance({k: v for k, v in self.stat.items() if k[0] == ln}))
        self.q = {}  # finalized nodes: (codes, fl, sign) NCHW
        self._pcache = {}
        self.trace = []
        self.last = last

    def _tensor(self, ln, d):
        if ln == "input":
            return self.g.x, self.fl_wl or 8
        sp = self.spec[ln]
        if d == "w":
            if self.fl_wl is not None and ln in self.edge:
                return sp["w"], self.fl_wl
            return sp["w"], self.w_wl or sp["wl"]
        if d == "b":
            return sp["b"], 32
        if d in PARAM:
            return sp[PARAM[d]], SCALE_WL[d]
        return self.g.act[ln], 8

    # ---- one quantized layer ----
    def _param(self, ln, d):
        """Codes (Eq. 12-13) and squared error of parameter d of layer ln at
        its current format (kept per format: parameters do not change)."""
        wl, fl, sign = self.qp[(ln, d)]
        hit = self._pcache.get((ln, d))
        if hit is not None and hit[0] == (wl, fl, sign):
            return hit[1], hit[2]
        x = self.spec[ln][PARAM.get(d, d)]
        c = orc.quantize_f32(x, wl, fl, sign).astype(np.int64)
        e = orc.layer_error(x.ravel(), c.ravel(), wl, fl, sign)[0]
        self._pcache[(ln, d)] = ((wl, fl, sign), c, e)
        return c, e

    def _quant_layer(self, ln, q=None):
        """(codes, fl, sign, errors {key: sse}) of layer ln at the current
        formats, its input taken from q (default: the finalized prefix).  The
        codes returned are the values the next layer multiplies (Eq. 13
        decoded); the errors use the codes as Eq. 12-13 define them."""
        q = self.q if q is None else q
        if ln == "input":
            wl, fl, sign = self.qp[("input", "a")]
            c = orc.quantize_f32(self.g.x, wl, fl, sign)
            return (_dec(c, wl, sign), fl, sign,
                    {("input", "a"): orc.layer_error(self.g.x.ravel(), c.ravel(), wl, fl, sign)[0]})
        sp = self.spec[ln]
        errs = {}
        x, fl_x, _ = q[sp["src"]]
        ww, flw, sw = self.qp[(ln, "w")]
        wc, errs[(ln, "w")] = self._param(ln, "w")
        wq = _dec(wc, ww, sw)
        b = a1 = a2 = None
        fl_b = fl_a1 = fl_a2 = 0
        if "b" in sp:
            bw, fl_b, sb = self.qp[(ln, "b")]
            bc, errs[(ln, "b")] = self._param(ln, "b")
            b = _dec(bc, bw, sb)
        if "a1" in sp:
            w1, fl_a1, g1 = self.qp[(ln, "s1")]
            c1, errs[(ln, "s1")] = self._param(ln, "s1")
            w2, fl_a2, g2 = self.qp[(ln, "s2")]
            c2, errs[(ln, "s2")] = self._param(ln, "s2")
            a1, a2 = _dec(c1, w1, g1), _dec(c2, w2, g2)
        if sp["fc"]:
            acc = orc.gemm(x.reshape(x.shape[0], -1), wq)
        else:
            acc = orc.conv2d(x, wq, sp["stride"], sp["pad"])
        v, s = orc.epilogue(acc, fl_x + flw, b, fl_b, a1, fl_a1, a2, fl_a2, sp["relu"])
        ref = self.g.act[ln]
        if sp["last"]:
            q = orc.quantize_i64(v, s, 32, s, 1)
            errs[(ln, "a")] = orc.layer_error(ref.ravel(), q.ravel(), 32, s, 1)[0]
            return q, s, 1, errs
        wl, fl, sign = self.qp[(ln, "a")]
        c = orc.quantize_i64(v, s, wl, fl, sign)
        errs[(ln, "a")] = orc.layer_error(ref.ravel(), c.ravel(), wl, fl, sign)[0]
        return _dec(c, wl, sign), fl, sign, errs

    def _fp32(self, codes, fl):
        return (np.asarray(codes, np.float64) * 2.0 ** -fl).astype(np.float32)

    def evaluate(self, ln):
        q, fl, sign, errs = self._quant_layer(ln)
        fp = {ln: self._fp32(q, fl)}
        after = False if ln != "input" else True
        logits = q if (ln != "input" and self.spec[ln]["last"]) else None
        for op, nm, sp in self.g.nodes:
            if nm == ln:
                after = True
                continue
            if not after or op == "input":
                continue
            get = lambda k: fp[k] if k in fp else self._fp32(self.q[k][0], self.q[k][1])
            if op == "conv":
                x = get(sp["src"])
                if sp["fc"]:
                    xin = x.reshape(x.shape[0], -1)
                    y = orc.teacher_conv2d(xin.reshape(xin.shape[0], -1, 1, 1),
                                           sp["w"].reshape(sp["cout"], -1, 1, 1), 1, 0)
                else:
                    y = orc.teacher_conv2d(x, sp["w"], sp["stride"], sp["pad"])
                if "b" in sp:
                    y = orc.teacher_affine(y, bias=sp["b"], relu=sp["relu"])
                elif "a1" in sp:
                    y = orc.teacher_affine(y, sp["a1"], sp["a2"], relu=sp["relu"])
                else:
                    y = orc.teacher_affine(y, relu=sp["relu"])
                errs[(nm, "a")] = _sse(self.g.act[nm], y)
            elif op == "maxpool":
                x = get(sp["src"])
                N, C, H, W = x.shape
                k, st, pd = sp["k"], sp["stride"], sp["pad"]
                Ho, Wo = (H + 2 * pd - k) // st + 1, (W + 2 * pd - k) // st + 1
                xp = np.full((N, C, H + 2 * pd, W + 2 * pd), -np.inf, np.float32)
                xp[:, :, pd:pd + H, pd:pd + W] = x
                y = np.full((N, C, Ho, Wo), -np.inf, np.float32)
                for r in range(k):
                    for s in range(k):
                        y = np.maximum(y, xp[:, :, r:r + st * Ho:st, s:s + st * Wo:st])
            elif op == "add":
                v = get(sp["a"]) + get(sp["b"])
                y = np.where(v > 0, v, np.float32(0)).astype(np.float32)
            else:
                y = orc.teacher_avgpool(get(sp["src"]))
                y = y.reshape(y.shape[0], y.shape[1], 1, 1)
            fp[nm] = y
        scores = logits if logits is not None else fp[self.last]
        un, extra = _ties(np.asarray(scores).reshape(self.B, -1))
        E = distillation_error(self.pi, self.stat, errs)
        C = int(np.asarray(scores).reshape(self.B, -1).shape[1])
        return E + un / self.B + extra / (self.B * C)

    def qparams_opt(self, ln, d, quantized=False):
        """Algorithm 1 for data structure (ln, d) from its current format;
        with quantized=True every candidate runs the whole quantized network
        (evaluate_quant) and self.acc_best receives the top-1 agreement of the
        chosen candidate."""
        key = (ln, d)
        fl0 = self.qp[key][1]

        def ev():
            if quantized:
                return self.evaluate_quant(ln)
            return self.evaluate(ln), None

        best, acc = ev()
        fl_best = fl0
        self.trace.append((ln, d, fl0, best))
        for i in (-1, +1):
            k, j = 1, 0
            while k <= self.K + j:
                fl = fl0 + i * k
                if fl < FL[0] or fl > FL[1]:
                    break
                self.qp[key][1] = fl
                cost, a = ev()
                self.trace.append((ln, d, fl, cost))
                if cost < best:
                    best, fl_best, acc, j = cost, fl, a, j + 1
                k += 1
        self.qp[key][1] = fl_best
        self.acc_best = acc
        return fl_best

    def _after(self, ln):
        """The nodes after ln in network order (all nodes for the input)."""
        names = [nm for _, nm, _ in self.g.nodes]
        i = 0 if ln == "input" else names.index(ln)
        return [nd for nd in self.g.nodes[i + 1:] if nd[0] != "input"]

    def _node_q(self, op, sp, q):
        """A quantized max-pool / eltwise / avg-pool node on the codes in q
        (the eltwise and avg-pool FxP-QLayers search their formats, Eq. 14)."""
        if op == "maxpool":
            x, f, s = q[sp["src"]]
            return orc.maxpool(x, sp["k"], sp["stride"], sp["pad"]), f, s
        if op == "add":
            xa, fa, _ = q[sp["a"]]
            xb, fb, _ = q[sp["b"]]
            v, s = orc.eltwise_add(xa, fa, xb, fb, relu=True)
            f, sg, _ = orc.fl_search_i64(v.ravel(), s, 8, orc.SIGN_AUTO, *FL)
            return orc.quantize_i64(v, s, 8, f, sg), f, sg
        x, f, _ = q[sp["src"]]
        hw = x.shape[2] * x.shape[3]
        r = np.repeat(np.array([np.float32(1.0) / np.float32(hw)], np.float32), 4)
        fr, sr, _ = orc.fl_search_f32(r, 16, orc.SIGN_AUTO, *FL)
        rq = orc.quantize_f32(r, 16, fr, sr)
        y = orc.avgpool_global(x, int(rq[0])).reshape(x.shape[0], x.shape[1], 1, 1)
        wl = self.fl_wl or 8  # the last layer's input
        fo, so, _ = orc.fl_search_i64(y.ravel(), f + fr, wl, orc.SIGN_AUTO, *FL)
        return orc.quantize_i64(y, f + fr, wl, fo, so), fo, so

    def finalize(self, ln):
        q, fl, sign, _ = self._quant_layer(ln)
        self.q[ln] = (q, fl, sign)
        for op, nm, sp in self._after(ln):
            if op == "conv":
                break
            self.q[nm] = self._node_q(op, sp, self.q)

    def refinalize(self, ln):
        """Re-quantizes the finalized network from layer ln on (after a
        format of ln changed)."""
        self.finalize(ln)
        for op, nm, _ in self._after(ln):
            if op == "conv":
                self.finalize(nm)

    def top1(self, logits):
        """Share of samples whose scores have a unique maximum at the
        teacher's top-1 class."""
        s = np.asarray(logits).reshape(self.B, -1)
        t = np.asarray(self.g.act[self.last]).reshape(self.B, -1).argmax(axis=1)
        unique = (s == s.max(axis=1, keepdims=True)).sum(axis=1) == 1
        return float(np.mean(unique & (s.argmax(axis=1) == t)))

    def evaluate_quant(self, ln):
        """Cost F of the current formats with the whole network quantized:
        the finalized prefix, layer ln at its current formats and every later
        layer quantized at its formats (the errors of all data structures
        from ln on, parameters included); also the top-1 agreement."""
        cur = dict(self.q)
        c, fl, sign, errs = self._quant_layer(ln, cur)
        cur[ln] = (c, fl, sign)
        for op, nm, sp in self._after(ln):
            if op == "conv":
                c, f, s, e = self._quant_layer(nm, cur)
                errs.update(e)
                cur[nm] = (c, f, s)
            else:
                cur[nm] = self._node_q(op, sp, cur)
        scores = np.asarray(cur[self.last][0]).reshape(self.B, -1)
        un, extra = _ties(scores)
        E = distillation_error(self.pi, self.stat, errs)
        cost = E + un / self.B + extra / (self.B * scores.shape[1])
        return cost, self.top1(scores)

    def run(self):
        layers = []
        for ln, d in self.order:
            if ln not in layers:
                layers.append(ln)
        keys = set(self.order)
        for ln in layers:
            for d in ("w", "b", "s1", "s2", "a"):
                if (ln, d) in keys:
                    self.qparams_opt(ln, d)
            self.finalize(ln)
        return {k: tuple(self.qp[k]) for k in self.order}

"""Forward optimizer with Algorithm 1 (QParamsOpt) over libfxpq.

Sec. "Quantization Parameters Optimization" and Algorithm 1: the fractional
length of each data structure (weights, then bias, then output activations of
each conv / FC layer, layer by layer from the input) is moved from the
preprocessor's initial value (Eq. 6-9) in both directions, one step at a
time, keeping the word length (alpha + beta = k), and the one with the
smallest cost

    F(d, l) = E(d, l) + UnClass + MisPred                         (Eq. 21)

is kept; a direction is searched K steps past the last improvement.  Every
candidate runs the network on the calibration batch with layers before l
quantized at their chosen formats, layer l quantized at the candidate, and
the layers after l in FP32 (the order-fixed teacher kernels), then

    E(d, l) = sum_{i >= l} sum_j pi_i^j L(X_i^j) / R_i^j          (Eq. 17)

with pi from Eq. 15-16 (dispersion x size, normalized per layer), R the
range of the FP32 data structure (Eq. 18), and L the squared error (Eq. 14):
for parameters their quantization error at the current format (zero for the
FP32 layers after l), for activations the distance of the network's
activation from the FP32 teacher's (post-training self-distillation), and
UnClass / MisPred from ties of the final scores (Eq. 19-20).

Readings: activations are the layers' outputs (the input image is the first
data structure, optimized before layer 1); a C-Block's data structures are
its output activations, its conv / FC weights and bias, and its Scale
parameters aleph_1 (multiplier, 16 bits) and aleph_2 (offset, 32 bits) of
Eq. 4-5, optimized in the order w, b, aleph_1, aleph_2, a; pi is normalized
over a layer's data structures; for activations sigma is the population
standard deviation of each calibration sample, averaged over the samples,
and the size nu is that of one sample (parameters: over the tensor);
eltwise and avg-pool FxP-QLayers keep their Eq. 14 searches; accuracy has no
labels here, so the report is the agreement of the quantized network's
top-1 with the FP32 teacher's.

Every tensor operation is a libfxpq call; the host only sequences the
candidates and adds up the per-tensor error sums the library returns.
"""
import numpy as np

from . import fxpq as fx
from .nets import A_WL, BIAS_WL, FL_HI, FL_LO, RECIP_WL
from .sweep import SCALE_WL, SHIFT_WL, Sweep

# Scale parameters of a C-Block as data structures (Eq. 4-5): s1 = aleph_1,
# s2 = aleph_2 (FP32 tensor key of the layer, initial word length)
SCALE = {"s1": ("a1_f32", SCALE_WL), "s2": ("a2_f32", SHIFT_WL)}


class ForwardOptimizer:
    def __init__(self, name, seed=None, batch=None, image=None, device="cuda:0", K=1,
                 strategy=fx.ROUND_CONSERVATIVE, psi_rule=fx.PSI_PRINTED, w_wl=None,
                 first_last_wl=None):
        self.sw = Sweep(name, seed, batch, image, device, wwls=(), awls=())
        self.T, self.h, self.B, self.K = self.sw.T, self.sw.h, self.sw.batch, K
        self.w_wl = w_wl  # one word length for every layer's weights (else the network's)
        # word length of the network input, the first and last layers' weights
        # and the last layer's input (the avg-pool FxP-QLayer); wide C-Blocks
        # above 8 bits
        self.fl_wl = first_last_wl
        T = self.T
        self.nodes = list(self.sw.graph)
        self.L = {L["node"].name: L for L in self.sw.layers}
        self.act = self.sw.act  # FP32 teacher activations, NHWC
        self.keep = []
        self.bufs = {}
        self.held = {}  # per layer: the ctypes structures its last calls used
        self.evals = 0
        # data structures in optimization order: the input, then per layer
        # weights, bias, Scale multiplier and offset, output activations
        # (none for the last layer)
        self.order = [("input", "a")]
        for n in self.nodes:
            if n.op in ("conv", "fc"):
                self.order.append((n.name, "w"))
                if n.bias:
                    self.order.append((n.name, "b"))
                if "a1_f32" in self.L[n.name]:
                    self.order += [(n.name, "s1"), (n.name, "s2")]
                if not n.last:
                    self.order.append((n.name, "a"))
        # per-tensor statistics and initial formats
        self.fmt = {}   # (layer, d) -> device int32[4] {wl, fl, sign, 0}
        self.qp = {}    # (layer, d) -> [wl, fl, sign] on the host
        self.stat = {}  # (layer, d) -> (sigma, size, range)
        out4 = self._empty((4,), T.float64)
        for (ln, d) in self.order + [(n.name, "a") for n in self.nodes if getattr(n, "last", False)]:
            ref, wl = self._tensor(ln, d)
            real = self._real(ln, d)  # without the layout's zero padding
            fmt = self._fmt()
            fx.preprocess(self.h, fx.src_f32(real), real.numel(), wl, strategy, psi_rule, FL_LO, FL_HI, fmt)
            fx.layer_error(self.h, real, real, fx.F32, None, real.numel(), out4)
            f, e = fmt.cpu().numpy(), out4.cpu().numpy()
            self.fmt[(ln, d)], self.qp[(ln, d)] = fmt, [int(f[0]), int(f[1]), int(f[2])]
            sigma, nu = float(e[3]), real.numel()
            if d == "a":
                # Eq. 16 for activations: sigma per calibration sample,
                # averaged; nu = the size of one sample
                per = real.reshape(self.B, -1)
                sig = []
                for i in range(self.B):
                    fx.layer_error(self.h, per[i], per[i], fx.F32, None, per.shape[1], out4)
                    sig.append(float(out4[3].item()))
                sigma, nu = float(np.mean(sig)), per.shape[1]
            self.stat[(ln, d)] = (sigma, nu, float(e[2] - e[1]))
        # Eq. 15, normalized over each layer's data structures
        self.pi = {}
        for ln in {k[0] for k in self.stat}:
            ks = [k for k in self.stat if k[0] == ln]
            tot = sum(self.stat[k][0] * self.stat[k][1] for k in ks)
            for k in ks:
                self.pi[k] = self.stat[k][0] * self.stat[k][1] / tot if tot > 0 else 0.0
        # quantized prefix: codes and formats of finalized nodes
        self.qcodes, self.qfmt, self.deq = {}, {}, {}
        self.pos = {n.name: i for i, n in enumerate(self.nodes)}
        self.logit_fmt = self._t(np.array([32, 0, 1, 0], np.int32))
        self.ties = self._empty((2,), T.int64)
        self.trace = []
        self.pfmt = {}  # (layer, d) -> the format its parameter codes hold
        self.acc_best = None

    # -- helpers ----------------------------------------------------------------
    def _t(self, a):
        t = self.T.from_numpy(np.ascontiguousarray(a)).to(self.sw.dev)
        self.keep.append(t)
        return t

    def _empty(self, shape, dtype):
        t = self.T.empty(shape, dtype=dtype, device=self.sw.dev)
        self.keep.append(t)
        return t

    def _fmt(self):
        return self._t(np.zeros(4, np.int32))

    def _buf(self, key, shape, dtype):
        """A device buffer reused by every evaluation (allocated once per key)."""
        b = self.bufs.get(key)
        if b is None or tuple(b.shape) != tuple(shape) or b.dtype != dtype:
            b = self.T.empty(shape, dtype=dtype, device=self.sw.dev)
            self.bufs[key] = b
        return b

    def _edge(self, ln):
        convs = [n.name for n in self.nodes if n.op in ("conv", "fc")]
        return self.fl_wl is not None and ln in (convs[0], convs[-1])

    def _ct32(self, key):
        """Storage of data structure key's codes wider than 8 bits: int32 for
        a signed format, uint32 for an unsigned one."""
        return fx.I32 if self.qp[key][2] else fx.U32

    def _first_wide(self):
        """The first layer's C-Block runs on int32 codes (input or weights
        wider than 8 bits); the input is stored as int32 codes then."""
        first = [n.name for n in self.nodes if n.op in ("conv", "fc")][0]
        return self.qp[("input", "a")][0] > 8 or self.qp[(first, "w")][0] > 8

    def _tensor(self, ln, d):
        """FP32 data structure (device) and its word length."""
        if ln == "input":
            return self.act["input"], self.fl_wl or A_WL
        L = self.L[ln]
        if d == "w":
            if self._edge(ln):
                return L["w_krsc"], self.fl_wl
            return L["w_krsc"], self.w_wl or L["node"].wl
        if d == "b":
            return L["b_f32"], BIAS_WL
        if d in SCALE:
            return L[SCALE[d][0]], SCALE[d][1]
        return L["y_ref"], A_WL

    def _real(self, ln, d):
        """The data structure as the model defines it (the input's three
        channels, the weights without the padded channel / row): its
        statistics and initial format do not see the layout's zeros."""
        if ln == "input":
            x = self.act["input"]
            return x[..., :3].contiguous()
        if d == "w":
            w = self.L[ln]["w_host"]
            return self._t(np.asarray(w, np.float32).ravel())
        return self._tensor(ln, d)[0]

    def _set(self, key, fl, wl=None):
        if wl is not None:
            self.qp[key][0] = wl
        self.qp[key][1] = fl
        wl, _, sign = self.qp[key]
        self.fmt[key].copy_(self.T.tensor([wl, fl, sign, 0], dtype=self.T.int32))

    # -- one quantized layer at the current formats ---------------------------------
    def _param(self, ln, d, codes, ctype, errs):
        """Quantizes parameter d of layer ln into codes at its current format
        (skipped while the format is the one its codes hold) and appends its
        error sums to errs."""
        L, key = self.L[ln], (ln, d)
        e = self._buf((ln, d, "err"), (4,), self.T.float64)
        fq = tuple(self.qp[key])
        if self.pfmt.get((key, ctype)) != fq:
            x = L["w_krsc"] if d == "w" else L[SCALE[d][0]] if d in SCALE else L["b_f32"]
            fx.quantize(self.h, x, x.numel(), self.fmt[key], codes, ctype)
            if d == "w" and ctype == fx.I8:
                fx.weight_colsum(self.h, codes, L["node"].cout, L["wlen"], self._buf((ln, "colsum"), (L["node"].cout,), self.T.int32))
            fx.layer_error(self.h, x, codes, ctype, self.fmt[key], x.numel(), e)
            self.pfmt[(key, ctype)] = fq
        errs.append((key, e))

    def _quant_layer(self, ln, errs, src=None):
        """Runs layer ln at the current formats on its quantized input (from
        src = (codes, formats) by node name, default the finalized prefix):
        its output codes (or integer logits), with the parameter and output
        error sums appended to errs as (key, device double[4])."""
        T, h, B = self.T, self.h, self.B
        qcodes, qfmt = src if src is not None else (self.qcodes, self.qfmt)
        if ln == "input":
            x = self.act["input"]
            wide = self._first_wide()
            ct = self._ct32(("input", "a")) if wide else fx.C8
            codes = self._buf(("input", "codes", ct), x.shape, T.int32 if wide else T.int8)
            fx.quantize(h, x, x.numel(), self.fmt[("input", "a")], codes, ct)
            e = self._buf(("input", "a", "err"), (4,), T.float64)
            fx.layer_error(h, x, codes, ct, self.fmt[("input", "a")], x.numel(), e)
            errs.append((("input", "a"), e))
            return codes, self.fmt[("input", "a")], ct
        L = self.L[ln]
        n = L["node"]
        wide = qcodes[n.inp].dtype == T.int32
        assert wide or self.qp[(ln, "w")][0] <= 8, ln
        wct = self._ct32((ln, "w")) if wide else fx.I8
        wcodes = self._buf((ln, "wcodes", wct), (L["w_krsc"].numel(),), T.int32 if wide else T.int8)
        self._param(ln, "w", wcodes, wct, errs)
        cs = self._buf((ln, "colsum"), (n.cout,), T.int32)
        kw = {}
        if n.bias:
            bcodes = self._buf((ln, "bcodes"), (n.cout,), T.int32)
            self._param(ln, "b", bcodes, fx.I32, errs)
            kw.update(bias=bcodes, fl_bias=self.qp[(ln, "b")][1])
        if "a1_f32" in L:
            c1 = self._buf((ln, "s1codes"), (n.cout,), T.int32)
            c2 = self._buf((ln, "s2codes"), (n.cout,), T.int32)
            self._param(ln, "s1", c1, fx.I32, errs)
            self._param(ln, "s2", c2, fx.I32, errs)
            kw.update(scale=c1, fl_scale=self.qp[(ln, "s1")][1], shift=c2,
                      fl_shift=self.qp[(ln, "s2")][1])
        xin = qcodes[n.inp]
        ep = fx.epilogue(n.cout, self.qp[(ln, "w")][1], qfmt[n.inp], relu=n.relu, **kw)
        if wide:
            # codes wider than 8 bits: the int8 plane contractions of fxpq_qconv_wide
            xf = qfmt[n.inp].cpu().numpy()
            wl_w, _, sw = self.qp[(ln, "w")]
            d = L["desc"]
            nb = fx.qconv_wide_workspace(d, int(xf[0]), int(xf[2]), wl_w, sw)
            ws = self._buf((ln, "wide-ws"), (nb,), T.uint8)
            v = self._buf((ln, "wide-v"), (L["M"] * n.cout,), T.int64)
            sc = self._buf((ln, "wide-s"), (1,), T.int32)
            fx.qconv_wide(h, d, xin, int(xf[0]), int(xf[2]), wcodes, wl_w, sw, ep, v, sc, ws, nb)
            src = fx.src_int(v, fx.I64, sc)
            acc = v
        else:
            acc = self._buf(("acc",), (L["M"], n.cout), T.int32)
            mm = self._buf((ln, "mm"), (2,), T.float64)
            if L["fc"]:
                fx.qgemm(h, L["M"], n.cout, L["wlen"], xin, fx.C8, wcodes, cs, ep, acc, mm)
            else:
                fx.qconv(h, L["desc"], xin, fx.C8, wcodes, cs, ep, acc, mm)
            src = fx.src_acc(acc, ep, mm)
        self.held[ln] = (ep, src)
        y_ref = L["y_ref"]
        e = self._buf((ln, "a", "err"), (4,), T.float64)
        if n.last:
            fx.epilogue_scale(h, ep, self.logit_fmt[1:2])
            logits = self._buf((ln, "logits"), (L["M"], n.cout), T.int32)
            fx.requant(h, src, acc.numel(), self.logit_fmt, logits, fx.I32)
            fx.layer_error(h, y_ref, logits, fx.I32, self.logit_fmt, logits.numel(), e)
            errs.append(((ln, "a"), e))
            return logits, self.logit_fmt, fx.I32
        codes = self._buf((ln, "codes"), (L["M"], n.cout), T.int8)
        fx.requant(h, src, acc.numel(), self.fmt[(ln, "a")], codes, fx.C8)
        fx.layer_error(h, y_ref, codes, fx.C8, self.fmt[(ln, "a")], codes.numel(), e)
        errs.append(((ln, "a"), e))
        return codes, self.fmt[(ln, "a")], fx.C8

    def _recip(self, n, HW):
        """The avg-pool's reciprocal 1 / HW at its searched 16-bit format
        (code, fractional length), once per node."""
        key = (n.name, "recip")
        if key not in self.held:
            r = np.repeat(np.array([np.float32(1.0) / np.float32(HW)], np.float32), 4)
            rd, rf = self._t(r), self._fmt()
            fx.fl_search(self.h, fx.src_f32(rd), 4, RECIP_WL, fx.SIGN_AUTO, FL_LO, FL_HI, rf)
            rc = self._empty((4,), self.T.int32)
            fx.quantize(self.h, rd, 4, rf, rc, fx.I32)
            self.held[key] = (int(rc.cpu().numpy()[0]), int(rf.cpu().numpy()[1]))
        return self.held[key]

    def _quant_node(self, n, src=None):
        """Quantized max-pool / eltwise / avg-pool node on quantized inputs
        (src as in _quant_layer; the eltwise and avg-pool FxP-QLayers search
        their own formats).  Writes per-node buffers reused by every call."""
        T, h, B = self.T, self.h, self.B
        qcodes, qfmt = src if src is not None else (self.qcodes, self.qfmt)
        H, W, C = self.act[n.inp].shape[1:]
        y = self._buf((n.name, "codes"), tuple(self.act[n.name].shape), T.int8)
        if n.op == "maxpool":
            fx.maxpool(h, qcodes[n.inp], fx.C8, B, H, W, C, n.k, n.stride, n.pad, y)
            return y, qfmt[n.inp]
        f = self._buf((n.name, "fmt"), (4,), T.int32)
        if n.op == "add":
            s = fx.src_add(qcodes[n.inp], fx.C8, qfmt[n.inp], qcodes[n.other], fx.C8,
                           qfmt[n.other], n.relu)
            m = qcodes[n.inp].numel()
            self.held[(n.name, "src")] = s
        else:  # global avg-pool with the quantized reciprocal (same as the runner)
            rc, rfl = self._recip(n, H * W)
            acc = self._buf((n.name, "sum"), (B, C), T.int64)
            fx.avgpool_global(h, qcodes[n.inp], fx.C8, qfmt[n.inp], B, H * W, C, rc, acc)
            ep = fx.epilogue(C, rfl, qfmt[n.inp])
            sc = self._buf((n.name, "scale"), (1,), T.int32)
            fx.epilogue_scale(h, ep, sc)
            s = fx.src_int(acc, fx.I64, sc)
            self.held[(n.name, "src")] = (ep, s)
            m = acc.numel()
            if self.fl_wl is not None:  # the last layer's input, 32-bit storage
                y32 = self._buf((n.name, "codes32"), tuple(self.act[n.name].shape), T.int32)
                fx.fl_search(h, s, m, self.fl_wl, fx.SIGN_AUTO, FL_LO, FL_HI, f)
                # unsigned codes as uint32 (an unsigned 32-bit format's storage)
                ct = fx.U32 if int(f[2].item()) == 0 else fx.I32
                fx.requant(h, s, m, f, y32, ct)
                return y32, f
        fx.fl_search(h, s, m, A_WL, fx.SIGN_AUTO, FL_LO, FL_HI, f)
        fx.requant(h, s, m, f, y, fx.C8)
        return y, f

    def _dequant(self, name):
        if name not in self.deq:
            c = self.qcodes[name]
            y = self._empty(c.shape, self.T.float32)
            if c.dtype == self.T.int32:  # uint32 storage for unsigned formats
                ct = fx.U32 if int(self.qfmt[name][2].item()) == 0 else fx.I32
            else:
                ct = fx.C8
            fx.dequantize(self.h, c, ct, self.qfmt[name], c.numel(), y)
            self.deq[name] = y
        return self.deq[name]

    # -- cost of the current formats for layer ln --------------------------------
    def evaluate(self, ln):
        T, h, B = self.T, self.h, self.B
        self.evals += 1
        errs = []
        codes, cfmt, ctype = self._quant_layer(ln, errs)
        is_last = ln != "input" and self.L[ln]["node"].last
        y = None
        if not is_last:
            y = self._buf((ln, "deq-cur"), codes.shape, T.float32)
            fx.dequantize(h, codes, ctype, cfmt, codes.numel(), y)
        fp = {ln: y}
        start = 0 if ln == "input" else self.pos[ln] + 1
        logits32 = codes if is_last else None
        for n in self.nodes[start:]:
            if n.op == "input":
                continue
            get = lambda nm: fp[nm] if nm in fp else self._dequant(nm)
            ref = self.act[n.name]
            y = self._buf((n.name, "fp32"), ref.shape, T.float32)
            if n.op in ("conv", "fc"):
                L = self.L[n.name]
                fx.teacher_conv(h, L["tdesc"], get(n.inp), L["w_rsck"], y)
                aff = {}
                if n.bias:
                    aff["bias"] = L["b_f32"]
                if "a1_f32" in L:
                    aff = {"a1": L["a1_f32"], "a2": L["a2_f32"]}
                fx.teacher_affine(h, y, y.numel(), n.cout, y, relu=n.relu, **aff)
                e = self._buf((n.name, "a", "err"), (4,), T.float64)
                fx.layer_error(h, ref, y, fx.F32, None, y.numel(), e)
                errs.append(((n.name, "a"), e))
            elif n.op == "maxpool":
                H, W, C = self.act[n.inp].shape[1:]
                fx.teacher_maxpool(h, get(n.inp), B, H, W, C, n.k, n.stride, n.pad, y)
            elif n.op == "add":
                fx.teacher_add(h, get(n.inp), get(n.other), y.numel(), n.relu, y)
            elif n.op == "avgpool":
                H, W, C = self.act[n.inp].shape[1:]
                fx.teacher_avgpool(h, get(n.inp), B, H * W, C, y)
            fp[n.name] = y
        last = [n for n in self.nodes if getattr(n, "last", False)][0]
        if logits32 is not None:
            fx.prediction_ties(h, logits32, fx.I32, B, last.cout, self.ties)
        else:
            fx.prediction_ties(h, fp[last.name], fx.F32, B, last.cout, self.ties)
        T.cuda.synchronize(self.sw.dev)
        E = 0.0
        for key, e in errs:
            if key in self.pi and self.stat[key][2] > 0:
                E += self.pi[key] * float(e[0].item()) / self.stat[key][2]
        t = self.ties.cpu().numpy()
        unclass = float(t[0]) / B
        mispred = float(t[1]) / (B * last.cout)
        return E + unclass + mispred, (E, unclass, mispred)

    # -- Algorithm 1 ------------------------------------------------------------------
    def qparams_opt(self, ln, d, quantized=False):
        """Algorithm 1 for data structure (ln, d) from its current format;
        with quantized=True every candidate runs the whole quantized network
        (evaluate_quant) and acc_best receives the chosen candidate's top-1
        agreement."""
        key = (ln, d)
        fl0 = self.qp[key][1]

        def ev():
            if quantized:
                return self.evaluate_quant(ln)
            return self.evaluate(ln)[0], None

        best, acc = ev()
        fl_best = fl0
        self.trace.append((ln, d, fl0, best))
        for i in (-1, +1):
            k, j = 1, 0
            while k <= self.K + j:
                fl = fl0 + i * k
                if fl < FL_LO or fl > FL_HI:
                    break
                self._set(key, fl)
                cost, a = ev()
                self.trace.append((ln, d, fl, cost))
                if cost < best:
                    best, fl_best, acc, j = cost, fl, a, j + 1
                k += 1
        self._set(key, fl_best)
        self.acc_best = acc
        return fl_best, best

    def _after(self, ln):
        start = 0 if ln == "input" else self.pos[ln] + 1
        return [n for n in self.nodes[start:] if n.op != "input"]

    def finalize(self, ln):
        """Quantizes layer ln at its chosen formats into the prefix, then the
        max-pool / eltwise / avg-pool nodes that follow it (copies: the
        evaluation buffers are reused)."""
        errs = []
        codes, cfmt, ctype = self._quant_layer(ln, errs)
        self.qcodes[ln], self.qfmt[ln] = codes.clone(), cfmt
        self.deq.pop(ln, None)
        for n in self._after(ln):
            if n.op in ("conv", "fc"):
                break
            y, f = self._quant_node(n)
            self.qcodes[n.name], self.qfmt[n.name] = y.clone(), f.clone()
            self.deq.pop(n.name, None)

    def refinalize(self, ln):
        """Re-quantizes the finalized network from layer ln on (after a format
        of ln changed)."""
        self.finalize(ln)
        for n in self._after(ln):
            if n.op in ("conv", "fc"):
                self.finalize(n.name)

    def _top1(self, logits):
        """Share of samples whose integer scores have a unique maximum at the
        teacher's top-1 class."""
        last = [n for n in self.nodes if getattr(n, "last", False)][0]
        q = logits.cpu().numpy().reshape(self.B, -1)
        t = self.act[last.name].cpu().numpy().reshape(self.B, -1)
        unique = (q == q.max(1, keepdims=True)).sum(1) == 1
        return float(np.mean(unique & (q.argmax(1) == t.argmax(1))))

    def evaluate_quant(self, ln):
        """Cost F of the current formats with the whole network quantized:
        the finalized prefix, layer ln at its current formats and every later
        layer at its formats (the error sums of every data structure from ln
        on, parameters included), and the top-1 agreement."""
        T, h, B = self.T, self.h, self.B
        self.evals += 1
        errs = []
        cc, cf = dict(self.qcodes), dict(self.qfmt)
        codes, cfmt, ctype = self._quant_layer(ln, errs, (cc, cf))
        cc[ln], cf[ln] = codes, cfmt
        for n in self._after(ln):
            if n.op in ("conv", "fc"):
                codes, cfmt, ctype = self._quant_layer(n.name, errs, (cc, cf))
            else:
                codes, cfmt = self._quant_node(n, (cc, cf))
            cc[n.name], cf[n.name] = codes, cfmt
        last = [n for n in self.nodes if getattr(n, "last", False)][0]
        logits = cc[last.name]
        fx.prediction_ties(h, logits, fx.I32, B, last.cout, self.ties)
        T.cuda.synchronize(self.sw.dev)
        E = 0.0
        for key, e in errs:
            if key in self.pi and self.stat[key][2] > 0:
                E += self.pi[key] * float(e[0].item()) / self.stat[key][2]
        t = self.ties.cpu().numpy()
        cost = E + float(t[0]) / B + float(t[1]) / (B * last.cout)
        return cost, self._top1(logits)

    def run(self):
        """The forward optimizer: every data structure in order; returns the
        chosen formats."""
        layers = []
        for ln, d in self.order:
            if ln not in layers:
                layers.append(ln)
        for ln in layers:
            for d in ("w", "b", "s1", "s2", "a"):
                if (ln, d) in self.qp and (ln, d) in dict.fromkeys(self.order):
                    self.qparams_opt(ln, d)
            self.finalize(ln)
        return {k: tuple(v) for k, v in self.qp.items() if k in dict.fromkeys(self.order)}

    def mac_overflow(self, bits=16):
        """Per conv / FC layer between the first and the last: (accumulators
        outside `bits`-bit two's complement, accumulators) of the finalized
        network (Sec. "Integer-Only Inference" keeps those MAC results in 16
        bits)."""
        convs = [n for n in self.nodes if n.op in ("conv", "fc")]
        cnt = self._buf(("ovf",), (1,), self.T.int64)
        out = {}
        for n in convs[1:-1]:
            self._quant_layer(n.name, [])
            acc = self.bufs[("acc",)]
            m = self.L[n.name]["M"] * n.cout
            cnt.zero_()
            fx.acc_overflow(self.h, acc, m, bits, cnt)
            out[n.name] = (int(cnt.item()), m)
        return out

    def top1_agreement(self):
        """Share of samples whose quantized top-1 (unique maximum) is the
        teacher's top-1."""
        last = [n for n in self.nodes if getattr(n, "last", False)][0]
        return self._top1(self.qcodes[last.name])

    def close(self):
        self.sw.close()

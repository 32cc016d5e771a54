"""Per-layer sensitivity sweep of a ResNet through libfxpq (the fifth workload).

Mirrors the paper's sensitivity test (Sec. "Data-Structures Sensitivity to
Quantization": one layer's data structures quantized, every other layer
intact), as a tensor-wide error per step instead of a top-1 rate: for every
conv / FC layer l, activation word length a in `awls` and weight word length
w in `wwls`:

  1. the FP32 teacher's input activation of l is quantized at a (its own FL
     search, Eq. 14; Eq. 10-12);
  2. the layer's weights are quantized at w (FL searched once per (l, w));
  3. the C-Block runs on the codes (int8 MFMA, bias / BN-as-Scale, ReLU);
  4. its output is requantized at a by the layer's FxP-QLayer (none after the
     last layer, whose logits stay integer, Sec. "FxP-QLayer");
  5. the layer error of that output against the teacher's output of l
     (Eq. 14, with min / max / std of the reference, Eq. 16-18).

The FP32 teacher (fxpq_teacher_*) runs once, outside the timing; its
activations stay in HBM (about 17 GB for ResNet-50 at batch 256).  Weight
searches are set-up (parameters are quantized once per word length); the
timed part is every step's input search + quantize, conv, output search +
requant and layer error, with no host synchronization until the end.
"""
import time

import numpy as np

import synth

from . import fxpq as fx
from .nets import ARCH, BIAS_WL, BN_EPS, DEFAULT_SHAPE, FL_HI, FL_LO, SCALE_WL, SEEDS, SHIFT_WL

WWLS = (8, 7, 6, 5, 4, 3, 2)
AWLS = (8, 7, 6, 5, 4)


class Sweep:
    def __init__(self, name="resnet50", seed=None, batch=None, image=None, device="cuda:0",
                 wwls=WWLS, awls=AWLS, layers=None):
        import torch
        self.T = torch
        self.name = name
        self.seed = SEEDS[name] if seed is None else seed
        b0, s0 = DEFAULT_SHAPE[name]
        self.batch, self.image = batch or b0, image or s0
        self.dev = torch.device(device)
        self.h = fx.Handle(self.dev.index or 0)
        fx.set_stream(self.h, torch.cuda.current_stream(self.dev))
        self.graph = ARCH[name](self.seed)
        self.wwls, self.awls = tuple(wwls), tuple(awls)
        self.keep = []
        self._build(layers)

    # -- helpers --------------------------------------------------------------
    def _t(self, a):
        t = self.T.from_numpy(np.ascontiguousarray(a)).to(self.dev)
        self.keep.append(t)
        return t

    def _empty(self, shape, dtype):
        t = self.T.empty(shape, dtype=dtype, device=self.dev)
        self.keep.append(t)
        return t

    def _fmt(self):
        return self._t(np.zeros(4, np.int32))

    def _search_quantize(self, xd, wl, codes, code_type):
        f = self._fmt()
        fx.fl_search(self.h, fx.src_f32(xd), xd.numel(), wl, fx.SIGN_AUTO, FL_LO, FL_HI, f)
        fx.quantize(self.h, xd, xd.numel(), f, codes, code_type)
        return f

    # -- set-up ---------------------------------------------------------------
    def _build(self, layers):
        T, B, S, seed = self.T, self.batch, self.image, self.seed
        x = synth.normal(seed, "input", (B, 3, S, S))
        x4 = np.zeros((B, S, S, 4), np.float32)
        x4[..., :3] = np.transpose(x, (0, 2, 3, 1))
        shapes = {"input": (S, S, 4)}
        act = {"input": self._t(x4)}  # teacher activations, NHWC fp32
        self.layers = []
        pending = []
        for n in self.graph:
            if n.op == "input":
                continue
            if n.op in ("conv", "fc"):
                H, W, Cin = shapes[n.inp]
                real_cin = 3 if n.inp == "input" else Cin
                if n.op == "conv":
                    k, st, pd = n.k, n.stride, n.pad
                    w = synth.he_normal(seed, n.name + ".w", (n.cout, real_cin, k, k))
                    wk = np.transpose(w, (0, 2, 3, 1))  # KRSC
                    if Cin == 4:
                        wk = np.concatenate([wk, np.zeros((n.cout, k, k, 1), np.float32)], axis=3)
                    w_rsck = np.transpose(wk, (1, 2, 3, 0))
                    wk = wk.reshape(n.cout, -1)
                    if Cin == 4:
                        kp = (wk.shape[1] + 63) // 64 * 64
                        wk = np.concatenate([wk, np.zeros((n.cout, kp - wk.shape[1]), np.float32)], 1)
                    Ho, Wo = (H + 2 * pd - k) // st + 1, (W + 2 * pd - k) // st + 1
                    desc = fx.conv_desc(B, H, W, Cin, n.cout, k, k, st, pd)
                else:
                    fan_in = H * W * Cin
                    w = synth.he_normal(seed, n.name + ".w", (n.cout, fan_in))
                    wk = w.reshape(n.cout, Cin, H, W).transpose(0, 2, 3, 1).reshape(n.cout, fan_in)
                    w_rsck = wk.T.reshape(1, 1, fan_in, n.cout)
                    Ho = Wo = 1
                    desc = fx.conv_desc(B, 1, 1, fan_in, n.cout, 1, 1, 1, 0)
                L = {"node": n, "desc": desc, "M": B * Ho * Wo, "Cin": Cin, "wlen": wk.shape[1],
                     "in": n.inp, "fc": n.op == "fc"}
                wkd = self._t(wk.astype(np.float32).ravel())
                # teacher: conv, then BN-as-Scale or bias, then ReLU
                y = self._empty((B, Ho, Wo, n.cout), T.float32)
                tdesc = desc if n.op == "conv" else fx.conv_desc(B, 1, 1, H * W * Cin, n.cout, 1, 1, 1, 0)
                L["w_rsck"] = self._t(w_rsck.astype(np.float32))
                L["w_krsc"], L["w_host"], L["tdesc"] = wkd, w, tdesc
                fx.teacher_conv(self.h, tdesc, act[n.inp], L["w_rsck"], y)
                aff = {}
                if n.bias:
                    b = synth.normal(seed, n.name + ".b", (n.cout,), std=0.01)
                    L["b_f32"] = self._t(b)
                    aff["bias"] = L["b_f32"]
                if getattr(n, "bn", False):
                    gamma = synth.uniform(seed, n.name + ".bn.gamma", (n.cout,), 0.5, 1.5)
                    beta = synth.normal(seed, n.name + ".bn.beta", (n.cout,), std=0.1)
                    mean = np.zeros(n.cout, np.float32)
                    var = np.ones(n.cout, np.float32)
                    inv = np.sqrt(var + BN_EPS)
                    a1 = (gamma / inv).astype(np.float32)  # Eq. 5
                    a2 = (beta - gamma * mean / inv).astype(np.float32)
                    L["a1_f32"], L["a2_f32"] = self._t(a1), self._t(a2)
                    aff = {"a1": L["a1_f32"], "a2": L["a2_f32"]}
                fx.teacher_affine(self.h, y, y.numel(), n.cout, y, relu=n.relu, **aff)
                act[n.name] = y
                shapes[n.name] = (Ho, Wo, n.cout)
                # parameters of the quantized path: weights at every w, bias /
                # Scale at their fixed word lengths
                L["w"] = {}
                for wwl in self.wwls:
                    codes = self._empty((wkd.numel(),), T.int8)
                    f = self._search_quantize(wkd, wwl, codes, fx.I8)
                    cs = self._empty((n.cout,), T.int32)
                    fx.weight_colsum(self.h, codes, n.cout, wk.shape[1], cs)
                    L["w"][wwl] = (codes, cs, f)
                    pending.append((L, "w", wwl, f))
                if n.bias:
                    bq = self._empty((n.cout,), T.int32)
                    pending.append((L, "b", None, self._search_quantize(L["b_f32"], BIAS_WL, bq, fx.I32)))
                    L["b"] = bq
                if getattr(n, "bn", False):
                    a1q, a2q = self._empty((n.cout,), T.int32), self._empty((n.cout,), T.int32)
                    pending.append((L, "a1", None, self._search_quantize(L["a1_f32"], SCALE_WL, a1q, fx.I32)))
                    pending.append((L, "a2", None, self._search_quantize(L["a2_f32"], SHIFT_WL, a2q, fx.I32)))
                    L["a1"], L["a2"] = a1q, a2q
                L["y_ref"] = y
                self.layers.append(L)
            elif n.op == "maxpool":
                H, W, C = shapes[n.inp]
                Ho, Wo = (H + 2 * n.pad - n.k) // n.stride + 1, (W + 2 * n.pad - n.k) // n.stride + 1
                y = self._empty((B, Ho, Wo, C), T.float32)
                fx.teacher_maxpool(self.h, act[n.inp], B, H, W, C, n.k, n.stride, n.pad, y)
                act[n.name], shapes[n.name] = y, (Ho, Wo, C)
            elif n.op == "add":
                y = self._empty(act[n.inp].shape, T.float32)
                fx.teacher_add(self.h, act[n.inp], act[n.other], y.numel(), n.relu, y)
                act[n.name], shapes[n.name] = y, shapes[n.inp]
            elif n.op == "avgpool":
                H, W, C = shapes[n.inp]
                y = self._empty((B, 1, 1, C), T.float32)
                fx.teacher_avgpool(self.h, act[n.inp], B, H * W, C, y)
                act[n.name], shapes[n.name] = y, (1, 1, C)
        self.act = act
        T.cuda.synchronize(self.dev)
        for L, kind, wwl, f in pending:
            wl, fl, sign, st = (int(v) for v in f.cpu().numpy())
            if st:
                raise RuntimeError(f"parameter search of {L['node'].name}.{kind} failed ({st})")
            L.setdefault("fl", {})[(kind, wwl)] = (wl, fl, sign)
        if layers is not None:
            self.layers = [L for L in self.layers if L["node"].name in layers]
        # per-step buffers sized for the largest layer
        self.max_in = max(act[L["in"]].numel() for L in self.layers)
        self.max_out = max(L["M"] * L["node"].cout for L in self.layers)
        self.xq = self._empty((self.max_in,), T.int8)
        self.acc = self._empty((self.max_out,), T.int32)
        self.yq = self._empty((self.max_out,), T.int8)
        self.logits = self._empty((self.max_out,), T.int32)
        self.mm = self._empty((2,), T.float64)
        self.steps = [(li, a, w) for li in range(len(self.layers)) for a in self.awls for w in self.wwls]
        # per step: [input format of (l, a) -- written in the group's first step
        # only], [output format (or the logits' {32, s, signed})]
        f0 = np.zeros((len(self.steps), 2, 4), np.int32)
        for si, (li, a, w) in enumerate(self.steps):
            if self.layers[li]["node"].last:
                f0[si, 1] = (32, 0, 1, 0)
        self.fmts = self._t(f0)
        self.errs = self._t(np.zeros((len(self.steps), 4), np.float64))
        self._plan()

    def _plan(self):
        """Every library call of the sweep, pre-built as (fn, args)."""
        import ctypes as C
        Lb = fx.lib()
        h = self.h.value
        calls = []
        self.refs = []
        fstride = 2 * 4 * 4
        step = 0
        for L in self.layers:
            n = L["node"]
            xin = self.act[L["in"]]
            nin = xin.numel()
            src_in = fx.src_f32(xin)
            self.refs.append(src_in)
            n_out = L["M"] * n.cout
            acc = self.acc[:n_out]
            self.refs.append(acc)
            for a in self.awls:
                f_in = self.fmts.data_ptr() + step * fstride
                calls.append((Lb.fxpq_fl_search, (h, C.byref(src_in), nin, a, fx.SIGN_AUTO, FL_LO,
                                                   FL_HI, f_in, None)))
                calls.append((Lb.fxpq_quantize, (h, xin.data_ptr(), nin, f_in, self.xq.data_ptr(), fx.C8)))
                for w in self.wwls:
                    f_out = self.fmts.data_ptr() + step * fstride + 16
                    err = self.errs.data_ptr() + step * 32
                    codes, cs, _ = L["w"][w]
                    kw = {}
                    if "b" in L:
                        kw.update(bias=L["b"], fl_bias=L["fl"][("b", None)][1])
                    if "a1" in L:
                        kw.update(scale=L["a1"], fl_scale=L["fl"][("a1", None)][1],
                                  shift=L["a2"], fl_shift=L["fl"][("a2", None)][1])
                    ep = fx.epilogue(n.cout, L["fl"][("w", w)][1], f_in, relu=n.relu, **kw)
                    src = fx.src_acc(acc, ep, self.mm)
                    self.refs += [ep, src]
                    if L["fc"]:
                        calls.append((Lb.fxpq_qgemm, (h, L["M"], n.cout, L["wlen"], self.xq.data_ptr(),
                                                      fx.C8, codes.data_ptr(), cs.data_ptr(),
                                                      C.byref(ep), acc.data_ptr(), self.mm.data_ptr())))
                    else:
                        calls.append((Lb.fxpq_qconv, (h, C.byref(L["desc"]), self.xq.data_ptr(), fx.C8,
                                                      codes.data_ptr(), cs.data_ptr(), C.byref(ep),
                                                      acc.data_ptr(), self.mm.data_ptr())))
                    if n.last:
                        # the last layer keeps integer logits at the C-Block scale
                        calls.append((Lb.fxpq_epilogue_scale, (h, C.byref(ep), f_out + 4)))
                        calls.append((Lb.fxpq_requant, (h, C.byref(src), n_out, f_out,
                                                        self.logits.data_ptr(), fx.I32)))
                        calls.append((Lb.fxpq_layer_error, (h, L["y_ref"].data_ptr(),
                                                            self.logits.data_ptr(), fx.I32, f_out,
                                                            n_out, err)))
                    else:
                        calls.append((Lb.fxpq_fl_search, (h, C.byref(src), n_out, a, fx.SIGN_AUTO,
                                                           FL_LO, FL_HI, f_out, None)))
                        calls.append((Lb.fxpq_requant, (h, C.byref(src), n_out, f_out,
                                                        self.yq.data_ptr(), fx.C8)))
                        calls.append((Lb.fxpq_layer_error, (h, L["y_ref"].data_ptr(),
                                                            self.yq.data_ptr(), fx.C8, f_out, n_out,
                                                            err)))
                    step += 1
        self.calls = calls

    # -- run ------------------------------------------------------------------
    def run(self):
        """Enqueues every step of the sweep (no host synchronization)."""
        for fn, args in self.calls:
            st = fn(*args)
            if st:
                raise fx.FxpqError(fn.__name__, st)

    def timed_run(self):
        """Runs the sweep once between two synchronizations; returns seconds."""
        self.T.cuda.synchronize(self.dev)
        t0 = time.perf_counter()
        self.run()
        self.T.cuda.synchronize(self.dev)
        return time.perf_counter() - t0

    def results(self):
        """One record per step: layer, word lengths, formats, layer error."""
        self.T.cuda.synchronize(self.dev)
        flags = fx.sync_status(self.h)
        f = self.fmts.cpu().numpy()
        e = self.errs.cpu().numpy()
        recs = []
        per_group = len(self.wwls)
        for si, (li, a, w) in enumerate(self.steps):
            L = self.layers[li]
            g = si - si % per_group  # first step of the (l, a) group holds the input format
            recs.append({"layer": L["node"].name, "awl": a, "wwl": w,
                         "fmt_in": tuple(int(v) for v in f[g, 0, :3]),
                         "fmt_w": L["fl"][("w", w)],
                         "fmt_out": tuple(int(v) for v in f[si, 1, :3]),
                         "status": (int(f[g, 0, 3]), int(f[si, 1, 3])),
                         "sse": float(e[si, 0]), "ref_min": float(e[si, 1]),
                         "ref_max": float(e[si, 2]), "ref_std": float(e[si, 3])})
        return {"flags": flags, "records": recs}

    def close(self):
        self.h.close()

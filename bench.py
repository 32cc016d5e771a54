"""Benchmark: DFX calibration forward of ResNet-50 at batch 256 on one MI355X.

One step = one complete calibration forward over a 256x3x224x224 batch:
input FL search + quantize + layer error, every C-Block (int8 MFMA conv +
epilogue, FL search over the whole output tensor, requantization), max-pool,
residual adds (FL search + requant), global avg-pool (+ FxP-QLayer) and the
final FC to integer logits.  Parameters are quantized once during set-up
(weight FL searches are not part of a calibration step).  Inputs are resident
in HBM before timing starts.  The runner predicts each C-Block's and each
eltwise FxP-QLayer's window from the previous forward on the same batch and
reruns the standard calls from the first failed prediction, so every
forward's results are the standard calls' bits; the timed forwards are the
repeated (warm) ones, and the line also reports cold forwards.

Roofline: the predicted C-Block, the kernel that takes most of the forward:
conv + epilogue + the FL-search window + codes in one contraction, bound by
its fp64 / int32 vector arithmetic (PRED_OPS_PER_VALUE lane-ops per output
value against 256 CUs x 64 lanes x 2.4 GHz), timed by the library's events
(fxpq_timer_start / fxpq_timer_read).  `traffic` comes from the committed
rocprofv3 FETCH_SIZE / WRITE_SIZE summary and is reported only while the
kernel sources match the profiled ones.  The contraction alone, the window
passes and per-layer rooflines are reported beside it.

Prints ONE JSON line.  --gpus above 1 exits: this build runs on one GPU.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
INT8_PEAK_TOPS = 5000.0
# fp64 / int32 vector ALU: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz lane-ops/s
ALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
# lane-ops per output value the predicted C-Block's epilogue must execute:
# value (colsum restore, convert, Scale / bias fma, ReLU) 4; per window
# candidate (scale, round, clamp, sum q^2, sum W q) 2 x 5; clipping bound 3;
# sum W^2 1; min / max 2; code (convert, pack) 2
PRED_OPS_PER_VALUE = 22
BATCH, IMAGE = 256, 224
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "cblock_predicted_resnet50_b256_traffic.md")
WINDOW_SOURCES = ["k_conv.hip", "fls.hpp", "values.hpp", "common.hpp"]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the per-layer sensitivity sweep reported alongside")
    ap.add_argument("--cpu-sample-batch", type=int, default=12)
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads' figures (FC layer, AlexNet, VGG-16, ResNet-18)")
    ap.add_argument("--mode", choices=["bench", "profile", "copy", "sweep", "qparams", "reduction",
                                       "wide", "steps"],
                    default="bench",
                    help="profile: set up and run --warmup forwards only (for counter runs); "
                         "copy: one plain 1 GiB device copy (counter calibration); "
                         "sweep: the sensitivity sweep figures only")
    return ap.parse_args()


def window_source_hash():
    """Hash of the sources of the kernel the committed traffic summary covers."""
    h = hashlib.sha256()
    for f in WINDOW_SOURCES:
        with open(os.path.join(ROOT, "paper_2203_12091_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic():
    """Per-launch HBM bytes of the predicted C-Block from the committed counter
    summary, or None when the summary is missing or the kernel changed since."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    m_hash = re.search(r"source_hash:\s*(\w+)", text)
    m_val = re.search(r"traffic_bytes_per_launch:\s*([0-9.]+)", text)
    if not m_hash or not m_val or m_hash.group(1) != window_source_hash():
        return None
    return float(m_val.group(1))


def host_info():
    """The GPU machine's host as the oracle sees it: CPU model, logical CPUs, the
    threads the oracle's OpenMP regions use, compiler and flags."""
    import subprocess
    from oracle import build as ob
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        cc = subprocess.run(["gcc", "--version"], capture_output=True, text=True).stdout.splitlines()[0]
    except (OSError, IndexError):
        cc = None
    return {"cpu_model": model, "logical_cpus": os.cpu_count(),
            "threads": int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1)),
            "compiler": cc, "flags": " ".join(ob.CFLAGS)}


def cpu_baseline(batch):
    """The oracle, as it stands, on a bounded sample: a calibration forward of
    `batch` images at 224x224 (parameters quantized beforehand), on the host;
    plus the single-core rates of its streaming steps."""
    import oracle
    t_prep = time.perf_counter()
    f = oracle.nets.prepare("resnet50", batch=batch, image=IMAGE)
    t0 = time.perf_counter()
    f.run()
    t = time.perf_counter() - t0
    info = host_info()
    out = {"value": round(batch / t, 5), "unit": "images/s", "cores": info["threads"],
           "kind": "oracle",
           "sample": f"ResNet-50 DFX calibration forward of {batch} images 224x224 "
                     f"(exact CPU oracle, parameters pre-quantized; {t:.1f} s forward, "
                     f"{t0 - t_prep:.1f} s set-up untimed)"}
    out.update({k: v for k, v in info.items() if k != "threads"})
    out["single_core"] = cpu_single_core()
    return out


def cpu_single_core():
    """GB/s of the oracle's quantize, FL search, requantization and layer
    error on one core (its OpenMP regions limited to one thread): fp32 /
    int32 values in, codes out, the algorithmic bytes of the GPU steps."""
    import ctypes
    import numpy as np
    import oracle
    import synth
    gomp = ctypes.CDLL("libgomp.so.1")
    gomp.omp_get_max_threads.restype = ctypes.c_int
    prev = gomp.omp_get_max_threads()
    n = 1 << 22
    x = synth.normal(1, "cpu-x", (n,))
    v = synth.integers(1, "cpu-v", (n,), -2 ** 20, 2 ** 20).astype(np.int64)
    out = {"values": n}
    gomp.omp_set_num_threads(1)
    try:
        steps = {
            "quantize": (lambda: oracle.quantize_f32(x, 8, 5, 1), 5),
            "fl_search": (lambda: oracle.fl_search_f32(x, 8, oracle.SIGN_AUTO, -8, 15), 4),
            "requant": (lambda: oracle.quantize_i64(v, 14, 8, -3, 1), 5),
        }
        codes = oracle.quantize_f32(x, 8, 5, 1)
        steps["layer_error"] = (lambda: oracle.layer_error(x, codes, 8, 5, 1), 5)
        for name, (fn, bpv) in steps.items():
            t0 = time.perf_counter()
            fn()
            t = time.perf_counter() - t0
            out[name + "_gbs"] = round(bpv * n / t / 1e9, 4)
    finally:
        gomp.omp_set_num_threads(prev)
    return out


def cpu_configs():
    """The oracle's forwards of the other workloads on bounded samples (all
    host threads): the FC layer at its full size, AlexNet / VGG-16 /
    ResNet-18 on a few images at 224x224 (parameters quantized beforehand)."""
    import oracle
    out = {}
    t0 = time.perf_counter()
    oracle.nets.run_fc(0)
    out["fc"] = {"us_per_call": round((time.perf_counter() - t0) * 1e6, 1),
                 "sample": "the whole FC workload (WL 8, 6 and 4), exact CPU oracle"}
    for name, b in (("alexnet", 4), ("vgg16", 1), ("resnet18", 4)):
        f = oracle.nets.prepare(name, batch=b, image=IMAGE)
        t0 = time.perf_counter()
        f.run()
        t = time.perf_counter() - t0
        out[name] = {"images_per_s": round(b / t, 4),
                     "sample": f"{b} image(s) 224x224, exact CPU oracle, {t:.1f} s"}
    return out


def qparams_figures(dev, batch=32, image=224):
    """The forward optimizer (Algorithm 1, K = 1, conservative preprocessor
    formats) over ResNet-18 on a calibration batch, timed from the teacher
    onwards; the oracle's optimizer on a bounded sample beside it; and the
    preprocessor's initial-format call over the network input."""
    import torch
    from paper_2203_12091_amd import fxpq as fx
    from paper_2203_12091_amd import qparams
    t0 = time.perf_counter()
    fo = qparams.ForwardOptimizer("resnet18", batch=batch, image=image, device=str(dev))
    torch.cuda.synchronize(dev)
    t1 = time.perf_counter()
    fo.run()
    torch.cuda.synchronize(dev)
    t2 = time.perf_counter()
    out = {"metric": "forward optimizer (Algorithm 1) seconds, ResNet-18", "batch": batch,
           "image": image, "K": fo.K, "data_structures": len(fo.order), "evaluations": fo.evals,
           "setup_s": round(t1 - t0, 3), "optimize_s": round(t2 - t1, 3),
           "evaluations_per_s": round(fo.evals / (t2 - t1), 2),
           "top1_agreement_with_fp32": round(fo.top1_agreement(), 4)}
    # the preprocessor over the network input (min / max pass + exact decision)
    x = fo.act["input"]
    fmt = torch.zeros(4, dtype=torch.int32, device=dev)
    src = fx.src_f32(x)
    reps = 20
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fx.preprocess(fo.h, src, x.numel(), 8, fx.ROUND_CONSERVATIVE, fx.PSI_PRINTED, -8, 15, fmt)
    e1.record()
    torch.cuda.synchronize(dev)
    ms = e0.elapsed_time(e1) / reps
    out["preprocess"] = {"tensor": f"input {tuple(x.shape)} fp32", "ms": round(ms, 4),
                         "gbs": round(4 * x.numel() / (ms * 1e-3) / 1e9, 1)}
    fo.close()
    import oracle.qparams as oq
    t0 = time.perf_counter()
    ref = oq.ForwardOptimizer("resnet18", batch=1, image=16)
    ref.run()
    t = time.perf_counter() - t0
    out["cpu_baseline"] = {"seconds": round(t, 2), "evaluations": len(ref.trace), "kind": "oracle",
                           "sample": "ResNet-18, 1 image 16x16, K = 1 (exact CPU oracle)"}
    return out


def reduction_figures(dev, batch=32, image=224, thld=0.5, max_changes=None):
    """Bit-precision level reduction (Algorithm 2) on a calibration batch:
    ResNet-18 from two initial designs, 8-bit everywhere (biases 32) and the
    paper's wide first / last layers (32-bit input, first and last weights
    and last-layer input, over wide C-Blocks), and AlexNet and VGG-16 from
    the 8-bit design.  Each: the forward
    optimizer first (untimed set-up), then Algorithm 2 to convergence (or
    max_changes applied reductions), timed; the memory model and the 16-bit
    MAC accounting before and after; the oracle's reduction on a bounded
    sample beside it."""
    import torch
    from paper_2203_12091_amd import qparams, reduction
    out = {"metric": "bit-precision reduction (Algorithm 2) seconds", "batch": batch,
           "image": image, "threshold": thld, "max_changes": max_changes}
    runs = (("resnet18", "design_8bit", None), ("resnet18", "design_wide32", 32),
            ("alexnet", "design_8bit", None), ("vgg16", "design_8bit", None))
    for net, design, flw in runs:
        design = f"{net}_{design}"
        fo = qparams.ForwardOptimizer(net, batch=batch, image=image, device=str(dev), w_wl=8,
                                      first_last_wl=flw)
        fo.run()
        torch.cuda.synchronize(dev)
        before = reduction.memory_model(fo)
        acc0 = fo.top1_agreement()
        ovf0 = fo.mac_overflow(16)
        r = reduction.QReduction(fo, thld, max_changes=max_changes)
        e0 = fo.evals
        t0 = time.perf_counter()
        r.run()
        torch.cuda.synchronize(dev)
        t = time.perf_counter() - t0
        after = reduction.memory_model(fo)
        ovf1 = fo.mac_overflow(16)
        ev = fo.evals - e0
        out[design] = {
            "changes": len(r.changes),
            "word_lengths": {f"{ln}.{d}": v[0] for (ln, d), v in r.formats().items()},
            "trials": len(r.trials), "evaluations": ev, "seconds": round(t, 3),
            "evaluations_per_s": round(ev / t, 2), "top1_agreement_before": round(acc0, 4),
            "top1_agreement_after": round(r.accuracy(), 4),
            "memory_mb_before": {k: round(v, 4) for k, v in before.items()},
            "memory_mb_after": {k: round(v, 4) for k, v in after.items()},
            "mac16_overflow_before": [sum(c for c, _ in ovf0.values()), sum(m for _, m in ovf0.values())],
            "mac16_overflow_after": [sum(c for c, _ in ovf1.values()), sum(m for _, m in ovf1.values())]}
        fo.close()
        del fo, r
    import oracle.qparams as oq
    import oracle.reduction as orr
    ref = oq.ForwardOptimizer("resnet18", batch=1, image=16, w_wl=8)
    ref.run()
    rr = orr.QReduction(ref, thld, max_changes=2)
    n0 = len(ref.trace)
    t0 = time.perf_counter()
    rr.run()
    t = time.perf_counter() - t0
    out["cpu_baseline"] = {"seconds": round(t, 2), "evaluations": len(ref.trace) - n0,
                           "changes": len(rr.changes), "kind": "oracle",
                           "sample": "ResNet-18, 1 image 16x16, 2 changes (exact CPU oracle)"}
    return out


def wide_figures(dev, batch=256):
    """Wide C-Blocks (fxpq_qconv_wide) at the shapes of ResNet-50's first and
    last layers, with 32-bit activations and weights (the paper's initial
    design) and with 16-bit ones: the first conv (7x7/2 over 224x224 RGB,
    Scale + ReLU epilogue) and the FC (2048 -> 1000, bias), each timed over 5
    calls after one untimed call.  One contraction walks the plane pairs
    (int8 operations: pairs x 2 M N depth) and writes the int64 values (8 B
    each); the codes are random over the whole 32- / 16-bit range."""
    import torch
    from paper_2203_12091_amd import fxpq as fx
    h = fx.Handle(0)
    fx.set_stream(h, torch.cuda.current_stream())
    gen = torch.Generator(device=dev).manual_seed(11)

    def codes(shape, wl):
        return torch.randint(-(1 << (wl - 1)), 1 << (wl - 1), shape, generator=gen, device=dev,
                             dtype=torch.int64).to(torch.int32)

    def planes(wl_x, wl_w):
        px = (wl_x + 7) // 8
        pw = next(n for n in range(1, 6) if (2 ** (wl_w - 1) - 1) <= 127 * ((256 ** n - 1) // 255))
        return px * pw

    out = {}
    shapes = {"resnet50_conv1_b256": (fx.conv_desc(batch, 224, 224, 4, 64, 7, 7, 2, 3), True),
              "resnet50_fc_b256": (fx.conv_desc(batch, 1, 1, 2048, 1000, 1, 1, 1, 0), False)}
    for bits in (32, 16):
        for name, (d, first) in shapes.items():
            depth = d.r * d.s * d.c
            wrow = (depth + 63) // 64 * 64 if d.c == 4 else depth
            x = codes((d.n, d.h, d.w, d.c), bits)
            if d.c == 4:
                x[..., 3] = 0
            w = codes((d.k, wrow), bits)
            if d.c == 4:
                w.view(d.k, -1)[:, depth:] = 0
            # fractional lengths small enough that full-range codes stay exact
            fin = torch.tensor([bits, 2, 1, 0], dtype=torch.int32, device=dev)
            if first:
                a1 = codes((d.k,), 16)
                a2 = codes((d.k,), 32)
                ep = fx.epilogue(d.k, 2, fin, relu=True, scale=a1, fl_scale=1, shift=a2,
                                 fl_shift=5)
            else:
                b = codes((d.k,), 32)
                ep = fx.epilogue(d.k, 2, fin, bias=b, fl_bias=4)
            nb = fx.qconv_wide_workspace(d, bits, 1, bits, 1)
            ws = torch.empty(nb, dtype=torch.uint8, device=dev)
            Ho = (d.h + 2 * d.pad - d.r) // d.stride + 1
            Wo = (d.w + 2 * d.pad - d.s) // d.stride + 1
            mk = d.n * Ho * Wo * d.k
            v = torch.empty(mk, dtype=torch.int64, device=dev)
            sc = torch.empty(1, dtype=torch.int32, device=dev)
            call = lambda: fx.qconv_wide(h, d, x, bits, 1, w, bits, 1, ep, v, sc, ws, nb)
            call()
            torch.cuda.synchronize(dev)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = 5
            e0.record()
            for _ in range(reps):
                call()
            e1.record()
            torch.cuda.synchronize(dev)
            ms = e0.elapsed_time(e1) / reps
            pairs = planes(bits, bits)
            ops = pairs * 2.0 * (mk // d.k) * d.k * wrow
            out[f"{name}_{bits}x{bits}"] = {
                "ms": round(ms, 4), "plane_pairs": pairs, "workspace_mb": round(nb / 2 ** 20, 1),
                "int8_tops_per_call": round(ops / (ms * 1e-3) / 1e12, 1), "outputs": mk,
                "value_bytes": 8 * mk}
            flags = fx.sync_status(h)
            assert flags & ~fx.FLAG_RANGE == 0, flags
            del ws
    h.close()
    return out


def steps_figures(dev):
    """Each hot-path call alone at ResNet-50 b256's largest tensors, inputs
    resident in HBM: quantize of the padded network input (256x224x224x4
    fp32), and over conv1-shaped int32 accumulators (256x112x112x64, Scale +
    ReLU epilogue) the FL search (min / max pass included), the
    requantization, the fused FxP-QLayer and the layer error against an fp32
    reference.  Algorithmic bytes: 4 B per fp32 or int32 value read, 1 B per
    code written (the search writes none); 5 timed calls after one untimed."""
    import torch
    from paper_2203_12091_amd import fxpq as fx
    h = fx.Handle(0)
    fx.set_stream(h, torch.cuda.current_stream())
    gen = torch.Generator(device=dev).manual_seed(12)
    x = torch.randn((256, 224, 224, 4), generator=gen, device=dev)
    acc = torch.randint(-2 ** 20, 2 ** 20, (256 * 112 * 112, 64), generator=gen, device=dev,
                        dtype=torch.int32)
    ref = torch.randn(acc.shape, generator=gen, device=dev)
    a1 = torch.randint(2 ** 14, 2 ** 15, (64,), generator=gen, device=dev, dtype=torch.int32)
    a2 = torch.randint(-2 ** 20, 2 ** 20, (64,), generator=gen, device=dev, dtype=torch.int32)
    fin = torch.tensor([8, 5, 1, 0], dtype=torch.int32, device=dev)
    ep = fx.epilogue(64, 9, fin, relu=True, scale=a1, fl_scale=15, shift=a2, fl_shift=20)
    fmt_x = torch.tensor([8, 5, 1, 0], dtype=torch.int32, device=dev)
    fmt_a = torch.zeros(4, dtype=torch.int32, device=dev)
    fmt_q = torch.zeros(4, dtype=torch.int32, device=dev)
    cx = torch.empty(x.numel(), dtype=torch.int8, device=dev)
    ca = torch.empty(acc.numel(), dtype=torch.int8, device=dev)
    alt = torch.empty(acc.numel(), dtype=torch.int8, device=dev)
    err = torch.empty(4, dtype=torch.float64, device=dev)
    n_x, n_a = x.numel(), acc.numel()
    src = fx.src_acc(acc, ep)
    calls = {
        "a1_quantize_fp32": (lambda: fx.quantize(h, x, n_x, fmt_x, cx, fx.C8), 5 * n_x),
        "a2_fl_search_acc": (lambda: fx.fl_search(h, src, n_a, 8, fx.SIGN_AUTO, -8, 15, fmt_a), 4 * n_a),
        "a4_requant_acc": (lambda: fx.requant(h, src, n_a, fmt_a, ca, fx.C8), 5 * n_a),
        "a2a4_qlayer_acc": (lambda: fx.qlayer(h, src, n_a, 8, fx.SIGN_AUTO, -8, 15, fmt_q, ca, fx.C8, alt),
                            5 * n_a),
        "a5_layer_error": (lambda: fx.layer_error(h, ref, ca, fx.C8, fmt_a, n_a, err), 5 * n_a),
    }
    out = {"tensors": {"input": list(x.shape), "acc": [256, 112, 112, 64]}}
    for name, (call, nbytes) in calls.items():
        call()
        torch.cuda.synchronize(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            call()
        e1.record()
        torch.cuda.synchronize(dev)
        ms = e0.elapsed_time(e1) / 5
        gbs = nbytes / (ms * 1e-3) / 1e9
        out[name] = {"ms": round(ms, 4), "algorithmic_bytes": nbytes, "gbs": round(gbs, 1),
                     "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}
    assert fx.sync_status(h) == 0
    h.close()
    return out


def conv_rooflines(net, dev, predict=False):
    """Per conv / FC call of one more (untimed, warm) forward, an event pair
    around each: its int8 TOP/s against its own roofline min(peak, AI x HBM
    peak), AI = int8 ops per HBM byte the call must move: input codes and
    weights, plus the int32 accumulators (fxpq_qconv) or the 8-bit codes
    (fxpq_cblock_predicted, which keeps the accumulators on chip); and the
    aggregate over the calls above the ridge point (peak / HBM bandwidth =
    625 ops/B), the ones the matrix cores bound."""
    import torch
    ridge = INT8_PEAK_TOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    classes = ("qconv", "cblock_pred")
    net.prepare_timers(1, classes=classes)
    m0 = net.misses
    net.forward(predict=predict)
    torch.cuda.synchronize(dev)
    run = net.pcalls if (net.predict and predict) else net.calls
    calls = [c for c in run if c[0] in classes]
    assert net.misses == m0 and len(calls) == len(net.timers), "a warm forward missed"
    names = [n.name for op, n, *r in net.ops if op in ("conv", "fc")]
    ops = ms = 0.0
    layers = 0
    per = []
    for name, (cls, work, fn, args), (_, _, e0, e1) in zip(names, calls, net.timers):
        t = e0.elapsed_time(e1)
        if fn.__name__ == "fxpq_qgemm":  # M, N, K
            m, n_, k, cin_bytes = args[1], args[2], args[3], args[1] * args[3]
        else:
            d = args[1]._obj
            ho = (d.h + 2 * d.pad - d.r) // d.stride + 1
            wo = (d.w + 2 * d.pad - d.s) // d.stride + 1
            m, n_, k, cin_bytes = d.n * ho * wo, d.k, d.r * d.s * d.c, d.n * d.h * d.w * d.c
        out_bytes = (1 if cls == "cblock_pred" else 4) * m * n_
        hbm = cin_bytes + n_ * k + out_bytes
        ai = work / hbm
        roof = min(INT8_PEAK_TOPS, ai * HBM_PEAK_GBS / 1000.0)
        tops = work / (t * 1e-3) / 1e12
        e = {"layer": name, "call": cls, "M": m, "N": n_, "K": k, "ms": round(t, 4),
             "tops": round(tops, 1), "ai": round(ai, 1), "roofline_tops": round(roof, 1),
             "frac_of_roofline": round(tops / roof, 3)}
        if cls == "cblock_pred":
            alu = PRED_OPS_PER_VALUE * m * n_ / (t * 1e-3) / 1e12
            e.update(alu_tops=round(alu, 2), alu_frac=round(alu / ALU_PEAK_TOPS, 3))
        per.append(e)
        if ai > ridge:
            ops += work
            ms += t
            layers += 1
    net.timers = None
    agg = None
    if layers:
        tops = ops / (ms * 1e-3) / 1e12
        agg = {"layers": layers, "ridge_ops_per_byte": round(ridge, 1), "achieved": round(tops, 1),
               "frac": round(tops / INT8_PEAK_TOPS, 4), "ms_per_forward": round(ms, 3)}
    roof_ms = sum(p["ms"] * p["frac_of_roofline"] for p in per)
    tot_ms = sum(p["ms"] for p in per)
    return agg, per, {"ms_at_own_roofline": round(roof_ms, 3), "ms": round(tot_ms, 3),
                      "frac": round(roof_ms / tot_ms, 4) if tot_ms else None}


def contraction_times(net):
    """(ms, launches, int8 ops) of the contraction alone: every conv / FC of
    one more (untimed) forward with the standard calls (fxpq_qconv /
    fxpq_qgemm, int32 accumulators)."""
    from paper_2203_12091_amd import fxpq as fx
    fx.timer_start(net.h, fx.TIMER_QCONV)
    net.forward(predict=False)
    out = fx.timer_read(net.h)
    fx.timer_start(net.h, fx.TIMER_OFF)
    return out


def predicted_times(net):
    """(ms, launches, int8 ops, output values) of the predicted C-Blocks of
    one more (untimed, warm) forward."""
    from paper_2203_12091_amd import fxpq as fx
    if not net.predict:
        return 0.0, 0, 0.0, 0
    vals = 0
    for cls, work, fn, args in net.pcalls:
        if cls == "cblock_pred":
            d = args[1]._obj
            ho = (d.h + 2 * d.pad - d.r) // d.stride + 1
            wo = (d.w + 2 * d.pad - d.s) // d.stride + 1
            vals += d.n * ho * wo * d.k
    fx.timer_start(net.h, fx.TIMER_CBLOCK_PRED)
    m0 = net.misses
    net.forward()
    ms, n, ops = fx.timer_read(net.h)
    fx.timer_start(net.h, fx.TIMER_OFF)
    assert net.misses == m0, "a warm forward missed"
    return ms, n, ops, vals


def cold_forward_ms(net, dev, reps=3):
    """Forwards right after every activation format changed (the formats
    reset to zero), as in an Algorithm 1 / 2 trial: (ms of such a forward
    with the standard calls, which a caller that changed formats runs; ms of
    one with predicted calls whose predictions fail, rerun from the first
    miss), each averaged over reps."""
    import torch
    out = []
    for predict in (False, True):
        tot = 0.0
        for _ in range(reps):
            for f in net.act_fmt.values():
                f.zero_()
            for op, n, *r in net.ops:
                if r and "mm" in r[0]:
                    r[0]["mm"].fill_(float("nan"))
            if hasattr(net, "input_mm"):
                net.input_mm.fill_(float("nan"))
            torch.cuda.synchronize(dev)
            t0 = time.perf_counter()
            net.forward(predict=predict)
            torch.cuda.synchronize(dev)
            tot += time.perf_counter() - t0
        out.append(round(tot * 1000.0 / reps, 3))
    return tuple(out)


def network_figures(dev, name, steps=5):
    """Another workload at its stated size (AlexNet b64, VGG-16 b128,
    ResNet-18 b256, 224x224): one untimed forward, `steps` timed forwards,
    then one forward each with the window pass and the contraction timed by
    the library's events, the compute-bound convolutions, and a cold
    forward."""
    import torch
    from paper_2203_12091_amd import fxpq as fx
    from paper_2203_12091_amd import nets
    net = nets.CalibNet(name, device=str(dev))
    b = net.batch
    net.forward()
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for i in range(steps):
        net.forward()
    torch.cuda.synchronize(dev)
    el = time.perf_counter() - t0
    fx.timer_start(net.h, fx.TIMER_FLS_WINDOW)
    net.forward()
    win_ms, win_n, win_bytes = fx.timer_read(net.h)
    cv_ms, cv_n, cv_ops = contraction_times(net)
    agg, _, own = conv_rooflines(net, dev)
    if net.results()["flags"]:
        print(f"bench.py: {name}: device flags", file=sys.stderr)
        sys.exit(1)
    gbs = win_bytes / (win_ms * 1e-3) / 1e9
    out = {"workload": f"{name}_b{b}_{net.image}_dfx_calibration_forward", "batch": b,
           "images_per_s": round(b * steps / el, 1), "ms_per_forward": round(el * 1000 / steps, 3),
           "ms_per_forward_cold": cold_forward_ms(net, dev)[0],
           "fl_search_gbs": round(gbs, 1), "fl_search_frac": round(gbs / HBM_PEAK_GBS, 4),
           "mfma_tops": round(cv_ops / (cv_ms * 1e-3) / 1e12, 1),
           "mfma_frac": round(cv_ops / (cv_ms * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4),
           "conv_frac_of_own_roofline": own["frac"], "compute_bound_layers": agg}
    net.close()
    return out


def fc_figures(dev, reps=200):
    """The single-FC-layer workload at WL 8 as one device pipeline: FL
    search + quantize of W (256x512) and A (32x512), the int8 GEMM with
    int32 accumulation, the fused FxP-QLayer of the 32x256 product (FL search
    + requantization to WL 8); microseconds per pipeline over `reps` calls
    after one untimed one (latency-bound: no roofline fraction)."""
    import torch
    import synth
    from paper_2203_12091_amd import fxpq as fx
    h = fx.Handle(0)
    fx.set_stream(h, torch.cuda.current_stream())
    W = torch.from_numpy(synth.normal(0, "fc.w", (256, 512), std=0.05).ravel()).to(dev)
    A = torch.from_numpy(synth.relu_normal(0, "fc.a", (32, 512)).ravel()).to(dev)
    fw, fa, fy = (torch.zeros(4, dtype=torch.int32, device=dev) for _ in range(3))
    wc = torch.empty(W.numel(), dtype=torch.int8, device=dev)
    ac = torch.empty(A.numel(), dtype=torch.int8, device=dev)
    cs = torch.empty(256, dtype=torch.int32, device=dev)
    acc = torch.empty((32, 256), dtype=torch.int32, device=dev)
    mm = torch.empty(2, dtype=torch.float64, device=dev)
    yc = torch.empty(acc.numel(), dtype=torch.int8, device=dev)
    alt = torch.empty(acc.numel() + 16, dtype=torch.int8, device=dev)
    sw, sa = fx.src_f32(W), fx.src_f32(A)
    fx.fl_search(h, sw, W.numel(), 8, fx.SIGN_AUTO, -8, 15, fw)
    torch.cuda.synchronize(dev)
    ep = fx.epilogue(256, int(fw.cpu()[1]), fa)
    sy = fx.src_acc(acc, ep, mm)

    def pipeline():
        fx.fl_search(h, sw, W.numel(), 8, fx.SIGN_AUTO, -8, 15, fw)
        fx.fl_search(h, sa, A.numel(), 8, fx.SIGN_AUTO, -8, 15, fa)
        fx.quantize(h, W, W.numel(), fw, wc, fx.I8)
        fx.quantize(h, A, A.numel(), fa, ac, fx.C8)
        fx.weight_colsum(h, wc, 256, 512, cs)
        fx.qgemm(h, 32, 256, 512, ac, fx.C8, wc, cs, ep, acc, mm)
        fx.qlayer(h, sy, acc.numel(), 8, fx.SIGN_AUTO, -8, 15, fy, yc, fx.C8, alt)

    pipeline()
    torch.cuda.synchronize(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        pipeline()
    e1.record()
    torch.cuda.synchronize(dev)
    us = e0.elapsed_time(e1) * 1000.0 / reps
    assert fx.sync_status(h) == 0
    h.close()
    return {"workload": "fc_256x512_b32_wl8", "us_per_call": round(us, 2),
            "calls": "fl_search W, fl_search A, quantize W, quantize A, colsum, qgemm, qlayer"}


def sweep_figures(dev):
    """The per-layer sensitivity sweep of ResNet-50 b256 (54 layers x activation
    WL 8..4 x weight WL 8..2 = 1890 layer evaluations), reported alongside: the
    FP32 teacher and the weight quantization are set-up; one untimed sweep,
    then one timed sweep between two synchronizations."""
    import torch
    from paper_2203_12091_amd import sweep
    t0 = time.perf_counter()
    sw = sweep.Sweep("resnet50", batch=BATCH, image=IMAGE, device=str(dev))
    torch.cuda.synchronize(dev)
    setup = time.perf_counter() - t0
    sw.run()
    t = sw.timed_run()
    res = sw.results()
    if res["flags"]:
        print(f"bench.py: sweep device flags {res['flags']:#x}", file=sys.stderr)
        sys.exit(1)
    steps = len(sw.steps)
    sw.close()
    return {"workload": "resnet50_b256_224_sensitivity_sweep", "layer_evaluations": steps,
            "seconds": round(t, 4), "layer_eval_images_per_s": round(BATCH * steps / t, 1),
            "setup_seconds_untimed": round(setup, 2)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only; --gpus {args.gpus} is not supported",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2203_12091_amd import fxpq as fx
    from paper_2203_12091_amd import nets

    dev = torch.device("cuda:0")
    if args.mode == "copy":
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize(dev)
        dst.copy_(src)
        torch.cuda.synchronize(dev)
        print(json.dumps({"copy_bytes": src.numel() * 4}), flush=True)
        return

    if args.mode == "sweep":
        print(json.dumps(sweep_figures(dev)), flush=True)
        return
    if args.mode == "qparams":
        print(json.dumps(qparams_figures(dev)), flush=True)
        return
    if args.mode == "reduction":
        print(json.dumps(reduction_figures(dev)), flush=True)
        return
    if args.mode == "wide":
        print(json.dumps(wide_figures(dev)), flush=True)
        return
    if args.mode == "steps":
        print(json.dumps(steps_figures(dev)), flush=True)
        return

    net = nets.CalibNet("resnet50", batch=BATCH, image=IMAGE, device="cuda:0")
    for _ in range(args.warmup):
        net.forward()
    torch.cuda.synchronize(dev)
    if args.mode == "profile":
        print(json.dumps({"profile_forwards": args.warmup}), flush=True)
        return

    # timed region: exactly `steps` forwards; the library brackets the window
    # launches of the last one with events (one forward's worth of event
    # records instead of all of them).  The library creates its timer events
    # on the first fxpq_timer_start (tens of thousands of hipEventCreate):
    # done here, before the timed region, so that only the event records are
    # inside it.
    fx.timer_start(net.h, fx.TIMER_FLS_WINDOW)
    fx.timer_start(net.h, fx.TIMER_OFF)
    torch.cuda.synchronize(dev)
    m0 = net.misses
    t0 = time.perf_counter()
    for i in range(args.steps):
        if i == args.steps - 1:
            fx.timer_start(net.h, fx.TIMER_FLS_WINDOW)
        net.forward()
    torch.cuda.synchronize(dev)
    elapsed = time.perf_counter() - t0
    timed_misses = net.misses - m0
    win_ms, win_n, win_bytes = fx.timer_read(net.h)
    res = net.results()
    if res["flags"]:
        print(f"bench.py: device flags {res['flags']:#x}", file=sys.stderr)
        sys.exit(1)

    # more (untimed) forwards: the predicted C-Blocks (the dominant kernel),
    # the contraction alone and the requantization (standard calls), the
    # per-layer rooflines of both, cold forwards
    pr_ms, pr_n, pr_ops, pr_vals = predicted_times(net)
    cv_ms, cv_n, cv_ops = contraction_times(net)
    fx.timer_start(net.h, fx.TIMER_REQUANT)
    net.forward(predict=False)
    rq_ms, rq_n, rq_bytes = fx.timer_read(net.h)
    fx.timer_start(net.h, fx.TIMER_OFF)
    net.forward()
    cbound, per_layer, own = conv_rooflines(net, dev, predict=False)
    _, per_pred, _ = conv_rooflines(net, dev, predict=True) if net.predict else (None, [], None)
    cold_ms, miss_ms = cold_forward_ms(net, dev)
    net.forward()  # back to the steady state (formats of the batch known)

    ms = elapsed * 1000.0 / args.steps
    value = BATCH * args.steps / elapsed
    achieved = win_bytes / (win_ms * 1e-3) / 1e9
    traffic = committed_traffic()
    pr_alu = PRED_OPS_PER_VALUE * pr_vals / (pr_ms * 1e-3) / 1e12 if pr_ms else 0.0
    out = {
        "metric": "calibration images/s (ResNet-50 b256 DFX); FL-search GB/s; int8 MFMA % peak",
        "value": round(value, 2),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "ms_per_step_cold": cold_ms,
        "ms_per_step_mispredicted": miss_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "resnet50_b256_224_dfx_calibration_forward", "batch": BATCH,
                   "image": IMAGE, "weight_wl": 8, "act_wl": 8, "fl_range": [-8, 15],
                   "parallelism": "single_gpu", "predicted_cblocks": sum(
                       1 for c in (net.pcalls if net.predict else []) if c[0] == "cblock_pred"),
                   "timed_forwards_rerun": timed_misses},
        "roofline": {"bound": "alu", "achieved": round(pr_alu, 2), "peak": round(ALU_PEAK_TOPS, 2),
                     "unit": "TOP/s", "frac": round(pr_alu / ALU_PEAK_TOPS, 4), "traffic": traffic,
                     "kernel": "k_qconv predicted C-Block (conv + epilogue + FL-search window + codes)",
                     "launches": pr_n, "avg_launch_ms": round(pr_ms / max(pr_n, 1), 5),
                     "algorithmic_ops_per_launch": round(PRED_OPS_PER_VALUE * pr_vals / max(pr_n, 1)),
                     "ops_per_output_value": PRED_OPS_PER_VALUE, "ms_per_forward": round(pr_ms, 3),
                     "int8_tops": round(pr_ops / (pr_ms * 1e-3) / 1e12, 1) if pr_ms else None},
        "fl_search_gbs": round(achieved, 1),
        "fl_search": {"kernel": "predicted / standard FL-search window passes over the network input "
                                "and the eltwise sums", "achieved": round(achieved, 1), "unit": "GB/s",
                      "frac": round(achieved / HBM_PEAK_GBS, 4), "launches": win_n,
                      "ms_per_forward": round(win_ms, 3),
                      "algorithmic_bytes_per_launch": round(win_bytes / max(win_n, 1))},
        "mfma": {"kernel": "k_qconv", "achieved": round(cv_ops / (cv_ms * 1e-3) / 1e12, 1),
                 "unit": "TOP/s", "peak": INT8_PEAK_TOPS,
                 "frac": round(cv_ops / (cv_ms * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4),
                 "ms_per_forward": round(cv_ms, 3), "launches": cv_n},
    }
    if rq_n:
        out["requant"] = {"kernel": "k_requant", "achieved": round(rq_bytes / (rq_ms * 1e-3) / 1e9, 1),
                          "unit": "GB/s", "ms_per_forward": round(rq_ms, 3), "launches": rq_n}
    if cbound:
        out["mfma"]["compute_bound_layers"] = cbound
    out["mfma"]["own_roofline"] = own
    out["mfma"]["per_layer"] = per_layer
    out["predicted_cblock"] = {"per_layer": per_pred}
    if not args.no_sweep:
        out["sweep"] = sweep_figures(dev)
    net.close()
    del net
    if not args.no_configs:
        out["configs"] = {"fc": fc_figures(dev)}
        for name in ("alexnet", "vgg16", "resnet18"):
            out["configs"][name] = network_figures(dev, name)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_sample_batch)
        if not args.no_configs:
            out["cpu_baseline"]["configs"] = cpu_configs()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

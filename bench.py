"""Benchmark: DFX calibration forward of ResNet-50 at batch 256 on one MI355X.

One step = one complete calibration forward over a 256x3x224x224 batch:
input FL search + quantize + layer error, every C-Block (int8 MFMA conv +
epilogue, FL search over the whole output tensor, requantization), max-pool,
residual adds (FL search + requant), global avg-pool (+ FxP-QLayer) and the
final FC to integer logits.  Parameters are quantized once during set-up
(weight FL searches are not part of a calibration step).  Inputs are resident
in HBM before timing starts.

Prints ONE JSON line (see the repository contract).  --gpus above 1 exits: this
build runs on one GPU.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BATCH, IMAGE = 256, 224


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-image", type=int, default=224)
    return ap.parse_args()


def cpu_baseline(image):
    """The oracle, as it stands, on a bounded sample: a calibration forward of
    one image (parameters quantized beforehand), timed on the host cores."""
    import oracle
    t_prep = time.perf_counter()
    f = oracle.nets.prepare("resnet50", batch=1, image=image)
    t0 = time.perf_counter()
    f.run()
    t = time.perf_counter() - t0
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": round(1.0 / t, 5), "unit": "images/s", "cores": cores, "kind": "oracle",
            "sample": f"ResNet-50 DFX calibration forward of 1 image {image}x{image} "
                      f"(parameters pre-quantized, {t:.1f} s forward, "
                      f"{t0 - t_prep:.1f} s parameter set-up untimed)"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only; --gpus {args.gpus} is not supported",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2203_12091_amd import nets

    dev = torch.device("cuda:0")
    net = nets.CalibNet("resnet50", batch=BATCH, image=IMAGE, device="cuda:0")
    for _ in range(args.warmup):
        net.forward()
    torch.cuda.synchronize(dev)

    # timed region: exactly `steps` forwards; the FL-search calls (the dominant
    # kernel) are bracketed by pre-created events on the library's stream.
    net.prepare_timers(args.steps, classes=("fl_search",))
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        net.forward()
    torch.cuda.synchronize(dev)
    elapsed = time.perf_counter() - t0
    res = net.results()
    if res["flags"]:
        print(f"bench.py: device flags {res['flags']:#x}", file=sys.stderr)
        sys.exit(1)

    ms = elapsed * 1000.0 / args.steps
    value = BATCH * args.steps / elapsed
    roof = net.roofline()
    out = {
        "metric": "calibration images/s (ResNet-50 b256 DFX); FL-search GB/s; int8 MFMA % peak",
        "value": round(value, 2),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "resnet50_b256_224_dfx_calibration_forward", "batch": BATCH,
                   "image": IMAGE, "weight_wl": 8, "act_wl": 8, "fl_range": [-8, 15],
                   "parallelism": "single_gpu"},
        "roofline": roof,
        "fl_search_gbs": roof.get("achieved"),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_sample_image)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

"""Helpers for the GPU parity tests (imported by test modules, not collected)."""
import sys

import numpy as np

DEV = "cuda:0"


def note(*a):
    """Names the case about to run on the GPU (flushed, so a fault still shows it)."""
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def torch():
    import torch as T
    return T


def dev(a):
    T = torch()
    return T.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    T = torch()
    T.cuda.synchronize()
    return t.cpu().numpy()


def empty(shape, dtype):
    T = torch()
    return T.empty(shape, dtype=dtype, device=DEV)


def fmt_dev(wl, fl, sign):
    T = torch()
    return T.tensor([wl, fl, sign, 0], dtype=T.int32, device=DEV)


def fmt_new():
    T = torch()
    return T.full((4,), -999, dtype=T.int32, device=DEV)


def fmt_host(t):
    wl, fl, sign, status = (int(v) for v in host(t))
    return wl, fl, sign, status


def decode8(codes, off):
    c = np.asarray(codes).astype(np.int64)
    return c + 128 if off else c

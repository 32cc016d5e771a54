"""ctypes wrappers over the oracle's C library (test infrastructure only)."""
import ctypes as C
import os

import numpy as np

from . import build as _build

SIGN_AUTO = -1
_lib = None


class OracleError(RuntimeError):
    pass


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _lib = C.CDLL(_build.LIB)
        _declare(_lib)
    return _lib


def _declare(L):
    p = C.c_void_p
    i = C.c_int
    i64 = C.c_int64
    sigs = {
        "orc_qrange": [i, i, p, p],
        "orc_sign_f32": [p, i64],
        "orc_sign_i64": [p, i64],
        "orc_quantize_f32": [p, i64, i, i, i, p],
        "orc_quantize_i64": [p, i64, i, i, i, i, p],
        "orc_sse_f32": [p, i64, i, i, i, p],
        "orc_sse_i64": [p, i64, i, i, i, i, p],
        "orc_fl_search_f32": [p, i64, i, i, i, i, p, p, p],
        "orc_fl_search_i64": [p, i64, i, i, i, i, i, p, p, p],
        "orc_gemm": [p, p, i64, i64, i64, p],
        "orc_conv2d": [p, i, i, i, i, p, i, i, i, i, i, p],
        "orc_conv2d_point": [p, i, i, i, i, p, i, i, i, i, i, i, i, i, i, p],
        "orc_epilogue": [p, i, i, i64, i, p, i, p, i, p, i, i, p, p],
        "orc_maxpool": [p, i, i, i, i, i, i, i, p],
        "orc_avgpool_global": [p, i, i, i, i64, p],
        "orc_eltwise_add": [p, i, p, i, i64, i, p, p],
        "orc_layer_error": [p, p, i64, i, i, i, p],
        "orc_teacher_conv2d": [p, i, i, i, i, p, i, i, i, i, i, p],
        "orc_teacher_affine": [p, i, i, i64, p, p, p, i, p],
        "orc_teacher_avgpool": [p, i, i, i64, p],
    }
    for name, args in sigs.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = C.c_int


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p) if a is not None else None


def _check(st, what):
    if st != 0:
        raise OracleError(f"{what}: oracle status {st}")


def _f32(x):
    return np.ascontiguousarray(x, dtype=np.float32)


def _i64(x):
    return np.ascontiguousarray(x, dtype=np.int64)


def _i32(x):
    return np.ascontiguousarray(x, dtype=np.int32)


def qrange(k, sign):
    """Eq. 12: (Qmin, Qmax) of a k-bit code with sign strategy S."""
    lo, hi = C.c_int64(), C.c_int64()
    _check(lib().orc_qrange(k, sign, C.byref(lo), C.byref(hi)), "qrange")
    return lo.value, hi.value


def sign_of(x):
    """Eq. 6: 1 if the smallest value is negative."""
    if np.asarray(x).dtype == np.float32:
        x = _f32(x)
        return lib().orc_sign_f32(_ptr(x), x.size)
    x = _i64(x)
    return lib().orc_sign_i64(_ptr(x), x.size)


def quantize_f32(x, k, fl, sign):
    """Eq. 10-13 on fp32 data; returns int32 codes."""
    x = _f32(x)
    out = np.empty(x.shape, np.int32)
    _check(lib().orc_quantize_f32(_ptr(x), x.size, k, fl, sign, _ptr(out)), "quantize_f32")
    return out


def quantize_i64(v, s, k, fl, sign):
    """Eq. 10-13 on the exact values v * 2^-s; returns int32 codes."""
    v = _i64(v)
    out = np.empty(v.shape, np.int32)
    _check(lib().orc_quantize_i64(_ptr(v), v.size, s, k, fl, sign, _ptr(out)), "quantize_i64")
    return out


def sse_f32(x, k, fl, sign):
    x = _f32(x)
    r = C.c_double()
    _check(lib().orc_sse_f32(_ptr(x), x.size, k, fl, sign, C.byref(r)), "sse_f32")
    return r.value


def sse_i64(v, s, k, fl, sign):
    v = _i64(v)
    r = C.c_double()
    _check(lib().orc_sse_i64(_ptr(v), v.size, s, k, fl, sign, C.byref(r)), "sse_i64")
    return r.value


def fl_search_f32(x, k, sign=SIGN_AUTO, fl_lo=-8, fl_hi=15):
    """Exhaustive search; returns (fl, sign, sse[fl_lo..fl_hi])."""
    x = _f32(x)
    fl, sg = C.c_int(), C.c_int()
    sse = np.empty(fl_hi - fl_lo + 1, np.float64)
    _check(lib().orc_fl_search_f32(_ptr(x), x.size, k, sign, fl_lo, fl_hi, C.byref(fl),
                                   C.byref(sg), _ptr(sse)), "fl_search_f32")
    return fl.value, sg.value, sse


def fl_search_i64(v, s, k, sign=SIGN_AUTO, fl_lo=-8, fl_hi=15):
    v = _i64(v)
    fl, sg = C.c_int(), C.c_int()
    sse = np.empty(fl_hi - fl_lo + 1, np.float64)
    _check(lib().orc_fl_search_i64(_ptr(v), v.size, s, k, sign, fl_lo, fl_hi, C.byref(fl),
                                   C.byref(sg), _ptr(sse)), "fl_search_i64")
    return fl.value, sg.value, sse


def gemm(A, B):
    """C[m][n] = sum_k A[m][k] * B[n][k], exact (codes of up to 32 bits, signed
    or unsigned); int64 result."""
    A, B = _i64(A), _i64(B)
    M, K = A.shape
    N = B.shape[0]
    assert B.shape[1] == K
    out = np.empty((M, N), np.int64)
    _check(lib().orc_gemm(_ptr(A), _ptr(B), M, N, K, _ptr(out)), "gemm")
    return out


def conv_out_hw(H, W, R, S, stride, pad):
    return (H + 2 * pad - R) // stride + 1, (W + 2 * pad - S) // stride + 1


def conv2d(x, w, stride, pad):
    """Direct convolution, NCHW x KCRS -> NKHW int64 (codes as gemm)."""
    x, w = _i64(x), _i64(w)
    N, Cc, H, W = x.shape
    K, C2, R, S = w.shape
    assert C2 == Cc
    Ho, Wo = conv_out_hw(H, W, R, S, stride, pad)
    out = np.empty((N, K, Ho, Wo), np.int64)
    _check(lib().orc_conv2d(_ptr(x), N, Cc, H, W, _ptr(w), K, R, S, stride, pad, _ptr(out)),
           "conv2d")
    return out


def conv2d_point(x, w, stride, pad, n, k, oh, ow):
    x, w = _i64(x), _i64(w)
    N, Cc, H, W = x.shape
    K, _, R, S = w.shape
    y = C.c_int64()
    _check(lib().orc_conv2d_point(_ptr(x), N, Cc, H, W, _ptr(w), K, R, S, stride, pad,
                                  n, k, oh, ow, C.byref(y)), "conv2d_point")
    return y.value


def epilogue(acc, s_acc, bias=None, fl_b=0, a1=None, fl_a1=0, a2=None, fl_a2=0, relu=False):
    """C-Block epilogue on NCHW (or NC) accumulators; returns (v int64, s_out)."""
    acc = _i64(acc)
    N, Cc = acc.shape[0], acc.shape[1]
    hw = int(np.prod(acc.shape[2:])) if acc.ndim > 2 else 1
    v = np.empty_like(acc)
    s_out = C.c_int()
    b = _i64(bias) if bias is not None else None
    m1 = _i64(a1) if a1 is not None else None
    m2 = _i64(a2) if a2 is not None else None
    _check(lib().orc_epilogue(_ptr(acc), N, Cc, hw, s_acc, _ptr(b), fl_b, _ptr(m1), fl_a1,
                              _ptr(m2), fl_a2, int(bool(relu)), _ptr(v), C.byref(s_out)),
           "epilogue")
    return v, s_out.value


def maxpool(x, k, stride, pad):
    x = _i32(x)
    N, Cc, H, W = x.shape
    Ho, Wo = conv_out_hw(H, W, k, k, stride, pad)
    out = np.empty((N, Cc, Ho, Wo), np.int32)
    _check(lib().orc_maxpool(_ptr(x), N, Cc, H, W, k, stride, pad, _ptr(out)), "maxpool")
    return out


def avgpool_global(x, recip):
    x = _i32(x)
    N, Cc = x.shape[:2]
    hw = int(np.prod(x.shape[2:]))
    out = np.empty((N, Cc), np.int64)
    _check(lib().orc_avgpool_global(_ptr(x), N, Cc, hw, int(recip), _ptr(out)), "avgpool")
    return out


def eltwise_add(a, fa, b, fb, relu):
    a, b = _i32(a), _i32(b)
    assert a.shape == b.shape
    v = np.empty(a.shape, np.int64)
    s_out = C.c_int()
    _check(lib().orc_eltwise_add(_ptr(a), fa, _ptr(b), fb, a.size, int(bool(relu)), _ptr(v),
                                 C.byref(s_out)), "eltwise_add")
    return v, s_out.value


def layer_error(ref, codes, k, fl, sign):
    """Returns [exact SSE, min(ref), max(ref), population std(ref)]."""
    ref, codes = _f32(ref), _i32(codes)
    assert ref.size == codes.size
    out = np.empty(4, np.float64)
    _check(lib().orc_layer_error(_ptr(ref), _ptr(codes), ref.size, k, fl, sign, _ptr(out)),
           "layer_error")
    return out


# ---- FP32 teacher (reference activations of the sensitivity sweep) ----------
def teacher_conv2d(x, w, stride, pad):
    """fp32 conv, NCHW x KCRS -> NKHW: fp64 sum of the exact products in the
    order r, s, c (padded taps skipped), rounded once to fp32."""
    x, w = _f32(x), _f32(w)
    N, Cc, H, W = x.shape
    K, C2, R, S = w.shape
    assert C2 == Cc
    Ho, Wo = conv_out_hw(H, W, R, S, stride, pad)
    out = np.empty((N, K, Ho, Wo), np.float32)
    _check(lib().orc_teacher_conv2d(_ptr(x), N, Cc, H, W, _ptr(w), K, R, S, stride, pad,
                                    _ptr(out)), "teacher_conv2d")
    return out


def teacher_affine(t, a1=None, a2=None, bias=None, relu=False):
    """Per channel (axis 1): relu?(fmaf(t, a1, a2)) or relu?(t + bias)."""
    t = _f32(t)
    N, Cc = t.shape[0], t.shape[1]
    hw = int(np.prod(t.shape[2:])) if t.ndim > 2 else 1
    m1 = None if a1 is None else _f32(a1)
    m2 = None if a2 is None else _f32(a2)
    b = None if bias is None else _f32(bias)
    out = np.empty_like(t)
    _check(lib().orc_teacher_affine(_ptr(t), N, Cc, hw, _ptr(m1), _ptr(m2), _ptr(b),
                                    int(bool(relu)), _ptr(out)), "teacher_affine")
    return out


def teacher_avgpool(x):
    """NCHW -> NC: (float)(sequential fp64 sum over h, w / (h * w))."""
    x = _f32(x)
    N, Cc = x.shape[:2]
    hw = int(np.prod(x.shape[2:]))
    out = np.empty((N, Cc), np.float32)
    _check(lib().orc_teacher_avgpool(_ptr(x), N, Cc, hw, _ptr(out)), "teacher_avgpool")
    return out

"""ctypes binding of libfxpq (include/fxpq.h): argument marshalling only.

Every function keeps the C name without the ``fxpq_`` prefix and takes device
pointers as Python ints or torch tensors (``tensor.data_ptr()`` is used).  All
arithmetic of the hot path runs in the HIP kernels of ``libfxpq.so``; when the
library is missing this module raises instead of falling back to anything.
"""
import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfxpq.so")

# enums (keep in sync with include/fxpq.h)
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_NONFINITE, ERR_OVERFLOW, ERR_HIP, ERR_ALLOC = range(7)
I8, U8OFF, I16, I32, I64, F32, C8, U32 = range(8)
SRC_F32, SRC_INT, SRC_ACC, SRC_ADD = range(4)
SIGN_AUTO = -1
FLAG_NONFINITE, FLAG_RANGE, FLAG_CODE = 0x1, 0x2, 0x4

EXPORTS = [
    "fxpq_create", "fxpq_destroy", "fxpq_set_stream", "fxpq_status_string", "fxpq_sync_status",
    "fxpq_quantize", "fxpq_requant", "fxpq_requant_addmm", "fxpq_fl_search", "fxpq_fl_search_static", "fxpq_qlayer", "fxpq_qlayer_predicted", "fxpq_preprocess", "fxpq_qconv", "fxpq_qgemm",
    "fxpq_qconv_wide_workspace", "fxpq_qconv_wide", "fxpq_acc_overflow",
    "fxpq_cblock", "fxpq_cblock_predicted", "fxpq_predicted_defer", "fxpq_predicted_decide",
    "fxpq_set_conv_tiling", "fxpq_weight_colsum", "fxpq_maxpool", "fxpq_avgpool_global", "fxpq_layer_error",
    "fxpq_epilogue_scale", "fxpq_dequantize", "fxpq_prediction_ties", "fxpq_timer_start",
    "fxpq_timer_read",
    "fxpq_teacher_conv", "fxpq_teacher_affine", "fxpq_teacher_add", "fxpq_teacher_maxpool",
    "fxpq_teacher_avgpool",
]
TIMER_OFF, TIMER_FLS_WINDOW, TIMER_QCONV, TIMER_REQUANT, TIMER_CBLOCK_PASS, TIMER_CBLOCK_PRED = range(6)
TILING_AUTO, TILING_GEMM, TILING_HALO = range(3)
ROUND_CONSERVATIVE, ROUND_NEUTRAL, ROUND_AGGRESSIVE = range(3)
PSI_PRINTED, PSI_MAX = range(2)


class Fmt(C.Structure):
    _fields_ = [("wl", C.c_int32), ("fl", C.c_int32), ("sign", C.c_int32), ("status", C.c_int32)]


class Epilogue(C.Structure):
    _fields_ = [("channels", C.c_int32), ("fl_w", C.c_int32), ("d_fmt_in", C.c_void_p),
                ("bias", C.c_void_p), ("fl_bias", C.c_int32), ("relu", C.c_int32),
                ("scale", C.c_void_p), ("fl_scale", C.c_int32), ("pad0", C.c_int32),
                ("shift", C.c_void_p), ("fl_shift", C.c_int32), ("pad1", C.c_int32)]


class Src(C.Structure):
    _fields_ = [("kind", C.c_int32), ("dtype", C.c_int32), ("x", C.c_void_p), ("x2", C.c_void_p),
                ("dtype2", C.c_int32), ("relu", C.c_int32), ("d_scale", C.c_void_p),
                ("d_fmt_a", C.c_void_p), ("d_fmt_b", C.c_void_p), ("ep", C.c_void_p),
                ("d_minmax", C.c_void_p)]


class ConvDesc(C.Structure):
    _fields_ = [(f, C.c_int32) for f in ("n", "h", "w", "c", "k", "r", "s", "stride", "pad")]


class FxpqError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {status_string(status)} ({status})")


_lib = None


def lib():
    """Loads libfxpq.so; raises when it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FileNotFoundError(
                f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                "(python -m paper_2203_12091_amd.build)")
        L = C.CDLL(LIB_PATH)
        p, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
        sig = {
            "fxpq_create": [p, C.c_int],
            "fxpq_destroy": [p],
            "fxpq_set_stream": [p, p],
            "fxpq_sync_status": [p, p],
            "fxpq_quantize": [p, p, i64, p, p, C.c_int],
            "fxpq_requant": [p, p, i64, p, p, C.c_int],
            "fxpq_requant_addmm": [p, p, i64, p, p, C.c_int, p, C.c_int, p, i32, p],
            "fxpq_fl_search": [p, p, i64, i32, i32, i32, i32, p, p],
            "fxpq_fl_search_static": [p, i64, i32, i32, i32, i32, p, p, p],
            "fxpq_qlayer": [p, p, i64, i32, i32, i32, i32, p, p, C.c_int, p],
            "fxpq_qlayer_predicted": [p, p, i64, i32, i32, i32, i32, p, p, C.c_int, p, p],
            "fxpq_preprocess": [p, p, i64, i32, i32, i32, i32, i32, p],
            "fxpq_qconv": [p, p, p, C.c_int, p, p, p, p, p],
            "fxpq_qgemm": [p, i64, i64, i64, p, C.c_int, p, p, p, p, p],
            "fxpq_qconv_wide_workspace": [p, i32, i32, i32, i32, p],
            "fxpq_qconv_wide": [p, p, p, i32, i32, p, i32, i32, p, p, p, p, i64],
            "fxpq_acc_overflow": [p, p, i64, i32, p],
            "fxpq_cblock": [p, p, p, C.c_int, p, p, p, i32, i32, i32, i32, p, p, C.c_int, p, p],
            "fxpq_cblock_predicted": [p, p, p, C.c_int, p, p, p, i32, i32, i32, i32, p, p, C.c_int,
                                      p, p],
            "fxpq_predicted_defer": [p, i32],
            "fxpq_predicted_decide": [p],
            "fxpq_weight_colsum": [p, p, i64, i64, p],
            "fxpq_set_conv_tiling": [p, i32],
            "fxpq_maxpool": [p, p, C.c_int, i32, i32, i32, i32, i32, i32, i32, p],
            "fxpq_avgpool_global": [p, p, C.c_int, p, i32, i32, i32, i64, p],
            "fxpq_layer_error": [p, p, p, C.c_int, p, i64, p],
            "fxpq_epilogue_scale": [p, p, p],
            "fxpq_dequantize": [p, p, C.c_int, p, i64, p],
            "fxpq_prediction_ties": [p, p, C.c_int, i32, i32, p],
            "fxpq_timer_start": [p, C.c_int],
            "fxpq_timer_read": [p, p, p, p],
            "fxpq_teacher_conv": [p, p, p, p, p],
            "fxpq_teacher_affine": [p, p, i64, i32, p, p, p, i32, p],
            "fxpq_teacher_add": [p, p, p, i64, i32, p],
            "fxpq_teacher_maxpool": [p, p, i32, i32, i32, i32, i32, i32, i32, p],
            "fxpq_teacher_avgpool": [p, p, i32, i32, i32, p],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = C.c_int
        L.fxpq_status_string.argtypes = [C.c_int]
        L.fxpq_status_string.restype = C.c_char_p
        _lib = L
    return _lib


def status_string(st):
    return lib().fxpq_status_string(st).decode()


def ptr(t):
    """Device pointer of a torch tensor (or an int / None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _call(name, *args):
    st = getattr(lib(), name)(*args)
    if st != OK:
        raise FxpqError(name, st)


class Handle:
    """Owns an fxpq_handle (and its scratch) on one device."""

    def __init__(self, device=0):
        self.h = C.c_void_p()
        _call("fxpq_create", C.byref(self.h), device)
        self.device = device

    def close(self):
        if self.h:
            _call("fxpq_destroy", self.h)
            self.h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def value(self):
        return self.h


def create(device=0):
    return Handle(device)


def destroy(h):
    h.close()


def set_stream(h, stream):
    """stream: a torch.cuda.Stream, a raw hipStream_t int, or None."""
    raw = getattr(stream, "cuda_stream", stream)
    _call("fxpq_set_stream", h.value, raw)


def sync_status(h):
    flags = C.c_uint32()
    _call("fxpq_sync_status", h.value, C.byref(flags))
    return flags.value


def quantize(h, x, n, d_fmt, codes, code_type):
    _call("fxpq_quantize", h.value, ptr(x), n, ptr(d_fmt), ptr(codes), code_type)


def requant(h, src, n, d_fmt, codes, code_type):
    _call("fxpq_requant", h.value, C.byref(src), n, ptr(d_fmt), ptr(codes), code_type)


def requant_addmm(h, src, n, d_fmt, codes, code_type, b, b_type, d_fmt_b, relu, d_add_minmax):
    _call("fxpq_requant_addmm", h.value, C.byref(src), n, ptr(d_fmt), ptr(codes), code_type, ptr(b),
          b_type, ptr(d_fmt_b), int(relu), ptr(d_add_minmax))


def fl_search(h, src, n, wl, sign, fl_lo, fl_hi, d_fmt_out, d_sse=None):
    _call("fxpq_fl_search", h.value, C.byref(src), n, wl, sign, fl_lo, fl_hi, ptr(d_fmt_out),
          ptr(d_sse))


def fl_search_static(src, n, wl, sign, fl_lo, fl_hi, d_fmt_out, d_sse=None, stream=None):
    """fxpq_fl_search_static: no handle, no allocation; stream is a raw HIP
    stream (int), a torch stream, or None for the default stream."""
    st = getattr(stream, "cuda_stream", stream)
    _call("fxpq_fl_search_static", C.byref(src), n, wl, sign, fl_lo, fl_hi, ptr(d_fmt_out),
          ptr(d_sse), st)


def preprocess(h, src, n, wl, strategy, psi_rule, fl_lo, fl_hi, d_fmt_out):
    _call("fxpq_preprocess", h.value, C.byref(src), n, wl, strategy, psi_rule, fl_lo, fl_hi,
          ptr(d_fmt_out))


def set_conv_tiling(h, mode):
    _call("fxpq_set_conv_tiling", h.value, mode)


def predicted_defer(h, on):
    _call("fxpq_predicted_defer", h.value, int(bool(on)))


def predicted_decide(h):
    _call("fxpq_predicted_decide", h.value)


def qlayer(h, src, n, wl, sign, fl_lo, fl_hi, d_fmt_out, codes, code_type, codes_alt):
    _call("fxpq_qlayer", h.value, C.byref(src), n, wl, sign, fl_lo, fl_hi, ptr(d_fmt_out), ptr(codes),
          code_type, ptr(codes_alt))


def cblock_predicted(h, desc, x, x_type, w, w_colsum, ep, wl, sign, fl_lo, fl_hi, d_fmt_out, y,
                     y_type, d_minmax, d_miss):
    _call("fxpq_cblock_predicted", h.value, C.byref(desc), ptr(x), x_type, ptr(w), ptr(w_colsum),
          C.byref(ep), wl, sign, fl_lo, fl_hi, ptr(d_fmt_out), ptr(y), y_type, ptr(d_minmax),
          ptr(d_miss))


def qlayer_predicted(h, src, n, wl, sign, fl_lo, fl_hi, d_fmt_out, codes, code_type, d_minmax,
                     d_miss):
    _call("fxpq_qlayer_predicted", h.value, C.byref(src), n, wl, sign, fl_lo, fl_hi,
          ptr(d_fmt_out), ptr(codes), code_type, ptr(d_minmax), ptr(d_miss))


def qconv(h, desc, x, x_type, w, w_colsum, ep, acc, d_minmax=None):
    _call("fxpq_qconv", h.value, C.byref(desc), ptr(x), x_type, ptr(w), ptr(w_colsum),
          C.byref(ep) if ep is not None else None, ptr(acc), ptr(d_minmax))


def qconv_wide_workspace(desc, wl_x, sign_x, wl_w, sign_w):
    b = C.c_int64(0)
    _call("fxpq_qconv_wide_workspace", C.byref(desc), wl_x, sign_x, wl_w, sign_w, C.byref(b))
    return b.value


def qconv_wide(h, desc, x, wl_x, sign_x, w, wl_w, sign_w, ep, v, d_scale, workspace, ws_bytes):
    _call("fxpq_qconv_wide", h.value, C.byref(desc), ptr(x), wl_x, sign_x, ptr(w), wl_w, sign_w,
          C.byref(ep), ptr(v), ptr(d_scale), ptr(workspace), ws_bytes)


def acc_overflow(h, acc, n, bits, d_count):
    _call("fxpq_acc_overflow", h.value, ptr(acc), n, bits, ptr(d_count))


def qgemm(h, M, N, K, A, a_type, B, b_colsum, ep, Cout, d_minmax=None):
    _call("fxpq_qgemm", h.value, M, N, K, ptr(A), a_type, ptr(B), ptr(b_colsum),
          C.byref(ep) if ep is not None else None, ptr(Cout), ptr(d_minmax))


def cblock(h, desc, x, x_type, w, w_colsum, ep, wl, sign, fl_lo, fl_hi, d_fmt_out, y, y_type,
           acc, d_minmax):
    _call("fxpq_cblock", h.value, C.byref(desc), ptr(x), x_type, ptr(w), ptr(w_colsum),
          C.byref(ep), wl, sign, fl_lo, fl_hi, ptr(d_fmt_out), ptr(y), y_type, ptr(acc),
          ptr(d_minmax))


def weight_colsum(h, w, k, length, colsum):
    _call("fxpq_weight_colsum", h.value, ptr(w), k, length, ptr(colsum))


def maxpool(h, x, dtype, n, hgt, wid, c, ksize, stride, pad, y):
    _call("fxpq_maxpool", h.value, ptr(x), dtype, n, hgt, wid, c, ksize, stride, pad, ptr(y))


def avgpool_global(h, x, dtype, d_fmt, n, hw, c, recip, y):
    _call("fxpq_avgpool_global", h.value, ptr(x), dtype, ptr(d_fmt), n, hw, c, recip, ptr(y))


def layer_error(h, ref, codes, code_type, d_fmt, n, d_out):
    _call("fxpq_layer_error", h.value, ptr(ref), ptr(codes), code_type, ptr(d_fmt), n, ptr(d_out))


def dequantize(h, codes, code_type, d_fmt, n, out):
    _call("fxpq_dequantize", h.value, ptr(codes), code_type, ptr(d_fmt), n, ptr(out))


def prediction_ties(h, scores, dtype, rows, cols, d_out):
    _call("fxpq_prediction_ties", h.value, ptr(scores), dtype, rows, cols, ptr(d_out))


def epilogue_scale(h, ep, d_scale):
    _call("fxpq_epilogue_scale", h.value, C.byref(ep), ptr(d_scale))


def teacher_conv(h, desc, x, w_rsck, y):
    _call("fxpq_teacher_conv", h.value, C.byref(desc), ptr(x), ptr(w_rsck), ptr(y))


def teacher_affine(h, t, n, channels, y, a1=None, a2=None, bias=None, relu=False):
    _call("fxpq_teacher_affine", h.value, ptr(t), n, channels, ptr(a1), ptr(a2), ptr(bias),
          int(relu), ptr(y))


def teacher_add(h, a, b, n, relu, y):
    _call("fxpq_teacher_add", h.value, ptr(a), ptr(b), n, int(relu), ptr(y))


def teacher_maxpool(h, x, n, hgt, wid, c, ksize, stride, pad, y):
    _call("fxpq_teacher_maxpool", h.value, ptr(x), n, hgt, wid, c, ksize, stride, pad, ptr(y))


def teacher_avgpool(h, x, n, hw, c, y):
    _call("fxpq_teacher_avgpool", h.value, ptr(x), n, hw, c, ptr(y))


def timer_start(h, kind):
    _call("fxpq_timer_start", h.value, kind)


def timer_read(h):
    """(total ms, launches, algorithmic work) of the timed kernel."""
    ms, n, work = C.c_double(), C.c_int64(), C.c_double()
    _call("fxpq_timer_read", h.value, C.byref(ms), C.byref(n), C.byref(work))
    return ms.value, n.value, work.value


# ---- descriptor helpers (plain struct filling) --------------------------------
# A descriptor holds raw device addresses; it also keeps the tensors it points
# to alive for as long as the descriptor itself lives.
def _keep(obj, *refs):
    obj._refs = [r for r in refs if r is not None and not isinstance(r, int)]
    return obj


def src_f32(x, d_minmax=None):
    return _keep(Src(kind=SRC_F32, dtype=F32, x=ptr(x), d_minmax=ptr(d_minmax)), x, d_minmax)


def src_int(x, dtype, d_scale, d_minmax=None):
    return _keep(Src(kind=SRC_INT, dtype=dtype, x=ptr(x), d_scale=ptr(d_scale),
                     d_minmax=ptr(d_minmax)), x, d_scale, d_minmax)


def src_acc(acc, ep, d_minmax=None):
    s = Src(kind=SRC_ACC, dtype=I32, x=ptr(acc), d_minmax=ptr(d_minmax))
    s.ep = C.addressof(ep)
    return _keep(s, acc, ep, d_minmax)


def src_add(a, a_type, d_fmt_a, b, b_type, d_fmt_b, relu, d_minmax=None):
    s = Src(kind=SRC_ADD, dtype=a_type, x=ptr(a), x2=ptr(b), dtype2=b_type, relu=int(relu),
            d_fmt_a=ptr(d_fmt_a), d_fmt_b=ptr(d_fmt_b), d_minmax=ptr(d_minmax))
    return _keep(s, a, b, d_fmt_a, d_fmt_b, d_minmax)


def epilogue(channels, fl_w, d_fmt_in, bias=None, fl_bias=0, relu=False, scale=None, fl_scale=0,
             shift=None, fl_shift=0):
    e = Epilogue(channels=channels, fl_w=fl_w, d_fmt_in=ptr(d_fmt_in), bias=ptr(bias),
                 fl_bias=fl_bias, relu=int(relu), scale=ptr(scale), fl_scale=fl_scale,
                 shift=ptr(shift), fl_shift=fl_shift)
    return _keep(e, d_fmt_in, bias, scale, shift)


def conv_desc(n, h, w, c, k, r, s, stride, pad):
    return ConvDesc(n, h, w, c, k, r, s, stride, pad)

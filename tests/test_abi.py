"""The C-ABI library loads and exports every call include/fxpq.h declares, and
host-side argument checks reject bad calls before touching a device."""
import ctypes as C
import os
import re

import pytest

from conftest import ROOT


def header_symbols():
    text = open(os.path.join(ROOT, "include", "fxpq.h")).read()
    return sorted(set(re.findall(r"^(?:fxpq_status|const char\*)\s+(fxpq_\w+)\(", text, re.M)))


@pytest.fixture(scope="module")
def fx():
    from paper_2203_12091_amd import fxpq
    if not os.path.exists(fxpq.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return fxpq


def test_every_declared_symbol_is_exported(fx):
    syms = header_symbols()
    assert len(syms) >= 15
    L = fx.lib()
    for s in syms:
        assert hasattr(L, s), s
    assert sorted(fx.EXPORTS) == syms


def test_struct_layouts_match_header(fx):
    assert C.sizeof(fx.Fmt) == 16
    assert C.sizeof(fx.Epilogue) == 64
    assert C.sizeof(fx.Src) == 72
    assert C.sizeof(fx.ConvDesc) == 36


def test_status_strings(fx):
    for st in range(7):
        assert fx.status_string(st)
    assert fx.status_string(99) == "unknown status"


def test_null_handle_and_bad_args_rejected_on_host(fx):
    L = fx.lib()
    assert L.fxpq_destroy(None) == fx.ERR_INVALID_ARG
    assert L.fxpq_sync_status(None, None) == fx.ERR_INVALID_ARG
    assert L.fxpq_quantize(None, None, 10, None, None, fx.I8) == fx.ERR_INVALID_ARG
    src = fx.Src(kind=fx.SRC_F32, dtype=fx.F32, x=None)
    assert L.fxpq_fl_search(None, C.byref(src), 10, 8, -1, -8, 15, None, None) == fx.ERR_INVALID_ARG
    # the no-allocation search: the same host checks, before any device call
    fmt = C.c_void_p(16)  # never dereferenced: every call below is rejected first
    assert L.fxpq_fl_search_static(C.byref(src), 10, 8, -1, -8, 15, None, None, None) == fx.ERR_INVALID_ARG
    assert L.fxpq_fl_search_static(C.byref(src), 0, 8, -1, -8, 15, fmt, None, None) == fx.ERR_INVALID_ARG
    assert L.fxpq_fl_search_static(C.byref(src), 10, 33, -1, -8, 15, fmt, None, None) == fx.ERR_INVALID_ARG
    assert L.fxpq_fl_search_static(C.byref(src), 10, 8, 2, -8, 15, fmt, None, None) == fx.ERR_INVALID_ARG
    assert L.fxpq_fl_search_static(C.byref(src), 10, 8, -1, 15, -8, fmt, None, None) == fx.ERR_INVALID_ARG
    assert L.fxpq_fl_search_static(None, 10, 8, -1, -8, 15, fmt, None, None) == fx.ERR_INVALID_ARG
    d = fx.ConvDesc(1, 8, 8, 64, 64, 3, 3, 1, 1)
    assert L.fxpq_qconv(None, C.byref(d), None, fx.I8, None, None, None, None, None) == fx.ERR_INVALID_ARG
    assert L.fxpq_cblock(None, C.byref(d), None, fx.I8, None, None, None, 8, -1, -8, 15, None, None,
                         fx.C8, None, None) == fx.ERR_INVALID_ARG
    h = C.c_void_p()
    # no GPU in this container: creating a handle must fail cleanly
    st = L.fxpq_create(C.byref(h), 0)
    if st == fx.OK:
        pytest.skip("a GPU is visible here")
    assert st == fx.ERR_INVALID_ARG and not h.value


def test_missing_library_fails_loudly(fx, monkeypatch, tmp_path):
    monkeypatch.setattr(fx, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(fx, "_lib", None)
    with pytest.raises(FileNotFoundError):
        fx.lib()


def test_wide_workspace_layout_on_host(fx):
    """Plane counts and workspace bytes of fxpq_qconv_wide (host arithmetic):
    ceil(wl / 8) input planes; balanced base-256 digits for the weights'
    code range (16-bit signed needs 3: 32767 > 127 * 257); 256-byte aligned
    regions for the input planes, weight planes and column sums, plus one
    int32 accumulator tensor per plane pair when the contraction is too deep
    for the fused path."""
    d = fx.ConvDesc(2, 8, 8, 16, 32, 3, 3, 1, 1)

    def want(px, pw):
        # one fused contraction: planes and column sums only
        a = lambda b: (b + 255) // 256 * 256
        n_in, wrow = 2 * 8 * 8 * 16, 9 * 16
        return px * a(n_in) + pw * a(32 * wrow) + a(pw * 32 * 4)

    for (wx, sx, ww, sw), (px, pw) in [((16, 1, 16, 1), (2, 3)), ((16, 1, 15, 1), (2, 2)),
                                       ((8, 1, 8, 1), (1, 1)), ((8, 0, 8, 0), (1, 2)),
                                       ((32, 1, 32, 1), (4, 5)), ((31, 0, 24, 1), (4, 4)),
                                       ((1, 1, 1, 1), (1, 1)), ((9, 1, 17, 1), (2, 3)),
                                       ((32, 0, 8, 1), (4, 1)), ((8, 1, 32, 0), (1, 5))]:
        assert fx.qconv_wide_workspace(d, wx, sx, ww, sw) == want(px, pw), (wx, sx, ww, sw)
    # the padded RGB layout rounds each weight row up to 64 bytes
    d4 = fx.ConvDesc(1, 10, 10, 4, 64, 7, 7, 2, 3)
    ho = (10 + 6 - 7) // 2 + 1
    a = lambda b: (b + 255) // 256 * 256
    assert fx.qconv_wide_workspace(d4, 16, 1, 8, 1) == 2 * a(400) + a(64 * 256) + a(64 * 4)
    # a contraction too deep for the fused path's int32 group sums (pairs of
    # one shift * padded depth * 2^14 must stay below 2^31): one int32
    # accumulator tensor per plane pair as well
    dd = fx.ConvDesc(1, 2, 2, 8192, 16, 3, 3, 1, 1)
    depth = 9 * 8192
    assert fx.qconv_wide_workspace(dd, 16, 1, 16, 1) == (
        2 * a(4 * 8192) + 3 * a(16 * depth) + a(3 * 16 * 4) + 2 * 3 * 4 * 16 * 4)
    for bad in [(0, 1, 8, 1), (8, 2, 8, 1), (33, 1, 8, 1), (8, 1, 33, 0), (32, -1, 8, 1)]:
        with pytest.raises(fx.FxpqError):
            fx.qconv_wide_workspace(d, *bad)

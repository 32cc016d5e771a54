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

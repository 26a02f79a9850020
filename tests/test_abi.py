"""The C-ABI library: it loads, exports what include/spdp.h declares, and
rejects bad arguments with the documented status (host-side checks only;
nothing here launches a kernel)."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2607_21985_amd as spdp
from conftest import ROOT

ERR_INVALID, ERR_UNSUPPORTED = -1, -2


def _declared():
    with open(os.path.join(ROOT, "include", "spdp.h")) as fh:
        text = fh.read()
    return sorted(set(re.findall(r"\b(spdp_[a-z_]+)\s*\(", text)))


def test_header_declares_what_binding_expects():
    assert _declared() == sorted(spdp.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol():
    L = ctypes.CDLL(spdp.lib_path())
    for name in _declared():
        assert hasattr(L, name), name


def test_strerror_and_last_error():
    L = spdp.lib()
    for st, text in [(0, b"success"), (-1, b"invalid argument"), (-2, b"unsupported"),
                     (-3, b"out of memory"), (-4, b"HIP runtime error"), (7, b"unknown status")]:
        assert L.spdp_strerror(st) == text
    with pytest.raises(spdp.SpdpError) as ei:
        spdp.threshold_code(float("nan"))
    assert ei.value.status == ERR_INVALID
    assert b"NaN" in L.spdp_last_error()


@pytest.mark.parametrize("tm,tk,status", [
    (32, 16, ERR_INVALID), (100, 16, ERR_INVALID), (0, 1, ERR_INVALID), (64, 0, ERR_INVALID),
    (64, 3, ERR_INVALID), (64, 512, ERR_INVALID), (512, 16, ERR_UNSUPPORTED),
    (1024, 16, ERR_UNSUPPORTED), (1088, 16, ERR_INVALID),
])
def test_encode_rejects_bad_tiles(tm, tk, status):
    w = np.ones((8, 8), dtype=np.float16)
    for fn in (spdp.encode_host,):
        with pytest.raises(spdp.SpdpError) as ei:
            fn(w, (tm, tk))
        assert ei.value.status == status


def test_null_and_size_errors():
    L = spdp.lib()
    h = ctypes.c_void_p()
    w = np.ones((4, 4), dtype=np.uint16)
    assert L.spdp_encode_host(None, 4, 4, 64, 16, ctypes.byref(h)) == ERR_INVALID and not h.value
    assert L.spdp_encode_host(ctypes.c_void_p(w.ctypes.data), 0, 4, 64, 16, ctypes.byref(h)) == ERR_INVALID
    assert L.spdp_encode_host(ctypes.c_void_p(w.ctypes.data), 4, -1, 64, 16, ctypes.byref(h)) == ERR_INVALID
    assert L.spdp_encode_host(ctypes.c_void_p(w.ctypes.data), 4, 4, 64, 16, None) == ERR_INVALID
    assert L.spdp_encode(None, 4, 4, 64, 16, ctypes.byref(h)) == ERR_INVALID and not h.value
    assert L.spdp_format(None, None) == ERR_INVALID
    assert L.spdp_reserve(None, 1) == ERR_INVALID
    assert L.spdp_spmspv(None, None, 1, ctypes.c_float(0.0), None, None) == ERR_INVALID
    assert L.spdp_spmspv_noalloc(None, None, 1, ctypes.c_float(0.0), None, None) == ERR_INVALID
    assert L.spdp_spmm(None, None, 1, None, None) == ERR_INVALID
    L.spdp_free(None)  # no-op
    out = np.empty(16, dtype=np.uint16)
    assert L.spdp_prune_magnitude(None, 16, ctypes.c_double(0.5), ctypes.c_void_p(out.ctypes.data)) == ERR_INVALID
    t = ctypes.c_float()
    assert L.spdp_calibrate_threshold(None, 4, ctypes.c_double(0.5), ctypes.byref(t)) == ERR_INVALID
    assert L.spdp_threshold_code(ctypes.c_float(1.0), None) == ERR_INVALID


def test_spmspv_on_host_only_handle_is_rejected():
    m = spdp.encode_host(np.ones((64, 16), dtype=np.float16), (64, 16))
    L = spdp.lib()
    x = np.zeros(64, dtype=np.uint16)
    st = L.spdp_spmspv(m._h, ctypes.c_void_p(x.ctypes.data), 1, ctypes.c_float(0.0),
                       ctypes.c_void_p(x.ctypes.data + 64), None)
    assert st == ERR_INVALID
    assert b"device" in L.spdp_last_error()
    st = L.spdp_spmspv_noalloc(m._h, ctypes.c_void_p(x.ctypes.data), 1, ctypes.c_float(0.0),
                               ctypes.c_void_p(x.ctypes.data + 64), None)
    assert st == ERR_INVALID
    st = L.spdp_spmm(m._h, ctypes.c_void_p(x.ctypes.data), 1, ctypes.c_void_p(x.ctypes.data + 64), None)
    assert st == ERR_INVALID
    assert b"device" in L.spdp_last_error()
    assert L.spdp_reserve(m._h, 4) == ERR_INVALID
    m.close()


def test_rtn_encode_argument_errors():
    w = np.ones((64, 16), dtype=np.float16)
    for bits in (0, 1, 9, 16):
        with pytest.raises(spdp.SpdpError) as e:
            spdp.encode_rtn_host(w, (64, 16), bits)
        assert e.value.status == ERR_INVALID and "bits" in str(e.value)
    w[3, 4] = np.inf
    with pytest.raises(spdp.SpdpError) as e:
        spdp.encode_rtn_host(w, (64, 16), 4)
    assert e.value.status == ERR_INVALID and "finite" in str(e.value)
    w[3, 4] = np.nan
    with pytest.raises(spdp.SpdpError):
        spdp.encode_rtn_host(w, (64, 16), 4)
    with pytest.raises(spdp.SpdpError) as e:
        spdp.encode_rtn_host(np.ones((64, 16), dtype=np.float16), (100, 16), 4)
    assert e.value.status == ERR_INVALID
    # a host-only code handle cannot run a product
    m = spdp.encode_rtn_host(np.ones((64, 16), dtype=np.float16), (64, 16), 4)
    L = spdp.lib()
    x = np.zeros(64, dtype=np.uint16)
    st = L.spdp_spmspv(m._h, ctypes.c_void_p(x.ctypes.data), 1, ctypes.c_float(0.0),
                       ctypes.c_void_p(x.ctypes.data + 64), None)
    assert st == ERR_INVALID
    f = m.format()
    assert f["value_bits"] == 4 and f["codes"].dtype == np.int8 and np.all(f["scales"] == np.float32(1.0 / 7.0))
    m.close()


def test_prune_and_calibrate_argument_errors():
    w = np.ones(10, dtype=np.float16)
    for bad in (-0.1, 1.5, float("nan")):
        with pytest.raises(spdp.SpdpError):
            spdp.prune_magnitude(w, bad)
        with pytest.raises(spdp.SpdpError):
            spdp.calibrate_threshold(w, bad)
    nanw = np.array([1.0, np.nan], dtype=np.float16)
    with pytest.raises(spdp.SpdpError):
        spdp.prune_magnitude(nanw, 0.5)
    with pytest.raises(spdp.SpdpError):
        spdp.calibrate_threshold(nanw, 0.5)


def test_format_view_fields():
    w = np.zeros((130, 37), dtype=np.float16)
    w[5, 3] = 1
    m = spdp.encode_host(w, (64, 4))
    f = m.format()
    assert (f["rows"], f["cols"], f["tile_m"], f["tile_k"]) == (130, 37, 64, 4)
    assert (f["n_stripes"], f["n_colblocks"], f["n_gtiles"]) == (3, 10, 30)
    assert f["tile_offset"].size == 31 and f["col_info"].size == 120 and f["bitmap"].size == 120
    assert m.device == -1
    assert all(v is None for v in m.device_pointers().values())


def test_spmspv_many_argument_errors():
    """Host-side checks of the grouped call (no device needed)."""
    L = spdp.lib()
    a = spdp.encode_host(np.ones((64, 16), dtype=np.float16), (64, 16))
    b = spdp.encode_host(np.ones((64, 16), dtype=np.float16), (64, 16))
    x = np.zeros(256, dtype=np.uint16)
    H = ctypes.c_void_p
    P = ctypes.c_void_p
    xs = (P * 2)(x.ctypes.data, x.ctypes.data)
    ys = (P * 2)(x.ctypes.data + 128, x.ctypes.data + 256)
    ts = (ctypes.c_float * 2)(0.0, 0.0)
    hs = (H * 2)(a._h.value, b._h.value)
    assert L.spdp_spmspv_many(None, 1, xs, 1, ts, ys, None) == ERR_INVALID
    assert L.spdp_spmspv_many(hs, 1, None, 1, ts, ys, None) == ERR_INVALID
    assert L.spdp_spmspv_many(hs, 1, xs, 1, None, ys, None) == ERR_INVALID
    for count in (0, 9, -1):
        assert L.spdp_spmspv_many(hs, count, xs, 1, ts, ys, None) == ERR_INVALID
    assert L.spdp_spmspv_many(hs, 2, xs, 0, ts, ys, None) == ERR_INVALID
    assert L.spdp_spmspv_many(hs, 2, xs, 33, ts, ys, None) == ERR_INVALID
    nul = (H * 2)(None, a._h.value)
    assert L.spdp_spmspv_many(nul, 2, xs, 1, ts, ys, None) == ERR_INVALID
    assert b"NULL" in L.spdp_last_error()
    # host-only handles are rejected before any device work
    assert L.spdp_spmspv_many(hs, 2, xs, 1, ts, ys, None) == ERR_INVALID
    assert b"device" in L.spdp_last_error()
    # the mask choice: only the two declared values
    for mask in (-1, 2, 7):
        assert L.spdp_spmspv_many_mask(hs, 2, xs, 1, ts, mask, ys, None) == ERR_INVALID
        assert b"mask" in L.spdp_last_error()
    for mask in (0, 1):  # valid masks reach the same device check
        assert L.spdp_spmspv_many_mask(hs, 2, xs, 1, ts, mask, ys, None) == ERR_INVALID
        assert b"device" in L.spdp_last_error()
    with pytest.raises(ValueError):
        spdp._mask_code("mean")
    a.close()
    b.close()


def test_chain_host_side_errors():
    """Chain: nothing to capture, replay before capture, a bad mask name."""
    ch = spdp.Chain()
    with pytest.raises(RuntimeError):
        ch.replay()
    with pytest.raises(RuntimeError):
        ch.capture()
    m = spdp.encode_host(np.ones((64, 16), dtype=np.float16), (64, 16))
    with pytest.raises(ValueError):
        ch.add(m, None, 0.5, None, mask="rows")
    m.close()

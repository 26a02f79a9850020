"""Python binding of libspdp: the MI355X Tiled-CBC spMspV library.

Argument marshalling only. Every step of the decode path (activity test,
column selection, bitmap decode, accumulation, split-K reduction) runs in
the HIP kernel behind ``spdp_spmspv``; the encoder, pruning and threshold
calibration run in the library's host C++. PyTorch supplies device memory
and streams. There is no fallback: if ``libspdp.so`` is not built, every
entry point raises.

    import paper_2607_21985_amd as spdp
    w_sp = spdp.prune_magnitude(w16, 0.5)          # numpy fp16, host
    m = spdp.encode(w_sp, tile=(256, 16))          # device copy on cuda:current
    t = spdp.calibrate_threshold(x16_calib, 0.5)   # TEAL-style quantile
    y = m(x_cuda_fp16, t)                          # torch fp16 [batch, rows]
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

__all__ = [
    "SpdpError",
    "Matrix",
    "lib",
    "lib_path",
    "encode",
    "encode_host",
    "encode_rtn",
    "encode_rtn_host",
    "spmspv_many",
    "MASKS",
    "Chain",
    "prune_magnitude",
    "calibrate_threshold",
    "threshold_code",
    "EXPORTED_SYMBOLS",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libspdp.so"

EXPORTED_SYMBOLS = (
    "spdp_encode", "spdp_encode_host", "spdp_spmspv", "spdp_spmspv_many", "spdp_spmspv_many_mask",
    "spdp_reserve", "spdp_split_plan", "spdp_free",
    "spdp_format", "spdp_prune_magnitude", "spdp_calibrate_threshold",
    "spdp_threshold_code", "spdp_strerror", "spdp_last_error",
    "spdp_encode_rtn", "spdp_encode_rtn_host", "spdp_spmspv_noalloc", "spdp_spmm",
)

SPDP_OK = 0
_STATUS = {0: "SPDP_OK", -1: "SPDP_ERR_INVALID_ARG", -2: "SPDP_ERR_UNSUPPORTED",
           -3: "SPDP_ERR_OOM", -4: "SPDP_ERR_HIP"}


class SpdpError(RuntimeError):
    """A libspdp call returned an error status."""

    def __init__(self, status: int, detail: str):
        super().__init__(f"{_STATUS.get(status, status)}: {detail}")
        self.status = status


class _Format(ctypes.Structure):
    _fields_ = [
        ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
        ("tile_m", ctypes.c_int32), ("tile_k", ctypes.c_int32),
        ("n_stripes", ctypes.c_int64), ("n_colblocks", ctypes.c_int64),
        ("n_gtiles", ctypes.c_int64), ("n_values", ctypes.c_int64),
        ("tile_offset", ctypes.POINTER(ctypes.c_uint32)),
        ("col_info", ctypes.POINTER(ctypes.c_uint32)),
        ("bitmap", ctypes.POINTER(ctypes.c_uint64)),
        ("values", ctypes.POINTER(ctypes.c_uint16)),
        ("d_tile_offset", ctypes.c_void_p), ("d_col_info", ctypes.c_void_p),
        ("d_bitmap", ctypes.c_void_p), ("d_values", ctypes.c_void_p),
        ("device", ctypes.c_int32),
        ("value_bits", ctypes.c_int32),
        ("codes", ctypes.POINTER(ctypes.c_int8)),
        ("scales", ctypes.POINTER(ctypes.c_float)),
        ("d_scales", ctypes.c_void_p),
    ]


_lib = None


def lib_path() -> str:
    return os.path.join(_HERE, _LIB_NAME)


def lib() -> ctypes.CDLL:
    """Load libspdp.so (built in-tree by ``build.py``); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    path = lib_path()
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2607_21985_amd.build`")
    L = ctypes.CDLL(path)
    u16p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    H = ctypes.c_void_p
    L.spdp_encode.argtypes = [u16p, i64, i64, i32, i32, ctypes.POINTER(H)]
    L.spdp_encode_host.argtypes = [u16p, i64, i64, i32, i32, ctypes.POINTER(H)]
    L.spdp_encode_rtn.argtypes = [u16p, i64, i64, i32, i32, i32, ctypes.POINTER(H)]
    L.spdp_encode_rtn_host.argtypes = [u16p, i64, i64, i32, i32, i32, ctypes.POINTER(H)]
    L.spdp_spmspv.argtypes = [H, ctypes.c_void_p, i32, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p]
    L.spdp_spmspv_noalloc.argtypes = [H, ctypes.c_void_p, i32, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p]
    L.spdp_spmm.argtypes = [H, ctypes.c_void_p, i64, ctypes.c_void_p, ctypes.c_void_p]
    L.spdp_spmspv_many.argtypes = [ctypes.POINTER(H), i32, ctypes.POINTER(ctypes.c_void_p), i32,
                                   ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_void_p),
                                   ctypes.c_void_p]
    L.spdp_spmspv_many_mask.argtypes = [ctypes.POINTER(H), i32, ctypes.POINTER(ctypes.c_void_p), i32,
                                        ctypes.POINTER(ctypes.c_float), i32, ctypes.POINTER(ctypes.c_void_p),
                                        ctypes.c_void_p]
    L.spdp_reserve.argtypes = [H, i32]
    L.spdp_split_plan.argtypes = [H, i32, ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i32)]
    L.spdp_free.argtypes = [H]
    L.spdp_free.restype = None
    L.spdp_format.argtypes = [H, ctypes.POINTER(_Format)]
    L.spdp_prune_magnitude.argtypes = [u16p, i64, ctypes.c_double, u16p]
    L.spdp_calibrate_threshold.argtypes = [u16p, i64, ctypes.c_double, ctypes.POINTER(ctypes.c_float)]
    L.spdp_threshold_code.argtypes = [ctypes.c_float, ctypes.POINTER(i32)]
    L.spdp_strerror.argtypes = [ctypes.c_int]
    L.spdp_strerror.restype = ctypes.c_char_p
    L.spdp_last_error.argtypes = []
    L.spdp_last_error.restype = ctypes.c_char_p
    for name in ("spdp_encode", "spdp_encode_host", "spdp_spmspv", "spdp_spmspv_noalloc", "spdp_spmm",
                 "spdp_spmspv_many",
                 "spdp_spmspv_many_mask",
                 "spdp_reserve", "spdp_split_plan",
                 "spdp_format",
                 "spdp_prune_magnitude", "spdp_calibrate_threshold", "spdp_threshold_code"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int) -> None:
    if status != SPDP_OK:
        raise SpdpError(status, lib().spdp_last_error().decode())


def _u16(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype == np.float16:
        return a.view(np.uint16)
    if a.dtype == np.uint16:
        return a
    raise TypeError(f"expected fp16 (or its uint16 bits), got {a.dtype}")


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data)


class Matrix:
    """An encoded weight matrix (owns the library handle)."""

    def __init__(self, handle: ctypes.c_void_p):
        self._h = handle
        f = _Format()
        _check(lib().spdp_format(self._h, ctypes.byref(f)))
        self.rows, self.cols = int(f.rows), int(f.cols)
        self.tile = (int(f.tile_m), int(f.tile_k))
        self.device = int(f.device)

    def _fmt(self) -> _Format:
        f = _Format()
        _check(lib().spdp_format(self._h, ctypes.byref(f)))
        return f

    def format(self) -> dict:
        """Copies of the four Tiled-CBC arrays (host) plus shape fields."""
        f = self._fmt()
        ngt, tk, tm = int(f.n_gtiles), int(f.tile_k), int(f.tile_m)

        def arr(p, n, dt):
            if n == 0:
                return np.zeros(0, dtype=dt)
            return np.ctypeslib.as_array(p, shape=(n,)).astype(dt, copy=True)

        out = {
            "rows": int(f.rows), "cols": int(f.cols), "tile_m": tm, "tile_k": tk,
            "n_stripes": int(f.n_stripes), "n_colblocks": int(f.n_colblocks), "n_gtiles": ngt,
            "tile_offset": arr(f.tile_offset, ngt + 1, np.uint32),
            "col_info": arr(f.col_info, ngt * tk, np.uint32),
            "bitmap": arr(f.bitmap, ngt * tk * tm // 64, np.uint64),
            "value_bits": int(f.value_bits),
        }
        if f.value_bits < 16:
            # one byte per code; "values" holds the codes' bytes
            out["codes"] = arr(f.codes, int(f.n_values), np.int8)
            out["values"] = out["codes"].view(np.uint8)
            out["scales"] = arr(f.scales, int(f.rows), np.float32)
        else:
            out["values"] = arr(f.values, int(f.n_values), np.uint16)
        return out

    def device_pointers(self) -> dict:
        f = self._fmt()
        return {"tile_offset": f.d_tile_offset, "col_info": f.d_col_info,
                "bitmap": f.d_bitmap, "values": f.d_values}

    def reserve(self, max_batch: int) -> None:
        _check(lib().spdp_reserve(self._h, int(max_batch)))

    def split_plan(self, batch: int) -> tuple:
        """(segments, wave_cols, passes) of a call with ``batch`` tokens (``spdp_split_plan``)."""
        sg, wc, ps = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(lib().spdp_split_plan(self._h, int(batch), ctypes.byref(sg), ctypes.byref(wc), ctypes.byref(ps)))
        return sg.value, wc.value, ps.value

    def spmspv_into(self, x, threshold: float, y, stream=None, mask: str = "token") -> None:
        """Enqueue ``y = W_sp . mask(x)`` on ``stream`` (torch stream, or the current one).

        ``mask``: "token" (each token's own columns) or "batch" (one column
        set for the batch, by its fp32 sum of magnitudes; see
        ``spmspv_many``)."""
        import torch
        if x.dtype != torch.float16 or y.dtype != torch.float16:
            raise TypeError("x and y must be torch.float16")
        if x.dim() != 2 or x.shape[1] != self.cols or not x.is_contiguous():
            raise ValueError(f"x must be a contiguous [batch, {self.cols}] tensor")
        b = x.shape[0]
        if tuple(y.shape) != (b, self.rows) or not y.is_contiguous():
            raise ValueError(f"y must be a contiguous [{b}, {self.rows}] tensor")
        if not (x.is_cuda and y.is_cuda):
            raise ValueError("x and y must be device tensors")
        s = stream if stream is not None else torch.cuda.current_stream(x.device)
        if mask == "token":
            _check(lib().spdp_spmspv(self._h, ctypes.c_void_p(x.data_ptr()), int(b),
                                     ctypes.c_float(threshold), ctypes.c_void_p(y.data_ptr()),
                                     ctypes.c_void_p(s.cuda_stream)))
        else:
            hs = (ctypes.c_void_p * 1)(self._h)
            xp = (ctypes.c_void_p * 1)(x.data_ptr())
            yp = (ctypes.c_void_p * 1)(y.data_ptr())
            ts = (ctypes.c_float * 1)(float(threshold))
            _check(lib().spdp_spmspv_many_mask(hs, 1, xp, int(b), ts, _mask_code(mask), yp,
                                               ctypes.c_void_p(s.cuda_stream)))

    def spmspv_noalloc_into(self, x, threshold: float, y, stream=None) -> None:
        """``spmspv_into`` through ``spdp_spmspv_noalloc``: the split-K partials
        go to the library's static workspace, so the call allocates nothing
        (per-token mask; calls on one GPU must not overlap)."""
        import torch
        if x.dtype != torch.float16 or y.dtype != torch.float16:
            raise TypeError("x and y must be torch.float16")
        if x.dim() != 2 or x.shape[1] != self.cols or not x.is_contiguous():
            raise ValueError(f"x must be a contiguous [batch, {self.cols}] tensor")
        b = x.shape[0]
        if tuple(y.shape) != (b, self.rows) or not y.is_contiguous():
            raise ValueError(f"y must be a contiguous [{b}, {self.rows}] tensor")
        if not (x.is_cuda and y.is_cuda):
            raise ValueError("x and y must be device tensors")
        s = stream if stream is not None else torch.cuda.current_stream(x.device)
        _check(lib().spdp_spmspv_noalloc(self._h, ctypes.c_void_p(x.data_ptr()), int(b),
                                         ctypes.c_float(threshold), ctypes.c_void_p(y.data_ptr()),
                                         ctypes.c_void_p(s.cuda_stream)))

    def spmm_into(self, x, y, stream=None) -> None:
        """Enqueue the prefill product ``y = x W_sp^T`` (every column, no
        threshold) for ``x`` [tokens, cols] into ``y`` [tokens, rows]."""
        import torch
        if x.dtype != torch.float16 or y.dtype != torch.float16:
            raise TypeError("x and y must be torch.float16")
        if x.dim() != 2 or x.shape[1] != self.cols or not x.is_contiguous():
            raise ValueError(f"x must be a contiguous [tokens, {self.cols}] tensor")
        n = x.shape[0]
        if tuple(y.shape) != (n, self.rows) or not y.is_contiguous():
            raise ValueError(f"y must be a contiguous [{n}, {self.rows}] tensor")
        if not (x.is_cuda and y.is_cuda):
            raise ValueError("x and y must be device tensors")
        s = stream if stream is not None else torch.cuda.current_stream(x.device)
        _check(lib().spdp_spmm(self._h, ctypes.c_void_p(x.data_ptr()), int(n), ctypes.c_void_p(y.data_ptr()),
                               ctypes.c_void_p(s.cuda_stream)))

    def spmm(self, x, stream=None):
        """The prefill product ``x W_sp^T`` as a new fp16 tensor."""
        import torch
        y = torch.empty((x.shape[0], self.rows), dtype=torch.float16, device=x.device)
        self.spmm_into(x, y, stream)
        return y

    def __call__(self, x, threshold: float, stream=None, mask: str = "token"):
        import torch
        y = torch.empty((x.shape[0], self.rows), dtype=torch.float16, device=x.device)
        self.spmspv_into(x, threshold, y, stream, mask)
        return y

    def close(self) -> None:
        """Free the handle (synchronizes the device; never while a stream capture runs)."""
        if getattr(self, "_h", None):
            lib().spdp_free(self._h)
            self._h = None
        _free_deferred()

    def __del__(self):
        # spdp_free synchronizes the device, which would invalidate a HIP
        # graph capture in progress: a handle that becomes garbage during a
        # capture is freed at the next close() or encode() instead.
        try:
            h = getattr(self, "_h", None)
            if not h:
                return
            self._h = None
            if _capturing():
                _DEFERRED.append(h)
            else:
                lib().spdp_free(h)
        except Exception:
            pass


_DEFERRED: list = []


def _capturing() -> bool:
    try:
        import torch
        return bool(torch.cuda.is_available() and torch.cuda.is_current_stream_capturing())
    except Exception:
        return False


def _free_deferred() -> None:
    while _DEFERRED and not _capturing():
        lib().spdp_free(_DEFERRED.pop())


def encode(w: np.ndarray, tile=(256, 16)) -> Matrix:
    """Encode a pruned fp16 matrix (host numpy) and upload it to the current HIP device."""
    wb = _u16(w)
    if wb.ndim != 2:
        raise ValueError("w must be 2-D")
    _free_deferred()
    h = ctypes.c_void_p()
    _check(lib().spdp_encode(_ptr(wb), wb.shape[0], wb.shape[1], int(tile[0]), int(tile[1]),
                             ctypes.byref(h)))
    return Matrix(h)


MASKS = {"token": 0, "batch": 1}  # SPDP_MASK_TOKEN, SPDP_MASK_BATCH


def _mask_code(mask: str) -> int:
    if mask not in MASKS:
        raise ValueError(f"mask must be one of {sorted(MASKS)}")
    return MASKS[mask]


def spmspv_many(mats, xs, thresholds, ys, stream=None, mask: str = "token") -> None:
    """Enqueue ``ys[i] = W_i . mask(xs[i])`` for every i in one launch.

    ``mats`` are encoded matrices with one tile height, ``xs``/``ys`` torch
    fp16 device tensors ``[batch, cols_i]`` / ``[batch, rows_i]`` (one batch
    for all), ``thresholds`` one float per product. Inputs may be shared.
    ``mask="token"``: column k takes part for token b iff |x[b, k]| > t;
    ``mask="batch"``: one column set for the batch, column k taking part for
    every token iff the fp32 running sum of |x[b, k]| over the tokens exceeds
    fp32(batch * t) (the batch's mean magnitude exceeds t).
    """
    import torch
    n = len(mats)
    if not (len(xs) == len(ys) == len(thresholds) == n):
        raise ValueError("mats, xs, thresholds and ys must have one entry per product")
    for m, x, y in zip(mats, xs, ys):
        if x.dtype != torch.float16 or y.dtype != torch.float16:
            raise TypeError("x and y must be torch.float16")
        if x.dim() != 2 or x.shape[1] != m.cols or not x.is_contiguous():
            raise ValueError(f"x must be a contiguous [batch, {m.cols}] tensor")
        if tuple(y.shape) != (x.shape[0], m.rows) or not y.is_contiguous():
            raise ValueError(f"y must be a contiguous [{x.shape[0]}, {m.rows}] tensor")
        if x.shape[0] != xs[0].shape[0]:
            raise ValueError("every product of one call takes the same batch")
        if not (x.is_cuda and y.is_cuda):
            raise ValueError("x and y must be device tensors")
    s = stream if stream is not None else torch.cuda.current_stream(xs[0].device)
    hs = (ctypes.c_void_p * n)(*[m._h for m in mats])
    xp = (ctypes.c_void_p * n)(*[x.data_ptr() for x in xs])
    yp = (ctypes.c_void_p * n)(*[y.data_ptr() for y in ys])
    ts = (ctypes.c_float * n)(*[float(t) for t in thresholds])
    _check(lib().spdp_spmspv_many_mask(hs, n, xp, int(xs[0].shape[0]), ts, _mask_code(mask), yp,
                                       ctypes.c_void_p(s.cuda_stream)))


def encode_rtn(w: np.ndarray, tile=(256, 16), bits: int = 4) -> Matrix:
    """Quantize a pruned fp16 matrix to ``bits``-bit round-to-nearest codes
    (one scale per row), encode it with one byte per code and upload it."""
    wb = _u16(w)
    if wb.ndim != 2:
        raise ValueError("w must be 2-D")
    _free_deferred()
    h = ctypes.c_void_p()
    _check(lib().spdp_encode_rtn(_ptr(wb), wb.shape[0], wb.shape[1], int(tile[0]), int(tile[1]),
                                 int(bits), ctypes.byref(h)))
    return Matrix(h)


def encode_rtn_host(w: np.ndarray, tile=(256, 16), bits: int = 4) -> Matrix:
    """``encode_rtn`` without touching any device."""
    wb = _u16(w)
    if wb.ndim != 2:
        raise ValueError("w must be 2-D")
    h = ctypes.c_void_p()
    _check(lib().spdp_encode_rtn_host(_ptr(wb), wb.shape[0], wb.shape[1], int(tile[0]), int(tile[1]),
                                      int(bits), ctypes.byref(h)))
    return Matrix(h)


def encode_host(w: np.ndarray, tile=(256, 16)) -> Matrix:
    """Encode without touching any device (inspection, CPU-only machines)."""
    wb = _u16(w)
    if wb.ndim != 2:
        raise ValueError("w must be 2-D")
    h = ctypes.c_void_p()
    _check(lib().spdp_encode_host(_ptr(wb), wb.shape[0], wb.shape[1], int(tile[0]),
                                  int(tile[1]), ctypes.byref(h)))
    return Matrix(h)


def prune_magnitude(w: np.ndarray, sparsity: float) -> np.ndarray:
    """Global magnitude pruning (host C++); returns a new fp16 array."""
    wb = _u16(w)
    out = np.empty_like(wb)
    _check(lib().spdp_prune_magnitude(_ptr(wb), wb.size, float(sparsity), _ptr(out)))
    return out.view(np.float16)


def calibrate_threshold(x: np.ndarray, p: float) -> float:
    """Threshold that drops a fraction p of |x| under the strict rule |x| > t."""
    xb = _u16(x)
    t = ctypes.c_float()
    _check(lib().spdp_calibrate_threshold(_ptr(xb), xb.size, float(p), ctypes.byref(t)))
    return float(t.value)


def threshold_code(t: float) -> int:
    """Integer magnitude bound the kernels compare fp16 bits against."""
    c = ctypes.c_int32()
    _check(lib().spdp_threshold_code(ctypes.c_float(t), ctypes.byref(c)))
    return int(c.value)


class Chain:
    """A decoder layer's projections issued as one HIP graph.

    ``add`` records one launch: a list of products that read one input
    (q, k and v; gate and up) goes out as one grouped launch, a single
    product as a plain call. ``capture`` sizes every matrix's workspace for
    the batches recorded, issues the launches once eagerly and records them
    into a graph on a side stream; ``replay`` re-issues the whole chain on
    the current stream with one host call. Between replays the caller
    rewrites the input tensors in place (and the thresholds are fixed at
    capture); the calls keep no host-side state, so every replay computes on
    the tensors' current contents.
    """

    def __init__(self):
        self._calls = []
        self._graph = None

    def add(self, mats, xs, thresholds, ys, mask: str = "token") -> "Chain":
        if self._graph is not None:
            raise RuntimeError("the chain is captured already")
        if isinstance(mats, Matrix):
            mats, xs, thresholds, ys = [mats], [xs], [thresholds], [ys]
        _mask_code(mask)
        self._calls.append((list(mats), list(xs), [float(t) for t in thresholds], list(ys), mask))
        return self

    def _issue(self):
        for mats, xs, ts, ys, mask in self._calls:
            if len(mats) == 1:
                mats[0].spmspv_into(xs[0], ts[0], ys[0], mask=mask)
            else:
                spmspv_many(mats, xs, ts, ys, mask=mask)

    def capture(self) -> "Chain":
        import torch
        if not self._calls:
            raise RuntimeError("nothing to capture")
        for mats, xs, _, _, _ in self._calls:
            for m, x in zip(mats, xs):
                m.reserve(int(x.shape[0]))
        dev = self._calls[0][1][0].device
        self._issue()  # eager once: every workspace and phase in place
        torch.cuda.synchronize(dev)
        s = torch.cuda.Stream(device=dev)
        s.wait_stream(torch.cuda.current_stream(dev))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            self._issue()
        torch.cuda.current_stream(dev).wait_stream(s)
        self._graph = g
        return self

    def replay(self) -> None:
        if self._graph is None:
            raise RuntimeError("capture() first")
        self._graph.replay()

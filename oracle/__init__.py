"""CPU oracle for the Tiled-CBC spMspV path -- TEST INFRASTRUCTURE ONLY.

This package is the slow, plain, obviously-correct statement of what the
decode hot path of SPDP computes. It exists to check the HIP library, never
to stand in for it: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it. It shares no code with
the library (no common headers, helpers, tables or generators) and never
imports it.

Everything here is NumPy on the CPU. Floating point is float64 from the fp16
inputs (every fp16 x fp16 product is exact in float64); integer/bit work is
done on the raw fp16 bit patterns (``uint16``).

Functions and the passages of the paper they follow:

* ``magnitude_prune``   -- static pruning ``W_sp = W * M`` (Sec. 2.2, the SP
  definition) with magnitude as the criterion (Sec. 2.2 / 3.2, global over
  the matrix).
* ``threshold_for``     -- a TEAL-style threshold: the p-quantile of the
  empirical distribution of |x| (Sec. 5.1, ECDF quantile calibration).
* ``active_mask`` / ``masked_activations`` -- dynamic pruning: a column k is
  kept for a token iff |x_k| exceeds the threshold (Sec. 2.2 DP definition,
  Sec. 4.2 step (3)); or, batched DP (future work in Sec. 4.3 and Sec. 7,
  read here as one column set shared by the batch), kept for every token
  iff the batch's fp32 score ``batch_score`` exceeds ``batch_threshold``.
* ``encode`` / ``decode`` -- the Tiled-CBC format (Sec. 4.1, Tiling Design
  and Storage Structure; 16-byte column padding from Sec. 4.2.3).
* ``spmspv`` / ``spmspv_rows`` -- the masked product
  ``y = W_sp . mask(x)`` (Sec. 2.2 SP and DP definitions combined; Sec. 4.2
  says inactive columns contribute nothing).
* ``spmm`` / ``spmm_flops`` -- the prefill product ``Y = X W_sp^T`` for N
  tokens (Sec. 4.3: prefill keeps static pruning and drops dynamic pruning)
  and its useful and dense flop counts.
* ``storage_bytes`` -- the Tiled-CBC storage formula (Sec. 4.1).
* ``compression_ratio``, ``compute_intensity``, ``compute_intensity_spdp``,
  ``attainable``, ``combined_sparsity`` -- Eq. 1, Eq. 2, the roofline, Eq. 3
  and the combined-sparsity arithmetic of Sec. 3.
* ``algorithmic_bytes`` / ``useful_flops`` -- the bytes a call must move
  (active-column metadata + values + touched TileOffset entries + x + y)
  and the multiply-adds it must do.
* ``rtn_quantize`` / ``encode_codes`` / ``decode_codes`` / ``spmspv_rtn``
  -- low-bit Values: round-to-nearest weight-only quantization of the pruned
  matrix (Sec. 5.1's quantization setup: pruning first, then quantization,
  then dynamic pruning at inference), the same format with one byte per
  code (Sec. 6: Values are stored apart from the sparsity metadata), and
  the masked product with the dequantized weights.

Readings where the paper is silent (bit order, array order, padding value,
ColInfo offset unit, zero test, ragged shapes, threshold tie rule, batch>1
semantics) are the ones listed in the design notes; each function states the
one it uses.

Parity status: every function above is pinned by tests under ``tests/``
(brute force on tiny inputs, round trip, closed forms, the paper's printed
numbers, a hand-worked encoding). None is "parity unpinned".
"""

from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = [
    "TiledCBC",
    "magnitude_prune",
    "threshold_for",
    "calibrated_threshold",
    "realized_sparsity",
    "active_mask",
    "batch_score",
    "batch_threshold",
    "MASKS",
    "masked_activations",
    "encode",
    "encode_brute",
    "decode",
    "spmspv",
    "spmspv_rows",
    "spmm",
    "spmm_flops",
    "storage_bytes",
    "unpadded_bytes",
    "compression_ratio",
    "compute_intensity",
    "compute_intensity_spdp",
    "attainable",
    "combined_sparsity",
    "algorithmic_bytes",
    "useful_flops",
    "rtn_quantize",
    "rtn_dequantize",
    "encode_codes",
    "decode_codes",
    "spmspv_rtn",
    "algorithmic_bytes_codes",
]


def _bits(a: np.ndarray) -> np.ndarray:
    """fp16 array -> its uint16 bit patterns (no arithmetic)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return a
    if a.dtype != np.float16:
        raise TypeError(f"expected float16 or uint16 bits, got {a.dtype}")
    return a.view(np.uint16)


# --------------------------------------------------------------------------
# Static pruning (Sec. 2.2: W_sp = W (.) M; magnitude criterion)
# --------------------------------------------------------------------------

def magnitude_prune(w: np.ndarray, sparsity: float) -> np.ndarray:
    """Global unstructured magnitude pruning of an fp16 matrix.

    The ``n = floor(sparsity * W.size)`` entries of smallest magnitude are set
    to +0 (bits 0x0000); all other entries keep their bits. Ties in magnitude
    are broken by row-major linear index, lowest first, so the result is
    unique. NaN entries are rejected (their magnitude has no order).

    Steps: the n-th smallest magnitude is the cut; every entry below the cut
    is pruned, and the entries equal to the cut are pruned in index order
    until n entries are pruned in total.
    """
    if not 0.0 <= sparsity <= 1.0:
        raise ValueError("sparsity must lie in [0, 1]")
    w = np.asarray(w, dtype=np.float16)
    if np.isnan(w).any():
        raise ValueError("NaN weights cannot be magnitude-pruned")
    flat = w.reshape(-1)
    n = int(math.floor(sparsity * flat.size))
    out = flat.copy()
    if n == 0:
        return out.reshape(w.shape)
    mag = np.abs(flat.astype(np.float64))
    cut = np.partition(mag, n - 1)[n - 1]
    below = mag < cut
    quota = n - int(below.sum())
    tied = np.flatnonzero(mag == cut)[:quota]
    out[below] = np.float16(0.0)  # +0
    out[tied] = np.float16(0.0)
    return out.reshape(w.shape)


# --------------------------------------------------------------------------
# Dynamic pruning (Sec. 2.2: W_dp(x) = W (.) M(x); TEAL threshold, Sec. 5.1)
# --------------------------------------------------------------------------

def threshold_for(x: np.ndarray, p: float) -> np.float32:
    """Magnitude threshold whose strict rule ``|x| > t`` drops a fraction p.

    The empirical distribution of |x| over every entry of ``x`` (all tokens
    pooled) is sorted ascending and ``t`` is its ``ceil(p * n)``-th smallest
    value, so at least ``ceil(p * n)`` entries satisfy ``|x| <= t``. For
    ``p == 0`` the threshold is -1, which keeps every entry. The result is a
    float32 (every fp16 magnitude is exact in float32). NaN is rejected.
    """
    if not 0.0 <= p <= 1.0:
        raise ValueError("p must lie in [0, 1]")
    x = np.asarray(x, dtype=np.float16)
    if np.isnan(x).any():
        raise ValueError("NaN activations have no magnitude order")
    if p == 0.0 or x.size == 0:
        return np.float32(-1.0)
    v = np.sort(np.abs(x.astype(np.float64)).reshape(-1))
    idx = int(math.ceil(p * v.size)) - 1
    return np.float32(v[idx])


def calibrated_threshold(samples: np.ndarray, p: float) -> np.float32:
    """A layer's threshold calibrated offline (Sec. 5.1, the DP setup).

    The layer's activation magnitudes over a calibration set (tokens drawn
    separately from the inputs the threshold is later applied to) form an
    empirical CDF; the threshold for a target dynamic sparsity p is its
    p-quantile. That is the quantile rule of ``threshold_for`` applied to the
    calibration set instead of to the input itself.
    """
    return threshold_for(samples, p)


def realized_sparsity(x: np.ndarray, t: float) -> float:
    """Fraction of the entries of ``x`` the rule ``|x| > t`` drops."""
    x = np.asarray(x, dtype=np.float16)
    if x.size == 0:
        return 0.0
    return float(1.0 - active_mask(x.reshape(1, -1), t).mean())


MASKS = ("token", "batch")


def batch_score(x: np.ndarray) -> np.ndarray:
    """Per-column score of a batch: ``s_k = sum_b |x[b, k]|`` in float32,
    tokens added in ascending order, each addition rounded to nearest even
    (the first one exact). NaN entries make the score NaN."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float16))
    s = np.zeros(x.shape[1], dtype=np.float32)
    with np.errstate(invalid="ignore", over="ignore"):
        for b in range(x.shape[0]):
            s = (s + np.abs(x[b].astype(np.float32))).astype(np.float32)
    return s


def batch_threshold(t: float, batch: int) -> np.float32:
    """The score threshold ``T = fp32(batch * fp32(t))`` (one rounding)."""
    return np.float32(np.float64(np.float32(t)) * batch)


def active_mask(x: np.ndarray, t: float, mask: str = "token") -> np.ndarray:
    """Column activity per token, ``[batch, cols]`` booleans.

    ``mask="token"`` (the DP definition, Sec. 2.2): ``|x[b, k]| > t``
    (strict), float64 compare. ``mask="batch"`` (batched DP, one column set
    shared by the batch; the paper leaves batched DP to future work, this is
    the reading built here): column k is active for every token iff its batch
    score exceeds ``batch_threshold(t, batch)``, i.e. the batch's mean |x|
    exceeds t; at batch 1 the two rules coincide. NaN activations are never
    active (a NaN makes the comparison false).
    """
    x = np.atleast_2d(np.asarray(x, dtype=np.float16))
    if mask == "token":
        with np.errstate(invalid="ignore"):
            return np.abs(x.astype(np.float64)) > np.float64(np.float32(t))
    if mask == "batch":
        with np.errstate(invalid="ignore"):
            shared = batch_score(x) > batch_threshold(t, x.shape[0])
        return np.broadcast_to(shared[None, :], x.shape).copy()
    raise ValueError(f"unknown mask {mask!r}")


def masked_activations(x: np.ndarray, t: float, mask: str = "token") -> np.ndarray:
    """``xm[b, k] = x[b, k]`` where active, else +0; stays fp16 (exact)."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float16))
    return np.where(active_mask(x, t, mask), x, np.float16(0.0)).astype(np.float16)


# --------------------------------------------------------------------------
# Tiled-CBC (Sec. 4.1)
# --------------------------------------------------------------------------

@dataclasses.dataclass
class TiledCBC:
    """The four arrays of the Tiled-CBC format plus its shape parameters.

    * ``tile_offset`` uint32 [NGT + 1]: start (in fp16 elements) of each GTile
      in ``values``; the last entry is ``len(values)``.
    * ``col_info`` uint32 [NGT * tile_k]: ``(offset << 16) | nnz`` per column
      of each GTile; offset in fp16 elements from the GTile start, counting
      earlier columns' padding; nnz without padding.
    * ``bitmap`` uint64 [NGT * tile_k * tile_m / 64]: ``tile_m / 64`` words per
      column, a column's words contiguous; bit i of word w <-> row 64 w + i
      of the tile's row stripe.
    * ``values`` uint16 (fp16 bits): GTile-major, column-major inside a GTile,
      rows ascending inside a column, each column zero-padded to a multiple
      of 8 elements (16 bytes).

    GTiles are numbered row-major: ``g = r * C + c`` for row stripe r and
    column block c.
    """

    rows: int
    cols: int
    tile_m: int
    tile_k: int
    tile_offset: np.ndarray
    col_info: np.ndarray
    bitmap: np.ndarray
    values: np.ndarray

    @property
    def n_stripes(self) -> int:
        return -(-self.rows // self.tile_m)

    @property
    def n_colblocks(self) -> int:
        return -(-self.cols // self.tile_k)

    @property
    def n_gtiles(self) -> int:
        return self.n_stripes * self.n_colblocks

    @property
    def words_per_column(self) -> int:
        return self.tile_m // 64

    def column(self, r: int, k: int):
        """(base element index in values, nnz, bitmap words) of column k of stripe r."""
        g = r * self.n_colblocks + k // self.tile_k
        j = k % self.tile_k
        ci = int(self.col_info[g * self.tile_k + j])
        wpc = self.words_per_column
        words = self.bitmap[(g * self.tile_k + j) * wpc:(g * self.tile_k + j + 1) * wpc]
        return int(self.tile_offset[g]) + (ci >> 16), ci & 0xFFFF, words


def _check_tile(tile_m: int, tile_k: int) -> None:
    if tile_m < 64 or tile_m > 1024 or tile_m % 64:
        raise ValueError("tile_m must be a multiple of 64 in [64, 1024]")
    if tile_k < 1 or tile_k > 256 or (tile_k & (tile_k - 1)):
        raise ValueError("tile_k must be a power of two in [1, 256]")
    if (tile_k - 1) * tile_m > 0xFFFF:
        raise ValueError("(tile_k - 1) * tile_m must fit the 16-bit ColInfo offset")


def _pad8(n: int) -> int:
    return (n + 7) // 8 * 8


def encode(w: np.ndarray, tile_m: int, tile_k: int) -> TiledCBC:
    """Encode an fp16 matrix into Tiled-CBC, walking the format as Sec. 4.1 lays it out.

    The matrix is conceptually zero-padded to whole tiles. For every GTile in
    row-major order, for every column of the GTile left to right: set one
    bitmap bit per nonzero row (nonzero means the magnitude bits are nonzero,
    so -0 counts as zero), append the nonzero values top to bottom, pad the
    column to a multiple of 8 values with +0, and record the column's offset
    inside the GTile and its nonzero count in ColInfo. TileOffset is the
    running total of the GTiles' padded sizes.
    """
    _check_tile(tile_m, tile_k)
    wb = _bits(np.asarray(w))
    rows, cols = wb.shape
    R = -(-rows // tile_m)
    C = -(-cols // tile_k)
    wpc = tile_m // 64
    padded = np.zeros((R * tile_m, C * tile_k), dtype=np.uint16)
    padded[:rows, :cols] = wb
    tile_offset = np.zeros(R * C + 1, dtype=np.uint64)
    col_info = np.zeros(R * C * tile_k, dtype=np.uint32)
    bitmap = np.zeros(R * C * tile_k * wpc, dtype=np.uint64)
    chunks = []
    weights_of_bit = np.left_shift(np.uint64(1), np.arange(64, dtype=np.uint64))
    total = 0
    for r in range(R):
        for c in range(C):
            g = r * C + c
            off = 0
            for j in range(tile_k):
                col = padded[r * tile_m:(r + 1) * tile_m, c * tile_k + j]
                nz = (col & 0x7FFF) != 0
                for wi in range(wpc):
                    seg = nz[64 * wi:64 * (wi + 1)]
                    bitmap[(g * tile_k + j) * wpc + wi] = np.bitwise_or.reduce(
                        np.where(seg, weights_of_bit, np.uint64(0)))
                vals = col[nz]
                nnz = int(vals.size)
                padn = _pad8(nnz)
                chunks.append(vals)
                if padn > nnz:
                    chunks.append(np.zeros(padn - nnz, dtype=np.uint16))
                col_info[g * tile_k + j] = (off << 16) | nnz
                off += padn
            total += off
            tile_offset[g + 1] = total
    if total > 0xFFFFFFFF:
        raise ValueError("encoded matrix exceeds 2^32 - 1 values")
    values = np.concatenate(chunks) if chunks else np.zeros(0, dtype=np.uint16)
    return TiledCBC(rows, cols, tile_m, tile_k, tile_offset.astype(np.uint32),
                    col_info, bitmap, values.astype(np.uint16))


def encode_brute(w: np.ndarray, tile_m: int, tile_k: int) -> TiledCBC:
    """Scalar, bit-by-bit encoder in plain Python ints, for tiny matrices.

    Same definition as ``encode``, written element by element without NumPy
    vector operations, so that the two can check each other.
    """
    _check_tile(tile_m, tile_k)
    wb = _bits(np.asarray(w))
    rows, cols = wb.shape
    R = -(-rows // tile_m)
    C = -(-cols // tile_k)
    wpc = tile_m // 64

    def elem(m, k):
        return int(wb[m, k]) if (m < rows and k < cols) else 0

    tile_offset = [0]
    col_info, bitmap, values = [], [], []
    for r in range(R):
        for c in range(C):
            off = 0
            for j in range(tile_k):
                k = c * tile_k + j
                nnz = 0
                for wi in range(wpc):
                    word = 0
                    for i in range(64):
                        h = elem(r * tile_m + 64 * wi + i, k)
                        if h & 0x7FFF:
                            word |= 1 << i
                            values.append(h)
                            nnz += 1
                    bitmap.append(word)
                padded = nnz
                while padded % 8:
                    values.append(0)
                    padded += 1
                col_info.append((off << 16) | nnz)
                off += padded
            tile_offset.append(tile_offset[-1] + off)
    return TiledCBC(rows, cols, tile_m, tile_k,
                    np.array(tile_offset, dtype=np.uint32),
                    np.array(col_info, dtype=np.uint32),
                    np.array(bitmap, dtype=np.uint64),
                    np.array(values, dtype=np.uint16))


def decode(f: TiledCBC) -> np.ndarray:
    """Rebuild the (pruned) fp16 matrix from its Tiled-CBC arrays.

    For each GTile and column, the r-th set bit (rows ascending) takes the
    r-th value of the column; every other element is +0.
    """
    R, C, wpc = f.n_stripes, f.n_colblocks, f.words_per_column
    out = np.zeros((R * f.tile_m, C * f.tile_k), dtype=np.uint16)
    for r in range(R):
        for c in range(C):
            g = r * C + c
            for j in range(f.tile_k):
                ci = int(f.col_info[g * f.tile_k + j])
                base = int(f.tile_offset[g]) + (ci >> 16)
                rank = 0
                for wi in range(wpc):
                    word = int(f.bitmap[(g * f.tile_k + j) * wpc + wi])
                    for i in range(64):
                        if (word >> i) & 1:
                            out[r * f.tile_m + 64 * wi + i, c * f.tile_k + j] = f.values[base + rank]
                            rank += 1
                if rank != (ci & 0xFFFF):
                    raise ValueError("bitmap popcount disagrees with ColInfo nnz")
    return out[:f.rows, :f.cols].view(np.float16)


def unpadded_bytes(f: TiledCBC) -> int:
    """Bytes of the four arrays with column padding left out (the quantity Sec. 4.1 counts)."""
    nnz = int(sum(int(ci) & 0xFFFF for ci in f.col_info))
    return 4 * f.tile_offset.size + 4 * f.col_info.size + 8 * f.bitmap.size + 2 * nnz


def storage_bytes(rows: int, cols: int, tile_m: int, tile_k: int, nnz: int) -> int:
    """Sec. 4.1 storage formula: 4(NGT+1) + 4 NGT TILE_K + 8 NBM + 2 NNZ.

    NGT = (M / TILE_M)(K / TILE_K), NBM = M K / 64; M and K are taken as the
    tile-padded sizes.
    """
    M = -(-rows // tile_m) * tile_m
    K = -(-cols // tile_k) * tile_k
    ngt = (M // tile_m) * (K // tile_k)
    nbm = M * K // 64
    return 4 * (ngt + 1) + 4 * ngt * tile_k + 8 * nbm + 2 * nnz


# --------------------------------------------------------------------------
# The masked product (Sec. 2.2; inactive columns contribute nothing, Sec. 4.2)
# --------------------------------------------------------------------------

def spmspv(w_sp: np.ndarray, x: np.ndarray, t: float, mask: str = "token"):
    """``y[b, m] = sum_k W_sp[m, k] * xm[b, k]`` in float64.

    Returns ``(y64, s64, y16)``: the float64 result, the magnitude sum
    ``S[b, m] = sum_k |W_sp[m, k]| |xm[b, k]|`` that scales the error bound,
    and ``y64`` rounded once to fp16 (round to nearest even).
    """
    w64 = np.asarray(w_sp, dtype=np.float16).astype(np.float64)
    xm = masked_activations(np.atleast_2d(x), t, mask).astype(np.float64)
    y64 = xm @ w64.T
    s64 = np.abs(xm) @ np.abs(w64).T
    return y64, s64, y64.astype(np.float16)


def spmspv_rows(w_sp: np.ndarray, x: np.ndarray, t: float, rows, mask: str = "token"):
    """The same product for selected output rows only (one dot product each)."""
    rows = np.asarray(rows, dtype=np.int64)
    w64 = np.asarray(w_sp, dtype=np.float16)[rows].astype(np.float64)
    xm = masked_activations(np.atleast_2d(x), t, mask).astype(np.float64)
    return xm @ w64.T, np.abs(xm) @ np.abs(w64).T


# --------------------------------------------------------------------------
# The prefill product (Sec. 4.3: prefill applies static pruning only, a
# sparse matrix times many tokens)
# --------------------------------------------------------------------------

def spmm(w_sp: np.ndarray, x: np.ndarray):
    """``Y[n, m] = sum_k W_sp[m, k] * X[n, k]`` for N tokens, in float64.

    No dynamic pruning: every column takes part (the prefill path drops the
    DP stage). Returns ``(y64, s64, y16)`` like ``spmspv``: the float64
    result, ``S[n, m] = sum_k |W_sp[m, k]| |X[n, k]|`` for the error bound,
    and ``y64`` rounded once to fp16.
    """
    w64 = np.asarray(w_sp, dtype=np.float16).astype(np.float64)
    x64 = np.atleast_2d(np.asarray(x, dtype=np.float16)).astype(np.float64)
    y64 = x64 @ w64.T
    s64 = np.abs(x64) @ np.abs(w64).T
    return y64, s64, y64.astype(np.float16)


def spmm_flops(w_sp: np.ndarray, n_tokens: int):
    """(useful, dense) flops of a prefill product: 2 x nonzeros x tokens,
    and 2 M K N for the dense matrix of the same shape."""
    nnz = int(((_bits(np.asarray(w_sp, dtype=np.float16)) & 0x7FFF) != 0).sum())
    m, k = np.asarray(w_sp).shape
    return 2 * nnz * int(n_tokens), 2 * m * k * int(n_tokens)


# --------------------------------------------------------------------------
# Roofline arithmetic (Sec. 3.1 Eq. 1-2 and roofline; Sec. 3.2 Eq. 3)
# --------------------------------------------------------------------------

def compression_ratio(rows: int, cols: int, stor_compressed: float) -> float:
    """Eq. 1: CR = 2 M K / Stor_compressed (fp16 dense storage over compressed)."""
    return 2.0 * rows * cols / stor_compressed


def compute_intensity(rows: int, n: int, cr: float) -> float:
    """Eq. 2: CI = M N / (M / CR + N)."""
    return rows * n / (rows / cr + n)


def compute_intensity_spdp(rows: int, n: int, cr: float, s: float) -> float:
    """Eq. 3: CI_SPDP = M N / ((M / CR)(1 - s) + N), s = skipped-column fraction."""
    return rows * n / ((rows / cr) * (1.0 - s) + n)


def attainable(peak: float, ci: float, bandwidth: float) -> float:
    """Roofline: P = min(P_peak, CI * B_mem)."""
    return min(peak, ci * bandwidth)


def combined_sparsity(sp: float, dp: float):
    """(overlap, total) when an SP fraction and an independent DP fraction combine.

    Overlap is sp * dp; total pruned is sp + dp - sp * dp = 1 - (1 - sp)(1 - dp).
    """
    overlap = sp * dp
    return overlap, sp + dp - overlap


# --------------------------------------------------------------------------
# What one call must move and compute
# --------------------------------------------------------------------------

def algorithmic_bytes(f: TiledCBC, x: np.ndarray, t: float, mask: str = "token") -> int:
    """Bytes a call must read/write given the active columns (union over tokens).

    For every row stripe and every active column: its ColInfo word (4 B), its
    bitmap (tile_m / 8 B) and its padded values (2 * pad8(nnz) B); plus one
    TileOffset entry (4 B) for each GTile that has an active column; plus the
    activations (2 B K) and the outputs (2 B M) per token.
    """
    x = np.atleast_2d(np.asarray(x, dtype=np.float16))
    act = active_mask(x, t, mask).any(axis=0)
    total = 0
    for r in range(f.n_stripes):
        touched = set()
        for k in range(f.cols):
            if not act[k]:
                continue
            _, nnz, _ = f.column(r, k)
            total += 4 + f.tile_m // 8 + 2 * _pad8(nnz)
            touched.add(k // f.tile_k)
        total += 4 * len(touched)
    b = x.shape[0]
    return total + 2 * b * f.cols + 2 * b * f.rows


def useful_flops(w_sp: np.ndarray, x: np.ndarray, t: float, mask: str = "token") -> int:
    """2 x the number of (token, nonzero weight, active column) products."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float16))
    act = active_mask(x, t, mask)
    nnz_col = ((_bits(np.asarray(w_sp, dtype=np.float16)) & 0x7FFF) != 0).sum(axis=0)
    return int(2 * (act * nnz_col[None, :]).sum())


# --------------------------------------------------------------------------
# Low-bit Values (Sec. 5.1 quantization setup; Sec. 6 on low-precision Values)
# --------------------------------------------------------------------------

def rtn_quantize(w_sp: np.ndarray, bits: int = 4):
    """Round-to-nearest weight-only quantization of a pruned fp16 matrix.

    The paper quantizes after pruning and before dynamic pruning, with 4-bit
    round-to-nearest, and gives no further detail. Reading: symmetric, one
    fp32 scale per output row, no zero point:

        s_m = fp32(max_k |W_sp[m, k]|) / fp32(2^(bits-1) - 1)   (fp32 division)
        q[m, k] = clamp(rint_even(fp32(W_sp[m, k]) / s_m), -qmax, qmax)

    with the division in fp32 and ties to even. The sparsity pattern is the
    pruning's: an entry is stored iff its magnitude bits are nonzero, also
    when its code rounds to 0; pruned entries have code 0 and are not
    stored. A row with no stored entry has scale 0. Non-finite weights are
    rejected. Returns ``(codes int8 [M, K], scales float32 [M], pattern bool
    [M, K])``.
    """
    if not (2 <= int(bits) <= 8):
        raise ValueError("bits must be in [2, 8]")
    wb = _bits(np.asarray(w_sp))
    w32 = wb.view(np.float16).astype(np.float32)  # exact
    if not np.all(np.isfinite(w32)):
        raise ValueError("weights must be finite")
    pattern = (wb & 0x7FFF) != 0
    qmax = np.float32(2 ** (int(bits) - 1) - 1)
    amax = np.where(pattern, np.abs(w32), np.float32(0)).max(axis=1).astype(np.float32)
    scales = (amax / qmax).astype(np.float32)
    codes = np.zeros(wb.shape, dtype=np.int8)
    live = scales > 0
    q = np.rint(w32[live] / scales[live, None]).astype(np.float32)
    q = np.clip(q, -qmax, qmax)
    codes[live] = np.where(pattern[live], q, 0).astype(np.int8)
    return codes, scales, pattern


def rtn_dequantize(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """The weights the quantized format stands for, in float64: s_m * q[m, k]."""
    return np.asarray(scales, dtype=np.float64)[:, None] * np.asarray(codes, dtype=np.float64)


def _pad16(n: int) -> int:
    return (n + 15) // 16 * 16


def encode_codes(codes: np.ndarray, pattern: np.ndarray, tile_m: int, tile_k: int) -> TiledCBC:
    """Tiled-CBC with one byte per value: the layout of ``encode`` (same
    GTile and column order, same bitmaps from the sparsity pattern), the
    Values array holding the codes as two's-complement bytes, each column
    padded with 0 to a multiple of 16 codes (16 bytes), and TileOffset and
    the ColInfo offsets counted in codes.
    """
    _check_tile(tile_m, tile_k)
    codes = np.asarray(codes, dtype=np.int8)
    pattern = np.asarray(pattern, dtype=bool)
    rows, cols = codes.shape
    R = -(-rows // tile_m)
    C = -(-cols // tile_k)
    wpc = tile_m // 64
    pc = np.zeros((R * tile_m, C * tile_k), dtype=np.int8)
    pp = np.zeros((R * tile_m, C * tile_k), dtype=bool)
    pc[:rows, :cols] = codes
    pp[:rows, :cols] = pattern
    tile_offset = np.zeros(R * C + 1, dtype=np.uint64)
    col_info = np.zeros(R * C * tile_k, dtype=np.uint32)
    bitmap = np.zeros(R * C * tile_k * wpc, dtype=np.uint64)
    chunks = []
    weights_of_bit = np.left_shift(np.uint64(1), np.arange(64, dtype=np.uint64))
    total = 0
    for r in range(R):
        for c in range(C):
            g = r * C + c
            off = 0
            for j in range(tile_k):
                col = pc[r * tile_m:(r + 1) * tile_m, c * tile_k + j]
                nz = pp[r * tile_m:(r + 1) * tile_m, c * tile_k + j]
                for wi in range(wpc):
                    seg = nz[64 * wi:64 * (wi + 1)]
                    bitmap[(g * tile_k + j) * wpc + wi] = np.bitwise_or.reduce(
                        np.where(seg, weights_of_bit, np.uint64(0)))
                vals = col[nz]
                nnz = int(vals.size)
                padn = _pad16(nnz)
                chunks.append(vals)
                if padn > nnz:
                    chunks.append(np.zeros(padn - nnz, dtype=np.int8))
                col_info[g * tile_k + j] = (off << 16) | nnz
                off += padn
            total += off
            tile_offset[g + 1] = total
    if total > 0xFFFFFFFF:
        raise ValueError("encoded matrix exceeds 2^32 - 1 values")
    values = np.concatenate(chunks) if chunks else np.zeros(0, dtype=np.int8)
    return TiledCBC(rows, cols, tile_m, tile_k, tile_offset.astype(np.uint32),
                    col_info, bitmap, values.astype(np.int8).view(np.uint8))


def decode_codes(f: TiledCBC):
    """Rebuild ``(codes int8 [M, K], pattern bool [M, K])`` from a one-byte-per-value Tiled-CBC."""
    R, C, wpc = f.n_stripes, f.n_colblocks, f.words_per_column
    vals = np.asarray(f.values, dtype=np.uint8).view(np.int8)
    codes = np.zeros((R * f.tile_m, C * f.tile_k), dtype=np.int8)
    pattern = np.zeros((R * f.tile_m, C * f.tile_k), dtype=bool)
    for r in range(R):
        for c in range(C):
            g = r * C + c
            for j in range(f.tile_k):
                ci = int(f.col_info[g * f.tile_k + j])
                base = int(f.tile_offset[g]) + (ci >> 16)
                rank = 0
                for wi in range(wpc):
                    word = int(f.bitmap[(g * f.tile_k + j) * wpc + wi])
                    for i in range(64):
                        if (word >> i) & 1:
                            codes[r * f.tile_m + 64 * wi + i, c * f.tile_k + j] = vals[base + rank]
                            pattern[r * f.tile_m + 64 * wi + i, c * f.tile_k + j] = True
                            rank += 1
                if rank != (ci & 0xFFFF):
                    raise ValueError("bitmap popcount disagrees with ColInfo nnz")
    return codes[:f.rows, :f.cols], pattern[:f.rows, :f.cols]


def spmspv_rtn(codes: np.ndarray, scales: np.ndarray, x: np.ndarray, t: float, mask: str = "token"):
    """The masked product with the dequantized weights, in float64:
    ``y[b, m] = sum_k (s_m q[m, k]) xm[b, k]``. Returns ``(y64, s64, y16)``
    as ``spmspv`` does, with ``S[b, m] = sum_k |s_m q[m, k]| |xm[b, k]|``.
    """
    wq = rtn_dequantize(codes, scales)
    xm = masked_activations(np.atleast_2d(x), t, mask).astype(np.float64)
    y64 = xm @ wq.T
    s64 = np.abs(xm) @ np.abs(wq).T
    return y64, s64, y64.astype(np.float16)


def algorithmic_bytes_codes(f: TiledCBC, x: np.ndarray, t: float, mask: str = "token") -> int:
    """``algorithmic_bytes`` for one byte per value: padded codes (pad16(nnz)
    bytes) instead of fp16 values, plus the row scales (4 B per row)."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float16))
    act = active_mask(x, t, mask).any(axis=0)
    total = 0
    for r in range(f.n_stripes):
        touched = set()
        for k in range(f.cols):
            if not act[k]:
                continue
            _, nnz, _ = f.column(r, k)
            total += 4 + f.tile_m // 8 + _pad16(nnz)
            touched.add(k // f.tile_k)
        total += 4 * len(touched)
    b = x.shape[0]
    return total + 2 * b * f.cols + 2 * b * f.rows + 4 * f.rows

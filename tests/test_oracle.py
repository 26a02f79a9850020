"""Pins for the CPU oracle: each check ties it to something other than itself.

Sources of truth used here: values the paper prints (tests/golden/
paper_numbers.json), hand-worked encodings (tests/golden/tiled_cbc_hand.json),
brute force in exact arithmetic on tiny inputs, closed forms and invariants.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
from conftest import GOLDEN


def _hand_cases():
    with open(os.path.join(GOLDEN, "tiled_cbc_hand.json")) as fh:
        return json.load(fh)["cases"]


def _paper():
    with open(os.path.join(GOLDEN, "paper_numbers.json")) as fh:
        return json.load(fh)


def _hand_matrix(case):
    w = np.zeros((case["rows"], case["cols"]), dtype=np.uint16)
    for m, k, h in case["nonzeros"]:
        w[m, k] = int(h, 16)
    return w


def _exact(h):
    """Exact rational value of an fp16 bit pattern (finite only), no NumPy floats."""
    h = int(h)
    sign = -1 if h & 0x8000 else 1
    e = (h >> 10) & 0x1F
    f = h & 0x3FF
    assert e != 0x1F
    if e == 0:
        return sign * Fraction(f, 1 << 24)
    return sign * Fraction(1024 + f, 1024) * Fraction(2) ** (e - 15)


# ---------------------------------------------------------------------------
# Tiled-CBC encoding
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("case", _hand_cases(), ids=lambda c: c["name"])
def test_encode_matches_hand_worked_case(case):
    w = _hand_matrix(case)
    for enc in (oracle.encode, oracle.encode_brute):
        f = enc(w, case["tile_m"], case["tile_k"])
        assert f.tile_offset.tolist() == case["tile_offset"]
        assert f.col_info.tolist() == [int(v, 16) for v in case["col_info"]]
        assert f.bitmap.tolist() == [int(v, 16) for v in case["bitmap"]]
        assert f.values.tolist() == [int(v, 16) for v in case["values"]]


@pytest.mark.parametrize("case", _hand_cases(), ids=lambda c: c["name"])
def test_product_matches_hand_worked_case(case):
    w = _hand_matrix(case).view(np.float16)
    for prod in case["products"]:
        x = np.array([prod["x"]], dtype=np.float16)
        y64, s64, y16 = oracle.spmspv(w, x, prod["t"])
        expect = np.zeros(case["rows"])
        for m, v in prod["y_nonzero"]:
            expect[m] = v
        assert np.array_equal(y64[0], expect)
        assert np.array_equal(y16[0].astype(np.float64), expect)


def test_padding_example_from_paper():
    pad = _paper()["column_padding"]
    w = np.zeros((64, 1), dtype=np.float16)
    w[:pad["nnz"], 0] = np.float16(1.5)
    f = oracle.encode(w, 64, 1)
    assert f.values.size * 2 == pad["padded_bytes"]
    assert f.values.size * 2 - pad["nnz"] * 2 == pad["pad_bytes"]


def test_bitmap_words_per_column_from_paper():
    p = _paper()["bitmap_words_per_column"]
    w = synth.weights(p["tile_m"], 3, 7)
    f = oracle.encode(w, p["tile_m"], 1)
    assert f.bitmap.size == 3 * p["words"]


@pytest.mark.parametrize("rows,cols,tm,tk,sw,seed", [
    (64, 1, 64, 1, 0.0, 1), (64, 16, 64, 16, 0.5, 2), (130, 37, 64, 4, 0.6, 3),
    (200, 33, 128, 8, 0.3, 4), (256, 40, 256, 16, 0.7, 5), (70, 9, 192, 2, 0.9, 6),
    (65, 65, 64, 64, 0.5, 7), (129, 5, 1024, 1, 0.2, 8), (1, 1, 64, 1, 0.0, 9),
])
def test_encode_equals_scalar_brute_force(rows, cols, tm, tk, sw, seed):
    w = oracle.magnitude_prune(synth.weights(rows, cols, seed), sw)
    a = oracle.encode(w, tm, tk)
    b = oracle.encode_brute(w, tm, tk)
    for name in ("tile_offset", "col_info", "bitmap", "values"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name


@pytest.mark.parametrize("rows,cols,tm,tk,sw,seed", [
    (300, 70, 128, 16, 0.6, 11), (256, 256, 256, 16, 0.5, 12), (97, 130, 64, 32, 0.8, 13),
    (512, 64, 512, 8, 0.0, 14), (1024, 48, 1024, 16, 0.95, 15),
])
def test_encode_round_trip_and_invariants(rows, cols, tm, tk, sw, seed):
    w = oracle.magnitude_prune(synth.weights(rows, cols, seed), sw)
    f = oracle.encode(w, tm, tk)
    # round trip: decoding gives back W_sp bit for bit (pruned entries are +0)
    assert np.array_equal(oracle.decode(f).view(np.uint16), w.view(np.uint16))
    wb = w.view(np.uint16)
    nnz = int(((wb & 0x7FFF) != 0).sum())
    # popcount of every bitmap equals the number of stored nonzeros
    pop = sum(bin(int(v)).count("1") for v in f.bitmap)
    assert pop == nnz == int(sum(int(c) & 0xFFFF for c in f.col_info))
    wpc = tm // 64
    for idx, ci in enumerate(f.col_info):
        words = f.bitmap[idx * wpc:(idx + 1) * wpc]
        assert sum(bin(int(v)).count("1") for v in words) == (int(ci) & 0xFFFF)
        assert (int(ci) >> 16) % 8 == 0
    # TileOffset: starts at 0, nondecreasing, multiples of 8, ends at len(values)
    to = f.tile_offset.astype(np.int64)
    assert to[0] == 0 and np.all(np.diff(to) >= 0) and np.all(to % 8 == 0)
    assert to[-1] == f.values.size
    # padding entries are +0; stored entries are nonzero
    used = np.zeros(f.values.size, dtype=bool)
    for r in range(f.n_stripes):
        for k in range(f.n_colblocks * tk):
            g = r * f.n_colblocks + k // tk
            ci = int(f.col_info[g * tk + k % tk])
            base = int(f.tile_offset[g]) + (ci >> 16)
            used[base:base + (ci & 0xFFFF)] = True
    assert np.all(f.values[~used] == 0)
    assert np.all((f.values[used] & 0x7FFF) != 0)
    # Sec. 4.1 storage formula equals the byte count of the arrays without padding
    assert oracle.unpadded_bytes(f) == oracle.storage_bytes(rows, cols, tm, tk, nnz)


def test_storage_formula_worked_numbers():
    p = _paper()["storage_llama7b_attn_50"]
    total = oracle.storage_bytes(p["rows"], p["cols"], p["tile_m"], p["tile_k"], p["nnz"])
    assert total == p["total_bytes"]
    assert total == p["tile_offset_bytes"] + p["col_info_bytes"] + p["bitmap_bytes"] + p["values_bytes"]


def test_negative_zero_is_not_stored():
    w = np.zeros((64, 2), dtype=np.uint16)
    w[:, 0] = 0x8000
    w[7, 1] = 0x8001  # smallest negative subnormal: nonzero
    f = oracle.encode(w, 64, 2)
    assert f.bitmap.tolist() == [0, 1 << 7]
    assert f.values.tolist()[:1] == [0x8001]
    assert np.array_equal(oracle.decode(f).view(np.uint16)[:, 1], w[:, 1])
    assert np.all(oracle.decode(f).view(np.uint16)[:, 0] == 0)


@pytest.mark.parametrize("tm,tk", [(32, 1), (100, 1), (1088, 1), (64, 3), (64, 512), (1024, 65)])
def test_encode_rejects_bad_tiles(tm, tk):
    with pytest.raises(ValueError):
        oracle.encode(np.zeros((4, 4), dtype=np.float16), tm, tk)


# ---------------------------------------------------------------------------
# Magnitude pruning
# ---------------------------------------------------------------------------

def _prune_brute(w, sparsity):
    flat = [int(v) for v in w.view(np.uint16).reshape(-1)]
    n = math.floor(sparsity * len(flat))
    keyed = sorted(range(len(flat)), key=lambda i: (abs(_exact(flat[i])), i))
    out = list(flat)
    for i in keyed[:n]:
        out[i] = 0
    return np.array(out, dtype=np.uint16).reshape(w.shape)


@pytest.mark.parametrize("shape,sw,seed", [((8, 8), 0.5, 1), ((13, 7), 0.3, 2), ((5, 40), 0.77, 3),
                                           ((16, 16), 0.0, 4), ((9, 9), 1.0, 5)])
def test_prune_equals_brute_force(shape, sw, seed):
    w = synth.weights(*shape, seed)
    got = oracle.magnitude_prune(w, sw).view(np.uint16)
    assert np.array_equal(got, _prune_brute(w, sw))


def test_prune_tie_break_and_signed_zero():
    # equal magnitudes of both signs plus -0: the cut falls inside the tie
    w = np.array([[0.5, -0.5, 0.25, -0.0], [0.5, 1.0, -0.25, 0.5]], dtype=np.float16)
    got = oracle.magnitude_prune(w, 0.5).view(np.uint16)
    # order by (|w|, index): idx3 (-0), idx2 (0.25), idx6 (-0.25), idx0 (0.5) are the four smallest
    expect = w.view(np.uint16).copy().reshape(-1)
    expect[[3, 2, 6, 0]] = 0
    assert np.array_equal(got.reshape(-1), expect)


def test_prune_invariants_medium():
    w = synth.weights(256, 192, 21)
    w[3, :40] = np.float16(0.0)  # some entries already zero
    sw = 0.6
    p = oracle.magnitude_prune(w, sw)
    wb, pb = w.view(np.uint16).reshape(-1), p.view(np.uint16).reshape(-1)
    mag = np.abs(w.astype(np.float64)).reshape(-1)
    n = math.floor(sw * w.size)
    z = int(((wb & 0x7FFF) == 0).sum())
    # the output differs from the input only where it became +0
    assert np.all((pb == wb) | (pb == 0))
    # exactly max(n, #already-zero) entries have zero magnitude afterwards
    out_zero = (pb & 0x7FFF) == 0
    assert out_zero.sum() == max(n, z)
    # every kept magnitude is at least every pruned magnitude
    assert mag[~out_zero].min() >= mag[out_zero].max()


def test_prune_rejects_nan():
    with pytest.raises(ValueError):
        oracle.magnitude_prune(np.array([[np.nan, 1]], dtype=np.float16), 0.5)


# ---------------------------------------------------------------------------
# Threshold and activity
# ---------------------------------------------------------------------------

def _threshold_brute(x, p):
    if p == 0:
        return -1.0
    mags = [abs(_exact(h)) for h in x.view(np.uint16).reshape(-1)]
    need = math.ceil(p * len(mags))
    # smallest candidate magnitude v with #{|x| <= v} >= need
    return float(min(v for v in set(mags) if sum(1 for m in mags if m <= v) >= need))


@pytest.mark.parametrize("p", [0.0, 0.1, 0.25, 0.5, 0.7, 0.99, 1.0])
def test_threshold_equals_counting_definition(p):
    x = synth.laplace_activations(3, 50, 31)
    assert float(oracle.threshold_for(x, p)) == _threshold_brute(x, p)


def test_threshold_with_ties():
    x = np.array([[1.0, -1.0, 1.0, 2.0, 0.0, -0.0, 3.0, 1.0]], dtype=np.float16)
    t = oracle.threshold_for(x, 0.5)  # 4th smallest of 0,0,1,1,1,1,2,3 is 1
    assert t == np.float32(1.0)
    act = oracle.active_mask(x, t)
    assert act.tolist() == [[False, False, False, True, False, False, True, False]]


# ---------------------------------------------------------------------------
# Offline calibration (Sec. 5.1, the DP setup): a layer's threshold is the
# quantile of the empirical CDF of its activation magnitudes over a separate
# calibration set, then applied to inputs the calibration never saw.

def _mixture_quantile(p, frac_out, scale=20.0):
    """p-quantile of |x| for Laplace(0, 1) entries of which a fraction
    frac_out is scaled by `scale`: F(t) = (1 - f)(1 - e^-t) + f(1 - e^(-t/scale)),
    solved by bisection."""
    lo, hi = 0.0, 1000.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        f = (1 - frac_out) * (1 - math.exp(-mid)) + frac_out * (1 - math.exp(-mid / scale))
        lo, hi = (mid, hi) if f < p else (lo, mid)
    return 0.5 * (lo + hi)


@pytest.mark.parametrize("p", [0.25, 0.5, 0.7])
def test_calibrated_threshold_is_the_distributions_quantile(p):
    k = 4096
    cal = synth.laplace_activations(300, k, 211, draw=1)
    t = float(oracle.calibrated_threshold(cal, p))
    exact = _mixture_quantile(p, round(0.01 * k) / k)
    # the quantile of 1.2 M draws deviates by < 1e-3 (standard error ~ 2e-4
    # to 5e-4 here), fp16 rounding of |x| near t by < 4e-4
    assert abs(t - exact) < 5e-3, (t, exact)


def test_calibrated_threshold_holds_on_unseen_tokens():
    cal = synth.laplace_activations(300, 4096, 211, draw=1)
    held = synth.laplace_activations(64, 4096, 211, draw=2)
    x = synth.laplace_activations(1, 4096, 211)
    for p in (0.25, 0.5, 0.7):
        t = oracle.calibrated_threshold(cal, p)
        # 262144 held-out entries: standard deviation of the fraction < 1e-3
        assert abs(oracle.realized_sparsity(held, t) - p) < 0.01
        # the input's own percentile drops p of it, up to ties at t
        assert abs(oracle.realized_sparsity(x, oracle.threshold_for(x, p)) - p) < 5e-3


def test_realized_sparsity_counts_dropped_entries():
    x = np.array([[1.0, -1.0, 0.5, 2.0], [0.0, -3.0, 1.0, 0.25]], dtype=np.float16)
    assert oracle.realized_sparsity(x, 1.0) == 6 / 8      # |x| > 1 keeps 2.0 and -3.0
    assert oracle.realized_sparsity(x, -1.0) == 0.0
    assert oracle.realized_sparsity(x, 3.0) == 1.0


def test_calibration_draws_keep_the_layers_outlier_channels():
    base = synth.laplace_activations(2, 512, 77)
    assert np.array_equal(base.view(np.uint16), synth.laplace_activations(2, 512, 77, draw=0).view(np.uint16))
    d1 = synth.laplace_activations(200, 512, 77, draw=1)
    d2 = synth.laplace_activations(200, 512, 77, draw=2)
    assert not np.array_equal(d1.view(np.uint16), d2.view(np.uint16))
    # the 5 outlier channels (1 % of 512) stand out in both draws
    top = [set(np.argsort(-np.abs(d.astype(np.float64)).mean(axis=0))[:5].tolist()) for d in (d1, d2)]
    assert top[0] == top[1]
    s0 = synth.swiglu_activations(2, 300, 5)
    assert np.array_equal(s0.view(np.uint16), synth.swiglu_activations(2, 300, 5, draw=0).view(np.uint16))
    assert not np.array_equal(s0.view(np.uint16), synth.swiglu_activations(2, 300, 5, draw=1).view(np.uint16))


def test_active_mask_elementwise_definition():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16).reshape(1, -1)
    for t in (-1.0, 0.0, 6e-8, 0.5, 0.50006, 1.0, 65504.0, 70000.0, float("inf")):
        t32 = float(np.float32(t))
        act = oracle.active_mask(x, t)[0]
        for h in list(range(0, 1 << 16, 97)) + [0x7C00, 0xFC00, 0x7C01, 0xFE00, 0x7BFF, 0x0001, 0x8000]:
            e, f = (h >> 10) & 0x1F, h & 0x3FF
            if e == 0x1F:
                expect = (f == 0) and (math.inf > t32)  # +-inf vs t; NaN is never active
            else:
                expect = abs(float(_exact(h))) > t32  # both sides exact in a Python float
            assert bool(act[h]) == expect, (h, t)


def test_masked_activations_keep_bits():
    x = synth.laplace_activations(2, 64, 5)
    t = oracle.threshold_for(x, 0.5)
    xm = oracle.masked_activations(x, t)
    act = oracle.active_mask(x, t)
    assert np.array_equal(xm.view(np.uint16)[act], x.view(np.uint16)[act])
    assert np.all(xm.view(np.uint16)[~act] == 0)


# ---------------------------------------------------------------------------
# The masked product
# ---------------------------------------------------------------------------

def _product_exact(w, x, t):
    M, K = w.shape
    B = x.shape[0]
    tt = Fraction(float(np.float32(t)))
    out = [[Fraction(0)] * M for _ in range(B)]
    wb, xb = w.view(np.uint16), x.view(np.uint16)
    for b in range(B):
        for k in range(K):
            xv = _exact(xb[b, k])
            if not abs(xv) > tt:
                continue
            for m in range(M):
                out[b][m] += _exact(wb[m, k]) * xv
    return out


@pytest.mark.parametrize("M,K,B,sw,p,seed", [(7, 9, 1, 0.5, 0.5, 1), (16, 20, 3, 0.3, 0.25, 2),
                                             (5, 33, 2, 0.0, 0.0, 3), (12, 12, 4, 0.9, 0.7, 4)])
def test_product_equals_exact_brute_force(M, K, B, sw, p, seed):
    w = oracle.magnitude_prune(synth.weights(M, K, seed), sw)
    x = synth.laplace_activations(B, K, seed + 100)
    t = oracle.threshold_for(x, p)
    y64, s64, y16 = oracle.spmspv(w, x, t)
    ex = _product_exact(w, x, t)
    for b in range(B):
        for m in range(M):
            assert abs(Fraction(float(y64[b, m])) - ex[b][m]) <= Fraction(1, 10**12) * (1 + abs(ex[b][m]))
            # y16 is the fp16 nearest to the exact value (ties far from likely)
            assert abs(float(y16[b, m]) - float(ex[b][m])) <= abs(float(np.float16(float(ex[b][m]))) - float(ex[b][m])) + 1e-30


def test_dense_no_threshold_is_plain_gemv():
    w = synth.weights(40, 30, 9)
    x = synth.laplace_activations(1, 30, 10)
    y64, _, _ = oracle.spmspv(w, x, -1.0)
    ex = _product_exact(w, x, -1.0)
    assert np.allclose(y64[0], [float(v) for v in ex[0]], rtol=1e-13, atol=0)


def test_all_inactive_gives_zero():
    w = synth.weights(33, 17, 3)
    x = synth.laplace_activations(2, 17, 4)
    t = float(np.abs(x.astype(np.float64)).max())
    y64, s64, y16 = oracle.spmspv(w, x, t)
    assert np.all(y64 == 0) and np.all(s64 == 0) and np.all(y16.astype(np.float64) == 0)


def test_single_active_column_is_scaled_column():
    w = synth.weights(50, 12, 5)
    x = np.full((1, 12), 0.25, dtype=np.float16)
    x[0, 7] = np.float16(-3.0)
    y64, _, _ = oracle.spmspv(w, x, 1.0)
    assert np.array_equal(y64[0], -3.0 * w[:, 7].astype(np.float64))


def test_rows_subset_agrees():
    w = oracle.magnitude_prune(synth.weights(64, 48, 8), 0.5)
    x = synth.laplace_activations(3, 48, 9)
    t = oracle.threshold_for(x, 0.4)
    y64, s64, _ = oracle.spmspv(w, x, t)
    rows = [0, 5, 63, 17]
    ex = _product_exact(w, x, t)
    yr, sr = oracle.spmspv_rows(w, x, t, rows)
    for b in range(3):
        for i, m in enumerate(rows):
            assert abs(yr[b, i] - float(ex[b][m])) <= 1e-12 * (1 + abs(float(ex[b][m])))
    assert np.allclose(sr, s64[:, rows])


# ---------------------------------------------------------------------------
# Sec. 3 arithmetic and the byte model
# ---------------------------------------------------------------------------

def test_combined_sparsity_paper_numbers():
    for c in _paper()["combined_sparsity"]:
        ov, tot = oracle.combined_sparsity(c["sp"], c["dp"])
        assert tot == pytest.approx(c["total"], abs=1e-12)
        if "overlap" in c:
            assert ov == pytest.approx(c["overlap"], abs=1e-12)
        assert tot == pytest.approx(1 - (1 - c["sp"]) * (1 - c["dp"]), abs=1e-12)


def test_intensity_formulas_from_flops_and_bytes():
    # Eq. 2 is FLOPs / bytes with FLOPs = 2 M K N and bytes = 2 M K / CR + 2 K N
    for M, K, N, cr in [(4096, 4096, 1, 1.0), (8192, 1024, 8, 2.7), (11008, 4096, 32, 1.3)]:
        flops, byts = 2 * M * K * N, 2 * M * K / cr + 2 * K * N
        assert oracle.compute_intensity(M, N, cr) == pytest.approx(flops / byts, rel=1e-12)
        # Eq. 3 with s = 0 is Eq. 2; with s, only the weight bytes shrink
        assert oracle.compute_intensity_spdp(M, N, cr, 0.0) == pytest.approx(flops / byts, rel=1e-12)
        s = 0.5
        byts_s = 2 * M * K / cr * (1 - s) + 2 * K * N
        assert oracle.compute_intensity_spdp(M, N, cr, s) == pytest.approx(flops / byts_s, rel=1e-12)
    assert oracle.attainable(100.0, 2.0, 8.0) == 16.0 and oracle.attainable(10.0, 2.0, 8.0) == 10.0


def test_compression_ratio_pinned():
    # Eq. 1 for 4096 x 4096 at 50 % weight sparsity: 33,554,432 dense bytes over
    # the storage formula's 19,152,900 (pinned by hand in paper_numbers.json)
    # is 1.7519243561027311, worked out by hand (long division to 16 digits)
    assert oracle.compression_ratio(4096, 4096, 19152900) == pytest.approx(1.7519243561027311, rel=1e-15)
    # an uncompressed matrix (storage = 2 bytes per element) has CR = 1, and
    # storage above the dense size gives CR < 1 (the paper's remark that some
    # formats exceed the dense footprint at moderate sparsity)
    assert oracle.compression_ratio(1024, 512, 2 * 1024 * 512) == 1.0
    assert oracle.compression_ratio(64, 64, 3 * 64 * 64) == pytest.approx(2.0 / 3.0, rel=1e-15)
    # Eq. 2 fed with Eq. 1 is flops over the bytes actually moved: CI(M, N,
    # CR) = 2 M K N / (stor + 2 K N) for the storage of the real encoding
    w = oracle.magnitude_prune(np.random.default_rng(7).normal(0, 1, (512, 256)).astype(np.float16), 0.5)
    f = oracle.encode(w, 256, 16)
    stor = oracle.unpadded_bytes(f)
    M, K = 512, 256
    for n in (1, 8, 64):
        cr = oracle.compression_ratio(M, K, stor)
        assert oracle.compute_intensity(M, n, cr) == pytest.approx(2 * M * K * n / (stor + 2 * K * n),
                                                                    rel=1e-12)


def test_algorithmic_bytes_dense_closed_form():
    # a fully dense 512 x 64 matrix at tile 256 x 16 with every column active:
    # R = 2 stripes, K = 64 columns, each (stripe, column) moves 4 + 32 + 512 bytes,
    # 2 x 4 = 8 GTiles touched, plus x (2 * 64 B) and y (2 * 512 B) for one token
    w = np.ones((512, 64), dtype=np.float16)
    f = oracle.encode(w, 256, 16)
    x = np.ones((1, 64), dtype=np.float16)
    expect = 2 * 64 * (4 + 32 + 512) + 4 * 8 + 2 * 64 + 2 * 512
    assert oracle.algorithmic_bytes(f, x, -1.0) == expect
    # only column 5 active: 2 stripes x (4 + 32 + 512) + 2 GTiles x 4 + x + y
    x2 = np.zeros((1, 64), dtype=np.float16)
    x2[0, 5] = 1
    assert oracle.algorithmic_bytes(f, x2, 0.5) == 2 * (4 + 32 + 512) + 8 + 2 * 64 + 2 * 512


def test_algorithmic_bytes_hand_case():
    case = _hand_cases()[1]
    f = oracle.encode(_hand_matrix(case), case["tile_m"], case["tile_k"])
    x = np.array([[1.0, 4.0, -2.0]], dtype=np.float16)
    # 2 stripes x 3 real columns x (4 + 8) metadata + padded values:
    # stripe 0: cols 0,1,2 each 8 values; stripe 1: col 0 -> 8, col 1 -> 0, col 2 -> 8
    vals = 2 * (8 + 8 + 8 + 8 + 0 + 8)
    expect = 6 * (4 + 8) + vals + 4 * 4 + 2 * 3 + 2 * 70
    assert oracle.algorithmic_bytes(f, x, -1.0) == expect


def test_useful_flops_counts_products():
    w = oracle.magnitude_prune(synth.weights(20, 10, 2), 0.5)
    x = synth.laplace_activations(2, 10, 3)
    t = oracle.threshold_for(x, 0.5)
    cnt = 0
    wb, act = w.view(np.uint16), oracle.active_mask(x, t)
    for b in range(2):
        for k in range(10):
            for m in range(20):
                if act[b, k] and (wb[m, k] & 0x7FFF):
                    cnt += 1
    assert oracle.useful_flops(w, x, t) == 2 * cnt


# ---------------------------------------------------------------------------
# Batched DP with one column set shared by the batch (the paper leaves
# batched DP to future work, Sec. 4.3 and Sec. 7; the reading built here):
# column k is kept for every token iff the fp32 score sum_b |x[b, k]|
# (tokens in ascending order) exceeds T = fp32(B * t).

@pytest.mark.parametrize("t", [-1.0, 0.0, 6e-8, 0.5, 1.0, 65504.0])
def test_batch_mask_at_batch_one_is_the_token_rule(t):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16).reshape(1, -1)
    assert np.array_equal(oracle.active_mask(x, t, "batch"), oracle.active_mask(x, t, "token"))


def test_batch_mask_hand_worked():
    x = np.array([[1.0, 0.5, -2.0, 0.0], [0.5, 0.25, 0.0, 0.0]], dtype=np.float16)
    # scores 1.5, 0.75, 2.0, 0; T = fp32(2 * 0.7) = 1.4 (to fp32)
    assert oracle.batch_score(x).tolist() == [1.5, 0.75, 2.0, 0.0]
    act = oracle.active_mask(x, 0.7, "batch")
    assert act.tolist() == [[True, False, True, False]] * 2
    xm = oracle.masked_activations(x, 0.7, "batch")
    # token 1 keeps its 0.5 in column 0 although 0.5 < t: the set is shared
    assert xm.astype(np.float64).tolist() == [[1.0, 0.0, -2.0, 0.0], [0.5, 0.0, 0.0, 0.0]]
    # the per-token rule differs: each token keeps only its own entries above t
    assert oracle.masked_activations(x, 0.7, "token").astype(np.float64).tolist() == [[1.0, 0.0, -2.0, 0.0],
                                                                                      [0.0, 0.0, 0.0, 0.0]]


def test_batch_score_is_an_fp32_running_sum():
    # 65504 + 2^-14 is not representable in fp32 near 65504 (spacing 2^-8):
    # the running sum stays 65504, so with T = 65504 the column is inactive,
    # where an exact (or float64) sum would make it active
    x = np.array([[65504.0], [2.0 ** -14]], dtype=np.float16)
    assert oracle.batch_score(x)[0] == np.float32(65504.0)
    assert oracle.batch_threshold(32752.0, 2) == np.float32(65504.0)
    assert not oracle.active_mask(x, 32752.0, "batch")[0, 0]
    # order matters for the rounding: small terms first accumulate
    y = np.array([[2.0 ** -10]] * 3 + [[2048.0]], dtype=np.float16)
    assert oracle.batch_score(y)[0] == np.float32(np.float32(3 * 2.0 ** -10) + np.float32(2048.0))


def test_batch_mask_special_values():
    x = np.array([[np.nan, np.inf, 0.0, 1.0], [1.0, 1.0, 0.0, 1.0]], dtype=np.float16)
    act = oracle.active_mask(x, 0.5, "batch")[0]
    assert act.tolist() == [False, True, False, True]       # NaN never, inf always
    assert oracle.active_mask(x[:, 2:], -1.0, "batch").all()  # negative t keeps every column
    with pytest.raises(ValueError):
        oracle.active_mask(x, 0.5, "mean")


def test_batch_mask_bytes_and_flops_brute_force():
    w = oracle.magnitude_prune(synth.weights(70, 40, 3), 0.5)
    x = synth.laplace_activations(3, 40, 4)
    t = float(oracle.threshold_for(x, 0.6))
    act = oracle.active_mask(x, t, "batch")[0]
    nnz = ((w.view(np.uint16) & 0x7FFF) != 0).sum(axis=0)
    assert oracle.useful_flops(w, x, t, "batch") == 2 * 3 * int(nnz[act].sum())
    f = oracle.encode(w, 64, 8)
    per_col = [sum(4 + 8 + 2 * ((f.column(r, k)[1] + 7) // 8 * 8) for r in range(f.n_stripes)) for k in range(40)]
    touched = len({k // 8 for k in range(40) if act[k]}) * f.n_stripes
    expect = sum(c for c, a in zip(per_col, act) if a) + 4 * touched + 2 * 3 * (40 + 70)
    assert oracle.algorithmic_bytes(f, x, t, "batch") == expect


# ---------------------------------------------------------------------------
# Low-bit Values: round-to-nearest quantization after pruning

def test_rtn_hand_worked():
    """Row 0: max |w| = 0.875, s = 0.875 / 7 = 0.125 exactly; 0.1875 / s = 1.5
    and 0.3125 / s = 2.5 are ties (to even: 2 and 2); 0.0625 / s = 0.5 ties to
    0 and stays stored (code 0); the pruned 0 and -0 are not stored. Row 1
    has nothing stored: scale 0."""
    w = np.array([[0.875, -0.1875, 0.0, 0.3125, 0.0625, -0.0],
                  [0.0, 0.0, 0.0, 0.0, 0.0, 0.0]], dtype=np.float16)
    codes, scales, pattern = oracle.rtn_quantize(w, 4)
    assert scales.dtype == np.float32 and list(scales) == [0.125, 0.0]
    assert codes.tolist() == [[7, -2, 0, 2, 0, 0], [0, 0, 0, 0, 0, 0]]
    assert pattern.tolist() == [[True, True, False, True, True, False], [False] * 6]
    f = oracle.encode_codes(codes, pattern, 64, 2)
    # GTile 0 (columns 0, 1): {7}, {-2}, each padded to 16 codes; GTile 1
    # (columns 2, 3): {}, {2}; GTile 2 (columns 4, 5): {0}, {}
    assert f.tile_offset.tolist() == [0, 32, 48, 64]
    assert f.col_info.tolist() == [1, (16 << 16) | 1, 0, 1, 1, 16 << 16]
    v = f.values.view(np.int8)
    assert v[0] == 7 and v[16] == -2 and v[32] == 2 and v[48] == 0 and len(v) == 64
    assert [int(b) for b in f.bitmap] == [1, 1, 0, 1, 1, 0]


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_rtn_exact_when_representable(bits):
    """Weights that are s * q for integer q with |q| <= qmax and each row
    reaching +-qmax come back exactly."""
    rng = np.random.default_rng(bits)
    qmax = 2 ** (bits - 1) - 1
    q = rng.integers(-qmax, qmax + 1, size=(40, 70))
    q[q == 0] = 1
    q[:, 3] = qmax * np.where(rng.random(40) < 0.5, -1, 1)
    s = 2.0 ** rng.integers(-9, -3, size=40)
    w = (s[:, None] * q).astype(np.float16)
    assert np.array_equal(w.astype(np.float64), s[:, None] * q)  # exactly fp16
    codes, scales, pattern = oracle.rtn_quantize(w, bits)
    assert pattern.all()
    assert np.array_equal(codes, q) and np.array_equal(scales.astype(np.float64), s)
    assert np.array_equal(oracle.rtn_dequantize(codes, scales), w.astype(np.float64))


@pytest.mark.parametrize("bits", [2, 4, 6, 8])
def test_rtn_error_bound_and_range(bits):
    w = oracle.magnitude_prune(synth.weights(120, 300, 40 + bits), 0.6)
    codes, scales, pattern = oracle.rtn_quantize(w, bits)
    qmax = 2 ** (bits - 1) - 1
    w64 = w.astype(np.float64)
    assert np.all(np.abs(codes) <= qmax)
    assert np.all(codes[~pattern] == 0)
    # every row with a stored entry reaches +-qmax at its largest magnitude
    for m in range(w.shape[0]):
        if pattern[m].any():
            k = int(np.argmax(np.where(pattern[m], np.abs(w64[m]), -1)))
            assert abs(int(codes[m, k])) == qmax and np.sign(codes[m, k]) == np.sign(w64[m, k])
    # round to nearest: within half a step, plus the fp32 rounding of the
    # quotient w / s (relative 2^-24 of a quotient of at most qmax steps)
    err = np.abs(oracle.rtn_dequantize(codes, scales) - np.where(pattern, w64, 0))
    assert np.all(err <= scales.astype(np.float64)[:, None] * (0.5 + (qmax + 1) * 2.0 ** -24))
    # the sign of a nonzero code is the weight's
    nz = codes != 0
    assert np.all(np.sign(codes[nz]) == np.sign(w64[nz]))


def test_rtn_matches_scalar_loop():
    """Element-by-element fp32 arithmetic in plain Python (NumPy scalars)."""
    w = oracle.magnitude_prune(synth.weights(9, 23, 77), 0.4)
    codes, scales, pattern = oracle.rtn_quantize(w, 4)
    wb = w.view(np.uint16)
    for m in range(9):
        amax = np.float32(0)
        for k in range(23):
            if wb[m, k] & 0x7FFF:
                amax = max(amax, np.float32(abs(float(w[m, k]))))
        s = np.float32(amax / np.float32(7))
        assert scales[m] == s
        for k in range(23):
            if not (wb[m, k] & 0x7FFF) or s == 0:
                assert codes[m, k] == 0
                continue
            qv = float(np.float32(np.float32(float(w[m, k])) / s))
            r = math.floor(qv)
            frac = qv - r
            q = r + 1 if frac > 0.5 or (frac == 0.5 and r % 2 == 1) else r
            assert codes[m, k] == max(-7, min(7, q)), (m, k)


def test_rtn_rejects_bad_input():
    with pytest.raises(ValueError):
        oracle.rtn_quantize(np.ones((2, 2), dtype=np.float16), 1)
    with pytest.raises(ValueError):
        oracle.rtn_quantize(np.ones((2, 2), dtype=np.float16), 9)
    w = np.ones((2, 2), dtype=np.float16)
    w[0, 1] = np.inf
    with pytest.raises(ValueError):
        oracle.rtn_quantize(w, 4)


@pytest.mark.parametrize("rows,cols,tile", [(300, 200, (128, 16)), (70, 33, (64, 4)), (256, 64, (256, 64)), (5, 1, (64, 1))])
def test_encode_codes_shares_the_pattern_of_encode(rows, cols, tile):
    """Same bitmaps and nonzero counts as the fp16 encoding of the pruned
    matrix; offsets are the running sums of pad16(nnz); decoding gives the
    codes and the pattern back."""
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows + cols), 0.5)
    codes, scales, pattern = oracle.rtn_quantize(w, 4)
    f16 = oracle.encode(w, *tile)
    fq = oracle.encode_codes(codes, pattern, *tile)
    assert np.array_equal(fq.bitmap, f16.bitmap)
    assert np.array_equal(fq.col_info & 0xFFFF, f16.col_info & 0xFFFF)
    nnz = (fq.col_info & 0xFFFF).astype(np.int64).reshape(-1, tile[1])
    pad = (nnz + 15) // 16 * 16
    assert np.array_equal(fq.col_info >> 16, (np.cumsum(pad, axis=1) - pad).reshape(-1).astype(np.uint32))
    assert np.array_equal(fq.tile_offset[1:], np.cumsum(pad.sum(axis=1)).astype(np.uint32))
    assert fq.values.dtype == np.uint8 and len(fq.values) == int(fq.tile_offset[-1])
    c2, p2 = oracle.decode_codes(fq)
    assert np.array_equal(c2, codes) and np.array_equal(p2, pattern)


def test_spmspv_rtn_exact_on_tiny_input():
    """Exact rational arithmetic: y = sum_k s_m q[m,k] xm[k]."""
    w = oracle.magnitude_prune(synth.weights(5, 11, 3), 0.3)
    x = synth.laplace_activations(2, 11, 4)
    t = float(oracle.threshold_for(x, 0.4))
    codes, scales, _ = oracle.rtn_quantize(w, 4)
    y64, s64, _ = oracle.spmspv_rtn(codes, scales, x, t)
    xm = oracle.masked_activations(x, t)
    for b in range(2):
        for m in range(5):
            exact = sum(Fraction(float(scales[m])) * int(codes[m, k]) * Fraction(float(xm[b, k])) for k in range(11))
            mag = sum(abs(Fraction(float(scales[m])) * int(codes[m, k]) * Fraction(float(xm[b, k]))) for k in range(11))
            assert abs(Fraction(y64[b, m]) - exact) <= Fraction(1, 2 ** 40) * (mag + 1)
            assert abs(Fraction(s64[b, m]) - mag) <= Fraction(1, 2 ** 40) * (mag + 1)


def test_algorithmic_bytes_codes_brute():
    w = oracle.magnitude_prune(synth.weights(130, 40, 8), 0.5)
    x = synth.laplace_activations(1, 40, 9)
    t = float(oracle.threshold_for(x, 0.5))
    codes, scales, pattern = oracle.rtn_quantize(w, 4)
    f = oracle.encode_codes(codes, pattern, 64, 8)
    act = oracle.active_mask(x, t).any(axis=0)
    total = 0
    for r in range(f.n_stripes):
        for k in range(40):
            if act[k]:
                nnz = int(pattern[64 * r:64 * (r + 1), k].sum())
                total += 4 + 8 + (nnz + 15) // 16 * 16
        total += 4 * len({k // 8 for k in range(40) if act[k]})
    total += 2 * 40 + 2 * 130 + 4 * 130
    assert oracle.algorithmic_bytes_codes(f, x, t) == total


# ---------------------------------------------------------------------------
# The prefill product (Sec. 4.3: static pruning only, N tokens)

def test_spmm_exact_rational_brute_force():
    from fractions import Fraction
    rng = np.random.default_rng(123)
    for rows, cols, n in [(3, 5, 2), (7, 4, 5), (1, 9, 3), (6, 6, 1)]:
        w = oracle.magnitude_prune(rng.normal(0, 1, (rows, cols)).astype(np.float16), 0.4)
        x = (rng.normal(0, 2, (n, cols))).astype(np.float16)
        y64, s64, y16 = oracle.spmm(w, x)
        for t in range(n):
            for m in range(rows):
                exact = sum(Fraction(float(w[m, k])) * Fraction(float(x[t, k])) for k in range(cols))
                mag = sum(abs(Fraction(float(w[m, k])) * Fraction(float(x[t, k]))) for k in range(cols))
                assert abs(Fraction(y64[t, m]) - exact) <= Fraction(cols, 2 ** 52) * mag
                assert Fraction(s64[t, m]) == mag or abs(Fraction(s64[t, m]) - mag) <= Fraction(cols, 2 ** 52) * mag
    # small integers: every sum is exact, so the float64 result is the integer
    w = rng.integers(-5, 6, (9, 13)).astype(np.float16)
    x = rng.integers(-5, 6, (4, 13)).astype(np.float16)
    y64, _, _ = oracle.spmm(w, x)
    ref = [[sum(int(w[m, k]) * int(x[t, k]) for k in range(13)) for m in range(9)] for t in range(4)]
    assert np.array_equal(y64, np.array(ref, dtype=np.float64))


def test_spmm_special_cases():
    rng = np.random.default_rng(5)
    x = rng.normal(0, 1, (6, 40)).astype(np.float16)
    # identity weights give the tokens back, bit for bit
    y64, _, y16 = oracle.spmm(np.eye(40, dtype=np.float16), x)
    assert np.array_equal(y16.view(np.uint16), x.view(np.uint16))
    # unit tokens pick columns of W
    w = oracle.magnitude_prune(rng.normal(0, 1, (30, 40)).astype(np.float16), 0.5)
    e = np.zeros((3, 40), dtype=np.float16)
    e[0, 7] = e[1, 0] = e[2, 39] = 1.0
    y64, _, _ = oracle.spmm(w, e)
    assert np.array_equal(y64[0], w[:, 7].astype(np.float64))
    assert np.array_equal(y64[1], w[:, 0].astype(np.float64))
    assert np.array_equal(y64[2], w[:, 39].astype(np.float64))
    # all-zero weights: exact zeros; and no threshold drops anything, so it
    # is the decode product with a negative threshold
    assert not oracle.spmm(np.zeros((5, 40), np.float16), x)[0].any()
    assert np.array_equal(oracle.spmm(w, x)[0], oracle.spmspv(w, x, -1.0)[0])


def test_spmm_flops_hand_count():
    w = np.zeros((4, 6), dtype=np.float16)
    w[0, 1] = 1.0
    w[2, 3] = -2.0
    w[3, 5] = np.float16(-0.0)  # -0 is not a nonzero
    w[1, 0] = 3.0
    assert oracle.spmm_flops(w, 10) == (2 * 3 * 10, 2 * 4 * 6 * 10)

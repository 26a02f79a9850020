"""Bit-exact parity of the library's host C++ (Tiled-CBC encoder, magnitude
pruning, threshold calibration, threshold code) against the CPU oracle, on
the same seeded inputs. No GPU involved."""

import numpy as np
import pytest

import oracle
import paper_2607_21985_amd as spdp
import synth


def _same_format(lib_fmt, ref):
    for name in ("tile_offset", "col_info", "bitmap", "values"):
        a, b = lib_fmt[name], getattr(ref, name)
        assert a.dtype == b.dtype and a.shape == b.shape, name
        assert np.array_equal(a, b), name


@pytest.mark.parametrize("rows,cols,tm,tk,sw,seed", [
    (1, 1, 64, 1, 0.0, 1), (64, 16, 64, 16, 0.5, 2), (130, 37, 64, 4, 0.6, 3),
    (200, 33, 128, 8, 0.3, 4), (256, 40, 256, 16, 0.7, 5), (70, 9, 192, 2, 0.9, 6),
    (65, 65, 64, 64, 0.5, 7), (300, 70, 256, 256, 0.2, 8), (513, 1000, 256, 16, 0.5, 9),
    (1024, 1024, 64, 64, 0.5, 101), (777, 300, 128, 1, 0.95, 10), (257, 129, 256, 128, 1.0, 11),
])
def test_encoder_bit_exact_small(rows, cols, tm, tk, sw, seed):
    w = oracle.magnitude_prune(synth.weights(rows, cols, seed), sw)
    _same_format(spdp.encode_host(w, (tm, tk)).format(), oracle.encode(w, tm, tk))


def test_encoder_keeps_signed_zero_and_subnormals_exact():
    w = synth.weights(256, 64, 77)
    wb = w.view(np.uint16).copy()
    wb[::7, ::3] = 0x8000          # -0: not stored
    wb[1::11, 1::5] = 0x0001       # smallest subnormal: stored
    wb[2::13, 2::7] = 0x83FF       # largest negative subnormal: stored
    w2 = wb.view(np.float16)
    _same_format(spdp.encode_host(w2, (256, 16)).format(), oracle.encode(w2, 256, 16))


@pytest.mark.slow
@pytest.mark.parametrize("rows,cols,sw,seed", [(4096, 4096, 0.5, 201), (11008, 4096, 0.6, 301),
                                               (4096, 11008, 0.6, 303)])
def test_encoder_bit_exact_full_size(rows, cols, sw, seed):
    w = spdp.prune_magnitude(synth.weights(rows, cols, seed), sw)
    _same_format(spdp.encode_host(w, (256, 16)).format(), oracle.encode(w, 256, 16))


@pytest.mark.parametrize("shape,sw,seed", [((8, 8), 0.5, 1), ((13, 7), 0.3, 2), ((300, 70), 0.6, 3),
                                           ((64, 64), 0.0, 4), ((9, 9), 1.0, 5), ((1000, 333), 0.77, 6)])
def test_prune_bit_exact(shape, sw, seed):
    w = synth.weights(*shape, seed)
    assert np.array_equal(spdp.prune_magnitude(w, sw).view(np.uint16),
                          oracle.magnitude_prune(w, sw).view(np.uint16))


def test_prune_ties_cross_chunks():
    # many equal magnitudes of both signs, far more than one worker chunk
    rng = np.random.default_rng(5)
    vals = np.array([0.5, -0.5, 0.25, -0.25, 1.0, 0.0, -0.0], dtype=np.float16)
    w = vals[rng.integers(0, vals.size, size=(3000, 3000))]
    for sw in (0.1, 0.37, 0.5, 0.93):
        assert np.array_equal(spdp.prune_magnitude(w, sw).view(np.uint16),
                              oracle.magnitude_prune(w, sw).view(np.uint16))


@pytest.mark.slow
def test_prune_bit_exact_full_size():
    w = synth.weights(4096, 4096, 201)
    assert np.array_equal(spdp.prune_magnitude(w, 0.5).view(np.uint16),
                          oracle.magnitude_prune(w, 0.5).view(np.uint16))


@pytest.mark.parametrize("p", [0.0, 0.1, 0.25, 0.5, 0.7, 0.999, 1.0])
@pytest.mark.parametrize("kind,b,k,seed", [("laplace", 1, 4096, 211), ("laplace", 8, 5120, 411),
                                           ("swiglu", 4, 11008, 313), ("laplace", 1, 7, 3)])
def test_calibrate_matches_oracle(p, kind, b, k, seed):
    x = (synth.laplace_activations if kind == "laplace" else synth.swiglu_activations)(b, k, seed)
    assert np.float32(spdp.calibrate_threshold(x, p)) == oracle.threshold_for(x, p)


def test_calibrate_on_a_calibration_set_matches_oracle():
    """Offline calibration over 300 separately drawn tokens of a layer."""
    for x in (synth.laplace_activations(300, 4096, 211, draw=1),
              synth.swiglu_activations(300, 11008, 313, draw=1)):
        for p in (0.25, 0.5, 0.7):
            assert np.float32(spdp.calibrate_threshold(x, p)) == oracle.calibrated_threshold(x, p)


def test_calibrate_empty_and_ties():
    assert spdp.calibrate_threshold(np.zeros(0, dtype=np.float16), 0.5) == -1.0
    x = np.array([[1.0, -1.0, 1.0, 2.0, 0.0, -0.0, 3.0, 1.0]], dtype=np.float16)
    assert spdp.calibrate_threshold(x, 0.5) == float(oracle.threshold_for(x, 0.5))


def test_threshold_code_decides_like_oracle_for_every_fp16():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16).reshape(1, -1)
    mag = (bits & 0x7FFF).astype(np.int64)
    ts = [-1.0, -0.0, 0.0, 5.96e-8, 6e-8, 1e-7, 6.1e-5, 0.1, 0.5, 0.50006, 1.0, 1.0009765625,
          3.14159, 1000.0, 65504.0, 65519.0, 65520.0, 1e30, float("inf"), float("-inf")]
    rng = np.random.default_rng(0)
    ts += list(rng.uniform(0, 10, 30)) + list(np.float16(rng.uniform(0, 10, 10)).astype(float))
    for t in ts:
        code = spdp.threshold_code(t)
        lib_act = (mag > code) & (mag <= 0x7C00)
        assert np.array_equal(lib_act, oracle.active_mask(x, t)[0]), t


# ---------------------------------------------------------------------------
# Low-bit Values: round-to-nearest codes, one byte each, one scale per row

def _same_rtn(m, w, tile, bits):
    f = m.format()
    codes, scales, pattern = oracle.rtn_quantize(w, bits)
    ref = oracle.encode_codes(codes, pattern, *tile)
    _same_format(f, ref)
    assert f["value_bits"] == bits
    assert f["scales"].dtype == np.float32 and np.array_equal(f["scales"].view(np.uint32), scales.view(np.uint32))
    assert np.array_equal(f["codes"], ref.values.view(np.int8))


@pytest.mark.parametrize("rows,cols,tm,tk,sw,bits,seed", [
    (1, 1, 64, 1, 0.0, 4, 1), (64, 16, 64, 16, 0.5, 4, 2), (130, 37, 64, 4, 0.6, 2, 3),
    (200, 33, 128, 8, 0.3, 8, 4), (256, 40, 256, 16, 0.7, 4, 5), (70, 9, 192, 2, 0.9, 3, 6),
    (513, 1000, 256, 16, 0.5, 4, 9), (777, 300, 128, 1, 0.95, 5, 10), (257, 129, 256, 128, 1.0, 4, 11),
])
def test_rtn_encoder_bit_exact(rows, cols, tm, tk, sw, bits, seed):
    w = oracle.magnitude_prune(synth.weights(rows, cols, seed), sw)
    _same_rtn(spdp.encode_rtn_host(w, (tm, tk), bits), w, (tm, tk), bits)


def test_rtn_encoder_ties_zero_rows_and_subnormals():
    """The hand-worked tie rows of the oracle pins, rows with nothing stored,
    -0 entries and subnormal weights (scales far below the fp16 range)."""
    w = synth.weights(256, 64, 78)
    wb = w.view(np.uint16).copy()
    wb[3] = 0                       # a row with nothing stored: scale 0
    wb[5] = 0x8000                  # -0 everywhere: also nothing stored
    wb[7, :] = 0
    wb[7, :4] = [0x0001, 0x0002, 0x0003, 0x8001]   # subnormals only
    row = np.array([0.875, -0.1875, 0.0, 0.3125, 0.0625, -0.0] * 10 + [0.0] * 4, dtype=np.float16)
    wb[9] = row.view(np.uint16)     # ties at 1.5, 2.5 and 0.5 steps
    w2 = wb.view(np.float16)
    for bits in (4, 8):
        m = spdp.encode_rtn_host(w2, (256, 16), bits)
        _same_rtn(m, w2, (256, 16), bits)
        f = m.format()
        assert f["scales"][3] == 0 and f["scales"][5] == 0
    m = spdp.encode_rtn_host(w2, (256, 16), 4)
    codes, _ = oracle.decode_codes(oracle.encode_codes(*oracle.rtn_quantize(w2, 4)[::2], 256, 16))
    assert codes[9, :6].tolist() == [7, -2, 0, 2, 0, 0]


@pytest.mark.slow
def test_rtn_encoder_bit_exact_full_size():
    w = spdp.prune_magnitude(synth.weights(4096, 4096, 201), 0.5)
    _same_rtn(spdp.encode_rtn_host(w, (256, 16), 4), w, (256, 16), 4)

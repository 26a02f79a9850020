"""bench.py's byte model agrees with the oracle's (CPU only)."""

import numpy as np
import pytest

import bench
import oracle
import paper_2607_21985_amd as spdp
import synth


@pytest.mark.parametrize("rows,cols,tile,sw,p,batch", [
    (1024, 1024, (64, 64), 0.5, 0.5, 1), (700, 900, (256, 16), 0.6, 0.25, 1),
    (300, 1000, (128, 8), 0.5, 0.0, 3), (333, 517, (192, 4), 0.7, 0.5, 8),
])
def test_call_bytes_matches_oracle(rows, cols, tile, sw, p, batch):
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows + cols), sw)
    x = synth.laplace_activations(batch, cols, 5)
    t = float(oracle.threshold_for(x, p))
    f = spdp.encode_host(w, tile).format()
    got, frac = bench.call_bytes(f, bench.token_activity(x, spdp.threshold_code(t)))
    ref = oracle.encode(w, *tile)
    assert got == oracle.algorithmic_bytes(ref, x, t)
    assert frac == pytest.approx(oracle.active_mask(x, t).any(axis=0).mean())


@pytest.mark.parametrize("rows,cols,tile,sw,p,batch,bits", [
    (1024, 1024, (64, 64), 0.5, 0.5, 1, 4), (700, 900, (256, 16), 0.6, 0.25, 1, 4),
    (333, 517, (192, 4), 0.7, 0.5, 8, 8),
])
def test_call_bytes_of_codes_matches_oracle(rows, cols, tile, sw, p, batch, bits):
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows + cols), sw)
    x = synth.laplace_activations(batch, cols, 5)
    t = float(oracle.threshold_for(x, p))
    f = spdp.encode_rtn_host(w, tile, bits).format()
    got, _ = bench.call_bytes(f, bench.token_activity(x, spdp.threshold_code(t)))
    codes, _, pattern = oracle.rtn_quantize(w, bits)
    assert got == oracle.algorithmic_bytes_codes(oracle.encode_codes(codes, pattern, *tile), x, t)


@pytest.mark.parametrize("p,batch,draw_t", [(0.5, 1, 0), (0.25, 4, 1), (0.7, 2, 1), (0.0, 1, 0)])
def test_dropped_fraction_matches_oracle(p, batch, draw_t):
    """Realized dynamic sparsity as the bench reports it, with the threshold
    taken from the input itself (draw 0) or from a calibration set (draw 1)."""
    x = synth.laplace_activations(batch, 2048, 9)
    src = x if draw_t == 0 else synth.laplace_activations(100, 2048, 9, draw=1)
    t = float(oracle.calibrated_threshold(src, p))
    assert bench.dropped_fraction(bench.token_activity(x, spdp.threshold_code(t))) == oracle.realized_sparsity(x, t)


@pytest.mark.parametrize("rows,cols,tile,sw,p,batch", [
    (700, 900, (256, 16), 0.6, 0.25, 1), (300, 1000, (128, 8), 0.5, 0.0, 3),
    (333, 517, (192, 4), 0.7, 0.5, 8), (129, 2000, (64, 64), 0.5, 0.6, 32),
])
def test_call_flops_matches_oracle(rows, cols, tile, sw, p, batch):
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows * cols), sw)
    x = synth.laplace_activations(batch, cols, 11)
    t = float(oracle.threshold_for(x, p))
    f = spdp.encode_host(w, tile).format()
    assert bench.call_flops(f, bench.token_activity(x, spdp.threshold_code(t))) == oracle.useful_flops(w, x, t)


def test_kernel_hash_ignores_comments_and_layout():
    src = "int f(int a) { // one\n  return a + 1; /* two\n three */ }\n"
    assert bench.kernel_source_sha(src) == bench.kernel_source_sha("int f(int a) {\n return a + 1; }")
    assert bench.kernel_source_sha(src) != bench.kernel_source_sha("int f(int a) { return a + 2; }")


@pytest.mark.parametrize("rows,cols,tile,sw,p,batch", [
    (700, 900, (256, 16), 0.6, 0.25, 1), (300, 1000, (128, 8), 0.5, 0.5, 3),
    (333, 517, (192, 4), 0.7, 0.5, 8), (129, 2000, (64, 64), 0.5, 0.6, 32),
])
def test_batch_mask_models_match_oracle(rows, cols, tile, sw, p, batch):
    """The bench's batch-shared activity, bytes and flops against the oracle's."""
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows + 7 * cols), sw)
    x = synth.laplace_activations(batch, cols, 13)
    assert np.array_equal(bench.batch_scores(x), oracle.batch_score(x))
    t = bench.batch_threshold_for(x, p)
    act = bench.batch_activity(x, t)
    assert np.array_equal(act, oracle.active_mask(x, t, "batch"))
    # the own-percentile choice drops about p of the columns
    assert abs((1 - act[0].mean()) - p) <= 2 / cols
    f = spdp.encode_host(w, tile).format()
    got, frac = bench.call_bytes(f, act)
    assert got == oracle.algorithmic_bytes(oracle.encode(w, *tile), x, t, "batch")
    assert bench.call_flops(f, act) == oracle.useful_flops(w, x, t, "batch")

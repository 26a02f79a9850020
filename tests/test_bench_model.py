"""bench.py's byte model agrees with the oracle's (CPU only)."""

import json

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


@pytest.mark.parametrize("rows,cols,tile,sw,p,batch,bits", [
    (700, 900, (256, 16), 0.6, 0.25, 1, 16), (300, 1000, (128, 8), 0.5, 0.5, 3, 16),
    (333, 517, (192, 4), 0.7, 0.5, 8, 16), (520, 700, (256, 16), 0.5, 0.4, 2, 4),
])
def test_line_model_against_brute_force(rows, cols, tile, sw, p, batch, bits):
    """Per-source bytes: the algorithmic parts add up to call_bytes, and the
    128-byte lines are those a scalar walk over every active (stripe,
    column) range touches."""
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows + 3 * cols), sw)
    x = synth.laplace_activations(batch, cols, 17)
    t = float(oracle.threshold_for(x, p))
    f = (spdp.encode_rtn_host(w, tile, bits) if bits < 16 else spdp.encode_host(w, tile)).format()
    act = bench.token_activity(x, spdp.threshold_code(t))
    lm = bench.line_model(f, act)
    total, _ = bench.call_bytes(f, act)
    assert sum(a for a, _ in lm.values()) == total
    assert all(l >= a for a, l in lm.values())
    tm, tk = tile
    R, C = f["n_stripes"], f["n_colblocks"]
    vb, pad = (1, 16) if bits < 16 else (2, 8)
    union = act.any(axis=0)
    vlines, blines = set(), set()
    for r in range(R):
        for k in range(cols):
            if not union[k]:
                continue
            g = r * C + k // tk
            ci = int(f["col_info"][g * tk + k % tk])
            nnz = ci & 0xFFFF
            start = (int(f["tile_offset"][g]) + (ci >> 16)) * vb
            n = -(-nnz // pad) * pad * vb
            vlines.update(range(start // 128, (start + n - 1) // 128 + 1) if n else [])
            boff = (g * tk + k % tk) * (tm // 8)
            blines.add(boff // 128)
    assert lm["values"][1] == 128 * len(vlines)
    assert lm["bitmap"][1] == 128 * len(blines)


def test_profile_summaries_from_raw_counters(tmp_path):
    """--summarize-profiles: kernel time from the trace pass, read bytes by
    request size and write bytes from the two counter passes, checked on a
    made-up raw output directory."""
    d = tmp_path / "raw"
    out = tmp_path / "profiles"
    out.mkdir()
    tag = "wl_decoder"
    pj = {"profile_only": True, "argv": ["--profile-only", "--workload", "wl"], "ms_per_step": 0.02,
          "launches": 4, "launches_per_step": 2, "algorithmic_bytes_per_launch": 10000.0,
          "y_bytes_per_launch": 100.0, "calib_read_bytes": 4096,
          "line_model_per_launch": {"values": [8000, 8192], "bitmap": [1000, 1280], "colinfo": [500, 512],
                                    "tileoffset": [100, 128], "x": [300, 384], "y": [100, 128],
                                    "scales": [0, 0]}}
    for kind in ("trace", "pmcR", "pmcW"):
        (d / f"{kind}_{tag}").mkdir(parents=True)
        (d / f"{kind}_{tag}.log").write_text("noise\n" + json.dumps(dict(pj, argv=pj["argv"] + [kind])) + "\n")
    (d / f"trace_{tag}" / "run_kernel_stats.csv").write_text(
        '"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n'
        '"void spmspv_kernel<1, 4, true, false, false>(LaunchArgs)",4,40000,10000.0,90,9000,11000,1\n')
    hdr = '"Kernel_Name","Counter_Name","Counter_Value"\n'
    rows_r = [("spmspv_kernel<1>", "TCC_EA0_RDREQ_32B_sum", 10), ("spmspv_kernel<1>", "TCC_EA0_RDREQ_64B_sum", 20),
              ("spmspv_kernel<1>", "TCC_EA0_RDREQ_128B_sum", 80), ("spmspv_kernel<1>", "TCC_EA0_RDREQ_sum", 110),
              ("read_kernel", "TCC_EA0_RDREQ_32B_sum", 0), ("read_kernel", "TCC_EA0_RDREQ_64B_sum", 0),
              ("read_kernel", "TCC_EA0_RDREQ_128B_sum", 32), ("read_kernel", "TCC_EA0_RDREQ_sum", 32)]
    rows_w = [("spmspv_kernel<1>", "TCC_EA0_WRREQ_sum", 30), ("spmspv_kernel<1>", "TCC_EA0_WRREQ_64B_sum", 10),
              ("spmspv_kernel<1>", "TCC_BUBBLE_sum", 80), ("spmspv_kernel<1>", "TCC_EA0_RDREQ_DRAM_sum", 100),
              ("read_kernel", "TCC_BUBBLE_sum", 32), ("read_kernel", "TCC_EA0_WRREQ_sum", 1),
              ("read_kernel", "TCC_EA0_WRREQ_64B_sum", 0), ("read_kernel", "TCC_EA0_RDREQ_DRAM_sum", 32)]
    for kind, rows in (("pmcR", rows_r), ("pmcW", rows_w)):
        (d / f"{kind}_{tag}" / "run_counter_collection.csv").write_text(
            hdr + "".join(f'"{k}","{c}",{v}\n' for k, c, v in rows))
    bench.summarize_profiles(str(d), str(out))
    trace = (out / f"spmspv_{tag}_kernel_trace.txt").read_text()
    assert "kernel_us_per_launch: 10.0000" in trace and "1.0 GB/s algorithmic" in trace
    traffic = (out / f"traffic_spmspv_{tag}.txt").read_text()
    rd = 32 * 10 + 64 * 20 + 128 * 80
    wr = 64 * 10 + 32 * 20
    assert f"read bytes by request size = {rd}" in traffic
    assert f"write bytes = {wr}" in traffic
    assert f"hbm_bytes_per_launch: {rd + wr}" in traffic
    assert "= 4096 = 1.0000 x the bytes read" in traffic
    assert f"kernel_sha: {bench.kernel_source_sha()}" in traffic


def test_sq_summary_from_raw_counters(tmp_path):
    """--summarize-profiles: the shader-sequencer passes give the per-word
    instruction mix and the waves' cycle shares, on made-up counters."""
    d = tmp_path / "raw"
    out = tmp_path / "profiles"
    out.mkdir()
    tag = "wl_decoder"
    pj = {"profile_only": True, "argv": ["--profile-only", "--workload", "wl"], "ms_per_step": 0.02,
          "launches": 4, "launches_per_step": 2, "algorithmic_bytes_per_launch": 10000.0,
          "y_bytes_per_launch": 100.0,
          "line_model_per_launch": {"values": [8000, 8192], "bitmap": [800, 1024], "colinfo": [500, 512],
                                    "tileoffset": [100, 128], "x": [300, 384], "y": [100, 128],
                                    "scales": [0, 0]}}
    (d / f"trace_{tag}").mkdir(parents=True)
    (d / f"trace_{tag}.log").write_text(json.dumps(pj) + "\n")
    (d / f"trace_{tag}" / "run_kernel_stats.csv").write_text(
        '"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n'
        '"void spmspv_kernel<8, 4>(LaunchArgs)",4,40000,10000.0,90,9000,11000,1\n')
    values = {"SQ_WAVES": 64, "SQ_WAVE_CYCLES": 1000, "SQ_WAIT_ANY": 400, "SQ_WAIT_INST_ANY": 150,
              "SQ_ACTIVE_INST_ANY": 450, "SQ_LDS_BANK_CONFLICT": 3, "SQ_INSTS_LDS": 150, "SQ_INSTS_VALU": 800,
              "SQ_INSTS_MFMA": 50, "SQ_INSTS_SALU": 600, "SQ_INSTS_SMEM": 20, "SQ_INSTS_BRANCH": 10}
    hdr = '"Kernel_Name","Counter_Name","Counter_Value"\n'
    for i, names in enumerate(bench.PASS_S):
        kind = f"pmcS{i + 1}"
        (d / f"{kind}_{tag}").mkdir()
        (d / f"{kind}_{tag}.log").write_text(json.dumps(dict(pj, argv=pj["argv"] + [kind])) + "\n")
        rows = "".join(f'"spmspv_kernel<8, 4>","{n}",{values.get(n, 7)}\n' for n in names for _ in range(2))
        (d / f"{kind}_{tag}" / "run_counter_collection.csv").write_text(hdr + rows)
    bench.summarize_profiles(str(d), str(out))
    sq = (out / f"sq_spmspv_{tag}.txt").read_text()
    # 800 bitmap bytes = 100 words
    assert "instructions per word: VALU 8.00, SALU 6.00, LDS 1.50, MFMA 0.50, SMEM 0.20, branch 0.10" in sq
    assert "issuing 0.450, waiting (any) 0.400, waiting on dependencies 0.150" in sq
    assert "LDS bank conflicts per LDS instruction: 0.0200" in sq
    assert "rocprofv3 --pmc SQ_WAVES" in sq and f"kernel_sha: {bench.kernel_source_sha()}" in sq

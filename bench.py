"""Benchmark of the decode-time Tiled-CBC spMspV on one MI355X.

Headline workload: the four Llama-7B attention projections (q, k, v, o; each
4096 x 4096 fp16) swept over weight sparsity {50, 60, 70}% and activation
sparsity {0, 25, 50}% at batch 1. One "step" is the whole sweep: 36 spMspV
calls (3 x 3 points x 4 projections), each on its own encoded copy; copies
rotate between steps so that every call streams from HBM rather than from
the 256 MB Infinity Cache.

Calls are issued the way a decoder issues them: projections of one sweep
point that read the same layer input (q, k and v; gate and up) go out as one
grouped launch (spdp_spmspv_many), the others (o, down) as single launches;
--group none issues every product as its own launch, and the JSON line
reports that rate too. By default the steps are replayed from captured HIP
graphs of their launches, a whole rotation cycle of steps per graph, as a
decoder replays a token's pass over all its layers as one graph (the kernel
keeps no host-side state between calls, so replays are exact); --launch
stream issues one host launch per call instead.

Prints one JSON line. ``value`` is the whole step's algorithmic bytes over its
time (GB/s). Algorithmic bytes per call = for every row stripe and every
column active for some token: ColInfo (4 B) + bitmap (tile_m/8 B) + padded
values (2 B x pad8(nnz)); + 4 B per touched GTile (TileOffset); + x and y.
``secondary`` carries the other workloads, each timed the same way: the
1024 x 1024 single layer; the Llama-7B MLP at batch 1/2/4/8; the Llama-13B
decoder layer (seven calls chained) at batch 1/4/16; and a slice of the
Llama-70B layer sweep.

``prefill`` times the prefill product (spdp_spmm, Sec. 4.3) on Llama shapes
at prompt lengths against the dense fp16 matrix peak and F.linear.

``--summarize-profiles DIR`` turns rocprofv3 outputs written under DIR by the
commands it prints into the summaries under profiles/ (no GPU needed).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--launch graph|stream] [--no-secondary]
"""

from __future__ import annotations

import argparse
import csv
import ctypes
import hashlib
import json
import os
import platform
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X published HBM3E bandwidth
# MI355X published fp32 vector peak: 256 CUs x 4 SIMDs x 64 lanes x 4 flops
# per cycle (a two-wide fp32 FMA, or v_dot2_f32_f16's two fp16 products added
# into fp32) x 2.4 GHz
VEC_PEAK_TFLOPS = 157.3
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X published dense fp16 matrix peak
LINE = 128  # bytes per L2 cache line (the granularity the traffic model uses)


def parse(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama7b-attn")
    ap.add_argument("--batch", type=int, default=None, help="override the workload's batch")
    ap.add_argument("--sw", default=None, help="override the weight-sparsity sweep (comma list)")
    ap.add_argument("--p", default=None, help="override the activation-sparsity sweep (comma list)")
    ap.add_argument("--rotation-mb", type=float, default=600.0,
                    help="minimum distinct encoded bytes between two uses of one copy")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the other workloads (single layer, 7B MLP, 13B layer, 70B slice)")
    ap.add_argument("--secondary-steps", type=int, default=12)
    ap.add_argument("--no-prefill", action="store_true", help="skip the prefill products (spdp_spmm)")
    ap.add_argument("--prefill-only", action="store_true",
                    help="run only the prefill products and print them as one JSON line")
    ap.add_argument("--profile-only", action="store_true",
                    help="run warmup + timed steps only (for rocprofv3 runs)")
    ap.add_argument("--calib-read-mib", type=int, default=0,
                    help="after the timed steps, read this many MiB once with the streaming-read "
                         "kernel (a known-size reference for the hardware byte counters)")
    ap.add_argument("--group", choices=("decoder", "none"), default="decoder",
                    help="decoder: products that read one input are one grouped launch; none: one launch each")
    ap.add_argument("--calibration", type=int, default=0, metavar="TOKENS",
                    help="0: each input is thresholded at its own p-th |x| percentile (the workload "
                         "definition); N > 0: each layer's threshold is the p-quantile of |x| over N "
                         "separately drawn calibration tokens of that layer, applied to the inputs "
                         "(offline calibration as in the paper's DP setup)")
    ap.add_argument("--mask", choices=("token", "batch"), default="token",
                    help="token: each token's own active columns (their union is read); batch: one "
                         "column set for the batch, chosen by the batch's mean |x| (batched DP)")
    ap.add_argument("--rtn-bits", type=int, default=0, metavar="B",
                    help="0: fp16 Values; 2..8: the pruned weights quantized to B-bit round-to-nearest "
                         "codes (one byte each, one scale per row; the paper's quantization setup uses 4)")
    ap.add_argument("--launch", choices=("graph", "stream"), default="graph",
                    help="graph: each step is one captured HIP graph of its calls (how a decode "
                         "loop runs them); stream: one host launch per call")
    ap.add_argument("--summarize-profiles", metavar="DIR", default=None,
                    help="write profiles/*.txt from the rocprofv3 outputs under DIR and exit")
    return ap.parse_args(argv)


# ---------------------------------------------------------------------------
# byte model (measurement code: computed from the handle's format arrays)

def token_activity(x16: np.ndarray, code: int) -> np.ndarray:
    """[batch, cols] column activity per token, the kernel's integer rule."""
    mag = (x16.view(np.uint16) & 0x7FFF).astype(np.int64)
    return (mag > code) & (mag <= 0x7C00)


def batch_scores(x16: np.ndarray) -> np.ndarray:
    """Per-column fp32 running sum of |x| over the tokens (ascending)."""
    s = np.zeros(x16.shape[1], dtype=np.float32)
    with np.errstate(invalid="ignore", over="ignore"):
        for b in range(x16.shape[0]):
            s = (s + np.abs(x16[b].astype(np.float32))).astype(np.float32)
    return s


def batch_activity(x16: np.ndarray, t: float) -> np.ndarray:
    """[batch, cols]: one shared column set, score > fp32(batch * fp32(t))."""
    thr = np.float32(np.float64(np.float32(t)) * x16.shape[0])
    with np.errstate(invalid="ignore"):
        shared = batch_scores(x16) > thr
    return np.broadcast_to(shared[None, :], x16.shape).copy()


def batch_threshold_for(x16: np.ndarray, p: float) -> float:
    """Threshold t that drops the fraction p of the columns by batch score
    (the ceil(p K)-th smallest score over the batch size; p = 0 keeps all)."""
    if p <= 0.0:
        return -1.0
    s = np.sort(batch_scores(x16))
    return float(s[int(np.ceil(p * s.size)) - 1]) / x16.shape[0]


def call_bytes(fmt: dict, act: np.ndarray) -> tuple[int, float]:
    """Algorithmic bytes of one call and the fraction of columns it reads,
    given the [batch, cols] activity."""
    R, C, tk, tm = fmt["n_stripes"], fmt["n_colblocks"], fmt["tile_k"], fmt["tile_m"]
    K, M = fmt["cols"], fmt["rows"]
    union = act.any(axis=0)                                       # [K]
    actp = np.zeros(C * tk, dtype=bool)
    actp[:K] = union
    nnz = (fmt["col_info"].reshape(R, C * tk) & 0xFFFF).astype(np.int64)
    if fmt.get("value_bits", 16) < 16:
        # one byte per code, columns padded to 16 codes; one fp32 scale per row
        per_col = 4 + tm // 8 + (nnz + 15) // 16 * 16             # [R, C*tk]
        extra = 4 * M
    else:
        per_col = 4 + tm // 8 + 2 * ((nnz + 7) // 8 * 8)
        extra = 0
    total = int((per_col * actp[None, :]).sum())
    touched = actp.reshape(C, tk).any(axis=1).sum()
    total += 4 * int(touched) * R
    b = act.shape[0]
    total += 2 * b * K + 2 * b * M + extra
    return total, float(union.mean())


def call_flops(fmt: dict, act: np.ndarray) -> int:
    """Useful flops of one call: 2 x the (token, nonzero weight of an active
    column) products, the work the method cannot avoid."""
    R, C, tk = fmt["n_stripes"], fmt["n_colblocks"], fmt["tile_k"]
    K = fmt["cols"]
    nnz_col = (fmt["col_info"].reshape(R, C * tk) & 0xFFFF).astype(np.int64).sum(axis=0)[:K]
    return int(2 * (act * nnz_col[None, :]).sum())


def line_model(fmt: dict, act: np.ndarray) -> dict:
    """Bytes per source of one call: the algorithmic bytes (what the method
    must move) and the whole 128-byte lines that hold them (what an L2 fetch
    of exactly those bytes brings). The kernel reads ColInfo and TileOffset
    of every column (speculatively, with the activations), the bitmaps and
    padded values of the active (stripe, column) pairs, x once and writes y;
    split-K partials are measured, not modelled."""
    R, C, tk, tm = fmt["n_stripes"], fmt["n_colblocks"], fmt["tile_k"], fmt["tile_m"]
    K, M = fmt["cols"], fmt["rows"]
    codes = fmt.get("value_bits", 16) < 16
    vb, pad = (1, 16) if codes else (2, 8)
    union = act.any(axis=0)
    actp = np.zeros(C * tk, dtype=bool)
    actp[:K] = union
    ci = fmt["col_info"].reshape(R, C * tk).astype(np.int64)
    nnz, off = ci & 0xFFFF, ci >> 16
    to = fmt["tile_offset"][:-1].astype(np.int64).reshape(R, C)
    start = (to[:, np.arange(C * tk) // tk] + off) * vb          # [R, C*tk] byte offsets
    length = (nnz + pad - 1) // pad * pad * vb
    sel = actp[None, :] & (length > 0)
    s, e = start[sel], start[sel] + length[sel]                  # in layout order
    first, last = s // LINE, (e - 1) // LINE
    val_lines = int((last - first + 1).sum() - (first[1:] == last[:-1]).sum()) if s.size else 0
    bm_bytes = tm // 8
    pairs = np.broadcast_to(actp[None, :], (R, C * tk))            # (stripe, column) pairs read
    n_pairs = int(pairs.sum())
    g_col = (np.arange(R)[:, None] * (C * tk) + np.arange(C * tk)[None, :])[pairs]
    bm_lines = int(np.unique(g_col * bm_bytes // LINE).size) if g_col.size else 0
    touched = int(actp.reshape(C, tk).any(axis=1).sum()) * R
    b = act.shape[0]

    def lines(n):
        return -(-n // LINE) * LINE

    return {
        "values": (int(length[sel].sum()), val_lines * LINE),
        "bitmap": (n_pairs * bm_bytes, bm_lines * LINE),
        "colinfo": (4 * n_pairs, lines(4 * R * C * tk)),
        "tileoffset": (4 * touched, lines(4 * R * C)),
        "x": (2 * b * K, lines(2 * b * K)),
        "y": (2 * b * M, lines(2 * b * M)),
        "scales": ((4 * M, lines(4 * M)) if codes else (0, 0)),
    }


def dropped_fraction(act: np.ndarray) -> float:
    """Fraction of the entries (all tokens) the rule drops: the realized
    dynamic sparsity."""
    return float(1.0 - act.mean()) if act.size else 0.0


def _code_only(src: str) -> str:
    """Source text without comments and with whitespace collapsed, so that a
    comment edit does not count as a kernel change."""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def kernel_source_sha(src: str | None = None) -> str:
    """Hash of the kernel source's code (comments and layout ignored)."""
    if src is None:
        with open(os.path.join(ROOT, "paper_2607_21985_amd", "csrc", "spdp.hip")) as fh:
            src = fh.read()
    return hashlib.sha256(_code_only(src).encode()).hexdigest()[:16]


def read_traffic(workload: str, group: str):
    """HBM bytes per launch from committed rocprofv3 counter summaries, if they
    were taken on the current kernel source and launch grouping; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_spmspv_{workload}_{group}.txt")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_sha = re.search(r"kernel_sha:\s*(\w+)", text)
    m_b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_sha or not m_b or m_sha.group(1) != kernel_source_sha():
        return None
    return float(m_b.group(1))


# ---------------------------------------------------------------------------

def cpu_baseline(points, mask="token", budget_s=20.0, rtn_bits=0):
    """Time the CPU oracle's masked product on a bounded sample of the same
    calls: ``oracle.masked_activations`` and the float64 product
    ``xm @ W64^T``, with each matrix converted to float64 before the timer
    (the weights are static, their conversion is an offline cost as the
    encoding is; the oracle's error bound S is not part of the product). With
    low-bit Values W64 holds the dequantized weights (quantized before the
    timer too)."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas = [(i.get("internal_api"), i.get("num_threads")) for i in threadpool_info()
                if i.get("user_api") == "blas"]
    except Exception:
        blas = []
    cores = max((n for _, n in blas if n), default=len(os.sched_getaffinity(0)))
    sample = []
    t_total, b_total = 0.0, 0
    t_start = time.perf_counter()
    for pt in points:
        if rtn_bits:
            codes, scales, _ = oracle.rtn_quantize(pt["w"], rtn_bits)
            w64 = oracle.rtn_dequantize(codes, scales)
        else:
            w64 = np.asarray(pt["w"], dtype=np.float16).astype(np.float64)

        def product():
            xm = oracle.masked_activations(pt["x"], pt["t"], mask).astype(np.float64)
            return xm @ w64.T

        product()  # warm-up
        reps = []
        for _ in range(3):
            t0 = time.perf_counter()
            product()
            reps.append(time.perf_counter() - t0)
        del w64
        t_total += float(np.median(reps))
        b_total += pt["bytes"]
        sample.append(pt["label"])
        if time.perf_counter() - t_start > budget_s:
            break
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {
        "value": b_total / t_total / 1e9, "unit": "GB/s", "cores": int(cores), "kind": "oracle",
        "sample": f"{len(sample)} of the step's calls ({', '.join(sample[:4])}{', ...' if len(sample) > 4 else ''}), "
                  f"median of 3 after 1 warm-up: oracle.masked_activations + float64 xm @ W64^T, W64 converted "
                  f"before the timer{' (the dequantized weights)' if rtn_bits else ''}; value = the calls' "
                  f"algorithmic bytes over the oracle's time; cpu={cpu}; blas={blas}",
        "us_per_call": t_total / len(sample) * 1e6,
    }


# ---------------------------------------------------------------------------
# measurement engine

class Bench:
    """Device, stream, timing and graph capture shared by every measurement."""

    def __init__(self, launch: str):
        import torch

        import paper_2607_21985_amd as spdp
        import synth
        self.torch, self.spdp, self.synth = torch, spdp, synth
        self.dev = torch.device("cuda:0")
        torch.cuda.set_device(self.dev)
        self.stream = torch.cuda.current_stream(self.dev)
        self.launch = launch
        self._dense_w = {}

    def sync(self):
        self.torch.cuda.synchronize(self.dev)

    def timed(self, fn, n):
        """ms of n calls of fn(i), HIP events on the launch stream."""
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        for i in range(n):
            fn(i)
        e1.record(self.stream)
        self.sync()
        return e0.elapsed_time(e1)

    def capture(self, fn):
        """fn() captured into a graph on a side stream (replays go to the
        current stream)."""
        torch = self.torch
        s = torch.cuda.Stream(device=self.dev)
        s.wait_stream(torch.cuda.current_stream(self.dev))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            fn()
        torch.cuda.current_stream(self.dev).wait_stream(s)
        return g

    def to_dev(self, a16):
        return self.torch.from_numpy(np.ascontiguousarray(a16).view(np.int16)).view(self.torch.float16).to(self.dev)

    def dense_weight(self, proj):
        key = (proj.rows, proj.cols, proj.w_seed)
        if key not in self._dense_w:
            self._dense_w[key] = proj.weight()
        return self._dense_w[key]


def input_key(pt):
    return (pt["sw"], pt["p"], pt["proj"].x_seed, pt["proj"].x_kind, pt["proj"].cols)


def make_points(B, wl, sw_list, p_list, batch, mask, calibration, pruned):
    """The calls of one step: every (sw, p) point x every projection, each
    with its input and threshold (the input's own p-quantile, or offline
    calibration)."""
    spdp = B.spdp
    xs = {}
    for proj in wl["projections"]:
        key = (proj.x_seed, proj.x_kind, proj.cols)
        if key not in xs:
            xs[key] = proj.activations(batch)
    cal = {}
    if calibration > 0:
        for proj in wl["projections"]:
            key = (proj.x_seed, proj.x_kind, proj.cols)
            if key not in cal:
                cal[key] = proj.activations(calibration, draw=1)
    points = []
    for sw in sw_list:
        for p in p_list:
            for proj in wl["projections"]:
                key = (proj.x_seed, proj.x_kind, proj.cols)
                x = xs[key]
                if mask == "batch":
                    if cal:
                        cs = cal[key]
                        n = cs.shape[0] // batch * batch
                        groups = cs[:n].reshape(-1, batch, cs.shape[1])
                        sc = np.sort(np.concatenate([batch_scores(g) for g in groups]))
                        t = -1.0 if p <= 0 else float(sc[int(np.ceil(p * sc.size)) - 1]) / batch
                    else:
                        t = batch_threshold_for(x, p)
                elif cal:
                    t = spdp.calibrate_threshold(cal[key], p)
                else:
                    t = spdp.calibrate_threshold(x, p)
                points.append({"sw": sw, "p": p, "proj": proj, "x": x, "t": t, "w": pruned[(sw, proj.name)],
                               "label": f"{proj.name}@sw{sw:g}/p{p:g}"})
    return points


def make_units(points, idx, grouped):
    """Launch units: the products of one sweep point that read one input
    form a group (at most 8); every other product is a unit of its own."""
    units, open_ = [], {}
    for j in idx:
        key = input_key(points[j])
        if grouped and key in open_ and len(units[open_[key]]) < 8:
            units[open_[key]].append(j)
        else:
            open_[key] = len(units)
            units.append([j])
    return units


def encode_copies(B, points, tile, rtn_bits, rotation_mb):
    """Encoded copies of every call's matrix, enough of them that at least
    rotation_mb of distinct weights lie between two uses of one copy."""
    spdp = B.spdp
    enc = (lambda w: spdp.encode_rtn(w, tile, rtn_bits)) if rtn_bits else (lambda w: spdp.encode(w, tile))
    t0 = time.perf_counter()
    copy0 = [enc(pt["w"]) for pt in points]
    enc_s = (time.perf_counter() - t0) / len(points)
    fmts = [m.format() for m in copy0]
    dev_bytes = sum(len(f["values"]) * (1 if rtn_bits else 2) for f in fmts)
    n_copies = max(2, int(np.ceil(rotation_mb * 1e6 / max(dev_bytes, 1))) + 1)
    copies = [copy0] + [[enc(pt["w"]) for pt in points] for _ in range(n_copies - 1)]
    return copies, fmts, enc_s


def annotate(points, fmts, mask, spdp):
    for pt, f in zip(points, fmts):
        act = (batch_activity(pt["x"], pt["t"]) if mask == "batch"
               else token_activity(pt["x"], spdp.threshold_code(pt["t"])))
        pt["bytes"], pt["active_frac"] = call_bytes(f, act)
        pt["dropped"] = dropped_fraction(act)
        pt["flops"] = call_flops(f, act)
        pt["lines"] = line_model(f, act)
        pt["rows"], pt["cols"] = f["rows"], f["cols"]


def measure(B, points, copies, batch, mask, grouped, steps, warmup, *, floor=False, single=False,
            per_point=False, stream_rate=False, profile_only=False, n_proj=None, calib_read_mib=0):
    """Time steps of `points` (one call each, decoder grouping) over the
    rotation copies: whole rotation cycles replayed as one graph (or host
    launches). Returns the step time and what was asked for."""
    torch, spdp = B.torch, B.spdp
    n_copies = len(copies)
    X = []
    for _ in range(n_copies):
        by_input, row = {}, []
        for pt in points:
            key = input_key(pt)
            if key not in by_input:
                by_input[key] = B.to_dev(pt["x"])
            row.append(by_input[key])
        X.append(row)
    Y = [[torch.empty((batch, pt["rows"]), dtype=torch.float16, device=B.dev) for pt in points]
         for _ in range(n_copies)]
    for cp in copies:
        for m in cp:
            m.reserve(batch)
    all_idx = list(range(len(points)))
    step_units = make_units(points, all_idx, grouped)
    single_units = make_units(points, all_idx, False)

    def launch_calls(c, units, t_all=None):
        th = (lambda j: points[j]["t"]) if t_all is None else (lambda j: t_all)
        for u in units:
            if len(u) == 1:
                copies[c][u[0]].spmspv_into(X[c][u[0]], th(u[0]), Y[c][u[0]], mask=mask)
            else:
                spdp.spmspv_many([copies[c][j] for j in u], [X[c][j] for j in u],
                                 [th(j) for j in u], [Y[c][j] for j in u], mask=mask)

    graphs = {}

    def cycle_graph(key, units, t_all=None):
        graphs[key] = B.capture(lambda: [launch_calls(c, units, t_all) for c in range(n_copies)])

    def run_steps(first, n, key, units):
        # whole rotation cycles as one graph replay; steps outside a whole
        # cycle as host launches
        i, end = first, first + n
        while i < end:
            if B.launch == "graph" and i % n_copies == 0 and i + n_copies <= end:
                graphs[key].replay()
                i += n_copies
            else:
                launch_calls(i % n_copies, units)
                i += 1

    for i in range(max(1, warmup)):
        launch_calls(i % n_copies, step_units)
    B.sync()
    if B.launch == "graph":
        cycle_graph("step", step_units)
        B.sync()
    # whole cycles only, so that graph mode times graph replays alone
    steps = max(n_copies, steps // n_copies * n_copies) if B.launch == "graph" else steps
    run_steps(0, max(warmup // n_copies, 1) * n_copies, "step", step_units)
    B.sync()
    total_ms = B.timed(lambda _: run_steps(0, steps, "step", step_units), 1)
    res = {"ms_per_step": total_ms / steps, "steps": steps, "n_launch": len(step_units),
           "n_calls": len(points), "n_copies": n_copies,
           "step_bytes": sum(pt["bytes"] for pt in points), "step_flops": sum(pt["flops"] for pt in points)}
    if calib_read_mib:
        peak_read_once(B, calib_read_mib)
    if profile_only:
        res["launches_in_run"] = (max(1, warmup) + max(warmup // n_copies, 1) * n_copies + steps) * len(step_units)
        return res, step_units
    if stream_rate:
        res["stream_ms_per_step"] = B.timed(lambda i: launch_calls(i % n_copies, step_units), steps) / steps
    if floor and B.launch == "graph":
        # the same launches with threshold +inf: no column is active, every
        # step but the value stream runs
        cycle_graph("floor", step_units, float("inf"))
        run_steps(0, n_copies, "floor", step_units)
        B.sync()
        res["floor_ms_per_step"] = B.timed(lambda _: run_steps(0, steps, "floor", step_units), 1) / steps
    if single:
        if B.launch == "graph":
            cycle_graph("single", single_units)
        run_steps(0, n_copies, "single", single_units)
        B.sync()
        res["single_ms_per_step"] = B.timed(lambda _: run_steps(0, steps, "single", single_units), 1) / steps
    if per_point and n_proj:
        # each sweep point's calls back to back (a graph per copy)
        reps = max(2, min(10, steps))
        per_call = np.zeros(len(points))
        for k in range(0, len(points), n_proj):
            units = make_units(points, list(range(k, k + n_proj)), grouped)
            if B.launch == "graph":
                gs = [B.capture(lambda c=c: launch_calls(c, units)) for c in range(n_copies)]
                ms = B.timed(lambda r: gs[r % n_copies].replay(), reps)
                del gs
            else:
                ms = B.timed(lambda r: launch_calls(r % n_copies, units), reps)
            per_call[k:k + n_proj] = ms / (reps * n_proj)
        res["per_call_ms"] = per_call
    graphs.clear()
    return res, step_units


def dense_step_ms(B, projections, batch, steps, warmup, rotation_mb):
    """One fp16 torch F.linear per projection (the dense GEMV/GEMM on the
    same GPU), rotated over copies like the sparse calls."""
    import torch.nn.functional as F
    torch = B.torch
    w_bytes = sum(proj.rows * proj.cols * 2 for proj in projections)
    n_dc = max(2, int(np.ceil(rotation_mb * 1e6 / w_bytes)) + 1)
    dW = {}
    for proj in projections:
        w16 = B.dense_weight(proj)
        for c in range(n_dc):
            dW[(c, proj.name)] = B.to_dev(w16)
    dX = {proj.name: B.to_dev(proj.activations(batch)) for proj in projections}

    def dcalls(c):
        for proj in projections:
            F.linear(dX[proj.name], dW[(c, proj.name)])

    for c in range(n_dc):
        dcalls(c)
    B.sync()
    g = B.capture(lambda: [dcalls(c) for c in range(n_dc)]) if B.launch == "graph" else None
    steps = max(n_dc, steps // n_dc * n_dc)

    def run(n):
        for i in range(0, n, n_dc):
            if g is not None:
                g.replay()
            else:
                for c in range(n_dc):
                    dcalls(c)

    run(max(warmup // n_dc, 1) * n_dc)
    B.sync()
    ms = B.timed(lambda _: run(steps), 1) / steps
    del g, dW, dX
    torch.cuda.empty_cache()
    return ms


_PEAK = None


def peak_lib():
    global _PEAK
    if _PEAK is None:
        path = os.path.join(ROOT, "paper_2607_21985_amd", "libspdp_peak.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} is not built; run `python -m paper_2607_21985_amd.build`")
        L = ctypes.CDLL(path)
        L.spdp_peak_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                     ctypes.c_void_p]
        L.spdp_peak_read.restype = ctypes.c_int
        _PEAK = L
    return _PEAK


def _peak_read(B, buf, off, nbytes, sink, blocks):
    # the current stream: the capture stream while a graph is being captured
    s = B.torch.cuda.current_stream(B.dev)
    st = peak_lib().spdp_peak_read(ctypes.c_void_p(buf.data_ptr() + off), nbytes, ctypes.c_void_p(sink.data_ptr()),
                                   blocks, ctypes.c_void_p(s.cuda_stream))
    if st != 0:
        raise RuntimeError(f"spdp_peak_read failed ({st})")


def peak_read_once(B, mib):
    """One streaming read of `mib` MiB (a known-size reference for counters)."""
    torch = B.torch
    n = mib << 20
    buf = torch.ones(n // 2, dtype=torch.float16, device=B.dev)
    sink = torch.empty(8192, dtype=torch.int32, device=B.dev)
    B.sync()
    _peak_read(B, buf, 0, n, sink, 4096)
    B.sync()
    del buf, sink


def measured_peaks(B, launch_bytes):
    """Streaming-read roof of this GPU (the library's read kernel, best grid,
    1 GiB) and what the same kernel reaches on reads of one launch's
    algorithmic size (consecutive chunks of 1 GiB so that each comes from
    HBM, replayed as one graph like the spMspV launches); plus a 1 GiB torch
    device copy (read + write bytes)."""
    torch = B.torch
    n = 1 << 30
    buf = torch.ones(n // 2, dtype=torch.float16, device=B.dev)
    sink = torch.empty(16384, dtype=torch.int32, device=B.dev)
    best = (0.0, 0)
    for blocks in (1024, 2048, 4096, 8192, 16384):
        _peak_read(B, buf, 0, n, sink, blocks)
        B.sync()
        ms = B.timed(lambda i: _peak_read(B, buf, 0, n, sink, blocks), 5) / 5
        best = max(best, (n / (ms * 1e-3) / 1e9, blocks))
    chunk = max(16, int(launch_bytes) // 16 * 16)
    n_chunks = max(2, n // chunk)
    best_c = (0.0, 0)
    for blocks in (512, 1024, 2048, 4096):
        g = B.capture(lambda: [_peak_read(B, buf, i * chunk, chunk, sink, blocks) for i in range(n_chunks)])
        g.replay()
        B.sync()
        ms = B.timed(lambda i: g.replay(), 3) / (3 * n_chunks)
        best_c = max(best_c, (chunk / (ms * 1e-3) / 1e9, blocks))
        del g
    b_pk = torch.empty_like(buf)
    for _ in range(2):
        b_pk.copy_(buf)
    B.sync()
    copy_ms = B.timed(lambda i: b_pk.copy_(buf), 5) / 5
    del buf, b_pk, sink
    torch.cuda.empty_cache()
    return {"read_gbs": round(best[0], 1), "read_blocks": best[1],
            "read_gbs_at_launch_bytes": round(best_c[0], 1), "launch_bytes": chunk, "launch_blocks": best_c[1],
            "copy_gbs": round(2 * n / (copy_ms * 1e-3) / 1e9, 1),
            "how": "libspdp_peak streaming read (16-byte loads, 4 in flight per lane, best of 1024-16384 "
                   "workgroups) of 1 GiB, mean of 5; the same kernel on consecutive chunks of one launch's "
                   "algorithmic bytes, replayed as one graph; torch copy_ of 1 GiB (read + write bytes)"}


# ---------------------------------------------------------------------------
# one workload, end to end

def prune_all(B, wl, sw_list):
    return {(sw, proj.name): B.spdp.prune_magnitude(B.dense_weight(proj), sw)
            for sw in sw_list for proj in wl["projections"]}


# the library accumulates on the matrix cores above this many tokens (and
# on the vector ALUs up to it): the compute roof follows the form
MATRIX_CORE_MIN_BATCH = 17


def roof(step_bytes, step_flops, ms, batch=1):
    t_hbm = step_bytes / (HBM_PEAK_GBS * 1e9) * 1e3
    mfma = batch >= MATRIX_CORE_MIN_BATCH
    t_alu = step_flops / ((MFMA_F16_PEAK_TFLOPS if mfma else VEC_PEAK_TFLOPS) * 1e12) * 1e3
    return {"frac": round(max(t_hbm, t_alu) / ms, 4),
            "binding": ("mfma" if mfma else "alu") if t_alu > t_hbm else "hbm"}


# the other workloads, each a (name, sw, p, batches) slice measured like the
# headline: decoder grouping, graph replays of rotation cycles, dense fp16
# baseline on the same batches
SECONDARY = [
    ("single-1024", 0.5, 0.5, [1]),
    ("llama7b-mlp", 0.6, 0.5, [1, 2, 4, 8]),
    ("llama13b-layer", 0.7, 0.5, [1, 4, 8, 16]),
    ("llama70b-layer", 0.7, 0.5, [1, 8, 32]),
    ("llama70b-layer", 0.5, 0.0, [1, 8, 32]),
    ("llama70b-layer", 0.8, 0.7, [1]),
    ("llama70b-tp8", 0.7, 0.5, [1, 8]),
]


def secondary(B, args):
    out = []
    dense_cache = {}
    for name, sw, p, batches in SECONDARY:
        wl = B.synth.workload(name)
        pruned = prune_all(B, wl, [sw])
        pts0 = make_points(B, wl, [sw], [p], batches[0], "token", 0, pruned)
        copies, fmts, _ = encode_copies(B, pts0, wl["tile"], 0, args.rotation_mb)
        for b in batches:
            pts = make_points(B, wl, [sw], [p], b, "token", 0, pruned)
            annotate(pts, fmts, "token", B.spdp)
            r, _ = measure(B, pts, copies, b, "token", True, args.secondary_steps, 3)
            ms = r["ms_per_step"]
            if (name, b) not in dense_cache and not args.no_dense:
                dense_cache[(name, b)] = dense_step_ms(B, wl["projections"], b, args.secondary_steps, 3,
                                                       args.rotation_mb)
            d = dense_cache.get((name, b))
            e = {"workload": name, "sw": sw, "p": p, "batch": b,
                 "calls": r["n_calls"], "launches": r["n_launch"],
                 "us_per_product": round(ms * 1e3 / r["n_calls"], 3),
                 "gbs": round(r["step_bytes"] / (ms * 1e-3) / 1e9, 1),
                 "pct_of_hbm_peak": round(100 * r["step_bytes"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
                 "roofline": roof(r["step_bytes"], r["step_flops"], ms, b),
                 "active_frac": round(float(np.mean([pt["active_frac"] for pt in pts])), 4),
                 "speedup_vs_dense": round(d / ms, 3) if d else None,
                 "dense_us_per_product": round(d * 1e3 / r["n_calls"], 3) if d else None}
            print(f"[bench] secondary {json.dumps(e)}", file=sys.stderr, flush=True)
            out.append(e)
        for cp in copies:
            for m in cp:
                m.close()
        del copies
        B.torch.cuda.empty_cache()
    return out


# prefill products (Sec. 4.3): (workload, projection, sw, tokens)
PREFILL = [
    ("llama7b-attn", "q", 0.5, 512),
    ("llama7b-attn", "q", 0.5, 2048),
    ("llama7b-mlp", "gate", 0.6, 2048),
    ("llama7b-mlp", "down", 0.6, 2048),
    ("llama70b-layer", "gate", 0.7, 1024),
    ("llama70b-layer", "gate", 0.7, 256),   # a serving-size prefill chunk
]


def prefill(B, args, steps=10):
    """The prefill product spdp_spmm on Llama shapes at prompt lengths:
    MFMA work executed (every 256 x 16 tile expanded, the token count
    rounded up to the 128-token tile) against the dense fp16 matrix peak,
    useful flops (2 x nonzeros x tokens), and the dense fp16 F.linear on the
    same shapes. Two encoded copies alternate so that consecutive calls read
    different weights."""
    import torch.nn.functional as F
    torch, spdp, synth = B.torch, B.spdp, B.synth
    out = []
    for name, pname, sw, n in PREFILL:
        proj = next(p for p in synth.workload(name)["projections"] if p.name == pname)
        w16 = B.dense_weight(proj)
        w = spdp.prune_magnitude(w16, sw)
        mats = [spdp.encode(w, (256, 16)) for _ in range(2)]
        X = B.to_dev(proj.activations(n, draw=2))
        Ys = [torch.empty((n, proj.rows), dtype=torch.float16, device=B.dev) for _ in range(2)]
        Wd = [B.to_dev(w16) for _ in range(2)]
        for i in range(2):
            # eager calls first: the split-K workspace and the dense library's
            # state are set up outside the captures
            mats[i].spmm_into(X, Ys[i])
            F.linear(X, Wd[i])
        B.sync()
        g = B.capture(lambda: [mats[i % 2].spmm_into(X, Ys[i % 2]) for i in range(steps)])
        g.replay()
        B.sync()
        ms = B.timed(lambda _: g.replay(), 3) / (3 * steps)
        del g
        gd = B.capture(lambda: [F.linear(X, Wd[i % 2]) for i in range(steps)])
        gd.replay()
        B.sync()
        dms = B.timed(lambda _: gd.replay(), 3) / (3 * steps)
        del gd, Wd
        f = mats[0].format()
        nnz = int(((f["col_info"] & 0xFFFF).astype(np.int64)).sum())
        executed = 2.0 * f["n_stripes"] * 256 * f["n_colblocks"] * 16 * (-(-n // 128) * 128)
        useful = 2.0 * nnz * n
        dense_fl = 2.0 * proj.rows * proj.cols * n
        e = {"workload": name, "projection": f"{pname} {proj.rows}x{proj.cols}", "sw": sw, "tokens": n,
             "us_per_call": round(ms * 1e3, 3),
             "mfma_tflops": round(executed / (ms * 1e-3) / 1e12, 1),
             "useful_tflops": round(useful / (ms * 1e-3) / 1e12, 1),
             "roofline": {"bound": "mfma", "achieved": round(executed / (ms * 1e-3) / 1e12, 1),
                          "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                          "frac": round(executed / (ms * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS, 4)},
             "dense_us_per_call": round(dms * 1e3, 3),
             "dense_tflops": round(dense_fl / (dms * 1e-3) / 1e12, 1),
             "speedup_vs_dense": round(dms / ms, 3)}
        print(f"[bench] prefill {json.dumps(e)}", file=sys.stderr, flush=True)
        out.append(e)
        for m in mats:
            m.close()
        del X, Ys
        torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.summarize_profiles:
        summarize_profiles(args.summarize_profiles)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU: --gpus above 1 is not supported"}))
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no ROCm GPU visible"}))
        sys.exit(2)
    B = Bench(args.launch)
    spdp, synth = B.spdp, B.synth
    if args.prefill_only:
        print(json.dumps({"prefill_only": True, "prefill": prefill(B, args)}), flush=True)
        return
    wl = synth.workload(args.workload)
    tile = wl["tile"]
    batch = args.batch if args.batch is not None else wl["batch"][0]
    sw_list = [float(v) for v in args.sw.split(",")] if args.sw else wl["weight_sparsity"]
    p_list = [float(v) for v in args.p.split(",")] if args.p else wl["act_sparsity"]

    t_prep = time.perf_counter()
    pruned = prune_all(B, wl, sw_list)
    points = make_points(B, wl, sw_list, p_list, batch, args.mask, args.calibration, pruned)
    copies, fmts, enc_s = encode_copies(B, points, tile, args.rtn_bits, args.rotation_mb)
    annotate(points, fmts, args.mask, spdp)
    prep_s = time.perf_counter() - t_prep
    grouped = args.group == "decoder"
    n_proj = len(wl["projections"])

    if args.profile_only:
        r, units = measure(B, points, copies, batch, args.mask, grouped, args.steps, args.warmup,
                           profile_only=True, calib_read_mib=args.calib_read_mib)
        lines = {k: [0, 0] for k in points[0]["lines"]}
        for pt in points:
            for k, (a, l) in pt["lines"].items():
                lines[k][0] += a
                lines[k][1] += l
        n = len(units)
        print(json.dumps({"profile_only": True, "argv": sys.argv[1:], "launch": args.launch, "group": args.group,
                          "ms_per_step": r["ms_per_step"], "launches": r["launches_in_run"],
                          "launches_per_step": n,
                          "algorithmic_bytes_per_launch": r["step_bytes"] / n,
                          "y_bytes_per_launch": lines["y"][0] / n,
                          "line_model_per_launch": {k: [a / n, l / n] for k, (a, l) in lines.items()},
                          "calib_read_bytes": args.calib_read_mib << 20}), flush=True)
        return

    r, step_units = measure(B, points, copies, batch, args.mask, grouped, args.steps, args.warmup,
                            floor=True, single=True, per_point=True, stream_rate=True, n_proj=n_proj)
    # "hot": one sweep point's launches replayed with no rotation, so that its
    # matrices stay in the 256 MB Infinity Cache (a labelled secondary figure;
    # the headline rotates copies through HBM)
    hot = None
    hk = [i for i, pt in enumerate(points) if pt["sw"] == sw_list[0] and pt["p"] == p_list[-1]]
    if hk:
        hp = [points[i] for i in hk]
        # the same matrices 16 times per graph, so that the graph's start-up
        # is spread over as many launches as in the headline's cycles
        rh, _ = measure(B, hp, [[copies[0][i] for i in hk]] * 16, batch, args.mask, grouped, args.steps,
                        args.warmup)
        hot_bytes = sum(pt["bytes"] for pt in hp)
        hot = {"point": f"sw {sw_list[0]} / p {p_list[-1]}",
               "us_per_call": round(rh["ms_per_step"] * 1e3 / len(hp), 3),
               "gbs": round(hot_bytes / (rh["ms_per_step"] * 1e-3) / 1e9, 1),
               "how": "the point's calls (decoder grouping), 16 steps per graph replay, no rotation: their "
                      f"{hot_bytes / 1e6:.1f} MB of algorithmic bytes stay in the 256 MB Infinity Cache; "
                      "the headline rotates encoded copies through HBM"}
    for cp in copies:
        for m in cp:
            m.close()
    del copies
    torch.cuda.empty_cache()
    ms_per_step = r["ms_per_step"]
    step_bytes, step_flops = r["step_bytes"], r["step_flops"]
    n_launch = r["n_launch"]
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    t_hbm_us = step_bytes / (HBM_PEAK_GBS * 1e9) * 1e6
    t_alu_us = step_flops / (VEC_PEAK_TFLOPS * 1e12) * 1e6
    alu_bound = t_alu_us > t_hbm_us

    peaks = measured_peaks(B, step_bytes / n_launch)
    dense_ms = None if args.no_dense else dense_step_ms(B, wl["projections"], batch, args.steps, args.warmup,
                                                        args.rotation_mb)
    dense = None
    if dense_ms is not None:
        dense = {"us_per_call": dense_ms * 1e3 / n_proj,
                 "gbs": sum(proj.rows * proj.cols * 2 + 2 * batch * (proj.rows + proj.cols)
                            for proj in wl["projections"]) / (dense_ms * 1e-3) / 1e9}

    pts_out = []
    per_call = r["per_call_ms"]
    for k in range(0, len(points), n_proj):
        grp = points[k:k + n_proj]
        us = float(per_call[k:k + n_proj].sum() * 1e3 / n_proj)
        byts = sum(pt["bytes"] for pt in grp)
        d = {"sw": grp[0]["sw"], "p": grp[0]["p"], "us_per_call": round(us, 3),
             "gbs": round(byts / (us * n_proj * 1e-6) / 1e9, 1),
             "active_frac": round(float(np.mean([pt["active_frac"] for pt in grp])), 4),
             "act_sparsity_realized": round(float(np.mean([pt["dropped"] for pt in grp])), 4),
             "bytes_per_call": int(byts / n_proj)}
        if dense:
            d["speedup_vs_dense"] = round(dense["us_per_call"] / us, 3)
        pts_out.append(d)

    sec = None if args.no_secondary else secondary(B, args)
    pre = None if args.no_prefill else prefill(B, args)
    cpu = None if args.no_cpu_baseline else cpu_baseline(points, args.mask, rtn_bits=args.rtn_bits)
    traffic = None if args.rtn_bits else read_traffic(args.workload, args.group)
    us_per_call = ms_per_step * 1e3 / len(points)
    kernel_us = ms_per_step * 1e3 / n_launch
    out = {
        "metric": "spMspV µs/call + achieved HBM GB/s (% of peak), Llama-7B shapes, batch 1",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": r["steps"],
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded N(0,0.02) x per-column log-normal weights, Laplace+outlier activations)",
        "config": {
            "workload": args.workload,
            "shapes": sorted({f"{pt['rows']}x{pt['cols']}" for pt in points}),
            "projections": [proj.name for proj in wl["projections"]],
            "weight_sparsity": sw_list, "act_sparsity": p_list,
            "batch": batch, "tile": list(tile), "calls_per_step": len(points),
            "launches_per_step": n_launch, "grouping": args.group,
            "rotation_copies": r["n_copies"], "accumulate": "f32",
            "values": (f"rtn{args.rtn_bits}: {args.rtn_bits}-bit round-to-nearest codes, one byte each, one "
                       "fp32 scale per row" if args.rtn_bits else "fp16"),
            "mask": args.mask,
            "threshold": ({"rule": "offline calibration", "calibration_tokens": args.calibration,
                           "how": "p-quantile of |x| over separately drawn tokens of each layer input"}
                          if args.calibration > 0 else
                          {"rule": "own percentile", "how": "p-quantile of |x| over the input itself"}),
        },
        "us_per_call": round(us_per_call, 3),
        "us_per_call_ungrouped": round(r["single_ms_per_step"] * 1e3 / len(points), 3),
        "gbs_ungrouped": round(step_bytes / (r["single_ms_per_step"] * 1e-3) / 1e9, 2),
        "us_per_call_stream_launch": round(r["stream_ms_per_step"] * 1e3 / len(points), 3),
        "launch": args.launch,
        "pct_of_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "measured_peaks": peaks,
        "pct_of_measured_read_peak": round(100 * value / peaks["read_gbs"], 2),
        "pct_of_read_at_launch_bytes": round(100 * value / peaks["read_gbs_at_launch_bytes"], 2),
        "roofline": {
            **({"bound": "alu", "achieved": round(step_flops / (ms_per_step * 1e-3) / 1e12, 3),
                "peak": VEC_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(t_alu_us / (ms_per_step * 1e3), 4)} if alu_bound else
               {"bound": "hbm", "achieved": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 2),
                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}),
            "traffic": traffic,
            "t_roof_us_per_step": {"hbm": round(t_hbm_us, 3), "alu": round(t_alu_us, 3),
                                   "binding": "alu" if alu_bound else "hbm"},
            "useful_flops_per_launch": int(step_flops / n_launch),
            "kernel": "spmspv_kernel",
            "kernel_us_per_launch": round(kernel_us, 3),
            "duration_source": "HIP events around the timed steps on the launch stream "
                               f"({'one captured graph per rotation cycle of steps' if args.launch == 'graph' else 'back-to-back launches'})",
            "algorithmic_bytes_per_launch": int(step_bytes / n_launch),
        },
        "hot": hot,
        "latency_floor": ({"us_per_launch": round(r["floor_ms_per_step"] * 1e3 / n_launch, 3),
                           "frac_of_launch": round(r["floor_ms_per_step"] / ms_per_step, 4),
                           "how": "the same launches with threshold +inf: no column active, every step "
                                  "but the value stream runs"} if "floor_ms_per_step" in r else None),
        "cpu_baseline": cpu,
        "dense_gemv": dense,
        "speedup_vs_dense": round(dense["us_per_call"] / us_per_call, 3) if dense else None,
        "points": pts_out,
        "secondary": sec,
        "prefill": pre,
        "prep_s": round(prep_s, 2),
        "encode_s_per_matrix": round(enc_s, 4),
        "host": platform.node(),
    }
    print(json.dumps(out), flush=True)


# ---------------------------------------------------------------------------
# rocprofv3 summaries (profiles/*.txt) from the raw outputs of the commands
# below, written under DIR on the GPU machine:
#   rocprofv3 --kernel-trace --stats --output-format csv -d DIR/trace_TAG -o run -- \
#       python3 bench.py --profile-only ARGS > DIR/trace_TAG.log
#   rocprofv3 --pmc PASS_R --output-format csv -d DIR/pmcR_TAG -o run -- \
#       python3 bench.py --profile-only --calib-read-mib 256 ARGS > DIR/pmcR_TAG.log
#   rocprofv3 --pmc PASS_W ... -d DIR/pmcW_TAG ... > DIR/pmcW_TAG.log
# Read bytes are counted by request size (32, 64 and 128-byte requests from
# the L2 to memory), write bytes by the 32/64-byte write requests; the
# streaming-read kernel of known size checks those formulas.

PASS_R = ["TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum", "TCC_EA0_RDREQ_128B_sum", "TCC_EA0_RDREQ_sum"]
PASS_W = ["TCC_EA0_WRREQ_sum", "TCC_EA0_WRREQ_64B_sum", "TCC_BUBBLE_sum", "TCC_EA0_RDREQ_DRAM_sum"]
# shader-sequencer passes: where the waves' cycles go, and the instruction mix
PASS_S = [["SQ_WAVES", "SQ_BUSY_CYCLES", "SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY",
           "SQ_ACTIVE_INST_ANY", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "GRBM_GUI_ACTIVE"],
          ["SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_SCA", "SQ_WAIT_INST_LDS",
           "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_LDS", "SQ_INSTS_VALU", "SQ_INSTS_MFMA", "GRBM_GUI_ACTIVE"],
          ["SQ_INSTS_SALU", "SQ_INSTS_SMEM", "SQ_INSTS_BRANCH", "SQ_ACTIVE_INST_MISC", "GRBM_GUI_ACTIVE"]]


def _profile_line(path):
    with open(path) as fh:
        for line in fh:
            if line.startswith("{") and "profile_only" in line:
                return json.loads(line)
    raise ValueError(f"{path}: no --profile-only line")


def _counters(path):
    """{counter: ([per spmspv dispatch], [per read-kernel dispatch])}."""
    out = {}
    with open(path) as fh:
        for row in csv.DictReader(fh):
            name = row["Counter_Name"]
            k = row["Kernel_Name"]
            v = float(row["Counter_Value"])
            sp, rd = out.setdefault(name, ([], []))
            if "spmspv_kernel" in k or "spmspv_mm_kernel" in k:
                sp.append(v)
            elif "read_kernel" in k:
                rd.append(v)
    return out


def _cmd(kind, d, tag, pj, extra=""):
    prof = {"trace": "--kernel-trace --stats", "pmcR": "--pmc " + " ".join(PASS_R),
            "pmcW": "--pmc " + " ".join(PASS_W)}
    prof.update({f"pmcS{i + 1}": "--pmc " + " ".join(p) for i, p in enumerate(PASS_S)})
    prof = prof[kind]
    return (f"rocprofv3 {prof} --output-format csv -d {d}/{kind}_{tag} -o run -- python3 bench.py "
            + " ".join(pj["argv"]) + f" > {d}/{kind}_{tag}.log")


def summarize_prefill(d, prof_dir):
    """profiles/spmm_prefill_kernel_trace.txt: the prefill kernels' durations
    under rocprofv3 next to what bench.py --prefill-only timed in the same run."""
    with open(os.path.join(d, "trace_prefill.log")) as fh:
        pj = next(json.loads(l) for l in fh if l.startswith("{") and "prefill_only" in l)
    rows = list(csv.DictReader(open(os.path.join(d, "trace_prefill", "run_kernel_stats.csv"))))
    out = ["# spdp_spmm (prefill) kernels", "", "command (GPU box, repository root, TMPDIR=/tmp):",
           f"  rocprofv3 --kernel-trace --stats --output-format csv -d {d}/trace_prefill -o run -- "
           f"python3 bench.py --prefill-only > {d}/trace_prefill.log", "",
           "kernel_stats (durations in ns):", "Name | Calls | AverageNs | MinNs | MaxNs"]
    for r in rows:
        out.append(f"{r['Name'].replace('(anonymous namespace)::', '')[:70]} | {r['Calls']} | "
                   f"{float(r['AverageNs']):.1f} | {r['MinNs']} | {r['MaxNs']}")
    out += ["", "bench.py --prefill-only (same run; graph replays, two encoded copies alternating):",
            "projection | tokens | us per call | MFMA TFLOP/s executed | frac of 2500 | dense us | vs dense"]
    for e in pj["prefill"]:
        out.append(f"{e['projection']} | {e['tokens']} | {e['us_per_call']} | {e['mfma_tflops']} | "
                   f"{e['roofline']['frac']} | {e['dense_us_per_call']} | {e['speedup_vs_dense']}")
    out += [f"spmm_sha: {kernel_source_sha(open(os.path.join(ROOT, 'paper_2607_21985_amd', 'csrc', 'spmm.hip')).read())}",
            ""]
    with open(os.path.join(prof_dir, "spmm_prefill_kernel_trace.txt"), "w") as fh:
        fh.write("\n".join(out))
    print("\n".join(out))


def summarize_sq(d, tag, pj, prof_dir, sha):
    """profiles/sq_spmspv_<tag>.txt from three shader-sequencer counter passes:
    the mean per spMspV dispatch of each counter, the instruction mix per
    64-row bitmap word decoded (the algorithmic bitmap bytes / 8), and the
    fractions of the waves' cycles spent issuing and waiting."""
    cs, cmds = {}, []
    for i in range(len(PASS_S)):
        kind = f"pmcS{i + 1}"
        cs.update(_counters(os.path.join(d, f"{kind}_{tag}", "run_counter_collection.csv")))
        cmds.append("  " + _cmd(kind, d, tag, _profile_line(os.path.join(d, f"{kind}_{tag}.log"))))

    def mean(name):
        v = cs.get(name, ([], []))[0]
        return sum(v) / len(v) if v else float("nan")

    words = pj["line_model_per_launch"]["bitmap"][0] / 8.0
    wc = mean("SQ_WAVE_CYCLES")
    out = [f"# shader-sequencer counters of spmspv_kernel: {tag}", "",
           "commands (GPU box, repository root, TMPDIR=/tmp), one counter pass per run:"] + cmds + [
           "", f"mean per spMspV dispatch ({len(cs['SQ_WAVES'][0])} dispatches in the first pass):"]
    for p in PASS_S:
        for name in p:
            if name != "GRBM_GUI_ACTIVE" or p is PASS_S[0]:
                out.append(f"  {name:26s} {mean(name):16.0f}")
    out += ["", f"64-row bitmap words decoded per launch (algorithmic bitmap bytes / 8): {words:.0f}",
            "instructions per word: " + ", ".join(
                f"{k} {mean(n) / words:.2f}" for k, n in (("VALU", "SQ_INSTS_VALU"), ("SALU", "SQ_INSTS_SALU"),
                                                          ("LDS", "SQ_INSTS_LDS"), ("MFMA", "SQ_INSTS_MFMA"),
                                                          ("SMEM", "SQ_INSTS_SMEM"), ("branch", "SQ_INSTS_BRANCH"))),
            "share of the waves' cycles: " + ", ".join(
                f"{k} {mean(n) / wc:.3f}" for k, n in (("issuing", "SQ_ACTIVE_INST_ANY"),
                                                       ("waiting (any)", "SQ_WAIT_ANY"),
                                                       ("waiting on dependencies", "SQ_WAIT_INST_ANY"))),
            f"LDS bank conflicts per LDS instruction: "
            f"{mean('SQ_LDS_BANK_CONFLICT') / max(mean('SQ_INSTS_LDS'), 1):.4f}",
            f"kernel_sha: {sha}", ""]
    with open(os.path.join(prof_dir, f"sq_spmspv_{tag}.txt"), "w") as fh:
        fh.write("\n".join(out))
    print("\n".join(out))


def summarize_profiles(d, prof_dir=None):
    sha = kernel_source_sha()
    prof_dir = prof_dir or os.path.join(ROOT, "profiles")
    if os.path.isdir(os.path.join(d, "trace_prefill")):
        summarize_prefill(d, prof_dir)
    tags = sorted(n[len("trace_"):] for n in os.listdir(d)
                  if n.startswith("trace_") and os.path.isdir(os.path.join(d, n)) and n != "trace_prefill")
    for tag in tags:
        pj = _profile_line(os.path.join(d, f"trace_{tag}.log"))
        rows = list(csv.DictReader(open(os.path.join(d, f"trace_{tag}", "run_kernel_stats.csv"))))
        out = [f"# spmspv_kernel: {tag}", "", "command (GPU box, repository root, TMPDIR=/tmp):",
               "  " + _cmd("trace", d, tag, pj), "",
               "kernel_stats (durations in ns):", "Name | Calls | AverageNs | MinNs | MaxNs"]
        for r in rows:
            out.append(f"{r['Name'].replace('(anonymous namespace)::', '')[:70]} | {r['Calls']} | "
                       f"{float(r['AverageNs']):.1f} | {r['MinNs']} | {r['MaxNs']}")
        kr = [r for r in rows if "spmspv_kernel" in r["Name"] or "spmspv_mm_kernel" in r["Name"]]
        calls = sum(int(r["Calls"]) for r in kr)
        avg = sum(int(r["Calls"]) * float(r["AverageNs"]) for r in kr) / max(calls, 1)
        alg = pj["algorithmic_bytes_per_launch"]
        out += ["", f"all spMspV kernel variants: {calls} launches, launch-weighted average {avg:.1f} ns",
                f"  -> {alg / avg:.1f} GB/s algorithmic ({100 * alg / avg / HBM_PEAK_GBS:.2f} % of "
                f"{HBM_PEAK_GBS:.0f} GB/s)",
                "", "bench.py --profile-only (same command) reported:",
                f"  ms_per_step = {pj['ms_per_step']:.5f} ({pj['launches_per_step']} launches per step: "
                f"{pj['ms_per_step'] * 1e6 / pj['launches_per_step']:.1f} ns per launch)",
                f"  launches = {pj['launches']}", f"  algorithmic_bytes_per_launch = {alg:.0f}",
                f"kernel_us_per_launch: {avg / 1e3:.4f}", f"kernel_sha: {sha}", ""]
        with open(os.path.join(prof_dir, f"spmspv_{tag}_kernel_trace.txt"), "w") as fh:
            fh.write("\n".join(out))
        print("\n".join(out))

        if all(os.path.isdir(os.path.join(d, f"pmcS{i + 1}_{tag}")) for i in range(len(PASS_S))):
            summarize_sq(d, tag, pj, prof_dir, sha)

        pr, pw = os.path.join(d, f"pmcR_{tag}"), os.path.join(d, f"pmcW_{tag}")
        if not (os.path.isdir(pr) and os.path.isdir(pw)):
            continue
        cr = _counters(os.path.join(pr, "run_counter_collection.csv"))
        cw = _counters(os.path.join(pw, "run_counter_collection.csv"))
        pjr = _profile_line(os.path.join(d, f"pmcR_{tag}.log"))

        def mean(c, name, which=0):
            v = c[name][which]
            return sum(v) / len(v) if v else float("nan")

        n32, n64, n128, nall = (mean(cr, c) for c in PASS_R)
        nw, nw64, nbub, ndram = (mean(cw, c) for c in PASS_W)
        rd = 32 * n32 + 64 * n64 + 128 * n128
        wr = 64 * nw64 + 32 * (nw - nw64)
        fetch_formula = (nbub * 128 + (nall - nbub - n32) * 64 + n32 * 32)
        # the streaming read of known size
        c32, c64, c128, call_ = (mean(cr, c, 1) for c in PASS_R)
        crd = 32 * c32 + 64 * c64 + 128 * c128
        cbub = mean(cw, "TCC_BUBBLE_sum", 1)
        cfetch = (cbub * 128 + (call_ - cbub - c32) * 64 + c32 * 32)
        ref = pjr["calib_read_bytes"]
        y = pj["y_bytes_per_launch"]
        lm = pj["line_model_per_launch"]
        line_rd = sum(l for k, (a, l) in lm.items() if k != "y")
        alg_rd = sum(a for k, (a, l) in lm.items() if k != "y")
        partial_w = max(wr - y, 0.0)
        out = [f"# HBM traffic of spmspv_kernel: {tag}", "",
               "commands (GPU box, repository root, TMPDIR=/tmp), one counter pass per run:",
               "  " + _cmd("pmcR", d, tag, pjr), "  " + _cmd("pmcW", d, tag, _profile_line(os.path.join(d, f"pmcW_{tag}.log"))),
               "",
               f"reference: the streaming-read kernel over {ref} bytes (16-byte loads):",
               f"  read requests 32/64/128 B = {c32:.0f} / {c64:.0f} / {c128:.0f} (all sizes: {call_:.0f})",
               f"  bytes by request size = {crd:.0f} = {crd / ref:.4f} x the bytes read",
               f"  FETCH_SIZE's formula (TCC_BUBBLE as the 128-byte count) = {cfetch:.0f} = {cfetch / ref:.4f} x",
               "",
               f"spmspv_kernel, mean per dispatch ({len(cr[PASS_R[0]][0])} dispatches per pass):",
               f"  read requests 32/64/128 B = {n32:.0f} / {n64:.0f} / {n128:.0f} (all sizes: {nall:.0f}; "
               f"to DRAM: {ndram:.0f}; TCC_BUBBLE {nbub:.0f})",
               f"  read bytes by request size = {rd:.0f}",
               f"  write requests = {nw:.0f} ({nw64:.0f} of 64 B) -> write bytes = {wr:.0f}",
               f"  FETCH_SIZE's formula = {fetch_formula:.0f} B, WRITE_SIZE = {wr:.0f} B (raw derived counters)",
               "",
               "per source, bytes per launch: algorithmic | whole 128-byte lines holding them",
               ]
        for k, (a, l) in lm.items():
            out.append(f"  {k:11s} {a:14.0f} | {l:14.0f}")
        out += [f"  {'reads':11s} {alg_rd:14.0f} | {line_rd:14.0f}   (measured read bytes {rd:.0f}: "
                f"{rd / line_rd:.3f} x the lines, {rd / alg_rd:.3f} x the algorithmic reads)",
                f"  split-K partials written (measured writes - y) = {partial_w:.0f}; read back at least as many",
                f"  reads beyond the lines = {rd - line_rd:.0f} "
                f"({(rd - line_rd) / max(partial_w, 1):.2f} x the partial bytes written)",
                "",
                f"algorithmic bytes per launch = {pj['algorithmic_bytes_per_launch']:.0f}",
                f"measured traffic per launch (reads + writes) = {rd + wr:.0f} = "
                f"{(rd + wr) / pj['algorithmic_bytes_per_launch']:.3f} x algorithmic",
                f"hbm_bytes_per_launch: {rd + wr:.0f}", f"kernel_sha: {sha}", ""]
        with open(os.path.join(prof_dir, f"traffic_spmspv_{tag}.txt"), "w") as fh:
            fh.write("\n".join(out))
        print("\n".join(out))


if __name__ == "__main__":
    main()

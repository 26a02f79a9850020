"""Benchmark of the decode-time Tiled-CBC spMspV on one MI355X.

Default workload: the four Llama-7B attention projections (q, k, v, o; each
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

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--launch graph|stream]
"""

from __future__ import annotations

import argparse
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


def parse():
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
    ap.add_argument("--profile-only", action="store_true",
                    help="run warmup + timed steps only (for rocprofv3 runs)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the timed steps, run one device-to-device copy of this many MiB "
                         "(a known-size reference for hardware byte counters)")
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
    return ap.parse_args()


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


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    import torch

    import paper_2607_21985_amd as spdp
    import synth

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no ROCm GPU visible"}))
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = synth.workload(args.workload)
    tile = wl["tile"]
    batch = args.batch if args.batch is not None else wl["batch"][0]
    if args.sw:
        wl = dict(wl, weight_sparsity=[float(v) for v in args.sw.split(",")])
    if args.p:
        wl = dict(wl, act_sparsity=[float(v) for v in args.p.split(",")])

    # ---- inputs: prune (library host C++), calibrate, encode rotated copies
    t_prep = time.perf_counter()
    pruned = {}
    for sw in wl["weight_sparsity"]:
        for proj in wl["projections"]:
            pruned[(sw, proj.name)] = spdp.prune_magnitude(proj.weight(), sw)
    xs = {proj.name: proj.activations(batch) for proj in wl["projections"]}
    # offline calibration sets: one per layer input (projections that read
    # one input share it), drawn apart from the inputs (draw 1)
    cal = {}
    if args.calibration > 0:
        for proj in wl["projections"]:
            key = (proj.x_seed, proj.x_kind, proj.cols)
            if key not in cal:
                cal[key] = proj.activations(args.calibration, draw=1)
    points = []
    for sw in wl["weight_sparsity"]:
        for p in wl["act_sparsity"]:
            for proj in wl["projections"]:
                x = xs[proj.name]
                if args.mask == "batch":
                    if cal:
                        # the calibration tokens in batches of this size,
                        # their column scores pooled
                        cs = cal[(proj.x_seed, proj.x_kind, proj.cols)]
                        n = cs.shape[0] // batch * batch
                        groups = cs[:n].reshape(-1, batch, cs.shape[1])
                        sc = np.sort(np.concatenate([batch_scores(g) for g in groups]))
                        t = -1.0 if p <= 0 else float(sc[int(np.ceil(p * sc.size)) - 1]) / batch
                    else:
                        t = batch_threshold_for(x, p)
                elif cal:
                    t = spdp.calibrate_threshold(cal[(proj.x_seed, proj.x_kind, proj.cols)], p)
                else:
                    t = spdp.calibrate_threshold(x, p)
                points.append({"sw": sw, "p": p, "proj": proj, "x": x, "t": t,
                               "w": pruned[(sw, proj.name)],
                               "label": f"{proj.name}@sw{sw:g}/p{p:g}"})
    t_enc = time.perf_counter()
    if args.rtn_bits:
        enc = lambda w: spdp.encode_rtn(w, tile, args.rtn_bits)  # noqa: E731
    else:
        enc = lambda w: spdp.encode(w, tile)  # noqa: E731
    copy0 = [enc(pt["w"]) for pt in points]
    enc_s = (time.perf_counter() - t_enc) / len(points)
    dev_bytes = sum(len(m.format()["values"]) * (1 if args.rtn_bits else 2) for m in copy0)
    n_copies = max(2, int(np.ceil(args.rotation_mb * 1e6 / max(dev_bytes, 1))) + 1)
    copies = [copy0] + [[enc(pt["w"]) for pt in points] for _ in range(n_copies - 1)]
    for pt, m in zip(points, copy0):
        f = m.format()
        act = (batch_activity(pt["x"], pt["t"]) if args.mask == "batch"
               else token_activity(pt["x"], spdp.threshold_code(pt["t"])))
        pt["bytes"], pt["active_frac"] = call_bytes(f, act)
        pt["dropped"] = dropped_fraction(act)
        pt["flops"] = call_flops(f, act)
        pt["rows"], pt["cols"] = f["rows"], f["cols"]
        del f
    # one device copy of each distinct input per rotation copy (grouped
    # products share it, as a decoder's q, k and v share the layer input)
    X = []
    for _ in range(n_copies):
        by_input = {}
        row = []
        for pt in points:
            key = (pt["sw"], pt["p"], pt["proj"].x_seed, pt["proj"].x_kind, pt["proj"].cols)
            if key not in by_input:
                by_input[key] = torch.from_numpy(pt["x"].view(np.int16)).view(torch.float16).to(dev)
            row.append(by_input[key])
        X.append(row)

    # launch units: the products of one sweep point that read one input form a
    # group (at most 8), every other product is a unit of its own
    def make_units(idx, grouped):
        units, open_ = [], {}
        for j in idx:
            pt = points[j]
            key = (pt["sw"], pt["p"], pt["proj"].x_seed, pt["proj"].x_kind, pt["proj"].cols)
            if grouped and key in open_ and len(units[open_[key]]) < 8:
                units[open_[key]].append(j)
            else:
                open_[key] = len(units)
                units.append([j])
        return units
    Y = [[torch.empty((batch, pt["rows"]), dtype=torch.float16, device=dev) for pt in points]
         for _ in range(n_copies)]
    for cp in copies:
        for m in cp:
            m.reserve(batch)
    prep_s = time.perf_counter() - t_prep
    stream = torch.cuda.current_stream(dev)

    def launch_calls(c, units, t_all=None):
        # t_all: one threshold for every call instead of the points' own
        th = (lambda j: points[j]["t"]) if t_all is None else (lambda j: t_all)
        for u in units:
            if len(u) == 1:
                copies[c][u[0]].spmspv_into(X[c][u[0]], th(u[0]), Y[c][u[0]], mask=args.mask)
            else:
                spdp.spmspv_many([copies[c][j] for j in u], [X[c][j] for j in u],
                                 [th(j) for j in u], [Y[c][j] for j in u], mask=args.mask)

    all_idx = list(range(len(points)))
    grouped = args.group == "decoder"
    step_units = make_units(all_idx, grouped)
    single_units = make_units(all_idx, False)
    graphs = {}

    def capture(key, c, idx):
        # capture on a side stream; replays go to the current stream
        s = torch.cuda.Stream(device=dev)
        s.wait_stream(torch.cuda.current_stream(dev))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            launch_calls(c, idx)
        torch.cuda.current_stream(dev).wait_stream(s)
        graphs[key] = g

    def step(i, mode, key="step", units=None):
        c = i % n_copies
        if mode == "graph":
            graphs[(key, c)].replay()
        else:
            launch_calls(c, units if units is not None else step_units)

    def capture_cycle(key, units, t_all=None):
        # one rotation cycle (the steps of copies 0 .. n_copies-1, in order)
        # as one graph: a decoder replays a whole token's pass over all its
        # layers as one graph, so the graph's own start-up is paid once per
        # many launches, not once per layer
        s = torch.cuda.Stream(device=dev)
        s.wait_stream(torch.cuda.current_stream(dev))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for c in range(n_copies):
                launch_calls(c, units, t_all)
        torch.cuda.current_stream(dev).wait_stream(s)
        graphs[(key, "cycle")] = g

    def run_steps(first, n, mode, key="step", units=None):
        # steps first .. first+n-1; in graph mode whole rotation cycles are
        # one replay, the steps outside a whole cycle one replay each
        i, end = first, first + n
        while i < end:
            if mode == "graph" and i % n_copies == 0 and i + n_copies <= end:
                graphs[(key, "cycle")].replay()
                i += n_copies
            else:
                step(i, mode, key, units)
                i += 1

    def timed(fn, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(n):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize(dev)
        return e0.elapsed_time(e1)

    # warm up eagerly (first calls load code, size workspaces), then capture
    for i in range(max(1, args.warmup)):
        step(i, "stream")
    torch.cuda.synchronize(dev)
    if args.launch == "graph":
        for c in range(n_copies):
            capture(("step", c), c, step_units)
            capture(("single", c), c, single_units)
        capture_cycle("step", step_units)
        capture_cycle("single", single_units)
        torch.cuda.synchronize(dev)
    run_steps(0, args.warmup, args.launch)
    torch.cuda.synchronize(dev)
    total_ms = timed(lambda _: run_steps(args.warmup, args.steps, args.launch), 1)
    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20)
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty(n, dtype=torch.uint8, device=dev)
        torch.cuda.synchronize(dev)
        dst.copy_(src)
        torch.cuda.synchronize(dev)
        del src, dst
    if args.profile_only:
        print(json.dumps({"profile_only": True, "launch": args.launch, "group": args.group,
                          "ms_per_step": total_ms / args.steps,
                          "launches": (2 * args.warmup + args.steps) * len(step_units),
                          "algorithmic_bytes_per_launch": sum(pt["bytes"] for pt in points) / len(step_units)}),
              flush=True)
        return
    ms_per_step = total_ms / args.steps
    step_bytes = sum(pt["bytes"] for pt in points)
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    # the same steps with one host launch per call, and with every product
    # as its own launch, for comparison
    stream_ms = timed(lambda i: step(args.warmup + i, "stream"), args.steps) / args.steps
    # the latency floor: the same launches with a threshold of +inf, so that
    # no column is active and every step but the value stream runs (launch,
    # set-up loads, activity test, list, split-K exchange, output)
    floor_ms = None
    if args.launch == "graph":
        capture_cycle("floor", step_units, float("inf"))
        run_steps(0, n_copies, "graph", "floor")
        torch.cuda.synchronize(dev)
        floor_ms = timed(lambda _: run_steps(0, args.steps // n_copies * n_copies or n_copies, "graph", "floor"),
                         1) / (args.steps // n_copies * n_copies or n_copies)
    single_ms = timed(lambda _: run_steps(args.warmup, args.steps, args.launch, "single", single_units),
                      1) / args.steps

    # ---- duration per sweep point: the point's calls run back to back (as a
    # captured graph in graph mode), so HIP events around a run of them
    # divided by their number give the kernels' average duration; an event
    # pair around every single launch would add its own overhead.
    n_proj = len(wl["projections"])
    reps = max(2, min(10, args.steps))
    per_call = np.zeros(len(points))
    for k in range(0, len(points), n_proj):
        idx = make_units(list(range(k, k + n_proj)), grouped)
        if args.launch == "graph":
            for c in range(n_copies):
                capture(("pt", k, c), c, idx)
            ms = timed(lambda r: graphs[("pt", k, r % n_copies)].replay(), reps)
        else:
            ms = timed(lambda r: launch_calls(r % n_copies, idx), reps)
        per_call[k:k + n_proj] = ms / (reps * n_proj)
    kern_ms = ms_per_step
    achieved = step_bytes / (kern_ms * 1e-3) / 1e9
    # the two roofs: T_roof = max(bytes / HBM peak, useful flops / vector peak)
    step_flops = sum(pt["flops"] for pt in points)
    t_hbm_us = step_bytes / (HBM_PEAK_GBS * 1e9) * 1e6
    t_alu_us = step_flops / (VEC_PEAK_TFLOPS * 1e12) * 1e6
    alu_bound = t_alu_us > t_hbm_us
    graphs.clear()

    # ---- measured streaming peaks on this GPU: a 1 GiB device copy (read +
    # write bytes) and a 1 GiB read-only reduction
    n_pk = 1 << 30
    a_pk = torch.empty(n_pk // 2, dtype=torch.float16, device=dev).fill_(1.0)
    b_pk = torch.empty_like(a_pk)
    for _ in range(2):
        b_pk.copy_(a_pk)
        a_pk.sum(dtype=torch.float32)
    torch.cuda.synchronize(dev)
    copy_ms = timed(lambda i: b_pk.copy_(a_pk), 5) / 5
    read_ms = timed(lambda i: a_pk.sum(dtype=torch.float32), 5) / 5
    peaks = {"copy_gbs": round(2 * n_pk / (copy_ms * 1e-3) / 1e9, 1),
             "read_gbs": round(n_pk / (read_ms * 1e-3) / 1e9, 1),
             "how": "torch copy_ of 1 GiB fp16 (read + write bytes) and torch sum of 1 GiB fp16 (read bytes), "
                    "mean of 5 after 2 warm-ups"}
    del a_pk, b_pk

    # ---- dense fp16 GEMV baseline (torch F.linear), rotated the same way
    dense = None
    if not args.no_dense:
        import torch.nn.functional as F
        dW = {}
        names = [proj.name for proj in wl["projections"]]
        w_bytes = sum(proj.rows * proj.cols * 2 for proj in wl["projections"])
        n_dc = max(2, int(np.ceil(args.rotation_mb * 1e6 / w_bytes)) + 1)
        for proj in wl["projections"]:
            w16 = proj.weight()
            for c in range(n_dc):
                dW[(c, proj.name)] = torch.from_numpy(w16.view(np.int16)).view(torch.float16).to(dev)
        dX = {n: torch.from_numpy(xs[n].view(np.int16)).view(torch.float16).to(dev) for n in names}

        def dcalls(c):
            for n in names:
                F.linear(dX[n], dW[(c, n)])

        for c in range(n_dc):
            dcalls(c)
        torch.cuda.synchronize(dev)
        dgraphs = []
        if args.launch == "graph":
            # per copy, and one rotation cycle as one graph, as for spMspV
            for cs in [[c] for c in range(n_dc)] + [list(range(n_dc))]:
                s_cap = torch.cuda.Stream(device=dev)
                s_cap.wait_stream(torch.cuda.current_stream(dev))
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=s_cap):
                    for c in cs:
                        dcalls(c)
                torch.cuda.current_stream(dev).wait_stream(s_cap)
                dgraphs.append(g)

        def drun(first, n):
            i, end = first, first + n
            while i < end:
                if dgraphs and i % n_dc == 0 and i + n_dc <= end:
                    dgraphs[n_dc].replay()
                    i += n_dc
                else:
                    if dgraphs:
                        dgraphs[i % n_dc].replay()
                    else:
                        dcalls(i % n_dc)
                    i += 1

        drun(0, args.warmup)
        torch.cuda.synchronize(dev)
        d_us = timed(lambda _: drun(args.warmup, args.steps), 1) * 1e3 / (args.steps * len(names))
        del dgraphs
        dense = {"us_per_call": d_us,
                 "gbs": (w_bytes / len(names) + 2 * batch * (wl["projections"][0].rows + wl["projections"][0].cols)) / (d_us * 1e-6) / 1e9}
        del dW

    # ---- per-point summary
    pts_out = []
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

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(points, args.mask, rtn_bits=args.rtn_bits)

    # the committed counter summaries are of fp16 Values
    traffic = None if args.rtn_bits else read_traffic(args.workload, args.group)
    n_launch = len(step_units)
    us_per_call = ms_per_step * 1e3 / len(points)
    kernel_us = kern_ms * 1e3 / n_launch
    out = {
        "metric": "spMspV \u00b5s/call + achieved HBM GB/s (% of peak), Llama-7B shapes, batch 1",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
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
            "weight_sparsity": wl["weight_sparsity"], "act_sparsity": wl["act_sparsity"],
            "batch": batch, "tile": list(tile), "calls_per_step": len(points),
            "launches_per_step": n_launch, "grouping": args.group,
            "rotation_copies": n_copies, "accumulate": "f32",
            "values": (f"rtn{args.rtn_bits}: {args.rtn_bits}-bit round-to-nearest codes, one byte each, one "
                       "fp32 scale per row" if args.rtn_bits else "fp16"),
            "mask": args.mask,
            "threshold": ({"rule": "offline calibration", "calibration_tokens": args.calibration,
                           "how": "p-quantile of |x| over separately drawn tokens of each layer input"}
                          if args.calibration > 0 else
                          {"rule": "own percentile", "how": "p-quantile of |x| over the input itself"}),
        },
        "us_per_call": round(us_per_call, 3),
        "us_per_call_ungrouped": round(single_ms * 1e3 / len(points), 3),
        "gbs_ungrouped": round(step_bytes / (single_ms * 1e-3) / 1e9, 2),
        "us_per_call_stream_launch": round(stream_ms * 1e3 / len(points), 3),
        "launch": args.launch,
        "pct_of_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "measured_peaks": peaks,
        "pct_of_measured_read_peak": round(100 * value / peaks["read_gbs"], 2),
        "roofline": {
            **({"bound": "alu", "achieved": round(step_flops / (kern_ms * 1e-3) / 1e12, 3),
                "peak": VEC_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(t_alu_us / (kern_ms * 1e3), 4)} if alu_bound else
               {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4)}),
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
        "latency_floor": ({"us_per_launch": round(floor_ms * 1e3 / n_launch, 3),
                           "frac_of_launch": round(floor_ms / kern_ms, 4),
                           "how": "the same launches with threshold +inf: no column active, every step "
                                  "but the value stream runs"} if floor_ms is not None else None),
        "cpu_baseline": cpu,
        "dense_gemv": dense,
        "speedup_vs_dense": round(dense["us_per_call"] / us_per_call, 3) if dense else None,
        "points": pts_out,
        "prep_s": round(prep_s, 2),
        "encode_s_per_matrix": round(enc_s, 4),
        "host": platform.node(),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

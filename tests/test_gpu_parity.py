"""GPU parity: the HIP spMspV path (through the C ABI) against the CPU oracle.

Every case builds its inputs from ``synth`` (seeded), runs the oracle's own
pipeline (oracle.magnitude_prune -> oracle.threshold_for -> oracle.spmspv) on
the CPU and the library's pipeline (spdp.encode -> spdp_spmspv on the GPU),
and compares element by element:

    |Y_gpu - y64| <= 2e-3 * S + 1e-5,   S = sum_k |W_sp[m,k]| |xm[b,k]|,

with Y finite, and exactly 0 where no active term exists (S == 0). Small cases
are checked in full; full-size shapes (in the same launch configuration as
bench.py) are checked on sampled rows plus whole-output properties.
"""

import ctypes
import json
import os

import numpy as np
import pytest

import oracle
import synth
from conftest import GOLDEN

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2607_21985_amd as spdp  # noqa: E402

RTOL, ATOL = 2e-3, 1e-5


def _dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm GPU (torch.cuda.is_available() is False)")
    return torch.device("cuda:0")


def _to_dev(x16: np.ndarray):
    t = torch.from_numpy(np.ascontiguousarray(x16).view(np.int16)).view(torch.float16)
    return t.to(_dev())


def _run_gpu(m, x16, t, y_init=None, mask="token"):
    X = _to_dev(x16)
    if y_init is None:
        Y = torch.full((x16.shape[0], m.rows), float("nan"), dtype=torch.float16, device=X.device)
    else:
        Y = y_init
    m.spmspv_into(X, t, Y, mask=mask)
    torch.cuda.synchronize()
    return Y.cpu().numpy().astype(np.float64)


def _assert_close(y, y64, s64, label=""):
    assert np.all(np.isfinite(y)), f"{label}: non-finite output"
    err = np.abs(y - y64)
    bound = RTOL * s64 + ATOL
    bad = err > bound
    if bad.any():
        b, m = np.argwhere(bad)[0]
        raise AssertionError(f"{label}: {bad.sum()} elements out of tolerance; first at "
                             f"(b={b}, m={m}): gpu={y[b, m]} ref={y64[b, m]} S={s64[b, m]}")
    zero = s64 == 0
    assert np.all(y[zero] == 0), f"{label}: rows with no active term are not exactly 0"


def _case(rows, cols, tile, sw, p, batch, wseed, xseed, xkind="laplace"):
    w = oracle.magnitude_prune(synth.weights(rows, cols, wseed), sw)
    x = (synth.laplace_activations if xkind == "laplace" else synth.swiglu_activations)(batch, cols, xseed)
    t = float(oracle.threshold_for(x, p))
    return w, x, t


def _check_full(w, x, t, tile, label):
    print(f"[gpu] {label}", flush=True)
    m = spdp.encode(w, tile)
    y = _run_gpu(m, x, t)
    y64, s64, _ = oracle.spmspv(w, x, t)
    _assert_close(y, y64, s64, label)
    m.close()
    return y


# ---------------------------------------------------------------------------

def _hand_cases():
    with open(os.path.join(GOLDEN, "tiled_cbc_hand.json")) as fh:
        return json.load(fh)["cases"]


@pytest.mark.parametrize("case", _hand_cases(), ids=lambda c: c["name"])
def test_hand_worked_cases_exact(case):
    w = np.zeros((case["rows"], case["cols"]), dtype=np.uint16)
    for mm, k, h in case["nonzeros"]:
        w[mm, k] = int(h, 16)
    w = w.view(np.float16)
    m = spdp.encode(w, (case["tile_m"], case["tile_k"]))
    for prod in case["products"]:
        x = np.array([prod["x"]], dtype=np.float16)
        y = _run_gpu(m, x, prod["t"])
        expect = np.zeros(case["rows"])
        for mm, v in prod["y_nonzero"]:
            expect[mm] = v
        assert np.array_equal(y[0], expect)
    m.close()


SMALL = [
    # rows, cols, tile, sw, p, batch
    (64, 64, (64, 64), 0.5, 0.5, 1),
    (1024, 1024, (64, 64), 0.5, 0.5, 1),      # the 1024x1024 single-layer workload
    (1, 1, (64, 1), 0.0, 0.0, 1),
    (70, 3, (64, 2), 0.3, 0.0, 1),
    (333, 517, (256, 16), 0.5, 0.5, 1),
    (513, 1000, (256, 16), 0.6, 0.25, 2),
    (256, 4096, (256, 16), 0.7, 0.5, 3),
    (700, 900, (128, 8), 0.5, 0.3, 4),
    (450, 640, (192, 32), 0.4, 0.5, 5),
    (300, 2048, (64, 1), 0.5, 0.5, 8),
    (1000, 1536, (256, 256), 0.5, 0.6, 13),
    (257, 777, (256, 4), 0.8, 0.2, 16),
    (129, 300, (128, 64), 0.5, 0.5, 17),
    (512, 1111, (256, 16), 0.6, 0.4, 32),
    (96, 5000, (64, 16), 0.9, 0.7, 7),
]


@pytest.mark.parametrize("rows,cols,tile,sw,p,batch", SMALL)
def test_small_against_oracle(rows, cols, tile, sw, p, batch):
    w, x, t = _case(rows, cols, tile, sw, p, batch, rows * 7 + cols, cols * 3 + batch)
    _check_full(w, x, t, tile, f"small {rows}x{cols} tile={tile} sw={sw} p={p} B={batch}")


# Both launch forms, forced: each wave's first batch requested before the
# workgroup list is built (SPDP_EARLY_FIRST=1) or all batches taken from the
# list (0). The cases include waves left with fewer than four active columns
# or none (high p), several tokens, and full 128-column waves with every
# column active (the largest list either form builds).
EARLY = [
    # rows, cols, tile, sw, p, batch, splitk
    (333, 517, (256, 16), 0.5, 0.5, 1, None),
    (513, 1000, (256, 16), 0.6, 0.97, 1, None),
    (700, 2900, (128, 8), 0.5, 0.9, 3, 7),
    (300, 2048, (64, 1), 0.5, 0.5, 8, None),
    (512, 1111, (256, 16), 0.6, 0.4, 32, None),
    (1024, 8192, (256, 16), 0.5, 0.0, 1, 16),
    # many tokens: the gather's (row block, 8-token slice) units outnumber
    # the reducers, which then take several each
    (512, 1111, (256, 16), 0.6, 0.4, 32, 1),
    (300, 2048, (64, 1), 0.5, 0.5, 17, 3),
    (700, 900, (128, 8), 0.5, 0.3, 16, 5),
]


@pytest.mark.parametrize("early", ["0", "1"])
@pytest.mark.parametrize("rows,cols,tile,sw,p,batch,splitk", EARLY)
def test_launch_forms_against_oracle(monkeypatch, early, rows, cols, tile, sw, p, batch, splitk):
    monkeypatch.setenv("SPDP_EARLY_FIRST", early)
    if splitk:
        monkeypatch.setenv("SPDP_SPLITK", str(splitk))
    w, x, t = _case(rows, cols, tile, sw, p, batch, rows * 5 + cols, cols * 7 + batch)
    _check_full(w, x, t, tile, f"early={early} {rows}x{cols} tile={tile} sw={sw} p={p} B={batch}")


def test_dense_no_threshold_is_gemv():
    w, x, _ = _case(300, 700, (256, 16), 0.0, 0.0, 2, 5, 6)
    _check_full(w, x, -1.0, (256, 16), "dense")


def test_everything_inactive_gives_exact_zero():
    w, x, _ = _case(300, 700, (256, 16), 0.5, 0.0, 3, 7, 8)
    t = float(np.abs(x.astype(np.float64)).max())
    y = _check_full(w, x, t, (256, 16), "all inactive")
    assert np.all(y == 0)


def test_all_zero_weights():
    w = np.zeros((200, 300), dtype=np.float16)
    x = synth.laplace_activations(2, 300, 1)
    y = _check_full(w, x, -1.0, (128, 16), "zero W")
    assert np.all(y == 0)


def test_single_active_column():
    w, _, _ = _case(500, 333, (256, 16), 0.5, 0.0, 1, 11, 12)
    x = np.full((1, 333), 0.25, dtype=np.float16)
    x[0, 200] = np.float16(-3.0)
    y = _check_full(w, x, 1.0, (256, 16), "one column")
    assert np.array_equal(y[0], (np.float16(-3.0) * w[:, 200].astype(np.float64)).astype(np.float16).astype(np.float64))


def test_nan_activations_are_never_active():
    w, x, t = _case(256, 512, (256, 16), 0.5, 0.5, 2, 13, 14)
    x = x.copy()
    x[0, ::5] = np.float16(np.nan)
    _check_full(w, x, t, (256, 16), "NaN in x")


def test_negative_zero_threshold_and_ties():
    w, _, _ = _case(256, 256, (256, 16), 0.5, 0.0, 1, 15, 16)
    x = np.tile(np.array([1.0, -1.0, 0.5, 0.0, -0.0, 2.0, -2.0, 1.0], dtype=np.float16), (2, 32))
    for t in (1.0, 0.5, 0.0, -0.0, -1.0, 1.9999, 2.0):
        _check_full(w, x, t, (256, 16), f"ties t={t}")


# Activations at the threshold code's edges for every kernel form: the
# one-token and two-token forms test each token's magnitude per column; from
# four tokens on (and in the matrix-core form above 16 tokens) the masks are
# taken from one unsigned compare per token, which must agree with
# (code, 0x7C00] at code = -1 (t < 0: every non-NaN value, +-0 included),
# 0 (t = +-0), a subnormal, ties at 0.5 / 1 / 2, 65504 (nothing finite
# above it) and +inf (nothing at all). x holds +-0, a subnormal, ties, NaN
# and +-65504 (two columns per token, so the sums stay finite).
_EDGE_VALUES = np.array([1.0, -1.0, 0.5, 0.0, -0.0, 2.0, -2.0, np.nan, 6e-8, -6e-8, 1.9990234375, 0.25, -0.5],
                        dtype=np.float16)
_EDGE_THRESHOLDS = (1.0, 0.5, 0.0, -0.0, -1.0, 1.9999, 2.0, 65504.0, float("inf"), 5.9604645e-08)


def _edge_x(batch, cols):
    k = np.arange(cols)
    x = np.stack([_EDGE_VALUES[(k * 7 + b * 3) % _EDGE_VALUES.size] for b in range(batch)])
    for b in range(batch):
        x[b, (b * 37) % cols] = np.float16(65504.0)
        x[b, (b * 53 + 11) % cols] = np.float16(-65504.0)
    return x


@pytest.mark.parametrize("batch,mask,mfma,codes", [
    (1, "token", None, False), (2, "token", None, False), (4, "token", None, False),
    (5, "token", None, False), (8, "token", None, False), (8, "token", "1", False),
    (12, "token", None, False), (16, "token", None, False), (20, "token", None, False),
    (32, "token", None, False), (2, "batch", None, False), (8, "batch", None, False),
    (20, "batch", None, False), (32, "batch", None, False),
    (1, "token", None, True), (4, "token", None, True), (16, "token", None, True), (32, "token", None, True)])
def test_threshold_edges_every_form(monkeypatch, batch, mask, mfma, codes):
    if mfma is not None:
        monkeypatch.setenv("SPDP_MFMA", mfma)
    w = oracle.magnitude_prune(synth.weights(300, 512, 23), 0.5)
    x = _edge_x(batch, 512)
    if mask == "batch":
        # a NaN in any token drops its column for the batch: keep a few, so
        # that the other columns' batch scores decide
        x = np.where(np.isnan(x), np.float16(0.75), x)
        x[0, ::29] = np.float16(np.nan)
    if codes:
        # one-byte 4-bit codes, one scale per row (the low-bit Values form)
        q, scales, _ = oracle.rtn_quantize(w, 4)
        m = spdp.encode_rtn(w, (256, 16), 4)
    else:
        m = spdp.encode(w, (256, 16))
    for t in _EDGE_THRESHOLDS:
        label = f"B={batch} mask={mask} mfma={mfma} codes={codes} t={t}"
        print(f"[gpu] edges {label}", flush=True)
        y = _run_gpu(m, x, t, mask=mask)
        y64, s64, _ = oracle.spmspv_rtn(q, scales, x, t, mask) if codes else oracle.spmspv(w, x, t, mask)
        _assert_close(y, y64, s64, label)
    m.close()


def test_output_fully_overwritten_and_repeatable():
    w, x, t = _case(600, 1500, (256, 16), 0.5, 0.5, 4, 17, 18)
    m = spdp.encode(w, (256, 16))
    y1 = _run_gpu(m, x, t)
    y2 = _run_gpu(m, x, t)  # second call: the stripes' phases were advanced by the first
    assert np.array_equal(y1, y2), "two identical calls differ"
    y64, s64, _ = oracle.spmspv(w, x, t)
    _assert_close(y1, y64, s64, "repeat")
    # growing then shrinking the batch reuses / grows the workspace
    for b in (1, 9, 32, 2):
        xb = synth.laplace_activations(b, 1500, 100 + b)
        tb = float(oracle.threshold_for(xb, 0.5))
        yb = _run_gpu(m, xb, tb)
        y64, s64, _ = oracle.spmspv(w, xb, tb)
        _assert_close(yb, y64, s64, f"batch {b}")
    m.close()


def test_alternating_batches_never_read_stale_partials(monkeypatch):
    """Split-K partials from an older call with a larger batch stay in the
    workspace; every later call must ignore them (they carry an old phase)."""
    monkeypatch.setenv("SPDP_SPLITK", "5")
    w = oracle.magnitude_prune(synth.weights(520, 2600, 61), 0.5)
    m = spdp.encode(w, (256, 16))
    m.reserve(8)
    for i, b in enumerate((8, 1, 3, 1, 8, 2, 8)):
        print(f"[gpu] alternating batch {i}: b={b}", flush=True)
        xb = synth.laplace_activations(b, 2600, 300 + i)
        tb = float(oracle.threshold_for(xb, 0.4))
        yb = _run_gpu(m, xb, tb)
        y64, s64, _ = oracle.spmspv(w, xb, tb)
        _assert_close(yb, y64, s64, f"alternating batch {i} (b={b})")
    m.close()


def test_graph_replay_matches_eager():
    """Calls captured in a HIP graph and replayed: no host-side state is baked
    into the capture, so every replay (with other work and synchronizations
    in between) gives the eager result."""
    dev = _dev()
    cases = [_case(900, 2100, (256, 16), 0.5, p, b, 71 + i, 81 + i) for i, (p, b) in enumerate([(0.5, 1), (0.0, 3)])]
    # a third call with the batch-shared column set
    wb, xb, _ = _case(900, 2100, (256, 16), 0.5, 0.5, 5, 74, 84)
    cases.append((wb, xb, _batch_t(xb, 0.5)))
    masks = ["token", "token", "batch"]
    mats = [spdp.encode(w, (256, 16)) for w, _, _ in cases]
    for m, (_, x, _) in zip(mats, cases):
        m.reserve(x.shape[0])
    Xs = [_to_dev(x) for _, x, _ in cases]
    Ys = [torch.zeros((x.shape[0], m.rows), dtype=torch.float16, device=dev) for (_, x, _), m in zip(cases, mats)]
    eager = []
    for m, X, Y, (_, _, t), mk in zip(mats, Xs, Ys, cases, masks):
        m.spmspv_into(X, t, Y, mask=mk)
        eager.append(Y.clone())
    torch.cuda.synchronize()
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for m, X, Y, (_, _, t), mk in zip(mats, Xs, Ys, cases, masks):
            m.spmspv_into(X, t, Y, mask=mk)
    torch.cuda.synchronize()
    for rep in range(4):
        print(f"[gpu] graph replay {rep}", flush=True)
        for Y in Ys:
            Y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for i, (Y, E) in enumerate(zip(Ys, eager)):
            assert torch.equal(Y, E), f"replay {rep}, call {i}: differs from the eager result"
        # eager calls on the same handles between replays
        for m, X, (_, _, t), mk in zip(mats, Xs, cases, masks):
            m(X, t, mask=mk)
        torch.cuda.synchronize()
    for (w, x, t), E, mk in zip(cases, eager, masks):
        y64, s64, _ = oracle.spmspv(w, x, t, mk)
        _assert_close(E.cpu().numpy().astype(np.float64), y64, s64, "graph eager reference")
    del g
    for m in mats:
        m.close()


def test_workspace_growth_keeps_captured_graphs_valid():
    """A call with a larger batch grows the handle's workspace without waiting
    for the device; the old workspace stays allocated, so a graph captured
    before the growth still replays correctly. Growth while the stream is
    capturing is refused and launches nothing."""
    dev = _dev()
    w, x1, t = _case(1000, 3000, (256, 16), 0.5, 0.5, 1, 91, 92)
    m = spdp.encode(w, (256, 16))
    X1 = _to_dev(x1)
    Y1 = torch.zeros((1, m.rows), dtype=torch.float16, device=dev)
    m.spmspv_into(X1, t, Y1)
    torch.cuda.synchronize()
    ref1 = Y1.clone()
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        m.spmspv_into(X1, t, Y1)
    torch.cuda.synchronize()
    # grow: 8 tokens (a new workspace, the captured one retired but alive)
    x8 = synth.laplace_activations(8, 3000, 93)
    t8 = float(oracle.threshold_for(x8, 0.5))
    y8 = _run_gpu(m, x8, t8)
    y64, s64, _ = oracle.spmspv(w, x8, t8)
    _assert_close(y8, y64, s64, "after growth, 8 tokens")
    for rep in range(3):
        Y1.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y1, ref1), f"replay {rep} after the workspace grew"
        _assert_close(_run_gpu(m, x1, t), *oracle.spmspv(w, x1, t)[:2], f"eager one token, rep {rep}")
    # a batch beyond the workspace inside a capture: refused, nothing launched
    x16 = synth.laplace_activations(16, 3000, 94)
    X16 = _to_dev(x16)
    Y16 = torch.zeros((16, m.rows), dtype=torch.float16, device=dev)
    g2 = torch.cuda.CUDAGraph()
    err = None
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.graph(g2, stream=s):
        try:
            m.spmspv_into(X16, 0.5, Y16)
        except spdp.SpdpError as e:
            err = e
    torch.cuda.synchronize()
    assert err is not None and err.status == -1 and "spdp_reserve" in str(err)
    del g, g2
    m.close()


@pytest.mark.parametrize("splitk", ["1", "2", "3", "7", "64", "1000"])
def test_split_k_settings(splitk, monkeypatch):
    monkeypatch.setenv("SPDP_SPLITK", splitk)
    w, x, t = _case(777, 3000, (256, 16), 0.5, 0.5, 3, 19, 20)
    _check_full(w, x, t, (256, 16), f"splitk={splitk}")


def test_streams_and_interleaved_handles():
    dev = _dev()
    cases = [_case(400 + 64 * i, 900 + 100 * i, (256, 16), 0.5, 0.5, 1 + i, 30 + i, 40 + i) for i in range(3)]
    mats = [spdp.encode(w, (256, 16)) for w, _, _ in cases]
    s = torch.cuda.Stream(device=dev)
    outs = []
    with torch.cuda.stream(s):
        for (w, x, t), m in zip(cases, mats):
            X = _to_dev(x)
            Y = torch.empty((x.shape[0], m.rows), dtype=torch.float16, device=dev)
            m.spmspv_into(X, t, Y, stream=s)
            outs.append(Y)
    s.synchronize()
    for (w, x, t), Y in zip(cases, outs):
        y64, s64, _ = oracle.spmspv(w, x, t)
        _assert_close(Y.cpu().numpy().astype(np.float64), y64, s64, "stream")
    for m in mats:
        m.close()


def test_device_copy_matches_host_format():
    w, _, _ = _case(700, 900, (256, 16), 0.6, 0.0, 1, 21, 22)
    m = spdp.encode(w, (256, 16))
    f = m.format()
    ref = oracle.encode(w, 256, 16)
    for name in ("tile_offset", "col_info", "bitmap", "values"):
        assert np.array_equal(f[name], getattr(ref, name)), name
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    torch.cuda.synchronize()
    for name, ptr in m.device_pointers().items():
        host = np.empty_like(f[name])
        assert hip.hipMemcpy(host.ctypes.data, ptr, host.nbytes, 2) == 0
        assert np.array_equal(host, f[name]), name
    m.close()


def test_argument_errors_on_device():
    w, x, t = _case(128, 256, (128, 16), 0.5, 0.5, 2, 23, 24)
    m = spdp.encode(w, (128, 16))
    X = _to_dev(x)
    Y = torch.empty((2, 128), dtype=torch.float16, device=X.device)
    with pytest.raises(spdp.SpdpError):
        m.spmspv_into(X, float("nan"), Y)
    L = spdp.lib()
    for b in (0, 33, -1):
        assert L.spdp_spmspv(m._h, ctypes.c_void_p(X.data_ptr()), b, ctypes.c_float(0.1),
                             ctypes.c_void_p(Y.data_ptr()), None) == -1
    # misaligned and overlapping buffers
    assert L.spdp_spmspv(m._h, ctypes.c_void_p(X.data_ptr() + 2), 1, ctypes.c_float(0.1),
                         ctypes.c_void_p(Y.data_ptr()), None) == -1
    assert L.spdp_spmspv(m._h, ctypes.c_void_p(X.data_ptr()), 1, ctypes.c_float(0.1),
                         ctypes.c_void_p(X.data_ptr()), None) == -1
    m.close()


# ---------------------------------------------------------------------------
# Full-size workloads, same launch configuration as bench.py, every row: the
# oracle runs in row blocks. One shape per distinct projection of each
# workload, at its highest (sw, p) point, at 50/0 (no dynamic sparsity), and
# for the 70B layer also at 80/70; batch 1 and the workload's largest batch.

def _check_all_rows(m, w, x, t, label, block=2048):
    print(f"[gpu] {label}", flush=True)
    y = _run_gpu(m, x, t)
    assert np.all(np.isfinite(y)), label
    for r0 in range(0, w.shape[0], block):
        rows = np.arange(r0, min(w.shape[0], r0 + block))
        y64, s64 = oracle.spmspv_rows(w, x, t, rows)
        _assert_close(y[:, rows], y64, s64, f"{label} rows {rows[0]}..{rows[-1]}")


FULL = []
for name in ("llama7b-attn", "llama7b-mlp", "llama13b-layer", "llama70b-layer", "llama70b-tp8"):
    wl = synth.workload(name)
    seen = set()
    for proj in wl["projections"]:
        if (proj.rows, proj.cols, proj.x_kind) not in seen:
            seen.add((proj.rows, proj.cols, proj.x_kind))
            FULL.append((name, proj))


@pytest.mark.parametrize("name,proj", FULL, ids=[f"{n}-{p.name}" for n, p in FULL])
def test_full_size_all_rows(name, proj):
    wl = synth.workload(name)
    points = [(max(wl["weight_sparsity"]), max(wl["act_sparsity"])), (0.5, 0.0)]
    if name == "llama70b-layer":
        points.append((0.8, 0.7))
    batch = max(wl["batch"])
    w0 = proj.weight()
    for sw, p in sorted(set(points)):
        w = oracle.magnitude_prune(w0, sw)
        m = spdp.encode(w, wl["tile"])
        for b in sorted({1, batch}):
            x = proj.activations(b)
            t = float(oracle.threshold_for(x, p))
            _check_all_rows(m, w, x, t, f"{name}/{proj.name} {proj.rows}x{proj.cols} sw={sw} p={p} B={b}")
        m.close()


# ---------------------------------------------------------------------------
# Batched DP with one column set shared by the batch (mask="batch"): column k
# is read for every token iff the fp32 running sum of |x[b, k]| exceeds
# fp32(batch * t).

def _batch_t(x, p):
    """t dropping the fraction p of the columns by batch score (oracle side)."""
    s = np.sort(oracle.batch_score(x))
    return -1.0 if p <= 0 else float(s[int(np.ceil(p * s.size)) - 1]) / x.shape[0]


BATCH_MASK = [
    # rows, cols, tile, sw, p, batch
    (333, 517, (256, 16), 0.5, 0.5, 1),
    (513, 1000, (256, 16), 0.6, 0.4, 2),
    (256, 4096, (256, 16), 0.7, 0.5, 3),
    (700, 900, (128, 8), 0.5, 0.3, 4),
    (300, 2048, (64, 1), 0.5, 0.5, 8),
    (1000, 1536, (256, 256), 0.5, 0.6, 13),
    (129, 300, (128, 64), 0.5, 0.5, 17),
    (512, 1111, (256, 16), 0.6, 0.7, 32),
]


@pytest.mark.parametrize("rows,cols,tile,sw,p,batch", BATCH_MASK)
def test_batch_mask_against_oracle(rows, cols, tile, sw, p, batch):
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows * 3 + cols), sw)
    x = synth.laplace_activations(batch, cols, cols + 5 * batch)
    t = _batch_t(x, p)
    label = f"batch mask {rows}x{cols} tile={tile} sw={sw} p={p} B={batch}"
    print(f"[gpu] {label}", flush=True)
    m = spdp.encode(w, tile)
    y = _run_gpu(m, x, t, mask="batch")
    y64, s64, _ = oracle.spmspv(w, x, t, "batch")
    _assert_close(y, y64, s64, label)
    if batch == 1:  # the two rules coincide at one token, bit for bit
        assert np.array_equal(y, _run_gpu(m, x, t, mask="token"))
    m.close()


def test_batch_mask_edge_cases():
    w = oracle.magnitude_prune(synth.weights(300, 700, 91), 0.5)
    x = synth.laplace_activations(5, 700, 92)
    m = spdp.encode(w, (256, 16))
    # nothing active: exact zeros
    y = _run_gpu(m, x, float(np.abs(x.astype(np.float64)).max()) * 2, mask="batch")
    assert np.array_equal(y, np.zeros_like(y))
    # a negative threshold keeps every column: the plain product
    y = _run_gpu(m, x, -1.0, mask="batch")
    y64, s64, _ = oracle.spmspv(w, x, -1.0, "batch")
    _assert_close(y, y64, s64, "batch mask, t < 0")
    # a NaN in one token drops its column for the whole batch
    xn = x.copy()
    xn[2, 10] = np.float16(np.nan)
    t = _batch_t(x, 0.3)
    y = _run_gpu(m, xn, t, mask="batch")
    y64, s64, _ = oracle.spmspv(w, xn, t, "batch")
    assert not oracle.active_mask(xn, t, "batch")[0, 10]
    _assert_close(y, y64, s64, "batch mask, NaN token")
    m.close()


@pytest.mark.parametrize("mfma", ["0", "1"])
@pytest.mark.parametrize("passes", ["1", "2", "3", "5", "64"])
@pytest.mark.parametrize("batch", [4, 8, 17, 32])
def test_forced_passes_and_matrix_core_form(monkeypatch, passes, batch, mfma):
    """Several K ranges per workgroup, forced, in the vector forms (from 3
    tokens) and in the 32x32 matrix-core form (forced on from 5 tokens): fp16
    values and one-byte codes (which keep one range) must both match the
    oracle. 64 passes cover the whole K: one segment per stripe, Y written
    without partials."""
    if mfma == "1" and batch < 5:
        pytest.skip("the 32x32 matrix-core form starts at 5 tokens")
    monkeypatch.setenv("SPDP_PASSES", passes)
    monkeypatch.setenv("SPDP_MFMA", mfma)
    w, x, t = _case(700, 3000, (256, 16), 0.6, 0.4, batch, 123, 456)
    _check_full(w, x, t, (256, 16), f"passes={passes} mfma={mfma} B={batch} fp16")
    codes, scales, _ = oracle.rtn_quantize(w, 4)
    m = spdp.encode_rtn(w, (256, 16), 4)
    y = _run_gpu(m, x, t)
    y64, s64, _ = oracle.spmspv_rtn(codes, scales, x, t)
    _assert_close(y, y64, s64, f"passes={passes} mfma={mfma} B={batch} codes")
    m.close()


@pytest.mark.parametrize("codes", [False, True], ids=["fp16", "codes"])
@pytest.mark.parametrize("batch", [1, 2, 3, 8, 16, 32])
def test_one_segment_every_vector_form(batch, codes):
    """40 columns fit one segment (64 columns at the narrowest split), so
    every stripe's workgroup writes Y itself, also in the one- and two-token
    forms and the code forms (row scale applied at the write)."""
    w, x, t = _case(600, 40, (256, 16), 0.5, 0.3, batch, 131, 457)
    label = f"600x40 B={batch} {'codes' if codes else 'fp16'} one segment"
    print(f"[gpu] {label}", flush=True)
    if codes:
        q, scales, _ = oracle.rtn_quantize(w, 4)
        m = spdp.encode_rtn(w, (256, 16), 4)
        y64, s64, _ = oracle.spmspv_rtn(q, scales, x, t)
    else:
        m = spdp.encode(w, (256, 16))
        y64, s64, _ = oracle.spmspv(w, x, t)
    for rep in range(2):
        _assert_close(_run_gpu(m, x, t), y64, s64, f"{label} rep {rep}")
    m.close()

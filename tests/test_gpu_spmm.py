"""GPU parity of the prefill product (spdp_spmm, Sec. 4.3) against the oracle.

Y = X W_sp^T for N tokens, every column taking part, computed on the matrix
cores from the same Tiled-CBC handle the decode path uses. Checked against
``oracle.spmm``:

* realistic inputs (the workloads' weight and activation distributions),
  every output element within |Y - y64| <= 2e-3 S + 1e-5, S = sum |w||x|;
* dyadic inputs (weights k 2^-9, tokens j / 4) on which every fp32 sum is
  exact in any order, so Y must equal fp16(y64) bit for bit on every row;
* ragged rows, columns that are not a multiple of 8, token counts that are
  not a multiple of the 128-token workgroup tile, tile_k 16/32/64;
* every kernel form (SPDP_SPMM_FORM=1 the plain one, 2 and 3 the 128- and
  256-token warp-specialized ones; the default picks by token count) and the
  split-K path of the warp-specialized form (forced split counts with
  SPDP_SPMM_SPLITS, and a width whose TileOffsets need several splits),
  bit for bit; graph capture with the split-K workspace, and its refusal
  to grow the workspace inside a capture.
"""

import ctypes

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2607_21985_amd as spdp  # noqa: E402


def _dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm GPU (torch.cuda.is_available() is False)")
    return torch.device("cuda:0")


def _to_dev(a16):
    return torch.from_numpy(np.ascontiguousarray(a16).view(np.int16)).view(torch.float16).to(_dev())


def _run(m, x):
    X = _to_dev(x)
    Y = torch.full((x.shape[0], m.rows), float("nan"), dtype=torch.float16, device=X.device)
    m.spmm_into(X, Y)
    torch.cuda.synchronize()
    return Y


def _assert_close(Y, w, x, label, block=4096):
    y = Y.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(y)), f"{label}: non-finite output"
    for r0 in range(0, w.shape[0], block):
        y64, s64, _ = oracle.spmm(w[r0:r0 + block], x)
        err = np.abs(y[:, r0:r0 + block] - y64)
        bad = err > 2e-3 * s64 + 1e-5
        if bad.any():
            t, mm = np.argwhere(bad)[0]
            raise AssertionError(f"{label}: {bad.sum()} elements out of tolerance; first (token {t}, row "
                                 f"{r0 + mm}): gpu={y[t, r0 + mm]} ref={y64[t, mm]} S={s64[t, mm]}")


def _dyadic(rows, cols, n, seed, sw):
    rng = np.random.default_rng(seed)
    k = rng.integers(1, 16, size=(rows, cols)).astype(np.float32)
    k *= np.where(rng.integers(0, 2, size=(rows, cols)) == 0, 1.0, -1.0).astype(np.float32)
    w = oracle.magnitude_prune((k * np.float32(2.0 ** -9)).astype(np.float16), sw)
    j = rng.integers(1, 9, size=(n, cols)).astype(np.float32)
    j *= np.where(rng.integers(0, 2, size=(n, cols)) == 0, 1.0, -1.0).astype(np.float32)
    return w, (j * np.float32(0.25)).astype(np.float16)


def _assert_bits(Y, w, x, label, block=4096):
    got = Y.cpu().numpy().view(np.uint16)
    for r0 in range(0, w.shape[0], block):
        y64, _, _ = oracle.spmm(w[r0:r0 + block], x)
        exp = (y64 + 0.0).astype(np.float16).view(np.uint16)
        bad = got[:, r0:r0 + block] != exp
        if bad.any():
            t, mm = np.argwhere(bad)[0]
            raise AssertionError(f"{label}: {bad.sum()} outputs differ; first (token {t}, row {r0 + mm}): "
                                 f"gpu={got[t, r0 + mm]:#06x} ref={exp[t, mm]:#06x}")


SMALL = [
    # rows, cols, tile, sw, n
    (256, 16, (256, 16), 0.5, 1),
    (256, 64, (256, 16), 0.0, 32),
    (333, 517, (256, 16), 0.5, 5),       # ragged rows, cols not a multiple of 8
    (700, 1000, (256, 16), 0.6, 129),    # token tail past one 128-token tile
    (512, 1024, (256, 32), 0.7, 300),
    (1000, 1536, (256, 64), 0.5, 64),
    (1, 40, (256, 16), 0.3, 7),
    (1024, 1024, (256, 16), 0.5, 256),
]


@pytest.mark.parametrize("rows,cols,tile,sw,n", SMALL)
def test_spmm_small_against_oracle(rows, cols, tile, sw, n):
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows * 5 + cols), sw)
    x = synth.laplace_activations(n, cols, cols + n)
    m = spdp.encode(w, tile)
    label = f"spmm {rows}x{cols} tile={tile} sw={sw} N={n}"
    print(f"[gpu] {label}", flush=True)
    _assert_close(_run(m, x), w, x, label)
    m.close()


@pytest.mark.parametrize("rows,cols,tile,sw,n", SMALL)
def test_spmm_small_exact(rows, cols, tile, sw, n):
    w, x = _dyadic(rows, cols, n, rows + 3 * cols + n, sw)
    m = spdp.encode(w, tile)
    label = f"spmm exact {rows}x{cols} tile={tile} sw={sw} N={n}"
    print(f"[gpu] {label}", flush=True)
    _assert_bits(_run(m, x), w, x, label)
    m.close()


FULL = [
    # the Llama projection shapes at prefill lengths
    (4096, 4096, 0.5, 512),
    (11008, 4096, 0.6, 256),
    (4096, 11008, 0.6, 256),
    (5120, 13824, 0.7, 200),
    (28672, 8192, 0.7, 128),
]


@pytest.mark.parametrize("rows,cols,sw,n", FULL)
def test_spmm_full_size_exact_every_row(rows, cols, sw, n):
    w, x = _dyadic(rows, cols, n, rows + cols + n, sw)
    m = spdp.encode(w, (256, 16))
    label = f"spmm exact {rows}x{cols} sw={sw} N={n}"
    print(f"[gpu] {label}", flush=True)
    _assert_bits(_run(m, x), w, x, label)
    m.close()


@pytest.mark.parametrize("rows,cols,sw,n", [(4096, 4096, 0.5, 512), (11008, 4096, 0.6, 384)])
def test_spmm_full_size_realistic(rows, cols, sw, n):
    w = oracle.magnitude_prune(synth.weights(rows, cols, 77 + rows), sw)
    x = synth.laplace_activations(n, cols, 78 + cols)
    m = spdp.encode(w, (256, 16))
    label = f"spmm {rows}x{cols} sw={sw} N={n}"
    print(f"[gpu] {label}", flush=True)
    _assert_close(_run(m, x), w, x, label)
    m.close()


FORCED = [
    ({"SPDP_SPMM_FORM": "2"}, (1000, 1536, 0.5, 300)),
    ({"SPDP_SPMM_FORM": "2"}, (4096, 4096, 0.6, 512)),
    ({"SPDP_SPMM_FORM": "3"}, (700, 1000, 0.5, 100)),
    ({"SPDP_SPMM_FORM": "3"}, (4096, 4096, 0.5, 700)),
    ({"SPDP_SPMM_FORM": "1"}, (1000, 1536, 0.5, 200)),
    ({"SPDP_SPMM_FORM": "1"}, (4096, 4096, 0.5, 300)),
    ({"SPDP_SPMM_SPLITS": "1"}, (1024, 1024, 0.5, 256)),
    ({"SPDP_SPMM_SPLITS": "3"}, (700, 1000, 0.6, 129)),
    ({"SPDP_SPMM_SPLITS": "5"}, (4096, 4096, 0.5, 512)),
    ({"SPDP_SPMM_SPLITS": "1000"}, (333, 520, 0.5, 40)),  # clamped to one GTile per split
]


@pytest.mark.parametrize("env,shape", FORCED, ids=[f"{list(e.items())[0][0]}={list(e.items())[0][1]}-{s[0]}x{s[1]}"
                                                   for e, s in FORCED])
def test_spmm_forced_forms_exact(env, shape, monkeypatch):
    rows, cols, sw, n = shape
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    w, x = _dyadic(rows, cols, n, rows + 5 * cols + n, sw)
    m = spdp.encode(w, (256, 16))
    label = f"spmm exact {rows}x{cols} N={n} {env}"
    print(f"[gpu] {label}", flush=True)
    _assert_bits(_run(m, x), w, x, label)
    m.close()


def test_spmm_wide_needs_several_splits():
    # 40000 columns: 2500 GTiles per stripe, more than one split's LDS table
    # of TileOffsets holds, so the product is split over K whatever the grid
    # (every partial sum < 2^12 in multiples of 2^-11: exact in fp32)
    w, x = _dyadic(300, 40000, 70, 17, 0.5)
    m = spdp.encode(w, (256, 16))
    print("[gpu] spmm exact 300x40000 N=70", flush=True)
    _assert_bits(_run(m, x), w, x, "spmm 300x40000")
    m.close()


def test_spmm_split_workspace_not_grown_in_capture():
    dev = _dev()
    w, x = _dyadic(512, 2048, 64, 23, 0.5)
    m = spdp.encode(w, (256, 16))
    X = _to_dev(x)
    Y = torch.zeros((64, 512), dtype=torch.float16, device=dev)
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    g = torch.cuda.CUDAGraph()
    err = None
    with torch.cuda.graph(g, stream=s):
        try:
            m.spmm_into(X, Y)  # a fresh handle: the split-K workspace would have to grow here
        except spdp.SpdpError as e:
            err = e
        Y.add_(0)
    assert err is not None and err.status == -1, "growing the workspace inside a capture must be refused"
    g.replay()
    torch.cuda.synchronize()
    # eager first, then the same call captured: no growth, the graph replays it
    m.spmm_into(X, Y)
    torch.cuda.synchronize()
    ref = Y.clone()
    _assert_bits(ref, w, x, "eager after refusal")
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=s):
        m.spmm_into(X, Y)
    for _ in range(3):
        Y.fill_(float("nan"))
        g2.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y, ref)
    del g, g2
    m.close()


def test_spmm_repeatable_and_graph_replay():
    dev = _dev()
    w, x = _dyadic(700, 1200, 200, 9, 0.5)
    m = spdp.encode(w, (256, 16))
    X = _to_dev(x)
    Y = torch.zeros((200, 700), dtype=torch.float16, device=dev)
    m.spmm_into(X, Y)
    torch.cuda.synchronize()
    ref = Y.clone()
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        m.spmm_into(X, Y)
    torch.cuda.synchronize()
    for rep in range(3):
        Y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y, ref), f"replay {rep}"
        # the decode path on the same handle between replays
        yd = m(X[:2].contiguous(), -1.0)
        torch.cuda.synchronize()
        assert np.array_equal(yd.cpu().numpy().view(np.uint16), ref[:2].cpu().numpy().view(np.uint16))
    _assert_bits(ref, w, x, "graph reference")
    del g
    m.close()


def test_spmm_argument_errors():
    dev = _dev()
    w = oracle.magnitude_prune(synth.weights(300, 256, 3), 0.5)
    X = torch.zeros((4, 256), dtype=torch.float16, device=dev)
    Y = torch.zeros((4, 300), dtype=torch.float16, device=dev)
    L = spdp.lib()
    for tile in ((128, 16), (256, 8)):
        m = spdp.encode(w, tile)
        with pytest.raises(spdp.SpdpError) as ei:
            m.spmm_into(X, Y)
        assert ei.value.status == -2
        m.close()
    mq = spdp.encode_rtn(w, (256, 16), 4)
    with pytest.raises(spdp.SpdpError) as ei:
        mq.spmm_into(X, Y)
    assert ei.value.status == -2
    mq.close()
    m = spdp.encode(w, (256, 16))
    assert L.spdp_spmm(m._h, ctypes.c_void_p(X.data_ptr()), 0, ctypes.c_void_p(Y.data_ptr()), None) == -1
    assert L.spdp_spmm(m._h, ctypes.c_void_p(X.data_ptr() + 2), 4, ctypes.c_void_p(Y.data_ptr()), None) == -1
    assert L.spdp_spmm(m._h, ctypes.c_void_p(X.data_ptr()), 4, ctypes.c_void_p(X.data_ptr()), None) == -1
    m.close()

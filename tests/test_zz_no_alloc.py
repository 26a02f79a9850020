"""spdp_spmspv_noalloc (through the C ABI) against spdp_spmspv.

The no-allocation entry point runs the same kernel with the same split, so
its outputs must equal spdp_spmspv's bit for bit; only the split-K partials
live elsewhere (the library's static workspace, tagged with a device-wide
call epoch instead of the handle's per-stripe phases). Checked on calls in a
row whose sizes shrink, interleaved across handles that share the static
workspace, replayed from a captured graph, and against the oracle's bound.
"""

import ctypes

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2607_21985_amd as spdp  # noqa: E402

ERR_UNSUPPORTED = -2


def _dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm GPU (torch.cuda.is_available() is False)")
    return torch.device("cuda:0")


def _to_dev(a16):
    return torch.from_numpy(np.ascontiguousarray(a16).view(np.int16)).view(torch.float16).to(_dev())


def _nan_y(m, batch):
    return torch.full((batch, m.rows), float("nan"), dtype=torch.float16, device=_dev())


def _abi_noalloc(m, X, t, Y, stream=None):
    s = stream if stream is not None else torch.cuda.current_stream(X.device)
    return spdp.lib().spdp_spmspv_noalloc(m._h, ctypes.c_void_p(X.data_ptr()), int(X.shape[0]),
                                          ctypes.c_float(t), ctypes.c_void_p(Y.data_ptr()),
                                          ctypes.c_void_p(s.cuda_stream))


def _abi_spmspv(m, X, t, Y):
    s = torch.cuda.current_stream(X.device)
    return spdp.lib().spdp_spmspv(m._h, ctypes.c_void_p(X.data_ptr()), int(X.shape[0]), ctypes.c_float(t),
                                  ctypes.c_void_p(Y.data_ptr()), ctypes.c_void_p(s.cuda_stream))


def _bits(Y):
    return Y.cpu().numpy().view(np.uint16)


def _problem(rows, cols, sw, p, batch, seed):
    w = oracle.magnitude_prune(synth.weights(rows, cols, seed), sw)
    x = synth.laplace_activations(batch, cols, seed + 1)
    return w, x, float(oracle.threshold_for(x, p))


def _compare(m, w, x, t, label):
    X = _to_dev(x)
    Y0, Y1 = _nan_y(m, x.shape[0]), _nan_y(m, x.shape[0])
    print(f"[gpu] noalloc {label}", flush=True)
    assert _abi_noalloc(m, X, t, Y1) == 0, spdp.lib().spdp_last_error()
    assert _abi_spmspv(m, X, t, Y0) == 0, spdp.lib().spdp_last_error()
    torch.cuda.synchronize()
    assert np.array_equal(_bits(Y1), _bits(Y0)), f"{label}: noalloc differs from spdp_spmspv"
    y = Y1.cpu().numpy().astype(np.float64)
    y64, s64, _ = oracle.spmspv(w, x, t)
    assert np.all(np.isfinite(y)), label
    assert np.all(np.abs(y - y64) <= 2e-3 * s64 + 1e-5), f"{label}: outside the oracle's bound"


def test_noalloc_two_calls_second_smaller():
    _dev()
    w, x, t = _problem(4096, 4096, 0.5, 0.5, 4, 7001)
    m = spdp.encode(w, (256, 16))
    _compare(m, w, x, t, "4096x4096 B=4")
    # the second call is smaller: another handle, fewer rows, columns and tokens
    w2, x2, t2 = _problem(1000, 1536, 0.6, 0.25, 1, 7002)
    m2 = spdp.encode(w2, (256, 16))
    _compare(m2, w2, x2, t2, "1000x1536 B=1")
    # and the first handle again with one token
    _compare(m, w, x[:1].copy(), t, "4096x4096 B=1")
    m.close()
    m2.close()


def test_noalloc_interleaved_handles_share_the_workspace():
    # calls of different shapes, batches and tile heights reuse the same
    # partial slots; each must see only its own call's partials
    cases = [(700, 900, (128, 8), 0.5, 0.3, 3), (333, 517, (256, 16), 0.5, 0.5, 1),
             (2048, 2048, (256, 16), 0.7, 0.5, 8), (300, 2048, (64, 1), 0.5, 0.5, 17),
             (512, 1111, (256, 16), 0.6, 0.4, 32)]
    probs = []
    for i, (r, c, tile, sw, p, b) in enumerate(cases):
        w, x, t = _problem(r, c, sw, p, b, 7100 + 10 * i)
        probs.append((spdp.encode(w, tile), w, x, t, f"{r}x{c} tile={tile} B={b}"))
    for rep in range(2):
        for m, w, x, t, label in probs + probs[::-1]:
            _compare(m, w, x, t, f"{label} rep {rep}")
    for m, *_ in probs:
        m.close()


def test_noalloc_one_segment_between_split_calls(monkeypatch):
    # a stripe that one workgroup covers whole writes Y
    # directly and leaves the static workspace's epoch as it was; the calls
    # around it (split, tagged) must still see only their own partials
    w, x, t = _problem(512, 1111, 0.6, 0.4, 32, 7300)
    m = spdp.encode(w, (256, 16))
    w2, x2, t2 = _problem(300, 2048, 0.5, 0.5, 17, 7310)
    m2 = spdp.encode(w2, (128, 16))
    for rep in range(2):
        _compare(m, w, x, t, f"512x1111 B=32 split rep {rep}")
        monkeypatch.setenv("SPDP_PASSES", "64")
        _compare(m, w, x, t, f"512x1111 B=32 one segment rep {rep}")
        _compare(m2, w2, x2, t2, f"300x2048 B=17 one segment rep {rep}")
        monkeypatch.delenv("SPDP_PASSES")
        _compare(m2, w2, x2, t2, f"300x2048 B=17 split rep {rep}")
    m.close()
    m2.close()


def test_noalloc_graph_replay():
    dev = _dev()
    w, x, t = _problem(4096, 4096, 0.6, 0.5, 1, 7201)
    m = spdp.encode(w, (256, 16))
    w2, x2, t2 = _problem(1024, 3000, 0.5, 0.5, 2, 7202)
    m2 = spdp.encode(w2, (256, 16))
    X = _to_dev(x)
    Y = _nan_y(m, 1)
    assert _abi_noalloc(m, X, t, Y) == 0  # eager once before the capture
    torch.cuda.synchronize()
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        assert _abi_noalloc(m, X, t, Y, stream=s) == 0
    torch.cuda.current_stream(dev).wait_stream(s)
    for rep in range(4):
        xr = synth.laplace_activations(1, 4096, 7300 + rep)
        X.copy_(_to_dev(xr))
        Y.fill_(float("nan"))
        g.replay()
        # an eager no-allocation call of another handle between replays
        X2, Y2 = _to_dev(x2), _nan_y(m2, 2)
        assert _abi_noalloc(m2, X2, t2, Y2) == 0
        Yref = _nan_y(m, 1)
        assert _abi_spmspv(m, X, t, Yref) == 0
        torch.cuda.synchronize()
        assert np.array_equal(_bits(Y), _bits(Yref)), f"replay {rep} differs from the eager call"
        y64, s64, _ = oracle.spmspv(w2, x2, t2)
        y2 = Y2.cpu().numpy().astype(np.float64)
        assert np.all(np.abs(y2 - y64) <= 2e-3 * s64 + 1e-5), f"eager call between replays, rep {rep}"
    del g
    m.close()
    m2.close()


def test_noalloc_refuses_more_than_its_workspace(monkeypatch):
    w, x, t = _problem(4096, 8192, 0.5, 0.5, 32, 7401)
    m = spdp.encode(w, (256, 16))
    # 128 segments x 32 tokens x 4096 rows x 8 bytes = 128 MiB of partials
    monkeypatch.setenv("SPDP_SPLITK", "1000")
    monkeypatch.setenv("SPDP_PASSES", "1")
    X = _to_dev(x)
    Y = _nan_y(m, 32)
    assert _abi_noalloc(m, X, t, Y) == ERR_UNSUPPORTED
    assert b"static workspace" in spdp.lib().spdp_last_error()
    torch.cuda.synchronize()
    assert np.all(np.isnan(Y.cpu().numpy().astype(np.float64))), "a refused call wrote its output"
    # the handle's own workspace serves the same product
    Y0 = _nan_y(m, 32)
    assert _abi_spmspv(m, X, t, Y0) == 0
    monkeypatch.delenv("SPDP_SPLITK")
    torch.cuda.synchronize()
    assert np.all(np.isfinite(Y0.cpu().numpy().astype(np.float64)))
    m.close()

"""GPU parity of the low-bit Values form (spdp_encode_rtn): the pruned
weights quantized to round-to-nearest codes (one byte each, one fp32 scale
per row), run through the same kernel, against the oracle's product with the
dequantized weights, y = sum_k (s_m q[m, k]) xm[b, k], to the same bound:

    |Y_gpu - y64| <= 2e-3 * S + 1e-5,   S = sum_k |s_m q[m, k]| |xm[b, k]|,

Y finite and exactly 0 where S = 0."""

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2607_21985_amd as spdp  # noqa: E402

from test_gpu_parity import _assert_close, _dev, _to_dev  # noqa: E402


def _run(m, x, t, mask="token"):
    X = _to_dev(x)
    Y = torch.full((x.shape[0], m.rows), float("nan"), dtype=torch.float16, device=X.device)
    m.spmspv_into(X, t, Y, mask=mask)
    torch.cuda.synchronize()
    return Y.cpu().numpy().astype(np.float64)


def _check(w, x, t, tile, bits, label, mask="token"):
    print(f"[gpu] rtn {label}", flush=True)
    m = spdp.encode_rtn(w, tile, bits)
    y = _run(m, x, t, mask)
    m.close()
    codes, scales, _ = oracle.rtn_quantize(w, bits)
    y64, s64, _ = oracle.spmspv_rtn(codes, scales, x, t, mask)
    _assert_close(y, y64, s64, label)
    return y


CASES = [
    # rows, cols, tile, sw, p, batch, bits
    (64, 64, (64, 64), 0.5, 0.5, 1, 4),
    (1024, 1024, (64, 64), 0.5, 0.5, 1, 4),
    (333, 517, (256, 16), 0.5, 0.5, 1, 4),
    (513, 1000, (256, 16), 0.6, 0.25, 2, 4),
    (256, 4096, (256, 16), 0.7, 0.5, 3, 8),
    (700, 900, (128, 8), 0.5, 0.3, 4, 4),
    (450, 640, (192, 32), 0.4, 0.5, 5, 3),
    (300, 2048, (64, 1), 0.5, 0.5, 8, 4),
    (1000, 1536, (256, 256), 0.5, 0.6, 13, 2),
    (129, 300, (128, 64), 0.5, 0.5, 17, 4),
    (512, 1111, (256, 16), 0.6, 0.4, 32, 4),
    (4096, 4096, (256, 16), 0.5, 0.5, 1, 4),
]


@pytest.mark.parametrize("rows,cols,tile,sw,p,batch,bits", CASES)
def test_rtn_against_oracle(rows, cols, tile, sw, p, batch, bits):
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows * 3 + cols), sw)
    x = synth.laplace_activations(batch, cols, cols * 5 + batch)
    t = float(oracle.threshold_for(x, p))
    _check(w, x, t, tile, bits, f"{rows}x{cols} tile={tile} sw={sw} p={p} B={batch} bits={bits}")


@pytest.mark.parametrize("early", ["0", "1"])
@pytest.mark.parametrize("rows,cols,p,splitk", [(513, 1000, 0.97, None), (1024, 8192, 0.0, 16), (333, 517, 0.5, None)])
def test_rtn_launch_forms(monkeypatch, early, rows, cols, p, splitk):
    monkeypatch.setenv("SPDP_EARLY_FIRST", early)
    if splitk:
        monkeypatch.setenv("SPDP_SPLITK", str(splitk))
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows + 5), 0.5)
    x = synth.laplace_activations(1, cols, cols + 6)
    t = float(oracle.threshold_for(x, p))
    _check(w, x, t, (256, 16), 4, f"early={early} {rows}x{cols} p={p}")


@pytest.mark.parametrize("rows,cols,batch", [(513, 1000, 2), (700, 2048, 8), (300, 1111, 32)])
def test_rtn_batch_mask(rows, cols, batch):
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows + 7), 0.6)
    x = synth.laplace_activations(batch, cols, cols + 8)
    sc = np.sort(oracle.batch_score(x))
    t = float(sc[len(sc) // 2 - 1]) / batch
    _check(w, x, t, (256, 16), 4, f"batch mask {rows}x{cols} B={batch}", mask="batch")


def test_rtn_grouped_matches_single_and_oracle():
    dev = _dev()
    shapes = [(4096, 4096), (1024, 4096), (1024, 4096)]
    ws = [oracle.magnitude_prune(synth.weights(r, c, 1500 + i), 0.5) for i, (r, c) in enumerate(shapes)]
    mats = [spdp.encode_rtn(w, (256, 16), 4) for w in ws]
    x = synth.laplace_activations(1, 4096, 1600)
    t = float(oracle.threshold_for(x, 0.5))
    X = _to_dev(x)
    Yg = [torch.full((1, m.rows), float("nan"), dtype=torch.float16, device=dev) for m in mats]
    print("[gpu] rtn grouped q/k/v", flush=True)
    spdp.spmspv_many(mats, [X] * 3, [t] * 3, Yg)
    torch.cuda.synchronize()
    for i, (w, m, Y) in enumerate(zip(ws, mats, Yg)):
        codes, scales, _ = oracle.rtn_quantize(w, 4)
        y64, s64, _ = oracle.spmspv_rtn(codes, scales, x, t)
        _assert_close(Y.cpu().numpy().astype(np.float64), y64, s64, f"grouped product {i}")
        Ys = torch.full_like(Y, float("nan"))
        m.spmspv_into(X, t, Ys)
        torch.cuda.synchronize()
        assert torch.equal(Ys, Y), f"product {i}: grouped differs from single"
    for m in mats:
        m.close()


def test_rtn_and_fp16_do_not_mix_in_one_launch():
    dev = _dev()
    w = oracle.magnitude_prune(synth.weights(256, 256, 1700), 0.5)
    a, b = spdp.encode(w, (256, 16)), spdp.encode_rtn(w, (256, 16), 4)
    X = _to_dev(synth.laplace_activations(1, 256, 1701))
    Ys = [torch.zeros((1, 256), dtype=torch.float16, device=dev) for _ in range(2)]
    with pytest.raises(spdp.SpdpError) as e:
        spdp.spmspv_many([a, b], [X, X], [0.5, 0.5], Ys)
    assert "codes" in str(e.value)
    a.close()
    b.close()


def test_rtn_edge_cases():
    # rows with nothing stored (scale 0) and nothing active: exact zeros
    w = oracle.magnitude_prune(synth.weights(300, 700, 1800), 0.5).copy()
    w[10:20] = 0
    x = synth.laplace_activations(2, 700, 1801)
    y = _check(w, x, float(oracle.threshold_for(x, 0.5)), (256, 16), 4, "zero rows")
    assert np.all(y[:, 10:20] == 0)
    y = _check(w, x, float(np.abs(x.astype(np.float64)).max()), (256, 16), 4, "nothing active")
    assert np.all(y == 0)
    # every code 0 except one per row (tiny weights next to a large one)
    w2 = np.full((256, 64), np.float16(1e-3))
    w2[:, 5] = np.float16(2.0)
    x2 = synth.laplace_activations(1, 64, 1802)
    _check(w2, x2, -1.0, (256, 16), 4, "codes mostly 0")


@pytest.mark.parametrize("rows,cols,sw,p", [(4096, 4096, 0.5, 0.5), (28672, 8192, 0.7, 0.5), (8192, 28672, 0.7, 0.5)])
def test_rtn_full_size_all_rows(rows, cols, sw, p):
    w = oracle.magnitude_prune(synth.weights(rows, cols, rows // 7 + cols), sw)
    codes, scales, _ = oracle.rtn_quantize(w, 4)
    m = spdp.encode_rtn(w, (256, 16), 4)
    for b in (1, 8):
        x = synth.laplace_activations(b, cols, cols + b)
        t = float(oracle.threshold_for(x, p))
        print(f"[gpu] rtn full size {rows}x{cols} sw={sw} p={p} B={b}", flush=True)
        y = _run(m, x, t)
        assert np.all(np.isfinite(y))
        for r0 in range(0, rows, 2048):
            r1 = min(rows, r0 + 2048)
            y64, s64, _ = oracle.spmspv_rtn(codes[r0:r1], scales[r0:r1], x, t)
            _assert_close(y[:, r0:r1], y64, s64, f"{rows}x{cols} B={b} rows {r0}..{r1 - 1}")
    m.close()

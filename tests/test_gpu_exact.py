"""GPU parity in exact arithmetic: every output bit, every row, full size.

The tolerance-based parity tests cannot see one lost term once a row has
hundreds of active columns (one term is ~1/n of S = sum |w||x|, below the
2e-3 S bound). Here the inputs are chosen so that the kernel's fp32
arithmetic is exact whatever order it adds in:

* weights k * 2^-9 with k uniform in +-{1..15} (fp16-exact), then pruned by
  the oracle's global magnitude pruning -- with only 15 magnitudes the cut
  falls inside a tie class, so the index tie-break decides the pattern at
  full size;
* activations j * 2^-2 with j uniform in +-{1..8}, thresholded at the
  oracle's p-quantile (Sec. 5.1) or by the batch score.

Every product is a multiple of 2^-11 and every partial sum of a row is
bounded by K * 120 * 2^-11 < 2^11 for K <= 28672, so it has at most 22
significant bits: fp32 holds it exactly, in any summation order and split.
The kernel's output must therefore be fp16_RNE(y64) exactly, with y64 the
oracle's float64 product (the masked product of Sec. 2.2, inactive columns
contributing nothing as Sec. 4.2 states). A dropped, duplicated or
misplaced term changes the sum by at least 2^-11 and shows in the fp16
result unless the row's magnitude hides it -- compared over every row of
every shape, some row always shows it.

The low-bit Values form uses weights k * 2^-8, k in +-{1..7}, 4-bit codes:
every row keeps a +-7 after pruning, so the row scale is exactly 2^-8 and
the codes are the k themselves; y = 2^-8 * sum q x is exact too.

Shapes: every projection shape of the five workloads (1024^2 with 64x64
tiles; the Llama-7B, 13B and 70B projections with 256x16), at batch 1 and at
the workload's largest batch, with per-token and batch-shared masks, alone
and as the decoder's grouped launches.
"""

import functools

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2607_21985_amd as spdp  # noqa: E402


def _dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm GPU (torch.cuda.is_available() is False)")
    return torch.device("cuda:0")


def _to_dev(a16):
    return torch.from_numpy(np.ascontiguousarray(a16).view(np.int16)).view(torch.float16).to(_dev())


@functools.lru_cache(maxsize=4)
def _dyadic_weights(rows, cols, seed, levels, exp):
    """fp16 k * 2^exp, k uniform in +-{1..levels} (a seeded test input)."""
    rng = np.random.default_rng(seed)
    k = rng.integers(1, levels + 1, size=(rows, cols), dtype=np.int16)
    k *= np.where(rng.integers(0, 2, size=(rows, cols), dtype=np.int8) == 0, 1, -1).astype(np.int16)
    return (k.astype(np.float32) * np.float32(2.0 ** exp)).astype(np.float16)


@functools.lru_cache(maxsize=4)
def _pruned(rows, cols, seed, sw, levels=15, exp=-9):
    return oracle.magnitude_prune(_dyadic_weights(rows, cols, seed, levels, exp), sw)


def _dyadic_x(batch, cols, seed):
    rng = np.random.default_rng(seed)
    j = rng.integers(1, 9, size=(batch, cols)).astype(np.float32)
    j *= np.where(rng.integers(0, 2, size=(batch, cols)) == 0, 1.0, -1.0).astype(np.float32)
    return (j * np.float32(0.25)).astype(np.float16)


def _batch_t(x, p):
    """t dropping the fraction p of the columns by batch score (oracle side)."""
    s = np.sort(oracle.batch_score(x))
    return -1.0 if p <= 0 else float(s[int(np.ceil(p * s.size)) - 1]) / x.shape[0]


def _expected_bits(w, x, t, mask, rtn=None, block=2048):
    """fp16 bits of the oracle's float64 product, evaluated in row blocks
    (every row); -0 is mapped to +0 (an exact zero sum is +0 in fp32)."""
    rows = w.shape[0]
    out = np.empty((x.shape[0], rows), dtype=np.uint16)
    if rtn is not None:
        codes, scales, _ = rtn
    for r0 in range(0, rows, block):
        r1 = min(rows, r0 + block)
        if rtn is None:
            y64, _ = oracle.spmspv_rows(w, x, t, np.arange(r0, r1), mask)
        else:
            y64, _, _ = oracle.spmspv_rtn(codes[r0:r1], scales[r0:r1], x, t, mask)
        out[:, r0:r1] = (y64 + 0.0).astype(np.float16).view(np.uint16)
    return out


def _assert_bits(y_dev, expect, label):
    got = y_dev.cpu().numpy().view(np.uint16)
    bad = got != expect
    if bad.any():
        b, m = np.argwhere(bad)[0]
        raise AssertionError(
            f"{label}: {int(bad.sum())} of {bad.size} outputs differ; first at (b={b}, m={m}): "
            f"gpu={got.view(np.float16)[b, m]} ref={expect.view(np.float16)[b, m]}")


def _run(m, x, t, mask):
    X = _to_dev(x)
    Y = torch.full((x.shape[0], m.rows), float("nan"), dtype=torch.float16, device=X.device)
    m.spmspv_into(X, t, Y, mask=mask)
    torch.cuda.synchronize()
    return Y


# (label, rows, cols, tile, [(sw, p)], batches, weight seed)
SHAPES = [
    ("single-1024", 1024, 1024, (64, 64), [(0.5, 0.5)], [1], 11),
    ("7b-attn 4096x4096", 4096, 4096, (256, 16), [(0.5, 0.0), (0.7, 0.5)], [1], 12),
    ("7b-gate/up 11008x4096", 11008, 4096, (256, 16), [(0.6, 0.5)], [1, 8], 13),
    ("7b-down 4096x11008", 4096, 11008, (256, 16), [(0.6, 0.5)], [1, 8], 14),
    ("13b-qkvo 5120x5120", 5120, 5120, (256, 16), [(0.7, 0.5)], [1, 16], 15),
    ("13b-gate/up 13824x5120", 13824, 5120, (256, 16), [(0.7, 0.5)], [1, 16], 16),
    ("13b-down 5120x13824", 5120, 13824, (256, 16), [(0.7, 0.5)], [1, 16], 17),
    ("70b-qo 8192x8192", 8192, 8192, (256, 16), [(0.5, 0.0), (0.8, 0.7)], [1, 32], 18),
    ("70b-kv 1024x8192", 1024, 8192, (256, 16), [(0.6, 0.3)], [1, 32], 19),
    ("70b-gate/up 28672x8192", 28672, 8192, (256, 16), [(0.5, 0.0), (0.7, 0.5)], [1, 32], 20),
    ("70b-down 8192x28672", 8192, 28672, (256, 16), [(0.7, 0.5), (0.8, 0.7)], [1, 32], 21),
]


@pytest.mark.parametrize("label,rows,cols,tile,points,batches,seed", SHAPES, ids=[s[0] for s in SHAPES])
def test_exact_every_row(label, rows, cols, tile, points, batches, seed):
    for sw, p in points:
        w = _pruned(rows, cols, seed, sw)
        m = spdp.encode(w, tile)
        for b in batches:
            x = _dyadic_x(b, cols, seed * 100 + b)
            t = float(oracle.threshold_for(x, p))
            lab = f"{label} sw={sw} p={p} B={b} token mask"
            print(f"[gpu-exact] {lab}", flush=True)
            _assert_bits(_run(m, x, t, "token"), _expected_bits(w, x, t, "token"), lab)
            if b > 1:
                tb = _batch_t(x, p)
                lab = f"{label} sw={sw} p={p} B={b} batch mask"
                print(f"[gpu-exact] {lab}", flush=True)
                _assert_bits(_run(m, x, tb, "batch"), _expected_bits(w, x, tb, "batch"), lab)
        m.close()


# one segment per stripe: SPDP_PASSES covers the whole K, so each stripe's
# workgroup adds every column and writes Y itself (no split-K partials);
# a 70B gate/up shape and a ragged one (rows and columns past a tile edge)
@pytest.mark.parametrize("mfma", ["0", "1"], ids=["vector", "mfma32"])
@pytest.mark.parametrize("rows,cols,batch,seed", [(28672, 8192, 32, 20), (1000, 3000, 17, 51)],
                         ids=["28672x8192 B=32", "1000x3000 B=17"])
def test_exact_one_segment(monkeypatch, rows, cols, batch, seed, mfma):
    monkeypatch.setenv("SPDP_PASSES", "64")
    monkeypatch.setenv("SPDP_MFMA", mfma)
    w = _pruned(rows, cols, seed, 0.7)
    m = spdp.encode(w, (256, 16))
    x = _dyadic_x(batch, cols, seed * 100 + batch)
    t = float(oracle.threshold_for(x, 0.5))
    lab = f"{rows}x{cols} B={batch} mfma={mfma} one segment"
    print(f"[gpu-exact] {lab} token mask", flush=True)
    _assert_bits(_run(m, x, t, "token"), _expected_bits(w, x, t, "token"), lab + " token mask")
    tb = _batch_t(x, 0.5)
    print(f"[gpu-exact] {lab} batch mask", flush=True)
    _assert_bits(_run(m, x, tb, "batch"), _expected_bits(w, x, tb, "batch"), lab + " batch mask")
    m.close()


# the decoder's grouped launches (q, k, v; gate, up) at full size
GROUPS = [
    ("7b q/k/v", [(4096, 4096)] * 3, 0.5, 0.5, 1, 31),
    ("7b gate/up", [(11008, 4096)] * 2, 0.6, 0.5, 8, 32),
    ("70b q/k/v", [(8192, 8192), (1024, 8192), (1024, 8192)], 0.7, 0.5, 4, 33),
]


@pytest.mark.parametrize("label,shapes,sw,p,batch,seed", GROUPS, ids=[g[0] for g in GROUPS])
def test_exact_grouped(label, shapes, sw, p, batch, seed):
    cols = shapes[0][1]
    x = _dyadic_x(batch, cols, seed)
    t = float(oracle.threshold_for(x, p))
    ws = [_pruned(r, c, seed + 7 * i, sw) for i, (r, c) in enumerate(shapes)]
    mats = [spdp.encode(w, (256, 16)) for w in ws]
    X = _to_dev(x)
    ys = [torch.full((batch, r), float("nan"), dtype=torch.float16, device=X.device) for r, _ in shapes]
    print(f"[gpu-exact] grouped {label} B={batch}", flush=True)
    spdp.spmspv_many(mats, [X] * len(mats), [t] * len(mats), ys)
    torch.cuda.synchronize()
    for i, (w, y) in enumerate(zip(ws, ys)):
        _assert_bits(y, _expected_bits(w, x, t, "token"), f"grouped {label} product {i}")
    for mm in mats:
        mm.close()


RTN_SHAPES = [
    ("4096x4096", 4096, 4096, 0.5, 0.5, [1], 41),
    ("11008x4096", 11008, 4096, 0.6, 0.5, [1, 8], 42),
    ("5120x13824", 5120, 13824, 0.7, 0.5, [1, 16], 43),
    ("28672x8192", 28672, 8192, 0.7, 0.5, [1, 32], 44),
    ("8192x28672", 8192, 28672, 0.8, 0.7, [1, 32], 45),
]


@pytest.mark.parametrize("label,rows,cols,sw,p,batches,seed", RTN_SHAPES, ids=[s[0] for s in RTN_SHAPES])
def test_exact_rtn_every_row(label, rows, cols, sw, p, batches, seed):
    w = _pruned(rows, cols, seed, sw, levels=7, exp=-8)
    codes, scales, pattern = oracle.rtn_quantize(w, 4)
    # the input design: the scale of every row is 2^-8 and the codes are the
    # weights' own multipliers, so the dequantized weights are W itself
    assert np.all(scales == np.float32(2.0 ** -8)), "a row lost its +-7 weights to pruning"
    m = spdp.encode_rtn(w, (256, 16), 4)
    for b in batches:
        x = _dyadic_x(b, cols, seed * 100 + b)
        t = float(oracle.threshold_for(x, p))
        lab = f"rtn4 {label} sw={sw} p={p} B={b} token mask"
        print(f"[gpu-exact] {lab}", flush=True)
        _assert_bits(_run(m, x, t, "token"), _expected_bits(w, x, t, "token", rtn=(codes, scales, pattern)), lab)
        if b > 1:
            tb = _batch_t(x, p)
            lab = f"rtn4 {label} sw={sw} p={p} B={b} batch mask"
            print(f"[gpu-exact] {lab}", flush=True)
            _assert_bits(_run(m, x, tb, "batch"),
                         _expected_bits(w, x, tb, "batch", rtn=(codes, scales, pattern)), lab)
    m.close()

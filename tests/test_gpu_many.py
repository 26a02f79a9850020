"""GPU parity of the grouped call (spdp_spmspv_many): several independent
products in one launch. Each product is checked against the CPU oracle and
must be bit-identical to the same product run alone (the kernel's summation
order does not depend on what else the launch carries)."""

import ctypes

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2607_21985_amd as spdp  # noqa: E402

from test_gpu_parity import _assert_close, _dev, _to_dev  # noqa: E402


def _products(shapes, sw, p, batch, seed, share_x=False):
    out = []
    x_shared = None
    for i, (rows, cols) in enumerate(shapes):
        w = oracle.magnitude_prune(synth.weights(rows, cols, seed + i), sw)
        if share_x and x_shared is not None and x_shared.shape[1] == cols:
            x = x_shared
        else:
            x = synth.laplace_activations(batch, cols, seed + 100 + i)
            x_shared = x
        t = float(oracle.threshold_for(x, p))
        out.append((w, x, t))
    return out


@pytest.mark.parametrize("shapes,tile,sw,p,batch,share_x", [
    ([(512, 1024), (300, 1024), (1000, 777)], (256, 16), 0.5, 0.5, 1, False),
    ([(4096, 4096), (4096, 4096), (4096, 4096)], (256, 16), 0.6, 0.5, 1, True),   # q, k, v on one input
    ([(1100, 4096), (1100, 4096)], (256, 16), 0.6, 0.5, 3, True),                 # gate, up
    ([(130, 200), (64, 64), (257, 1000), (90, 33), (700, 300)], (64, 8), 0.5, 0.3, 2, False),
    ([(256, 256)] * 8, (128, 16), 0.7, 0.25, 1, False),
    # at 20 tokens the 4096x4096 product walks two K ranges per workgroup and
    # the 300x1024 one a single range: the launch runs the several-range
    # kernel, whose one-range products must keep their single-call bits
    ([(4096, 4096), (300, 1024)], (256, 16), 0.6, 0.5, 20, False),
    # 256x16384 tests 96 columns per wave and range, so from two tokens on
    # the launch runs the 128-column kernels, while the 300x1024 product
    # alone runs the 64-column ones: the same bits either way
    ([(256, 16384), (300, 1024)], (256, 16), 0.6, 0.5, 8, False),
    ([(256, 16384), (300, 1024)], (256, 16), 0.6, 0.5, 20, False),
])
def test_many_matches_oracle_and_single_calls(shapes, tile, sw, p, batch, share_x):
    dev = _dev()
    prods = _products(shapes, sw, p, batch, 900 + len(shapes), share_x)
    mats = [spdp.encode(w, tile) for w, _, _ in prods]
    Xs, xs_by_id = [], {}
    for _, x, _ in prods:
        if id(x) not in xs_by_id:
            xs_by_id[id(x)] = _to_dev(x)
        Xs.append(xs_by_id[id(x)])
    Yg = [torch.full((batch, m.rows), float("nan"), dtype=torch.float16, device=dev) for m in mats]
    print(f"[gpu] many: {len(mats)} products {shapes[:2]}... tile {tile} b={batch}", flush=True)
    spdp.spmspv_many(mats, Xs, [t for _, _, t in prods], Yg)
    torch.cuda.synchronize()
    for i, ((w, x, t), m, X, Y) in enumerate(zip(prods, mats, Xs, Yg)):
        y = Y.cpu().numpy().astype(np.float64)
        y64, s64, _ = oracle.spmspv(w, x, t)
        _assert_close(y, y64, s64, f"product {i}")
        Ys = torch.full_like(Y, float("nan"))
        m.spmspv_into(X, t, Ys)
        torch.cuda.synchronize()
        assert torch.equal(Ys, Y), f"product {i}: grouped result differs from the single call"
    for m in mats:
        m.close()


def test_many_mixes_early_and_plain_first_batches(monkeypatch):
    """One token: a product of at most 1024 workgroups requests each wave's
    first batch before the list is built, a larger one does not; in one
    launch both forms run, and each product still gives the bits of its
    single call. 64 segments make the 4200-row product 17 x 64 = 1088
    workgroups."""
    monkeypatch.setenv("SPDP_SPLITK", "64")
    dev = _dev()
    prods = _products([(4200, 4096), (512, 1024), (1300, 4096)], 0.6, 0.5, 1, 1234)
    mats = [spdp.encode(w, (256, 16)) for w, _, _ in prods]
    Xs = [_to_dev(x) for _, x, _ in prods]
    Yg = [torch.full((1, m.rows), float("nan"), dtype=torch.float16, device=dev) for m in mats]
    print("[gpu] many: mixed first-batch forms", flush=True)
    spdp.spmspv_many(mats, Xs, [t for _, _, t in prods], Yg)
    torch.cuda.synchronize()
    for i, ((w, x, t), m, X, Y) in enumerate(zip(prods, mats, Xs, Yg)):
        y = Y.cpu().numpy().astype(np.float64)
        y64, s64, _ = oracle.spmspv(w, x, t)
        _assert_close(y, y64, s64, f"product {i}")
        Ys = torch.full_like(Y, float("nan"))
        m.spmspv_into(X, t, Ys)
        torch.cuda.synchronize()
        assert torch.equal(Ys, Y), f"product {i}: grouped result differs from the single call"
    for m in mats:
        m.close()


def test_many_batch_mask_matches_oracle_and_single_calls():
    """The batch-shared mask in a grouped launch: every product against the
    oracle and bit-identical to its single call."""
    dev = _dev()
    prods = _products([(700, 1500), (300, 1500), (1300, 900)], 0.6, 0.5, 6, 4321)
    ts = []
    for _, x, _ in prods:
        sc = np.sort(oracle.batch_score(x))
        ts.append(float(sc[int(np.ceil(0.5 * sc.size)) - 1]) / x.shape[0])
    mats = [spdp.encode(w, (256, 16)) for w, _, _ in prods]
    Xs = [_to_dev(x) for _, x, _ in prods]
    Yg = [torch.full((6, m.rows), float("nan"), dtype=torch.float16, device=dev) for m in mats]
    print("[gpu] many: batch mask", flush=True)
    spdp.spmspv_many(mats, Xs, ts, Yg, mask="batch")
    torch.cuda.synchronize()
    for i, ((w, x, _), t, m, X, Y) in enumerate(zip(prods, ts, mats, Xs, Yg)):
        y = Y.cpu().numpy().astype(np.float64)
        y64, s64, _ = oracle.spmspv(w, x, t, "batch")
        _assert_close(y, y64, s64, f"product {i}")
        Ys = torch.full_like(Y, float("nan"))
        m.spmspv_into(X, t, Ys, mask="batch")
        torch.cuda.synchronize()
        assert torch.equal(Ys, Y), f"product {i}: grouped result differs from the single call"
    for m in mats:
        m.close()


def test_many_repeated_and_graph_replayed():
    """Grouped calls back to back, then captured and replayed with eager calls
    in between: every result equals the first eager one."""
    dev = _dev()
    prods = _products([(900, 2100), (600, 2100), (1300, 2100)], 0.5, 0.5, 1, 77, share_x=True)
    mats = [spdp.encode(w, (256, 16)) for w, _, _ in prods]
    X = _to_dev(prods[0][1])
    ts = [t for _, _, t in prods]
    Ys = [torch.zeros((1, m.rows), dtype=torch.float16, device=dev) for m in mats]
    spdp.spmspv_many(mats, [X] * 3, ts, Ys)
    torch.cuda.synchronize()
    ref = [Y.clone() for Y in Ys]
    for rep in range(3):
        spdp.spmspv_many(mats, [X] * 3, ts, Ys)
    torch.cuda.synchronize()
    assert all(torch.equal(Y, R) for Y, R in zip(Ys, ref))
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        spdp.spmspv_many(mats, [X] * 3, ts, Ys)
    torch.cuda.synchronize()
    for rep in range(4):
        print(f"[gpu] grouped graph replay {rep}", flush=True)
        for Y in Ys:
            Y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert all(torch.equal(Y, R) for Y, R in zip(Ys, ref)), f"replay {rep}"
        for m, t in zip(mats, ts):
            m(X, t)
        torch.cuda.synchronize()
    for (w, x, t), R in zip(prods, ref):
        y64, s64, _ = oracle.spmspv(w, x, t)
        _assert_close(R.cpu().numpy().astype(np.float64), y64, s64, "grouped reference")
    del g
    for m in mats:
        m.close()


def test_many_argument_errors_on_device():
    dev = _dev()
    L = spdp.lib()
    w = oracle.magnitude_prune(synth.weights(256, 512, 5), 0.5)
    a, b = spdp.encode(w, (256, 16)), spdp.encode(w, (256, 16))
    c = spdp.encode(w, (128, 16))
    X = torch.zeros((1, 512), dtype=torch.float16, device=dev)
    Y = torch.zeros((2, 256), dtype=torch.float16, device=dev)
    P = ctypes.c_void_p

    def call(hs, xs, ys, ts=(0.0, 0.0)):
        n = len(hs)
        return L.spdp_spmspv_many((P * n)(*[h._h.value for h in hs]), n,
                                  (P * n)(*[x.data_ptr() for x in xs]), 1,
                                  (ctypes.c_float * n)(*ts), (P * n)(*[y.data_ptr() for y in ys]), None)

    y0, y1 = Y[0:1], Y[1:2]
    assert call([a, a], [X, X], [y0, y1]) == -1 and b"twice" in L.spdp_last_error()
    assert call([a, c], [X, X], [y0, y1]) == -1 and b"tile_m" in L.spdp_last_error()
    assert call([a, b], [X, X], [y0, y0]) == -1 and b"overlap" in L.spdp_last_error()
    assert call([a, b], [X, y0], [y0, y1]) == -1 and b"overlap" in L.spdp_last_error()
    assert call([a, b], [X, X], [y0, y1], (0.0, float("nan"))) == -1
    assert call([a, b], [X, X], [y0, y1]) == 0
    torch.cuda.synchronize()
    for m in (a, b, c):
        m.close()


def test_decoder_layer_chain_in_one_graph():
    """A small decoder layer (q/k/v grouped, o, gate/up grouped, down) as one
    captured graph: every replay, with fresh inputs written in place between
    replays, matches the oracle on those inputs."""
    dev = _dev()
    d, f = 768, 2048
    shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "gate": (f, d), "up": (f, d), "down": (d, f)}
    ws = {n: oracle.magnitude_prune(synth.weights(r, c, 700 + i), 0.6) for i, (n, (r, c)) in enumerate(shapes.items())}
    mats = {n: spdp.encode(w, (256, 16)) for n, w in ws.items()}
    batch = 2
    inputs = {"qkv": d, "o": d, "gu": d, "down": f}
    X = {k: torch.zeros((batch, c), dtype=torch.float16, device=dev) for k, c in inputs.items()}
    Y = {n: torch.zeros((batch, r), dtype=torch.float16, device=dev) for n, (r, _) in shapes.items()}
    t = 0.6
    chain = spdp.Chain()
    chain.add([mats["q"], mats["k"], mats["v"]], [X["qkv"]] * 3, [t] * 3, [Y["q"], Y["k"], Y["v"]])
    chain.add(mats["o"], X["o"], t, Y["o"])
    chain.add([mats["gate"], mats["up"]], [X["gu"]] * 2, [t] * 2, [Y["gate"], Y["up"]], mask="batch")
    chain.add(mats["down"], X["down"], t, Y["down"], mask="batch")
    chain.capture()
    src = {"q": "qkv", "k": "qkv", "v": "qkv", "o": "o", "gate": "gu", "up": "gu", "down": "down"}
    mask = {"q": "token", "k": "token", "v": "token", "o": "token", "gate": "batch", "up": "batch", "down": "batch"}
    for rep in range(3):
        print(f"[gpu] chain replay {rep}", flush=True)
        xs = {k: synth.laplace_activations(batch, c, 900 + 10 * rep + i) for i, (k, c) in enumerate(inputs.items())}
        for k, x in xs.items():
            X[k].copy_(torch.from_numpy(x.view(np.int16)).view(torch.float16).to(dev))
        for yv in Y.values():
            yv.fill_(float("nan"))
        chain.replay()
        torch.cuda.synchronize()
        for n in shapes:
            y = Y[n].cpu().numpy().astype(np.float64)
            y64, s64, _ = oracle.spmspv(ws[n], xs[src[n]], t, mask[n])
            _assert_close(y, y64, s64, f"chain replay {rep}, {n}")
    del chain
    for m in mats.values():
        m.close()


def test_many_nothing_active_gives_exact_zeros():
    """A threshold of +inf leaves no column active (the bench's latency-floor
    launches): every product of a grouped launch comes out exactly 0, at one
    token and with both masks at several."""
    dev = _dev()
    shapes = [(4096, 4096), (1000, 4096), (300, 4096)]
    ws = [oracle.magnitude_prune(synth.weights(r, c, 1200 + i), 0.5) for i, (r, c) in enumerate(shapes)]
    mats = [spdp.encode(w, (256, 16)) for w in ws]
    for batch, mask in ((1, "token"), (3, "token"), (3, "batch")):
        print(f"[gpu] many, nothing active: batch {batch}, mask {mask}", flush=True)
        X = _to_dev(synth.laplace_activations(batch, 4096, 1300 + batch))
        Ys = [torch.full((batch, m.rows), float("nan"), dtype=torch.float16, device=dev) for m in mats]
        spdp.spmspv_many(mats, [X] * len(mats), [float("inf")] * len(mats), Ys, mask=mask)
        torch.cuda.synchronize()
        for i, Y in enumerate(Ys):
            assert torch.count_nonzero(Y).item() == 0 and not torch.isnan(Y).any().item(), f"product {i}"
    for m in mats:
        m.close()

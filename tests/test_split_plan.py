"""The split-K plan a call uses (spdp_split_plan, host-side only): every
column lies in exactly one K range, one- and two-token calls and code
values walk one range per workgroup, and larger batches walk 2 or 4 ranges
where the product keeps enough workgroups (the largest P of 4, 2, 1 with
W_P * batch >= 2560 P, W_P = stripes * ceil(segments at one range / P))."""

import ctypes

import numpy as np
import pytest

import paper_2607_21985_amd as spdp

ERR_INVALID = -1

# every projection shape of the Llama 7B/13B/70B workloads and the 70B
# one-GPU share of 8-way tensor parallelism, plus ragged and narrow ones
SHAPES = [(4096, 4096), (11008, 4096), (4096, 11008), (5120, 5120), (13824, 5120), (5120, 13824),
          (8192, 8192), (1024, 8192), (28672, 8192), (8192, 28672), (128, 8192), (8192, 1024),
          (3584, 8192), (8192, 3584), (1000, 3000), (300, 40), (64, 64)]


@pytest.fixture(scope="module")
def plans():
    out = {}
    for rows, cols in SHAPES:
        # the plan depends on the shape and the value form only: zeros encode fastest
        m = spdp.encode_host(np.zeros((rows, cols), np.float16), (256, 16))
        out[(rows, cols)] = (m.format()["n_stripes"], {b: m.split_plan(b) for b in range(1, 33)})
        m.close()
    return out


def _rule(stripes, segs1, batch):
    if batch < 3:
        return 1
    for p in (4, 2):
        if stripes * (-(-segs1 // p)) * batch >= 2560 * p:
            return p
    return 1


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{r}x{c}" for r, c in SHAPES])
def test_every_column_in_exactly_one_range(plans, shape):
    rows, cols = shape
    _, by_batch = plans[shape]
    for b, (segs, wc, passes) in by_batch.items():
        span = passes * 4 * wc  # the columns of one segment
        assert segs >= 1 and 16 <= wc <= 128 and wc % 16 == 0 and passes >= 1, (b, segs, wc, passes)
        assert segs * span >= cols, (b, segs, wc, passes)
        assert (segs - 1) * span < cols, f"B={b}: segment {segs - 1} holds no column"


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{r}x{c}" for r, c in SHAPES])
def test_pass_rule(plans, shape):
    stripes, by_batch = plans[shape]
    segs1, wc1, p1 = by_batch[1]
    assert p1 == 1
    for b, (segs, wc, passes) in by_batch.items():
        assert wc == wc1, "the range width does not depend on the batch"
        assert passes == _rule(stripes, segs1, b), (b, passes)
        assert segs == -(-segs1 // passes), (b, segs)


def test_documented_choices(plans):
    # the choices quoted for the Llama layers: 2 ranges for the large 70B
    # products at 8 and 16 tokens, 4 at 32, k and v (1024 rows) one range;
    # the 13B q and the 7B MLP one range at 8 tokens, two at 32
    P = lambda r, c, b: plans[(r, c)][1][b][2]
    assert [P(28672, 8192, b) for b in (1, 2, 4, 8, 16, 32)] == [1, 1, 1, 2, 2, 4]
    assert [P(8192, 28672, b) for b in (8, 16, 32)] == [2, 2, 4]
    assert [P(8192, 8192, b) for b in (8, 16, 32)] == [2, 2, 4]
    assert [P(1024, 8192, b) for b in (8, 16, 32)] == [1, 1, 1]
    assert [P(5120, 5120, b) for b in (8, 16, 32)] == [1, 1, 2]
    assert [P(13824, 5120, b) for b in (8, 16, 32)] == [2, 2, 4]
    assert [P(11008, 4096, b) for b in (8, 32)] == [1, 2]
    assert [P(4096, 11008, b) for b in (8, 32)] == [1, 2]


def test_codes_and_small_batches_walk_one_range(monkeypatch):
    w = np.zeros((28672, 8192), np.float16)
    w[0, 0] = 1.0  # a row scale that is not 0
    m = spdp.encode_rtn_host(w, (256, 16), 4)
    assert all(m.split_plan(b)[2] == 1 for b in (1, 8, 16, 32))
    monkeypatch.setenv("SPDP_PASSES", "4")
    assert m.split_plan(32)[2] == 1
    m.close()


def test_forced_passes(monkeypatch):
    m = spdp.encode_host(np.zeros((1000, 3000), np.float16), (256, 16))
    segs1, wc, _ = m.split_plan(1)
    monkeypatch.setenv("SPDP_PASSES", "3")
    for b in (1, 2):
        assert m.split_plan(b) == (segs1, wc, 1), "one or two tokens walk one range"
    for b in (3, 8, 17, 32):
        assert m.split_plan(b) == (-(-segs1 // 3), wc, 3)
    monkeypatch.setenv("SPDP_PASSES", "64")
    assert m.split_plan(32) == (1, wc, 64)
    m.close()


def test_invalid_arguments():
    L = spdp.lib()
    out = [ctypes.c_int32(-7) for _ in range(3)]
    refs = [ctypes.byref(o) for o in out]
    assert L.spdp_split_plan(None, 1, *refs) == ERR_INVALID
    m = spdp.encode_host(np.zeros((64, 64), np.float16), (64, 16))
    for b in (0, 33, -1):
        assert L.spdp_split_plan(m._h, b, *refs) == ERR_INVALID
    assert L.spdp_split_plan(m._h, 1, None, refs[1], refs[2]) == ERR_INVALID
    assert [o.value for o in out] == [-7, -7, -7], "a refused call wrote its outputs"
    m.close()


def test_noalloc_workspace_holds_every_llama_projection(plans):
    # the static workspace of spdp_spmspv_noalloc (SPDP_NOALLOC_PARTIAL_BYTES,
    # 40 MiB) holds the partials of every Llama 7B/13B/70B projection at
    # every batch up to 32: 8 bytes x segments x batch x rows rounded up to
    # the 256-row tile
    limit = 40 << 20
    worst = 0
    for (rows, cols), (stripes, by_batch) in plans.items():
        for b, (segs, _, _) in by_batch.items():
            need = 8 * segs * b * stripes * 256
            assert need <= limit, (rows, cols, b, need)
            worst = max(worst, need)
    assert worst == 8 * 22 * 29 * 32 * 256  # 8192x8192 at 29 tokens: 39.9 MiB, the most

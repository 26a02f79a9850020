"""Seeded synthetic inputs for the Tiled-CBC spMspV path.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic (no pruning, no thresholding, no encoding, no product).
Both the CPU oracle's tests and the GPU path's tests and benchmark take their
inputs from here, so that the two sides see the same bits.

Distributions stand in for the paper's workloads (LLM projection matrices at
decode time, Sec. 5.3; activations thresholded TEAL-style, Sec. 2.2 and 5.1):

* weights: N(0, 0.02) entries times a per-input-channel log-normal(0, 0.5)
  scale, rounded once to fp16 (round-to-nearest-even from float64);
* attention-input activations: Laplace(0, 1) with 1 % outlier channels x20,
  the outlier set shared by every token of a batch;
* down-projection inputs: SiLU(g) * u of standard-normal pre-activations.

Every array is returned as ``numpy.float16``. Draw order is fixed as written
so that a (shape, seed) pair always yields the same bits. ``draw`` > 0 gives
further, independent tokens of the same layer (a calibration set or held-out
inputs): their own random stream, the layer's outlier channels kept (those
belong to the layer, as in a trained model); ``draw`` = 0 is the original
draw.
"""

from __future__ import annotations

import dataclasses

import numpy as np

__all__ = [
    "weights",
    "laplace_activations",
    "swiglu_activations",
    "WORKLOADS",
    "Projection",
    "workload",
]


def weights(rows: int, cols: int, seed: int) -> np.ndarray:
    """Dense fp16 weight matrix, row-major ``rows x cols`` (out x in features).

    ``s = lognormal(0, 0.5, cols)`` is one scale per column (input channel),
    ``G = normal(0, 0.02, (rows, cols))``; the result is ``fp16(G * s)``.
    """
    rng = np.random.default_rng(seed)
    s = rng.lognormal(0.0, 0.5, cols)
    g = rng.normal(0.0, 0.02, (rows, cols))
    g *= s[None, :]
    return g.astype(np.float16)


def laplace_activations(batch: int, cols: int, seed: int, draw: int = 0) -> np.ndarray:
    """fp16 activations ``batch x cols``: Laplace(0, 1), 1 % outlier channels x20."""
    rng = np.random.default_rng(seed)
    n_out = int(round(0.01 * cols))
    outliers = rng.choice(cols, n_out, replace=False)
    if draw:
        rng = np.random.default_rng((seed, draw))
    x = rng.laplace(0.0, 1.0, (batch, cols))
    x[:, outliers] *= 20.0
    return x.astype(np.float16)


def swiglu_activations(batch: int, cols: int, seed: int, draw: int = 0) -> np.ndarray:
    """fp16 down-projection inputs ``SiLU(g) * u`` with g, u ~ N(0, 1)."""
    rng = np.random.default_rng((seed, draw) if draw else seed)
    g = rng.normal(0.0, 1.0, (batch, cols))
    u = rng.normal(0.0, 1.0, (batch, cols))
    x = g / (1.0 + np.exp(-g)) * u
    return x.astype(np.float16)


@dataclasses.dataclass(frozen=True)
class Projection:
    """One linear layer of a workload: ``W`` is ``rows x cols``."""

    name: str
    rows: int
    cols: int
    w_seed: int
    x_seed: int
    x_kind: str  # "laplace" or "swiglu"

    def weight(self) -> np.ndarray:
        return weights(self.rows, self.cols, self.w_seed)

    def activations(self, batch: int, draw: int = 0) -> np.ndarray:
        if self.x_kind == "laplace":
            return laplace_activations(batch, self.cols, self.x_seed, draw)
        if self.x_kind == "swiglu":
            return swiglu_activations(batch, self.cols, self.x_seed, draw)
        raise ValueError(f"unknown activation kind {self.x_kind!r}")


def _proj(name, rows, cols, ws, xs, kind="laplace"):
    return Projection(name, rows, cols, ws, xs, kind)


# The five workloads and one tensor-parallel shard: shapes, sweeps and seeds. Tile shapes are the paper's
# 256 x 16 GTile (Sec. 4.1, 4.2.3) except the small single-layer case.
WORKLOADS = {
    "single-1024": dict(
        projections=[_proj("w", 1024, 1024, 101, 102)],
        weight_sparsity=[0.5], act_sparsity=[0.5], batch=[1], tile=(64, 64)),
    "llama7b-attn": dict(
        projections=[_proj("q", 4096, 4096, 201, 211),   # q, k, v read the layer input
                     _proj("k", 4096, 4096, 202, 211),
                     _proj("v", 4096, 4096, 203, 211),
                     _proj("o", 4096, 4096, 204, 212)],  # o reads the attention output
        weight_sparsity=[0.5, 0.6, 0.7], act_sparsity=[0.0, 0.25, 0.5],
        batch=[1], tile=(256, 16)),
    "llama7b-mlp": dict(
        projections=[_proj("gate", 11008, 4096, 301, 311),
                     _proj("up", 11008, 4096, 302, 311),
                     _proj("down", 4096, 11008, 303, 313, "swiglu")],
        weight_sparsity=[0.6], act_sparsity=[0.5], batch=[1, 2, 4, 8],
        tile=(256, 16)),
    "llama13b-layer": dict(
        projections=[_proj("q", 5120, 5120, 401, 411),
                     _proj("k", 5120, 5120, 402, 411),
                     _proj("v", 5120, 5120, 403, 411),
                     _proj("o", 5120, 5120, 404, 412),
                     _proj("gate", 13824, 5120, 405, 413),
                     _proj("up", 13824, 5120, 406, 413),
                     _proj("down", 5120, 13824, 407, 414, "swiglu")],
        weight_sparsity=[0.7], act_sparsity=[0.5], batch=[1, 2, 4, 8, 16],
        tile=(256, 16)),
    "llama70b-layer": dict(
        projections=[_proj("q", 8192, 8192, 501, 511),
                     _proj("k", 1024, 8192, 502, 511),
                     _proj("v", 1024, 8192, 503, 511),
                     _proj("o", 8192, 8192, 504, 512),
                     _proj("gate", 28672, 8192, 505, 513),
                     _proj("up", 28672, 8192, 506, 513),
                     _proj("down", 8192, 28672, 507, 514, "swiglu")],
        weight_sparsity=[0.5, 0.6, 0.7, 0.8],
        act_sparsity=[0.0, 0.1, 0.2, 0.3, 0.4, 0.5, 0.6, 0.7],
        batch=[1, 2, 4, 8, 16, 32], tile=(256, 16)),
    # one GPU's share of the Llama-70B layer under 8-way tensor parallelism:
    # q/k/v and gate/up split their output rows (64 query heads and 8 key /
    # value heads of 128 over 8 GPUs), o and down their input columns; x is
    # the full layer input, o and down read the local attention output and
    # the local SwiGLU activations
    "llama70b-tp8": dict(
        projections=[_proj("q", 1024, 8192, 601, 611),
                     _proj("k", 128, 8192, 602, 611),
                     _proj("v", 128, 8192, 603, 611),
                     _proj("o", 8192, 1024, 604, 612),
                     _proj("gate", 3584, 8192, 605, 613),
                     _proj("up", 3584, 8192, 606, 613),
                     _proj("down", 8192, 3584, 607, 614, "swiglu")],
        weight_sparsity=[0.7], act_sparsity=[0.5],
        batch=[1, 8, 32], tile=(256, 16)),
}


def workload(name: str) -> dict:
    """Return the description of a named workload (see ``WORKLOADS``)."""
    return WORKLOADS[name]

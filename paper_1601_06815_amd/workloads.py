"""Seeded synthetic inputs for the OaA convolution layer.

This module only draws random numbers; it holds none of the convolution's
arithmetic. Both the GPU path's callers and the CPU checks take their inputs
from here, so they see identical arrays.

Recipe: one ``numpy.random.default_rng(seed)`` (PCG64) per workload, drawing
in float64 in the order x, w, g, then rounding each to float32. The paper
(arXiv:1601.06815, Section 3) times synthetic arrays of the sizes it names
(32x32 with 5x5 kernels, 64x64, inputs up to 256x256, and 224x224 with an
8x8 kernel); the named layers below stand in for those and for typical CNN
layers. ``N(0, s)`` below means variance s (fan-in initialisation).
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Layer:
    """One convolution layer: x[B,C,N,N], w[K,C,n,n], valid output of side
    N - n + 1, stride 1."""
    name: str
    B: int
    C: int
    K: int
    N: int
    n: int
    x_dist: str = "uniform"      # "uniform" U[-1,1], "relu_normal" max(N(0,1), 0)
    w_var: float | None = None   # None: 1 / (C n^2)
    g_dist: str = "uniform"      # "uniform" U[-1,1], "normal" N(0,1)
    passes: tuple = ("fwd", "bwd_data", "bwd_filter")

    @property
    def M(self):
        return self.N - self.n + 1

    def direct_flops(self):
        """Multiply-adds of the direct definition, times two, for one pass."""
        return 2.0 * self.B * self.K * self.C * self.M * self.M * self.n * self.n


LAYERS = {
    "tiny": Layer("tiny", 1, 3, 4, 32, 5),
    "plane224_n3": Layer("plane224_n3", 1, 1, 1, 224, 3, w_var=1 / 9, passes=("fwd",)),
    "plane224_n5": Layer("plane224_n5", 1, 1, 1, 224, 5, w_var=1 / 25, passes=("fwd",)),
    "plane224_n8": Layer("plane224_n8", 1, 1, 1, 224, 8, w_var=1 / 64, passes=("fwd",)),
    "first224": Layer("first224", 64, 3, 64, 224, 7, w_var=1 / (3 * 49)),
    "mid56": Layer("mid56", 128, 128, 128, 56, 3, x_dist="relu_normal", w_var=2 / (128 * 9)),
    "large128": Layer("large128", 32, 96, 256, 128, 16, w_var=1 / (96 * 256), g_dist="normal"),
}


def make_inputs(layer: Layer, seed: int = 0, want_g: bool = True, batch: int | None = None):
    """Return float32 arrays (x, w, g) for ``layer``; g is None when not wanted.
    ``batch`` overrides B (the draws then follow the smaller shape)."""
    B = layer.B if batch is None else batch
    rng = np.random.default_rng(seed)
    xs = (B, layer.C, layer.N, layer.N)
    if layer.x_dist == "uniform":
        x = rng.uniform(-1.0, 1.0, xs)
    elif layer.x_dist == "relu_normal":
        x = np.maximum(rng.standard_normal(xs), 0.0)
    else:
        raise ValueError(layer.x_dist)
    var = layer.w_var if layer.w_var is not None else 1.0 / (layer.C * layer.n * layer.n)
    w = rng.standard_normal((layer.K, layer.C, layer.n, layer.n)) * np.sqrt(var)
    g = None
    if want_g:
        gs = (B, layer.K, layer.M, layer.M)
        if layer.g_dist == "uniform":
            g = rng.uniform(-1.0, 1.0, gs)
        elif layer.g_dist == "normal":
            g = rng.standard_normal(gs)
        else:
            raise ValueError(layer.g_dist)
        g = g.astype(np.float32)
    return x.astype(np.float32), w.astype(np.float32), g


def random_layer(rng: np.random.Generator, max_B=3, max_C=5, max_K=5, max_N=40, max_n=12):
    """A random small layer shape for property tests."""
    n = int(rng.integers(1, max_n + 1))
    N = int(rng.integers(n, max(n, max_N) + 1))
    return Layer("random", int(rng.integers(1, max_B + 1)), int(rng.integers(1, max_C + 1)),
                 int(rng.integers(1, max_K + 1)), N, n)

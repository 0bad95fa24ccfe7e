"""Seeded synthetic inputs for the WpAq bipolar-INT GEMM.

Shared by the tests, the smoke check and the benchmark, for both the oracle
and the GPU path.  This module only draws numbers: it holds none of the
method's arithmetic (no conversion, packing or products).

Codes are signed b-bit integers stored as int8 in [-2^(b-1), 2^(b-1) - 1].
"Uniform over the bipolar-INT code set" is the uniform distribution over the
2^b codes.  Scales are drawn as float64 uniforms and cast to float16.

Random streams use numpy's PCG64 (``default_rng``) seeded with a list
``[seed, *sub]`` so that every workload has its own reproducible stream.  Draw
order inside a workload: weight codes, activation codes, weight scales,
activation scales.

The workloads stand in for the LLaMA-class linear layers the paper measures
(7B-class shapes: hidden 4096, MLP 11008); no model weights or datasets are
used.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

HIDDEN = 4096
MLP = 11008

# name -> (N, K) of the 7B-class decoder-layer linear set
LAYER_SHAPES = {
    "q": (HIDDEN, HIDDEN), "k": (HIDDEN, HIDDEN), "v": (HIDDEN, HIDDEN), "o": (HIDDEN, HIDDEN),
    "gate": (MLP, HIDDEN), "up": (MLP, HIDDEN), "down": (HIDDEN, MLP),
}

# (p, q) pairs of the arbitrary-precision sweep on the down-projection shape
SWEEP_BITS = [(1, 1), (1, 4), (2, 8), (3, 3), (3, 8), (4, 8)]


def rng(seed: int, *sub: int) -> np.random.Generator:
    return np.random.default_rng([seed, *sub])


def uniform_codes(g: np.random.Generator, rows: int, K: int, bits: int) -> np.ndarray:
    lo, hi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    return g.integers(lo, hi + 1, size=(rows, K), dtype=np.int64).astype(np.int8)


def gaussian_codes(g: np.random.Generator, rows: int, K: int, bits: int) -> np.ndarray:
    """Codes whose bipolar values 2x+1 follow a rounded Gaussian: t ~ N(0, sigma)
    with sigma a quarter of the value span 2(2^b - 1); x = floor(t / 2), so 2x+1
    is the odd integer nearest to t; then clipped to the b-bit code range."""
    sigma = (2.0 * ((1 << bits) - 1)) / 4.0
    t = g.normal(0.0, sigma, size=(rows, K))
    x = np.floor(t / 2.0)
    lo, hi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    return np.clip(x, lo, hi).astype(np.int8)


def scales(g: np.random.Generator, n: int, lo: float, hi: float) -> np.ndarray:
    return g.uniform(lo, hi, size=n).astype(np.float16)


def fp16_activations(g: np.random.Generator, rows: int, K: int,
                     outlier_frac: float = 0.01) -> np.ndarray:
    """fp16 activations [rows][K] shaped like a decoder layer's linear inputs:
    a Gaussian body whose per-token spread is log-normal (median 1), and a few
    outlier channels (``outlier_frac`` of K, the same channels in every row)
    whose magnitude is 10-50x larger."""
    tok = np.exp(g.normal(0.0, 0.75, size=(rows, 1)))
    x = g.normal(0.0, 1.0, size=(rows, K)) * tok
    n_out = int(round(outlier_frac * K))
    if n_out:
        ch = g.choice(K, size=n_out, replace=False)
        x[:, ch] *= g.uniform(10.0, 50.0, size=n_out)
    return x.astype(np.float16)


W_SCALE_RANGE = (0.005, 0.05)  # per output channel
A_SCALE_RANGE = (0.01, 0.1)    # per token


@dataclass
class Problem:
    """One GEMM problem: C = A W^T with A [M][K] q-bit and W [N][K] p-bit codes."""
    name: str
    M: int
    N: int
    K: int
    p: int
    q: int
    w_codes: np.ndarray
    a_codes: np.ndarray
    w_scale: Optional[np.ndarray] = None
    a_scale: Optional[np.ndarray] = None
    meta: dict = field(default_factory=dict)
    w_zero: Optional[np.ndarray] = None
    a_zero: Optional[np.ndarray] = None

    @property
    def ops(self) -> int:
        """Effective operations 2 M N K."""
        return 2 * self.M * self.N * self.K


def make(name: str, M: int, N: int, K: int, p: int, q: int, g: np.random.Generator,
         act: str = "uniform", with_scales: bool = False) -> Problem:
    w = uniform_codes(g, N, K, p)
    a = uniform_codes(g, M, K, q) if act == "uniform" else gaussian_codes(g, M, K, q)
    ws = scales(g, N, *W_SCALE_RANGE) if with_scales else None
    as_ = scales(g, M, *A_SCALE_RANGE) if with_scales else None
    return Problem(name, M, N, K, p, q, w, a, ws, as_)


def w1a2_small() -> Problem:
    """W1A2, M=16 N=512 K=512, uniform codes, seed 0, int32 output."""
    return make("w1a2_16x512x512", 16, 512, 512, 1, 2, rng(0))


def w2a2_decode(M: int, N: int, K: int = HIDDEN) -> Problem:
    """W2A2 decode GEMM with fp16 scales, seed 2; M in {1, 4, 8},
    (N, K) in {(4096, 4096), (11008, 4096)}."""
    return make("w2a2_decode_m%d_n%d_k%d" % (M, N, K), M, N, K, 2, 2, rng(2, M, N, K),
                with_scales=True)


def w4a4_prefill() -> Problem:
    """W4A4 prefill GEMM, M=2048 N=11008 K=4096, uniform codes, seed 3."""
    return make("w4a4_prefill_2048x11008x4096", 2048, MLP, HIDDEN, 4, 4, rng(3))


def sweep_down(index: int, M: int = 512) -> Problem:
    """Down-projection M=512 N=4096 K=11008 at SWEEP_BITS[index]; uniform weights,
    rounded-Gaussian activations, seed 40 + index."""
    p, q = SWEEP_BITS[index]
    return make("sweep_w%da%d_%dx4096x11008" % (p, q, M), M, HIDDEN, MLP, p, q,
                rng(40 + index), act="gaussian")


def layer_w2a4(layer: str, M: int) -> Problem:
    """One linear of the W2A4 7B-class decoder layer with fp16 scales, seed 5."""
    N, K = LAYER_SHAPES[layer]
    idx = list(LAYER_SHAPES).index(layer)
    return make("w2a4_%s_m%d" % (layer, M), M, N, K, 2, 4, rng(5, idx, M), with_scales=True)


def random_problem(g: np.random.Generator, M: int, N: int, K: int, p: int, q: int,
                   with_scales: bool = False) -> Problem:
    return make("rand_%dx%dx%d_w%da%d" % (M, N, K, p, q), M, N, K, p, q, g,
                with_scales=with_scales)


def zero_points(g: np.random.Generator, scale: np.ndarray, bits: int) -> np.ndarray:
    """Bipolar zero-points z' for bipolar scales s' (fp16): an asymmetric
    quantizer whose grid centre is shifted by up to a quarter of its half
    range s' (2^b - 1), i.e. z' ~ U(-1/4, 1/4) s' (2^b - 1), cast to fp16."""
    half = np.asarray(scale, dtype=np.float64) * ((1 << bits) - 1)
    return (g.uniform(-0.25, 0.25, size=half.shape) * half).astype(np.float16)


def affine_problem(name: str, M: int, N: int, K: int, p: int, q: int,
                   g: np.random.Generator) -> Problem:
    """Codes, fp16 scales and fp16 zero-points of two linear quantizers in
    bipolar form.  Draw order: weight codes, activation codes, weight scales,
    activation scales, weight zeros, activation zeros."""
    prob = make(name, M, N, K, p, q, g, with_scales=True)
    prob.w_zero = zero_points(g, prob.w_scale, p)
    prob.a_zero = zero_points(g, prob.a_scale, q)
    return prob


def layer_w2a4_affine(layer: str, M: int) -> Problem:
    """One linear of the W2A4 7B-class decoder layer with per-channel and
    per-token scales and zero-points, seed 6."""
    N, K = LAYER_SHAPES[layer]
    idx = list(LAYER_SHAPES).index(layer)
    return affine_problem("w2a4_affine_%s_m%d" % (layer, M), M, N, K, 2, 4, rng(6, idx, M))

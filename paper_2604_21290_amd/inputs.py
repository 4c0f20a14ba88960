"""Seeded synthetic inputs shaped like the paper's ViG workloads.

This module is shared by the GPU path's tests/benchmark and by the CPU oracle's
callers.  It holds *no* arithmetic of the method (no normalisation for the
graph, no distances, no selection, no aggregation, no FC): it only draws
numbers and rounds them to the storage dtype.

Every tensor is returned twice: as the exact storage bits handed to the GPU
(float32 array, or uint16 bfloat16 bit patterns) and as the same values
widened exactly to float64 for the oracle, so both sides see identical inputs.

Workloads (the model table of Sec. V-A gives the ViG widths and depths; the
patch grid follows from 224x224 inputs with 16x16 patches for the isotropic
models and the 4x downsampled 56x56 stage-1 grid of the pyramid models):

  single   1 isotropic layer, B=1,  14x14 grid, C=192, fp32, k=9, d=1
  vig_ti   ViG-Ti stack, 12 blocks, B=32, 14x14, C=192, bf16, k=9, d=ceil(l/4)
  vig_b    ViG-B stack, 16 blocks, B=64, 14x14, C=640, bf16, k=9, d=1..4
  pyr_s1   pyramid stage 1, 2 blocks, B=32, 56x56, C=80,  keys pooled r=4, bf16
  pyr_s2   pyramid stage 2, 2 blocks, B=32, 28x28, C=160, keys pooled r=2, bf16
  hires    4 blocks, B=8, 56x56, C=96, full N x N, k=16, d=2, bf16,
           8-component Gaussian mixture laid out in Voronoi regions
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

F32 = "f32"
BF16 = "bf16"


# ----------------------------------------------------------------------------
# dtype rounding (storage only)
# ----------------------------------------------------------------------------
def f64_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float64 -> float32 (RNE) -> bfloat16 (RNE); return uint16 bits."""
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    # round to nearest, ties to even, on the upper 16 bits
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = u + np.uint64(0x7FFF) + lsb
    out = (u >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    u = np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


@dataclasses.dataclass
class Stored:
    """A tensor as stored for the GPU (`bits`) and its exact float64 value."""

    bits: np.ndarray
    value: np.ndarray
    dtype: str

    @property
    def shape(self):
        return self.value.shape


def store(a: np.ndarray, dtype: str) -> Stored:
    if dtype == F32:
        bits = np.ascontiguousarray(np.asarray(a, dtype=np.float64).astype(np.float32))
        return Stored(bits, bits.astype(np.float64), dtype)
    if dtype == BF16:
        bits = f64_to_bf16_bits(a)
        return Stored(bits, bf16_bits_to_f64(bits), dtype)
    raise ValueError(dtype)


def from_bits(bits: np.ndarray, dtype: str) -> Stored:
    """Wrap storage bits read back from a device buffer."""
    if dtype == F32:
        b = np.ascontiguousarray(bits, dtype=np.float32)
        return Stored(b, b.astype(np.float64), dtype)
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return Stored(b, bf16_bits_to_f64(b), dtype)


# ----------------------------------------------------------------------------
# workload registry
# ----------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int           # patch-grid height
    W: int           # patch-grid width
    C: int
    k: int
    dilations: tuple  # one per block (0-based block index)
    dtype: str
    pool_r: int = 1   # key pooling window (1 = keys are the features)
    seed: int = 1
    features: str = "normal_unit"   # or "mixture"

    @property
    def N(self) -> int:
        return self.H * self.W

    @property
    def M(self) -> int:
        return (self.H // self.pool_r) * (self.W // self.pool_r)

    @property
    def L(self) -> int:
        return len(self.dilations)


WORKLOADS = {
    "single": Workload("single", 1, 14, 14, 192, 9, (1,), F32, seed=1),
    "vig_ti": Workload("vig_ti", 32, 14, 14, 192, 9,
                       tuple(math.ceil(l / 4) for l in range(1, 13)), BF16, seed=2),
    "vig_b": Workload("vig_b", 64, 14, 14, 640, 9,
                      tuple(1 + (l // 4) for l in range(16)), BF16, seed=3),
    "pyr_s1": Workload("pyr_s1", 32, 56, 56, 80, 9, (1, 1), BF16, pool_r=4, seed=4),
    "pyr_s2": Workload("pyr_s2", 32, 28, 28, 160, 9, (1, 1), BF16, pool_r=2, seed=41),
    "hires": Workload("hires", 8, 56, 56, 96, 16, (2, 2, 2, 2), BF16, seed=5,
                      features="mixture"),
    # further shapes of the paper's model table and its 448 x 448 inputs
    "vig_ti_448": Workload("vig_ti_448", 32, 28, 28, 192, 9,
                           tuple(math.ceil(l / 4) for l in range(1, 13)), BF16, seed=6),
    "vig_s": Workload("vig_s", 32, 14, 14, 320, 9,
                      tuple(math.ceil(l / 4) for l in range(1, 13)), BF16, seed=7),
    "pyr_s3": Workload("pyr_s3", 32, 14, 14, 400, 9, (1,) * 6, BF16, seed=42),
    "pyr_s4": Workload("pyr_s4", 32, 7, 7, 640, 9, (1, 1), BF16, seed=43),
}


def with_batch(w: Workload, B: int) -> Workload:
    return dataclasses.replace(w, B=B)


# ----------------------------------------------------------------------------
# generators
# ----------------------------------------------------------------------------
def _unit_rows(g: np.random.Generator, shape) -> np.ndarray:
    """N(0,1) rows scaled to unit length (the workload recipe says the input
    patch features are L2-normalised per node; this is data preparation)."""
    a = g.standard_normal(shape)
    return a / np.linalg.norm(a, axis=-1, keepdims=True)


def _mixture(g: np.random.Generator, B: int, H: int, W: int, C: int,
             n_comp: int = 8, sigma: float = 0.5) -> np.ndarray:
    """Per image: n_comp seeded grid sites split the H x W grid into Voronoi
    regions; every node of region c draws mu_c + sigma * N(0, I)."""
    out = np.empty((B, H * W, C))
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    pos = np.stack([yy.ravel(), xx.ravel()], axis=1).astype(np.float64)
    for b in range(B):
        mu = g.standard_normal((n_comp, C))
        sites = np.stack([g.integers(0, H, n_comp), g.integers(0, W, n_comp)], 1)
        d2 = ((pos[:, None, :] - sites[None, :, :]) ** 2).sum(-1)
        comp = np.argmin(d2, axis=1)
        out[b] = mu[comp] + sigma * g.standard_normal((H * W, C))
    return out


def make_features(w: Workload, seed: int | None = None, B: int | None = None) -> Stored:
    g = np.random.default_rng(w.seed if seed is None else seed)
    B = w.B if B is None else B
    if w.features == "mixture":
        a = _mixture(g, B, w.H, w.W, w.C)
    else:
        a = _unit_rows(g, (B, w.N, w.C))
    return store(a, w.dtype)


def make_weight(w: Workload, layer: int, Cout: int | None = None) -> Stored:
    """FC weight W[Cout, 2C], Kaiming-uniform: U(-sqrt(6/fan_in), +sqrt(6/fan_in))
    with fan_in = 2C; seed 1000*workload_seed + layer."""
    Cout = w.C if Cout is None else Cout
    g = np.random.default_rng(1000 * w.seed + layer)
    bound = math.sqrt(6.0 / (2 * w.C))
    return store(g.uniform(-bound, bound, (Cout, 2 * w.C)), w.dtype)


def make_bias(w: Workload, layer: int, Cout: int | None = None, zero: bool = True) -> Stored:
    Cout = w.C if Cout is None else Cout
    if zero:
        return store(np.zeros(Cout), w.dtype)
    g = np.random.default_rng(7000 * w.seed + layer)
    return store(g.uniform(-0.1, 0.1, Cout), w.dtype)


def make_vig_params(w: Workload, layer: int, bias: bool = True) -> dict:
    """Weights of one full ViG block (FC1, MRConv, FC2, FFN 4C), Kaiming-uniform
    per fan-in, as Stored tensors keyed like the oracle's VIG_PARAMS.  W_upd is
    make_weight(w, layer); the others draw from their own seeded streams.  The
    two layers that end a residual branch (W_out, W_2) are scaled by 0.2 so a
    12-block stack without normalisation layers keeps O(1) activations.
    Biases are uniform(-0.1, 0.1) when `bias`, else omitted."""
    C = w.C
    shapes = {"W_in": (C, C), "W_out": (C, C), "W_1": (4 * C, C), "W_2": (C, 4 * C)}
    p = {"W_upd": make_weight(w, layer)}
    for m, (name, shp) in enumerate(sorted(shapes.items())):
        g = np.random.default_rng([w.seed, layer, m, 17])
        bound = math.sqrt(6.0 / shp[1]) * (0.2 if name in ("W_out", "W_2") else 1.0)
        p[name] = store(g.uniform(-bound, bound, shp), w.dtype)
    if bias:
        outs = {"b_in": C, "b_upd": C, "b_out": C, "b_1": 4 * C, "b_2": C}
        for m, (name, n) in enumerate(sorted(outs.items())):
            g = np.random.default_rng([w.seed, layer, m, 29])
            p[name] = store(g.uniform(-0.1, 0.1, n), w.dtype)
    return p


def random_features(seed: int, B: int, N: int, C: int, dtype: str,
                    unit: bool = True) -> Stored:
    """Generic seeded features for edge-case tests."""
    g = np.random.default_rng(seed)
    a = _unit_rows(g, (B, N, C)) if unit else g.standard_normal((B, N, C))
    return store(a, dtype)


def random_weight(seed: int, Cout: int, C: int, dtype: str) -> Stored:
    g = np.random.default_rng(seed)
    bound = math.sqrt(6.0 / (2 * C))
    return store(g.uniform(-bound, bound, (Cout, 2 * C)), dtype)


def random_indices(seed: int, B: int, N: int, k: int, M: int) -> np.ndarray:
    g = np.random.default_rng(seed)
    return g.integers(0, M, (B, N, k)).astype(np.int32)

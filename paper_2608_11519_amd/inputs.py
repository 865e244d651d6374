"""Seeded synthetic inputs for the FLARE++ mixer forward.

This module generates data only: it holds none of the mixer's arithmetic, so
both the float64 oracle (``oracle/``) and the HIP path may draw their inputs
from it without sharing any computation.

Problem statement (Sec. 3.1 and App. A.1 of the paper): tokens
``X in R^{B x N x C}``, five ``C x C`` weights (``W_K, W_V, W~_K, W~_V, W_O``;
Sec. 3.2, Eqs. (7), (9)-(11) and Fig. 1) and the learned seeds
``Q~ in R^{H x M x D}`` with ``D = C / H`` (Sec. 3.2, Eq. (8); App. A.1).

Workload recipes (the paper's benchmarks are not available; these synthetic
inputs stand in for them, with the paper's token counts and widths):

* ``tiny``    B=1, N=1024,  C=64,  H=4, M=32,  fp32.  X ~ N(0, 1).
* ``grid2d``  B=4, N=16384, C=128, H=8, M=128, bf16.  X ~ N(0, 1).  Stands in
  for 2D structured-grid benchmarks (128 x 128 grid tokens).
* ``mesh``    B=2, N=50000, C=256, H=8, M=256, bf16.  X is a random Fourier
  embedding of N uniform points in the unit square plus N(0, 0.1) noise.
  Stands in for irregular-mesh benchmarks (~40K points).
* ``lra``     B=32, N=4096, C=128, H=8, M=64,  bf16.  X is a seeded N(0, 1)
  256 x C embedding table indexed by i.i.d. uniform ids in [0, 256).  Takes
  only the shape of a long-sequence classification layer; no dataset is used.
* ``mesh3d``  B=1, N=2^20, C=128, H=8, M=512, bf16.  X ~ N(0, 1).  The
  paper's 10^6-token single-GPU scale.

Conventions (the paper is silent on these; the readings are fixed here):

* Generator: ``numpy.random.Generator(PCG64(seed))``.  Float64 draws, in this
  order: X (or its ingredients), W_K, W_V, W~_K, W~_V, W_O, seeds.
* Weights: Xavier-uniform, ``U(-a, a)`` with ``a = sqrt(6 / (C + C))``.
  Row-major ``[C_in][C_out]``, applied as ``X @ W``.
* Seeds: ``N(0, 1/D)`` (the second argument is the variance).
* Storage: float64 draws are rounded to float32 (round to nearest even), and
  for the bf16 workloads further to bfloat16 (round to nearest even).  The
  oracle consumes exactly these rounded values, upcast to float64.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "WORKLOAD_ORDER",
    "workload",
    "make_inputs",
    "round_to_bf16",
    "bf16_bits",
    "bits_to_f32",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    N: int
    C: int
    H: int
    M: int
    dtype: str  # "f32" or "bf16"
    x_kind: str  # "normal", "fourier", "embedding"

    @property
    def D(self) -> int:
        return self.C // self.H

    @property
    def tokens(self) -> int:
        return self.B * self.N

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 1, 1024, 64, 4, 32, "f32", "normal"),
    "grid2d": Workload("grid2d", 4, 16384, 128, 8, 128, "bf16", "normal"),
    "mesh": Workload("mesh", 2, 50000, 256, 8, 256, "bf16", "fourier"),
    "lra": Workload("lra", 32, 4096, 128, 8, 64, "bf16", "embedding"),
    "mesh3d": Workload("mesh3d", 1, 1 << 20, 128, 8, 512, "bf16", "normal"),
}
WORKLOAD_ORDER = ["tiny", "grid2d", "mesh", "lra", "mesh3d"]

# Frequency scale of the random Fourier embedding of the "mesh" workload.
FOURIER_SIGMA = 4.0
# Variance of the additive noise of the "mesh" workload.
FOURIER_NOISE_VAR = 0.1
# Size of the embedding table of the "lra" workload.
EMBED_VOCAB = 256


def workload(name: str, **overrides) -> Workload:
    w = WORKLOADS[name]
    return w.replace(**overrides) if overrides else w


# ---------------------------------------------------------------------------
# storage rounding (data preparation, not part of the mixer)
# ---------------------------------------------------------------------------

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); uint16 bits.

    NaN is not expected in generated data and is not special-cased beyond
    keeping it a NaN.
    """
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    out = r.astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Expand bfloat16 bits (uint16) to the float32 values they encode."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Float32 array holding the bfloat16-rounded values of ``a``."""
    return bits_to_f32(bf16_bits(np.asarray(a, dtype=np.float32)))


# ---------------------------------------------------------------------------
# generators
# ---------------------------------------------------------------------------

def _draw_x(w: Workload, rng: np.random.Generator, x_scale: float) -> np.ndarray:
    B, N, C = w.B, w.N, w.C
    if w.x_kind == "normal":
        x = rng.standard_normal((B, N, C))
    elif w.x_kind == "fourier":
        if C % 2:
            raise ValueError("fourier embedding needs an even width")
        pts = rng.random((B, N, 2))
        freq = rng.standard_normal((C // 2, 2)) * FOURIER_SIGMA
        noise = rng.standard_normal((B, N, C)) * np.sqrt(FOURIER_NOISE_VAR)
        ang = 2.0 * np.pi * (pts @ freq.T)
        x = np.concatenate([np.cos(ang), np.sin(ang)], axis=-1) + noise
    elif w.x_kind == "embedding":
        table = rng.standard_normal((EMBED_VOCAB, C))
        ids = rng.integers(0, EMBED_VOCAB, size=(B, N))
        x = table[ids]
    else:
        raise ValueError(f"unknown x_kind {w.x_kind!r}")
    return x * x_scale


def make_inputs(
    w: Workload,
    seed: int = 0,
    *,
    seed_scale: float = 1.0,
    x_scale: float = 1.0,
    zero_seeds: bool = False,
) -> Dict[str, np.ndarray]:
    """Draw one set of mixer inputs.

    Returns float32 arrays holding the stored values (already rounded to the
    workload's storage type): ``X [B,N,C]``, ``Wk, Wv, Wkt, Wvt, Wo [C,C]``,
    ``seeds [H,M,D]``.  ``seed_scale`` and ``x_scale`` build the stress
    variants ("sharp" seeds, "hot" tokens); the scaling is applied to the
    float64 draws before storage rounding.
    """
    if w.C % w.H:
        raise ValueError("C must be a multiple of H")
    rng = np.random.Generator(np.random.PCG64(seed))
    C, H, M, D = w.C, w.H, w.M, w.D
    x = _draw_x(w, rng, x_scale)
    a = np.sqrt(6.0 / (C + C))
    ws = [rng.uniform(-a, a, size=(C, C)) for _ in range(5)]
    seeds = rng.standard_normal((H, M, D)) * np.sqrt(1.0 / D) * seed_scale
    if zero_seeds:
        seeds = np.zeros_like(seeds)

    def store(v: np.ndarray) -> np.ndarray:
        v32 = np.ascontiguousarray(v, dtype=np.float32)
        return round_to_bf16(v32) if w.dtype == "bf16" else v32

    out = {"X": store(x)}
    for name, v in zip(("Wk", "Wv", "Wkt", "Wvt", "Wo"), ws):
        out[name] = store(v)
    out["seeds"] = store(seeds)
    return out


def make_tensor(shape, seed: int, dtype: str = "f32", scale: float = 1.0,
                kind: str = "normal") -> np.ndarray:
    """Standalone seeded tensor (for routing-call tests): N(0, scale^2) draws
    or U(-scale, scale), rounded to the storage type."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if kind == "normal":
        v = rng.standard_normal(shape) * scale
    elif kind == "uniform":
        v = rng.uniform(-scale, scale, size=shape)
    else:
        raise ValueError(kind)
    v32 = np.ascontiguousarray(v, dtype=np.float32)
    return round_to_bf16(v32) if dtype == "bf16" else v32


def describe(w: Workload, seed: int = 0, variant: Optional[str] = None) -> str:
    s = f"{w.name}(B={w.B},N={w.N},C={w.C},H={w.H},M={w.M},{w.dtype},seed={seed}"
    return s + (f",{variant})" if variant else ")")

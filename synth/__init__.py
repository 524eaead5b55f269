"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This module only draws numbers and rounds them to storage formats; it holds none
of the method's arithmetic.  Both the CPU oracle and the HIP path receive
exactly the arrays produced here, so any disagreement between them comes from
their own arithmetic.

Generator: numpy PCG64 via ``numpy.random.default_rng(seed)``, standard normal
draws in float32.  bf16 values are the round-to-nearest-even truncation of the
float32 bit pattern (ties to even, no NaNs are ever drawn).  Weights are
``sigma * draw`` with sigma = 0.02, drawn in float32 before rounding.

The workloads mirror the video-latent shapes of the paper's experiment
appendix (spatial length 4096 = 64x64 latent of a 1024x1024 frame after an
8x VAE and 2x2 patches; hidden 1152, 16 heads of 72 for the 720M model) and
the scaled-down shapes used for correctness cases.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

WEIGHT_SIGMA = 0.02


def rng(seed: int) -> np.random.Generator:
    return np.random.default_rng(seed)


def normal_f32(gen: np.random.Generator, shape, sigma: float = 1.0) -> np.ndarray:
    x = gen.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        x = (x * np.float32(sigma)).astype(np.float32)
    return x


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 values that are exactly representable in bf16 (rounded RNE)."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


# ----------------------------------------------------------------------------
# Workloads
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class Workload:
    name: str
    kind: str            # "chain", "switch", "spatial", "temporal", "block"
    dtype: str           # "f32" or "bf16"
    B: int
    T: int
    S: int
    C: int
    H: int
    n_chunks: int = 1
    F: int = 0           # MLP hidden width (block only)
    seed: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def D(self) -> int:
        return self.C // self.H


WORKLOADS = {
    # tiny spatial-temporal chain in fp32
    "tiny_chain_f32": Workload("tiny_chain_f32", "chain", "f32", B=1, T=4, S=16, C=64, H=4, seed=0),
    # one GPU's T-shard of a 2M-token video latent (T=512 over 8 ranks), switched T->S into 8 chunks
    "switch_bf16_T64_S4096": Workload("switch_bf16_T64_S4096", "switch", "bf16", B=1, T=64, S=4096,
                                      C=1152, H=16, n_chunks=8, seed=1),
    # spatial attention on a temporal shard: 16 frames of 64x64 latent tokens
    "spatial_bf16_B2_T16_S4096": Workload("spatial_bf16_B2_T16_S4096", "spatial", "bf16", B=2, T=16,
                                          S=4096, C=1152, H=16, seed=2),
    # temporal attention on a spatial shard: 512 locations, 128 frames
    "temporal_bf16_B2_S512_T128": Workload("temporal_bf16_B2_S512_T128", "temporal", "bf16", B=2,
                                           T=128, S=512, C=1152, H=16, seed=3),
    # full spatial-temporal block of the 720M model at a 32x32 latent, 32 frames
    "block_bf16_B1_T32_S1024": Workload("block_bf16_B1_T32_S1024", "block", "bf16", B=1, T=32,
                                        S=1024, C=1152, H=16, F=4608, seed=4),
}


def activations(w: Workload, gen: np.random.Generator, shape=None) -> np.ndarray:
    """N(0,1) activations, rounded to bf16 values when the workload is bf16 (kept as float32)."""
    x = normal_f32(gen, shape if shape is not None else (w.B, w.T, w.S, w.C))
    return bf16_round(x) if w.dtype == "bf16" else x


def weight_stored(gen: np.random.Generator, n_out: int, n_in: int, bf16: bool) -> np.ndarray:
    """A weight drawn N(0, 0.02^2) in stored layout [out][in] (row-major, K-contiguous)."""
    w = normal_f32(gen, (n_out, n_in), WEIGHT_SIGMA)
    return bf16_round(w) if bf16 else w


BLOCK_WEIGHT_FIELDS = ("wqkv_s", "bqkv_s", "wo_s", "bo_s", "wqkv_t", "bqkv_t", "wo_t", "bo_t",
                       "w1", "b1", "w2", "b2")


def block_inputs(w: Workload, with_bias: bool = False):
    """Input activation and the twelve block parameters, drawn in field order.

    Weights are returned in stored layout [out][in]; biases (or None) as [out].
    The activation is returned in (B,T,S,C) float32 (bf16-representable values
    for a bf16 workload)."""
    gen = rng(w.seed)
    x = activations(w, gen)
    bf = w.dtype == "bf16"
    C, F = w.C, w.F
    dims = {"wqkv_s": (3 * C, C), "wo_s": (C, C), "wqkv_t": (3 * C, C), "wo_t": (C, C),
            "w1": (F, C), "w2": (C, F)}
    params = {}
    for name in BLOCK_WEIGHT_FIELDS:
        if name.startswith("b"):
            wname = "w" + name[1:]
            n_out = dims[wname][0] if wname in dims else 0
            if with_bias and n_out:
                b = normal_f32(gen, (n_out,), WEIGHT_SIGMA)
                params[name] = bf16_round(b) if bf else b
            else:
                params[name] = None
        else:
            if name in dims and dims[name][0] > 0 and dims[name][1] > 0:
                params[name] = weight_stored(gen, dims[name][0], dims[name][1], bf)
            else:
                params[name] = None
    return x, params


def chain_inputs(w: Workload):
    """Input and the four projection weights of the tiny chain (fp32, stored [out][in])."""
    gen = rng(w.seed)
    x = activations(w, gen)
    C = w.C
    wqkv_s = weight_stored(gen, 3 * C, C, False)
    wo_s = weight_stored(gen, C, C, False)
    wqkv_t = weight_stored(gen, 3 * C, C, False)
    wo_t = weight_stored(gen, C, C, False)
    return x, {"wqkv_s": wqkv_s, "wo_s": wo_s, "wqkv_t": wqkv_t, "wo_t": wo_t}


def qkv_inputs(w: Workload, layout: str):
    """Q, K, V drawn in that order, each (B, X, L, C) in the given layout.

    layout "BTSC" gives (B,T,S,C) (spatial), "BSTC" gives (B,S,T,C) (temporal)."""
    gen = rng(w.seed)
    shape = (w.B, w.T, w.S, w.C) if layout == "BTSC" else (w.B, w.S, w.T, w.C)
    q = activations(w, gen, shape)
    k = activations(w, gen, shape)
    v = activations(w, gen, shape)
    return q, k, v


def switch_input(w: Workload) -> np.ndarray:
    gen = rng(w.seed)
    return activations(w, gen)

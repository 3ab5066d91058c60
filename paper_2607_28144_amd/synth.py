"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

Holds none of the attention arithmetic: only random numbers and the
float32 -> bf16 rounding of them.  The paper's workloads (talking-head clips,
distilled weights) are not available, so i.i.d. N(0, 1) activations at the
paper's window shape stand in for post-normalization q/k/v.

Recipe: ``np.random.default_rng(seed)`` (PCG64), ``standard_normal`` in
float32, drawn in the order the caller asks for (Q, then K, then V, then the
conditioning K and V), each of shape [B, S, H, D]; then round-to-nearest-even
to bf16 by bit manipulation.  The returned arrays are the bf16 bit patterns
(uint16); the same host buffers feed the oracle and the GPU.
"""
from __future__ import annotations

import numpy as np


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(x)
    out = rounded.astype(np.uint16)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal_bf16(rng: np.random.Generator, shape, scale: float = 1.0) -> np.ndarray:
    """bf16 bits of scale * N(0, 1) float32 draws."""
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x = x * np.float32(scale)
    return f32_to_bf16_bits(x)


def qkv(seed: int, B: int, H: int, Sq: int, Skv: int, D: int, ctx: int = 0):
    """Q [B,Sq,H,D], K and V [B,Skv,H,D] (and, if ctx > 0, conditioning K and V
    [B,ctx,H,D] drawn after them), as bf16 bit arrays."""
    rng = np.random.default_rng(seed)
    q = normal_bf16(rng, (B, Sq, H, D))
    k = normal_bf16(rng, (B, Skv, H, D))
    v = normal_bf16(rng, (B, Skv, H, D))
    if ctx > 0:
        kc = normal_bf16(rng, (B, ctx, H, D))
        vc = normal_bf16(rng, (B, ctx, H, D))
        return q, k, v, kc, vc
    return q, k, v


def default_scale(D: int) -> float:
    """1/sqrt(D) rounded to float32 (the value both sides receive)."""
    return float(np.float32(1.0 / np.sqrt(D)))

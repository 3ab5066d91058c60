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


# Parameters of one diffusion-transformer block (model width 1536 = 12 heads
# x 128, feed-forward 8960, six adaLN vectors): name -> shape; linear-layer
# weights are [out, in].
DIT_WIDTH, DIT_HEADS, DIT_FFN = 1536, 12, 8960
DIT_PARAM_SHAPES = {
    "w_mod": (6 * DIT_WIDTH, DIT_WIDTH), "b_mod": (6 * DIT_WIDTH,),
    "w_qkv": (3 * DIT_WIDTH, DIT_WIDTH), "b_qkv": (3 * DIT_WIDTH,), "w_qn": (DIT_WIDTH,), "w_kn": (DIT_WIDTH,),
    "w_o": (DIT_WIDTH, DIT_WIDTH), "b_o": (DIT_WIDTH,),
    "w_n3": (DIT_WIDTH,), "b_n3": (DIT_WIDTH,),
    "w_qc": (DIT_WIDTH, DIT_WIDTH), "b_qc": (DIT_WIDTH,), "w_qcn": (DIT_WIDTH,),
    "w_oc": (DIT_WIDTH, DIT_WIDTH), "b_oc": (DIT_WIDTH,),
    "w_1": (DIT_FFN, DIT_WIDTH), "b_1": (DIT_FFN,),
    "w_2": (DIT_WIDTH, DIT_FFN), "b_2": (DIT_WIDTH,),
}
# per-channel scales of the normalizations: 1 + N(0, 0.02^2) (not N(0, 0.02),
# which would zero the signal); every other parameter N(0, 0.02^2)
DIT_NORM_SCALES = ("w_qn", "w_kn", "w_n3", "w_qcn")


def dit_params(seed: int) -> dict:
    """Synthetic bf16 parameters of one block (bits), in DIT_PARAM_SHAPES
    order from np.random.default_rng(seed): weights and biases N(0, 0.02^2),
    normalization scales 1 + N(0, 0.02^2) (trained weights are not
    available)."""
    rng = np.random.default_rng(seed)
    out = {}
    for name, shape in DIT_PARAM_SHAPES.items():
        x = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(0.02)
        if name in DIT_NORM_SCALES:
            x = x + np.float32(1.0)
        out[name] = f32_to_bf16_bits(x)
    return out


def dit_inputs(seed: int, S: int, S_ctx: int, steps: int = 4):
    """Block inputs: residual stream x float32 [S, 1536] ~ N(0, 1); one
    conditioning vector per denoising step, float32 [steps, 1536] ~ N(0, 1)
    (standing in for the timestep embeddings of the four-step schedule); and
    the context's precomputed key/values, bf16 bits [S_ctx, 12, 128] ~ N(0, 1)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(size=(S, DIT_WIDTH), dtype=np.float32)
    e = rng.standard_normal(size=(steps, DIT_WIDTH), dtype=np.float32)
    kc = normal_bf16(rng, (S_ctx, DIT_HEADS, DIT_WIDTH // DIT_HEADS))
    vc = normal_bf16(rng, (S_ctx, DIT_HEADS, DIT_WIDTH // DIT_HEADS))
    return x, e, kc, vc


def vae_inputs(seed: int, T: int, H: int, W: int, C: int, layers: int = 2):
    """A VAE decoder stage at latent resolution: activations bf16 bits
    [T, H, W, C] ~ N(0, 1) (channels-last), and `layers` causal 3D
    convolutions C -> C as bf16 bits, weights [C, 3, 3, 3, C] ~ N(0, 1 / (27 C))
    (unit gain at initialization) and biases [C] ~ N(0, 0.02^2) (trained VAE
    weights are not available)."""
    rng = np.random.default_rng(seed)
    x = normal_bf16(rng, (T, H, W, C))
    convs = [(normal_bf16(rng, (C, 3, 3, 3, C), float(1.0 / np.sqrt(27 * C))), normal_bf16(rng, (C,), 0.02))
             for _ in range(layers)]
    return x, convs

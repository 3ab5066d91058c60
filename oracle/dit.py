"""Reference oracle of the diffusion-transformer block around the attention --
TEST INFRASTRUCTURE ONLY.

Plain float64 numpy definitions (numpy's matmul is the only library step),
used by the tests, the smoke check and the benchmark's CPU leg; the product
never imports this module and it imports nothing from the product.

What is computed.  The paper's backbone (Sec. 3.4) is the transformer of a
pretrained video diffusion control model, run in bf16 (Sec. 5.1) at four
fixed timesteps; it prints no block formula.  The block below is the
configuration the workload names -- hidden C = 1536 = 12 heads x 128, RMSNorm
on q and k, 3D rotary embedding over (frame, row, column), adaLN
shift/scale/gate from a 1536-vector, self-attention, cross-attention to the
context tokens whose key/values are precomputed off-GPU (Sec. 3.9), and a
GELU(tanh) feed-forward 1536 -> 8960 -> 1536 -- laid out as the standard
adaLN-modulated DiT block (Peebles and Xie, 2023), per token row:

    (sh1, sc1, g1, sh2, sc2, g2) = W_mod silu(e) + b_mod           6 x C
    h1 = LN(x) (1 + sc1) + sh1                                       [bf16]
    q, k, v = split(h1 Wqkv^T + bqkv)                                [bf16]
    q, k = RoPE(RMSNorm_wq(q)), RoPE(RMSNorm_wk(k))                  [bf16]
    x = x + g1 (Attn(q, k, v) Wo^T + bo)                 (Attn out   [bf16])
    h2 = LN_{w3,b3}(x)                                               [bf16]
    qc = RMSNorm_wqc(h2 Wqc^T + bqc)                     (both steps [bf16])
    x = x + (Attn(qc, Kctx, Vctx) Woc^T + boc)           (Attn out   [bf16])
    h3 = LN(x) (1 + sc2) + sh2                                       [bf16]
    f = gelu_tanh(h3 W1^T + b1)                                      [bf16]
    x = x + g2 (f W2^T + b2)

LN is layer normalization over the C channels (biased variance, eps 1e-6),
without affine parameters where modulated and with (w3, b3) before the
cross-attention; RMSNorm and RoPE are oracle.norm_rope's (over all C
channels of a token); Attn is oracle.attn with scale 1/sqrt(128) in float32.
The model runs in bf16: every tensor marked [bf16] is stored rounded to bf16
(round to nearest, ties to even, from the exact float64 value), as the GPU
path stores it; the residual stream x and the modulation vectors stay wide
(float64 here).  Weights and context key/values are bf16 inputs.
"""
from __future__ import annotations

import numpy as np

from . import attn as _attn
from . import norm_rope as _norm_rope

C = 1536          # model width
HEADS = 12
HEAD_DIM = 128
FFN = 8960
EPS = 1e-6
N_MOD = 6         # shift, scale, gate (attention) and shift, scale, gate (feed-forward)


def widen(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exactly."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value of each float64 (ties to even), returned as float64:
    the significand is rounded to 8 bits directly from the exact value."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                       # x = m * 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def to_bits(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of float64 values that are already bf16 values."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def gemm(a: np.ndarray, w: np.ndarray, b: np.ndarray | None = None) -> np.ndarray:
    """a [M, K] times the transpose of w [N, K] (the weight layout of a linear
    layer, one row per output channel), plus an optional bias [N]."""
    y = np.matmul(np.asarray(a, dtype=np.float64), np.asarray(w, dtype=np.float64).T)
    return y if b is None else y + b


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """The tanh form of GELU: x/2 (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def layer_norm(x: np.ndarray, eps: float = EPS, w: np.ndarray | None = None,
               b: np.ndarray | None = None) -> np.ndarray:
    """Normalization of each row to zero mean and unit (biased) variance,
    then the optional per-channel affine map y w + b."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    y = (x - mu) / np.sqrt(var + eps)
    if w is not None:
        y = y * w
    if b is not None:
        y = y + b
    return y


def rms_norm(x: np.ndarray, w: np.ndarray, eps: float = EPS) -> np.ndarray:
    """Each row divided by its root mean square (plus eps), times w."""
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * w


def modulation(e: np.ndarray, w_mod: np.ndarray, b_mod: np.ndarray) -> np.ndarray:
    """The six adaLN vectors of a block from the conditioning vector e [C]:
    W_mod silu(e) + b_mod, as rows (sh1, sc1, g1, sh2, sc2, g2) of [6, C]."""
    return (gemm(silu(np.asarray(e, dtype=np.float64))[None, :], w_mod, b_mod)).reshape(N_MOD, -1)


def modulate(y: np.ndarray, shift: np.ndarray, scale: np.ndarray) -> np.ndarray:
    return y * (1.0 + scale) + shift


def _attention(q: np.ndarray, k_bits: np.ndarray, v_bits: np.ndarray) -> np.ndarray:
    """Attention of bf16-valued q [S, C] over bf16 key/values [Skv, H, D]
    (bits); output [S, C], rounded to bf16."""
    S = q.shape[0]
    scale = float(np.float32(1.0 / np.sqrt(HEAD_DIM)))
    qb = to_bits(q).reshape(1, S, HEADS, HEAD_DIM)
    o, _ = _attn(qb, k_bits.reshape(1, -1, HEADS, HEAD_DIM), v_bits.reshape(1, -1, HEADS, HEAD_DIM), scale)
    return round_bf16(o.reshape(S, C))


def block(x: np.ndarray, e: np.ndarray, p: dict, ctx_k: np.ndarray, ctx_v: np.ndarray, grid,
          token0: int = 0, theta: float = 10000.0, rows=None) -> np.ndarray:
    """One forward of the block.  x: float64 [S, C] residual stream (tokens in
    (frame, row, column) raster order on `grid`); e: [C] conditioning vector;
    p: the block's parameters as bf16 bits (w_* of linear layers [out, in]);
    ctx_k, ctx_v: the context's key/values, bf16 bits [Sctx, H, D].  Returns
    the new x; with `rows` (indices), only those rows of it -- every step but
    the self-attention's keys and values is row by row, and those still come
    from all S rows."""
    x = np.array(x, dtype=np.float64)
    sel = np.arange(x.shape[0]) if rows is None else np.asarray(rows)
    S = x.shape[0]
    W = {n: widen(v) for n, v in p.items()}
    sh1, sc1, g1, sh2, sc2, g2 = modulation(e, W["w_mod"], W["b_mod"])

    # self-attention branch
    h1 = round_bf16(modulate(layer_norm(x), sh1, sc1))
    qkv = round_bf16(gemm(h1, W["w_qkv"], W["b_qkv"]))
    q, k, v = qkv[:, :C], qkv[:, C:2 * C], qkv[:, 2 * C:]
    qr = round_bf16(_norm_rope(to_bits(q).reshape(1, S, HEADS, HEAD_DIM), p["w_qn"], grid, token0, EPS, theta))
    kr = round_bf16(_norm_rope(to_bits(k).reshape(1, S, HEADS, HEAD_DIM), p["w_kn"], grid, token0, EPS, theta))
    a = _attention(qr.reshape(S, C)[sel], to_bits(kr), to_bits(v))
    x = x[sel] + g1 * gemm(a, W["w_o"], W["b_o"])

    # cross-attention branch
    h2 = round_bf16(layer_norm(x, EPS, W["w_n3"], W["b_n3"]))
    qc = round_bf16(gemm(h2, W["w_qc"], W["b_qc"]))
    qc = round_bf16(rms_norm(qc, W["w_qcn"]))
    c = _attention(qc, ctx_k, ctx_v)
    x = x + gemm(c, W["w_oc"], W["b_oc"])

    # feed-forward branch
    h3 = round_bf16(modulate(layer_norm(x), sh2, sc2))
    f = round_bf16(gelu_tanh(gemm(h3, W["w_1"], W["b_1"])))
    return x + g2 * gemm(f, W["w_2"], W["b_2"])

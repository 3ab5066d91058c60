/*
 * regenvc_dit.h -- C ABI of the gfx950 kernels of the diffusion-transformer
 * block that hosts the window attention (the backbone of the paper's
 * four-step decoder, Sec. 3.4, run in bf16, Sec. 5.1), and of the block
 * forward itself.
 *
 * The paper names the backbone but prints no block formula; the block is
 * the adaLN-modulated DiT block of the workload's configuration (hidden C =
 * heads x D, q/k RMSNorm + 3D rotary embedding, adaLN from a C-vector,
 * self-attention, cross-attention to context tokens whose key/values are
 * precomputed off-GPU (Sec. 3.9), GELU-tanh feed-forward C -> F -> C).  Per
 * token row, with tensors marked [bf16] stored rounded to bf16:
 *     (sh1, sc1, g1, sh2, sc2, g2) = W_mod silu(e) + b_mod          (f32)
 *     h1 = LN(x) (1 + sc1) + sh1                                    [bf16]
 *     q, k, v = split(h1 Wqkv^T + bqkv)                             [bf16]
 *     q, k = RoPE(RMSNorm_wq(q)), RoPE(RMSNorm_wk(k))               [bf16]
 *     x = x + g1 (Attn(q, k, v) Wo^T + bo)           (Attn out      [bf16])
 *     h2 = LN_{w3,b3}(x)                                            [bf16]
 *     qc = RMSNorm_wqc(h2 Wqc^T + bqc)               (both steps    [bf16])
 *     x = x + (Attn(qc, Kctx, Vctx) Woc^T + boc)     (Attn out      [bf16])
 *     h3 = LN(x) (1 + sc2) + sh2                                    [bf16]
 *     f = gelu_tanh(h3 W1^T + b1)                                   [bf16]
 *     x = x + g2 (f W2^T + b2)
 * LN: over the C channels, biased variance, eps 1e-6; RMSNorm and RoPE as
 * regenvc_qk_norm_rope (regenvc_attn.h); Attn as regenvc_attn_fwd with scale
 * 1/sqrt(D); gelu_tanh(u) = u/2 (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3))).
 * The residual stream x stays float32.
 *
 * Conventions are those of regenvc_attn.h (status codes, regenvc_last_error,
 * device pointers owned by the caller, validation before any launch, work
 * enqueued on `stream`).  None of these calls allocates: the block forward
 * takes a caller workspace.
 */
#ifndef REGENVC_DIT_H
#define REGENVC_DIT_H

#include <stdint.h>

#include "regenvc_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Epilogues of regenvc_linear_fwd, per output element y = (a W^T)[m][n]: */
#define REGENVC_EPI_BIAS 0          /* out bf16 = y + bias[n]                       */
#define REGENVC_EPI_BIAS_GELU 1     /* out bf16 = gelu_tanh(y + bias[n])            */
#define REGENVC_EPI_GATED_RESIDUAL 2 /* out f32 += gate[n] (y + bias[n]), in place   */

/* A linear layer of the block on bf16 MFMA with fp32 accumulation, its
   pointwise follower fused into the epilogue (the fusion the paper's graph
   compilation step performs, Sec. 3.8):
     a:    bf16 [M, K], row stride lda elements
     w:    bf16 [N, K] contiguous (one row per output channel)
     bias: bf16 [N] or NULL (0)
     gate: f32 [N] or NULL (1); REGENVC_EPI_GATED_RESIDUAL only
     out:  bf16 [M, N] (row stride ldo) for BIAS and BIAS_GELU; f32 [M, N]
           (row stride ldo), read and rewritten, for GATED_RESIDUAL
   M, N, K >= 0; K a multiple of 64; N a multiple of 16; lda, ldo multiples
   of 8 and >= K, N; pointers 16-byte aligned (bias, gate too) -- else
   REGENVC_ERR_UNSUPPORTED.  out must not overlap a, w, bias or gate.  Rows
   go in tiles of 256 or 288 (whichever fills the compute units in fewer
   rounds) by 256 channels. */
regenvc_status regenvc_linear_fwd(const void *a, int64_t lda, const void *w, const void *bias,
                                  const float *gate, void *out, int64_t ldo, int32_t M, int32_t N,
                                  int32_t K, int32_t epilogue, void *stream);

/* Layer normalization of the f32 rows of x [rows, C] (row stride ldx) into
   bf16 y (row stride ldy): LN(x) (1 + scale) + shift with f32 shift, scale
   [C] (the adaLN-modulated form; w, b NULL), or LN(x) w + b with bf16 w, b
   [C] (the affine form; shift, scale NULL).  C a multiple of 512, at most
   2048; eps finite >= 0. */
regenvc_status regenvc_layer_norm_fwd(const float *x, int64_t ldx, void *y, int64_t ldy,
                                      const float *shift, const float *scale, const void *w,
                                      const void *b, int32_t rows, int32_t C, float eps,
                                      void *stream);

/* RMSNorm of bf16 rows: y = x / sqrt(mean(x^2) + eps) w, bf16 w [C]; y may
   be x itself (same pointer and stride).  C a multiple of 512, at most 2048. */
regenvc_status regenvc_rms_norm_fwd(const void *x, int64_t ldx, void *y, int64_t ldy, const void *w,
                                    int32_t rows, int32_t C, float eps, void *stream);

/* adaLN modulation vectors: mod[j] = sum_k w_mod[j][k] silu(e[k]) + b_mod[j],
   j < rows; w_mod bf16 [rows, C], b_mod bf16 [rows], e f32 [C], mod f32
   [rows]. */
regenvc_status regenvc_dit_modulation(const void *w_mod, const void *b_mod, const float *e, float *mod,
                                      int32_t rows, int32_t C, void *stream);

/* The block's parameters (device pointers, bf16): linear weights [out, in],
   biases [out], normalization scales [C]. */
typedef struct {
    const void *w_mod, *b_mod;  /* [6C, C], [6C]  */
    const void *w_qkv, *b_qkv;  /* [3C, C], [3C]  */
    const void *w_qn, *w_kn;    /* [C]            */
    const void *w_o, *b_o;      /* [C, C], [C]    */
    const void *w_n3, *b_n3;    /* [C]            */
    const void *w_qc, *b_qc;    /* [C, C], [C]    */
    const void *w_qcn;          /* [C]            */
    const void *w_oc, *b_oc;    /* [C, C], [C]    */
    const void *w_1, *b_1;      /* [F, C], [F]    */
    const void *w_2, *b_2;      /* [C, F], [C]    */
} regenvc_dit_params;

/* Bytes of workspace regenvc_dit_block_fwd needs for S tokens, S_ctx
   context tokens, width C = heads x D, feed-forward F, on a device with
   n_cu compute units: the modulation vectors, the bf16 activations
   (S x (5 C + F) values) and the attention calls' split-tile scratch.
   Host-only. */
regenvc_status regenvc_dit_block_workspace(int32_t S, int32_t S_ctx, int32_t C, int32_t heads, int32_t F,
                                           int32_t n_cu, int64_t *bytes);

/* One forward of the block over one window: x (f32 [S, C], contiguous) is
   updated in place.  e: f32 [C] conditioning vector of this denoising step;
   ctx_k, ctx_v: bf16 [S_ctx, heads, D] contiguous, the context's
   precomputed key/values; tokens in (frame, row, column) raster order on a
   grid_f x grid_h x grid_w latent grid from token0 (as
   regenvc_qk_norm_rope).  workspace: device, 256-byte aligned, at least
   regenvc_dit_block_workspace bytes, not overlapping any other argument.
   Constraints: S, S_ctx >= 1; D = C / heads in {64, 128}; C a multiple of
   512 (at most 2048); F a multiple of 64.  Allocates nothing. */
regenvc_status regenvc_dit_block_fwd(float *x, const float *e, const regenvc_dit_params *p,
                                     const void *ctx_k, const void *ctx_v, int32_t S_ctx, int32_t S,
                                     int32_t C, int32_t heads, int32_t F, int32_t grid_f, int32_t grid_h,
                                     int32_t grid_w, int32_t token0, void *workspace,
                                     int64_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* REGENVC_DIT_H */

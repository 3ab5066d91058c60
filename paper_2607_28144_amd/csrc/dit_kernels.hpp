// Internal launch interface of the diffusion-transformer block kernels
// (linear layers with fused epilogues, normalizations, adaLN modulation).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace regenvc {

// Epilogue of a linear layer y = a W^T (+ bias), applied per output element:
enum LinearEpi : int32_t {
    kEpiBias = 0,       // out bf16 = y + bias
    kEpiBiasGelu = 1,   // out bf16 = gelu_tanh(y + bias)
    kEpiGatedRes = 2,   // out f32 (in place) = out + gate[n] * (y + bias[n])   (gate may be null: 1)
};

// a: bf16 [M, K] (row stride lda elements), w: bf16 [N, K] contiguous
// (one row per output channel), bias: bf16 [N] or null, gate: f32 [N] or
// null, out: bf16 or f32 [M, N] with row stride ldo elements.
struct LinearArgs {
    const void *a;
    const void *w;
    const void *bias;
    const float *gate;
    void *out;
    int64_t lda, ldo;
    int32_t M, N, K;
    int32_t epi;
};

// Tile rows of the launch the planner picks for this shape on n_cu CUs
// (256 or 288; the tile is that many rows x 256 output channels).
int linear_tile_rows(int M, int N, int n_cu);
hipError_t launch_linear(const LinearArgs &a, hipStream_t stream);

// Row normalization of x (f32 [rows, C], row stride ldx) into bf16 y (row
// stride ldy): LN(x) (1 + scale) + shift with f32 shift/scale [C]
// (modulated), or LN(x) w + b with bf16 w, b [C] (affine).
struct LayerNormArgs {
    const float *x;
    void *y;
    int64_t ldx, ldy;
    const float *shift, *scale;  // modulated form (both set), or
    const void *w, *b;           // affine form (both set)
    int32_t rows, C;
    float eps;
};
hipError_t launch_layer_norm(const LayerNormArgs &a, hipStream_t stream);

// RMSNorm of bf16 rows (row stride ld, in place allowed): y = x / rms(x) w.
struct RmsNormArgs {
    const void *x;
    void *y;
    int64_t ldx, ldy;
    const void *w;  // bf16 [C]
    int32_t rows, C;
    float eps;
};
hipError_t launch_rms_norm(const RmsNormArgs &a, hipStream_t stream);

// adaLN modulation vectors: mod[j] = sum_k w[j][k] silu(e[k]) + b[j],
// j < rows (6 C); w bf16 [rows, C], b bf16 [rows], e f32 [C], mod f32.
struct ModulationArgs {
    const void *w, *b;
    const float *e;
    float *mod;
    int32_t rows, C;
};
hipError_t launch_modulation(const ModulationArgs &a, hipStream_t stream);

}  // namespace regenvc

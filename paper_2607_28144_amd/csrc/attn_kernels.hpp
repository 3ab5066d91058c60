// Internal launch interface between the C ABI layer and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace regenvc {

// One attention launch: Q [B,Sq,H,D], K/V [B,Skv,H,D] (bf16, element strides,
// d contiguous); O [B,Sq,H,D] bf16 or f32; optional f32 LSE [B,H,Sq].
struct AttnArgs {
    const void *q, *k, *v;
    void *o;
    float *lse;  // may be null
    int64_t q_sb, q_ss, q_sh;
    int64_t k_sb, k_ss, k_sh;
    int64_t v_sb, v_ss, v_sh;
    int64_t o_sb, o_ss, o_sh;
    int32_t B, H, Sq, Skv, D;
    bool o_f32;
    float scale;
};

struct MergeArgs {
    const float *o_parts[16];
    const float *lse_parts[16];
    int32_t num_parts;
    void *o;
    float *lse;  // may be null
    int64_t o_sb, o_ss, o_sh;
    int32_t B, H, Sq, D;
    bool o_f32;
};

struct FillArgs {  // empty-chunk partial: O = 0, LSE = -inf
    float *o;
    float *lse;
    int64_t o_sb, o_ss, o_sh;
    int32_t B, H, Sq, D;
};

hipError_t launch_attn(const AttnArgs &a, hipStream_t stream);
hipError_t launch_merge(const MergeArgs &a, hipStream_t stream);
hipError_t launch_empty_partial(const FillArgs &a, hipStream_t stream);

}  // namespace regenvc

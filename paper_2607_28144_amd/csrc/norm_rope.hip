// gfx950 q/k RMSNorm + 3D rotary position embedding: the steps between the
// QKV projection and self-attention in a block of the video diffusion
// transformer, producing the attention kernels' bf16 [B, S, H, D] inputs.
//
// Per token: r = 1/sqrt(mean of the squares of its H*D channels + eps),
// y = x * r * w, then per head a rotation of each (2i, 2i+1) pair by
// pos_a * theta^(-2k/d_a), with pairs split over the frame, row and column
// axes of the latent grid (22/21/21 pairs at D = 128).
//
// HBM-bound: a token's q and k are read once and written once.  One wave
// handles one token, q and k together (they share the rotation angles): each
// lane keeps its 16-byte chunks of both in registers between the sum of
// squares (wave reduction) and the scaled, rotated write-back.
#include "attn_kernels.hpp"

#include <math.h>

namespace regenvc {
namespace {

typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

constexpr int kWavesPerGroup = 1;  // one wave per workgroup: measured fastest (more, smaller workgroups in flight)
constexpr float kInv2Pi = 0.15915494309189535f;

__device__ __forceinline__ float bf16_to_f32(uint16_t b)
{
    return __uint_as_float(((uint32_t)b) << 16);
}

// float -> bf16, round to nearest even (inputs here are finite)
__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

// NCPL: 16-byte chunks per lane and tensor (C = H*D <= 64 * 8 * NCPL).
template <int NCPL>
__global__ __launch_bounds__(64 * kWavesPerGroup) void qk_norm_rope_kernel(NormRopeArgs a)
{
    const int lane = threadIdx.x & 63;
    const int64_t token = (int64_t)blockIdx.x * kWavesPerGroup + (threadIdx.x >> 6);  // over B * S
    if (token >= (int64_t)a.B * a.S) return;  // whole wave
    const int64_t b = token / a.S, t = token % a.S;
    const int D = a.D, C = a.H * a.D, nchunk = C / 8;
    const uint16_t *qi = static_cast<const uint16_t *>(a.q_in) + b * a.qi_sb + t * a.qi_ss;
    const uint16_t *ki = static_cast<const uint16_t *>(a.k_in) + b * a.ki_sb + t * a.ki_ss;

    // pass 1: this lane's chunks of q and k, and their sums of squares
    u16x8 qv[NCPL], kv[NCPL];
    float sq = 0.f, sk = 0.f;
#pragma unroll
    for (int j = 0; j < NCPL; ++j) {
        const int c = lane + 64 * j;
        if (c < nchunk) {
            const int h = (c * 8) / D, d0 = (c * 8) % D;
            qv[j] = *reinterpret_cast<const u16x8 *>(qi + h * a.qi_sh + d0);
            kv[j] = *reinterpret_cast<const u16x8 *>(ki + h * a.ki_sh + d0);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float x = bf16_to_f32(qv[j][e]), y = bf16_to_f32(kv[j][e]);
                sq = fmaf(x, x, sq);
                sk = fmaf(y, y, sk);
            }
        }
    }
    const float rq = 1.0f / sqrtf(wave_sum(sq) / (float)C + a.eps);
    const float rk = 1.0f / sqrtf(wave_sum(sk) / (float)C + a.eps);

    // this token's grid position
    const int64_t g = (int64_t)a.token0 + t;
    const int64_t hw = (int64_t)a.grid_h * a.grid_w;
    const float pos[3] = {(float)(g / hw), (float)((g / a.grid_w) % a.grid_h), (float)(g % a.grid_w)};
    const int P = D / 2, ph = D / 6, pf = P - 2 * ph;

    uint16_t *qo = static_cast<uint16_t *>(a.q_out) + b * a.qo_sb + t * a.qo_ss;
    uint16_t *ko = static_cast<uint16_t *>(a.k_out) + b * a.ko_sb + t * a.ko_ss;
#pragma unroll
    for (int j = 0; j < NCPL; ++j) {
        const int c = lane + 64 * j;
        if (c >= nchunk) continue;
        const int h = (c * 8) / D, d0 = (c * 8) % D;
        const u16x8 wq = *reinterpret_cast<const u16x8 *>(static_cast<const uint16_t *>(a.w_q) + c * 8);
        const u16x8 wk = *reinterpret_cast<const u16x8 *>(static_cast<const uint16_t *>(a.w_k) + c * 8);
        u16x8 oq, ok;
#pragma unroll
        for (int pp = 0; pp < 4; ++pp) {
            const int i = d0 / 2 + pp;  // pair index within the head
            int axis, kk, pairs;
            if (i < pf) {
                axis = 0, kk = i, pairs = pf;
            } else if (i < pf + ph) {
                axis = 1, kk = i - pf, pairs = ph;
            } else {
                axis = 2, kk = i - pf - ph, pairs = ph;
            }
            // angle pos_a * theta^(-2k/d_a), d_a = 2 * pairs, in turns; the
            // hardware sine/cosine take turns, reduced to [0, 1) first (exact)
            const float freq = exp2f(-(float)kk / (float)pairs * a.log2_theta);
            const float turns = __builtin_amdgcn_fractf(pos[axis] * freq * kInv2Pi);
            const float sn = __builtin_amdgcn_sinf(turns), cs = __builtin_amdgcn_cosf(turns);
            const int e0 = 2 * pp, e1 = 2 * pp + 1;
            const float q0 = bf16_to_f32(qv[j][e0]) * rq * bf16_to_f32(wq[e0]);
            const float q1 = bf16_to_f32(qv[j][e1]) * rq * bf16_to_f32(wq[e1]);
            const float k0 = bf16_to_f32(kv[j][e0]) * rk * bf16_to_f32(wk[e0]);
            const float k1 = bf16_to_f32(kv[j][e1]) * rk * bf16_to_f32(wk[e1]);
            oq[e0] = f32_to_bf16(q0 * cs - q1 * sn);
            oq[e1] = f32_to_bf16(q0 * sn + q1 * cs);
            ok[e0] = f32_to_bf16(k0 * cs - k1 * sn);
            ok[e1] = f32_to_bf16(k0 * sn + k1 * cs);
        }
        *reinterpret_cast<u16x8 *>(qo + h * a.qo_sh + d0) = oq;
        *reinterpret_cast<u16x8 *>(ko + h * a.ko_sh + d0) = ok;
    }
}

}  // namespace

hipError_t launch_norm_rope(const NormRopeArgs &a, hipStream_t stream)
{
    const int64_t tokens = (int64_t)a.B * a.S;
    const dim3 grid((unsigned)((tokens + kWavesPerGroup - 1) / kWavesPerGroup)), block(64 * kWavesPerGroup);
    const int nchunk = a.H * a.D / 8;
    if (nchunk <= 64 * 4)
        hipLaunchKernelGGL(qk_norm_rope_kernel<4>, grid, block, 0, stream, a);
    else if (nchunk <= 64 * 16)
        hipLaunchKernelGGL(qk_norm_rope_kernel<16>, grid, block, 0, stream, a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace regenvc

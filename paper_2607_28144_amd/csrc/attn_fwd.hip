// gfx950 blockwise exact attention: bf16 MFMA for Q K^T and P V with fp32
// accumulation, online softmax in registers, K/V tiles double-buffered in LDS.
//
// Method: exact softmax attention computed blockwise over key/value tiles with
// a running (max, sum) per query row -- the "online-softmax" combination the
// paper's Ring attention relies on (Sec. 3.5); a single launch covers one
// GPU's share (a subset of heads, all or a chunk of the keys).
//
// Work decomposition
//   workgroup = 4 waves = one (batch, head, BM-query tile); BM = 4 * 32 * QB.
//   wave      = QB blocks of 32 queries, all head dims, every key tile.
//   key tile  = 64 keys; K and V tiles live in LDS, two buffers.
//
// Layout trick: scores are computed transposed, S^T = K Q^T, with the MFMA
//   v_mfma_f32_32x32x16_bf16 (A = 32 keys x 16 dims from LDS, B = 16 dims x
//   32 queries held in registers).  In the 32x32 accumulator a lane owns ONE
//   query column and 16 of the 32 keys, so row max / row sum are in-register
//   reductions plus one exchange with lane^32 (v_permlane32_swap).  The same
//   accumulator, rounded to bf16, is directly the B operand of O^T = V^T P^T:
//   the MFMA's k-slot -> key assignment it implies is matched by reading V
//   with ds_read_b64_tr_b16 in that key order.  Attention is invariant under
//   a joint permutation of keys and values, so no shuffle is needed.
//
// Lazy rescaling: the running max used as the exponent reference is only
//   raised when a tile's max exceeds it by more than 8 (log2 units); the
//   exponentials are then bounded by 2^8, which fp32 sums and bf16 operands
//   hold exactly as well as values <= 1.  The final O / l and
//   LSE = ln2 * (m_ref + log2 l) are the same quantities for any reference,
//   so this only removes the O-rescale work from the common path.
#include "attn_kernels.hpp"

#include <math.h>

namespace regenvc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) uint16_t lds_u16;

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kBlockN = 64;                 // keys per tile
constexpr float kRescaleThreshold = 8.0f;  // log2 units
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// LDS placement of 16-byte chunk `ch` of tile row `row`.  K rows are read
// 16 B per lane, 32 consecutive rows at one chunk: XOR with the row spreads
// them over distinct banks.  V rows are read with the 8-byte transposing
// load, 4 consecutive rows x 2 adjacent chunks per 16 lanes: XOR with 4*(row%4)
// keeps those 8 (and, with the neighbouring 16 lanes, 16) chunks distinct.
template <int NCH>
__device__ __forceinline__ int k_slot(int row, int ch) { return ch ^ (row & (NCH - 1)); }
template <int NCH>
__device__ __forceinline__ int v_slot(int row, int ch) { return ch ^ ((4 * (row & 3)) & (NCH - 1)); }

// (x of this lane, x of lane^32) combined so both halves hold the same value.
__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D, int QB, bool OUT_F32>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attn_fwd_kernel(AttnArgs a, int n_qtiles)
{
    constexpr int NCH = D / 8;    // 16-byte chunks per row
    constexpr int DS = D / 16;    // k-steps of the Q K^T MFMA
    constexpr int DB = D / 32;    // 32-row blocks of O^T
    constexpr int BM = kWaves * 32 * QB;
    constexpr int LOADS = kBlockN * NCH / kThreads;  // 16-byte chunks per thread per tile
    static_assert(LOADS >= 1 && (kBlockN * NCH) % kThreads == 0, "tile load split");

    __shared__ __attribute__((aligned(16))) uint16_t smem[2][2][kBlockN * D];  // [buf][K|V]

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int hi = lane >> 5;   // which half of the wave
    const int col = lane & 31;  // query column owned in the 32x32 accumulators

    int bid = blockIdx.x;
    const int qt = bid % n_qtiles;
    bid /= n_qtiles;
    const int h = bid % a.H;
    const int b = bid / a.H;
    const int q0 = qt * BM + wave * 32 * QB;

    const uint16_t *qp = static_cast<const uint16_t *>(a.q) + b * a.q_sb + h * a.q_sh;
    const uint16_t *kp = static_cast<const uint16_t *>(a.k) + b * a.k_sb + h * a.k_sh;
    const uint16_t *vp = static_cast<const uint16_t *>(a.v) + b * a.v_sb + h * a.v_sh;
    const int Sq = a.Sq, Skv = a.Skv;

    // Q^T operand fragments stay in registers for the whole key loop.
    bf16x8 qf[QB][DS];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int qi = q0 + qb * 32 + col;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) {
            if (qi < Sq)
                qf[qb][ds] = *reinterpret_cast<const bf16x8 *>(qp + (int64_t)qi * a.q_ss + ds * 16 + hi * 8);
            else
                qf[qb][ds] = bf16x8{};
        }
    }

    f32x16 oacc[QB][DB];
    float mref[QB], lsum[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        mref[qb] = -INFINITY;
        lsum[qb] = 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[qb][db] = f32x16{};
    }
    const float c = a.scale * kLog2e;
    const int ntiles = (Skv + kBlockN - 1) / kBlockN;

    u32x4 kreg[LOADS], vreg[LOADS];
    auto gload = [&](int tile) {
#pragma unroll
        for (int j = 0; j < LOADS; ++j) {
            const int id = threadIdx.x + j * kThreads;
            const int row = id / NCH, ch = id % NCH;
            const int key = tile * kBlockN + row;
            if (key < Skv) {
                kreg[j] = *reinterpret_cast<const u32x4 *>(kp + (int64_t)key * a.k_ss + ch * 8);
                vreg[j] = *reinterpret_cast<const u32x4 *>(vp + (int64_t)key * a.v_ss + ch * 8);
            } else {  // keys past the end: finite zeros, masked out of the softmax below
                kreg[j] = u32x4{};
                vreg[j] = u32x4{};
            }
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int j = 0; j < LOADS; ++j) {
            const int id = threadIdx.x + j * kThreads;
            const int row = id / NCH, ch = id % NCH;
            *reinterpret_cast<u32x4 *>(&smem[buf][0][row * D + k_slot<NCH>(row, ch) * 8]) = kreg[j];
            *reinterpret_cast<u32x4 *>(&smem[buf][1][row * D + v_slot<NCH>(row, ch) * 8]) = vreg[j];
        }
    };

    gload(0);
    lstore(0);
    for (int t = 0; t < ntiles; ++t) {
        __syncthreads();  // tile t visible in buffer t&1; buffer (t+1)&1 free
        const int buf = t & 1;
        if (t + 1 < ntiles) gload(t + 1);

        // S^T = K Q^T for two 32-key blocks
        f32x16 sacc[QB][2];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) sacc[qb][0] = sacc[qb][1] = f32x16{};
        const uint16_t *kt = smem[buf][0];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int row = kb * 32 + col;
#pragma unroll
            for (int ds = 0; ds < DS; ++ds) {
                const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(kt + row * D + k_slot<NCH>(row, ds * 2 + hi) * 8);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    sacc[qb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qb][ds], sacc[qb][kb], 0, 0, 0);
            }
        }

        // Keys of this lane: accumulator register i of block kb holds key
        // kb*32 + (i/4)*8 + hi*4 + i%4 of the tile.
        const bool ragged = (t + 1) * kBlockN > Skv;
        const int kbase = t * kBlockN + hi * 4;

        float mt[QB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = kbase + kb * 32 + (i >> 2) * 8 + (i & 3);
                    const float x = (ragged && key >= Skv) ? -INFINITY : sacc[qb][kb][i];
                    mx = fmaxf(mx, x);
                }
            mt[qb] = pair_max(mx) * c;
        }
        bool need = false;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) need |= mt[qb] > mref[qb] + kRescaleThreshold;
        if (__builtin_amdgcn_ballot_w64(need) != 0) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                const float mnew = fmaxf(mref[qb], mt[qb]);
                const float alpha = __builtin_amdgcn_exp2f(mref[qb] - mnew);
                lsum[qb] *= alpha;
#pragma unroll
                for (int db = 0; db < DB; ++db) oacc[qb][db] *= alpha;
                mref[qb] = mnew;
            }
        }

        // P^T fragments (bf16) and row sums.
        bf16x8 pf[QB][4];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const float nm = -mref[qb];
            float ls = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = kbase + kb * 32 + (i >> 2) * 8 + (i & 3);
                    float p = __builtin_amdgcn_exp2f(fmaf(sacc[qb][kb][i], c, nm));
                    if (ragged && key >= Skv) p = 0.f;
                    ls += p;
                    pf[qb][kb * 2 + (i >> 3)][i & 7] = (__bf16)p;
                }
            lsum[qb] += ls;
        }

        // O^T += V^T P^T.  MFMA k-step kk covers tile keys 16kk..16kk+15; the
        // lower half-wave supplies keys {0-3, 8-11}, the upper {4-7, 12-15}.
        const uint16_t *vt = smem[buf][1];
        const int g = lane >> 4, x = lane & 15;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int dcol = db * 32 + 16 * (g & 1) + 4 * (x & 3);  // first of 4 dims this lane fetches
                bf16x8 vf;
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const int row = kk * 16 + 4 * (g >> 1) + 8 * half + (x >> 2);
                    const int off = row * D + v_slot<NCH>(row, dcol >> 3) * 8 + (dcol & 7);
                    const bf16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                        (lds_bf16x4 *)((lds_u16 *)vt + off));
                    vf[half * 4 + 0] = r[0];
                    vf[half * 4 + 1] = r[1];
                    vf[half * 4 + 2] = r[2];
                    vf[half * 4 + 3] = r[3];
                }
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    oacc[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qb][kk], oacc[qb][db], 0, 0, 0);
            }
        }

        if (t + 1 < ntiles) lstore((t + 1) & 1);
    }

    // Epilogue: O = O^T / l, LSE = ln2 * (m_ref + log2 l).
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const float lt = pair_sum(lsum[qb]);
        const float inv = 1.0f / lt;
        const int qi = q0 + qb * 32 + col;
        if (qi < Sq) {
            char *orow = static_cast<char *>(a.o) +
                         ((int64_t)b * a.o_sb + (int64_t)qi * a.o_ss + (int64_t)h * a.o_sh) * (OUT_F32 ? 4 : 2);
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    const int d = db * 32 + gq * 8 + hi * 4;
                    if constexpr (OUT_F32) {
                        f32x4 w;
#pragma unroll
                        for (int e = 0; e < 4; ++e) w[e] = oacc[qb][db][gq * 4 + e] * inv;
                        *reinterpret_cast<f32x4 *>(orow + d * 4) = w;
                    } else {
                        bf16x4 w;
#pragma unroll
                        for (int e = 0; e < 4; ++e) w[e] = (__bf16)(oacc[qb][db][gq * 4 + e] * inv);
                        *reinterpret_cast<bf16x4 *>(orow + d * 2) = w;
                    }
                }
            if (a.lse != nullptr && hi == 0)
                a.lse[((int64_t)b * a.H + h) * Sq + qi] = (mref[qb] + __log2f(lt)) * kLn2;
        }
    }
}

template <int D, int QB, bool OUT_F32>
hipError_t launch_attn_t(const AttnArgs &a, hipStream_t stream)
{
    constexpr int BM = kWaves * 32 * QB;
    const int n_qtiles = (a.Sq + BM - 1) / BM;
    const int64_t nblocks = (int64_t)n_qtiles * a.H * a.B;
    if (nblocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((attn_fwd_kernel<D, QB, OUT_F32>), dim3((unsigned)nblocks), dim3(kThreads), 0, stream, a,
                       n_qtiles);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Log-sum-exp merge of chunk partials: one thread per 4 dims of one row.
template <bool OUT_F32>
__global__ __launch_bounds__(256) void lse_merge_kernel(MergeArgs a)
{
    const int per_row = a.D / 4;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t rows = (int64_t)a.B * a.Sq * a.H;
    const int64_t row = gid / per_row;  // row index in [B, Sq, H] order
    if (row >= rows) return;
    const int d = (int)(gid % per_row) * 4;
    const int h = (int)(row % a.H);
    const int64_t bi = row / a.H;
    const int i = (int)(bi % a.Sq);
    const int b = (int)(bi / a.Sq);
    const int64_t li = ((int64_t)b * a.H + h) * a.Sq + i;

    float m = -INFINITY;
    for (int c = 0; c < a.num_parts; ++c) m = fmaxf(m, a.lse_parts[c][li]);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float L = -INFINITY;
    if (m != -INFINITY) {
        float s = 0.f;
        for (int c = 0; c < a.num_parts; ++c) s += expf(a.lse_parts[c][li] - m);
        L = m + logf(s);
        for (int c = 0; c < a.num_parts; ++c) {
            const float w = expf(a.lse_parts[c][li] - L);
            const f32x4 oc = *reinterpret_cast<const f32x4 *>(a.o_parts[c] + row * a.D + d);
            acc += w * oc;
        }
    }
    char *orow = static_cast<char *>(a.o) + ((int64_t)b * a.o_sb + (int64_t)i * a.o_ss + (int64_t)h * a.o_sh) *
                                                (OUT_F32 ? 4 : 2);
    if constexpr (OUT_F32) {
        *reinterpret_cast<f32x4 *>(orow + d * 4) = acc;
    } else {
        bf16x4 w;
        for (int e = 0; e < 4; ++e) w[e] = (__bf16)acc[e];
        *reinterpret_cast<bf16x4 *>(orow + d * 2) = w;
    }
    if (a.lse != nullptr && d == 0) a.lse[li] = L;
}

__global__ __launch_bounds__(256) void empty_partial_kernel(FillArgs a)
{
    const int per_row = a.D / 4;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t rows = (int64_t)a.B * a.Sq * a.H;
    const int64_t row = gid / per_row;
    if (row >= rows) return;
    const int d = (int)(gid % per_row) * 4;
    const int h = (int)(row % a.H);
    const int64_t bi = row / a.H;
    const int i = (int)(bi % a.Sq);
    const int b = (int)(bi / a.Sq);
    float *orow = a.o + (int64_t)b * a.o_sb + (int64_t)i * a.o_ss + (int64_t)h * a.o_sh;
    *reinterpret_cast<f32x4 *>(orow + d) = f32x4{0.f, 0.f, 0.f, 0.f};
    if (d == 0) a.lse[((int64_t)b * a.H + h) * a.Sq + i] = -INFINITY;
}

}  // namespace

hipError_t launch_attn(const AttnArgs &a, hipStream_t stream)
{
    if (a.D == 128)
        return a.o_f32 ? launch_attn_t<128, 2, true>(a, stream) : launch_attn_t<128, 2, false>(a, stream);
    if (a.D == 64)
        return a.o_f32 ? launch_attn_t<64, 2, true>(a, stream) : launch_attn_t<64, 2, false>(a, stream);
    return hipErrorInvalidValue;
}

static int64_t elementwise_blocks(int64_t rows, int D)
{
    return (rows * (D / 4) + 255) / 256;
}

hipError_t launch_merge(const MergeArgs &a, hipStream_t stream)
{
    const int64_t nb = elementwise_blocks((int64_t)a.B * a.Sq * a.H, a.D);
    if (nb > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (a.o_f32)
        hipLaunchKernelGGL(lse_merge_kernel<true>, dim3((unsigned)nb), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(lse_merge_kernel<false>, dim3((unsigned)nb), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_empty_partial(const FillArgs &a, hipStream_t stream)
{
    const int64_t nb = elementwise_blocks((int64_t)a.B * a.Sq * a.H, a.D);
    if (nb > 0x7fffffff) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(empty_partial_kernel, dim3((unsigned)nb), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace regenvc

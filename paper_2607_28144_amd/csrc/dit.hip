// gfx950 kernels of the diffusion-transformer block around the attention:
// linear layers (bf16 MFMA, fp32 accumulation) with the block's pointwise
// work fused into their epilogues, the layer normalizations with the adaLN
// modulation, the row RMSNorm of the cross-attention query and the adaLN
// modulation vectors.
//
// Linear layer y = a W^T, a [M, K] and W [N, K] both K-contiguous (the weight
// layout of a linear layer): the shared bf16 MFMA tile kernel (gemm_tile.hpp)
// with dense A rows and BM x 256 tiles (waves 2 x 4, each (BM/2) x 64), BM
// 256 or 288 by how the tiles fill whole rounds of the compute units.
#include "dit_kernels.hpp"

#include <math.h>

#include "gemm_tile.hpp"

namespace regenvc {
namespace {

using tile::bf;
using tile::kBK;
using tile::kThreads;
typedef tile::bf16x8 bf16x8;
typedef tile::f32x4 f32x4;

constexpr int kBN = 256;   // output channels per linear tile (four waves of 64 across)

// Dense A rows: row m of a [M, K] bf16 matrix with row stride lda.
struct DenseA {
    const uint16_t *a;
    int64_t lda;
    typedef const uint16_t *Row;
    __device__ Row row(int m, int chunk) const { return a + (int64_t)m * lda + chunk * 8; }
    __device__ const uint16_t *src(Row r, int kt) const { return r + kt * kBK; }
};

// Linear layer, one BM x 256 tile per workgroup.
template <int BM, int EPI>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void linear_kernel(LinearArgs a, int tiles_n, int n_tiles)
{
    __shared__ __attribute__((aligned(1024))) char smem[tile::lds_bytes<BM, 4>()];
    const DenseA src{static_cast<const uint16_t *>(a.a), a.lda};
    const tile::Out o{static_cast<const uint16_t *>(a.w), static_cast<const uint16_t *>(a.bias), a.gate, a.out,
                      a.ldo, a.M, a.N, a.K};
    tile::tile_body<BM, 4, EPI>(src, o, tiles_n, n_tiles, smem);
}

// ---------------------------------------------------------------- row norms
__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

// One wave per row of C = 512 * NCH channels; lane l holds channels
// 512 j + 8 l .. +7 for j < NCH.  Two-pass mean and variance in registers.
template <int NCH>
__global__ __launch_bounds__(256) void layer_norm_kernel(LayerNormArgs a)
{
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= a.rows) return;
    const float *xr = a.x + row * a.ldx;
    f32x4 v[NCH][2];
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int c = 512 * j + 8 * lane;
        v[j][0] = *reinterpret_cast<const f32x4 *>(xr + c);
        v[j][1] = *reinterpret_cast<const f32x4 *>(xr + c + 4);
        s += v[j][0][0] + v[j][0][1] + v[j][0][2] + v[j][0][3] + v[j][1][0] + v[j][1][1] + v[j][1][2] + v[j][1][3];
    }
    const float inv_c = 1.0f / (float)a.C;
    const float mu = wave_sum(s) * inv_c;
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[j][h][i] -= mu;
                q = fmaf(v[j][h][i], v[j][h][i], q);
            }
    const float rstd = rsqrtf(wave_sum(q) * inv_c + a.eps);
    uint16_t *yr = static_cast<uint16_t *>(a.y) + row * a.ldy;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int c = 512 * j + 8 * lane;
        f32x4 mul[2], add[2];
        if (a.scale != nullptr) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                mul[h] = *reinterpret_cast<const f32x4 *>(a.scale + c + 4 * h) + 1.0f;
                add[h] = *reinterpret_cast<const f32x4 *>(a.shift + c + 4 * h);
            }
        } else {
            const uint16_t *w = static_cast<const uint16_t *>(a.w), *b = static_cast<const uint16_t *>(a.b);
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    mul[h][i] = bf(w[c + 4 * h + i]);
                    add[h][i] = bf(b[c + 4 * h + i]);
                }
        }
        bf16x8 o;
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int i = 0; i < 4; ++i) o[4 * h + i] = (__bf16)fmaf(v[j][h][i] * rstd, mul[h][i], add[h][i]);
        *reinterpret_cast<bf16x8 *>(yr + c) = o;
    }
}

template <int NCH>
__global__ __launch_bounds__(256) void rms_norm_kernel(RmsNormArgs a)
{
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= a.rows) return;
    const uint16_t *xr = static_cast<const uint16_t *>(a.x) + row * a.ldx;
    const uint16_t *w = static_cast<const uint16_t *>(a.w);
    bf16x8 v[NCH];
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        v[j] = *reinterpret_cast<const bf16x8 *>(xr + 512 * j + 8 * lane);
#pragma unroll
        for (int i = 0; i < 8; ++i) q = fmaf((float)v[j][i], (float)v[j][i], q);
    }
    const float r = rsqrtf(wave_sum(q) / (float)a.C + a.eps);
    uint16_t *yr = static_cast<uint16_t *>(a.y) + row * a.ldy;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int c = 512 * j + 8 * lane;
        const bf16x8 wv = *reinterpret_cast<const bf16x8 *>(w + c);
        bf16x8 o;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = (__bf16)((float)v[j][i] * r * (float)wv[i]);
        *reinterpret_cast<bf16x8 *>(yr + c) = o;
    }
}

// adaLN vectors: one wave per output row j, lanes over the C inputs.
// Vector form (C a multiple of 8, 16-byte aligned rows and e): each wave
// takes kModRows consecutive rows; a lane walks 8-channel chunks, forms
// silu(e) of a chunk once and applies it to the chunk of every one of its
// rows (16-byte weight loads, all of a lane's issued before the first is
// used; C <= 2048).
constexpr int kModRows = 4;

__global__ __launch_bounds__(256) void modulation_vec_kernel(ModulationArgs a)
{
    constexpr int kIt = 4;  // 512-channel steps per lane: C <= 2048
    const int lane = threadIdx.x & 63;
    const int j0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * kModRows;
    if (j0 >= a.rows) return;
    const int nr = min(kModRows, a.rows - j0);
    const uint16_t *w = static_cast<const uint16_t *>(a.w) + (int64_t)j0 * a.C;
    // every weight chunk of this lane is requested before the first is used
    bf16x8 v[kIt][kModRows];
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
        const int c = lane * 8 + it * 512;
#pragma unroll
        for (int r = 0; r < kModRows; ++r)
            if (c < a.C && r < nr) v[it][r] = *reinterpret_cast<const bf16x8 *>(w + (int64_t)r * a.C + c);
    }
    float s[kModRows] = {};
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
        const int c = lane * 8 + it * 512;
        if (c >= a.C) break;
        const f32x4 e0 = *reinterpret_cast<const f32x4 *>(a.e + c);
        const f32x4 e1 = *reinterpret_cast<const f32x4 *>(a.e + c + 4);
        float u[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            u[i] = e0[i] / (1.0f + __expf(-e0[i]));
            u[4 + i] = e1[i] / (1.0f + __expf(-e1[i]));
        }
#pragma unroll
        for (int r = 0; r < kModRows; ++r) {
            if (r < nr) {
#pragma unroll
                for (int i = 0; i < 8; ++i) s[r] = fmaf((float)v[it][r][i], u[i], s[r]);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < kModRows; ++r) {
        const float t = wave_sum(s[r]);
        if (lane == 0 && r < nr) a.mod[j0 + r] = t + bf(static_cast<const uint16_t *>(a.b)[j0 + r]);
    }
}

// Scalar form, any C and alignment: one wave per row.
__global__ __launch_bounds__(256) void modulation_kernel(ModulationArgs a)
{
    const int lane = threadIdx.x & 63;
    const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= a.rows) return;
    const uint16_t *w = static_cast<const uint16_t *>(a.w) + (int64_t)j * a.C;
    float s = 0.f;
    for (int c = lane; c < a.C; c += 64) {
        const float e = a.e[c];
        s = fmaf(bf(w[c]), e / (1.0f + __expf(-e)), s);
    }
    s = wave_sum(s);
    if (lane == 0) a.mod[j] = s + bf(static_cast<const uint16_t *>(a.b)[j]);
}

template <int BM, int EPI>
hipError_t launch_linear_t(const LinearArgs &a, hipStream_t stream)
{
    const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.N + kBN - 1) / kBN;
    const int n_tiles = tiles_m * tiles_n;
    hipLaunchKernelGGL((linear_kernel<BM, EPI>), dim3((unsigned)n_tiles), dim3(kThreads), 0, stream, a, tiles_n,
                       n_tiles);
    return hipGetLastError();
}

template <int BM>
hipError_t launch_linear_bm(const LinearArgs &a, hipStream_t stream)
{
    switch (a.epi) {
    case kEpiBias: return launch_linear_t<BM, kEpiBias>(a, stream);
    case kEpiBiasGelu: return launch_linear_t<BM, kEpiBiasGelu>(a, stream);
    case kEpiGatedRes: return launch_linear_t<BM, kEpiGatedRes>(a, stream);
    }
    return hipErrorInvalidValue;
}

int cu_count_here()
{
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
    return n;
}

}  // namespace

// Rounds of tiles over the CUs, each tile costing its rows: the 288-row tile
// wins when the 256-row tiling spills a few tiles into an extra round (at
// M = 10920 rows, 43 row blocks of 256 x 6 channel blocks = 258 tiles on 256
// CUs; 38 blocks of 288 give 228 tiles, one round).
int linear_tile_rows(int M, int N, int n_cu)
{
    const int tn = (N + kBN - 1) / kBN;
    auto cost = [&](int bm) {
        const int64_t tiles = (int64_t)((M + bm - 1) / bm) * tn;
        return (double)((tiles + n_cu - 1) / n_cu) * bm;
    };
    return cost(288) < cost(256) ? 288 : 256;
}

hipError_t launch_linear(const LinearArgs &a, hipStream_t stream)
{
    if (a.M == 0 || a.N == 0) return hipSuccess;
    return linear_tile_rows(a.M, a.N, cu_count_here()) == 288 ? launch_linear_bm<288>(a, stream)
                                                               : launch_linear_bm<256>(a, stream);
}

hipError_t launch_layer_norm(const LayerNormArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)((a.rows + 3) / 4)), block(256);
    switch (a.C / 512) {
    case 1: hipLaunchKernelGGL(layer_norm_kernel<1>, grid, block, 0, stream, a); break;
    case 2: hipLaunchKernelGGL(layer_norm_kernel<2>, grid, block, 0, stream, a); break;
    case 3: hipLaunchKernelGGL(layer_norm_kernel<3>, grid, block, 0, stream, a); break;
    case 4: hipLaunchKernelGGL(layer_norm_kernel<4>, grid, block, 0, stream, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_rms_norm(const RmsNormArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)((a.rows + 3) / 4)), block(256);
    switch (a.C / 512) {
    case 1: hipLaunchKernelGGL(rms_norm_kernel<1>, grid, block, 0, stream, a); break;
    case 2: hipLaunchKernelGGL(rms_norm_kernel<2>, grid, block, 0, stream, a); break;
    case 3: hipLaunchKernelGGL(rms_norm_kernel<3>, grid, block, 0, stream, a); break;
    case 4: hipLaunchKernelGGL(rms_norm_kernel<4>, grid, block, 0, stream, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_modulation(const ModulationArgs &a, hipStream_t stream)
{
    const bool vec = a.C % 8 == 0 && a.C <= 2048 && ((uintptr_t)a.w & 15) == 0 && ((uintptr_t)a.e & 15) == 0;
    if (vec) {
        const int per_block = 4 * kModRows;
        hipLaunchKernelGGL(modulation_vec_kernel, dim3((unsigned)((a.rows + per_block - 1) / per_block)), dim3(256), 0,
                           stream, a);
    } else {
        hipLaunchKernelGGL(modulation_kernel, dim3((unsigned)((a.rows + 3) / 4)), dim3(256), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace regenvc

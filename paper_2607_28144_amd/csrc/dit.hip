// gfx950 kernels of the diffusion-transformer block around the attention:
// linear layers (bf16 MFMA, fp32 accumulation) with the block's pointwise
// work fused into their epilogues, the layer normalizations with the adaLN
// modulation, the row RMSNorm of the cross-attention query and the adaLN
// modulation vectors.
//
// Linear layer y = a W^T, a [M, K] and W [N, K] both K-contiguous (the weight
// layout of a linear layer), so every MFMA fragment is a plain 16-byte LDS
// read.  Workgroup = 8 waves (two per SIMD) = one BM x 256 output tile; wave
// (wm, wn) owns rows wm*BM/2 .. +BM/2 and channels wn*64 .. +64 on
// v_mfma_f32_16x16x32_bf16.  The product is formed transposed, C^T = W a^T,
// so that a lane's accumulator holds four consecutive output channels of one
// row -- the layout the epilogues (bias, GELU-tanh, gated fp32 residual)
// want.  K advances in steps of 64: both operand tiles go HBM -> LDS with
// global_load_lds_dwordx4 (no register staging) into a double-buffered LDS
// ring, rows 128 bytes long with 16-byte chunk c of row r stored at chunk
// c ^ ((r >> 1) & 7), which makes the fragment reads (16 rows, one chunk)
// bank-conflict free.  Tiles are dealt XCD-aware: each XCD takes a
// contiguous range of tiles (a few row blocks across all channel blocks), so
// the rows it reads stay in its L2.
#include "dit_kernels.hpp"

#include <math.h>

namespace regenvc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) char lds_char;

constexpr int kLinWaves = 8;
constexpr int kLinThreads = 64 * kLinWaves;
constexpr int kBN = 256;   // output channels per tile
constexpr int kBK = 64;    // K per step (two 32-deep MFMA steps)
constexpr int kRowBytes = kBK * 2;

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16-byte HBM -> LDS copy (global_load_lds_dwordx4): lane i's 16 bytes land
// at lds_base + 16 * i.  Inline asm so that the compiler does not order it
// against the LDS reads of the other ring stage; completion is awaited with
// an explicit s_waitcnt vmcnt before the barrier that publishes the stage.
__device__ __forceinline__ void lds_copy16(const void *gptr, uint32_t lds_base)
{
    const uint32_t base = __builtin_amdgcn_readfirstlane(lds_base);  // wave-uniform by construction
    __asm__ volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" : : "s"(base), "v"(gptr) : "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ void wait_all_copies()
{
    __asm__ volatile("s_waitcnt vmcnt(0)" : : : "memory");
}

__device__ __forceinline__ int swz(int row, int chunk)
{
    return chunk ^ ((row >> 1) & 7);
}

__device__ __forceinline__ float gelu_tanh(float x)
{
    // x/2 (1 + tanh(u)), tanh(u) = 1 - 2 / (e^(2u) + 1); u = sqrt(2/pi) (x + 0.044715 x^3)
    const float u = 0.7978845608028654f * fmaf(0.044715f * x, x * x, x);
    const float t = 1.0f - 2.0f / (__expf(2.0f * u) + 1.0f);
    return 0.5f * x * (1.0f + t);
}

__device__ __forceinline__ float bf(uint16_t b)
{
    return __uint_as_float(((uint32_t)b) << 16);
}

// Linear layer, one BM x 256 tile per workgroup.
template <int BM, int EPI>
__global__ __launch_bounds__(kLinThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void linear_kernel(LinearArgs a, int tiles_n, int n_tiles)
{
    constexpr int WM = BM / 2;           // rows per wave
    constexpr int MB = WM / 16;          // 16-row MFMA blocks per wave
    constexpr int NB = 4;                // 16-channel MFMA blocks per wave
    constexpr int A_BYTES = BM * kRowBytes;
    constexpr int W_BYTES = kBN * kRowBytes;
    constexpr int STAGE = A_BYTES + W_BYTES;
    constexpr int A_INSTR = A_BYTES / 1024;  // 1 KB (8 rows) per wave copy instruction
    constexpr int W_INSTR = W_BYTES / 1024;
    constexpr int A_PER = (A_INSTR + kLinWaves - 1) / kLinWaves;
    constexpr int W_PER = W_INSTR / kLinWaves;
    static_assert(WM % 16 == 0 && W_INSTR % kLinWaves == 0, "tile shape");
    __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave >> 2, wn = wave & 3;
    const int g = lane >> 4, x = lane & 15;

    // XCD-aware tile: workgroup i runs on XCD i % 8; XCD x takes a contiguous
    // range of tiles, channel blocks fastest
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int tile = xcd * (n_tiles >> 3) + min(xcd, n_tiles & 7) + slot;
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const int m0 = tm * BM, n0 = tn * kBN;

    const uint16_t *A = static_cast<const uint16_t *>(a.a);
    const uint16_t *W = static_cast<const uint16_t *>(a.w);

    // this lane's copy sources: instruction j of the tile covers rows 8j..8j+7;
    // lane l fills LDS chunk l % 8 of row 8j + l / 8, which holds global chunk
    // swz(row, l % 8).  Rows past the end re-read the last row (never stored).
    const uint16_t *asrc[A_PER];
    const uint16_t *wsrc[W_PER];
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
        const int j = wave + i * kLinWaves;
        const int r = min(j, A_INSTR - 1) * 8 + (lane >> 3);
        const int gr = min(m0 + r, a.M - 1);
        asrc[i] = A + (int64_t)gr * a.lda + swz(r, lane & 7) * 8;
    }
#pragma unroll
    for (int i = 0; i < W_PER; ++i) {
        const int r = (wave + i * kLinWaves) * 8 + (lane >> 3);
        const int gr = min(n0 + r, a.N - 1);
        wsrc[i] = W + (int64_t)gr * a.K + swz(r, lane & 7) * 8;
    }
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char *)smem;
    auto issue = [&](int kt, int st) {
        const uint32_t sa = lds0 + st * STAGE, sw = sa + A_BYTES;
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            const int j = wave + i * kLinWaves;
            if (j < A_INSTR) lds_copy16(asrc[i] + kt * kBK, sa + j * 1024);
        }
#pragma unroll
        for (int i = 0; i < W_PER; ++i) lds_copy16(wsrc[i] + kt * kBK, sw + (wave + i * kLinWaves) * 1024);
    };

    // fragment offsets within a stage: A block mb (rows wm*WM + mb*16 + x),
    // W block nb (rows wn*64 + nb*16 + x), 16-byte chunk ks*4 + g
    f32x4 acc[NB][MB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = a.K / kBK;
    issue(0, 0);
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        wait_all_copies();   // this wave's copies of step kt landed
        __syncthreads();     // ... and every wave's; step kt-1's stage is free
        if (kt + 1 < nk) issue(kt + 1, st ^ 1);
        const lds_char *sa = (const lds_char *)smem + st * STAGE;
        const lds_char *sw = sa + A_BYTES;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int ch = ks * 4 + g;
            bf16x8 wf[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const int r = wn * 64 + nb * 16 + x;
                wf[nb] = *(const lds_bf16x8 *)(sw + r * kRowBytes + swz(r, ch) * 16);
            }
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                const int r = wm * WM + mb * 16 + x;
                const bf16x8 af = *(const lds_bf16x8 *)(sa + r * kRowBytes + swz(r, ch) * 16);
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[nb], af, acc[nb][mb], 0, 0, 0);
            }
        }
    }

    // epilogue: acc[nb][mb][i] = y[m0 + wm*WM + mb*16 + x][n0 + wn*64 + nb*16 + 4g + i]
    const uint16_t *bias = static_cast<const uint16_t *>(a.bias);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int n = n0 + wn * 64 + nb * 16 + 4 * g;
        if (n >= a.N) continue;
        f32x4 bv = {0.f, 0.f, 0.f, 0.f};
        if (bias != nullptr) {
            const uint64_t b4 = *reinterpret_cast<const uint64_t *>(bias + n);
#pragma unroll
            for (int i = 0; i < 4; ++i) bv[i] = bf((uint16_t)(b4 >> (16 * i)));
        }
        f32x4 gv = {1.f, 1.f, 1.f, 1.f};
        if (EPI == kEpiGatedRes && a.gate != nullptr) gv = *reinterpret_cast<const f32x4 *>(a.gate + n);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const int m = m0 + wm * WM + mb * 16 + x;
            if (m >= a.M) continue;
            const f32x4 y = acc[nb][mb] + bv;
            if constexpr (EPI == kEpiGatedRes) {
                f32x4 *o = reinterpret_cast<f32x4 *>(static_cast<float *>(a.out) + (int64_t)m * a.ldo + n);
                *o = *o + gv * y;
            } else {
                bf16x4 w;
#pragma unroll
                for (int i = 0; i < 4; ++i) w[i] = (__bf16)(EPI == kEpiBiasGelu ? gelu_tanh(y[i]) : y[i]);
                *reinterpret_cast<bf16x4 *>(static_cast<uint16_t *>(a.out) + (int64_t)m * a.ldo + n) = w;
            }
        }
    }
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
    hipLaunchKernelGGL((linear_kernel<BM, EPI>), dim3((unsigned)n_tiles), dim3(kLinThreads), 0, stream, a, tiles_n,
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
    hipLaunchKernelGGL(modulation_kernel, dim3((unsigned)((a.rows + 3) / 4)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace regenvc

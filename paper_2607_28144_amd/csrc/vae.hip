// gfx950 kernels of the spatially split VAE tile (paper Sec. 3.6): the
// causal 3D convolutions of a VAE stage run on each tile's region (its core
// widened by a halo), and the blended gather of the tiles into the plane.
//
// Convolution as an implicit GEMM on the shared bf16 MFMA tile kernel
// (gemm_tile.hpp): rows are the output pixels (tile, frame, row, column) of
// the listed tiles, K runs over the 27 taps x Cin channels, and the weights
// [Cout, 3, 3, 3, Cin] are K-contiguous per output channel -- the linear
// layer's layout.  Channels-last activations make every (pixel, tap) a
// contiguous run of Cin values, so a K step of 64 channels of one tap is
// one 128-byte row per pixel, copied HBM -> LDS like a dense row; a tap
// that falls before the first frame or outside the tile's region is copied
// from a page of zeros instead (the zero padding).  Tiles of 128 pixel
// rows x 384 output channels; when they are too few to fill the compute
// units (one GPU's single tile), K is split into ranges whose f32 partial
// sums a second kernel adds, with the bias and the activation.
//
// Blend: one thread per (pixel, 8 channels) walks the tiles whose region
// covers the pixel and adds weight x value, the weight the product of the
// two axes' ramps (fp32).  HBM-bound.
#include "vae_kernels.hpp"

#include <stdint.h>

#include <algorithm>

#include "gemm_tile.hpp"

// 128 bytes of zeros in device memory: the source of the copies that stand
// for padding taps (read only).
static __device__ __align__(256) uint16_t vae_zero_page[64] = {0};

namespace regenvc {
namespace {

using tile::kBK;
using tile::kThreads;

// Output tile of the convolution: 128 rows x 384 channels (all of Cout up to
// 384: each gathered A row block is read once for every output channel);
// waves 2 x 4, each 64 rows x 96 channels.
constexpr int kConvBM = 128;
constexpr int kConvNB = 6;
constexpr int kConvBN = 16 * kConvNB * 4;
typedef tile::bf16x8 bf16x8;
typedef tile::f32x4 f32x4;

// A rows of the convolution: pixel m of the listed tiles' regions, K step kt
// = tap kt / (Cin / 64), channels 64 (kt % (Cin / 64)) .. +63.  A row keeps
// the address of its own pixel (the centre tap of the current frame) and
// its position and region size; everything that depends on the tap is
// wave-uniform (scalar): the tap's offset from the row's address and which
// bounds it can cross.
struct ConvA {
    const uint16_t *in;
    const ConvArgs *a;
    int cpt;              // K steps per tap
    int64_t frame_px;     // pixels per frame of the input (plane, or a tile buffer)
    int64_t row_px;       // pixels per row of the input
    struct Row {
        const uint16_t *base;
        int t, y, x, h, w;
    };
    __device__ Row row(int m, int chunk) const
    {
        Row r;
        r.x = m % a->Wr;
        int q = m / a->Wr;
        r.y = q % a->Hr;
        q /= a->Hr;
        r.t = q % a->T;
        const int ti = q / a->T;
        const VaeTile &tl = a->tiles[ti];
        r.h = tl.reg_y1 - tl.reg_y0;
        r.w = tl.reg_x1 - tl.reg_x0;
        int64_t pix;
        if (a->in_is_plane)
            pix = ((int64_t)r.t * a->H + tl.reg_y0 + r.y) * a->W + tl.reg_x0 + r.x;
        else
            pix = ((int64_t)ti * a->T + r.t) * frame_px + (int64_t)r.y * a->Wr + r.x;
        r.base = in + pix * a->Cin + chunk * 8;
        return r;
    }
    __device__ const uint16_t *src(const Row &r, int kt) const
    {
        const int tap = kt / cpt, c0 = (kt - tap * cpt) * kBK;  // wave-uniform
        const int dt = tap / 9 - 2, dy = (tap / 3) % 3 - 1, dx = tap % 3 - 1;
        const int64_t off = ((int64_t)dt * frame_px + (int64_t)dy * row_px + dx) * a->Cin + c0;
        const bool ok = r.t + dt >= 0 && (unsigned)(r.y + dy) < (unsigned)r.h && (unsigned)(r.x + dx) < (unsigned)r.w;
        return ok ? r.base + off : vae_zero_page;
    }
};

// EPI == kPartial: split-K, f32 partial sums of `splits` K ranges into the
// workspace (bias and activation follow in vae_reduce_kernel).
template <int BM, int EPI>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void conv3d_kernel(ConvArgs a, int tiles_n, int n_tiles, int splits)
{
    __shared__ __attribute__((aligned(1024))) char smem[tile::lds_bytes<BM, 4, kConvNB>()];
    const ConvA src{static_cast<const uint16_t *>(a.in), &a, a.Cin / kBK,
                    a.in_is_plane ? (int64_t)a.H * a.W : (int64_t)a.Hr * a.Wr, a.in_is_plane ? a.W : a.Wr};
    const bool part = EPI == tile::kPartial;
    const tile::Out o{static_cast<const uint16_t *>(a.w), part ? nullptr : static_cast<const uint16_t *>(a.bias),
                      nullptr, part ? a.ws : a.out, a.Cout, a.n_tiles * a.T * a.Hr * a.Wr, a.Cout, 27 * a.Cin, splits};
    tile::tile_body<BM, 4, EPI, ConvA, kConvNB>(src, o, tiles_n, n_tiles, smem);
}

// Sum of the split-K partials, bias and activation: one thread per 8
// channels of one output row.
template <bool SILU>
__global__ __launch_bounds__(256) void vae_reduce_kernel(ConvArgs a, int splits)
{
    const int64_t M = (int64_t)a.n_tiles * a.T * a.Hr * a.Wr;
    const int cg = a.Cout / 8;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= M * cg) return;
    const int64_t m = gid / cg;
    const int c = (int)(gid - m * cg) * 8;
    const float *p = static_cast<const float *>(a.ws) + m * a.Cout + c;
    f32x4 s0 = *reinterpret_cast<const f32x4 *>(p), s1 = *reinterpret_cast<const f32x4 *>(p + 4);
    for (int k = 1; k < splits; ++k) {
        const float *q = p + (int64_t)k * M * a.Cout;
        s0 += *reinterpret_cast<const f32x4 *>(q);
        s1 += *reinterpret_cast<const f32x4 *>(q + 4);
    }
    const bf16x8 bb = *reinterpret_cast<const bf16x8 *>(static_cast<const uint16_t *>(a.bias) + c);
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float y = (e < 4 ? s0[e] : s1[e - 4]) + (float)bb[e];
        o[e] = (__bf16)(SILU ? tile::silu(y) : y);
    }
    *reinterpret_cast<bf16x8 *>(static_cast<uint16_t *>(a.out) + m * a.Cout + c) = o;
}

__device__ __forceinline__ float ramp(int p, int c0, int c1, int n, int band)
{
    if (band == 0) return (p >= c0 && p < c1) ? 1.f : 0.f;
    const float pc = (float)p + 0.5f, inv = 0.5f / (float)band;
    float w = 1.f;
    if (c0 > 0) w = fminf(w, fminf(fmaxf(((float)band + (pc - (float)c0)) * inv, 0.f), 1.f));
    if (c1 < n) w = fminf(w, fminf(fmaxf(((float)band + ((float)c1 - pc)) * inv, 0.f), 1.f));
    return w;
}

__global__ __launch_bounds__(256) void vae_blend_kernel(BlendArgs a)
{
    const int cg = a.C / 8;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (int64_t)a.T * a.H * a.W * cg) return;
    const int c = (int)(gid % cg) * 8;
    int64_t q = gid / cg;
    const int x = (int)(q % a.W);
    q /= a.W;
    const int y = (int)(q % a.H);
    const int t = (int)(q / a.H);
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const uint16_t *src = static_cast<const uint16_t *>(a.tiles_out);
    for (int i = 0; i < a.n_tiles; ++i) {
        const VaeTile &tl = a.tiles[i];
        if (y < tl.reg_y0 || y >= tl.reg_y1 || x < tl.reg_x0 || x >= tl.reg_x1) continue;
        const float w = ramp(y, tl.core_y0, tl.core_y1, a.H, a.band) * ramp(x, tl.core_x0, tl.core_x1, a.W, a.band);
        if (w == 0.f) continue;
        const int64_t pix = (((int64_t)i * a.T + t) * a.Hr + (y - tl.reg_y0)) * a.Wr + (x - tl.reg_x0);
        const bf16x8 v = *reinterpret_cast<const bf16x8 *>(src + pix * a.C + c);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(w, (float)v[e], acc[e]);
    }
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (__bf16)acc[e];
    *reinterpret_cast<bf16x8 *>(static_cast<uint16_t *>(a.out) + (((int64_t)t * a.H + y) * a.W + x) * a.C + c) = o;
}

hipError_t launch_conv(const ConvArgs &a, int splits, hipStream_t stream)
{
    constexpr int BM = kConvBM;
    const int64_t M = (int64_t)a.n_tiles * a.T * a.Hr * a.Wr;
    const int tiles_n = tile::tiles_along(a.Cout, kConvBN);
    const int n_tiles = (int)((M + BM - 1) / BM) * tiles_n;
    if (splits > 1) {
        hipLaunchKernelGGL((conv3d_kernel<BM, tile::kPartial>), dim3((unsigned)(n_tiles * splits)), dim3(kThreads), 0,
                           stream, a, tiles_n, n_tiles, splits);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t n = M * (a.Cout / 8);
        const dim3 grid((unsigned)((n + 255) / 256));
        if (a.silu)
            hipLaunchKernelGGL(vae_reduce_kernel<true>, grid, dim3(256), 0, stream, a, splits);
        else
            hipLaunchKernelGGL(vae_reduce_kernel<false>, grid, dim3(256), 0, stream, a, splits);
    } else if (a.silu) {
        hipLaunchKernelGGL((conv3d_kernel<BM, tile::kBiasSilu>), dim3((unsigned)n_tiles), dim3(kThreads), 0, stream,
                           a, tiles_n, n_tiles, 1);
    } else {
        hipLaunchKernelGGL((conv3d_kernel<BM, tile::kBias>), dim3((unsigned)n_tiles), dim3(kThreads), 0, stream, a,
                           tiles_n, n_tiles, 1);
    }
    return hipGetLastError();
}

int cu_count_here()
{
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
    return n;
}

}  // namespace

// Split-K when the output tiles (128 rows x all channels) leave more than
// half the compute units idle: K (27 taps x Cin) cut into as many ranges as
// fill the CUs in one round (at most 8), limited by the workspace (one f32
// copy of the output per range).  One split VAE tile of the window (8092
// pixels: 64 row tiles) runs as 64 x 4 workgroups.
int conv_splits(int64_t M, int N, int Cin, int n_cu, int64_t ws_bytes)
{
    const int64_t tiles = (M + kConvBM - 1) / kConvBM * ((N + kConvBN - 1) / kConvBN);
    const int nk = 27 * Cin / kBK;
    if (tiles * 2 > n_cu) return 1;
    int s = (int)std::min<int64_t>(8, n_cu / tiles);
    s = std::min(s, nk);
    const int64_t plane = M * N * (int64_t)sizeof(float);
    if (plane > 0) s = (int)std::min<int64_t>(s, ws_bytes / plane);
    return s >= 2 ? s : 1;
}

size_t conv_workspace_bytes(int64_t M, int N, int Cin, int n_cu)
{
    const int s = conv_splits(M, N, Cin, n_cu, INT64_MAX);
    return s > 1 ? (size_t)s * M * N * sizeof(float) : 0;
}

hipError_t launch_vae_conv(const ConvArgs &a, hipStream_t stream)
{
    const int64_t M = (int64_t)a.n_tiles * a.T * a.Hr * a.Wr;
    if (M == 0) return hipSuccess;
    const int splits = a.ws != nullptr ? conv_splits(M, a.Cout, a.Cin, cu_count_here(), a.ws_bytes) : 1;
    return launch_conv(a, splits, stream);
}

hipError_t launch_vae_blend(const BlendArgs &a, hipStream_t stream)
{
    const int64_t n = (int64_t)a.T * a.H * a.W * (a.C / 8);
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(vae_blend_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace regenvc

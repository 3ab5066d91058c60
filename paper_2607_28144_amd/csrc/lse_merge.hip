// gfx950 log-sum-exp merge of key/value-chunk partials, and the empty-chunk
// partial (the merge identity).  Streaming, HBM-bound: one thread per four
// head dims of one (batch, token, head) row, 16-byte loads and stores.
//
// Method: partials over disjoint key chunks combine exactly by the
// log-sum-exp identity (the Ring side of the paper's sequence parallelism,
// Sec. 3.5): L = m + log sum_c exp(L_c - m), O = sum_c exp(L_c - L) O_c.
// Parts are visited in their given order, so a launch is deterministic.
#include "attn_kernels.hpp"

#include <math.h>

namespace regenvc {
namespace {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Log-sum-exp merge of chunk partials: one thread per 4 dims of one row.
// Parts are visited in batches of MB whose LSE and O loads are all issued
// before any is used, and combined online (running max, sum and weighted O).
// A part with LSE = -inf (an empty chunk) has weight 0; if every part is
// empty the row is O = 0, LSE = -inf.
template <bool OUT_F32>
__global__ __launch_bounds__(256) void lse_merge_kernel(MergeArgs a)
{
    constexpr int MB = 4;
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

    float m = -INFINITY, s = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < a.num_parts; c0 += MB) {
        float l[MB];
        f32x4 o[MB];
#pragma unroll
        for (int k = 0; k < MB; ++k) {
            const int c = min(c0 + k, a.num_parts - 1);
            l[k] = c0 + k < a.num_parts ? a.lse_parts[c][li] : -INFINITY;
            o[k] = *reinterpret_cast<const f32x4 *>(a.o_parts[c] + row * a.D + d);
        }
        float mb = m;
#pragma unroll
        for (int k = 0; k < MB; ++k) mb = fmaxf(mb, l[k]);
        if (mb == -INFINITY) continue;  // nothing but empty parts so far
        const float sc = expf(m - mb);  // 0 while m is still -inf
        s *= sc;
        acc *= sc;
#pragma unroll
        for (int k = 0; k < MB; ++k) {
            const float w = expf(l[k] - mb);
            s += w;
            acc += w * o[k];
        }
        m = mb;
    }
    float L = -INFINITY;
    if (m != -INFINITY) {
        L = m + logf(s);
        acc *= 1.0f / s;
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

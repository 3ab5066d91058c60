// The bf16 MFMA tile kernel shared by the linear layers of the diffusion
// block (dense rows) and the VAE's causal 3D convolution (rows gathered as
// an implicit GEMM): out[m][n] = epilogue(sum_k A[m][k] W[n][k]).
//
// Workgroup = 8 waves (two per SIMD) = one BM x BN output tile, BN = 16 NB
// WN; the waves form an (8 / WN) x WN grid, each owning (BM / (8 / WN)) rows
// x 16 NB channels on v_mfma_f32_16x16x32_bf16.  The product is formed
// transposed, C^T = W A^T, so that a lane's accumulator holds four
// consecutive output channels of one row (what the epilogues want).  K
// advances in steps of 64: both operand tiles go HBM -> LDS with
// global_load_lds_dwordx4 (no register staging) into a double-buffered LDS
// ring; rows are 128 bytes, 16-byte chunk c of row r stored at chunk
// c ^ ((r >> 1) & 7), which makes the fragment reads (16 rows, one chunk)
// bank-conflict free.  Tiles are dealt XCD-aware: each XCD takes a
// contiguous range of tiles, numbered in groups of four row blocks swept
// across the channel blocks, so that the tiles resident on an XCD share
// their operand blocks through its L2.
//
// The A source is a policy: for each of this lane's copy rows it gives the
// address of the 16 bytes to copy at K step kt (a dense row, or a tap of a
// convolution patch, or a page of zeros for padding).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace regenvc {
namespace tile {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) char lds_char;

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kBK = 64;               // K per step (two 32-deep MFMA steps)
constexpr int kRowBytes = kBK * 2;
constexpr int kGroupM = 4;            // row blocks per group of the tile order

enum Epi : int32_t {
    kBias = 0,        // out bf16 = y + bias
    kBiasGelu = 1,    // out bf16 = gelu_tanh(y + bias)
    kGatedRes = 2,    // out f32 (in place) = out + gate[n] * (y + bias[n])   (gate may be null: 1)
    kBiasSilu = 3,    // out bf16 = silu(y + bias)
    kPartial = 4,     // out f32 = y over this workgroup's share of K (split-K partial, no bias)
};

// Output side of a tile launch.
struct Out {
    const uint16_t *w;    // [N, K] bf16, K contiguous
    const uint16_t *bias; // [N] bf16 or null
    const float *gate;    // [N] f32 or null (kGatedRes)
    void *out;            // bf16 or f32 [M, N], row stride ldo
    int64_t ldo;
    int32_t M, N, K;
    int32_t splits;       // kPartial: K split into this many contiguous ranges, one per launch slice
};

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

// Activations of the epilogues, in the sigmoid form with the hardware
// base-2 exponential and reciprocal (both within an ulp or two of fp32,
// far below the bf16 rounding that follows): no fp32 division.
//   gelu_tanh(x) = x/2 (1 + tanh(u)) = x sigmoid(2u),  u = sqrt(2/pi) (x + 0.044715 x^3),
//   sigmoid(2u) = 1 / (1 + 2^z),  z = -2 log2(e) u = x (kG1 + kG3 x^2).
__device__ __forceinline__ float gelu_tanh(float x)
{
    constexpr float kG1 = -2.0f * 1.4426950408889634f * 0.7978845608028654f;
    constexpr float kG3 = kG1 * 0.044715f;
    const float z = x * fmaf(kG3, x * x, kG1);
    return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}

// silu(x) = x sigmoid(x) = x / (1 + 2^(-x log2 e)).
__device__ __forceinline__ float silu(float x)
{
    return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}

__device__ __forceinline__ float bf(uint16_t b)
{
    return __uint_as_float(((uint32_t)b) << 16);
}

// One BM x BN output tile.  The launch has n_tiles workgroups per K slice;
// with EPI == kPartial it has o.splits slices (workgroup s * n_tiles + t:
// tile t over the s-th of o.splits contiguous ranges of K steps), each
// writing its partial sums to its own f32 [M][ldo] plane of o.out.
template <int BM, int WN, int EPI, class ASrc, int NB = 4>
__device__ __forceinline__ void tile_body(const ASrc &asrc, const Out &o, int tiles_n, int n_tiles, char *smem)
{
    constexpr int BN = 16 * NB * WN;     // NB 16-channel MFMA blocks per wave across
    constexpr int WGM = kWaves / WN;     // waves along M
    constexpr int WM = BM / WGM;         // rows per wave
    constexpr int MB = WM / 16;          // 16-row MFMA blocks per wave
    constexpr int A_BYTES = BM * kRowBytes;
    constexpr int W_BYTES = BN * kRowBytes;
    constexpr int STAGE = A_BYTES + W_BYTES;
    constexpr int A_INSTR = A_BYTES / 1024;  // 1 KB (8 rows) per wave copy instruction
    constexpr int W_INSTR = W_BYTES / 1024;
    constexpr int A_PER = (A_INSTR + kWaves - 1) / kWaves;
    constexpr int W_PER = W_INSTR / kWaves;
    static_assert(WM % 16 == 0 && W_INSTR % kWaves == 0, "tile shape");

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave / WN, wn = wave % WN;
    const int g = lane >> 4, x = lane & 15;

    // XCD-aware tile: workgroup i runs on XCD i % 8; XCD x takes a contiguous
    // range of tiles.  Tiles are numbered in groups of kGroupM row blocks
    // swept across the channel blocks (row block fastest), so the ~32 tiles
    // resident on an XCD at a time cover about 4 row blocks x 8 channel
    // blocks: each A row block and W block they read serves several of them
    // from the XCD's L2.
    const int sp = EPI == kPartial ? (int)blockIdx.x / n_tiles : 0;  // K slice
    const int bid = EPI == kPartial ? (int)blockIdx.x - sp * n_tiles : (int)blockIdx.x;
    const int xcd = bid & 7, slot = bid >> 3;
    const int tile = xcd * (n_tiles >> 3) + min(xcd, n_tiles & 7) + slot;
    const int tiles_m = n_tiles / tiles_n;
    const int group = tile / (kGroupM * tiles_n), in_group = tile - group * kGroupM * tiles_n;
    const int gm = min(tiles_m - group * kGroupM, kGroupM);
    const int tm = group * kGroupM + in_group % gm, tn = in_group / gm;
    const int m0 = tm * BM, n0 = tn * BN;

    // this lane's copies: instruction j of a tile covers its rows 8j..8j+7;
    // lane l fills LDS chunk l % 8 of row 8j + l / 8, which holds global
    // chunk swz(row, l % 8).  Rows past the end re-read the last row (never
    // stored).
    typename ASrc::Row arow[A_PER];
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
        const int j = min(wave + i * kWaves, A_INSTR - 1);
        const int r = j * 8 + (lane >> 3);
        arow[i] = asrc.row(min(m0 + r, o.M - 1), swz(r, lane & 7));
    }
    const uint16_t *wsrc[W_PER];
#pragma unroll
    for (int i = 0; i < W_PER; ++i) {
        const int r = (wave + i * kWaves) * 8 + (lane >> 3);
        const int gr = min(n0 + r, o.N - 1);
        wsrc[i] = o.w + (int64_t)gr * o.K + swz(r, lane & 7) * 8;
    }
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char *)smem;
    auto issue = [&](int kt, int st) {
        const uint32_t sa = lds0 + st * STAGE, sw = sa + A_BYTES;
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            const int j = wave + i * kWaves;
            if (j < A_INSTR) lds_copy16(asrc.src(arow[i], kt), sa + j * 1024);
        }
#pragma unroll
        for (int i = 0; i < W_PER; ++i) lds_copy16(wsrc[i] + kt * kBK, sw + (wave + i * kWaves) * 1024);
    };

    f32x4 acc[NB][MB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk_all = o.K / kBK;
    const int k_begin = EPI == kPartial ? (int)((int64_t)sp * nk_all / o.splits) : 0;
    const int nk = EPI == kPartial ? (int)((int64_t)(sp + 1) * nk_all / o.splits) : nk_all;
    issue(k_begin, 0);
    for (int kt = k_begin; kt < nk; ++kt) {
        const int st = (kt - k_begin) & 1;
        wait_all_copies();   // this wave's copies of step kt landed
        __syncthreads();     // ... and every wave's; step kt-1's stage is free
        if (kt + 1 < nk) issue(kt + 1, st ^ 1);
        const lds_char *sa = (const lds_char *)smem + st * STAGE;
        const lds_char *sw = sa + A_BYTES;
        // the step's 2 x MB groups of 4 MFMAs (k half ks, row block mb),
        // each A fragment read two groups ahead of its MFMAs (a ring of 3)
        // and the second k half's W fragments read at the start, the order
        // pinned so that the LDS latency passes under earlier MFMAs
        auto afrag = [&](int s) {
            const int r = wm * WM + (s % MB) * 16 + x;
            return *(const lds_bf16x8 *)(sa + r * kRowBytes + swz(r, (s / MB) * 4 + g) * 16);
        };
        auto wfrag = [&](int ks, int nb) {
            const int r = wn * (16 * NB) + nb * 16 + x;
            return *(const lds_bf16x8 *)(sw + r * kRowBytes + swz(r, ks * 4 + g) * 16);
        };
        bf16x8 wf[2][NB], ar[3];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) wf[0][nb] = wfrag(0, nb);
        ar[0] = afrag(0);
        ar[1] = afrag(1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s = 0; s < 2 * MB; ++s) {
            if (s + 2 < 2 * MB) ar[(s + 2) % 3] = afrag(s + 2);
            if (s == 0) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) wf[1][nb] = wfrag(1, nb);
            }
            const int ks = s / MB, mb = s % MB;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[ks][nb], ar[s % 3], acc[nb][mb], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // epilogue: acc[nb][mb][i] = y[m0 + wm*WM + mb*16 + x][n0 + wn*16*NB + nb*16 + 4g + i]
    constexpr bool BF16_OUT = EPI == kBias || EPI == kBiasGelu || EPI == kBiasSilu;
    if constexpr (BF16_OUT) {
        // A whole-width tile with 16-byte aligned rows goes out as full rows:
        // the values are staged in the (now idle) LDS, row-major with 16-byte
        // chunk c of row r at chunk c ^ (r & 15), and each store instruction
        // then writes whole 16-byte chunks of consecutive rows instead of 8
        // bytes of each of 16 rows.
        if (n0 + BN <= o.N && (reinterpret_cast<uintptr_t>(o.out) & 15) == 0 && (o.ldo & 7) == 0) {
            constexpr int CH = BN / 8;  // 16-byte chunks per staged row
            static_assert(CH % 16 == 0 && (BM * CH) % kThreads == 0, "staging shape");
            __syncthreads();  // every wave is done reading the ring
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const int n = n0 + wn * (16 * NB) + nb * 16 + 4 * g;
                f32x4 bv = {0.f, 0.f, 0.f, 0.f};
                if (o.bias != nullptr) {
                    const uint64_t b4 = *reinterpret_cast<const uint64_t *>(o.bias + n);
#pragma unroll
                    for (int i = 0; i < 4; ++i) bv[i] = bf((uint16_t)(b4 >> (16 * i)));
                }
                const int c = wn * 2 * NB + nb * 2 + g / 2;
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const int r = wm * WM + mb * 16 + x;
                    const f32x4 y = acc[nb][mb] + bv;
                    bf16x4 w;
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        w[i] = (__bf16)(EPI == kBiasGelu ? gelu_tanh(y[i]) : EPI == kBiasSilu ? silu(y[i]) : y[i]);
                    *(__attribute__((address_space(3))) bf16x4 *)((lds_char *)smem + r * (BN * 2) +
                                                                 ((c ^ (r & 15)) * 16) + (g & 1) * 8) = w;
                }
            }
            __syncthreads();
#pragma unroll
            for (int it = 0; it < BM * CH / kThreads; ++it) {
                const int id = it * kThreads + (int)threadIdx.x;
                const int r = id / CH, c = id % CH;
                const bf16x8 v = *(const lds_bf16x8 *)((const lds_char *)smem + r * (BN * 2) + ((c ^ (r & 15)) * 16));
                if (m0 + r < o.M)
                    *reinterpret_cast<bf16x8 *>(static_cast<uint16_t *>(o.out) + (int64_t)(m0 + r) * o.ldo + n0 +
                                                c * 8) = v;
            }
            return;
        }
    }
    if constexpr (EPI == kGatedRes) {
        // The same for the read-modify-write of the fp32 residual, in two
        // passes over half the tile's channels each (the staged fp32 half
        // tile fits the LDS): y + bias is staged, and the lane that owns a
        // 16-byte chunk of a row adds gate * y to it with whole-chunk loads
        // and stores of consecutive rows.
        if (n0 + BN <= o.N && (reinterpret_cast<uintptr_t>(o.out) & 15) == 0 && (o.ldo & 3) == 0) {
            constexpr int HALF = BN / 2;  // channels per pass
            constexpr int CH = HALF / 4;  // 16-byte chunks per staged row
            constexpr int WCH = 16 * NB;  // channels of one wave column
            static_assert(HALF % WCH == 0 && CH % 16 == 0 && (BM * CH) % kThreads == 0, "staging shape");
#pragma unroll
            for (int pass = 0; pass < 2; ++pass) {
                __syncthreads();  // the ring (first pass) or the previous half is no longer read
                if (wn * WCH / HALF == pass) {
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb) {
                        const int col = wn * WCH + nb * 16 + 4 * g;  // channel within the tile
                        f32x4 bv = {0.f, 0.f, 0.f, 0.f};
                        if (o.bias != nullptr) {
                            const uint64_t b4 = *reinterpret_cast<const uint64_t *>(o.bias + n0 + col);
#pragma unroll
                            for (int i = 0; i < 4; ++i) bv[i] = bf((uint16_t)(b4 >> (16 * i)));
                        }
                        const int c = (col - pass * HALF) / 4;
#pragma unroll
                        for (int mb = 0; mb < MB; ++mb) {
                            const int r = wm * WM + mb * 16 + x;
                            *(__attribute__((address_space(3))) f32x4 *)((lds_char *)smem + r * (HALF * 4) +
                                                                        ((c ^ (r & 15)) * 16)) = acc[nb][mb] + bv;
                        }
                    }
                }
                __syncthreads();
#pragma unroll 2
                for (int it = 0; it < BM * CH / kThreads; ++it) {
                    const int id = it * kThreads + (int)threadIdx.x;
                    const int r = id / CH, c = id % CH;
                    if (m0 + r >= o.M) continue;
                    const int n = n0 + pass * HALF + c * 4;
                    const f32x4 y =
                        *(const __attribute__((address_space(3))) f32x4 *)((const lds_char *)smem + r * (HALF * 4) +
                                                                         ((c ^ (r & 15)) * 16));
                    const f32x4 gv = o.gate != nullptr ? *reinterpret_cast<const f32x4 *>(o.gate + n)
                                                       : f32x4{1.f, 1.f, 1.f, 1.f};
                    f32x4 *p = reinterpret_cast<f32x4 *>(static_cast<float *>(o.out) + (int64_t)(m0 + r) * o.ldo + n);
                    *p = *p + gv * y;
                }
            }
            return;
        }
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int n = n0 + wn * (16 * NB) + nb * 16 + 4 * g;
        if (n >= o.N) continue;
        f32x4 bv = {0.f, 0.f, 0.f, 0.f};
        if (o.bias != nullptr) {
            const uint64_t b4 = *reinterpret_cast<const uint64_t *>(o.bias + n);
#pragma unroll
            for (int i = 0; i < 4; ++i) bv[i] = bf((uint16_t)(b4 >> (16 * i)));
        }
        f32x4 gv = {1.f, 1.f, 1.f, 1.f};
        if (EPI == kGatedRes && o.gate != nullptr) gv = *reinterpret_cast<const f32x4 *>(o.gate + n);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const int m = m0 + wm * WM + mb * 16 + x;
            if (m >= o.M) continue;
            const f32x4 y = acc[nb][mb] + bv;
            if constexpr (EPI == kPartial) {
                *reinterpret_cast<f32x4 *>(static_cast<float *>(o.out) + ((int64_t)sp * o.M + m) * o.ldo + n) =
                    acc[nb][mb];
            } else if constexpr (EPI == kGatedRes) {
                f32x4 *p = reinterpret_cast<f32x4 *>(static_cast<float *>(o.out) + (int64_t)m * o.ldo + n);
                *p = *p + gv * y;
            } else {
                bf16x4 w;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    w[i] = (__bf16)(EPI == kBiasGelu ? gelu_tanh(y[i]) : EPI == kBiasSilu ? silu(y[i]) : y[i]);
                *reinterpret_cast<bf16x4 *>(static_cast<uint16_t *>(o.out) + (int64_t)m * o.ldo + n) = w;
            }
        }
    }
}

// LDS bytes of a BM x (16 NB WN) tile: its double-buffered ring, or the
// bf16 output staging if that is larger.
template <int BM, int WN, int NB = 4>
constexpr int lds_bytes()
{
    constexpr int ring = 2 * (BM + 16 * NB * WN) * kRowBytes;
    constexpr int staging = BM * 16 * NB * WN * 2;  // bf16 tile, or half of it in fp32
    return ring > staging ? ring : staging;
}

// XCD-aware tile count helpers for the launchers.
inline int tiles_along(int n, int b)
{
    return (n + b - 1) / b;
}

}  // namespace tile
}  // namespace regenvc

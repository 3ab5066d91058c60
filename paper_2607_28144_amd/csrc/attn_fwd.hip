// gfx950 blockwise exact attention: bf16 MFMA for Q K^T and P V with fp32
// accumulation, online softmax in registers, K/V tiles streamed through LDS.
//
// Method: exact softmax attention computed blockwise over key/value tiles with
// a running (max, sum) per query row -- the same rescaling recurrence by
// which the paper's Ring attention folds key/value blocks together (Sec.
// 3.5); a single launch covers one
// GPU's share (a subset of heads, all or a chunk of the keys).
//
// Work decomposition
//   workgroup = 8 waves = one (batch, head, 256-query tile); one per CU, so
//               each SIMD runs two waves and one wave's exponentials overlap
//               the other's matrix instructions.  Short key ranges use 4-wave
//               workgroups of 128 queries instead, two per CU ("paired").
//   wave      = 32 queries, all head dims, every key tile.
//   key tile  = 64 keys.  K and V tiles are copied HBM -> LDS with
//               global_load_lds_dwordx4 (no register staging) into a ring of
//               LDS stages (3 in the interleaved schedule, 4 in ping-pong,
//               separate K and V rings of 2 when paired).
//   Workgroups are renumbered so that the tiles of one head run on the same
//   XCD (each XCD has its own L2; the hardware deals workgroups round-robin).
//
// Layout trick (interleaved kernel; the ping-pong kernel uses the 16x16x32
//   form, see there): scores are computed transposed, S^T = K Q^T, with
//   v_mfma_f32_32x32x16_bf16 (A = 32 keys x 16 dims from LDS, B = 16 dims x
//   32 queries held in registers).  In the 32x32 accumulator a lane owns ONE
//   query column and 16 of the 32 keys, so row max / row sum are in-register
//   reductions plus one exchange with lane^32 (v_permlane32_swap).  The same
//   accumulator, rounded to bf16, is directly the B operand of O^T = V^T P^T:
//   the MFMA's k-slot -> key assignment it implies is matched by reading V
//   with ds_read_b64_tr_b16 in that key order.  Attention is invariant under
//   a joint permutation of keys and values, so no shuffle is needed.
//
// Two schedules of the key loop (the launch picks one by the number of key
// tiles; results agree to rounding; the interleaved one runs 8 waves or, in
// pairs, 4):
//   interleaved (attn_fwd_kernel), per wave and tile t:
//     phase X:  MFMA  S_{t+1} = K_{t+1} Q^T   beside  VALU  softmax of S_t
//     phase Y:  MFMA  O^T += V_t^T P_t^T       beside  the rest of it
//   ping-pong (attn_fwd_pingpong_kernel): each wave alternates a pure MFMA
//     phase (P V of the previous tile, then Q K^T of the current one) and a
//     pure VALU phase (the weights), the two waves of a SIMD in opposite
//     phases, separated by workgroup barriers; faster on long key ranges,
//     slower on short ones (longer prologue, two barriers per tile).
//
// Lazy rescaling: the running max used as the exponent reference is only
//   raised when a tile's max exceeds it by more than 8 (log2 units); the
//   exponentials are then bounded by 2^8, which fp32 sums and bf16 operands
//   hold as well as values <= 1.  The final O / l and
//   LSE = ln2 * (m_ref + log2 l) are the same quantities for any reference,
//   so this only removes the O-rescale work from the common path; when it is
//   needed it is applied between the phases, outside the MFMA streams.
//
// Two running sums per query: l_r, of the weights as rounded to bf16 for the
//   P V product, divides O (O is then exactly a convex combination of the V
//   rows, whatever the rounding: when one key carries nearly all the weight,
//   its rounding cancels instead of reaching O); l, of the unrounded fp32
//   weights, gives LSE (a single dominant weight's bf16 rounding would move
//   LSE by up to 2^-9).
#include "attn_kernels.hpp"

#include <math.h>

#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <type_traits>

// Split-tile partials of regenvc_attn_fwd_noalloc (callers that cannot
// allocate).  In host code this name is only a stand-in for the symbol:
// kernels get the device address from regenvc::noalloc_scratch().
static __device__ __align__(256) char scratch[regenvc::kNoAllocScratchBytes];

namespace regenvc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) char lds_char;

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kBlockN = 64;                 // keys per tile
constexpr int kStages = 3;                  // LDS ring depth (interleaved schedule)
constexpr int kAhead = kStages - 1;         // tiles in flight (interleaved schedule)
constexpr int kStagesPP = 4;                // LDS ring depth (ping-pong schedule)
// Launches whose work items span at least this many key tiles use the
// ping-pong schedule; shorter ones (cross-attention to a few hundred
// context tokens) the interleaved one, whose prologue and epilogue are
// shorter (measured: ping-pong 2.5 % faster at 171 key tiles, 1 % at 43,
// 6.6 % slower at 8).
constexpr int kPingPongMinTiles = 32;
constexpr float kRescaleThreshold = 8.0f;   // log2 units
// Largest sum of one lane's 16 weights of a key half accepted against a
// speculative reference (the same bound on each weight as kRescaleThreshold).
constexpr float kSpecLimit = 256.f;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int D, int STAGES = kStages, int THREADS = kThreads>
struct Geo {
    static constexpr int NCH = D / 8;                      // 16-byte chunks per row
    static constexpr int DS = D / 16;                      // k-steps of Q K^T
    static constexpr int DB = D / 32;                      // 32-row blocks of O^T
    static constexpr int TILE = kBlockN * D * 2;           // bytes of one K or V tile
    static constexpr int STAGE = 2 * TILE;                 // K tile then V tile
    static constexpr int LDS = STAGES * STAGE;
    static constexpr int LOADS = kBlockN * NCH / THREADS;  // 16-byte loads per thread per tensor per tile
    static_assert(LOADS >= 1 && (kBlockN * NCH) % THREADS == 0, "tile load split");
};

// LDS placement of 16-byte chunk `ch` of tile row `row` (an involution in ch).
// K rows are read 16 B per lane, 32 consecutive rows at one chunk: XOR with the
// row spreads them over distinct banks.  V rows are read with the 8-byte
// transposing load, 4 consecutive rows x 2 adjacent chunks per 16 lanes: XOR
// with 4*(row%4) keeps those 8 (and, with the neighbouring 16 lanes, 16)
// chunks distinct.
template <int NCH>
__device__ __forceinline__ int k_slot(int row, int ch) { return ch ^ (row & (NCH - 1)); }
template <int NCH>
__device__ __forceinline__ int v_slot(int row, int ch) { return ch ^ ((4 * (row & 3)) & (NCH - 1)); }
// V placement of the ping-pong kernel, whose transposing reads take 4
// consecutive rows x 2 adjacent chunks per 16 lanes but rows 4g.. for lane
// group g, so that two 16-lane groups read the same bank columns under the
// XOR above.  With d = 128 the extra XOR of 2 (rows 4-11 of every 16) moves
// groups 1 and 2 to the other half of the banks: any two of the four groups
// that differ in one index bit then read 16 distinct chunks together.
template <int NCH>
__device__ __forceinline__ int vp_slot(int row, int ch)
{
    if constexpr (NCH == 16)
        return ch ^ (4 * (row & 3) + 2 * (((row >> 2) ^ (row >> 3)) & 1));
    else
        return v_slot<NCH>(row, ch);
}

// The copies below name M0 as clobbered: they set it to the LDS destination,
// and the compiler must not keep a value of its own there across them.  Clang
// warns that M0 is a reserved register; the clobber is still honoured (it
// reloads M0 before its own uses), so the warning is silenced here only.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16-byte HBM -> LDS copy (global_load_lds_dwordx4): lane i's 16 bytes land at
// lds_base + 16 * i.  Written as inline asm so the compiler does not treat it
// as an LDS store it must wait for before every later LDS read (it cannot
// tell the ring stages apart); completion is awaited explicitly with
// s_waitcnt vmcnt before the barrier that publishes a stage.
__device__ __forceinline__ void lds_dma16(const void *gptr, uint32_t lds_base)
{
    const uint32_t base = __builtin_amdgcn_readfirstlane(lds_base);  // wave-uniform by construction
    __asm__ volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" : : "s"(base), "v"(gptr) : "m0");
}

// Same copy with a scalar (wave-uniform) base address and a 32-bit lane offset.
__device__ __forceinline__ void lds_dma16_s(const void *gbase, uint32_t off, uint32_t lds_base)
{
    const uint32_t base = __builtin_amdgcn_readfirstlane(lds_base);
    const uint64_t g = (uint64_t)(uintptr_t)gbase;
    // readfirstlane yields an int: widen each half through uint32_t so the low
    // half is zero-extended (a sign-extended low half corrupts the address)
    const uint32_t ghi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(g >> 32));
    const uint32_t glo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)g);
    const uint64_t gs = ((uint64_t)ghi << 32) | (uint64_t)glo;
    __asm__ volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                     :
                     : "s"(base), "v"(off), "s"((const void *)(uintptr_t)gs)
                     : "m0");
}

// The LOADS copies of one tile tensor by this thread with a wave-uniform
// source base and LDS address: lane offsets off[j], LDS block j at
// lds_base + j KB.  M0 is set once per group; the immediate offset (applied
// to the global and the LDS address alike) steps the LDS block, and the
// scalar base is lowered by the same amount so that the global address is
// base + off[j].  The leading nop covers a scalar base written just before by
// a vector instruction (readfirstlane).
template <int LOADS>
__device__ __forceinline__ void lds_dma16_group(const uint16_t *base, const uint32_t (&off)[LOADS], uint32_t lds_base)
{
    const uint64_t b = (uint64_t)(uintptr_t)base;  // integer arithmetic: b - 1024 may precede the tensor
    if constexpr (LOADS == 1) {
        __asm__ volatile("s_nop 4\n\ts_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :
                         : "s"(lds_base), "v"(off[0]), "s"(b)
                         : "m0");
    } else {
        static_assert(LOADS == 2, "copy group of one or two chunks");
        __asm__ volatile("s_nop 4\n\ts_mov_b32 m0, %0\n\t"
                         "global_load_lds_dwordx4 %1, %3\n\t"
                         "global_load_lds_dwordx4 %2, %4 offset:1024"
                         :
                         : "s"(lds_base), "v"(off[0]), "v"(off[1]), "s"(b), "s"(b - 1024)
                         : "m0");
    }
}
#pragma clang diagnostic pop

// A pointer the caller knows to be wave-uniform, moved to scalar registers.
__device__ __forceinline__ const uint16_t *uniform_ptr(const uint16_t *p)
{
    const uint64_t g = (uint64_t)(uintptr_t)p;
    const uint32_t ghi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(g >> 32));
    const uint32_t glo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)g);
    return (const uint16_t *)(uintptr_t)(((uint64_t)ghi << 32) | (uint64_t)glo);
}

// (x of this lane, x of lane^32) combined so both halves hold the same value.
__device__ __forceinline__ float pair_max(float x)
{
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x)
{
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// x combined over the four lanes l, l^16, l^32, l^48 (each gets the result).
__device__ __forceinline__ float quad_max(float x)
{
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float t = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    auto u = __builtin_amdgcn_permlane32_swap(__float_as_uint(t), __float_as_uint(t), false, false);
    return fmaxf(__uint_as_float(u[0]), __uint_as_float(u[1]));
}
__device__ __forceinline__ float quad_sum(float x)
{
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float t = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    auto u = __builtin_amdgcn_permlane32_swap(__float_as_uint(t), __float_as_uint(t), false, false);
    return __uint_as_float(u[0]) + __uint_as_float(u[1]);
}

// Stores the weights (x0, x1), rounded to bf16 (nearest even, one packed
// conversion), as weights j, j+1 of a P operand, and adds the two rounded
// values to rs: one v_dot2c_f32_bf16 of the packed pair against (1, 1), so
// that the sum that normalizes O is the sum of exactly the weights the P V
// product multiplies (O is then a convex combination of V rows).
__device__ __forceinline__ void put_pair(bf16x8 &dst, int j, float x0, float x1, float &rs)
{
    bf16x2 pk;
    pk[0] = (__bf16)x0;
    pk[1] = (__bf16)x1;
    dst[j] = pk[0];
    dst[j + 1] = pk[1];
    const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
    rs = __builtin_amdgcn_fdot2_f32_bf16(pk, one, rs, false);
}

// Online-softmax step for one 32-query block over one 64-key tile.
//   s      : S^T accumulators of the two 32-key halves (raw q.k dot products);
//            register i of half kb holds key kb*32 + (i/4)*8 + hi*4 + i%4 of
//            the tile for this lane's query
//   c      : scale * log2(e)
//   mref   : exponent reference (log2 units), raised lazily
//   lsum   : running fp32 sum of exp2(s*c - mref) over this lane's keys (the
//            unrounded weights; it gives LSE)
//   rsum   : running sum of the same weights rounded to bf16 (it normalizes O)
//   p      : bf16 P^T operands of the four 16-key MFMA steps of the tile
//   alpha  : factor the O accumulator must be multiplied by (1 if unchanged)
//   upd    : wave-uniform flag: some lane raised its reference
// MASK: keys at or past Skv (only in the last tile) get weight exactly 0.
template <bool MASK>
__device__ __forceinline__ void softmax_block(const f32x16 (&s)[2], float c, float &mref, float &lsum, float &rsum,
                                              bf16x8 (&p)[4], float &alpha, bool &upd, int key0, int Skv)
{
    const int hi = (threadIdx.x >> 5) & 1;
    auto valid = [&](int kb, int i) { return key0 + kb * 32 + (i >> 2) * 8 + hi * 4 + (i & 3) < Skv; };
    float m0 = -INFINITY, m1 = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        m0 = fmaxf(m0, (!MASK || valid(0, i)) ? s[0][i] : -INFINITY);
        m1 = fmaxf(m1, (!MASK || valid(1, i)) ? s[1][i] : -INFINITY);
    }
    const float mt = pair_max(fmaxf(m0, m1)) * c;
    upd = __builtin_amdgcn_ballot_w64(mt > mref + kRescaleThreshold) != 0;
    const float mnew = upd ? fmaxf(mref, mt) : mref;
    alpha = __builtin_amdgcn_exp2f(mref - mnew);
    mref = mnew;
    const float nm = -mnew;
    float acc0 = 0.f, acc1 = 0.f, racc = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; i += 2) {
            float e0 = __builtin_amdgcn_exp2f(fmaf(s[kb][i], c, nm));
            float e1 = __builtin_amdgcn_exp2f(fmaf(s[kb][i + 1], c, nm));
            if (MASK) {
                e0 = valid(kb, i) ? e0 : 0.f;
                e1 = valid(kb, i + 1) ? e1 : 0.f;
            }
            put_pair(p[kb * 2 + (i >> 3)], i & 7, e0, e1, racc);
            acc0 += e0;
            acc1 += e1;
        }
    lsum = fmaf(lsum, alpha, acc0 + acc1);
    rsum = fmaf(rsum, alpha, racc);
}

// One key/value context of a (batch, head): K and V base pointers, row
// strides (elements), length, key tiles, and whether tile copies can use
// 32-bit lane offsets.
struct KvSrc {
    const uint16_t *k, *v;
    int64_t k_ss, v_ss;
    int Skv, n_kt;
    bool off32;
};

// Work item of a workgroup: one key range of a split tile (the first
// n_units workgroups, so that these short items start with the first round
// instead of trailing the last one) or a whole query tile.  Whole tiles are
// renumbered XCD-aware: workgroup i runs on XCD i % 8, i.e. whole tile j on
// XCD (j + n_units) % 8, a fixed rotation of j % 8; each XCD gets a
// contiguous range of tiles so that one head's tiles share an L2.
struct WorkItem {
    int tile, kt0, kt1, slot;  // slot: workspace row block of a key range, -1 for a whole tile
    int src;                   // context of a key range (dual launches: 1 = the second)
};
__device__ __forceinline__ WorkItem work_item(const AttnPlan &pl, int item)
{
    WorkItem w;
    w.src = 0;
    if (item < pl.n_units) {
        const int per = pl.seg + pl.seg2;
        int sgi = item % per, seg = pl.seg, nkt = pl.n_kt;
        if (sgi >= pl.seg) {
            sgi -= pl.seg;
            seg = pl.seg2;
            nkt = pl.n_kt2;
            w.src = 1;
        }
        w.tile = pl.n_dp + item / per;
        w.kt0 = (int)((int64_t)sgi * nkt / seg);
        w.kt1 = (int)((int64_t)(sgi + 1) * nkt / seg);
        w.slot = item;
    } else {
        const int j = item - pl.n_units;
        const int xcd = j & 7;
        w.tile = xcd * (pl.n_dp >> 3) + min(xcd, pl.n_dp & 7) + (j >> 3);
        w.kt0 = 0;
        w.kt1 = pl.n_kt;
        w.slot = -1;
    }
    return w;
}

// Chunked-partials launches: the chunk of a tile gives its key range (K/V
// bases moved to the chunk's first key, the chunk length as Skv) and its
// outputs, and the tile index becomes the one within the chunk.  Other
// launches pass through unchanged.
__device__ __forceinline__ AttnArgs chunk_of(const AttnArgs &a, const AttnPlan &pl, int &tile)
{
    if (pl.tiles_per_chunk == 0) return a;
    const int c = tile / pl.tiles_per_chunk;
    tile -= c * pl.tiles_per_chunk;
    AttnArgs r = a;
    r.k = static_cast<const uint16_t *>(a.k) + (int64_t)a.ck0[c] * a.k_ss;
    r.v = static_cast<const uint16_t *>(a.v) + (int64_t)a.ck0[c] * a.v_ss;
    r.Skv = a.clen[c];
    r.o = a.co[c];
    r.lse = a.clse[c];
    return r;
}

// The same for a work item, with the key tiles of its chunk (n_kt) and, for
// a whole tile, its key range.  A split tile's ranges were planned on the
// last chunk's key tiles, which every split tile's chunk has.
__device__ __forceinline__ AttnArgs chunk_view(const AttnArgs &a, const AttnPlan &pl, WorkItem &wi, int &n_kt)
{
    const AttnArgs r = chunk_of(a, pl, wi.tile);
    n_kt = pl.tiles_per_chunk == 0 ? pl.n_kt : (r.Skv + kBlockN - 1) / kBlockN;
    if (wi.slot < 0) wi.kt1 = n_kt;
    return r;
}

// Ring accumulate: how a row's running state (normalized O_run over the key
// chunks seen so far, and its LSE L_run) and this launch's normalized result
// (O_c, L_c) combine, by the log-sum-exp identity of the chunk merge:
// L = log(e^L_run + e^L_c), O = e^(L_run - L) O_run + e^(L_c - L) O_c.  A row
// with L_run = -inf has seen no key: its O_run values (anything, NaN
// included) do not enter the result.
struct RunMerge {
    float wr, wc, lse;
    bool run;  // O_run enters the result
};
__device__ __forceinline__ RunMerge run_merge(float lr, float lc)
{
    RunMerge m;
    m.run = !(lr == -INFINITY);
    if (!m.run) {
        m.wr = 0.f;
        m.wc = 1.f;
        m.lse = lc;
        return m;
    }
    const float mx = fmaxf(lr, lc);
    const float er = expf(lr - mx), ec = expf(lc - mx);
    const float s = er + ec;
    m.wr = er / s;
    m.wc = ec / s;
    m.lse = mx + logf(s);
    return m;
}

// Four consecutive output values of a row: w.wc * oc (+ w.wr * run, the
// running output's values, when the running state enters), stored as f32 or
// bf16 at element d of the row.
template <bool OUT_F32>
__device__ __forceinline__ void put_out4(char *orow, const RunMerge &w, int d, f32x4 oc, f32x4 run)
{
    f32x4 r = oc * w.wc;
    if (w.run) r += run * w.wr;
    if constexpr (OUT_F32) {
        *reinterpret_cast<f32x4 *>(orow + d * 4) = r;
    } else {
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (__bf16)r[e];
        *reinterpret_cast<bf16x4 *>(orow + d * 2) = o;
    }
}

// The running state of row qi (clamped into the sequence, so that a padded
// query row reads a real row it then ignores): LSE and the f32x4 chunks at
// d = d0 + j * dstep of the running output, all loaded before any output is
// written (the output may be the running output itself, so a store must not
// come between them).
template <int N>
__device__ __forceinline__ float load_run(const AttnArgs &a, int b, int h, int qi, int d0, int dstep, f32x4 (&run)[N])
{
    qi = min(qi, a.Sq - 1);
    const float *rrow = a.run_o + ((int64_t)b * a.r_sb + (int64_t)qi * a.r_ss + (int64_t)h * a.r_sh);
#pragma unroll
    for (int j = 0; j < N; ++j) run[j] = *reinterpret_cast<const f32x4 *>(rrow + d0 + j * dstep);
    return a.run_lse[((int64_t)b * a.H + h) * a.Sq + qi];
}

// Epilogue of one lane's query row: O = O^T / l_r and LSE = ln2 * (m_ref +
// log2 l), with l_r the sum of the rounded weights and l of the unrounded
// ones; a split tile's key range writes its normalized partial to the
// workspace instead.  lsum and rsum are this lane's halves of l and l_r (the
// other halves are in lane^32).
template <int D, bool OUT_F32, bool ACC, int BM>
__device__ __forceinline__ void store_row(const AttnArgs &a, const AttnPlan &pl, const f32x16 (&oacc)[D / 32],
                                          float lsum, float rsum, float mref, int b, int h, int qi, int qrow, int slot)
{
    constexpr int DB = D / 32;
    const int hi = (threadIdx.x >> 5) & 1;
    const float lt = pair_sum(lsum);
    const float inv = 1.0f / pair_sum(rsum);
    const float lse_val = (mref + __log2f(lt)) * kLn2;
    if (qi >= a.Sq) return;
    if (slot >= 0) {
        float *orow = pl.ws_o + ((int64_t)slot * BM + qrow) * D;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                f32x4 w;
#pragma unroll
                for (int e = 0; e < 4; ++e) w[e] = oacc[db][gq * 4 + e] * inv;
                *reinterpret_cast<f32x4 *>(orow + db * 32 + gq * 8 + hi * 4) = w;
            }
        if (hi == 0) pl.ws_lse[(int64_t)slot * BM + qrow] = lse_val;
    } else {
        char *orow = static_cast<char *>(a.o) +
                     ((int64_t)b * a.o_sb + (int64_t)qi * a.o_ss + (int64_t)h * a.o_sh) * (OUT_F32 ? 4 : 2);
        f32x4 run[ACC ? DB * 4 : 1] = {};
        RunMerge w{0.f, 1.f, lse_val, false};
        if constexpr (ACC) w = run_merge(load_run(a, b, h, qi, hi * 4, 8, run), lse_val);
        w.wc *= inv;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                f32x4 oc;
#pragma unroll
                for (int e = 0; e < 4; ++e) oc[e] = oacc[db][gq * 4 + e];
                put_out4<OUT_F32>(orow, w, db * 32 + gq * 8 + hi * 4, oc, run[ACC ? db * 4 + gq : 0]);
            }
        if (a.lse != nullptr && hi == 0) a.lse[((int64_t)b * a.H + h) * a.Sq + qi] = w.lse;
    }
}

// bf16 output of a whole tile as full rows: each wave stages its 32 rows in
// LDS at `stg` (32 * D * 2 bytes, 16-byte chunks XOR-swizzled by row) with
// stage_out4, then store_staged_rows writes 64 / (D/8) whole rows of 16-byte
// chunks per store instruction.  Writing straight from the accumulator
// layouts instead scatters each instruction over 16 or 32 rows, a few bytes
// apiece, and the stores of a 256-row tile then take about 60 % longer to
// drain.  The caller has made sure that no wave still reads the LDS at `stg`;
// a wave reads back only what it wrote, so its own LDS ordering suffices.
template <int D>
__device__ __forceinline__ void stage_out4(lds_char *stg, int r, int d, const bf16x4 &w)
{
    constexpr int CPR = D / 8;  // 16-byte chunks per row
    *(lds_bf16x4 *)(stg + r * D * 2 + (((d >> 3) ^ (r & (CPR - 1))) << 4) + (d & 4) * 2) = w;
}

template <int D>
__device__ __forceinline__ void store_staged_rows(const AttnArgs &a, const lds_char *stg, int lane, int b, int h,
                                                  int row0)
{
    constexpr int CPR = D / 8;     // 16-byte chunks per row
    constexpr int RPI = 64 / CPR;  // rows per store instruction
#pragma unroll
    for (int it = 0; it < 32 / RPI; ++it) {
        const int r = it * RPI + lane / CPR, c = lane % CPR;
        const bf16x8 w = *(const lds_bf16x8 *)(stg + r * D * 2 + (c ^ (r & (CPR - 1))) * 16);
        const int qr = row0 + r;
        if (qr < a.Sq)
            *reinterpret_cast<bf16x8 *>(static_cast<char *>(a.o) +
                                        ((int64_t)b * a.o_sb + (int64_t)qr * a.o_ss + (int64_t)h * a.o_sh) * 2 + c * 16) = w;
    }
}

// The same for f32 rows (32 * D * 4 bytes of LDS per wave).
template <int D>
__device__ __forceinline__ void stage_out4_f32(lds_char *stg, int r, int d, const f32x4 &w)
{
    constexpr int CPR = D / 4;  // 16-byte chunks per row
    *(__attribute__((address_space(3))) f32x4 *)(stg + r * D * 4 + (((d >> 2) ^ (r & (CPR - 1))) << 4)) = w;
}

template <int D>
__device__ __forceinline__ void store_staged_rows_f32(const AttnArgs &a, const lds_char *stg, int lane, int b, int h,
                                                      int row0)
{
    constexpr int CPR = D / 4;     // 16-byte chunks per row
    constexpr int RPI = 64 / CPR;  // rows per store instruction
#pragma unroll
    for (int it = 0; it < 32 / RPI; ++it) {
        const int r = it * RPI + lane / CPR, c = lane % CPR;
        const f32x4 w = *(const __attribute__((address_space(3))) f32x4 *)(stg + r * D * 4 + (c ^ (r & (CPR - 1))) * 16);
        const int qr = row0 + r;
        if (qr < a.Sq)
            *reinterpret_cast<f32x4 *>(static_cast<char *>(a.o) +
                                       ((int64_t)b * a.o_sb + (int64_t)qr * a.o_ss + (int64_t)h * a.o_sh) * 4 + c * 16) = w;
    }
}

// Staged rows of the ring accumulate: the staged values are this launch's
// normalized O times its merge weight; row r then adds w_r * O_run, with w_r
// < 0 marking a row without running state (O_run ignored).  w_r is held by
// lane r % 16 of the ping-pong layout, as wr[r / 16].  All O_run chunks are
// loaded before the first store (the output may be O_run itself).
template <int D, bool OUT_F32>
__device__ __forceinline__ void store_staged_rows_run(const AttnArgs &a, const lds_char *stg, int lane, int b, int h,
                                                      int row0, const float (&wr)[2])
{
    constexpr int ESZ = OUT_F32 ? 4 : 2;
    constexpr int CPR = D * ESZ / 16;  // 16-byte chunks per row
    constexpr int VPC = 16 / ESZ;      // values per chunk
    constexpr int RPI = 64 / CPR;      // rows per instruction (divides 16)
    constexpr int NIT = 32 / RPI;
    static_assert(16 % RPI == 0, "one query block per instruction");
    f32x4 run[NIT][VPC / 4];
    float w[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int r = it * RPI + lane / CPR, c = lane % CPR;
        w[it] = __shfl(it * RPI < 16 ? wr[0] : wr[1], r & 15, 64);
        const int qc = min(row0 + r, a.Sq - 1);
        const float *rrow = a.run_o + ((int64_t)b * a.r_sb + (int64_t)qc * a.r_ss + (int64_t)h * a.r_sh) + c * VPC;
#pragma unroll
        for (int k = 0; k < VPC / 4; ++k) run[it][k] = *reinterpret_cast<const f32x4 *>(rrow + 4 * k);
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int r = it * RPI + lane / CPR, c = lane % CPR;
        const int qr = row0 + r;
        const lds_char *src = stg + r * D * ESZ + (c ^ (r & (CPR - 1))) * 16;
        char *dst = static_cast<char *>(a.o) + ((int64_t)b * a.o_sb + (int64_t)qr * a.o_ss + (int64_t)h * a.o_sh) * ESZ +
                    c * 16;
        if constexpr (OUT_F32) {
            f32x4 v = *(const __attribute__((address_space(3))) f32x4 *)src;
            if (w[it] >= 0.f) v += run[it][0] * w[it];
            if (qr < a.Sq) *reinterpret_cast<f32x4 *>(dst) = v;
        } else {
            const bf16x8 sv = *(const lds_bf16x8 *)src;
            bf16x8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float v = (float)sv[e];
                if (w[it] >= 0.f) v += run[it][e / 4][e % 4] * w[it];
                o[e] = (__bf16)v;
            }
            if (qr < a.Sq) *reinterpret_cast<bf16x8 *>(dst) = o;
        }
    }
}

// Interleaved layout: this lane holds row `col` (lane % 32), values at
// d = db*32 + gq*8 + hi*4 + e, already final.
template <int D>
__device__ __forceinline__ void store_tile_bf16(const AttnArgs &a, lds_char *stg, const f32x16 (&val)[D / 32], int lane,
                                                int b, int h, int row0)
{
    constexpr int DB = D / 32;
    const int col = lane & 31, hi = lane >> 5;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            bf16x4 w;
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = (__bf16)val[db][gq * 4 + e];
            stage_out4<D>(stg, col, db * 32 + gq * 8 + hi * 4, w);
        }
    store_staged_rows<D>(a, stg, lane, b, h, row0);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    __asm__ volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// ACC: the ring-accumulate epilogue; DUAL: two contexts summed (each a
// separate instantiation, so that the plain kernels keep their register
// allocation).  A dual launch runs the key pipeline twice over one query
// tile: first context, then, with the first result parked in LDS as bf16
// (the precision of a single context-attention output), the second.
template <int D, bool OUT_F32, bool ACC, bool DUAL = false, int WAVES = kWaves>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_fwd_kernel(AttnArgs a_in, AttnPlan pl)
{
    // Paired launches (WAVES = 4): two workgroups of 128 query rows share a
    // CU, one wave of each per SIMD, so that one's Q load and output drain
    // run beside the other's key loop; K and V then go through rings of two
    // tiles each (64 KB of LDS per workgroup for d = 128), see `step`.
    constexpr bool PAIRED = WAVES != kWaves;
    static_assert(!PAIRED || (WAVES == 4 && !DUAL), "paired launches: 4 waves, one context");
    constexpr int THREADS = 64 * WAVES;
    using G = Geo<D, PAIRED ? 2 : kStages, THREADS>;
    constexpr int NCH = G::NCH, DS = G::DS, DB = G::DB, LOADS = G::LOADS;
    constexpr int BM = WAVES * 32;
    constexpr int PER_TILE = 2 * LOADS;  // copies in flight per thread per tile (K and V)

    // dual launches: + the first context's normalized O (bf16), 16-byte chunk
    // j of thread t at byte G::LDS + 16 * (j * THREADS + t)
    __shared__ __attribute__((aligned(1024))) char smem[G::LDS + (DUAL ? BM * D * 2 : 0)];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const int hi = lane >> 5;   // which half of the wave
    const int col = lane & 31;  // query column owned in the 32x32 accumulators

    WorkItem wi = work_item(pl, blockIdx.x);
    int n_kt;
    const AttnArgs a = chunk_view(a_in, pl, wi, n_kt);
    const int tile = wi.tile, slot = wi.slot;
    const int qt = tile % pl.n_qtiles;
    const int bh = tile / pl.n_qtiles;
    const int h = bh % a.H;
    const int b = bh / a.H;
    const int qrow = wave * 32 + col;  // this lane's query within the tile
    const int qi = qt * BM + qrow;     // ... and in the sequence

    const uint16_t *qp = static_cast<const uint16_t *>(a.q) + b * a.q_sb + h * a.q_sh;
    const int Sq = a.Sq;
    // key/value contexts of this (b, h)
    const KvSrc src0{static_cast<const uint16_t *>(a.k) + b * a.k_sb + h * a.k_sh,
                     static_cast<const uint16_t *>(a.v) + b * a.v_sb + h * a.v_sh,
                     a.k_ss, a.v_ss, a.Skv, n_kt, a.kv_off32};

    // Q^T operand fragments stay in registers for the whole key loop.
    bf16x8 qf[DS];
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
        if (qi < Sq)
            qf[ds] = *reinterpret_cast<const bf16x8 *>(qp + (int64_t)qi * a.q_ss + ds * 16 + hi * 8);
        else
            qf[ds] = bf16x8{};
    }

    const KvSrc src1 = DUAL ? KvSrc{static_cast<const uint16_t *>(a.k2) + b * a.k2_sb + h * a.k2_sh,
                                    static_cast<const uint16_t *>(a.v2) + b * a.v2_sb + h * a.v2_sh,
                                    a.k2_ss, a.v2_ss, a.Skv2, pl.n_kt2, a.kv2_off32}
                            : src0;
    f32x16 oacc[DB];
    float mref, lsum, rsum;
    const float c = a.scale * kLog2e;
    float lse1 = 0.f;  // dual launches: LSE of the first context

    // Passes of the key pipeline, each from the empty state into (oacc, mref,
    // lsum): one over the work item's key range, or (dual launches, whole
    // tiles) one over each context.
    const int n_pass = DUAL && slot < 0 ? 2 : 1;
    // unrolled for dual launches: each pass then gets its own register
    // allocation (as a loop, the state carried between the passes spilled)
#pragma unroll
    for (int ps = 0; ps < (DUAL ? 2 : 1); ++ps) {
    if (ps >= n_pass) break;
    if (DUAL && ps == 1) {
        // the second pass reads its Q fragments again (from L2, as a rule)
        // rather than keeping them live through the first pass's epilogue
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) {
            if (qi < Sq)
                qf[ds] = *reinterpret_cast<const bf16x8 *>(qp + (int64_t)qi * a.q_ss + ds * 16 + hi * 8);
            else
                qf[ds] = bf16x8{};
        }
    }
    const KvSrc src = (DUAL && (slot >= 0 ? wi.src : ps) == 1) ? src1 : src0;
    const int kt0 = wi.kt0;
    const int kt1 = DUAL && slot < 0 ? src.n_kt : wi.kt1;
    const uint16_t *kp = src.k, *vp = src.v;
    const int Skv = src.Skv;
    // only the last key tile of the whole context can be ragged
    const bool ragged_end = kt1 == src.n_kt && (Skv % kBlockN) != 0;

    // HBM -> LDS copy of one key tile into a ring stage.  Each wave
    // instruction fills 1 KB of LDS (64 lanes x 16 B, in lane order); the
    // lane fetches the chunk the swizzle places there.  Rows past the last
    // key re-read the last key (finite data; their softmax weight is 0).
    // Copies requested past the last tile repeat it into the otherwise unused
    // stage, so every call issues exactly PER_TILE copies per thread and the
    // vmcnt waits below count whole tiles.
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char *)smem;
    uint32_t kofs[LOADS], vofs[LOADS];
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
        const int slot16 = (wave * LOADS + j) * 64 + lane;
        const int row = slot16 / NCH, phys = slot16 % NCH;
        kofs[j] = (uint32_t)((row * src.k_ss + k_slot<NCH>(row, phys) * 8) * 2);
        vofs[j] = (uint32_t)((row * src.v_ss + v_slot<NCH>(row, phys) * 8) * 2);
    }
    // Tiles are copied in order kt0, kt0+1, ... (one call per tile); the
    // scalar source bases advance by one tile per call and stay on the last
    // tile once it is reached.  `stage` is the ring stage to fill.
    const int64_t k_step = (int64_t)kBlockN * src.k_ss, v_step = (int64_t)kBlockN * src.v_ss;
    const int last_full = Skv / kBlockN - 1;  // last tile with kBlockN keys
    int tl_copy = kt0;
    const uint16_t *kb_copy = kp + kt0 * k_step;
    const uint16_t *vb_copy = vp + kt0 * v_step;
    auto issue_next = [&](int stage) {
        const uint32_t kdst = lds0 + stage * G::STAGE;
        const uint32_t vdst = kdst + G::TILE;
        if (src.off32 && tl_copy <= last_full) {
            // full tile: scalar tile base + precomputed 32-bit lane offsets
#pragma unroll
            for (int j = 0; j < LOADS; ++j) {
                const uint32_t blk = (wave * LOADS + j) * 1024;
                lds_dma16_s(kb_copy, kofs[j], kdst + blk);
                lds_dma16_s(vb_copy, vofs[j], vdst + blk);
            }
        } else {
            const int key0 = tl_copy * kBlockN;
            const int last = Skv - 1 - key0;
#pragma unroll
            for (int j = 0; j < LOADS; ++j) {
                const int blk = wave * LOADS + j;
                const int slot16 = blk * 64 + lane;
                const int row = slot16 / NCH, phys = slot16 % NCH;
                const int64_t key = key0 + min(row, last);
                lds_dma16(kp + key * src.k_ss + k_slot<NCH>(row, phys) * 8, kdst + blk * 1024);
                lds_dma16(vp + key * src.v_ss + v_slot<NCH>(row, phys) * 8, vdst + blk * 1024);
            }
        }
        if (tl_copy < kt1 - 1) {
            ++tl_copy;
            kb_copy += k_step;
            vb_copy += v_step;
        }
    };
    auto next_stage = [](int st) { return st == G::LDS / G::STAGE - 1 ? 0 : st + 1; };
    static_assert(PAIRED || (kAhead == 2 && kStages == 3), "the step issues tile t+2 into the stage of tile t-1");
    // Paired launches: one tensor's copy of tile tl into the K or V half of
    // the stage at LDS byte dst (same lane layout and clamping as above).
    auto issue_one = [&](int tl, uint32_t dst, auto is_v) __attribute__((always_inline)) {
        constexpr bool V = decltype(is_v)::value;
        const uint16_t *base = V ? vp : kp;
        const int64_t ss = V ? src.v_ss : src.k_ss;
        if (src.off32 && tl <= last_full) {
            const uint16_t *tb = base + (int64_t)tl * kBlockN * ss;
#pragma unroll
            for (int j = 0; j < LOADS; ++j)
                lds_dma16_s(tb, V ? vofs[j] : kofs[j], dst + (wave * LOADS + j) * 1024);
        } else {
            const int key0 = tl * kBlockN;
            const int last = Skv - 1 - key0;
#pragma unroll
            for (int j = 0; j < LOADS; ++j) {
                const int blk = wave * LOADS + j;
                const int slot16 = blk * 64 + lane;
                const int row = slot16 / NCH, phys = slot16 % NCH;
                const int64_t key = key0 + min(row, last);
                const int ch = V ? v_slot<NCH>(row, phys) : k_slot<NCH>(row, phys);
                lds_dma16(base + key * ss + ch * 8, dst + blk * 1024);
            }
        }
    };

    // Per-lane LDS byte offsets of the MFMA operand fragments (stage 0).
    int koff[DS];
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) koff[ds] = (col * D + k_slot<NCH>(col, ds * 2 + hi) * 8) * 2;
    const int g = lane >> 4, x = lane & 15;
    int voff[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        const int row = 4 * (g >> 1) + (x >> 2);
        const int dcol = db * 32 + 16 * (g & 1) + 4 * (x & 3);
        voff[db] = G::TILE + (row * D + v_slot<NCH>(row, dcol >> 3) * 8 + (dcol & 7)) * 2;
    }

    constexpr int NK = 2 * DS;  // K fragments (MFMAs) per tile for S^T
    constexpr int NV = 4 * DB;  // V fragments (MFMAs) per tile for O^T
    constexpr int PF = 4;       // fragments read ahead of their MFMA
    static_assert(NK >= 8 && NV >= PF, "schedule assumes d >= 64");

    // K fragment i (i = 2*ds + kb): rows kb*32.., dims 16*ds.. of the tile.
    auto kfrag = [&](const lds_char *kt, int i) -> bf16x8 {
        return *(const lds_bf16x8 *)(kt + koff[i >> 1] + (i & 1) * 32 * D * 2);
    };
    // V^T fragment i (i = kk*DB + db): dims 32*db.., keys 16*kk.. of the tile;
    // the lower half-wave supplies keys {0-3, 8-11}, the upper {4-7, 12-15}
    // (the S^T accumulator order).
    auto vfrag = [&](const lds_char *vt, int i) -> bf16x8 {
        const int kk = i / DB, db = i % DB;
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(vt + voff[db] + kk * 16 * D * 2));
        const bf16x4 up =
            __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(vt + voff[db] + (kk * 16 + 8) * D * 2));
        return bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
    };
    auto stage_ptr = [&](int st) { return (const lds_char *)(smem + st * G::STAGE); };

    // S^T (two 32-key halves) of the key tile in stage `st`, plain (prologue
    // only).
    auto qk = [&](int st, f32x16 (&s)[2]) {
        const lds_char *kt = stage_ptr(st);
        s[0] = s[1] = f32x16{};
#pragma unroll
        for (int i = 0; i < NK; ++i)
            s[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kfrag(kt, i), qf[i >> 1], s[i & 1], 0, 0, 0);
    };

#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
    mref = -INFINITY;
    lsum = rsum = 0.f;
    f32x16 scur[2], snext[2];
    bf16x8 p[4];
    float alpha = 1.f;
    bool upd = false;
    // softmax state carried from phase X into phase Y of a step: -mref, the
    // first half's weight sums (unrounded, rounded) and the second half's
    // partial sums
    float nm = 0.f, acc0 = 0.f, acc1 = 0.f, acc2 = 0.f, racc0 = 0.f, racc1 = 0.f;

    // O^T += V^T P^T for the key tile in stage `st`: each MFMA's V fragment is read PF
    // MFMAs ahead; the order is pinned so that the waits stay PF deep.  With
    // `tail`, the MFMAs carry the weights of the second key half of this tile
    // (P operands 2 and 3): one piece after each of the first NV/2 MFMAs,
    // then the overflow check of that half, before P operand 2 is first used.
    auto pv = [&](int st, auto tail, const f32x16 (&sc)[2]) {
        constexpr bool TAIL = decltype(tail)::value;
        constexpr int TN = 32 / NV;  // weights per piece
        const lds_char *vt = stage_ptr(st);
        bf16x8 vr[PF];
#pragma unroll
        for (int i = 0; i < PF; ++i) vr[i] = vfrag(vt, i);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            oacc[i % DB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vr[i % PF], p[i / DB], oacc[i % DB], 0, 0, 0);
            if (i + PF < NV) vr[i % PF] = vfrag(vt, i + PF);
            if constexpr (TAIL) {
                if (i < NV / 2) {
#pragma unroll
                    for (int e = i * TN; e < (i + 1) * TN; e += 2) {
                        const float x0 = __builtin_amdgcn_exp2f(fmaf(sc[1][e], c, nm));
                        const float x1 = __builtin_amdgcn_exp2f(fmaf(sc[1][e + 1], c, nm));
                        put_pair(p[2 + (e >> 3)], e & 7, x0, x1, racc1);
                        acc1 += x0;
                        acc2 += x1;
                    }
                }
                if (i == NV / 2 - 1) {
                    // second key half against the same reference: raise it
                    // (and rescale everything accumulated so far, including
                    // this tile's first half) if its weights overflow the limit
                    __builtin_amdgcn_sched_barrier(0);
                    float a2 = acc1 + acc2;
                    const bool up2 = __builtin_amdgcn_ballot_w64(!(a2 <= kSpecLimit) && a2 == a2) != 0;
                    if (up2) {
                        float m1 = -INFINITY;
#pragma unroll
                        for (int e = 0; e < 16; ++e) m1 = fmaxf(m1, sc[1][e]);
                        const float mnew = fmaxf(mref, pair_max(m1) * c);
                        const float al = __builtin_amdgcn_exp2f(mref - mnew);
                        mref = mnew;
#pragma unroll
                        for (int db = 0; db < DB; ++db) oacc[db] *= al;
                        lsum *= al;
                        rsum *= al;
                        acc0 *= al;
                        racc0 *= al;
                        acc1 = acc2 = racc1 = 0.f;
#pragma unroll
                        for (int e = 0; e < 16; e += 2) {
                            const float x0 = __builtin_amdgcn_exp2f(fmaf(sc[1][e], c, -mnew));
                            const float x1 = __builtin_amdgcn_exp2f(fmaf(sc[1][e + 1], c, -mnew));
                            put_pair(p[2 + (e >> 3)], e & 7, x0, x1, racc1);
                            acc1 += x0;
                            acc2 += x1;
                        }
                        a2 = acc1 + acc2;
                    }
                    lsum += acc0 + a2;
                    rsum += racc0 + racc1;
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };


    // Phase X of a tile that has a successor: S_{t+1} = K_{t+1} Q^T on the
    // MFMA pipe, and beside it the weights of the first key half of S_t
    // (P operands 0 and 1), one pair after every NK/8-th MFMA, with K
    // fragments read PF MFMAs ahead.  The weights are taken against the
    // current reference without a tile max: if some lane's 16 weights sum to
    // more than kSpecLimit (a jump of the running max, or the first tile,
    // where mref = -inf), the exact max of the tile is taken, the reference
    // raised and the weights recomputed, outside the MFMA stream.  Weights
    // then stay <= kSpecLimit, as with a lazily raised exact max.
    auto qk_softmax = [&](int st_next, const f32x16 (&sc)[2], f32x16 (&sn)[2]) {
        const lds_char *kt = stage_ptr(st_next);
        // The two waves sharing a SIMD contend for its MFMA pipe; the one in
        // this (VALU-heavy) phase goes first, and the other's P V products
        // fill the gaps between its MFMAs.
        __builtin_amdgcn_s_setprio(1);
        constexpr int STRIDE = NK / 8;
        bf16x8 kr[PF];
        acc0 = acc1 = racc0 = 0.f;
        const float nm0 = -mref;
#pragma unroll
        for (int i = 0; i < PF; ++i) kr[i] = kfrag(kt, i);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < NK; ++i) {
            if (i < 2)
                sn[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kr[i % PF], qf[i >> 1], f32x16{}, 0, 0, 0);
            else
                sn[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kr[i % PF], qf[i >> 1], sn[i & 1], 0, 0, 0);
            if (i + PF < NK) kr[i % PF] = kfrag(kt, i + PF);
            if (i % STRIDE == STRIDE - 1) {
                const int e = 2 * (i / STRIDE);
                const float x0 = __builtin_amdgcn_exp2f(fmaf(sc[0][e], c, nm0));
                const float x1 = __builtin_amdgcn_exp2f(fmaf(sc[0][e + 1], c, nm0));
                put_pair(p[e >> 3], e & 7, x0, x1, racc0);
                acc0 += x0;
                acc1 += x1;
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        float a1 = acc0 + acc1;
        // keep this half of the softmax in this phase: without a use here the
        // compiler sinks it past the branch below, next to the P V products
        __asm__ volatile("" : : "v"(p[0]), "v"(p[1]), "v"(a1), "v"(racc0));
        upd = __builtin_amdgcn_ballot_w64(!(a1 <= kSpecLimit) && a1 == a1) != 0;
        if (upd) {
            float m0 = -INFINITY, m1 = -INFINITY;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                m0 = fmaxf(m0, sc[0][e]);
                m1 = fmaxf(m1, sc[1][e]);
            }
            const float mnew = fmaxf(mref, pair_max(fmaxf(m0, m1)) * c);
            alpha = __builtin_amdgcn_exp2f(mref - mnew);
            mref = mnew;
            lsum *= alpha;
            rsum *= alpha;
            acc0 = acc1 = racc0 = 0.f;
#pragma unroll
            for (int e = 0; e < 16; e += 2) {
                const float x0 = __builtin_amdgcn_exp2f(fmaf(sc[0][e], c, -mnew));
                const float x1 = __builtin_amdgcn_exp2f(fmaf(sc[0][e + 1], c, -mnew));
                put_pair(p[e >> 3], e & 7, x0, x1, racc0);
                acc0 += x0;
                acc1 += x1;
            }
            a1 = acc0 + acc1;
        }
        acc0 = a1;
        acc1 = acc2 = racc1 = 0.f;
        nm = -mref;
    };

    // Prologue: kAhead tiles in flight (paired launches: K of the first two
    // tiles and V of the first); S of the first tile.
    int st = kt0 % (G::LDS / G::STAGE);  // stage of tile t
    if constexpr (PAIRED) {
        const uint32_t s0 = lds0 + st * G::STAGE;
        issue_one(kt0, s0, std::false_type{});
        if (kt1 - kt0 > 1) {
            issue_one(kt0 + 1, lds0 + (st ^ 1) * G::STAGE, std::false_type{});
            issue_one(kt0, s0 + G::TILE, std::true_type{});
            wait_vmcnt<2 * LOADS>();
        } else {
            issue_one(kt0, s0 + G::TILE, std::true_type{});
            wait_vmcnt<LOADS>();
        }
    } else {
        int sl = st;
#pragma unroll
        for (int i = 0; i < kAhead; ++i) {
            issue_next(sl);
            sl = next_stage(sl);
        }
        wait_vmcnt<(kAhead - 1) * PER_TILE>();
    }
    __syncthreads();
    qk(st, scur);

    // One tile of the pipeline on the S buffers sc (S_t) and sn (S_{t+1}).
    // HAS_NEXT: tile t+1 exists (S_{t+1} is computed here, beside the softmax
    // of S_t); MASK: tile t is the ragged last one.
    auto step = [&](int t, f32x16 (&sc)[2], f32x16 (&sn)[2], auto has_next, auto mask) {
        constexpr bool HAS_NEXT = decltype(has_next)::value;
        constexpr bool MASK = decltype(mask)::value;
        const int st1 = next_stage(st);  // stage of tile t+1
        // ---- phase X
        if constexpr (PAIRED) {
            // K of tile t+1 and V of tile t were copied during the previous
            // step (or the prologue); K of tile t+2 goes into the stage whose
            // K (tile t) the previous step's Q K^T consumed, V of tile t+1
            // into the stage whose V (tile t-1) its P V consumed.
            wait_vmcnt<0>();  // this wave's copies landed
            __syncthreads();  // ... and every other wave's, which is past the previous step
            if (t + 2 < kt1) issue_one(t + 2, lds0 + st * G::STAGE, std::false_type{});
            if (t + 1 < kt1) issue_one(t + 1, lds0 + st1 * G::STAGE + G::TILE, std::true_type{});
            if constexpr (HAS_NEXT)
                qk_softmax(st1, sc, sn);
            else
                softmax_block<MASK>(sc, c, mref, lsum, rsum, p, alpha, upd, t * kBlockN, Skv);
        } else if constexpr (HAS_NEXT) {
            // tiles up to t + kAhead - 1 have been issued; tile t+1 must have
            // landed, so at most kAhead - 2 tiles' copies may still be in flight
            wait_vmcnt<(kAhead - 2) * PER_TILE>();  // this wave's copies of tile t+1 landed
            __syncthreads();                         // ... and every other wave's
            issue_next(next_stage(st1));             // tile t+kAhead, into the stage tile t-1 used
            qk_softmax(st1, sc, sn);
        } else {
            softmax_block<MASK>(sc, c, mref, lsum, rsum, p, alpha, upd, t * kBlockN, Skv);
        }
        // ---- O rescale (rare), outside the MFMA streams
        if (upd) {
#pragma unroll
            for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
        }
        // ---- phase Y, at normal priority (phase X raised it)
        __builtin_amdgcn_s_setprio(0);
        if constexpr (HAS_NEXT)
            pv(st, std::true_type{}, sc);
        else
            pv(st, std::false_type{}, sc);
        st = st1;
    };

    using T_ = std::true_type;
    using F_ = std::false_type;
    // Two tiles per trip with the roles of the S buffers swapped in the
    // second, so that S_{t+1} is never copied.
    int t = kt0;
    for (; t + 2 < kt1; t += 2) {
        step(t, scur, snext, T_{}, F_{});
        step(t + 1, snext, scur, T_{}, F_{});
    }
    if (t + 1 < kt1) {  // two tiles left: one more step with a successor
        step(t, scur, snext, T_{}, F_{});
        scur[0] = snext[0];
        scur[1] = snext[1];
        ++t;
    }
    if (ragged_end)
        step(t, scur, snext, F_{}, T_{});
    else
        step(t, scur, snext, F_{}, F_{});
    wait_vmcnt<0>();  // the clamped trailing copies must land before the workgroup exits
    if (DUAL && n_pass == 2 && ps == 0) {
        // park the first context's normalized O in LDS (bf16) and its LSE
        const float lt1 = pair_sum(lsum);
        lse1 = (mref + __log2f(lt1)) * kLn2;
        const float inv = 1.0f / pair_sum(rsum);
        lds_char *park = (lds_char *)smem + G::LDS + threadIdx.x * 16;
#pragma unroll
        for (int j = 0; j < DB * 2; ++j) {  // chunk j: values 8j .. 8j+7 of (db, gq, e) order
            bf16x8 w;
#pragma unroll
            for (int e = 0; e < 8; ++e) w[e] = (__bf16)(oacc[j / 2][(j % 2) * 8 + e] * inv);
            *(lds_bf16x8 *)(park + j * THREADS * 16) = w;
        }
        __syncthreads();  // every wave is done with the ring before the second pass refills it
    }
    }

    if (slot >= 0 || OUT_F32 || ACC) {
        store_row<D, OUT_F32, ACC, BM>(a, pl, oacc, lsum, rsum, mref, b, h, qi, qrow, slot);
        return;
    }
    // whole tile, bf16 output: final values in oacc, then full-row stores
    const float lt = pair_sum(lsum);
    const float inv = 1.0f / pair_sum(rsum);
    const float lse_last = (mref + __log2f(lt)) * kLn2;
    if constexpr (DUAL) {
        if (hi == 0 && qi < Sq) {
            const int64_t li = ((int64_t)b * a.H + h) * a.Sq + qi;
            if (a.lse != nullptr) a.lse[li] = lse1;
            if (a.lse2 != nullptr) a.lse2[li] = lse_last;
        }
        // the sum, staged in the (now idle) ring and written as full rows
        const lds_char *park = (const lds_char *)smem + G::LDS + threadIdx.x * 16;
        __syncthreads();  // every wave is done with the ring
        lds_char *stg = (lds_char *)smem + wave * 32 * D * 2;
#pragma unroll
        for (int j = 0; j < DB * 2; ++j) {
            const bf16x8 o1 = *(const lds_bf16x8 *)(park + j * THREADS * 16);
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int db = j / 2, gq = (j % 2) * 2 + half;
                bf16x4 w;
#pragma unroll
                for (int e = 0; e < 4; ++e) w[e] = (__bf16)(oacc[db][gq * 4 + e] * inv + (float)o1[half * 4 + e]);
                stage_out4<D>(stg, col, db * 32 + gq * 8 + hi * 4, w);
            }
        }
        store_staged_rows<D>(a, stg, lane, b, h, qt * BM + wave * 32);
        return;
    } else {
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] *= inv;
    }
    if (a.lse != nullptr && hi == 0 && qi < Sq) a.lse[((int64_t)b * a.H + h) * a.Sq + qi] = lse_last;
    __syncthreads();  // every wave is done with the ring, which now stages the output
    store_tile_bf16<D>(a, (lds_char *)smem + wave * 32 * D * 2, oacc, lane, b, h, qt * BM + wave * 32);
}

// Ping-pong schedule of the same computation (launches with many key tiles).
// Waves w and w+4 share a SIMD; group 0 (waves 0-3) and group 1 (waves 4-7)
// alternate, in opposite phases, between
//   M(u): a straight MFMA stream: O^T += V^T P^T of tile u-1, then
//         S^T = K Q^T of tile u, operand fragments read PF MFMAs ahead;
//   V(u): the weights of tile u (vector instructions only),
// with a workgroup barrier between phases, so that on every SIMD one wave
// streams MFMAs while the other computes weights.  (A wave that interleaves
// its own weights with its MFMAs keeps the matrix pipe about half busy; two
// waves in opposite phases keep it about 80 % busy in a probe of the same
// instruction mix.)  Tiles go through a 4-stage LDS ring: each wave copies its
// share of tile u+2 right after M(u), into the stage of tile u-2.  A wave
// reads the first PF operand fragments of its next M phase (V fragments of a
// tile that landed a pair earlier) before the barrier that starts the phase,
// so their LDS latency passes while it waits there rather than before its
// first MFMA.
//
// The products use v_mfma_f32_16x16x32_bf16 rather than the 32x32x16 form
// of the interleaved kernel: the same FLOPs at the same issue rate, but half
// the accumulator bytes read and written per FLOP.  The chip runs this load
// at its power limit, and a pure MFMA stream of the 16x16x32 form holds a
// ~15 % higher shader clock than one of the 32x32x16 form.  Layout: a lane
// (group g = lane/16, column x = lane%16) holds queries x and 16 + x of the
// wave's 32, each with keys 4g .. 4g+3 of every 16-key block of S^T; row
// sums and maxima are in-lane over those keys plus an exchange across the
// four lane groups (only at the end, and when the reference is raised).
//
// Weights use the speculative reference of the interleaved kernel, checked
// once per tile (a lane's 16 weights of one query summing to more than
// kSpecLimit), and the same running sum.
template <int D, bool OUT_F32, bool ACC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_fwd_pingpong_kernel(AttnArgs a_in, AttnPlan pl)
{
    using G = Geo<D, kStagesPP>;
    constexpr int NCH = G::NCH, LOADS = G::LOADS;
    constexpr int KS = D / 32;           // 32-dim k-steps of Q K^T
    constexpr int DB = D / 16;           // 16-dim blocks of O^T
    constexpr int BM = kWaves * 32;
    constexpr int PER_TILE = 2 * LOADS;  // copies per thread per tile (K and V)
    static_assert(kStagesPP == 4, "tile u+2 is copied into the stage of tile u-2");
    static_assert(kBlockN == 64, "four 16-key blocks per tile");

    __shared__ __attribute__((aligned(1024))) char smem[G::LDS];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const int grp = wave >> 2;
    const int g = lane >> 4;   // lane group: 4 keys of each 16-key block, 4 dims of each 16-dim block
    const int x = lane & 15;   // query column within a 16-query block

    WorkItem wi = work_item(pl, blockIdx.x);
    int n_kt;
    const AttnArgs a = chunk_view(a_in, pl, wi, n_kt);
    const int tile = wi.tile, kt0 = wi.kt0, kt1 = wi.kt1, slot = wi.slot;
    const int qt = tile % pl.n_qtiles;
    const int bh = tile / pl.n_qtiles;
    const int h = bh % a.H;
    const int b = bh / a.H;
    // this lane's two queries: row wave*32 + qb*16 + x of the tile, qb = 0, 1
    const int qrow0 = wave * 32 + x;
    const int qi0 = qt * BM + qrow0;

    const uint16_t *qp = static_cast<const uint16_t *>(a.q) + b * a.q_sb + h * a.q_sh;
    const uint16_t *kp = static_cast<const uint16_t *>(a.k) + b * a.k_sb + h * a.k_sh;
    const uint16_t *vp = static_cast<const uint16_t *>(a.v) + b * a.v_sb + h * a.v_sh;
    const int Skv = a.Skv;
    const int T = kt1 - kt0;  // key tiles of this work item, >= 1
    const bool ragged_end = kt1 == n_kt && (Skv % kBlockN) != 0;

    // Q^T operand fragments (B of S^T = K Q^T): query block qb, dims
    // 32*ks + 8*g .. +7 of query qb*16 + x.
    bf16x8 qf[2][KS];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int qi = qi0 + qb * 16;
            if (qi < a.Sq)
                qf[qb][ks] = *reinterpret_cast<const bf16x8 *>(qp + (int64_t)qi * a.q_ss + ks * 32 + g * 8);
            else
                qf[qb][ks] = bf16x8{};
        }

    // HBM -> LDS copies: tiles in order kt0, kt0+1, ... into ring stages 0,
    // 1, 2, ...; every tile is PER_TILE copies per thread, in two halves, K
    // (LOADS copies) and V (LOADS copies), issued at different points of the
    // schedule; advance_copy moves on to the next tile once both are out.
    // Past the last tile the copies repeat it into stages that are not read
    // again (every tile issues PER_TILE copies, so the vmcnt waits count
    // tiles); the schedule's tail asks for none.
    using T_ = std::true_type;
    using F_ = std::false_type;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char *)smem;
    uint32_t kofs[LOADS], vofs[LOADS];
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
        const int slot16 = (wave * LOADS + j) * 64 + lane;
        const int row = slot16 / NCH, phys = slot16 % NCH;
        kofs[j] = (uint32_t)((row * a.k_ss + k_slot<NCH>(row, phys) * 8) * 2);
        vofs[j] = (uint32_t)((row * a.v_ss + vp_slot<NCH>(row, phys) * 8) * 2);
    }
    const int64_t k_step = (int64_t)kBlockN * a.k_ss, v_step = (int64_t)kBlockN * a.v_ss;
    const int last_full = Skv / kBlockN - 1;  // last tile with kBlockN keys
    int tl_copy = kt0;
    int st_copy = 0;
    const uint16_t *kb_copy = kp + kt0 * k_step;
    const uint16_t *vb_copy = vp + kt0 * v_step;
    auto issue_half = [&](auto is_v) __attribute__((always_inline)) {
        constexpr bool V = decltype(is_v)::value;
        const uint32_t dst = lds0 + st_copy * G::STAGE + (V ? G::TILE : 0);
        if (a.kv_off32 && tl_copy <= last_full) {
            const uint32_t blk = __builtin_amdgcn_readfirstlane(wave * LOADS * 1024);
            lds_dma16_group<LOADS>(uniform_ptr(V ? vb_copy : kb_copy), V ? vofs : kofs,
                                   __builtin_amdgcn_readfirstlane(dst) + blk);
        } else {
            const int key0 = tl_copy * kBlockN;
            const int last = Skv - 1 - key0;
#pragma unroll
            for (int j = 0; j < LOADS; ++j) {
                const int blk = wave * LOADS + j;
                const int slot16 = blk * 64 + lane;
                const int row = slot16 / NCH, phys = slot16 % NCH;
                const int64_t key = key0 + min(row, last);
                if (V)
                    lds_dma16(vp + key * a.v_ss + vp_slot<NCH>(row, phys) * 8, dst + blk * 1024);
                else
                    lds_dma16(kp + key * a.k_ss + k_slot<NCH>(row, phys) * 8, dst + blk * 1024);
            }
        }
    };
    auto advance_copy = [&]() __attribute__((always_inline)) {
        st_copy = st_copy == kStagesPP - 1 ? 0 : st_copy + 1;
        if (tl_copy < kt1 - 1) {
            ++tl_copy;
            kb_copy += k_step;
            vb_copy += v_step;
        }
    };

    // Per-lane LDS byte offsets of the MFMA operand fragments (stage 0).
    // K fragment (kb, ks): key kb*16 + x, dims 32*ks + 8*g .. +7 (one 16-byte
    // chunk; the key block is an immediate offset, the swizzle depends on
    // the key only through x).  V^T fragment (db, ks): dim db*16 + x of keys
    // 32*ks + 4*g .. +3 and 32*ks + 16 + 4*g .. +3, two transposing 8-byte
    // reads in which lane x of each 16-lane group supplies key 4*g + x/4,
    // dims db*16 + 4*(x%4) .. +3 and receives the column of dim db*16 + x.
    // That key order is the one the S^T accumulators give the P operand.
    int koff[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) koff[ks] = (x * D + k_slot<NCH>(x, ks * 4 + g) * 8) * 2;
    int voff[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        const int row = 4 * g + (x >> 2);
        const int dcol = db * 16 + 4 * (x & 3);
        voff[db] = G::TILE + (row * D + vp_slot<NCH>(row, dcol >> 3) * 8 + (dcol & 7)) * 2;
    }
    constexpr int NK = 4 * KS;  // K fragments per tile (each feeds two MFMAs)
    constexpr int NV = 2 * DB;  // V^T fragments per tile (each feeds two MFMAs)
    constexpr int PF = 4;       // fragments read ahead of their MFMAs
    static_assert(NK >= PF && NV >= PF, "schedule assumes d >= 64");
    auto kfrag = [&](const lds_char *kt, int i) -> bf16x8 {  // i = ks*4 + kb
        return *(const lds_bf16x8 *)(kt + koff[i >> 2] + (i & 3) * 16 * D * 2);
    };
    auto vfrag = [&](const lds_char *vt, int i) -> bf16x8 {  // i = ks*DB + db
        const int ks = i / DB, db = i % DB;
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(vt + voff[db] + ks * 32 * D * 2));
        const bf16x4 up =
            __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(vt + voff[db] + (ks * 32 + 16) * D * 2));
        return bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
    };
    auto stage_ptr = [&](int st) { return (const lds_char *)(smem + st * G::STAGE); };

    // Accumulators: oacc[db][qb] = O^T dims db*16 + 4*g .. +3 of query
    // qb*16 + x; s[kb][qb] = S^T keys kb*16 + 4*g .. +3 of that query.
    f32x4 oacc[DB][2];
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db][0] = oacc[db][1] = f32x4{};
    f32x4 s[4][2];
    bf16x8 p[2][2];  // P^T operands: 32-key step ks, query block qb
    const float c = a.scale * kLog2e;
    // per query block: reference, sum of the unrounded weights (LSE) and of
    // the bf16-rounded weights (the normalizer of O)
    float mref[2] = {-INFINITY, -INFINITY}, lsum[2] = {0.f, 0.f}, rsum[2] = {0.f, 0.f};

    // First PF operand fragments of an M phase (see mphase), read ahead of it.
    bf16x8 r[PF];
    auto mprefetch = [&](int stq, int stv, auto do_pv) __attribute__((always_inline)) {
        constexpr int N0 = decltype(do_pv)::value ? NV : 0;
        const lds_char *vt = stage_ptr(stv);
        const lds_char *kt = stage_ptr(stq);
#pragma unroll
        for (int j = 0; j < PF; ++j) r[j] = j < N0 ? vfrag(vt, j) : kfrag(kt, j - N0);
    };

    // M phase: PV of the tile in stage stv (weights p), then QK of the tile in
    // stage stq (into s); every fragment feeds the MFMAs of both query blocks;
    // the order is pinned so the fragment reads stay PF fragments ahead.  The
    // first PF fragments are in r (mprefetch, same stages).
    auto mphase = [&](int stq, int stv, auto do_pv, auto do_qk) __attribute__((always_inline)) {
        constexpr bool PV = decltype(do_pv)::value, QK = decltype(do_qk)::value;
        constexpr int N0 = PV ? NV : 0;
        constexpr int N = N0 + (QK ? NK : 0);
        const lds_char *vt = stage_ptr(stv);
        const lds_char *kt = stage_ptr(stq);
        auto frag = [&](int j) -> bf16x8 { return j < N0 ? vfrag(vt, j) : kfrag(kt, j - N0); };
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < N; ++j) {
            if (j < N0) {
                const int ks = j / DB, db = j % DB;
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
                    oacc[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(r[j % PF], p[ks][qb], oacc[db][qb], 0, 0, 0);
            } else {
                const int i = j - N0, ks = i >> 2, kb = i & 3;
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
                    s[kb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(r[j % PF], qf[qb][ks],
                                                                       ks == 0 ? f32x4{} : s[kb][qb], 0, 0, 0);
            }
            if (j + PF < N) r[j % PF] = frag(j + PF);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // V phase: weights of the tile whose first key is key0, from s into p,
    // against the running references; if some lane's 16 weights of one of
    // its queries sum to more than kSpecLimit (or are not finite: the first
    // tile), the references are raised to the exact running maxima (over the
    // four lanes that hold a query's keys), O and the sums are rescaled and
    // the weights recomputed.  MASK: keys at or past Skv get weight exactly 0.
    auto vphase = [&](int key0, auto mask) __attribute__((always_inline)) {
        constexpr bool MASK = decltype(mask)::value;
        auto valid = [&](int kb, int i) { return key0 + kb * 16 + g * 4 + i < Skv; };
        float e_sum[2], r_sum[2];
        auto weights = [&]() __attribute__((always_inline)) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                const float nm = -mref[qb];
                // -0 starts the sums (0 + x is not foldable: it turns -0 into +0)
                float a0 = -0.f, a1 = -0.f, ar = -0.f;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int i = 0; i < 4; i += 2) {
                        float e0 = __builtin_amdgcn_exp2f(fmaf(s[kb][qb][i], c, nm));
                        float e1 = __builtin_amdgcn_exp2f(fmaf(s[kb][qb][i + 1], c, nm));
                        if (MASK) {
                            e0 = valid(kb, i) ? e0 : 0.f;
                            e1 = valid(kb, i + 1) ? e1 : 0.f;
                        }
                        put_pair(p[kb >> 1][qb], (kb & 1) * 4 + i, e0, e1, ar);
                        a0 += e0;
                        a1 += e1;
                    }
                e_sum[qb] = a0 + a1;
                r_sum[qb] = ar;
            }
        };
        weights();
        const bool over = !(e_sum[0] <= kSpecLimit) || !(e_sum[1] <= kSpecLimit);
        if (__builtin_amdgcn_ballot_w64(over) != 0) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                float m0 = -INFINITY, m1 = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 4; kb += 2)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        m0 = fmaxf(m0, (!MASK || valid(kb, i)) ? s[kb][qb][i] : -INFINITY);
                        m1 = fmaxf(m1, (!MASK || valid(kb + 1, i)) ? s[kb + 1][qb][i] : -INFINITY);
                    }
                const float mnew = fmaxf(mref[qb], quad_max(fmaxf(m0, m1)) * c);
                const float alpha = __builtin_amdgcn_exp2f(mref[qb] - mnew);
                mref[qb] = mnew;
#pragma unroll
                for (int db = 0; db < DB; ++db) oacc[db][qb] *= alpha;
                lsum[qb] *= alpha;
                rsum[qb] *= alpha;
            }
            weights();
        }
        lsum[0] += e_sum[0];
        lsum[1] += e_sum[1];
        rsum[0] += r_sum[0];
        rsum[1] += r_sum[1];
    };

    auto st = [](int u) { return u & (kStagesPP - 1); };  // ring stage of the work item's tile u
    auto key0 = [&](int u) { return (kt0 + u) * kBlockN; };
    auto vlast = [&](int u) __attribute__((always_inline)) {  // V phase of the last (possibly ragged) tile
        if (ragged_end)
            vphase(key0(u), T_{});
        else
            vphase(key0(u), F_{});
    };
    // Barrier between phases.  Nothing moves across it (the compiler would
    // otherwise hoist a V phase's register-only work above it, into the same
    // interval as the wave's own M phase), and the score and weight registers
    // are pinned to their side of it.
    auto phase_barrier = [&]() __attribute__((always_inline)) {
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
        __asm__ volatile("" : "+v"(s[0][0]), "+v"(s[0][1]), "+v"(s[1][0]), "+v"(s[1][1]), "+v"(s[2][0]),
                         "+v"(s[2][1]), "+v"(s[3][0]), "+v"(s[3][1]));
        __asm__ volatile("" : "+v"(p[0][0]), "+v"(p[0][1]), "+v"(p[1][0]), "+v"(p[1][1]));
        __builtin_amdgcn_sched_barrier(0);
    };
    // The barriers after a wave's last M phase: no score or weight register
    // is live any more, so nothing is pinned.
    auto end_barrier = [&]() __attribute__((always_inline)) {
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
    };

    // Prologue: tiles 0 and 1 in flight, tile 0 landed.
    issue_half(F_{});
    issue_half(T_{});
    advance_copy();
    issue_half(F_{});
    issue_half(T_{});
    advance_copy();
    wait_vmcnt<PER_TILE>();
    __syncthreads();

    // Interval pairs u = 0..T, two barriers each (the same count in both
    // groups).  Group 0 runs M(u) | V(u), group 1 runs V(u-1) | M(u).  Each
    // wave copies its part of tile u+2 in pair u (stage of tile u-2, last
    // read by PV(u-2) in pair u-1): the K half right after its M(u), the V
    // half at the start of its V interval of pair u (so that the two halves'
    // issue, which the CU's address unit serializes, is shared between the M
    // and the V interval).  Before the barrier that ends pair u, a wave waits
    // for its copies of tile u+1, which M(u+1) reads after that barrier.  The
    // fragments an M phase starts with are read before the barrier ahead of
    // it: V fragments of its tile u-1, which landed a pair earlier and is not
    // overwritten before pair u+1.  The M phase runs at raised priority.
    if (grp == 0) {
        // (distinct markers at the head of the two schedules: their common
        // first reads are not hoisted above the branch, which would keep
        // them live through the other group's whole schedule)
        __asm__ volatile("; group 0 schedule");
        mprefetch(st(0), st(0), F_{});
        __builtin_amdgcn_s_setprio(1);
        mphase(st(0), st(0), F_{}, T_{});
        __builtin_amdgcn_s_setprio(0);
        issue_half(F_{});
        phase_barrier();
        issue_half(T_{});
        if (T == 1)
            vlast(0);
        else
            vphase(key0(0), F_{});
        advance_copy();
        wait_vmcnt<PER_TILE>();
        mprefetch(st(1), st(0), T_{});
        phase_barrier();
        for (int u = 1; u < T - 1; ++u) {
            __builtin_amdgcn_s_setprio(1);
            mphase(st(u), st(u - 1), T_{}, T_{});
            __builtin_amdgcn_s_setprio(0);
            issue_half(F_{});
            phase_barrier();
            issue_half(T_{});
            vphase(key0(u), F_{});
            advance_copy();
            wait_vmcnt<PER_TILE>();
            mprefetch(st(u + 1), st(u), T_{});
            phase_barrier();
        }
        if (T >= 2) {
            __builtin_amdgcn_s_setprio(1);
            mphase(st(T - 1), st(T - 2), T_{}, T_{});
            __builtin_amdgcn_s_setprio(0);
            phase_barrier();
            vlast(T - 1);
            wait_vmcnt<0>();  // (left in flight: the repeat copy of the pair before)
            mprefetch(st(T), st(T - 1), T_{});
            phase_barrier();
        }
        __builtin_amdgcn_s_setprio(1);
        __asm__ volatile("; last M phase, group 0");  // keeps the two groups' last M phases apart
        mphase(st(T), st(T - 1), T_{}, F_{});
        __builtin_amdgcn_s_setprio(0);
        end_barrier();
        end_barrier();
    } else {
        // (the V half of a tile goes out a whole interval before its K half)
        __asm__ volatile("; group 1 schedule");
        mprefetch(st(0), st(0), F_{});
        issue_half(T_{});
        phase_barrier();
        __builtin_amdgcn_s_setprio(1);
        mphase(st(0), st(0), F_{}, T_{});
        __builtin_amdgcn_s_setprio(0);
        issue_half(F_{});
        advance_copy();
        wait_vmcnt<PER_TILE>();
        phase_barrier();
        for (int u = 1; u < T; ++u) {
            issue_half(T_{});
            vphase(key0(u - 1), F_{});
            mprefetch(st(u), st(u - 1), T_{});
            phase_barrier();
            __builtin_amdgcn_s_setprio(1);
            mphase(st(u), st(u - 1), T_{}, T_{});
            __builtin_amdgcn_s_setprio(0);
            issue_half(F_{});
            advance_copy();
            wait_vmcnt<PER_TILE>();
            phase_barrier();
        }
        vlast(T - 1);
        mprefetch(st(T), st(T - 1), T_{});
        phase_barrier();
        __builtin_amdgcn_s_setprio(1);
        __asm__ volatile("; last M phase, group 1");
        mphase(st(T), st(T - 1), T_{}, F_{});
        __builtin_amdgcn_s_setprio(0);
        end_barrier();
    }
    wait_vmcnt<0>();  // the repeat copies past the last tile must land before the workgroup exits

    // The epilogue's lane indices come from a fresh copy of the thread index
    // (opaque to the compiler), so that no index or address computed before
    // the key loop has to stay live across it.
    int tid_e = (int)threadIdx.x;
    __asm__ volatile("" : "+v"(tid_e));
    const int lane_e = tid_e & 63, x_e = lane_e & 15, g_e = lane_e >> 4;
    const int qrow0_e = wave * 32 + x_e, qi0_e = qt * BM + qrow0_e;

    // Epilogue: per query, l and l_r = the sums of the four lanes' partial
    // sums; O = O^T / l_r, LSE = ln2 * (m_ref + log2 l); a split tile's key
    // range writes its normalized partial to the workspace instead.
    {
        if (slot < 0) {  // whole tile: staged full-row stores (f32 rows take the whole 128 KB ring)
            float wr[2] = {0.f, 0.f};  // ring accumulate: the running output's weight per query block
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                const float lt = quad_sum(lsum[qb]);
                float sc = 1.0f / quad_sum(rsum[qb]);
                float lse_val = (mref[qb] + __log2f(lt)) * kLn2;
                const int qi = qi0_e + qb * 16;
                if constexpr (ACC) {
                    const int qc = min(qi, a.Sq - 1);
                    const RunMerge m = run_merge(a.run_lse[((int64_t)b * a.H + h) * a.Sq + qc], lse_val);
                    lse_val = m.lse;
                    sc *= m.wc;
                    wr[qb] = m.run ? m.wr : -1.f;
                }
                if (a.lse != nullptr && g_e == 0 && qi < a.Sq) a.lse[((int64_t)b * a.H + h) * a.Sq + qi] = lse_val;
#pragma unroll
                for (int db = 0; db < DB; ++db) oacc[db][qb] *= sc;
            }
            __syncthreads();  // every wave is done with the ring, which now stages the output
            lds_char *stg = (lds_char *)smem + wave * 32 * D * (OUT_F32 ? 4 : 2);
            static_assert(!OUT_F32 || kWaves * 32 * D * 4 <= G::LDS, "f32 staging fits the ring");
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    if constexpr (OUT_F32) {
                        stage_out4_f32<D>(stg, qb * 16 + x_e, db * 16 + g_e * 4, oacc[db][qb]);
                    } else {
                        bf16x4 w;
#pragma unroll
                        for (int e = 0; e < 4; ++e) w[e] = (__bf16)oacc[db][qb][e];
                        stage_out4<D>(stg, qb * 16 + x_e, db * 16 + g_e * 4, w);
                    }
                }
            if constexpr (ACC)
                store_staged_rows_run<D, OUT_F32>(a, stg, lane_e, b, h, qt * BM + wave * 32, wr);
            else if constexpr (OUT_F32)
                store_staged_rows_f32<D>(a, stg, lane_e, b, h, qt * BM + wave * 32);
            else
                store_staged_rows<D>(a, stg, lane_e, b, h, qt * BM + wave * 32);
            return;
        }
    }
    // A split tile's key range: its normalized partial (f32) to the
    // workspace, staged in the ring and written as full rows like a whole
    // tile's f32 output, and its LSE.
    __syncthreads();  // every wave is done with the ring
    lds_char *stg = (lds_char *)smem + wave * 32 * D * 4;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float lt = quad_sum(lsum[qb]);
        const float inv = 1.0f / quad_sum(rsum[qb]);
        const int qrow = qrow0_e + qb * 16, qi = qi0_e + qb * 16;
        if (g_e == 0 && qi < a.Sq) pl.ws_lse[(int64_t)slot * BM + qrow] = (mref[qb] + __log2f(lt)) * kLn2;
#pragma unroll
        for (int db = 0; db < DB; ++db) stage_out4_f32<D>(stg, qb * 16 + x_e, db * 16 + g_e * 4, oacc[db][qb] * inv);
    }
    constexpr int CPR = D / 4;     // 16-byte chunks per row
    constexpr int RPI = 64 / CPR;  // rows per store instruction
#pragma unroll
    for (int it = 0; it < 32 / RPI; ++it) {
        const int r = it * RPI + lane_e / CPR, c = lane_e % CPR;
        const f32x4 w = *(const __attribute__((address_space(3))) f32x4 *)(stg + r * D * 4 + (c ^ (r & (CPR - 1))) * 16);
        if (qt * BM + wave * 32 + r < a.Sq)
            *reinterpret_cast<f32x4 *>(pl.ws_o + ((int64_t)slot * BM + wave * 32 + r) * D + c * 4) = w;
    }
}

// Log-sum-exp combination of the key-range partials of each split tile
// (the same identity as the chunk merge): one thread per 4 dims of one row.
// The partials are visited in batches of FB whose LSE and O loads are all
// issued before any of them is used, combined online (running max, sum and
// weighted O), so the loop is not a chain of dependent memory accesses.
// Key-range slices of the fixup: the waves of a workgroup take the same 64
// (row, 4-dim) pairs, wave i merging key ranges i, i + slices, ...; the
// first wave combines the slices' results (read through LDS) and stores.
// A lane then waits for one batch of (at most 8) partial loads instead of
// several in turn.  Tiles split into fewer than 9 ranges per context take
// one slice: there the extra waves and the combine cost more than they save
// (measured: 8 + 5 ranges 4.4 -> 5.3 us, 2 ranges 12.2 -> 27.7 us with four).
// A workgroup holds 256 / (64 * slices) groups of 64 pairs (one for three
// slices).
constexpr int kFixSlices = 4;  // at most
__host__ __device__ inline int fix_slices(const AttnPlan &pl)
{
    const int most = pl.seg > pl.seg2 ? pl.seg : pl.seg2;
    const int s = (most + 7) / 8;
    return s < 1 ? 1 : (s > kFixSlices ? kFixSlices : s);
}
__host__ __device__ inline int fix_groups(int slices) { return kFixSlices / slices; }

template <bool OUT_F32>
__global__ __launch_bounds__(64 * kFixSlices) void split_fixup_kernel(AttnArgs a_in, AttnPlan pl)
{
    const int BM = pl.bm;
    constexpr int FB = 8;
    const int n_sl = fix_slices(pl), n_grp = fix_groups(n_sl);  // blockDim.x == 64 * n_sl * n_grp
    __shared__ float red[2][kFixSlices - 1][6][64];
    const int per_row = a_in.D / 4;
    const int lane = threadIdx.x & 63;
    const int slice = (threadIdx.x >> 6) % n_sl, grp = (threadIdx.x >> 6) / n_sl;
    const int entry = grp * (n_sl - 1) + slice - 1;  // this wave's LDS entry (slice > 0): < kFixSlices - 1
    const int64_t rows = (int64_t)(pl.n_tiles - pl.n_dp) * BM;
    const int64_t pair = ((int64_t)blockIdx.x * n_grp + grp) * 64 + lane;
    // lanes past the last row merge the last one again (in bounds) and store nothing
    const int64_t row = min(pair / per_row, rows - 1);
    const int d = (int)(pair % per_row) * 4;
    const int j = (int)(row / BM), r = (int)(row % BM);
    int tile = pl.n_dp + j;
    const AttnArgs a = chunk_of(a_in, pl, tile);
    const int qt = tile % pl.n_qtiles;
    const int bh = tile / pl.n_qtiles;
    const int h = bh % a.H, b = bh / a.H;
    const int qi = qt * BM + r;
    const bool live = pair / per_row < rows && qi < a.Sq;
    // LSE merge of this slice's units among n from u0 on: (max m, sum s,
    // weighted O acc); m = -inf, s = 0 and acc = 0 for a slice without units
    auto merge_units = [&](int64_t u0, int n, float &m, float &s, f32x4 &acc) {
        m = -INFINITY;
        s = 0.f;
        acc = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int c0 = slice; c0 < n; c0 += FB * n_sl) {
            float l[FB];
            f32x4 o[FB];
#pragma unroll
            for (int k = 0; k < FB; ++k) {
                const int c = c0 + k * n_sl;  // wave-uniform
                if (c < n) {
                    const int64_t u = u0 + c;
                    l[k] = pl.ws_lse[u * BM + r];
                    o[k] = *reinterpret_cast<const f32x4 *>(pl.ws_o + (u * BM + r) * a.D + d);
                } else {  // past this slice's last unit: weight 0, nothing loaded
                    l[k] = -INFINITY;
                    o[k] = f32x4{0.f, 0.f, 0.f, 0.f};
                }
            }
            float mb = m;
#pragma unroll
            for (int k = 0; k < FB; ++k) mb = fmaxf(mb, l[k]);
            // every key range holds at least one key and each batch starts
            // with a unit, so mb is finite
            const float sc = expf(m - mb);
            s *= sc;
            acc *= sc;
#pragma unroll
            for (int k = 0; k < FB; ++k) {
                const float w = expf(l[k] - mb);
                s += w;
                acc += w * o[k];
            }
            m = mb;
        }
    };
    // The slices' results combined on the first wave (buffer i of red);
    // slice 0 always holds unit 0, so the common maximum is finite.
    auto combine = [&](int i, float &m, float &s, f32x4 &acc) {
        if (n_sl == 1) return;
        if (slice > 0) {
            float *e = &red[i][entry][0][lane];
            e[0] = m;
            e[64] = s;
#pragma unroll
            for (int k = 0; k < 4; ++k) e[(2 + k) * 64] = acc[k];
        }
        __syncthreads();
        if (slice == 0) {
            float mx = m;
            const int e0 = grp * (n_sl - 1) - 1;  // entry of slice t: e0 + t
#pragma unroll
            for (int t = 1; t < kFixSlices; ++t)
                if (t < n_sl) mx = fmaxf(mx, red[i][e0 + t][0][lane]);
            const float w0 = expf(m - mx);
            s *= w0;
            acc *= w0;
#pragma unroll
            for (int t = 1; t < kFixSlices; ++t)
                if (t < n_sl) {
                    const float w = expf(red[i][e0 + t][0][lane] - mx);
                    s += w * red[i][e0 + t][1][lane];
#pragma unroll
                    for (int k = 0; k < 4; ++k) acc[k] += w * red[i][e0 + t][2 + k][lane];
                }
            m = mx;
        }
    };
    const int64_t u0 = (int64_t)j * (pl.seg + pl.seg2);
    float m, s;
    f32x4 acc;
    merge_units(u0, pl.seg, m, s, acc);
    combine(0, m, s, acc);
    float m2 = 0.f, s2 = 1.f;
    f32x4 acc2{};
    if (pl.seg2 > 0) {  // dual context: the second context's units, merged alike
        merge_units(u0 + pl.seg, pl.seg2, m2, s2, acc2);
        combine(1, m2, s2, acc2);
    }
    if (slice != 0 || !live) return;
    const float L = m + logf(s);
    char *orow = static_cast<char *>(a.o) +
                 ((int64_t)b * a.o_sb + (int64_t)qi * a.o_ss + (int64_t)h * a.o_sh) * (OUT_F32 ? 4 : 2);
    const int64_t li = ((int64_t)b * a.H + h) * a.Sq + qi;
    if (pl.seg2 > 0) {  // the two contexts' results summed
        put_out4<OUT_F32>(orow, RunMerge{1.f, 1.0f / s, L, true}, d, acc, acc2 * (1.0f / s2));
        if (d == 0) {
            if (a.lse != nullptr) a.lse[li] = L;
            if (a.lse2 != nullptr) a.lse2[li] = m2 + logf(s2);
        }
        return;
    }
    RunMerge w{0.f, 1.f, L, false};
    f32x4 run[1] = {};
    if (a.run_lse != nullptr) w = run_merge(load_run(a, b, h, qi, d, 0, run), L);
    w.wc *= 1.0f / s;
    put_out4<OUT_F32>(orow, w, d, acc, run[0]);
    if (a.lse != nullptr && d == 0) a.lse[li] = w.lse;
}

// Chooses the work plan by a cost model in units of one key-tile iteration
// of one workgroup: whole tiles cost n_kt + 1 (prologue and epilogue), a
// split unit costs its key range + 1.5 (the partial store), and the partials'
// write + read traffic is priced at 5 TB/s against ~1 us per iteration.
// n_cu counts workgroup slots: in paired launches (128-row tiles) two per
// CU.  In a paired launch that does not fill one round, tiles that get a CU
// of their own run at about 0.65 of the paired time, and a split adds the
// fixup launch (~2 iterations).  After full rounds the leftover tiles start
// only as the last round drains, so they cost a whole tile each, and the
// fixup runs back to back with the attention kernel (measured on the window
// cross-attention, 1032 tiles of 8 key tiles on 512 slots: 8 leftover
// tiles split into 64 one-tile ranges, 53.5 -> 52.5 us).
AttnPlan make_plan(int n_qtiles, int n_tiles, int n_kt, int n_cu, int D, int BM)
{
    const bool paired = BM != kWaves * 32;
    AttnPlan pl{};
    pl.bm = BM;
    pl.n_qtiles = n_qtiles;
    pl.n_tiles = n_tiles;
    pl.n_kt = n_kt;
    pl.n_dp = n_tiles;
    pl.seg = 1;
    pl.n_units = 0;
    const double whole = n_kt + 1.0;
    const int rounds = n_tiles / n_cu;
    const int rem = n_tiles - rounds * n_cu;
    const bool lone = paired && rounds == 0;  // an underfilled paired launch
    const double tail = rem == 0 ? 0.0 : (lone && rem <= n_cu / 2 ? 0.65 : 1.0) * whole;
    double best = rounds * whole + tail;
    if (rem == 0 || n_kt < 2) return pl;
    for (int seg = 2; seg <= n_kt && seg <= 256; ++seg) {
        const int64_t units = (int64_t)rem * seg;
        if (units > 0x7fffffff - (int64_t)n_tiles) break;
        const int64_t sk_rounds = (units + n_cu - 1) / n_cu;
        const int len = (n_kt + seg - 1) / seg;
        const double traffic = 2.0 * units * BM * (D + 1) * 4 / 5e12 / 1e-6;
        const double cost = rounds * whole + sk_rounds * (len + 1.5) + traffic + (lone ? 2.0 : 0.0);
        if (cost < best) {
            best = cost;
            pl.n_dp = rounds * n_cu;
            pl.seg = seg;
            pl.n_units = (int)units;
        }
    }
    return pl;
}

// Plan of a dual-context launch (key tiles n_kt of the first context, n_kt2
// of the second): whole tiles run both passes (cost n_kt + n_kt2 + 2); a
// split tile becomes seg ranges of the first context and seg2 of the second,
// seg : seg2 close to n_kt : n_kt2, with the same cost model as above.
AttnPlan make_plan_dual(int n_qtiles, int n_tiles, int n_kt, int n_kt2, int n_cu, int D)
{
    constexpr int BM = kWaves * 32;
    AttnPlan pl{};
    pl.bm = BM;
    pl.n_qtiles = n_qtiles;
    pl.n_tiles = n_tiles;
    pl.n_kt = n_kt;
    pl.n_kt2 = n_kt2;
    pl.n_dp = n_tiles;
    pl.seg = 1;
    pl.seg2 = 1;
    pl.n_units = 0;
    const double whole = n_kt + n_kt2 + 2.0;
    double best = (double)((n_tiles + n_cu - 1) / n_cu) * whole;
    const int rounds = n_tiles / n_cu;
    const int rem = n_tiles - rounds * n_cu;
    if (rem == 0) return pl;
    for (int tot = 2; tot <= n_kt + n_kt2 && tot <= 256; ++tot) {
        const int s1 = min(max((int)lround((double)tot * n_kt / (n_kt + n_kt2)), 1), min(n_kt, tot - 1));
        const int s2 = tot - s1;
        if (s2 < 1 || s2 > n_kt2) continue;
        const int64_t units = (int64_t)rem * tot;
        if (units > 0x7fffffff - (int64_t)n_tiles) break;
        const int64_t sk_rounds = (units + n_cu - 1) / n_cu;
        const int len = max((n_kt + s1 - 1) / s1, (n_kt2 + s2 - 1) / s2);
        const double traffic = 2.0 * units * BM * (D + 1) * 4 / 5e12 / 1e-6;
        const double cost = rounds * whole + sk_rounds * (len + 1.5) + traffic;
        if (cost < best) {
            best = cost;
            pl.n_dp = rounds * n_cu;
            pl.seg = s1;
            pl.seg2 = s2;
            pl.n_units = (int)units;
        }
    }
    return pl;
}

int cu_count()
{
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (dev >= 0 && dev < 64 && cached[dev].load() > 0) return cached[dev].load();
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    if (dev >= 0 && dev < 64) cached[dev].store(n);
    return n;
}

std::atomic<int64_t> g_pool_draws{0};

// Stream-ordered workspace for split-tile partials, from a per-device pool
// that keeps its memory (so steady-state calls do not go back to the driver).
// Used only by calls that are not given a workspace.
hipMemPool_t workspace_pool()
{
    static std::mutex mu;
    static hipMemPool_t pools[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    if (pools[dev] == nullptr) {
        hipMemPoolProps props{};
        props.allocType = hipMemAllocationTypePinned;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        hipMemPool_t p = nullptr;
        if (hipMemPoolCreate(&p, &props) != hipSuccess) return nullptr;
        uint64_t keep = UINT64_MAX;
        (void)hipMemPoolSetAttribute(p, hipMemPoolAttrReleaseThreshold, &keep);
        pools[dev] = p;
    }
    return pools[dev];
}

// REGENVC_ATTN_SCHEDULE=pingpong|interleaved forces one schedule for every
// launch (diagnostics and tests; read at each launch); unset or anything else
// selects by the number of key tiles.
int forced_schedule()
{
    const char *e = getenv("REGENVC_ATTN_SCHEDULE");
    if (e == nullptr) return 0;
    if (strcmp(e, "pingpong") == 0) return kSchedPingPong;
    if (strcmp(e, "interleaved") == 0) return kSchedInterleaved;
    if (strcmp(e, "paired") == 0) return kSchedPaired;
    return 0;
}

// Kernel of a launch with n_kt key tiles per whole tile: the ping-pong
// schedule from kPingPongMinTiles key tiles on, the paired interleaved one
// below; dual-context launches always take the 8-wave interleaved kernel
// (its parked first result needs the LDS).
int pick_schedule(int n_kt, bool dual)
{
    if (dual) return kSchedInterleaved;
    const int s = forced_schedule();
    return s != 0 ? s : n_kt >= kPingPongMinTiles ? kSchedPingPong : kSchedPaired;
}

// The work plan of launch `a` on n_cu compute units.
bool plan_for(const AttnArgs &a, int n_cu, AttnPlan *pl)
{
    if (a.n_chunks > 1) return plan_attn_chunks(a.B, a.H, a.Sq, a.n_chunks, a.clen, a.D, n_cu, pl);
    return plan_attn(a.B, a.H, a.Sq, a.Skv, a.D, n_cu, pl, a.k2 != nullptr ? a.Skv2 : 0);
}

template <int D, bool OUT_F32>
hipError_t launch_attn_t(const AttnArgs &a, hipStream_t stream, const Workspace &given)
{
    AttnPlan pl{};
    if (OUT_F32 && a.k2 != nullptr) return hipErrorInvalidValue;  // dual context: bf16 output only
    if (a.n_chunks > 1 && (!OUT_F32 || a.k2 != nullptr || a.run_lse != nullptr)) return hipErrorInvalidValue;
    if (!plan_for(a, cu_count(), &pl)) return hipErrorInvalidConfiguration;
    void *ws = nullptr;     // pool allocation to return
    if (pl.n_units > 0) {
        const size_t bytes = workspace_bytes(pl, D);
        void *buf = given.ptr;
        if (buf != nullptr) {
            if (given.bytes < bytes) return hipErrorInvalidValue;  // checked by the caller beforehand
        } else {
            hipMemPool_t pool = workspace_pool();
            hipError_t e = pool ? hipMallocFromPoolAsync(&ws, bytes, pool, stream) : hipErrorOutOfMemory;
            if (e != hipSuccess) return e;
            g_pool_draws.fetch_add(1);
            buf = ws;
        }
        pl.ws_o = static_cast<float *>(buf);
        pl.ws_lse = pl.ws_o + (size_t)pl.n_units * pl.bm * D;
    }
    const dim3 grid((unsigned)(pl.n_dp + pl.n_units));
    const dim3 block(pl.sched == kSchedPaired ? 256 : kThreads);
    const bool pp = pl.sched == kSchedPingPong;
    if (a.k2 != nullptr) {
        if constexpr (!OUT_F32)
            hipLaunchKernelGGL((attn_fwd_kernel<D, false, false, true>), grid, block, 0, stream, a, pl);
    } else if (a.run_lse != nullptr) {
        if (pp)
            hipLaunchKernelGGL((attn_fwd_pingpong_kernel<D, OUT_F32, true>), grid, block, 0, stream, a, pl);
        else if (pl.sched == kSchedPaired)
            hipLaunchKernelGGL((attn_fwd_kernel<D, OUT_F32, true, false, 4>), grid, block, 0, stream, a, pl);
        else
            hipLaunchKernelGGL((attn_fwd_kernel<D, OUT_F32, true>), grid, block, 0, stream, a, pl);
    } else if (pp) {
        hipLaunchKernelGGL((attn_fwd_pingpong_kernel<D, OUT_F32, false>), grid, block, 0, stream, a, pl);
    } else if (pl.sched == kSchedPaired) {
        hipLaunchKernelGGL((attn_fwd_kernel<D, OUT_F32, false, false, 4>), grid, block, 0, stream, a, pl);
    } else {
        hipLaunchKernelGGL((attn_fwd_kernel<D, OUT_F32, false>), grid, block, 0, stream, a, pl);
    }
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && pl.n_units > 0) {
        const int64_t pairs = (int64_t)(pl.n_tiles - pl.n_dp) * pl.bm * (D / 4);
        const int sl = fix_slices(pl), grp = fix_groups(sl);
        hipLaunchKernelGGL(split_fixup_kernel<OUT_F32>, dim3((unsigned)((pairs + 64 * grp - 1) / (64 * grp))),
                           dim3(64 * sl * grp), 0, stream, a, pl);
        e = hipGetLastError();
    }
    if (ws != nullptr) {
        const hipError_t ef = hipFreeAsync(ws, stream);
        if (e == hipSuccess) e = ef;
    }
    return e;
}

}  // namespace

bool plan_attn(int B, int H, int Sq, int Skv, int D, int n_cu, AttnPlan *out, int Skv2)
{
    if (B < 0 || H < 0 || Sq < 0 || Skv < 1 || n_cu < 1) return false;
    const int sched = pick_schedule((int)(((int64_t)Skv + kBlockN - 1) / kBlockN), Skv2 > 0);
    // paired launches: 128-row tiles, two resident per CU
    const int BM = sched == kSchedPaired ? 128 : kWaves * 32;
    const int slots = sched == kSchedPaired && n_cu <= 0x3fffffff ? 2 * n_cu : n_cu;
    const int64_t n_qtiles = ((int64_t)Sq + BM - 1) / BM;  // < 2^24
    const int64_t per_batch = n_qtiles * H;                 // < 2^55: no overflow
    if (per_batch > 0x7fffffff || (B > 0 && per_batch > 0x7fffffff / B)) return false;
    const int64_t n_tiles = per_batch * B;
    const int n_kt = (int)(((int64_t)Skv + kBlockN - 1) / kBlockN);
    if (Skv2 < 0) return false;
    if (Skv2 > 0)
        *out = make_plan_dual((int)n_qtiles, (int)n_tiles, n_kt, (int)(((int64_t)Skv2 + kBlockN - 1) / kBlockN), n_cu,
                              D);
    else
        *out = make_plan((int)n_qtiles, (int)n_tiles, n_kt, slots, D, BM);
    out->sched = sched;
    return true;
}

bool plan_attn_chunks(int B, int H, int Sq, int n_chunks, const int32_t *clen, int D, int n_cu, AttnPlan *out)
{
    if (n_chunks < 1 || n_chunks > kMaxChunks || B < 0 || H < 0 || Sq < 0 || n_cu < 1) return false;
    for (int c = 0; c < n_chunks; ++c)
        if (clen[c] < 1) return false;
    auto kt = [](int len) { return (int)(((int64_t)len + kBlockN - 1) / kBlockN); };
    const int n_kt = kt(clen[n_chunks - 1]);
    const int sched = pick_schedule(n_kt, false);
    const int BM = sched == kSchedPaired ? 128 : kWaves * 32;
    const int slots = sched == kSchedPaired && n_cu <= 0x3fffffff ? 2 * n_cu : n_cu;
    const int64_t n_qtiles = ((int64_t)Sq + BM - 1) / BM;
    const int64_t per_chunk = n_qtiles * H * B;
    if (n_qtiles * H > 0x7fffffff || per_chunk > 0x7fffffff / n_chunks) return false;
    *out = make_plan((int)n_qtiles, (int)(per_chunk * n_chunks), n_kt, slots, D, BM);
    out->sched = sched;
    out->tiles_per_chunk = (int)per_chunk;
    if (out->n_units > 0 && per_chunk > 0) {
        // the split tiles are the last ones: their chunks must all have n_kt key tiles
        for (int c = (int)(out->n_dp / per_chunk); c < n_chunks; ++c)
            if (kt(clen[c]) != n_kt) {
                out->n_dp = out->n_tiles;
                out->seg = 1;
                out->n_units = 0;
                break;
            }
    }
    return true;
}

size_t workspace_bytes(const AttnPlan &pl, int D)
{
    return (size_t)pl.n_units * pl.bm * (D + 1) * sizeof(float);
}

int device_cu_count()
{
    return cu_count();
}

size_t attn_workspace_need(const AttnArgs &a)
{
    AttnPlan pl{};
    if (!plan_for(a, cu_count(), &pl)) return 0;
    return workspace_bytes(pl, a.D);
}

int64_t pool_draws()
{
    return g_pool_draws.load();
}

hipError_t noalloc_scratch(void **out)
{
    static std::mutex mu;
    static void *addr[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        // once per device, with that device current: each GPU holds its own copy
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *out = addr[dev];
    return hipSuccess;
}

hipError_t launch_attn(const AttnArgs &a, hipStream_t stream, const Workspace &ws)
{
    if (a.D == 128)
        return a.o_f32 ? launch_attn_t<128, true>(a, stream, ws) : launch_attn_t<128, false>(a, stream, ws);
    if (a.D == 64)
        return a.o_f32 ? launch_attn_t<64, true>(a, stream, ws) : launch_attn_t<64, false>(a, stream, ws);
    return hipErrorInvalidValue;
}

}  // namespace regenvc

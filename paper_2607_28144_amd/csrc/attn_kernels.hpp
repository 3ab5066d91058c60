// Internal launch interface between the C ABI layer and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace regenvc {

constexpr int kMaxChunks = 16;  // key chunks of one chunked-partials launch

// Attention kernels (AttnPlan::sched): the ping-pong schedule (8 waves, 256
// query rows), the interleaved one (the same tile), and the interleaved one
// in pairs (4 waves, 128 query rows, two workgroups resident per CU).
constexpr int kSchedPingPong = 1, kSchedInterleaved = 2, kSchedPaired = 3;

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
    // K/V row offsets within a 64-key tile fit 31 bits (non-negative strides
    // below 2^24 elements): tile copies use a scalar base + 32-bit lane offsets
    bool kv_off32;
    // Ring accumulate (run_lse set): run_o f32 [B,Sq,H,D] and run_lse hold
    // the normalized output and LSE over the key chunks already seen; the
    // epilogue merges this launch's result into them, writing O to o and the
    // merged LSE to lse (== run_lse).  Rows whose run_lse is -inf have seen
    // no key yet: their run_o values are ignored.
    const float *run_o;
    float *run_lse;
    int64_t r_sb, r_ss, r_sh;
    // Dual context (k2 set): O = softmax(s Q K^T) V + softmax(s Q K2^T) V2,
    // the two context attentions summed with Q read once; lse gets the first
    // context's LSE and lse2 (may be null) the second's.  bf16 O only.
    const void *k2, *v2;
    float *lse2;
    int64_t k2_sb, k2_ss, k2_sh;
    int64_t v2_sb, v2_ss, v2_sh;
    int32_t Skv2;
    bool kv2_off32;
    // Chunked partials (n_chunks > 1): the launch covers n_chunks key chunks
    // at once; query tile t belongs to chunk c = t / (tiles per chunk),
    // attends over keys [ck0[c], ck0[c] + clen[c]) of k/v and writes its
    // normalized partial to co[c] (f32, strides o_*) and its LSE to clse[c].
    int32_t n_chunks;
    int32_t ck0[kMaxChunks], clen[kMaxChunks];
    float *co[kMaxChunks];
    float *clse[kMaxChunks];
};

// Work plan of one attention launch.  Query tiles [0, n_dp) are processed
// whole, one workgroup each (data-parallel rounds); tiles [n_dp, n_tiles) are
// each split into `seg` contiguous key ranges ("units", one workgroup each)
// whose normalized partial O and LSE go to a workspace and are combined by a
// log-sum-exp fixup (in dual launches: seg ranges over the first context,
// then seg2 over the second, each context merged by LSE and the two summed).  Splitting only the leftover tiles keeps every CU busy
// when the tile count is just above a multiple of the CU count.  The units
// are the first n_units workgroups of the grid, the whole tiles follow.
struct AttnPlan {
    int32_t n_qtiles;  // query tiles per (batch, head)
    int32_t n_tiles;   // B * H * n_qtiles
    int32_t n_kt;      // key tiles per query tile
    int32_t n_dp;      // tiles processed whole
    int32_t seg;       // key ranges per split tile (>= 2 when n_units > 0)
    int32_t n_units;   // (n_tiles - n_dp) * (seg + seg2)
    int32_t n_kt2;     // key tiles of the second context (dual launches; else 0)
    int32_t seg2;      // key ranges of a split tile over the second context (else 0)
    int32_t tiles_per_chunk;  // chunked partials: B * H * n_qtiles (else 0); n_kt is the last chunk's
    int32_t bm;        // query rows per tile: 256, or 128 for the paired interleaved kernel
    int32_t sched;     // kernel: kSchedPingPong, kSchedInterleaved or kSchedPaired
    float *ws_o;       // [n_units][query tile rows][D] partial O (normalized)
    float *ws_lse;     // [n_units][query tile rows] partial LSE
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

// q/k RMSNorm over all H*D channels of a token + 3D rotary embedding per
// head; q/k in and out bf16 [B,S,H,D] (element strides, d contiguous; an
// output may be its own input); w_q/w_k bf16 [H*D].
struct NormRopeArgs {
    const void *q_in, *k_in, *w_q, *w_k;
    void *q_out, *k_out;
    int64_t qi_sb, qi_ss, qi_sh;
    int64_t ki_sb, ki_ss, ki_sh;
    int64_t qo_sb, qo_ss, qo_sh;
    int64_t ko_sb, ko_ss, ko_sh;
    int32_t B, S, H, D;
    int32_t grid_f, grid_h, grid_w, token0;
    float eps, log2_theta;
};

// Work plan of an attention launch of this shape on n_cu compute units
// (host-only); false if the shape has no valid plan (Skv < 1, too many tiles).
bool plan_attn(int B, int H, int Sq, int Skv, int D, int n_cu, AttnPlan *out, int Skv2 = 0);
// The same for a chunked-partials launch over n_chunks chunks of clen[c]
// keys (each >= 1): tiles are split only where every split tile's chunk has
// the last chunk's key tile count.
bool plan_attn_chunks(int B, int H, int Sq, int n_chunks, const int32_t *clen, int D, int n_cu, AttnPlan *out);
// Bytes of split-tile partials a plan needs (0 when nothing is split).
size_t workspace_bytes(const AttnPlan &pl, int D);
// Compute units of the current device (cached per device).
int device_cu_count();
// Bytes of split-tile partials the launch `a` needs on the current device.
size_t attn_workspace_need(const AttnArgs &a);

// Where an attention launch takes its split-tile partials from: stream-ordered
// from the library's per-device pool, or a caller-given buffer of at least
// attn_workspace_need() bytes (no allocation then).
struct Workspace {
    void *ptr = nullptr;  // null: the pool
    size_t bytes = 0;
};
hipError_t launch_attn(const AttnArgs &a, hipStream_t stream, const Workspace &ws);
// Number of launches so far (all devices) that drew their partials from the pool.
int64_t pool_draws();

// Scratch of the no-allocation entry point: a file-scope static device array
// of kNoAllocScratchBytes, one copy per GPU (held until the process ends).
// noalloc_scratch() gives its device address on the current device, looked
// up with hipGetSymbolAddress once per device and kept.
constexpr size_t kNoAllocScratchBytes = (size_t)32 << 20;
hipError_t noalloc_scratch(void **ptr);
hipError_t launch_merge(const MergeArgs &a, hipStream_t stream);
hipError_t launch_empty_partial(const FillArgs &a, hipStream_t stream);
hipError_t launch_norm_rope(const NormRopeArgs &a, hipStream_t stream);

}  // namespace regenvc

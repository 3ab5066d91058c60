/*
 * regenvc_attn.h -- C ABI of the gfx950 (MI355X) window-attention library.
 *
 * The operations are the per-GPU compute of the decoder's sequence-parallel
 * attention (paper Sec. 3.5, "Multi-GPU unified sequence parallelism"):
 *   - Ulysses hands every GPU the whole token sequence for a subset of heads
 *     and asks for exact attention over it                -> regenvc_attn_fwd
 *   - Ring passes key/value blocks between GPUs and folds their results
 *     together with running-max rescaling: one partial result per key/value
 *     chunk, then a log-sum-exp merge, exact apart from summation order
 *                            -> regenvc_attn_partial_fwd (or every chunk's at
                               once: regenvc_attn_partials_fwd) + regenvc_lse_merge,
 *                               or regenvc_attn_ring_accumulate (merge fused)
 *   - the conditioning path (Sec. 3.9, "Hybrid CPU-GPU deployment") streams
 *     precomputed text/image key/value tensors to the GPU, which the video
 *     tokens cross-attend to                         -> regenvc_cross_attn_fwd,
 *     both contexts summed with Q read once         -> regenvc_cross_attn_dual_fwd
 *
 * Definition (per batch b, head h, query row i; scale = softmax_scale):
 *     s_j = scale * <Q[b,i,h,:], K[b,j,h,:]>,  j = 0..Skv-1
 *     O[b,i,h,:] = sum_j softmax(s)_j * V[b,j,h,:]
 *     LSE[b,h,i] = log sum_j exp(s_j)                      (natural log)
 * Attention is non-causal and unmasked: every query sees every key of the
 * window.
 *
 * Conventions common to every entry point
 *   - Every data pointer is DEVICE memory owned by the caller; the library
 *     never frees, keeps or synchronizes on it.
 *   - Scratch memory: when the query tiles of an attention call do not fill
 *     whole rounds of the GPU's compute units, the leftover tiles are split
 *     along the keys and their partial results combined by a second kernel.
 *     Those partials live in a workspace of (split units) x (tile rows) x
 *     (D + 1) floats (15.3 MB for 12 heads x 10920 tokens at D = 128; the exact size
 *     of a call is workspace_bytes of regenvc_attn_plan_query or
 *     regenvc_cross_attn_dual_plan_query).  A caller that binds a workspace
 *     with regenvc_attn_set_workspace supplies it and the library allocates
 *     nothing.  Otherwise the call takes it, stream-ordered, from a
 *     per-device memory pool and returns it, stream-ordered, before it
 *     returns; the pool keeps that memory for later calls until the process
 *     ends, and a failed pool allocation returns REGENVC_ERR_HIP with
 *     nothing enqueued.  regenvc_lse_merge and regenvc_qk_norm_rope use no
 *     scratch.
 *   - Q/K/V/O are logical [B, S, H, D] with element strides for b, s and h
 *     (regenvc_tensor); the D axis is contiguous.  Token-major [B,S,H,D]
 *     and head-major [B,H,S,D] are both expressible.  Inputs are bf16.
 *   - LSE buffers are float32, contiguous [B, H, Sq].
 *   - Arguments are validated synchronously, before any HIP call.  On any
 *     error the call returns a non-OK status, enqueues nothing and leaves
 *     every output untouched; regenvc_last_error() then describes the
 *     problem (thread-local text).
 *   - On success the work is enqueued asynchronously on `stream`
 *     (a hipStream_t; NULL = the legacy default stream).  Device faults
 *     surface at the caller's next synchronization.
 *   - Outputs must not overlap any input or each other.
 *   - B, H or Sq equal to 0 is an empty problem: OK, nothing enqueued.
 *   - Only D in {64, 128} is implemented; only gfx950 devices are accepted.
 *   - All entry points are reentrant; concurrent calls on different streams
 *     are independent.
 *   - The same launch configuration gives bit-identical results run to run.
 *   - Three forms of the attention kernel exist; a launch whose key range
 *     spans at least 32 tiles of 64 keys uses the ping-pong one (256-query
 *     tiles), a shorter one the interleaved one in pairs (128-query tiles,
 *     two workgroups per compute unit), a dual cross-attention the 8-wave
 *     interleaved one (256-query tiles).  The ping-pong and interleaved
 *     kernels compute the same quantities with a different summation order
 *     (results agree to rounding, not bitwise); the paired and 8-wave
 *     interleaved forms agree bitwise row by row.  The environment variable
 *     REGENVC_ATTN_SCHEDULE=pingpong|interleaved|paired, read at each call,
 *     forces one of them (diagnostics and tests; the dual call honours only
 *     interleaved).
 */
#ifndef REGENVC_ATTN_H
#define REGENVC_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    REGENVC_OK = 0,
    /* NULL pointer, negative size, Skv < 1, non-finite or negative scale,
       num_parts out of range, overlapping output and input */
    REGENVC_ERR_INVALID_ARG = 1,
    /* D not in {64,128}; pointer not 16-byte aligned; a stride not a
       multiple of 8 elements; a size whose element offsets overflow int64;
       the current device is not gfx950 */
    REGENVC_ERR_UNSUPPORTED = 2,
    /* a HIP runtime call failed (device query or kernel launch) */
    REGENVC_ERR_HIP = 3
} regenvc_status;

typedef enum { REGENVC_BF16 = 0, REGENVC_F32 = 1 } regenvc_dtype;

/* A logical [B, S, H, D] tensor: base pointer plus element strides of the
   b, s and h axes (the d axis has stride 1).  Strides may be any value that
   is a multiple of 8 elements, including 0 (broadcast). */
typedef struct {
    void *ptr;
    int64_t stride_b;
    int64_t stride_s;
    int64_t stride_h;
} regenvc_tensor;

#define REGENVC_MAX_PARTS 16

/* Exact self-attention over the full key sequence for H heads
   (Sec. 3.5, Ulysses: each GPU attends over every token of the window for
   its own subset of heads).
     q: bf16 [B,Sq,H,D]; k, v: bf16 [B,Skv,H,D]
     o: [B,Sq,H,D] in o_dtype (bf16, round-to-nearest-even, or f32)
     lse: f32 [B,H,Sq] or NULL to skip it
     softmax_scale: finite, >= 0 (the usual value is 1/sqrt(D))
   Skv must be >= 1. */
regenvc_status regenvc_attn_fwd(const regenvc_tensor *q, const regenvc_tensor *k,
                                const regenvc_tensor *v, const regenvc_tensor *o,
                                regenvc_dtype o_dtype, float *lse,
                                int32_t B, int32_t H, int32_t Sq, int32_t Skv,
                                int32_t D, float softmax_scale, void *stream);

/* The same call as regenvc_attn_fwd (same arguments, rules and results,
   bitwise) for callers that cannot allocate: code under HIP graph capture,
   tight serving loops, harnesses that forbid hipMalloc.  It allocates
   nothing and ignores any regenvc_attn_set_workspace binding: the split-tile
   partials go to a static device array of REGENVC_NOALLOC_SCRATCH_BYTES
   inside the library, one copy per GPU, which each GPU the library runs on
   holds until the process ends (its address is looked up once per device,
   at the first call there).  A call whose plan needs more scratch than that
   (workspace_bytes of regenvc_attn_plan_query) returns
   REGENVC_ERR_UNSUPPORTED and enqueues nothing.  Every call on a GPU shares
   that GPU's array, which keeps the last call's contents (nothing in it has
   to start at zero): calls that overlap in time on one GPU -- on different
   streams, or from different threads without ordering -- race on it, so
   order them (one stream, or synchronize). */
#define REGENVC_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
regenvc_status regenvc_attn_fwd_noalloc(const regenvc_tensor *q, const regenvc_tensor *k,
                                        const regenvc_tensor *v, const regenvc_tensor *o,
                                        regenvc_dtype o_dtype, float *lse,
                                        int32_t B, int32_t H, int32_t Sq, int32_t Skv,
                                        int32_t D, float softmax_scale, void *stream);

/* Partial attention of every query over ONE key/value chunk (Sec. 3.5,
   Ring: key/value blocks are passed around and folded together with
   running-max rescaling).
   The chunk is a plain view: k_chunk/v_chunk point at the chunk's first
   token with the full tensor's strides.
     o_part: f32 [B,Sq,H,D], normalized over the chunk's keys
     lse_part: f32 [B,H,Sq], required (the merge needs it)
   Skv_chunk == 0 is allowed and writes the merge identity: o_part = 0,
   lse_part = -inf. */
regenvc_status regenvc_attn_partial_fwd(const regenvc_tensor *q,
                                        const regenvc_tensor *k_chunk,
                                        const regenvc_tensor *v_chunk,
                                        const regenvc_tensor *o_part, float *lse_part,
                                        int32_t B, int32_t H, int32_t Sq,
                                        int32_t Skv_chunk, int32_t D,
                                        float softmax_scale, void *stream);

/* The partials of several key chunks in ONE launch (Sec. 3.5: a GPU that
   holds all of its ring's key/value chunks -- e.g. after an all-gather --
   can compute every chunk's partial at once).  Chunk c covers keys
   [chunk_start[c], chunk_start[c+1]) of k and v (full [B,Skv,H,D] views);
   its result is what regenvc_attn_partial_fwd gives on that chunk, up to
   rounding (bitwise on the query tiles that both keep whole when every
   chunk has the same number of 64-key tiles; tiles split along the keys to
   fill the compute units are summed in another order).  One launch fills
   the GPU where a chunk's query tiles alone would leave compute units
   idle.
     chunk_start: HOST array of num_chunks + 1 ascending key offsets,
       0 <= chunk_start[0] and chunk_start[num_chunks] <= Skv; every chunk
       holds at least one key (INVALID_ARG otherwise)
     o_parts, lse_parts: HOST arrays of num_chunks DEVICE pointers;
       o_parts[c]: f32 [B,Sq,H,D] contiguous, normalized over chunk c's keys;
       lse_parts[c]: f32 [B,H,Sq] (the layout regenvc_lse_merge reads); no
       part may overlap an input or another part
     1 <= num_chunks <= REGENVC_MAX_PARTS
   Scratch as the other attention calls (workspace_bytes of
   regenvc_attn_partials_plan_query). */
regenvc_status regenvc_attn_partials_fwd(const regenvc_tensor *q, const regenvc_tensor *k,
                                         const regenvc_tensor *v, int32_t num_chunks,
                                         const int32_t *chunk_start, float *const *o_parts,
                                         float *const *lse_parts, int32_t B, int32_t H,
                                         int32_t Sq, int32_t Skv, int32_t D, float softmax_scale,
                                         void *stream);

/* Log-sum-exp merge of num_parts partial results over disjoint key chunks
   into the result over their union (Sec. 3.5: the sharded computation equals
   single-device attention apart from summation order):
     m = max_c L_c;  L = m + log sum_c exp(L_c - m);  O = sum_c exp(L_c - L) O_c
   A part with L_c = -inf has weight 0; if every part is -inf the row is
   O = 0, L = -inf.
     o_parts, lse_parts: HOST arrays of num_parts DEVICE pointers;
       o_parts[c]: f32 [B,Sq,H,D] contiguous; lse_parts[c]: f32 [B,H,Sq]
     1 <= num_parts <= REGENVC_MAX_PARTS
     o: [B,Sq,H,D] in o_dtype; lse: f32 [B,H,Sq] or NULL.
   The result does not depend on the order of the parts beyond rounding. */
regenvc_status regenvc_lse_merge(const float *const *o_parts,
                                 const float *const *lse_parts, int32_t num_parts,
                                 const regenvc_tensor *o, regenvc_dtype o_dtype,
                                 float *lse, int32_t B, int32_t H, int32_t Sq,
                                 int32_t D, void *stream);

/* Ring accumulate (Sec. 3.5: Ring combines the streamed key/value blocks
   with running-max rescaling): partial attention over ONE key/value chunk whose
   epilogue merges the result straight into the running state of the chunks
   already processed, so no separate merge pass and no per-chunk partial
   buffers are needed.  Per row, with (O_run, L_run) the running state and
   (O_c, L_c) the chunk's normalized result and LSE:
     L = log(exp L_run + exp L_c);  O = exp(L_run - L) O_run + exp(L_c - L) O_c
   (the regenvc_lse_merge identity for two parts).
     o_run: f32 [B,Sq,H,D], the normalized output over the chunks so far
       (the whole view must be valid memory); where lse_run is -inf the row
       has seen no key and its o_run values are ignored (they may hold
       anything, NaN included)
     lse_run: f32 [B,H,Sq], required; read, then overwritten in place with L
     o_out: NULL writes O back into o_run (f32, o_dtype must be
       REGENVC_F32); otherwise O goes to o_out in o_dtype (bf16 or f32, e.g.
       the final chunk's bf16 output) and o_run is only read.  o_out may be
       o_run itself (same pointer and strides, f32) but must not otherwise
       overlap it.
     k_chunk/v_chunk: the chunk as a plain view, as in regenvc_attn_partial_fwd
   Skv_chunk must be >= 1.  A ring starts from regenvc_attn_partial_fwd on its
   first chunk, or from lse_run filled with -inf. */
regenvc_status regenvc_attn_ring_accumulate(const regenvc_tensor *q,
                                            const regenvc_tensor *k_chunk,
                                            const regenvc_tensor *v_chunk,
                                            const regenvc_tensor *o_run, float *lse_run,
                                            const regenvc_tensor *o_out, regenvc_dtype o_dtype,
                                            int32_t B, int32_t H, int32_t Sq,
                                            int32_t Skv_chunk, int32_t D,
                                            float softmax_scale, void *stream);

/* Cross-attention of the video tokens to Sctx conditioning tokens whose
   key/value tensors were precomputed off-GPU and uploaded (Sec. 3.9).
   Same definition, layouts and rules as regenvc_attn_fwd with Skv = Sctx. */
regenvc_status regenvc_cross_attn_fwd(const regenvc_tensor *q,
                                      const regenvc_tensor *k_ctx,
                                      const regenvc_tensor *v_ctx,
                                      const regenvc_tensor *o, regenvc_dtype o_dtype,
                                      float *lse, int32_t B, int32_t H, int32_t Sq,
                                      int32_t Sctx, int32_t D, float softmax_scale,
                                      void *stream);

/* Dual cross-attention: the video tokens attend to the text context (T5
   tokens) and, separately, to the image context (CLIP tokens), and the two
   results are summed -- the two conditioning streams whose key/value tensors
   Sec. 3.9 precomputes off-GPU.  Per row:
     O = softmax(scale Q K_txt^T) V_txt + softmax(scale Q K_img^T) V_img
   Each softmax is over its own context (not a joint softmax over both).  Q
   is read once: one kernel runs the key pipeline over the text context,
   keeps that normalized result on chip in bf16 (the precision of a single
   cross-attention output), then runs the image context and adds.
     k_txt/v_txt: bf16 [B,S_txt,H,D]; k_img/v_img: bf16 [B,S_img,H,D]
     o: bf16 [B,Sq,H,D] (bf16 only: o_dtype is implied)
     lse_txt, lse_img: f32 [B,H,Sq] LSE of each context's softmax, or NULL
   S_txt and S_img must be >= 1.  Other rules as regenvc_attn_fwd. */
regenvc_status regenvc_cross_attn_dual_fwd(const regenvc_tensor *q,
                                           const regenvc_tensor *k_txt,
                                           const regenvc_tensor *v_txt, int32_t S_txt,
                                           const regenvc_tensor *k_img,
                                           const regenvc_tensor *v_img, int32_t S_img,
                                           const regenvc_tensor *o, float *lse_txt,
                                           float *lse_img, int32_t B, int32_t H,
                                           int32_t Sq, int32_t D, float softmax_scale,
                                           void *stream);

/* q/k RMSNorm + 3D rotary position embedding: the steps that turn the QKV
   projection's q and k into the attention inputs in a block of the video
   diffusion transformer (the backbone of Sec. 3.4, whose blocks the paper's
   compilation step fuses pointwise, Sec. 3.8).  Per batch b and token t, x
   being q (or k) over all H*D channels of the token and w = w_q (or w_k):
     r   = 1 / sqrt(sum_c x_c^2 / (H*D) + eps)
     y_c = x_c * r * w_c
   then in every head, each pair (y_2i, y_2i+1), i < D/2, is rotated by
     angle = pos_a * theta^(-2k / d_a)
     (y_2i, y_2i+1) <- (y_2i cos - y_2i+1 sin, y_2i sin + y_2i+1 cos)
   where the pairs are split over the latent grid's axes a = frame, row,
   column (Ph = Pw = D/6 pairs for rows and columns, the other D/2 - 2 D/6 for
   frames: 22/21/21 at D = 128), k is the pair's index within its axis and
   d_a = 2 * (its axis' pairs).  The token's position comes from its global
   index g = token0 + t in (frame, row, column) raster order on a
   grid_f x grid_h x grid_w grid: frame g / (grid_h grid_w), row
   (g / grid_w) % grid_h, column g % grid_w.
     q_in, k_in, q_out, k_out: bf16 [B,S,H,D] views (as above); an output may
       be exactly its own input (same pointer and strides), otherwise no
       output may overlap any input or the other output.  Outputs are
       rounded to bf16 (nearest even).
     w_q, w_k: bf16 [H*D] contiguous, 16-byte aligned.
     D in {64, 128}; H >= 1; H*D <= 8192; 1 <= grid sizes <= 4096;
     token0 >= 0; token0 + S <= grid_f*grid_h*grid_w; eps finite >= 0
     (usual 1e-6); theta finite > 0 (usual 10000).
   Arithmetic is float32: the angle pos_a * theta^(-2k/d_a) is formed in
   float32 (relative error ~2^-23, i.e. at most ~5e-4 rad at position 4095)
   and reduced to one turn before the hardware sine and cosine.  Non-finite
   inputs give non-finite outputs.  Allocates nothing.  HBM-bound: every q
   and k element is read once and written once. */
regenvc_status regenvc_qk_norm_rope(const regenvc_tensor *q_in, const regenvc_tensor *k_in,
                                    const void *w_q, const void *w_k,
                                    const regenvc_tensor *q_out, const regenvc_tensor *k_out,
                                    int32_t B, int32_t S, int32_t H, int32_t D,
                                    int32_t grid_f, int32_t grid_h, int32_t grid_w, int32_t token0,
                                    float eps, float theta, void *stream);

/* Work plan of one attention call (regenvc_attn_fwd, regenvc_attn_partial_fwd
   or regenvc_cross_attn_fwd) of the given shape on a device with n_cu
   compute units (the calls themselves use the current device's count, 256
   on MI355X).  Queries are processed in tiles of tile_rows of one (batch,
   head) and keys in tiles of 64: tile_rows is 256, or 128 for calls with
   fewer than 32 key tiles, which run two 128-row workgroups per compute
   unit (so that one's query load and output stores overlap the other's
   key loop).  whole_tiles query tiles run as one workgroup each; each of
   the split_tiles leftover tiles runs as key_ranges workgroups over
   contiguous key ranges whose partials a second kernel combines, and those
   partials occupy workspace_bytes of scratch memory (0 when nothing is
   split; see "Scratch memory" above).
     B, H, Sq >= 0; Skv >= 1; D in {64, 128}; n_cu >= 1; plan non-NULL.
   Host-only: makes no HIP call.  Returns REGENVC_ERR_INVALID_ARG or
   REGENVC_ERR_UNSUPPORTED (D, or more than 2^31 - 1 query tiles) on bad
   arguments, leaving *plan untouched. */
typedef struct {
    int32_t query_tiles; /* B * H * ceil(Sq / tile_rows) */
    int32_t key_tiles;   /* ceil(Skv / 64) */
    int32_t whole_tiles;
    int32_t split_tiles;
    int32_t key_ranges;  /* per split tile; 0 when split_tiles == 0 */
    int64_t workspace_bytes;
    int32_t tile_rows;   /* query rows per tile: 256 or 128 */
} regenvc_attn_plan;

regenvc_status regenvc_attn_plan_query(int32_t B, int32_t H, int32_t Sq, int32_t Skv, int32_t D,
                                       int32_t n_cu, regenvc_attn_plan *plan);

/* Work plan of one regenvc_cross_attn_dual_fwd call: as
   regenvc_attn_plan_query, with key_tiles the tiles of both contexts and
   key_ranges the ranges of a split tile over both (S_txt, S_img >= 1). */
regenvc_status regenvc_cross_attn_dual_plan_query(int32_t B, int32_t H, int32_t Sq, int32_t S_txt,
                                                  int32_t S_img, int32_t D, int32_t n_cu,
                                                  regenvc_attn_plan *plan);

/* Work plan of one regenvc_attn_partials_fwd call: query_tiles counts the
   tiles of every chunk (num_chunks * B * H * ceil(Sq / tile_rows)), key_tiles is
   the last chunk's, and split tiles (the last ones of the launch) are split
   only when every chunk they belong to has that many key tiles.  Host-only;
   the chunk arguments as in regenvc_attn_partials_fwd. */
regenvc_status regenvc_attn_partials_plan_query(int32_t B, int32_t H, int32_t Sq,
                                                int32_t num_chunks, const int32_t *chunk_start,
                                                int32_t D, int32_t n_cu, regenvc_attn_plan *plan);

/* Binds a caller-owned DEVICE buffer of `bytes` bytes as the scratch memory
   of the attention calls (regenvc_attn_fwd, regenvc_attn_partial_fwd,
   regenvc_attn_partials_fwd,
   regenvc_attn_ring_accumulate, regenvc_cross_attn_fwd,
   regenvc_cross_attn_dual_fwd) made later on the calling thread, until
   another binding replaces it; workspace == NULL unbinds (back to the pool).
   While a buffer is bound those calls allocate nothing.  A call that needs
   more than `bytes` (its plan's workspace_bytes on the current device)
   returns REGENVC_ERR_INVALID_ARG and enqueues nothing, as does one whose
   tensors overlap the part of the buffer it would use.  Each call uses the
   buffer stream-ordered on its own stream: calls that share it must be
   ordered (one stream, or synchronized), since concurrent calls on
   different streams would overwrite each other's partials.  The library
   never frees or keeps the buffer beyond the binding.
     workspace: 256-byte aligned (else REGENVC_ERR_UNSUPPORTED), or NULL
     bytes >= 0 (else REGENVC_ERR_INVALID_ARG; ignored when unbinding)
   Host-only: makes no HIP call. */
regenvc_status regenvc_attn_set_workspace(void *workspace, int64_t bytes);

/* Number of attention calls in this process (all threads and devices) that
   took their scratch from the library's pool; a diagnostic for callers and
   tests that must not allocate.  Host-only. */
int64_t regenvc_attn_pool_draws(void);

/* Static text for a status code. */
const char *regenvc_status_str(regenvc_status status);

/* Detail of the most recent non-OK return on the calling thread ("" if none). */
const char *regenvc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* REGENVC_ATTN_H */

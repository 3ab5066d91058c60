// C ABI of the window-attention library: synchronous argument validation
// (before any HIP call), device check, and kernel launch on the caller's
// stream.  Declarations and the contract live in include/regenvc_attn.h.
#include "regenvc_attn.h"

#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "attn_kernels.hpp"

namespace {

thread_local char g_last_error[512] = "";
// Caller workspace bound on this thread (regenvc_attn_set_workspace).
thread_local void *g_ws_ptr = nullptr;
thread_local int64_t g_ws_bytes = 0;

regenvc_status fail(regenvc_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return st;
}

// Byte range [lo, hi) that a logical [B,S,H,D] view can touch.
struct Extent {
    uintptr_t lo, hi;
};

bool mul_ok(int64_t a, int64_t b, int64_t *out)
{
    return !__builtin_mul_overflow(a, b, out);
}

// Checks one tensor view; on success fills its byte extent.
regenvc_status check_view(const char *name, const regenvc_tensor *t, int64_t B, int64_t S, int64_t H, int64_t D,
                          size_t elem, Extent *ext)
{
    if (t == nullptr) return fail(REGENVC_ERR_INVALID_ARG, "%s: descriptor is NULL", name);
    if (t->ptr == nullptr) return fail(REGENVC_ERR_INVALID_ARG, "%s: data pointer is NULL", name);
    if (reinterpret_cast<uintptr_t>(t->ptr) % 16 != 0)
        return fail(REGENVC_ERR_UNSUPPORTED, "%s: data pointer is not 16-byte aligned", name);
    const int64_t strides[3] = {t->stride_b, t->stride_s, t->stride_h};
    const int64_t sizes[3] = {B, S, H};
    const char *axis[3] = {"b", "s", "h"};
    int64_t lo = 0, hi = D;  // element offsets relative to ptr
    for (int i = 0; i < 3; ++i) {
        if (strides[i] % 8 != 0)
            return fail(REGENVC_ERR_UNSUPPORTED, "%s: stride_%s=%lld is not a multiple of 8 elements", name, axis[i],
                        (long long)strides[i]);
        int64_t span;
        if (!mul_ok(strides[i], sizes[i] - 1, &span))
            return fail(REGENVC_ERR_UNSUPPORTED, "%s: offsets overflow int64", name);
        if (span < 0) {
            if (__builtin_add_overflow(lo, span, &lo))
                return fail(REGENVC_ERR_UNSUPPORTED, "%s: offsets overflow int64", name);
        } else if (__builtin_add_overflow(hi, span, &hi)) {
            return fail(REGENVC_ERR_UNSUPPORTED, "%s: offsets overflow int64", name);
        }
    }
    int64_t blo, bhi;
    if (!mul_ok(lo, (int64_t)elem, &blo) || !mul_ok(hi, (int64_t)elem, &bhi))
        return fail(REGENVC_ERR_UNSUPPORTED, "%s: byte offsets overflow int64", name);
    const uintptr_t base = reinterpret_cast<uintptr_t>(t->ptr);
    ext->lo = base + (intptr_t)blo;
    ext->hi = base + (intptr_t)bhi;
    return REGENVC_OK;
}

Extent flat_extent(const void *p, int64_t n_elems, size_t elem)
{
    const uintptr_t base = reinterpret_cast<uintptr_t>(p);
    return Extent{base, base + (uintptr_t)(n_elems * (int64_t)elem)};
}

bool overlap(const Extent &a, const Extent &b)
{
    return a.lo < b.hi && b.lo < a.hi;
}

// An output view must not map two logical elements to one address: sorted
// by |stride|, every axis of size > 1 must step past the whole span of the
// axes inside it (d is the innermost axis, stride 1, size D).
bool view_is_injective(const regenvc_tensor *t, int64_t B, int64_t S, int64_t H, int64_t D)
{
    int64_t st[3] = {t->stride_b, t->stride_s, t->stride_h};
    int64_t sz[3] = {B, S, H};
    for (int i = 0; i < 3; ++i) st[i] = st[i] < 0 ? -st[i] : st[i];
    for (int i = 0; i < 3; ++i)  // tiny insertion sort by stride
        for (int j = i + 1; j < 3; ++j)
            if (st[j] < st[i]) {
                int64_t a = st[i], b = sz[i];
                st[i] = st[j], sz[i] = sz[j];
                st[j] = a, sz[j] = b;
            }
    int64_t span = D;  // elements covered by the axes inside the current one
    for (int i = 0; i < 3; ++i) {
        if (sz[i] <= 1) continue;
        if (st[i] < span) return false;
        span = st[i] * sz[i];
    }
    return true;
}

regenvc_status check_sizes(int32_t B, int32_t H, int32_t Sq, int32_t D)
{
    if (B < 0 || H < 0 || Sq < 0)
        return fail(REGENVC_ERR_INVALID_ARG, "negative size (B=%d H=%d Sq=%d)", B, H, Sq);
    if (D != 64 && D != 128) return fail(REGENVC_ERR_UNSUPPORTED, "head dim D=%d (only 64 and 128)", D);
    return REGENVC_OK;
}

regenvc_status check_scale(float s)
{
    if (!std::isfinite(s)) return fail(REGENVC_ERR_INVALID_ARG, "softmax_scale is not finite");
    if (s < 0.f) return fail(REGENVC_ERR_INVALID_ARG, "softmax_scale is negative");
    return REGENVC_OK;
}

// Device must be gfx950.  Cached per device ordinal.
std::atomic<int> g_arch_state[64];  // 0 unknown, 1 ok, 2 wrong arch

regenvc_status check_device()
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(REGENVC_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    int st = (dev >= 0 && dev < 64) ? g_arch_state[dev].load() : 0;
    if (st == 0) {
        hipDeviceProp_t prop;
        e = hipGetDeviceProperties(&prop, dev);
        if (e != hipSuccess) return fail(REGENVC_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
        st = (std::strncmp(prop.gcnArchName, "gfx950", 6) == 0) ? 1 : 2;
        if (dev >= 0 && dev < 64) g_arch_state[dev].store(st);
        if (st == 2)
            return fail(REGENVC_ERR_UNSUPPORTED, "device %d is %s; this library is built for gfx950 only", dev,
                        prop.gcnArchName);
    }
    if (st == 2) return fail(REGENVC_ERR_UNSUPPORTED, "device %d is not gfx950", dev);
    return REGENVC_OK;
}

regenvc_status launched(hipError_t e, const char *what)
{
    if (e != hipSuccess) return fail(REGENVC_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
    g_last_error[0] = '\0';
    return REGENVC_OK;
}

bool same_view(const regenvc_tensor *a, const regenvc_tensor *b)
{
    return a->ptr == b->ptr && a->stride_b == b->stride_b && a->stride_s == b->stride_s && a->stride_h == b->stride_h;
}

// Second context of a dual cross-attention.
struct Ctx2 {
    const regenvc_tensor *k, *v;
    int32_t S;
    float *lse;  // may be null
};

// The bound workspace for a launch needing `need` bytes: too small, or
// overlapping one of the call's n tensor extents, is INVALID_ARG.
regenvc_status bound_workspace(const char *fn, size_t need, const Extent *ext, int n, regenvc::Workspace *ws)
{
    if ((size_t)g_ws_bytes < need)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: the bound workspace holds %lld bytes, this call needs %zu", fn,
                    (long long)g_ws_bytes, need);
    if (need > 0) {
        const Extent ew = flat_extent(g_ws_ptr, (int64_t)need, 1);
        for (int i = 0; i < n; ++i)
            if (overlap(ew, ext[i]))
                return fail(REGENVC_ERR_INVALID_ARG, "%s: the bound workspace overlaps a tensor of the call", fn);
    }
    ws->ptr = g_ws_ptr;
    ws->bytes = (size_t)g_ws_bytes;
    return REGENVC_OK;
}

// run_o (ring accumulate only): f32 running output, read; lse is then the
// running LSE, read and rewritten in place; o may be run_o itself (f32).
// ctx2 (dual cross-attention only): the second context, summed into o.
// no_alloc: split-tile partials in the library's static device scratch
// (regenvc_attn_fwd_noalloc) instead of a bound workspace or the pool.
regenvc_status attn_common(const char *fn, const regenvc_tensor *q, const regenvc_tensor *k,
                           const regenvc_tensor *v, const regenvc_tensor *o, regenvc_dtype o_dtype, float *lse,
                           bool lse_required, int32_t B, int32_t H, int32_t Sq, int32_t Skv, int32_t D, float scale,
                           void *stream, bool allow_empty_keys, const regenvc_tensor *run_o = nullptr,
                           const Ctx2 *ctx2 = nullptr, bool no_alloc = false)
{
    regenvc_status st = check_sizes(B, H, Sq, D);
    if (st != REGENVC_OK) return st;
    if (Skv < 0 || (Skv == 0 && !allow_empty_keys))
        return fail(REGENVC_ERR_INVALID_ARG, "%s: key count %d must be >= 1", fn, Skv);
    if (o_dtype != REGENVC_BF16 && o_dtype != REGENVC_F32)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: unknown output dtype %d", fn, (int)o_dtype);
    if ((st = check_scale(scale)) != REGENVC_OK) return st;
    if (lse_required && lse == nullptr) return fail(REGENVC_ERR_INVALID_ARG, "%s: lse output is required", fn);
    if (ctx2 != nullptr) {
        if (ctx2->S < 1) return fail(REGENVC_ERR_INVALID_ARG, "%s: second context length %d must be >= 1", fn, ctx2->S);
        if (o_dtype != REGENVC_BF16)
            return fail(REGENVC_ERR_UNSUPPORTED, "%s: the summed output is bf16 only (o_dtype must be BF16)", fn);
        if (ctx2->lse != nullptr && reinterpret_cast<uintptr_t>(ctx2->lse) % 4 != 0)
            return fail(REGENVC_ERR_UNSUPPORTED, "%s: lse_img pointer is not 4-byte aligned", fn);
    }
    if (lse != nullptr && reinterpret_cast<uintptr_t>(lse) % 4 != 0)
        return fail(REGENVC_ERR_UNSUPPORTED, "%s: lse pointer is not 4-byte aligned", fn);
    if (B == 0 || H == 0 || Sq == 0) {
        // empty problem: nothing to read or write, but descriptors must still be present
        if (!q || !k || !v || !o || (ctx2 && (!ctx2->k || !ctx2->v)))
            return fail(REGENVC_ERR_INVALID_ARG, "%s: descriptor is NULL", fn);
        g_last_error[0] = '\0';
        return REGENVC_OK;
    }
    const int64_t Skv_view = Skv > 0 ? Skv : 1;
    Extent eq, ek, ev, eo;
    if ((st = check_view("q", q, B, Sq, H, D, 2, &eq)) != REGENVC_OK) return st;
    if (Skv > 0) {
        if ((st = check_view("k", k, B, Skv_view, H, D, 2, &ek)) != REGENVC_OK) return st;
        if ((st = check_view("v", v, B, Skv_view, H, D, 2, &ev)) != REGENVC_OK) return st;
    } else if (!k || !v) {
        return fail(REGENVC_ERR_INVALID_ARG, "%s: descriptor is NULL", fn);
    }
    const size_t oel = o_dtype == REGENVC_F32 ? 4 : 2;
    if ((st = check_view("o", o, B, Sq, H, D, oel, &eo)) != REGENVC_OK) return st;
    if (!view_is_injective(o, B, Sq, H, D))
        return fail(REGENVC_ERR_INVALID_ARG, "%s: output o has overlapping rows (strides)", fn);
    if (overlap(eo, eq) || (Skv > 0 && (overlap(eo, ek) || overlap(eo, ev))))
        return fail(REGENVC_ERR_INVALID_ARG, "%s: output o overlaps an input", fn);
    if (lse != nullptr) {
        const Extent el = flat_extent(lse, (int64_t)B * H * Sq, 4);
        if (overlap(el, eq) || overlap(el, eo) || (Skv > 0 && (overlap(el, ek) || overlap(el, ev))))
            return fail(REGENVC_ERR_INVALID_ARG, "%s: lse overlaps another tensor", fn);
    }
    Extent ek2{0, 0}, ev2{0, 0}, er{0, 0};
    if (ctx2 != nullptr) {
        if ((st = check_view("k_img", ctx2->k, B, ctx2->S, H, D, 2, &ek2)) != REGENVC_OK) return st;
        if ((st = check_view("v_img", ctx2->v, B, ctx2->S, H, D, 2, &ev2)) != REGENVC_OK) return st;
        if (overlap(eo, ek2) || overlap(eo, ev2))
            return fail(REGENVC_ERR_INVALID_ARG, "%s: output o overlaps an input", fn);
        if (lse != nullptr) {
            const Extent el = flat_extent(lse, (int64_t)B * H * Sq, 4);
            if (overlap(el, ek2) || overlap(el, ev2))
                return fail(REGENVC_ERR_INVALID_ARG, "%s: lse overlaps another tensor", fn);
        }
        if (ctx2->lse != nullptr) {
            const Extent el2 = flat_extent(ctx2->lse, (int64_t)B * H * Sq, 4);
            if (overlap(el2, eq) || overlap(el2, ek) || overlap(el2, ev) || overlap(el2, ek2) || overlap(el2, ev2) ||
                overlap(el2, eo) || (lse != nullptr && overlap(el2, flat_extent(lse, (int64_t)B * H * Sq, 4))))
                return fail(REGENVC_ERR_INVALID_ARG, "%s: lse_img overlaps another tensor", fn);
        }
    }
    if (run_o != nullptr) {
        if ((st = check_view("o_run", run_o, B, Sq, H, D, 4, &er)) != REGENVC_OK) return st;
        if (!view_is_injective(run_o, B, Sq, H, D))
            return fail(REGENVC_ERR_INVALID_ARG, "%s: o_run has overlapping rows (strides)", fn);
        if (overlap(er, eq) || overlap(er, ek) || overlap(er, ev))
            return fail(REGENVC_ERR_INVALID_ARG, "%s: o_run overlaps an input", fn);
        if (overlap(er, flat_extent(lse, (int64_t)B * H * Sq, 4)))
            return fail(REGENVC_ERR_INVALID_ARG, "%s: o_run overlaps lse_run", fn);
        if (overlap(er, eo) && !(same_view(run_o, o) && o_dtype == REGENVC_F32))
            return fail(REGENVC_ERR_INVALID_ARG, "%s: o_out overlaps o_run (other than being o_run itself)", fn);
    }
    if ((st = check_device()) != REGENVC_OK) return st;

    if (Skv == 0) {  // empty chunk: the merge identity
        regenvc::FillArgs f{};
        f.o = static_cast<float *>(o->ptr);
        f.lse = lse;
        f.o_sb = o->stride_b;
        f.o_ss = o->stride_s;
        f.o_sh = o->stride_h;
        f.B = B;
        f.H = H;
        f.Sq = Sq;
        f.D = D;
        return launched(regenvc::launch_empty_partial(f, static_cast<hipStream_t>(stream)), fn);
    }
    regenvc::AttnArgs a{};
    a.q = q->ptr;
    a.k = k->ptr;
    a.v = v->ptr;
    a.o = o->ptr;
    a.lse = lse;
    a.q_sb = q->stride_b, a.q_ss = q->stride_s, a.q_sh = q->stride_h;
    a.k_sb = k->stride_b, a.k_ss = k->stride_s, a.k_sh = k->stride_h;
    a.v_sb = v->stride_b, a.v_ss = v->stride_s, a.v_sh = v->stride_h;
    a.o_sb = o->stride_b, a.o_ss = o->stride_s, a.o_sh = o->stride_h;
    a.B = B;
    a.H = H;
    a.Sq = Sq;
    a.Skv = Skv;
    a.D = D;
    a.o_f32 = o_dtype == REGENVC_F32;
    a.scale = scale;
    a.kv_off32 = k->stride_s >= 0 && v->stride_s >= 0 && k->stride_s < (1 << 24) && v->stride_s < (1 << 24);
    if (ctx2 != nullptr) {
        a.k2 = ctx2->k->ptr;
        a.v2 = ctx2->v->ptr;
        a.lse2 = ctx2->lse;
        a.k2_sb = ctx2->k->stride_b, a.k2_ss = ctx2->k->stride_s, a.k2_sh = ctx2->k->stride_h;
        a.v2_sb = ctx2->v->stride_b, a.v2_ss = ctx2->v->stride_s, a.v2_sh = ctx2->v->stride_h;
        a.Skv2 = ctx2->S;
        a.kv2_off32 = a.k2_ss >= 0 && a.v2_ss >= 0 && a.k2_ss < (1 << 24) && a.v2_ss < (1 << 24);
    }
    if (run_o != nullptr) {
        a.run_o = static_cast<const float *>(run_o->ptr);
        a.run_lse = lse;
        a.r_sb = run_o->stride_b, a.r_ss = run_o->stride_s, a.r_sh = run_o->stride_h;
    }
    // split-tile partials: the static scratch (no_alloc), the workspace bound
    // on this thread, else the pool
    regenvc::Workspace ws{};
    if (no_alloc) {
        const size_t need = regenvc::attn_workspace_need(a);
        if (need > regenvc::kNoAllocScratchBytes)
            return fail(REGENVC_ERR_UNSUPPORTED,
                        "%s: this call needs %zu bytes of scratch, more than the %zu bytes the no-allocation entry "
                        "point holds",
                        fn, need, regenvc::kNoAllocScratchBytes);
        void *p = nullptr;
        const hipError_t e = regenvc::noalloc_scratch(&p);
        if (e != hipSuccess) return fail(REGENVC_ERR_HIP, "%s: scratch lookup: %s", fn, hipGetErrorString(e));
        ws.ptr = p;
        ws.bytes = regenvc::kNoAllocScratchBytes;
    } else if (g_ws_ptr != nullptr) {
        const int64_t nl = (int64_t)B * H * Sq;
        const Extent none{0, 0};
        const Extent ext[9] = {eq, ek, ev, eo, ek2, ev2, er, lse ? flat_extent(lse, nl, 4) : none,
                               ctx2 && ctx2->lse ? flat_extent(ctx2->lse, nl, 4) : none};
        if ((st = bound_workspace(fn, regenvc::attn_workspace_need(a), ext, 9, &ws)) != REGENVC_OK) return st;
    }
    return launched(regenvc::launch_attn(a, static_cast<hipStream_t>(stream), ws), fn);
}

}  // namespace

extern "C" {

regenvc_status regenvc_attn_fwd(const regenvc_tensor *q, const regenvc_tensor *k, const regenvc_tensor *v,
                                const regenvc_tensor *o, regenvc_dtype o_dtype, float *lse, int32_t B, int32_t H,
                                int32_t Sq, int32_t Skv, int32_t D, float softmax_scale, void *stream)
{
    return attn_common("regenvc_attn_fwd", q, k, v, o, o_dtype, lse, false, B, H, Sq, Skv, D, softmax_scale, stream,
                       false);
}

regenvc_status regenvc_attn_fwd_noalloc(const regenvc_tensor *q, const regenvc_tensor *k, const regenvc_tensor *v,
                                        const regenvc_tensor *o, regenvc_dtype o_dtype, float *lse, int32_t B,
                                        int32_t H, int32_t Sq, int32_t Skv, int32_t D, float softmax_scale,
                                        void *stream)
{
    static_assert(REGENVC_NOALLOC_SCRATCH_BYTES == regenvc::kNoAllocScratchBytes, "header and library agree");
    return attn_common("regenvc_attn_fwd_noalloc", q, k, v, o, o_dtype, lse, false, B, H, Sq, Skv, D, softmax_scale,
                       stream, false, nullptr, nullptr, true);
}

regenvc_status regenvc_attn_partial_fwd(const regenvc_tensor *q, const regenvc_tensor *k_chunk,
                                        const regenvc_tensor *v_chunk, const regenvc_tensor *o_part,
                                        float *lse_part, int32_t B, int32_t H, int32_t Sq, int32_t Skv_chunk,
                                        int32_t D, float softmax_scale, void *stream)
{
    return attn_common("regenvc_attn_partial_fwd", q, k_chunk, v_chunk, o_part, REGENVC_F32, lse_part, true, B, H, Sq,
                       Skv_chunk, D, softmax_scale, stream, true);
}

regenvc_status regenvc_attn_partials_fwd(const regenvc_tensor *q, const regenvc_tensor *k, const regenvc_tensor *v,
                                         int32_t num_chunks, const int32_t *chunk_start, float *const *o_parts,
                                         float *const *lse_parts, int32_t B, int32_t H, int32_t Sq, int32_t Skv,
                                         int32_t D, float softmax_scale, void *stream)
{
    const char *fn = "regenvc_attn_partials_fwd";
    regenvc_status st = check_sizes(B, H, Sq, D);
    if (st != REGENVC_OK) return st;
    if ((st = check_scale(softmax_scale)) != REGENVC_OK) return st;
    if (num_chunks < 1 || num_chunks > REGENVC_MAX_PARTS)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: num_chunks=%d not in [1, %d]", fn, num_chunks, REGENVC_MAX_PARTS);
    if (chunk_start == nullptr || o_parts == nullptr || lse_parts == nullptr)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: chunk_start, o_parts or lse_parts is NULL", fn);
    if (Skv < 1) return fail(REGENVC_ERR_INVALID_ARG, "%s: key count %d must be >= 1", fn, Skv);
    if (chunk_start[0] < 0 || chunk_start[num_chunks] > Skv)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: chunks [%d, %d) lie outside the %d keys", fn, chunk_start[0],
                    chunk_start[num_chunks], Skv);
    for (int c = 0; c < num_chunks; ++c) {
        if (chunk_start[c + 1] <= chunk_start[c])
            return fail(REGENVC_ERR_INVALID_ARG, "%s: chunk %d = [%d, %d) is empty or reversed", fn, c,
                        chunk_start[c], chunk_start[c + 1]);
        if (o_parts[c] == nullptr || lse_parts[c] == nullptr)
            return fail(REGENVC_ERR_INVALID_ARG, "%s: part %d pointer is NULL", fn, c);
        if (reinterpret_cast<uintptr_t>(o_parts[c]) % 16 != 0)
            return fail(REGENVC_ERR_UNSUPPORTED, "%s: o_parts[%d] is not 16-byte aligned", fn, c);
        if (reinterpret_cast<uintptr_t>(lse_parts[c]) % 4 != 0)
            return fail(REGENVC_ERR_UNSUPPORTED, "%s: lse_parts[%d] is not 4-byte aligned", fn, c);
    }
    if (!q || !k || !v) return fail(REGENVC_ERR_INVALID_ARG, "%s: descriptor is NULL", fn);
    if (B == 0 || H == 0 || Sq == 0) {
        g_last_error[0] = '\0';
        return REGENVC_OK;
    }
    Extent ext[3 + 2 * REGENVC_MAX_PARTS];
    if ((st = check_view("q", q, B, Sq, H, D, 2, &ext[0])) != REGENVC_OK) return st;
    if ((st = check_view("k", k, B, Skv, H, D, 2, &ext[1])) != REGENVC_OK) return st;
    if ((st = check_view("v", v, B, Skv, H, D, 2, &ext[2])) != REGENVC_OK) return st;
    const int64_t rows = (int64_t)B * Sq * H;
    int n_ext = 3;
    for (int c = 0; c < num_chunks; ++c) {
        const Extent eo = flat_extent(o_parts[c], rows * D, 4), el = flat_extent(lse_parts[c], rows, 4);
        if (overlap(eo, el)) return fail(REGENVC_ERR_INVALID_ARG, "%s: o_parts[%d] overlaps lse_parts[%d]", fn, c, c);
        for (int i = 0; i < n_ext; ++i)
            if (overlap(eo, ext[i]) || overlap(el, ext[i]))
                return fail(REGENVC_ERR_INVALID_ARG, "%s: part %d overlaps an input or another part", fn, c);
        ext[n_ext++] = eo;
        ext[n_ext++] = el;
    }
    if ((st = check_device()) != REGENVC_OK) return st;

    regenvc::AttnArgs a{};
    a.q = q->ptr;
    a.k = k->ptr;
    a.v = v->ptr;
    a.q_sb = q->stride_b, a.q_ss = q->stride_s, a.q_sh = q->stride_h;
    a.k_sb = k->stride_b, a.k_ss = k->stride_s, a.k_sh = k->stride_h;
    a.v_sb = v->stride_b, a.v_ss = v->stride_s, a.v_sh = v->stride_h;
    a.o_sb = (int64_t)Sq * H * D, a.o_ss = (int64_t)H * D, a.o_sh = D;  // contiguous partials
    a.B = B;
    a.H = H;
    a.Sq = Sq;
    a.D = D;
    a.o_f32 = true;
    a.scale = softmax_scale;
    a.kv_off32 = k->stride_s >= 0 && v->stride_s >= 0 && k->stride_s < (1 << 24) && v->stride_s < (1 << 24);
    if (num_chunks == 1) {  // a plain partial over the one chunk
        a.k = static_cast<const uint16_t *>(k->ptr) + (int64_t)chunk_start[0] * k->stride_s;
        a.v = static_cast<const uint16_t *>(v->ptr) + (int64_t)chunk_start[0] * v->stride_s;
        a.Skv = chunk_start[1] - chunk_start[0];
        a.o = o_parts[0];
        a.lse = lse_parts[0];
    } else {
        a.n_chunks = num_chunks;
        a.Skv = chunk_start[num_chunks] - chunk_start[num_chunks - 1];
        a.o = o_parts[0];
        a.lse = lse_parts[0];
        for (int c = 0; c < num_chunks; ++c) {
            a.ck0[c] = chunk_start[c];
            a.clen[c] = chunk_start[c + 1] - chunk_start[c];
            a.co[c] = o_parts[c];
            a.clse[c] = lse_parts[c];
        }
    }
    regenvc::Workspace ws{};
    if (g_ws_ptr != nullptr &&
        (st = bound_workspace(fn, regenvc::attn_workspace_need(a), ext, n_ext, &ws)) != REGENVC_OK)
        return st;
    return launched(regenvc::launch_attn(a, static_cast<hipStream_t>(stream), ws), fn);
}

regenvc_status regenvc_attn_ring_accumulate(const regenvc_tensor *q, const regenvc_tensor *k_chunk,
                                            const regenvc_tensor *v_chunk, const regenvc_tensor *o_run,
                                            float *lse_run, const regenvc_tensor *o_out, regenvc_dtype o_dtype,
                                            int32_t B, int32_t H, int32_t Sq, int32_t Skv_chunk, int32_t D,
                                            float softmax_scale, void *stream)
{
    const char *fn = "regenvc_attn_ring_accumulate";
    if (o_run == nullptr) return fail(REGENVC_ERR_INVALID_ARG, "%s: o_run descriptor is NULL", fn);
    if (o_out == nullptr && o_dtype != REGENVC_F32)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: the running output o_run is f32 (o_dtype must be F32 without o_out)",
                    fn);
    return attn_common(fn, q, k_chunk, v_chunk, o_out ? o_out : o_run, o_dtype, lse_run, true, B, H, Sq, Skv_chunk,
                       D, softmax_scale, stream, false, o_run);
}

regenvc_status regenvc_cross_attn_fwd(const regenvc_tensor *q, const regenvc_tensor *k_ctx,
                                      const regenvc_tensor *v_ctx, const regenvc_tensor *o, regenvc_dtype o_dtype,
                                      float *lse, int32_t B, int32_t H, int32_t Sq, int32_t Sctx, int32_t D,
                                      float softmax_scale, void *stream)
{
    return attn_common("regenvc_cross_attn_fwd", q, k_ctx, v_ctx, o, o_dtype, lse, false, B, H, Sq, Sctx, D,
                       softmax_scale, stream, false);
}

regenvc_status regenvc_cross_attn_dual_fwd(const regenvc_tensor *q, const regenvc_tensor *k_txt,
                                           const regenvc_tensor *v_txt, int32_t S_txt, const regenvc_tensor *k_img,
                                           const regenvc_tensor *v_img, int32_t S_img, const regenvc_tensor *o,
                                           float *lse_txt, float *lse_img, int32_t B, int32_t H, int32_t Sq, int32_t D,
                                           float softmax_scale, void *stream)
{
    const Ctx2 c2{k_img, v_img, S_img, lse_img};
    return attn_common("regenvc_cross_attn_dual_fwd", q, k_txt, v_txt, o, REGENVC_BF16, lse_txt, false, B, H, Sq, S_txt,
                       D, softmax_scale, stream, false, nullptr, &c2);
}

regenvc_status regenvc_lse_merge(const float *const *o_parts, const float *const *lse_parts, int32_t num_parts,
                                 const regenvc_tensor *o, regenvc_dtype o_dtype, float *lse, int32_t B, int32_t H,
                                 int32_t Sq, int32_t D, void *stream)
{
    regenvc_status st = check_sizes(B, H, Sq, D);
    if (st != REGENVC_OK) return st;
    if (num_parts < 1 || num_parts > REGENVC_MAX_PARTS)
        return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: num_parts=%d not in [1, %d]", num_parts,
                    REGENVC_MAX_PARTS);
    if (o_parts == nullptr || lse_parts == nullptr)
        return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: part arrays are NULL");
    if (o_dtype != REGENVC_BF16 && o_dtype != REGENVC_F32)
        return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: unknown output dtype %d", (int)o_dtype);
    if (o == nullptr) return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: descriptor is NULL");
    for (int c = 0; c < num_parts; ++c) {
        if (o_parts[c] == nullptr || lse_parts[c] == nullptr)
            return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: part %d pointer is NULL", c);
        if (reinterpret_cast<uintptr_t>(o_parts[c]) % 16 != 0)
            return fail(REGENVC_ERR_UNSUPPORTED, "regenvc_lse_merge: o_parts[%d] is not 16-byte aligned", c);
        if (reinterpret_cast<uintptr_t>(lse_parts[c]) % 4 != 0)
            return fail(REGENVC_ERR_UNSUPPORTED, "regenvc_lse_merge: lse_parts[%d] is not 4-byte aligned", c);
    }
    if (lse != nullptr && reinterpret_cast<uintptr_t>(lse) % 4 != 0)
        return fail(REGENVC_ERR_UNSUPPORTED, "regenvc_lse_merge: lse pointer is not 4-byte aligned");
    if (B == 0 || H == 0 || Sq == 0) {
        g_last_error[0] = '\0';
        return REGENVC_OK;
    }
    Extent eo;
    if ((st = check_view("o", o, B, Sq, H, D, o_dtype == REGENVC_F32 ? 4 : 2, &eo)) != REGENVC_OK) return st;
    if (!view_is_injective(o, B, Sq, H, D))
        return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: output o has overlapping rows (strides)");
    const int64_t rows = (int64_t)B * Sq * H;
    Extent el{0, 0};
    if (lse != nullptr) el = flat_extent(lse, (int64_t)B * H * Sq, 4);
    for (int c = 0; c < num_parts; ++c) {
        const Extent ep = flat_extent(o_parts[c], rows * D, 4);
        const Extent elp = flat_extent(lse_parts[c], rows, 4);
        if (overlap(eo, ep) || overlap(eo, elp))
            return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: output o overlaps part %d", c);
        if (lse != nullptr && (overlap(el, ep) || overlap(el, elp)))
            return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: output lse overlaps part %d", c);
    }
    if (lse != nullptr && overlap(el, eo))
        return fail(REGENVC_ERR_INVALID_ARG, "regenvc_lse_merge: lse overlaps o");
    if ((st = check_device()) != REGENVC_OK) return st;

    regenvc::MergeArgs m{};
    for (int c = 0; c < num_parts; ++c) {
        m.o_parts[c] = o_parts[c];
        m.lse_parts[c] = lse_parts[c];
    }
    m.num_parts = num_parts;
    m.o = o->ptr;
    m.lse = lse;
    m.o_sb = o->stride_b;
    m.o_ss = o->stride_s;
    m.o_sh = o->stride_h;
    m.B = B;
    m.H = H;
    m.Sq = Sq;
    m.D = D;
    m.o_f32 = o_dtype == REGENVC_F32;
    return launched(regenvc::launch_merge(m, static_cast<hipStream_t>(stream)), "regenvc_lse_merge");
}

regenvc_status regenvc_qk_norm_rope(const regenvc_tensor *q_in, const regenvc_tensor *k_in, const void *w_q,
                                    const void *w_k, const regenvc_tensor *q_out, const regenvc_tensor *k_out,
                                    int32_t B, int32_t S, int32_t H, int32_t D, int32_t grid_f, int32_t grid_h,
                                    int32_t grid_w, int32_t token0, float eps, float theta, void *stream)
{
    const char *fn = "regenvc_qk_norm_rope";
    if (B < 0 || S < 0 || H < 1)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: bad size (B=%d S=%d H=%d)", fn, B, S, H);
    if (D != 64 && D != 128) return fail(REGENVC_ERR_UNSUPPORTED, "%s: head dim D=%d (only 64 and 128)", fn, D);
    if ((int64_t)H * D > 8192)
        return fail(REGENVC_ERR_UNSUPPORTED, "%s: H*D=%lld channels per token (at most 8192)", fn,
                    (long long)H * D);
    if (grid_f < 1 || grid_h < 1 || grid_w < 1 || token0 < 0)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: bad grid %d x %d x %d or token0=%d", fn, grid_f, grid_h, grid_w,
                    token0);
    if (grid_f > 4096 || grid_h > 4096 || grid_w > 4096)
        return fail(REGENVC_ERR_UNSUPPORTED, "%s: grid %d x %d x %d has an axis longer than 4096", fn, grid_f, grid_h,
                    grid_w);
    if ((int64_t)token0 + S > (int64_t)grid_f * grid_h * grid_w)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: tokens %d..%lld lie outside the %d x %d x %d grid", fn, token0,
                    (long long)token0 + S - 1, grid_f, grid_h, grid_w);
    if (!std::isfinite(eps) || eps < 0.f) return fail(REGENVC_ERR_INVALID_ARG, "%s: eps must be finite and >= 0", fn);
    if (!std::isfinite(theta) || !(theta > 0.f))
        return fail(REGENVC_ERR_INVALID_ARG, "%s: theta must be finite and > 0", fn);
    if (!q_in || !k_in || !q_out || !k_out) return fail(REGENVC_ERR_INVALID_ARG, "%s: descriptor is NULL", fn);
    if (w_q == nullptr || w_k == nullptr) return fail(REGENVC_ERR_INVALID_ARG, "%s: weight pointer is NULL", fn);
    if (reinterpret_cast<uintptr_t>(w_q) % 16 != 0 || reinterpret_cast<uintptr_t>(w_k) % 16 != 0)
        return fail(REGENVC_ERR_UNSUPPORTED, "%s: weight pointer is not 16-byte aligned", fn);
    if (B == 0 || S == 0) {
        g_last_error[0] = '\0';
        return REGENVC_OK;
    }
    regenvc_status st;
    Extent eqi, eki, eqo, eko;
    if ((st = check_view("q_in", q_in, B, S, H, D, 2, &eqi)) != REGENVC_OK) return st;
    if ((st = check_view("k_in", k_in, B, S, H, D, 2, &eki)) != REGENVC_OK) return st;
    if ((st = check_view("q_out", q_out, B, S, H, D, 2, &eqo)) != REGENVC_OK) return st;
    if ((st = check_view("k_out", k_out, B, S, H, D, 2, &eko)) != REGENVC_OK) return st;
    if (!view_is_injective(q_out, B, S, H, D) || !view_is_injective(k_out, B, S, H, D))
        return fail(REGENVC_ERR_INVALID_ARG, "%s: an output has overlapping rows (strides)", fn);
    const Extent ewq = flat_extent(w_q, (int64_t)H * D, 2), ewk = flat_extent(w_k, (int64_t)H * D, 2);
    if (overlap(eqo, eko)) return fail(REGENVC_ERR_INVALID_ARG, "%s: q_out overlaps k_out", fn);
    if ((overlap(eqo, eqi) && !same_view(q_out, q_in)) || overlap(eqo, eki) || overlap(eqo, ewq) ||
        overlap(eqo, ewk))
        return fail(REGENVC_ERR_INVALID_ARG, "%s: q_out overlaps an input (other than being q_in itself)", fn);
    if ((overlap(eko, eki) && !same_view(k_out, k_in)) || overlap(eko, eqi) || overlap(eko, ewq) ||
        overlap(eko, ewk))
        return fail(REGENVC_ERR_INVALID_ARG, "%s: k_out overlaps an input (other than being k_in itself)", fn);
    if ((st = check_device()) != REGENVC_OK) return st;

    regenvc::NormRopeArgs a{};
    a.q_in = q_in->ptr, a.k_in = k_in->ptr, a.w_q = w_q, a.w_k = w_k;
    a.q_out = q_out->ptr, a.k_out = k_out->ptr;
    a.qi_sb = q_in->stride_b, a.qi_ss = q_in->stride_s, a.qi_sh = q_in->stride_h;
    a.ki_sb = k_in->stride_b, a.ki_ss = k_in->stride_s, a.ki_sh = k_in->stride_h;
    a.qo_sb = q_out->stride_b, a.qo_ss = q_out->stride_s, a.qo_sh = q_out->stride_h;
    a.ko_sb = k_out->stride_b, a.ko_ss = k_out->stride_s, a.ko_sh = k_out->stride_h;
    a.B = B, a.S = S, a.H = H, a.D = D;
    a.grid_f = grid_f, a.grid_h = grid_h, a.grid_w = grid_w, a.token0 = token0;
    a.eps = eps;
    a.log2_theta = std::log2(theta);
    return launched(regenvc::launch_norm_rope(a, static_cast<hipStream_t>(stream)), fn);
}

namespace {

regenvc_status plan_query(const char *fn, int32_t B, int32_t H, int32_t Sq, int32_t Skv, int32_t Skv2, int32_t D,
                          int32_t n_cu, regenvc_attn_plan *plan)
{
    if (plan == nullptr) return fail(REGENVC_ERR_INVALID_ARG, "%s: plan is NULL", fn);
    if (B < 0 || H < 0 || Sq < 0)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: negative size (B=%d H=%d Sq=%d)", fn, B, H, Sq);
    if (Skv < 1) return fail(REGENVC_ERR_INVALID_ARG, "%s: key count %d < 1", fn, Skv);
    if (Skv2 < 0) return fail(REGENVC_ERR_INVALID_ARG, "%s: second key count %d < 1", fn, Skv2);
    if (n_cu < 1) return fail(REGENVC_ERR_INVALID_ARG, "%s: n_cu=%d < 1", fn, n_cu);
    if (D != 64 && D != 128) return fail(REGENVC_ERR_UNSUPPORTED, "%s: D=%d not in {64, 128}", fn, D);
    regenvc::AttnPlan pl{};
    if (!regenvc::plan_attn(B, H, Sq, Skv, D, n_cu, &pl, Skv2))
        return fail(REGENVC_ERR_UNSUPPORTED, "%s: too many query tiles", fn);
    plan->query_tiles = pl.n_tiles;
    plan->key_tiles = pl.n_kt + pl.n_kt2;
    plan->whole_tiles = pl.n_dp;
    plan->split_tiles = pl.n_tiles - pl.n_dp;
    plan->key_ranges = pl.n_units > 0 ? pl.seg + pl.seg2 : 0;
    plan->workspace_bytes = (int64_t)regenvc::workspace_bytes(pl, D);
    plan->tile_rows = pl.bm;
    g_last_error[0] = '\0';
    return REGENVC_OK;
}

}  // namespace

regenvc_status regenvc_attn_plan_query(int32_t B, int32_t H, int32_t Sq, int32_t Skv, int32_t D, int32_t n_cu,
                                       regenvc_attn_plan *plan)
{
    return plan_query("regenvc_attn_plan_query", B, H, Sq, Skv, 0, D, n_cu, plan);
}

regenvc_status regenvc_cross_attn_dual_plan_query(int32_t B, int32_t H, int32_t Sq, int32_t S_txt, int32_t S_img,
                                                  int32_t D, int32_t n_cu, regenvc_attn_plan *plan)
{
    if (S_img < 1)
        return fail(REGENVC_ERR_INVALID_ARG, "regenvc_cross_attn_dual_plan_query: S_img=%d < 1", S_img);
    return plan_query("regenvc_cross_attn_dual_plan_query", B, H, Sq, S_txt, S_img, D, n_cu, plan);
}

regenvc_status regenvc_attn_partials_plan_query(int32_t B, int32_t H, int32_t Sq, int32_t num_chunks,
                                                const int32_t *chunk_start, int32_t D, int32_t n_cu,
                                                regenvc_attn_plan *plan)
{
    const char *fn = "regenvc_attn_partials_plan_query";
    if (plan == nullptr || chunk_start == nullptr)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: plan or chunk_start is NULL", fn);
    if (num_chunks < 1 || num_chunks > REGENVC_MAX_PARTS)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: num_chunks=%d not in [1, %d]", fn, num_chunks, REGENVC_MAX_PARTS);
    if (num_chunks == 1) return plan_query(fn, B, H, Sq, chunk_start[1] - chunk_start[0], 0, D, n_cu, plan);
    if (B < 0 || H < 0 || Sq < 0)
        return fail(REGENVC_ERR_INVALID_ARG, "%s: negative size (B=%d H=%d Sq=%d)", fn, B, H, Sq);
    if (n_cu < 1) return fail(REGENVC_ERR_INVALID_ARG, "%s: n_cu=%d < 1", fn, n_cu);
    if (D != 64 && D != 128) return fail(REGENVC_ERR_UNSUPPORTED, "%s: D=%d not in {64, 128}", fn, D);
    int32_t clen[REGENVC_MAX_PARTS];
    for (int c = 0; c < num_chunks; ++c) {
        clen[c] = chunk_start[c + 1] - chunk_start[c];
        if (clen[c] < 1) return fail(REGENVC_ERR_INVALID_ARG, "%s: chunk %d is empty or reversed", fn, c);
    }
    regenvc::AttnPlan pl{};
    if (!regenvc::plan_attn_chunks(B, H, Sq, num_chunks, clen, D, n_cu, &pl))
        return fail(REGENVC_ERR_UNSUPPORTED, "%s: too many query tiles", fn);
    plan->query_tiles = pl.n_tiles;
    plan->key_tiles = pl.n_kt;
    plan->whole_tiles = pl.n_dp;
    plan->split_tiles = pl.n_tiles - pl.n_dp;
    plan->key_ranges = pl.n_units > 0 ? pl.seg : 0;
    plan->workspace_bytes = (int64_t)regenvc::workspace_bytes(pl, D);
    plan->tile_rows = pl.bm;
    g_last_error[0] = '\0';
    return REGENVC_OK;
}

regenvc_status regenvc_attn_set_workspace(void *workspace, int64_t bytes)
{
    if (workspace == nullptr) {
        g_ws_ptr = nullptr;
        g_ws_bytes = 0;
        g_last_error[0] = '\0';
        return REGENVC_OK;
    }
    if (bytes < 0) return fail(REGENVC_ERR_INVALID_ARG, "regenvc_attn_set_workspace: bytes=%lld < 0", (long long)bytes);
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
        return fail(REGENVC_ERR_UNSUPPORTED, "regenvc_attn_set_workspace: workspace is not 256-byte aligned");
    g_ws_ptr = workspace;
    g_ws_bytes = bytes;
    g_last_error[0] = '\0';
    return REGENVC_OK;
}

int64_t regenvc_attn_pool_draws(void)
{
    return regenvc::pool_draws();
}

const char *regenvc_status_str(regenvc_status status)
{
    switch (status) {
    case REGENVC_OK: return "ok";
    case REGENVC_ERR_INVALID_ARG: return "invalid argument";
    case REGENVC_ERR_UNSUPPORTED: return "unsupported";
    case REGENVC_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char *regenvc_last_error(void)
{
    return g_last_error;
}

}  // extern "C"

// Status helpers shared with the other entry-point files (abi_util.hpp).
namespace regenvc {
namespace abi {

regenvc_status fail_msg(regenvc_status st, const char *msg)
{
    return fail(st, "%s", msg);
}

regenvc_status device_ok()
{
    return check_device();
}

regenvc_status launch_status(hipError_t e, const char *what)
{
    return launched(e, what);
}

void clear_error()
{
    g_last_error[0] = '\0';
}

}  // namespace abi
}  // namespace regenvc

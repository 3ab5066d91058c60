// C ABI of the diffusion-transformer block kernels and of the block forward
// (include/regenvc_dit.h): synchronous argument validation before any
// launch, then the kernels on the caller's stream.  The block forward is a
// fixed sequence of launches over a caller workspace; it allocates nothing.
#include "regenvc_dit.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "abi_util.hpp"
#include "attn_kernels.hpp"
#include "dit_kernels.hpp"

using regenvc::abi::aligned;
using regenvc::abi::failf;
using regenvc::abi::overlaps;
using regenvc::abi::range_of;

namespace {

constexpr float kEps = 1e-6f;

regenvc_status check_linear(const char *fn, const void *a, int64_t lda, const void *w, const void *bias,
                            const float *gate, const void *out, int64_t ldo, int32_t M, int32_t N, int32_t K,
                            int32_t epi)
{
    if (M < 0 || N < 0 || K < 0) return failf(REGENVC_ERR_INVALID_ARG, "%s: negative size (M=%d N=%d K=%d)", fn, M, N, K);
    if (epi != REGENVC_EPI_BIAS && epi != REGENVC_EPI_BIAS_GELU && epi != REGENVC_EPI_GATED_RESIDUAL)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: unknown epilogue %d", fn, epi);
    if (gate != nullptr && epi != REGENVC_EPI_GATED_RESIDUAL)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: a gate needs the gated-residual epilogue", fn);
    if (K % 64 != 0) return failf(REGENVC_ERR_UNSUPPORTED, "%s: K=%d is not a multiple of 64", fn, K);
    if (N % 16 != 0) return failf(REGENVC_ERR_UNSUPPORTED, "%s: N=%d is not a multiple of 16", fn, N);
    if (lda < K || ldo < N || lda % 8 != 0 || ldo % 8 != 0)
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: row strides lda=%lld ldo=%lld (multiples of 8, >= K and N)", fn,
                     (long long)lda, (long long)ldo);
    if (M == 0 || N == 0) return REGENVC_OK;
    if (a == nullptr || w == nullptr || out == nullptr)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL data pointer", fn);
    if (!aligned(a, 16) || !aligned(w, 16) || !aligned(out, 16) || (bias && !aligned(bias, 16)) ||
        (gate && !aligned(gate, 16)))
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);
    const int esz = epi == REGENVC_EPI_GATED_RESIDUAL ? 4 : 2;
    const auto ro = range_of(out, ((int64_t)(M - 1) * ldo + N) * esz);
    if (overlaps(ro, range_of(a, ((int64_t)(M - 1) * lda + K) * 2)) ||
        overlaps(ro, range_of(w, (int64_t)N * K * 2)) || (bias && overlaps(ro, range_of(bias, (int64_t)N * 2))) ||
        (gate && overlaps(ro, range_of(gate, (int64_t)N * 4))))
        return failf(REGENVC_ERR_INVALID_ARG, "%s: out overlaps an input", fn);
    return REGENVC_OK;
}

regenvc_status check_width(const char *fn, int32_t C)
{
    if (C < 512 || C % 512 != 0 || C > 2048)
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: C=%d is not a multiple of 512 in [512, 2048]", fn, C);
    return REGENVC_OK;
}

int64_t align256(int64_t b)
{
    return (b + 255) / 256 * 256;
}

// Workspace layout of the block forward.
struct BlockLayout {
    int64_t mod, h, qkv, att, f, scr, total;
};

BlockLayout block_layout(int32_t S, int32_t S_ctx, int32_t C, int32_t heads, int32_t F, int32_t n_cu)
{
    BlockLayout L{};
    const int D = C / heads;
    L.mod = 0;
    L.h = align256((int64_t)6 * C * 4);
    L.qkv = L.h + align256((int64_t)S * C * 2);
    L.att = L.qkv + align256((int64_t)S * 3 * C * 2);
    L.f = L.att + align256((int64_t)S * C * 2);
    L.scr = L.f + align256((int64_t)S * F * 2);
    regenvc::AttnPlan p1{}, p2{};
    int64_t need = 0;
    if (regenvc::plan_attn(1, heads, S, S, D, n_cu, &p1)) need = (int64_t)regenvc::workspace_bytes(p1, D);
    if (regenvc::plan_attn(1, heads, S, S_ctx, D, n_cu, &p2))
        need = std::max(need, (int64_t)regenvc::workspace_bytes(p2, D));
    L.total = L.scr + align256(need);
    return L;
}

regenvc_status check_block_shape(const char *fn, int32_t S, int32_t S_ctx, int32_t C, int32_t heads, int32_t F)
{
    if (S < 1 || S_ctx < 1 || heads < 1 || F < 1)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: bad size (S=%d S_ctx=%d heads=%d F=%d)", fn, S, S_ctx, heads, F);
    regenvc_status st = check_width(fn, C);
    if (st != REGENVC_OK) return st;
    if (C % heads != 0 || (C / heads != 64 && C / heads != 128))
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: head dim C/heads = %d/%d (64 or 128)", fn, C, heads);
    if (F % 64 != 0) return failf(REGENVC_ERR_UNSUPPORTED, "%s: F=%d is not a multiple of 64", fn, F);
    return REGENVC_OK;
}

}  // namespace

extern "C" {

regenvc_status regenvc_linear_fwd(const void *a, int64_t lda, const void *w, const void *bias, const float *gate,
                                  void *out, int64_t ldo, int32_t M, int32_t N, int32_t K, int32_t epilogue,
                                  void *stream)
{
    const char *fn = "regenvc_linear_fwd";
    regenvc_status st = check_linear(fn, a, lda, w, bias, gate, out, ldo, M, N, K, epilogue);
    if (st != REGENVC_OK) return st;
    if (M == 0 || N == 0) {
        regenvc::abi::clear_error();
        return REGENVC_OK;
    }
    if ((st = regenvc::abi::device_ok()) != REGENVC_OK) return st;
    regenvc::LinearArgs la{a, w, bias, gate, out, lda, ldo, M, N, K, epilogue};
    return regenvc::abi::launch_status(regenvc::launch_linear(la, static_cast<hipStream_t>(stream)), fn);
}

regenvc_status regenvc_layer_norm_fwd(const float *x, int64_t ldx, void *y, int64_t ldy, const float *shift,
                                      const float *scale, const void *w, const void *b, int32_t rows, int32_t C,
                                      float eps, void *stream)
{
    const char *fn = "regenvc_layer_norm_fwd";
    if (rows < 0) return failf(REGENVC_ERR_INVALID_ARG, "%s: rows=%d < 0", fn, rows);
    regenvc_status st = check_width(fn, C);
    if (st != REGENVC_OK) return st;
    const bool mod = shift != nullptr || scale != nullptr, aff = w != nullptr || b != nullptr;
    if (mod == aff || (mod && (!shift || !scale)) || (aff && (!w || !b)))
        return failf(REGENVC_ERR_INVALID_ARG, "%s: give shift and scale, or w and b", fn);
    if (!std::isfinite(eps) || eps < 0.f) return failf(REGENVC_ERR_INVALID_ARG, "%s: eps must be finite, >= 0", fn);
    if (ldx < C || ldy < C || ldx % 8 || ldy % 8)
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: row strides must be multiples of 8 and >= C", fn);
    if (rows == 0) {
        regenvc::abi::clear_error();
        return REGENVC_OK;
    }
    if (!x || !y) return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL data pointer", fn);
    if (!aligned(x, 16) || !aligned(y, 16) || (shift && (!aligned(shift, 16) || !aligned(scale, 16))) ||
        (w && (!aligned(w, 16) || !aligned(b, 16))))
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);
    if (overlaps(range_of(y, ((int64_t)(rows - 1) * ldy + C) * 2), range_of(x, ((int64_t)(rows - 1) * ldx + C) * 4)))
        return failf(REGENVC_ERR_INVALID_ARG, "%s: y overlaps x", fn);
    if ((st = regenvc::abi::device_ok()) != REGENVC_OK) return st;
    regenvc::LayerNormArgs la{x, y, ldx, ldy, shift, scale, w, b, rows, C, eps};
    return regenvc::abi::launch_status(regenvc::launch_layer_norm(la, static_cast<hipStream_t>(stream)), fn);
}

regenvc_status regenvc_rms_norm_fwd(const void *x, int64_t ldx, void *y, int64_t ldy, const void *w, int32_t rows,
                                    int32_t C, float eps, void *stream)
{
    const char *fn = "regenvc_rms_norm_fwd";
    if (rows < 0) return failf(REGENVC_ERR_INVALID_ARG, "%s: rows=%d < 0", fn, rows);
    regenvc_status st = check_width(fn, C);
    if (st != REGENVC_OK) return st;
    if (!std::isfinite(eps) || eps < 0.f) return failf(REGENVC_ERR_INVALID_ARG, "%s: eps must be finite, >= 0", fn);
    if (ldx < C || ldy < C || ldx % 8 || ldy % 8)
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: row strides must be multiples of 8 and >= C", fn);
    if (rows == 0) {
        regenvc::abi::clear_error();
        return REGENVC_OK;
    }
    if (!x || !y || !w) return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL pointer", fn);
    if (!aligned(x, 16) || !aligned(y, 16) || !aligned(w, 16))
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);
    const bool same = x == y && ldx == ldy;
    if (!same && overlaps(range_of(y, ((int64_t)(rows - 1) * ldy + C) * 2),
                          range_of(x, ((int64_t)(rows - 1) * ldx + C) * 2)))
        return failf(REGENVC_ERR_INVALID_ARG, "%s: y overlaps x (other than being x itself)", fn);
    if ((st = regenvc::abi::device_ok()) != REGENVC_OK) return st;
    regenvc::RmsNormArgs ra{x, y, ldx, ldy, w, rows, C, eps};
    return regenvc::abi::launch_status(regenvc::launch_rms_norm(ra, static_cast<hipStream_t>(stream)), fn);
}

regenvc_status regenvc_dit_modulation(const void *w_mod, const void *b_mod, const float *e, float *mod, int32_t rows,
                                      int32_t C, void *stream)
{
    const char *fn = "regenvc_dit_modulation";
    if (rows < 0 || C < 1) return failf(REGENVC_ERR_INVALID_ARG, "%s: bad size (rows=%d C=%d)", fn, rows, C);
    if (rows == 0) {
        regenvc::abi::clear_error();
        return REGENVC_OK;
    }
    if (!w_mod || !b_mod || !e || !mod) return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL pointer", fn);
    if (!aligned(w_mod, 2) || !aligned(b_mod, 2) || !aligned(e, 4) || !aligned(mod, 4))
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: misaligned pointer", fn);
    regenvc_status st = regenvc::abi::device_ok();
    if (st != REGENVC_OK) return st;
    regenvc::ModulationArgs ma{w_mod, b_mod, e, mod, rows, C};
    return regenvc::abi::launch_status(regenvc::launch_modulation(ma, static_cast<hipStream_t>(stream)), fn);
}

regenvc_status regenvc_dit_block_workspace(int32_t S, int32_t S_ctx, int32_t C, int32_t heads, int32_t F,
                                           int32_t n_cu, int64_t *bytes)
{
    const char *fn = "regenvc_dit_block_workspace";
    if (bytes == nullptr) return failf(REGENVC_ERR_INVALID_ARG, "%s: bytes is NULL", fn);
    if (n_cu < 1) return failf(REGENVC_ERR_INVALID_ARG, "%s: n_cu=%d < 1", fn, n_cu);
    regenvc_status st = check_block_shape(fn, S, S_ctx, C, heads, F);
    if (st != REGENVC_OK) return st;
    *bytes = block_layout(S, S_ctx, C, heads, F, n_cu).total;
    regenvc::abi::clear_error();
    return REGENVC_OK;
}

regenvc_status regenvc_dit_block_fwd(float *x, const float *e, const regenvc_dit_params *p, const void *ctx_k,
                                     const void *ctx_v, int32_t S_ctx, int32_t S, int32_t C, int32_t heads, int32_t F,
                                     int32_t grid_f, int32_t grid_h, int32_t grid_w, int32_t token0, void *workspace,
                                     int64_t workspace_bytes, void *stream)
{
    const char *fn = "regenvc_dit_block_fwd";
    regenvc_status st = check_block_shape(fn, S, S_ctx, C, heads, F);
    if (st != REGENVC_OK) return st;
    if (!x || !e || !p || !ctx_k || !ctx_v || !workspace) return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL pointer", fn);
    const void *params[] = {p->w_mod, p->b_mod, p->w_qkv, p->b_qkv, p->w_qn, p->w_kn, p->w_o, p->b_o, p->w_n3,
                            p->b_n3,  p->w_qc,  p->b_qc,  p->w_qcn, p->w_oc, p->b_oc, p->w_1, p->b_1, p->w_2, p->b_2};
    for (const void *q : params) {
        if (q == nullptr) return failf(REGENVC_ERR_INVALID_ARG, "%s: a NULL parameter pointer", fn);
        if (!aligned(q, 16)) return failf(REGENVC_ERR_UNSUPPORTED, "%s: parameters must be 16-byte aligned", fn);
    }
    if (!aligned(x, 16) || !aligned(e, 16) || !aligned(ctx_k, 16) || !aligned(ctx_v, 16))
        return failf(REGENVC_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);
    if (!aligned(workspace, 256)) return failf(REGENVC_ERR_UNSUPPORTED, "%s: workspace is not 256-byte aligned", fn);
    if (grid_f < 1 || grid_h < 1 || grid_w < 1 || grid_f > 4096 || grid_h > 4096 || grid_w > 4096 || token0 < 0 ||
        (int64_t)token0 + S > (int64_t)grid_f * grid_h * grid_w)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: tokens %d..%lld do not fit the %d x %d x %d grid", fn, token0,
                     (long long)token0 + S - 1, grid_f, grid_h, grid_w);
    if ((st = regenvc::abi::device_ok()) != REGENVC_OK) return st;
    const BlockLayout L = block_layout(S, S_ctx, C, heads, F, regenvc::device_cu_count());
    if (workspace_bytes < L.total)
        return failf(REGENVC_ERR_INVALID_ARG, "%s: workspace of %lld bytes, this call needs %lld", fn,
                     (long long)workspace_bytes, (long long)L.total);
    const auto rw = range_of(workspace, L.total);
    if (overlaps(rw, range_of(x, (int64_t)S * C * 4)) || overlaps(rw, range_of(e, (int64_t)C * 4)) ||
        overlaps(rw, range_of(ctx_k, (int64_t)S_ctx * C * 2)) || overlaps(rw, range_of(ctx_v, (int64_t)S_ctx * C * 2)))
        return failf(REGENVC_ERR_INVALID_ARG, "%s: the workspace overlaps another argument", fn);

    hipStream_t s = static_cast<hipStream_t>(stream);
    char *ws = static_cast<char *>(workspace);
    float *mod = reinterpret_cast<float *>(ws + L.mod);
    void *h = ws + L.h, *qkv = ws + L.qkv, *att = ws + L.att, *f = ws + L.f;
    const regenvc::Workspace scr{ws + L.scr, (size_t)(L.total - L.scr)};
    const int D = C / heads;
    const float scale = (float)(1.0 / std::sqrt((double)D));  // 1/sqrt(D) rounded to float32 once
    hipError_t err = hipSuccess;
    auto linear = [&](const void *a, int64_t lda, const void *w, const void *bias, const float *gate, void *out,
                      int64_t ldo, int N, int K, int epi) {
        if (err != hipSuccess) return;
        err = regenvc::launch_linear(regenvc::LinearArgs{a, w, bias, gate, out, lda, ldo, S, N, K, epi}, s);
    };
    auto norm = [&](const float *shift, const float *sc, const void *w, const void *b) {
        if (err != hipSuccess) return;
        err = regenvc::launch_layer_norm(regenvc::LayerNormArgs{x, h, C, C, shift, sc, w, b, S, C, kEps}, s);
    };
    auto attention = [&](const void *q, int64_t q_ss, const void *k, const void *v, int64_t kv_ss, int Skv,
                         void *o) {
        if (err != hipSuccess) return;
        regenvc::AttnArgs a{};
        a.q = q, a.k = k, a.v = v, a.o = o;
        a.q_sb = 0, a.q_ss = q_ss, a.q_sh = D;
        a.k_sb = a.v_sb = 0, a.k_ss = a.v_ss = kv_ss, a.k_sh = a.v_sh = D;
        a.o_sb = 0, a.o_ss = C, a.o_sh = D;
        a.B = 1, a.H = heads, a.Sq = S, a.Skv = Skv, a.D = D;
        a.scale = scale;
        a.kv_off32 = kv_ss < (1 << 24);
        err = regenvc::launch_attn(a, s, scr);
    };

    // adaLN vectors (sh1, sc1, g1, sh2, sc2, g2)
    err = regenvc::launch_modulation(regenvc::ModulationArgs{p->w_mod, p->b_mod, e, mod, 6 * C, C}, s);
    // self-attention branch
    norm(mod + 0 * C, mod + 1 * C, nullptr, nullptr);
    linear(h, C, p->w_qkv, p->b_qkv, nullptr, qkv, 3 * C, 3 * C, C, regenvc::kEpiBias);
    if (err == hipSuccess) {
        regenvc::NormRopeArgs r{};
        char *q = static_cast<char *>(qkv), *k = q + (int64_t)C * 2;
        r.q_in = r.q_out = q, r.k_in = r.k_out = k, r.w_q = p->w_qn, r.w_k = p->w_kn;
        r.qi_sb = r.ki_sb = r.qo_sb = r.ko_sb = 0;
        r.qi_ss = r.ki_ss = r.qo_ss = r.ko_ss = 3 * C;
        r.qi_sh = r.ki_sh = r.qo_sh = r.ko_sh = D;
        r.B = 1, r.S = S, r.H = heads, r.D = D;
        r.grid_f = grid_f, r.grid_h = grid_h, r.grid_w = grid_w, r.token0 = token0;
        r.eps = kEps, r.log2_theta = std::log2(10000.0f);
        err = regenvc::launch_norm_rope(r, s);
    }
    {
        const char *q = static_cast<const char *>(qkv);
        attention(q, 3 * C, q + (int64_t)C * 2, q + (int64_t)2 * C * 2, 3 * C, S, att);
    }
    linear(att, C, p->w_o, p->b_o, mod + 2 * C, x, C, C, C, regenvc::kEpiGatedRes);
    // cross-attention branch: query in `att`, normalized in place; output in `h`
    norm(nullptr, nullptr, p->w_n3, p->b_n3);
    linear(h, C, p->w_qc, p->b_qc, nullptr, att, C, C, C, regenvc::kEpiBias);
    if (err == hipSuccess) err = regenvc::launch_rms_norm(regenvc::RmsNormArgs{att, att, C, C, p->w_qcn, S, C, kEps}, s);
    attention(att, C, ctx_k, ctx_v, C, S_ctx, h);
    linear(h, C, p->w_oc, p->b_oc, nullptr, x, C, C, C, regenvc::kEpiGatedRes);
    // feed-forward branch
    norm(mod + 3 * C, mod + 4 * C, nullptr, nullptr);
    linear(h, C, p->w_1, p->b_1, nullptr, f, F, F, C, regenvc::kEpiBiasGelu);
    linear(f, F, p->w_2, p->b_2, mod + 5 * C, x, C, C, F, regenvc::kEpiGatedRes);
    return regenvc::abi::launch_status(err, fn);
}

}  // extern "C"

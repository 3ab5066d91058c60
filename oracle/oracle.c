/*
 * Reference oracle for exact softmax attention and log-sum-exp merging.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously-correct CPU
 * definition that the GPU kernels are checked against.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product library never links, calls or falls back to it, and it shares no
 * source, header, table or helper with the GPU path.
 *
 * What is computed (paper, Sec. 3.5 "Multi-GPU unified sequence parallelism"):
 *   under Ulysses every GPU attends over all tokens of the window for its own
 *   subset of heads; under Ring key/value blocks travel between GPUs and their
 *   partial results are folded together with running-max rescaling; either
 *   way the result is single-device attention, apart from the order of the
 *   floating-point reductions.  The plain definition of it, per batch b,
 *   head h and query row i, with the caller's float32 scale widened to double:
 *
 *       s_j  = scale * sum_t Q[b,i,h,t] * K[b,j,h,t]          j = 0..Skv-1
 *       m    = max_j s_j
 *       l    = sum_j exp(s_j - m)
 *       O[b,i,h,:]  = sum_j exp(s_j - m) * V[b,j,h,:] / l
 *       LSE[b,h,i]  = m + log(l)                     (natural log)
 *
 *   This is written as two passes over each row (all scores first, then the
 *   max, the sum and the weighted sum): deliberately NOT the blockwise online
 *   recurrence the kernels use.  A key/value chunk's partial result is the same
 *   function applied to that chunk's rows.
 *
 *   Merging n partial results (O_c, L_c) of disjoint key chunks back into the
 *   result over their union is the log-sum-exp identity:
 *       m* = max_c L_c,   L = m* + log sum_c exp(L_c - m*),
 *       O  = sum_c exp(L_c - L) * O_c.
 *   A part with L_c = -inf carries no keys and weight 0; if every part has
 *   L_c = -inf the merged row is O = 0, L = -inf.
 *
 * Inputs are bf16 bit patterns (uint16), widened exactly to double.  Tensors
 * are logical [B, S, H, D] with element strides for b, s and h, and D
 * contiguous.  Outputs are double: O [B, Sq, H, D] contiguous, LSE [B, H, Sq].
 * Rounding: every product and sum is done in double precision.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double bf16_to_double(uint16_t bits)
{
    /* a bf16 value is the top half of the float32 with the same bits */
    uint32_t u = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Exact attention over all Skv keys; returns 0 on success, -1 on bad sizes
 * or allocation failure. */
int oracle_attn(const uint16_t *q, int64_t q_sb, int64_t q_ss, int64_t q_sh,
                const uint16_t *k, int64_t k_sb, int64_t k_ss, int64_t k_sh,
                const uint16_t *v, int64_t v_sb, int64_t v_ss, int64_t v_sh,
                double *o, double *lse,
                int B, int H, int Sq, int Skv, int D, float scale_f32)
{
    if (B < 0 || H < 0 || Sq < 0 || Skv < 1 || D < 1)
        return -1;
    const double scale = (double)scale_f32;
    int failed = 0;

#pragma omp parallel
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)Skv);
        double *acc = (double *)malloc(sizeof(double) * (size_t)D);
        if (!s || !acc) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for collapse(3) schedule(dynamic, 4)
        for (int b = 0; b < B; b++)
            for (int h = 0; h < H; h++)
                for (int i = 0; i < Sq; i++) {
                    if (!s || !acc)
                        continue;
                    const uint16_t *qi = q + b * q_sb + i * q_ss + h * q_sh;
                    /* pass 1: every scaled score of the row */
                    for (int j = 0; j < Skv; j++) {
                        const uint16_t *kj = k + b * k_sb + j * k_ss + h * k_sh;
                        double dot = 0.0;
                        for (int t = 0; t < D; t++)
                            dot += bf16_to_double(qi[t]) * bf16_to_double(kj[t]);
                        s[j] = scale * dot;
                    }
                    /* pass 2: max, normaliser and weighted sum of value rows */
                    double m = -INFINITY;
                    for (int j = 0; j < Skv; j++)
                        if (s[j] > m)
                            m = s[j];
                    double l = 0.0;
                    for (int t = 0; t < D; t++)
                        acc[t] = 0.0;
                    for (int j = 0; j < Skv; j++) {
                        const double p = exp(s[j] - m);
                        const uint16_t *vj = v + b * v_sb + j * v_ss + h * v_sh;
                        l += p;
                        for (int t = 0; t < D; t++)
                            acc[t] += p * bf16_to_double(vj[t]);
                    }
                    double *oi = o + (((int64_t)b * Sq + i) * H + h) * D;
                    for (int t = 0; t < D; t++)
                        oi[t] = acc[t] / l;
                    lse[((int64_t)b * H + h) * Sq + i] = m + log(l);
                }
        free(s);
        free(acc);
    }
    return failed ? -1 : 0;
}

/* Log-sum-exp merge of num_parts partial results of disjoint key chunks.
 * o_parts[c]: [B, Sq, H, D] contiguous; lse_parts[c]: [B, H, Sq]. */
int oracle_merge(const double *const *o_parts, const double *const *lse_parts,
                 int num_parts, double *o, double *lse,
                 int B, int H, int Sq, int D)
{
    if (num_parts < 1 || B < 0 || H < 0 || Sq < 0 || D < 1)
        return -1;
#pragma omp parallel for collapse(3) schedule(static)
    for (int b = 0; b < B; b++)
        for (int h = 0; h < H; h++)
            for (int i = 0; i < Sq; i++) {
                const int64_t li = ((int64_t)b * H + h) * Sq + i;
                const int64_t oi = (((int64_t)b * Sq + i) * H + h) * D;
                double mstar = -INFINITY;
                for (int c = 0; c < num_parts; c++)
                    if (lse_parts[c][li] > mstar)
                        mstar = lse_parts[c][li];
                if (mstar == -INFINITY) {
                    /* no part holds any key: the empty-set result */
                    for (int t = 0; t < D; t++)
                        o[oi + t] = 0.0;
                    lse[li] = -INFINITY;
                    continue;
                }
                double sum = 0.0;
                for (int c = 0; c < num_parts; c++)
                    sum += exp(lse_parts[c][li] - mstar);
                const double L = mstar + log(sum);
                for (int t = 0; t < D; t++) {
                    double acc = 0.0;
                    for (int c = 0; c < num_parts; c++) {
                        const double w = exp(lse_parts[c][li] - L);
                        acc += w * o_parts[c][oi + t];
                    }
                    o[oi + t] = acc;
                }
                lse[li] = L;
            }
    return 0;
}

/* Sets the number of OpenMP threads of later oracle calls (n >= 1); used to
 * time the oracle on one host core as well as on all of them. */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n >= 1)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Number of OpenMP threads the oracle runs on (reported next to its timing). */
int oracle_num_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}

/*
 * q/k RMSNorm + 3D rotary position embedding: the steps between the QKV
 * projection and self-attention in a block of the video diffusion
 * transformer (the backbone of Sec. 3.4; the block shape -- RMSNorm on q and
 * k, rotary embedding split over frame / row / column -- is the workload's
 * configuration, the paper does not print it).  Per batch b and token t, with
 * x the C = H*D values of the token (all heads) and w the C norm weights:
 *
 *     r   = 1 / sqrt(sum_c x_c^2 / C + eps)
 *     y_c = x_c * r * w_c
 *
 * then per head, on pairs (y_2i, y_2i+1), i = 0..D/2-1, a rotation by
 *
 *     angle_i = pos_a * theta^(-2 k / d_a)
 *
 * where pair i belongs to axis a = frame for i < Pf, row for Pf <= i < Pf+Ph,
 * column otherwise, k is its index within that axis, d_a = 2 * (pairs of the
 * axis), Ph = Pw = D/6 (integer division) and Pf = D/2 - Ph - Pw (22/21/21
 * pairs, 44/42/42 dims, at D = 128); the token's global index g = token0 + t
 * in (frame, row, column) raster order over a grid_f x grid_h x grid_w
 * latent grid gives pos_frame = g / (grid_h grid_w),
 * pos_row = (g / grid_w) % grid_h, pos_col = g % grid_w:
 *
 *     (y_2i, y_2i+1) -> (y_2i cos a - y_2i+1 sin a,  y_2i sin a + y_2i+1 cos a)
 *
 * This is the rotary embedding of RoFormer (rotation of coordinate pairs by
 * position times a geometric frequency), applied per axis.  eps and theta are
 * the caller's float32 values widened to double; all arithmetic in double.
 * x: bf16 [B, S, H, D] with element strides; w: bf16 [H*D]; y: double
 * [B, S, H, D] contiguous.  Returns 0, or -1 on bad sizes.
 */
int oracle_norm_rope(const uint16_t *x, int64_t x_sb, int64_t x_ss, int64_t x_sh, const uint16_t *w,
                     double *y, int B, int S, int H, int D, int grid_f, int grid_h, int grid_w, int token0,
                     float eps_f32, float theta_f32)
{
    if (B < 0 || S < 0 || H < 1 || D < 6 || D % 2 != 0 || grid_f < 1 || grid_h < 1 || grid_w < 1 ||
        token0 < 0 || (int64_t)token0 + S > (int64_t)grid_f * grid_h * grid_w)
        return -1;
    const double eps = (double)eps_f32, theta = (double)theta_f32;
    const int C = H * D, P = D / 2;
    const int ph = D / 6, pw = D / 6, pf = P - ph - pw;
#pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b)
        for (int t = 0; t < S; ++t) {
            double ss = 0.0;
            for (int h = 0; h < H; ++h)
                for (int d = 0; d < D; ++d) {
                    const double xv = bf16_to_double(x[b * x_sb + t * x_ss + h * x_sh + d]);
                    ss += xv * xv;
                }
            const double r = 1.0 / sqrt(ss / C + eps);
            const int64_t g = (int64_t)token0 + t;
            const double pos[3] = {(double)(g / ((int64_t)grid_h * grid_w)), (double)((g / grid_w) % grid_h),
                                   (double)(g % grid_w)};
            for (int h = 0; h < H; ++h) {
                double *yr = y + (((int64_t)b * S + t) * H + h) * D;
                for (int d = 0; d < D; ++d)
                    yr[d] = bf16_to_double(x[b * x_sb + t * x_ss + h * x_sh + d]) * r *
                            bf16_to_double(w[h * D + d]);
                for (int i = 0; i < P; ++i) {
                    int axis, kk, pairs;
                    if (i < pf) {
                        axis = 0, kk = i, pairs = pf;
                    } else if (i < pf + ph) {
                        axis = 1, kk = i - pf, pairs = ph;
                    } else {
                        axis = 2, kk = i - pf - ph, pairs = pw;
                    }
                    const double ang = pos[axis] * pow(theta, -2.0 * kk / (2.0 * pairs));
                    const double c = cos(ang), sn = sin(ang);
                    const double a0 = yr[2 * i], a1 = yr[2 * i + 1];
                    yr[2 * i] = a0 * c - a1 * sn;
                    yr[2 * i + 1] = a0 * sn + a1 * c;
                }
            }
        }
    return 0;
}

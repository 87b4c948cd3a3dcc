/*
 * oracle.c -- plain, slow, obviously correct CPU reference for the fused
 * BitLinear forward of "Scalable MatMul-free Language Modeling"
 * (arXiv 2406.02528).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no source with the HIP library: it has
 * its own packer, its own decoder and its own arithmetic.
 *
 * What is computed, and where the paper defines it:
 *   weight quantisation  -- Algorithm 1, function weight_quant: scale by the
 *                           reciprocal of mean|W| over the whole tensor, round,
 *                           clip to [-1, 1].
 *   RMSNorm              -- Sec. "Implementation Details on Intel Loihi 2",
 *                           RMSNorm equation (learned scale w, eps = 1e-6),
 *                           read with the mean of squares as in the
 *                           "Double RMSNorm Derivation" appendix.
 *   activation quant     -- Algorithm 1, function activation_quant: scale by
 *                           127 / max|X| per token, round, clip to [-128, 127].
 *   ternary accumulation -- Sec. "MatMul-free Dense Layers with Ternary
 *                           Weights": each output is the sum of the inputs whose
 *                           weight is +1 minus the sum of those whose weight is
 *                           -1; a zero weight contributes nothing.
 *   dequantisation       -- Algorithm 1: the quantisers return the rounded value
 *                           times 1/s, so the product of two fake-quantised
 *                           operands is the integer sum times (1/s_a)(1/s_w).
 *   GLU gate             -- Sec. "MatMul-free Channel Mixer": SiLU(g) * u.
 *   MLGRU                -- Sec. "MatMul-free Language Model Architecture",
 *                           MLGRU equations: forget/candidate/output gate
 *                           activations, the recurrence over time and the
 *                           output gate o' = g * sigma(h); bias of a layer.
 *   backward             -- Algorithm 1, backward_pass and rms_norm_bwd, with
 *                           the straight-through estimator of Sec.
 *                           "Surrogate Gradient".
 *
 * Precision.  The paper fixes none.  Where a floating-point value decides an
 * integer (the ternary code, the int8 activation) the oracle takes that
 * decision in the same precision as the GPU kernels: sums of squares and of
 * |W| in fp64, everything after in fp32 with round-half-to-even.  Everything
 * that does not decide an integer (the dequantised output) is computed in
 * fp64 and rounded to fp32 once at the end.
 *
 * Conventions: row-major arrays; x is [M][K] (tokens x in-features); the
 * latent weight W is [N][K] (out-features x in-features); ternary codes t are
 * int8 in {-1, 0, +1}, [N][K].
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Number of OpenMP threads the parallel loops below use (1 without OpenMP). */
int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_num_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Round half to even in fp32 (the rounding the paper writes as a bracketed
 * round; read as IEEE round-to-nearest-even, the default rounding mode). */
static float round_half_even_f32(float v) {
    float r = nearbyintf(v);   /* honours the current mode: nearest-even */
    return r;
}

/* ---------------------------------------------------------------------- */
/* weight_quant (Algorithm 1): W -> t in {-1,0,1}, w_scale = mean|W|.     */
/* Returns 0.                                                              */
/* ---------------------------------------------------------------------- */
int oracle_weight_quant(const float *W, int64_t N, int64_t K, int8_t *t,
                        float *w_scale) {
    /* mean(|W|) over the whole tensor, summed sequentially in fp64 */
    double sum_abs = 0.0;
    int64_t count = N * K;
    for (int64_t i = 0; i < count; ++i) sum_abs += fabs((double)W[i]);
    double mean_abs = count > 0 ? sum_abs / (double)count : 0.0;

    /* the stored statistic, kept away from zero so s = 1/mean is finite */
    float mean_f = (float)mean_abs;
    if (mean_f < 1e-5f) mean_f = 1e-5f;
    float s = 1.0f / mean_f;

    for (int64_t i = 0; i < count; ++i) {
        float v = round_half_even_f32(W[i] * s);
        if (v > 1.0f) v = 1.0f;
        if (v < -1.0f) v = -1.0f;
        t[i] = (int8_t)v;
    }
    *w_scale = mean_f;   /* the dequantisation multiplier 1/s */
    return 0;
}

/* ---------------------------------------------------------------------- */
/* 2-bit packing of ternary codes, the library's storage format.          */
/*   Wpacked has K/16 rows of N uint32 words; word (j, n) is Wpacked[j*N+n]*/
/*   and holds the 16 weights t[n][16j .. 16j+15].                         */
/*   For k = 16j + 4i + b (i, b in 0..3) the code c = t + 1 in {0,1,2}     */
/*   occupies bits 8b + 2i and 8b + 2i + 1.  Code 3 is invalid.            */
/* ---------------------------------------------------------------------- */
static int packed_bit_position(int kk /* 0..15 */) {
    int i = kk / 4, b = kk % 4;
    return 8 * b + 2 * i;
}

/* Returns 0, or -1 if K is not a multiple of 16 or a code is out of range. */
int oracle_pack(const int8_t *t, int64_t N, int64_t K, uint32_t *Wpacked) {
    if (K % 16 != 0) return -1;
    int64_t J = K / 16;
    for (int64_t j = 0; j < J; ++j) {
        for (int64_t n = 0; n < N; ++n) {
            uint32_t word = 0;
            for (int kk = 0; kk < 16; ++kk) {
                int tv = t[n * K + 16 * j + kk];
                if (tv < -1 || tv > 1) return -1;
                uint32_t code = (uint32_t)(tv + 1);
                word |= code << packed_bit_position(kk);
            }
            Wpacked[j * N + n] = word;
        }
    }
    return 0;
}

/* Returns the number of invalid (== 3) codes met; those decode to 0. */
int64_t oracle_unpack(const uint32_t *Wpacked, int64_t N, int64_t K, int8_t *t) {
    if (K % 16 != 0) return -1;
    int64_t J = K / 16, bad = 0;
    for (int64_t j = 0; j < J; ++j) {
        for (int64_t n = 0; n < N; ++n) {
            uint32_t word = Wpacked[j * N + n];
            for (int kk = 0; kk < 16; ++kk) {
                uint32_t code = (word >> packed_bit_position(kk)) & 3u;
                int tv;
                if (code == 3u) { ++bad; tv = 0; }
                else tv = (int)code - 1;
                t[n * K + 16 * j + kk] = (int8_t)tv;
            }
        }
    }
    return bad;
}

/* ---------------------------------------------------------------------- */
/* RMSNorm: r_m = 1 / sqrt(mean_k x_mk^2 + eps); y_mk = (x_mk r_m) gamma_k */
/* gamma may be NULL (all ones).  r (length M) may be NULL.                */
/* ---------------------------------------------------------------------- */
void oracle_rms_norm(const float *x, const float *gamma, int64_t M, int64_t K,
                     double eps, float *y, float *r_out) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        const float *xr = x + m * K;
        double ss = 0.0;                       /* sequential fp64 sum */
        for (int64_t k = 0; k < K; ++k) ss += (double)xr[k] * (double)xr[k];
        double ms = K > 0 ? ss / (double)K : 0.0;
        float r = (float)(1.0 / sqrt(ms + eps));
        if (r_out) r_out[m] = r;
        for (int64_t k = 0; k < K; ++k) {
            float v = xr[k] * r;
            if (gamma) v = v * gamma[k];
            y[m * K + k] = v;
        }
    }
}

/* ---------------------------------------------------------------------- */
/* activation_quant (Algorithm 1), one scale per token (row):             */
/*   a = max_k |y_k| (floored at 1e-5), s = 127 / a,                       */
/*   q_k = clamp(round(s y_k), -128, 127), a_scale = a / 127 (= 1/s).      */
/* ---------------------------------------------------------------------- */
void oracle_act_quant(const float *y, int64_t M, int64_t K, int8_t *q,
                      float *a_scale) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        const float *yr = y + m * K;
        float amax = 0.0f;
        for (int64_t k = 0; k < K; ++k) {
            float a = fabsf(yr[k]);
            if (a > amax) amax = a;
        }
        if (amax < 1e-5f) amax = 1e-5f;
        float s = 127.0f / amax;
        for (int64_t k = 0; k < K; ++k) {
            float v = round_half_even_f32(yr[k] * s);
            if (v > 127.0f) v = 127.0f;
            if (v < -128.0f) v = -128.0f;
            q[m * K + k] = (int8_t)v;
        }
        a_scale[m] = amax / 127.0f;
    }
}

/* ---------------------------------------------------------------------- */
/* Ternary accumulation: acc[m][n] = sum_{k: t=+1} q - sum_{k: t=-1} q.    */
/* Written as the case analysis of the paper: add, skip or subtract.       */
/* Returns 0, or -1 if a sum does not fit int32 or a code is not ternary.  */
/* ---------------------------------------------------------------------- */
int oracle_ternary_accumulate(const int8_t *q, const int8_t *t, int64_t M,
                              int64_t K, int64_t N, int32_t *acc) {
    int status = 0;
#pragma omp parallel for collapse(2) schedule(static) reduction(min : status)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            const int8_t *qr = q + m * K;
            const int8_t *tr = t + n * K;
            int64_t plus = 0, minus = 0;
            for (int64_t k = 0; k < K; ++k) {
                if (tr[k] == 1) plus += qr[k];
                else if (tr[k] == -1) minus += qr[k];
                else if (tr[k] != 0) status = -1;
            }
            int64_t v = plus - minus;
            if (v > INT32_MAX || v < INT32_MIN) status = -1;
            acc[m * N + n] = (int32_t)v;
        }
    }
    return status;
}

/* Same sum for an explicit list of (m, n) pairs; out[p] for pair p. */
int oracle_ternary_accumulate_pairs(const int8_t *q, const int8_t *t,
                                    int64_t K, const int64_t *ms,
                                    const int64_t *ns, int64_t P,
                                    int32_t *out) {
    int status = 0;
#pragma omp parallel for schedule(static) reduction(min : status)
    for (int64_t p = 0; p < P; ++p) {
        const int8_t *qr = q + ms[p] * K;
        const int8_t *tr = t + ns[p] * K;
        int64_t plus = 0, minus = 0;
        for (int64_t k = 0; k < K; ++k) {
            if (tr[k] == 1) plus += qr[k];
            else if (tr[k] == -1) minus += qr[k];
            else if (tr[k] != 0) status = -1;
        }
        int64_t v = plus - minus;
        if (v > INT32_MAX || v < INT32_MIN) status = -1;
        out[p] = (int32_t)v;
    }
    return status;
}

/* ---------------------------------------------------------------------- */
/* Dequantisation: y[m][n] = acc[m][n] * (1/s_a,m) * (1/s_w), in fp64,     */
/* rounded once to fp32.                                                    */
/* ---------------------------------------------------------------------- */
void oracle_dequant(const int32_t *acc, const float *a_scale, float w_scale,
                    int64_t M, int64_t N, float *y) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n)
            y[m * N + n] = (float)((double)acc[m * N + n] * (double)a_scale[m] *
                                   (double)w_scale);
}

/* ---------------------------------------------------------------------- */
/* The whole forward: RMSNorm -> act quant -> ternary accumulation ->     */
/* dequant, with the ternary codes t and w_scale from oracle_weight_quant. */
/* Scratch: ybuf float[M*K], q int8[M*K], a_scale float[M], acc int32[M*N] */
/* supplied by the caller so that the oracle allocates nothing.            */
/* ---------------------------------------------------------------------- */
int oracle_bitlinear_fwd(const float *x, const float *gamma, const int8_t *t,
                         float w_scale, int64_t M, int64_t K, int64_t N,
                         double eps, float *ybuf, int8_t *q, float *a_scale,
                         int32_t *acc, float *y) {
    oracle_rms_norm(x, gamma, M, K, eps, ybuf, NULL);
    oracle_act_quant(ybuf, M, K, q, a_scale);
    int st = oracle_ternary_accumulate(q, t, M, K, N, acc);
    oracle_dequant(acc, a_scale, w_scale, M, N, y);
    return st;
}

/* ---------------------------------------------------------------------- */
/* GLU channel-mixer gate (Sec. "MatMul-free Channel Mixer"): the gated   */
/* representation is p = tau(g) (.) u, with g and u the outputs of the two */
/* up-projections and tau the SiLU activation, tau(v) = v / (1 + e^-v).    */
/* Evaluated in fp64 from the fp32 inputs and rounded to fp32 once.        */
/* ---------------------------------------------------------------------- */
void oracle_glu(const float *g, const float *u, int64_t n, float *p) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const double gv = (double)g[i];
        const double silu = gv / (1.0 + exp(-gv));
        p[i] = (float)(silu * (double)u[i]);
    }
}

/* ---------------------------------------------------------------------- */
/* MLGRU gate activations (Sec. "MatMul-free Language Model Architecture", */
/* paragraph "MatMul-free Linear Gated Recurrent Unit").  z is [M][3d]: the */
/* three ternary projections of a token side by side, forget gate columns  */
/* [0, d), candidate [d, 2d), output gate [2d, 3d).  With the biases b     */
/* ([3d], NULL => 0) and the forget-gate lower bound lb ([d], NULL => 0):  */
/*   f = lb + (1 - lb) sigma(z_f + b_f)                                   */
/*   c = SiLU(z_c + b_c) = v / (1 + e^-v)                                 */
/*   g = z_g + b_g                                                        */
/* The lower bound is the form of HGRN that the paper's cummax remark      */
/* refers to (a per-layer vector in [0, 1) raising the forget gate towards */
/* 1 in deeper layers); lb = 0 is the equations as printed.  Each value is */
/* evaluated in fp64 from the fp32 inputs and rounded to fp32 once.        */
/* ---------------------------------------------------------------------- */
void oracle_mlgru_gates(const float *z, const float *bias, const float *lb,
                        int64_t M, int64_t d, float *fcg) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        const float *zr = z + m * 3 * d;
        float *o = fcg + m * 3 * d;
        for (int64_t i = 0; i < d; ++i) {
            const double vf = (double)zr[i] + (bias ? (double)bias[i] : 0.0);
            const double vc = (double)zr[d + i] + (bias ? (double)bias[d + i] : 0.0);
            const double vg = (double)zr[2 * d + i] + (bias ? (double)bias[2 * d + i] : 0.0);
            const double low = lb ? (double)lb[i] : 0.0;
            o[i] = (float)(low + (1.0 - low) / (1.0 + exp(-vf)));
            o[d + i] = (float)(vc / (1.0 + exp(-vc)));
            o[2 * d + i] = (float)vg;
        }
    }
}

/* ---------------------------------------------------------------------- */
/* MLGRU recurrence and output gate (same paragraph): for each of B        */
/* sequences of T tokens (rows b*T + t of fcg, laid out as above)          */
/*   h_t  = f_t (.) h_{t-1} + (1 - f_t) (.) c_t,   h_0 = h0 (NULL => 0)    */
/*   o'_t = g_t (.) sigma(h_t)                                            */
/* taken one step after the other in token order, the state carried in     */
/* fp64.  o' [B*T][d] is rounded to fp32 once per value; h_last [B][d]     */
/* (may be NULL) receives the state after the last token, rounded.        */
/* ---------------------------------------------------------------------- */
void oracle_mlgru_scan(const float *fcg, const float *h0, int64_t B, int64_t T,
                       int64_t d, float *o, float *h_last) {
#pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t i = 0; i < d; ++i) {
            double h = h0 ? (double)h0[b * d + i] : 0.0;
            for (int64_t t = 0; t < T; ++t) {
                const float *row = fcg + (b * T + t) * 3 * d;
                const double f = (double)row[i];
                const double c = (double)row[d + i];
                const double g = (double)row[2 * d + i];
                h = f * h + (1.0 - f) * c;
                o[(b * T + t) * d + i] = (float)(g / (1.0 + exp(-h)));
            }
            if (h_last) h_last[b * d + i] = (float)h;
        }
    }
}

/* ---------------------------------------------------------------------- */
/* Bias of a dense layer (Algorithm 1, forward_pass: the ternary product   */
/* plus b): y [M][N] fp32 outputs of the dequantised product, b [N];       */
/* out = y + b in fp64, rounded once.                                      */
/* ---------------------------------------------------------------------- */
void oracle_add_bias(const float *y, const float *b, int64_t M, int64_t N, float *out) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n)
            out[m * N + n] = (float)((double)y[m * N + n] + (double)b[n]);
}

/* ---------------------------------------------------------------------- */
/* bfloat16 storage of a float: round to nearest, ties to even, on the     */
/* top 16 bits (the 16-bit activations the training path stores).         */
/* ---------------------------------------------------------------------- */
static float round_to_bf16(float v) {
    uint32_t b;
    memcpy(&b, &v, 4);
    const uint32_t lsb = (b >> 16) & 1u;
    b = (b + 0x7FFFu + lsb) & 0xFFFF0000u;
    float out;
    memcpy(&out, &b, 4);
    return out;
}

/* ---------------------------------------------------------------------- */
/* Backward of the BitLinear (Algorithm 1, backward_pass and rms_norm_bwd; */
/* Sec. "Surrogate Gradient": the straight-through estimator passes the    */
/* gradient through both quantisers unchanged).  In the RMSNorm reading    */
/* (no mean subtracted, so the mean term of rms_norm_bwd vanishes) with    */
/* the learned scale applied after the normalisation, y = (x r) gamma:     */
/*   dY  = dO x Wt^T            Wt = t * w_scale, the forward's weights    */
/*   g   = gamma (.) dY,  s = sum_k g_k x_k                                */
/*   dX  = r g - (r^3 / K) x s                                             */
/*   dW  = dO^T x Yq            Yq = q * a_scale stored as bfloat16        */
/*   db  = sum over tokens of dO;  dgamma = sum over tokens of dY x r      */
/* dO [M][N] holds the values of the bf16 output gradient; r [M] is the    */
/* forward's fp32 rstd.  Sums in fp64, each output rounded to fp32 once;   */
/* Yq is rounded to bf16 from the fp32 product q * a_scale, as stored.     */
/* Scratch: dY double[M*K], yq float[M*K] supplied by the caller.          */
/* ---------------------------------------------------------------------- */
void oracle_bitlinear_bwd(const float *dO, const float *x, const float *gamma,
                          const float *r, const int8_t *q, const float *a_scale,
                          const int8_t *t, float w_scale, int64_t M, int64_t K,
                          int64_t N, double *dY, float *yq, float *dx, float *dW,
                          float *db, float *dgamma) {
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int64_t n = 0; n < N; ++n)
                acc += (double)dO[m * N + n] * (double)t[n * K + k];
            dY[m * K + k] = acc * (double)w_scale;
        }
        const double rm = (double)r[m];
        double s = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double gk = gamma ? (double)gamma[k] : 1.0;
            s += gk * dY[m * K + k] * (double)x[m * K + k];
        }
        for (int64_t k = 0; k < K; ++k) {
            const double gk = gamma ? (double)gamma[k] : 1.0;
            dx[m * K + k] = (float)(rm * gk * dY[m * K + k] -
                                    rm * rm * rm / (double)K * (double)x[m * K + k] * s);
            yq[m * K + k] = round_to_bf16((float)q[m * K + k] * a_scale[m]);
        }
    }
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int64_t m = 0; m < M; ++m) acc += (double)dO[m * N + n] * (double)yq[m * K + k];
            dW[n * K + k] = (float)acc;
        }
        if (db) {
            double acc = 0.0;
            for (int64_t m = 0; m < M; ++m) acc += (double)dO[m * N + n];
            db[n] = (float)acc;
        }
    }
    if (dgamma) {
#pragma omp parallel for schedule(static)
        for (int64_t k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int64_t m = 0; m < M; ++m)
                acc += dY[m * K + k] * (double)x[m * K + k] * (double)r[m];
            dgamma[k] = (float)acc;
        }
    }
}

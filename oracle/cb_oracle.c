/*
 * cb_oracle.c -- plain fp64 CPU oracle for the CacheBridge mapper path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the reference that the GPU library is
 * checked against.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it; the product library never links, includes or
 * calls anything here, and this file includes nothing from the product.
 *
 * What it computes (CacheBridge, "Efficient Cross-Model KV Cache Transfer"):
 *
 *   Head-local feature (Sec. 3.2, Eq. localfeature, one selected source layer):
 *     the map for target (layer l, head h, component z in {K,V}) reads the
 *     source row Z^S[src_layer, z, seq, src_head, t] (width d_s) and the
 *     target row Z^T[l, z, seq, h, t] (width d_t).
 *
 *   Sufficient statistics (Sec. 3.4, Eq. fusedstats, in augmented form):
 *     x~ = [x ; 1] (width P = d_s + 1), w = weights[weight_row][token],
 *       G += sum_t w x~ x~^T        (P x P)
 *       C += sum_t w x~ y^T         (P x d_t)
 *     The centered A_h, B_h and the weighted means of the paper are all
 *     contained in G and C (the last row/column holds sum w, sum w x, sum w y).
 *
 *   Ridge solve (Sec. 3.1 Eq. closedform; Sec. 3.4 solver):
 *     M = G + lambda_m * D,  W~ = M^{-1} C   (fp64 Cholesky)
 *     D = I (bias penalized)  or  diag(1,..,1,0) (bias not penalized, which is
 *     exactly the centered weighted ridge of Eq. closedform by a Schur
 *     complement on the bias row).  lambda_m = lambda * tr(G)/P when relative.
 *     Rows 0..d_s-1 of W~ are W, row d_s is the bias b^T.
 *
 *   Online application (Sec. 1 pipeline; Sec. 2.3 Eq. support-cost):
 *     out[l, z, seq, h, t, :] = RNE_bf16( x~ W~ ) with the sum taken in fp64 and
 *     rounded once, to nearest with ties to even, to bfloat16.
 *
 *   Multi-layer feature (Sec. 3.2, Eq. localfeature with k selected source
 *   layers): x~ = [x_0 ; ... ; x_{k-1} ; 1], P = k d_s + 1, over the sampled
 *   calibration rows (oracle_stats_multi, oracle_apply_multi); the solve above
 *   takes any P.  Its two-pass centered form (oracle_stats_multi_centered)
 *   feeds oracle_ridge_solve_centered with the feature width k d_s.
 *
 * Parity status: stats, solve and apply are pinned by the tests in
 * tests/test_oracle_pins.py (closed forms, invariants, library special cases,
 * brute-force minimality of the paper's objective).  No worked numerical
 * example exists in the paper, so no value of the paper itself pins them.
 *
 * Everything is plain loops in fp64, parallel over maps only (OpenMP), with no
 * blocking or reordering beyond the definitions above.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* bfloat16 bits -> double (exact: bf16 is the top half of an IEEE binary32). */
static double bf16_bits_to_double(uint16_t b) {
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * double -> bfloat16 bits, rounded once to nearest with ties to even.
 * bfloat16 carries 8 significant bits and the binary32 exponent range
 * (normals from 2^-126, subnormal quantum 2^-133, largest finite
 * (2 - 2^-7) * 2^127).  The value is scaled by a power of two so that the
 * retained bits become an integer, rounded with nearbyint (round-half-even in
 * the default floating-point environment), and scaled back; both scalings are
 * exact.  The result is representable in binary32, whose top 16 bits are the
 * bfloat16 encoding.
 */
uint16_t oracle_double_to_bf16(double v) {
    if (isnan(v)) return (uint16_t)0x7FC0u;
    if (isinf(v)) return v > 0 ? (uint16_t)0x7F80u : (uint16_t)0xFF80u;
    if (v == 0.0) return signbit(v) ? (uint16_t)0x8000u : (uint16_t)0x0000u;
    double a = fabs(v);
    int e;
    (void)frexp(a, &e);            /* a = m * 2^e, m in [0.5, 1): leading bit is 2^(e-1) */
    int q = e - 8;                 /* weight of the 8th significant bit */
    if (q < -133) q = -133;        /* below the normal range the quantum is fixed */
    double r = ldexp(nearbyint(ldexp(a, -q)), q);
    const double bf16_max = ldexp(255.0, 120);   /* (2 - 2^-7) * 2^127 */
    uint16_t bits;
    if (r > bf16_max) {
        bits = 0x7F80u;            /* rounds past the largest finite value */
    } else {
        float f = (float)r;        /* exact */
        uint32_t u;
        memcpy(&u, &f, sizeof u);
        bits = (uint16_t)(u >> 16);
    }
    return signbit(v) ? (uint16_t)(bits | 0x8000u) : bits;
}

/* Element offset of row (layer, kv, seq, head, tok) in a strided cache view. */
static int64_t row_offset(const int64_t *s, int layer, int kv, int seq, int head, int tok) {
    return (int64_t)layer * s[0] + (int64_t)kv * s[1] + (int64_t)seq * s[2] +
           (int64_t)head * s[3] + (int64_t)tok * s[4];
}

static void set_threads(int n_threads) {
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
}

/*
 * Weighted augmented moments, accumulated into G [n_maps][P][P] and
 * C [n_maps][P][d_t] (both fp64, row-major, P = d_s + 1).
 *   src/tgt: bf16 bits, strides {layer, kv, seq, head, tok} in elements,
 *            channel stride 1.
 *   weights: fp32, weights[row * w_row_stride + seq * seq_len + tok].
 * Every token of every sequence is visited.  Returns 0.
 */
int oracle_stats(int n_maps,
                 const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                 const int32_t *src_layer, const int32_t *src_head, const int32_t *weight_row,
                 const uint16_t *src, const int64_t *src_strides, int d_s,
                 const uint16_t *tgt, const int64_t *tgt_strides, int d_t,
                 const float *weights, int64_t w_row_stride,
                 int n_seqs, int seq_len,
                 double *G, double *C, int n_threads) {
    const int P = d_s + 1;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        double *Gm = G + (int64_t)m * P * P;
        double *Cm = C + (int64_t)m * P * d_t;
        double *xt = (double *)malloc(sizeof(double) * (size_t)P);
        double *y = (double *)malloc(sizeof(double) * (size_t)d_t);
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                const uint16_t *xr = src + row_offset(src_strides, src_layer[m], kv[m], b, src_head[m], t);
                const uint16_t *yr = tgt + row_offset(tgt_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                const double w = (double)weights[(int64_t)weight_row[m] * w_row_stride +
                                                 (int64_t)b * seq_len + t];
                for (int i = 0; i < d_s; ++i) xt[i] = bf16_bits_to_double(xr[i]);
                xt[d_s] = 1.0;
                for (int j = 0; j < d_t; ++j) y[j] = bf16_bits_to_double(yr[j]);
                for (int i = 0; i < P; ++i) {
                    const double wi = w * xt[i];
                    for (int j = 0; j < P; ++j) Gm[(int64_t)i * P + j] += wi * xt[j];
                    for (int j = 0; j < d_t; ++j) Cm[(int64_t)i * d_t + j] += wi * y[j];
                }
            }
        }
        free(xt);
        free(y);
    }
    return 0;
}

/*
 * Batched ridge solve in fp64.
 *   G [n_maps][P][P], C [n_maps][P][d_t]  ->  W [n_maps][P][d_t]
 *   lambda_relative != 0: lambda_m = lambda * trace(G_m) / P, else lambda.
 *   bias_unpenalized != 0: the ridge term is left off the last diagonal entry.
 * Cholesky M = L L^T (row by row), then L Z = C and L^T W = Z.
 * info[m] = 0 on success, else the 1-based index of the first pivot that is not
 * positive and finite; W_m is then zero-filled.  Returns 0.
 */
int oracle_ridge_solve(int n_maps, int P, int d_t, const double *G, const double *C,
                       double lambda, int lambda_relative, int bias_unpenalized,
                       double *W, int32_t *info, int n_threads) {
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        const double *Gm = G + (int64_t)m * P * P;
        const double *Cm = C + (int64_t)m * P * d_t;
        double *Wm = W + (int64_t)m * P * d_t;
        double *L = (double *)calloc((size_t)P * P, sizeof(double));
        double *Z = (double *)calloc((size_t)P * d_t, sizeof(double));
        double tr = 0.0;
        for (int i = 0; i < P; ++i) tr += Gm[(int64_t)i * P + i];
        const double lam = lambda_relative ? lambda * tr / (double)P : lambda;
        int bad = 0;
        for (int i = 0; i < P && !bad; ++i) {
            for (int j = 0; j <= i; ++j) {
                double s = Gm[(int64_t)i * P + j];
                if (i == j && !(bias_unpenalized && i == P - 1)) s += lam;
                for (int k = 0; k < j; ++k) s -= L[(int64_t)i * P + k] * L[(int64_t)j * P + k];
                if (i == j) {
                    if (!(s > 0.0) || !isfinite(s)) { bad = i + 1; break; }
                    L[(int64_t)i * P + i] = sqrt(s);
                } else {
                    L[(int64_t)i * P + j] = s / L[(int64_t)j * P + j];
                }
            }
        }
        info[m] = bad;
        if (bad) {
            memset(Wm, 0, sizeof(double) * (size_t)P * d_t);
        } else {
            for (int c = 0; c < d_t; ++c) {
                for (int i = 0; i < P; ++i) {          /* forward: L z = c */
                    double s = Cm[(int64_t)i * d_t + c];
                    for (int k = 0; k < i; ++k) s -= L[(int64_t)i * P + k] * Z[(int64_t)k * d_t + c];
                    Z[(int64_t)i * d_t + c] = s / L[(int64_t)i * P + i];
                }
                for (int i = P - 1; i >= 0; --i) {     /* backward: L^T w = z */
                    double s = Z[(int64_t)i * d_t + c];
                    for (int k = i + 1; k < P; ++k) s -= L[(int64_t)k * P + i] * Wm[(int64_t)k * d_t + c];
                    Wm[(int64_t)i * d_t + c] = s / L[(int64_t)i * P + i];
                }
            }
        }
        free(L);
        free(Z);
    }
    return 0;
}

/*
 * Two-pass centered statistics of Sec. 3.4 for every map: pass 1 accumulates
 * sum w, sum w x, sum w y over all tokens; pass 2 revisits the tokens and
 * accumulates A = sum w (x - mu_x)(x - mu_x)^T and B = sum w (x - mu_x)(y - mu_y)^T
 * with the means of pass 1.  Outputs (overwritten, fp64):
 *   sums [n_maps][1 + d_s + d_t] = (sum w, sum w x, sum w y),
 *   A [n_maps][d_s][d_s], B [n_maps][d_s][d_t].
 * A map whose weights sum to zero gets zero means.  Returns 0.
 */
int oracle_stats_centered(int n_maps,
                          const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                          const int32_t *src_layer, const int32_t *src_head, const int32_t *weight_row,
                          const uint16_t *src, const int64_t *src_strides, int d_s,
                          const uint16_t *tgt, const int64_t *tgt_strides, int d_t,
                          const float *weights, int64_t w_row_stride,
                          int n_seqs, int seq_len,
                          double *sums, double *A, double *B, int n_threads) {
    const int NS = 1 + d_s + d_t;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        double *sm = sums + (int64_t)m * NS;
        double *Am = A + (int64_t)m * d_s * d_s;
        double *Bm = B + (int64_t)m * d_s * d_t;
        double *x = (double *)malloc(sizeof(double) * (size_t)d_s);
        double *y = (double *)malloc(sizeof(double) * (size_t)d_t);
        memset(sm, 0, sizeof(double) * (size_t)NS);
        memset(Am, 0, sizeof(double) * (size_t)d_s * d_s);
        memset(Bm, 0, sizeof(double) * (size_t)d_s * d_t);
        /* pass 1: weighted sums */
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                const uint16_t *xr = src + row_offset(src_strides, src_layer[m], kv[m], b, src_head[m], t);
                const uint16_t *yr = tgt + row_offset(tgt_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                const double w = (double)weights[(int64_t)weight_row[m] * w_row_stride +
                                                 (int64_t)b * seq_len + t];
                sm[0] += w;
                for (int i = 0; i < d_s; ++i) sm[1 + i] += w * bf16_bits_to_double(xr[i]);
                for (int j = 0; j < d_t; ++j) sm[1 + d_s + j] += w * bf16_bits_to_double(yr[j]);
            }
        }
        const double sw = sm[0];
        /* pass 2: centered moments */
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                const uint16_t *xr = src + row_offset(src_strides, src_layer[m], kv[m], b, src_head[m], t);
                const uint16_t *yr = tgt + row_offset(tgt_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                const double w = (double)weights[(int64_t)weight_row[m] * w_row_stride +
                                                 (int64_t)b * seq_len + t];
                for (int i = 0; i < d_s; ++i)
                    x[i] = bf16_bits_to_double(xr[i]) - (sw != 0.0 ? sm[1 + i] / sw : 0.0);
                for (int j = 0; j < d_t; ++j)
                    y[j] = bf16_bits_to_double(yr[j]) - (sw != 0.0 ? sm[1 + d_s + j] / sw : 0.0);
                for (int i = 0; i < d_s; ++i) {
                    const double wi = w * x[i];
                    for (int j = 0; j < d_s; ++j) Am[(int64_t)i * d_s + j] += wi * x[j];
                    for (int j = 0; j < d_t; ++j) Bm[(int64_t)i * d_t + j] += wi * y[j];
                }
            }
        }
        free(x);
        free(y);
    }
    return 0;
}

/*
 * Centered ridge solve (Sec. 3.1, Eq. closedform) in fp64:
 *   W = (A + lambda_m I)^{-1} B  (Cholesky),  b = mu_y - W^T mu_x,
 * written as W~ [n_maps][d_s + 1][d_t] (rows 0..d_s-1 = W, row d_s = b^T).
 * lambda_m as in the file comment; info as in oracle_ridge_solve (first pivot of
 * A + lambda_m I that is not positive and finite, 1-based; W~ zero-filled).
 */
int oracle_ridge_solve_centered(int n_maps, int d_s, int d_t, const double *sums, const double *A,
                                const double *B, double lambda, int lambda_relative,
                                double *W, int32_t *info, int n_threads) {
    const int NS = 1 + d_s + d_t, P = d_s + 1;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        const double *sm = sums + (int64_t)m * NS;
        const double *Am = A + (int64_t)m * d_s * d_s;
        const double *Bm = B + (int64_t)m * d_s * d_t;
        double *Wm = W + (int64_t)m * P * d_t;
        double *L = (double *)calloc((size_t)d_s * d_s, sizeof(double));
        double *Z = (double *)calloc((size_t)d_s * d_t, sizeof(double));
        const double sw = sm[0];
        double tr = sw;
        for (int i = 0; i < d_s; ++i) {
            const double mu = sw != 0.0 ? sm[1 + i] / sw : 0.0;
            tr += Am[(int64_t)i * d_s + i] + sw * mu * mu;
        }
        const double lam = lambda_relative ? lambda * tr / (double)P : lambda;
        int bad = 0;
        for (int i = 0; i < d_s && !bad; ++i) {
            for (int j = 0; j <= i; ++j) {
                double s = Am[(int64_t)i * d_s + j];
                if (i == j) s += lam;
                for (int k = 0; k < j; ++k) s -= L[(int64_t)i * d_s + k] * L[(int64_t)j * d_s + k];
                if (i == j) {
                    if (!(s > 0.0) || !isfinite(s)) { bad = i + 1; break; }
                    L[(int64_t)i * d_s + i] = sqrt(s);
                } else {
                    L[(int64_t)i * d_s + j] = s / L[(int64_t)j * d_s + j];
                }
            }
        }
        info[m] = bad;
        if (bad) {
            memset(Wm, 0, sizeof(double) * (size_t)P * d_t);
        } else {
            for (int c = 0; c < d_t; ++c) {
                for (int i = 0; i < d_s; ++i) {
                    double s = Bm[(int64_t)i * d_t + c];
                    for (int k = 0; k < i; ++k) s -= L[(int64_t)i * d_s + k] * Z[(int64_t)k * d_t + c];
                    Z[(int64_t)i * d_t + c] = s / L[(int64_t)i * d_s + i];
                }
                for (int i = d_s - 1; i >= 0; --i) {
                    double s = Z[(int64_t)i * d_t + c];
                    for (int k = i + 1; k < d_s; ++k) s -= L[(int64_t)k * d_s + i] * Wm[(int64_t)k * d_t + c];
                    Wm[(int64_t)i * d_t + c] = s / L[(int64_t)i * d_s + i];
                }
                double bias = sw != 0.0 ? sm[1 + d_s + c] / sw : 0.0;
                for (int i = 0; i < d_s; ++i) bias -= Wm[(int64_t)i * d_t + c] * (sw != 0.0 ? sm[1 + i] / sw : 0.0);
                Wm[(int64_t)d_s * d_t + c] = bias;
            }
        }
        free(L);
        free(Z);
    }
    return 0;
}

/*
 * Weighted sums of squares per channel (the diagonal second moments that the
 * total sum of squares of a probe needs):
 *   sq [n_maps][d_s + d_t] = (sum w x_i^2 for i < d_s, sum w y_j^2 for j < d_t).
 * Same input conventions as oracle_stats.  Overwrites sq.  Returns 0.
 */
int oracle_weighted_squares(int n_maps,
                            const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                            const int32_t *src_layer, const int32_t *src_head, const int32_t *weight_row,
                            const uint16_t *src, const int64_t *src_strides, int d_s,
                            const uint16_t *tgt, const int64_t *tgt_strides, int d_t,
                            const float *weights, int64_t w_row_stride,
                            int n_seqs, int seq_len, double *sq, int n_threads) {
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        double *q = sq + (int64_t)m * (d_s + d_t);
        memset(q, 0, sizeof(double) * (size_t)(d_s + d_t));
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                const uint16_t *xr = src + row_offset(src_strides, src_layer[m], kv[m], b, src_head[m], t);
                const uint16_t *yr = tgt + row_offset(tgt_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                const double w = (double)weights[(int64_t)weight_row[m] * w_row_stride +
                                                 (int64_t)b * seq_len + t];
                for (int i = 0; i < d_s; ++i) {
                    const double v = bf16_bits_to_double(xr[i]);
                    q[i] += w * v * v;
                }
                for (int j = 0; j < d_t; ++j) {
                    const double v = bf16_bits_to_double(yr[j]);
                    q[d_s + j] += w * v * v;
                }
            }
        }
    }
    return 0;
}

/*
 * Held-in R^2 of fitted probes (Sec. 3.1, layer selection), from its
 * definition: with the map's weighted target mean mu_y,
 *   RSS = sum_t w_t |y_t - [x_t, 1] W~|^2,   TSS = sum_t w_t |y_t - mu_y|^2,
 *   r2[m] = 1 - RSS / TSS   (0 when TSS = 0),
 * pooled over the d_t output channels.  W [n_maps][d_s + 1][d_t] fp64 with the
 * bias as the last row; same input conventions as oracle_stats.  Two passes over
 * the tokens: the mean, then the residuals.  Returns 0.
 */
int oracle_probe_r2(int n_maps,
                    const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                    const int32_t *src_layer, const int32_t *src_head, const int32_t *weight_row,
                    const double *W,
                    const uint16_t *src, const int64_t *src_strides, int d_s,
                    const uint16_t *tgt, const int64_t *tgt_strides, int d_t,
                    const float *weights, int64_t w_row_stride,
                    int n_seqs, int seq_len, double *r2, int n_threads) {
    const int P = d_s + 1;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        const double *Wm = W + (int64_t)m * P * d_t;
        double *x = (double *)malloc(sizeof(double) * (size_t)d_s);
        double *mu = (double *)calloc((size_t)d_t, sizeof(double));
        double sw = 0.0, rss = 0.0, tss = 0.0;
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                const uint16_t *yr = tgt + row_offset(tgt_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                const double w = (double)weights[(int64_t)weight_row[m] * w_row_stride +
                                                 (int64_t)b * seq_len + t];
                sw += w;
                for (int j = 0; j < d_t; ++j) mu[j] += w * bf16_bits_to_double(yr[j]);
            }
        }
        for (int j = 0; j < d_t; ++j) mu[j] = sw != 0.0 ? mu[j] / sw : 0.0;
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                const uint16_t *xr = src + row_offset(src_strides, src_layer[m], kv[m], b, src_head[m], t);
                const uint16_t *yr = tgt + row_offset(tgt_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                const double w = (double)weights[(int64_t)weight_row[m] * w_row_stride +
                                                 (int64_t)b * seq_len + t];
                for (int i = 0; i < d_s; ++i) x[i] = bf16_bits_to_double(xr[i]);
                for (int j = 0; j < d_t; ++j) {
                    double pred = Wm[(int64_t)d_s * d_t + j];
                    for (int i = 0; i < d_s; ++i) pred += x[i] * Wm[(int64_t)i * d_t + j];
                    const double y = bf16_bits_to_double(yr[j]);
                    rss += w * (y - pred) * (y - pred);
                    tss += w * (y - mu[j]) * (y - mu[j]);
                }
            }
        }
        r2[m] = tss > 0.0 ? 1.0 - rss / tss : 0.0;
        free(x);
        free(mu);
    }
    return 0;
}

/*
 * Attention-aligned sensitivities (Sec. 3.3, Eq. attentionlinearization and
 * Eq. sensitivity), raw and before the global normalization.
 * For every target layer l, KV head h and sequence b, every boundary
 * c = boundaries[k] (the position of the first query after the prefix
 * [0, c)) and every query head u of h's group (u = h*G .. h*G + G-1,
 * G = n_qheads / n_heads):
 *   s_i = q_u . k_i / sqrt(d),  a_i = softmax over keys i = 0 .. c (causal,
 *   the query's own position included),  o_u = sum_i a_i v_i,
 * and for the eligible prefix positions E_c = {i < c : i mod sample_stride = 0}:
 *   p^V_i += a_i^2,   p^K_i += a_i^2 |v_i - o_u|^2 |q_u|^2 / d   (summed over u).
 * Each boundary's p^V and p^K are scaled to unit mass over E_c (skipped when
 * the mass is zero) and added into r:
 *   r [n_layers][2][n_heads][n_seqs * seq_len] (fp64, overwritten), component
 *   0 = K (from p^K), 1 = V (from p^V); the row of (l, z, h) is (l*2 + z)*H + h.
 * K, V: bf16 bits of the target cache, kv 0 and 1 of the strides
 * {layer, kv, seq, head, tok}.  q: bf16 bits, element (l, b, k, u, j) at
 * l*q_strides[0] + b*q_strides[1] + k*q_strides[2] + u*q_strides[3] + j.
 * Returns 0.
 */
int oracle_attn_sensitivity(int n_layers, int n_heads, int n_qheads, int d, int n_seqs, int seq_len,
                            const uint16_t *kvc, const int64_t *kv_strides, const uint16_t *q,
                            const int64_t *q_strides, const int32_t *boundaries, int n_bounds,
                            int sample_stride, double *r, int n_threads) {
    const int G = n_qheads / n_heads;
    const int64_t N = (int64_t)n_seqs * seq_len;
    set_threads(n_threads);
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int l = 0; l < n_layers; ++l) {
        for (int h = 0; h < n_heads; ++h) {
            double *rK = r + ((int64_t)(l * 2 + 0) * n_heads + h) * N;
            double *rV = r + ((int64_t)(l * 2 + 1) * n_heads + h) * N;
            memset(rK, 0, sizeof(double) * (size_t)N);
            memset(rV, 0, sizeof(double) * (size_t)N);
            double *a = (double *)malloc(sizeof(double) * (size_t)seq_len);
            double *pK = (double *)malloc(sizeof(double) * (size_t)seq_len);
            double *pV = (double *)malloc(sizeof(double) * (size_t)seq_len);
            double *qv = (double *)malloc(sizeof(double) * (size_t)d);
            double *o = (double *)malloc(sizeof(double) * (size_t)d);
            for (int b = 0; b < n_seqs; ++b) {
                for (int k = 0; k < n_bounds; ++k) {
                    const int c = boundaries[k];
                    for (int i = 0; i < seq_len; ++i) pK[i] = pV[i] = 0.0;
                    for (int u = h * G; u < (h + 1) * G; ++u) {
                        const uint16_t *qr = q + (int64_t)l * q_strides[0] + (int64_t)b * q_strides[1] +
                                             (int64_t)k * q_strides[2] + (int64_t)u * q_strides[3];
                        double qq = 0.0;
                        for (int j = 0; j < d; ++j) {
                            qv[j] = bf16_bits_to_double(qr[j]);
                            qq += qv[j] * qv[j];
                        }
                        double mx = -HUGE_VAL;
                        for (int i = 0; i <= c; ++i) {
                            const uint16_t *kr = kvc + row_offset(kv_strides, l, 0, b, h, i);
                            double sc = 0.0;
                            for (int j = 0; j < d; ++j) sc += qv[j] * bf16_bits_to_double(kr[j]);
                            a[i] = sc / sqrt((double)d);
                            if (a[i] > mx) mx = a[i];
                        }
                        double z = 0.0;
                        for (int i = 0; i <= c; ++i) {
                            a[i] = exp(a[i] - mx);
                            z += a[i];
                        }
                        for (int j = 0; j < d; ++j) o[j] = 0.0;
                        for (int i = 0; i <= c; ++i) {
                            a[i] /= z;
                            const uint16_t *vr = kvc + row_offset(kv_strides, l, 1, b, h, i);
                            for (int j = 0; j < d; ++j) o[j] += a[i] * bf16_bits_to_double(vr[j]);
                        }
                        for (int i = 0; i < c; i += sample_stride) {
                            const uint16_t *vr = kvc + row_offset(kv_strides, l, 1, b, h, i);
                            double dv = 0.0;
                            for (int j = 0; j < d; ++j) {
                                const double e = bf16_bits_to_double(vr[j]) - o[j];
                                dv += e * e;
                            }
                            pV[i] += a[i] * a[i];
                            pK[i] += a[i] * a[i] * dv * qq / (double)d;
                        }
                    }
                    double mK = 0.0, mV = 0.0;
                    for (int i = 0; i < c; i += sample_stride) {
                        mK += pK[i];
                        mV += pV[i];
                    }
                    for (int i = 0; i < c; i += sample_stride) {
                        if (mK > 0.0) rK[(int64_t)b * seq_len + i] += pK[i] / mK;
                        if (mV > 0.0) rV[(int64_t)b * seq_len + i] += pV[i] / mV;
                    }
                }
            }
            free(a);
            free(pK);
            free(pV);
            free(qv);
            free(o);
        }
    }
    return 0;
}

/*
 * Shrinkage of the raw sensitivities toward uniform weights (Sec. 3.3), per
 * row of r [n_rows][n_seqs * seq_len]: over the n calibration rows (positions
 * t with t mod sample_stride = 0 of every sequence),
 *   r_i <- r_i / mean(r)                       (mean one; all ones if the mean is 0)
 *   CV^2 = mean((r_i - 1)^2),  tau = min(n, 2 p),
 *   alpha = 1 if CV^2 = 0, else min(1, sqrt((n / tau - 1) / CV^2)),
 *   w_i = 1 + alpha (r_i - 1),
 * the largest alpha whose Kish effective sample size n / (1 + alpha^2 CV^2)
 * is at least tau.  Positions that are not calibration rows get w = 0.
 * Outputs w (same shape as r) and alpha [n_rows], fp64.  Returns 0.
 */
int oracle_attn_weights(int n_rows, int n_seqs, int seq_len, int sample_stride, const double *r, int p,
                        double *w, double *alpha) {
    const int64_t N = (int64_t)n_seqs * seq_len;
    for (int row = 0; row < n_rows; ++row) {
        const double *rr = r + (int64_t)row * N;
        double *ww = w + (int64_t)row * N;
        double sum = 0.0;
        int64_t n = 0;
        for (int b = 0; b < n_seqs; ++b)
            for (int t = 0; t < seq_len; t += sample_stride) {
                sum += rr[(int64_t)b * seq_len + t];
                ++n;
            }
        const double mean = n > 0 ? sum / (double)n : 0.0;
        double cv2 = 0.0;
        for (int b = 0; b < n_seqs; ++b)
            for (int t = 0; t < seq_len; t += sample_stride) {
                const double x = mean > 0.0 ? rr[(int64_t)b * seq_len + t] / mean : 1.0;
                cv2 += (x - 1.0) * (x - 1.0);
            }
        cv2 = n > 0 ? cv2 / (double)n : 0.0;
        const double tau = (double)(n < 2 * (int64_t)p ? n : 2 * (int64_t)p);
        double al = 1.0;
        if (cv2 > 0.0) {
            al = sqrt(((double)n / tau - 1.0) / cv2);
            if (al > 1.0) al = 1.0;
        }
        alpha[row] = al;
        for (int64_t i = 0; i < N; ++i) ww[i] = 0.0;
        for (int b = 0; b < n_seqs; ++b)
            for (int t = 0; t < seq_len; t += sample_stride) {
                const int64_t i = (int64_t)b * seq_len + t;
                const double x = mean > 0.0 ? rr[i] / mean : 1.0;
                ww[i] = 1.0 + al * (x - 1.0);
            }
    }
    return 0;
}

/*
 * Rotary position transform of the keys (Sec. 2.1, Sec. 3.1: source RoPE is
 * inverted before fitting and target RoPE applied after mapping; RoFormer's
 * rotation).  For every K row (kv = 0) of a cache at position
 * pos = pos_offset + tok, channel pairs are rotated by the angle pos * f_i,
 * f_i = theta^(-2 i / d), i < d/2:
 *   style 0 (half split): pair (i, i + d/2);  style 1 (interleaved): pair (2i, 2i + 1);
 *   (a, b) -> (a cos - b sin, b cos + a sin), with the angle negated when inverse.
 * Angles, sines and products in fp64, one rounding to bf16 (RNE).  V rows
 * (kv = 1) are copied unchanged.  in/out: bf16 bits with strides {layer, kv,
 * seq, head, tok}.  Returns 0.
 */
int oracle_rope(int n_layers, int n_heads, int d, int n_seqs, int seq_len, const uint16_t *in,
                const int64_t *in_strides, uint16_t *out, const int64_t *out_strides, double theta, int style,
                int inverse, int pos_offset) {
    const int h = d / 2;
    for (int l = 0; l < n_layers; ++l)
        for (int z = 0; z < 2; ++z)
            for (int b = 0; b < n_seqs; ++b)
                for (int g = 0; g < n_heads; ++g)
                    for (int t = 0; t < seq_len; ++t) {
                        const uint16_t *xr = in + row_offset(in_strides, l, z, b, g, t);
                        uint16_t *yr = out + row_offset(out_strides, l, z, b, g, t);
                        if (z == 1) {
                            for (int j = 0; j < d; ++j) yr[j] = xr[j];
                            continue;
                        }
                        const double pos = (double)(pos_offset + t);
                        for (int i = 0; i < h; ++i) {
                            const double ang = (inverse ? -pos : pos) * pow(theta, -2.0 * i / (double)d);
                            const double c = cos(ang), s = sin(ang);
                            const int ia = style == 0 ? i : 2 * i, ib = style == 0 ? i + h : 2 * i + 1;
                            const double a = bf16_bits_to_double(xr[ia]), bb = bf16_bits_to_double(xr[ib]);
                            yr[ia] = oracle_double_to_bf16(a * c - bb * s);
                            yr[ib] = oracle_double_to_bf16(bb * c + a * s);
                        }
                    }
    return 0;
}

/*
 * Online application of the fitted maps.
 *   W [n_maps][P][d_t] (fp64 copies of the coefficients; row d_s is the bias)
 *   out[tgt_layer, kv, seq, tgt_head, tok, j] = RNE_bf16( sum_k x~_k W[k][j] )
 * for every token of every sequence.  Returns 0.
 */
int oracle_apply(int n_maps,
                 const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                 const int32_t *src_layer, const int32_t *src_head,
                 const double *W,
                 const uint16_t *src, const int64_t *src_strides, int d_s,
                 uint16_t *out, const int64_t *out_strides, int d_t,
                 int n_seqs, int seq_len, int n_threads) {
    const int P = d_s + 1;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        const double *Wm = W + (int64_t)m * P * d_t;
        double *xt = (double *)malloc(sizeof(double) * (size_t)P);
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                const uint16_t *xr = src + row_offset(src_strides, src_layer[m], kv[m], b, src_head[m], t);
                uint16_t *orow = out + row_offset(out_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                for (int i = 0; i < d_s; ++i) xt[i] = bf16_bits_to_double(xr[i]);
                xt[d_s] = 1.0;
                for (int j = 0; j < d_t; ++j) {
                    double s = 0.0;
                    for (int k = 0; k < P; ++k) s += xt[k] * Wm[(int64_t)k * d_t + j];
                    orow[j] = oracle_double_to_bf16(s);
                }
            }
        }
        free(xt);
    }
    return 0;
}

/*
 * Multi-layer head-local feature (Sec. 3.2, Eq. localfeature with k selected
 * source layers).  Map m reads, for each calibration row, the k source rows
 *   Z^S[src_layers[m*k + i], kv[m], seq, src_head[m], t],  i = 0..k-1,
 * concatenated in that order, and appends 1:
 *   x~ = [x_0 ; x_1 ; ... ; x_{k-1} ; 1]   (width P = k d_s + 1).
 * The calibration rows are the tokens t of every sequence with
 * t mod sample_stride == 0 (Sec. 4.1 samples every fourth token).
 *   G [n_maps][P][P] += sum w x~ x~^T,   C [n_maps][P][d_t] += sum w x~ y^T
 * with w = weights[weight_row[m] * w_row_stride + seq * seq_len + t].
 * Returns 0.
 */
int oracle_stats_multi(int n_maps, int k,
                       const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                       const int32_t *src_layers, const int32_t *src_head, const int32_t *weight_row,
                       const uint16_t *src, const int64_t *src_strides, int d_s,
                       const uint16_t *tgt, const int64_t *tgt_strides, int d_t,
                       const float *weights, int64_t w_row_stride,
                       int n_seqs, int seq_len, int sample_stride,
                       double *G, double *C, int n_threads) {
    const int P = k * d_s + 1;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        double *Gm = G + (int64_t)m * P * P;
        double *Cm = C + (int64_t)m * P * d_t;
        double *xt = (double *)malloc(sizeof(double) * (size_t)P);
        double *y = (double *)malloc(sizeof(double) * (size_t)d_t);
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; t += sample_stride) {
                for (int i = 0; i < k; ++i) {
                    const uint16_t *xr = src + row_offset(src_strides, src_layers[(int64_t)m * k + i], kv[m], b,
                                                          src_head[m], t);
                    for (int c = 0; c < d_s; ++c) xt[i * d_s + c] = bf16_bits_to_double(xr[c]);
                }
                xt[k * d_s] = 1.0;
                const uint16_t *yr = tgt + row_offset(tgt_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                for (int j = 0; j < d_t; ++j) y[j] = bf16_bits_to_double(yr[j]);
                const double w = (double)weights[(int64_t)weight_row[m] * w_row_stride + (int64_t)b * seq_len + t];
                for (int i = 0; i < P; ++i) {
                    const double wi = w * xt[i];
                    double *gr = Gm + (int64_t)i * P;
                    double *cr = Cm + (int64_t)i * d_t;
                    for (int j = 0; j < P; ++j) gr[j] += wi * xt[j];
                    for (int j = 0; j < d_t; ++j) cr[j] += wi * y[j];
                }
            }
        }
        free(xt);
        free(y);
    }
    return 0;
}

/*
 * Two-pass centered statistics (Sec. 3.4) over the multi-layer feature of
 * Sec. 3.2: x = [x_0 ; ... ; x_{k-1}] (width Dx = k d_s, no bias entry), the
 * calibration rows t with t mod sample_stride == 0.  Pass 1 sums w, w x and
 * w y over every row; pass 2 revisits the rows and accumulates the moments
 * about the weighted means of pass 1.  Outputs (overwritten, fp64):
 *   sums [n_maps][1 + Dx + d_t] = (sum w, sum w x, sum w y),
 *   A [n_maps][Dx][Dx] = sum w (x - mu_x)(x - mu_x)^T,
 *   B [n_maps][Dx][d_t] = sum w (x - mu_x)(y - mu_y)^T.
 * A map whose weights sum to zero gets zero means.  Returns 0.
 */
int oracle_stats_multi_centered(int n_maps, int k,
                                const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                                const int32_t *src_layers, const int32_t *src_head, const int32_t *weight_row,
                                const uint16_t *src, const int64_t *src_strides, int d_s,
                                const uint16_t *tgt, const int64_t *tgt_strides, int d_t,
                                const float *weights, int64_t w_row_stride,
                                int n_seqs, int seq_len, int sample_stride,
                                double *sums, double *A, double *B, int n_threads) {
    const int Dx = k * d_s, NS = 1 + Dx + d_t;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        double *sm = sums + (int64_t)m * NS;
        double *Am = A + (int64_t)m * Dx * Dx;
        double *Bm = B + (int64_t)m * Dx * d_t;
        double *x = (double *)malloc(sizeof(double) * (size_t)Dx);
        double *y = (double *)malloc(sizeof(double) * (size_t)d_t);
        memset(sm, 0, sizeof(double) * (size_t)NS);
        memset(Am, 0, sizeof(double) * (size_t)Dx * Dx);
        memset(Bm, 0, sizeof(double) * (size_t)Dx * d_t);
        for (int pass = 0; pass < 2; ++pass) {
            const double sw = sm[0];
            for (int b = 0; b < n_seqs; ++b) {
                for (int t = 0; t < seq_len; t += sample_stride) {
                    for (int i = 0; i < k; ++i) {
                        const uint16_t *xr = src + row_offset(src_strides, src_layers[(int64_t)m * k + i], kv[m], b,
                                                              src_head[m], t);
                        for (int c = 0; c < d_s; ++c) x[i * d_s + c] = bf16_bits_to_double(xr[c]);
                    }
                    const uint16_t *yr = tgt + row_offset(tgt_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                    for (int j = 0; j < d_t; ++j) y[j] = bf16_bits_to_double(yr[j]);
                    const double w = (double)weights[(int64_t)weight_row[m] * w_row_stride + (int64_t)b * seq_len + t];
                    if (pass == 0) {                       /* pass 1: weighted sums */
                        sm[0] += w;
                        for (int i = 0; i < Dx; ++i) sm[1 + i] += w * x[i];
                        for (int j = 0; j < d_t; ++j) sm[1 + Dx + j] += w * y[j];
                        continue;
                    }
                    /* pass 2: moments about the means */
                    for (int i = 0; i < Dx; ++i) x[i] -= sw != 0.0 ? sm[1 + i] / sw : 0.0;
                    for (int j = 0; j < d_t; ++j) y[j] -= sw != 0.0 ? sm[1 + Dx + j] / sw : 0.0;
                    for (int i = 0; i < Dx; ++i) {
                        const double wi = w * x[i];
                        double *ar = Am + (int64_t)i * Dx;
                        double *br = Bm + (int64_t)i * d_t;
                        for (int j = 0; j < Dx; ++j) ar[j] += wi * x[j];
                        for (int j = 0; j < d_t; ++j) br[j] += wi * y[j];
                    }
                }
            }
        }
        free(x);
        free(y);
    }
    return 0;
}

/*
 * Online application with the target's rotary transform (Sec. 1 pipeline;
 * Sec. 2.1, Sec. 3.1: the mapped keys receive the target RoPE).  For every map
 * and token, s = x~ W~ in fp64 as in oracle_apply; when the map is a K map
 * (kv = 0), the pairs of s (style 0: (i, i + d_t/2), style 1: (2i, 2i + 1))
 * are turned by the angle pos * theta^(-2 i / d_t), pos = pos_offset + t:
 *   (a, b) -> (a cos - b sin, b cos + a sin),
 * in fp64; then every channel is rounded once to bf16 (RNE).  V maps write
 * RNE_bf16(s).  Returns 0.
 */
int oracle_apply_rope(int n_maps,
                      const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                      const int32_t *src_layer, const int32_t *src_head,
                      const double *W,
                      const uint16_t *src, const int64_t *src_strides, int d_s,
                      uint16_t *out, const int64_t *out_strides, int d_t,
                      int n_seqs, int seq_len, double theta, int style, int pos_offset, int n_threads) {
    const int P = d_s + 1;
    const int h = d_t / 2;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        const double *Wm = W + (int64_t)m * P * d_t;
        double *xt = (double *)malloc(sizeof(double) * (size_t)P);
        double *s = (double *)malloc(sizeof(double) * (size_t)d_t);
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                const uint16_t *xr = src + row_offset(src_strides, src_layer[m], kv[m], b, src_head[m], t);
                uint16_t *orow = out + row_offset(out_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                for (int i = 0; i < d_s; ++i) xt[i] = bf16_bits_to_double(xr[i]);
                xt[d_s] = 1.0;
                for (int j = 0; j < d_t; ++j) {
                    double acc = 0.0;
                    for (int k = 0; k < P; ++k) acc += xt[k] * Wm[(int64_t)k * d_t + j];
                    s[j] = acc;
                }
                if (kv[m] == 0) {
                    const double pos = (double)(pos_offset + t);
                    for (int i = 0; i < h; ++i) {
                        const double ang = pos * pow(theta, -2.0 * i / (double)d_t);
                        const double c = cos(ang), sn = sin(ang);
                        const int ia = style == 0 ? i : 2 * i, ib = style == 0 ? i + h : 2 * i + 1;
                        const double a = s[ia], bb = s[ib];
                        s[ia] = a * c - bb * sn;
                        s[ib] = bb * c + a * sn;
                    }
                }
                for (int j = 0; j < d_t; ++j) orow[j] = oracle_double_to_bf16(s[j]);
            }
        }
        free(s);
        free(xt);
    }
    return 0;
}

/*
 * Online application of multi-layer maps (Sec. 3.2 feature, Sec. 1 pipeline):
 *   W [n_maps][P][d_t], P = k d_s + 1, rows i d_s .. (i+1) d_s - 1 act on the
 *   source row of src_layers[m*k + i], the last row is the bias;
 *   out[tgt_layer, kv, seq, tgt_head, tok, j] = RNE_bf16( sum_p x~_p W[p][j] )
 * for every token of every sequence, the sum in fp64, rounded once.  Returns 0.
 */
int oracle_apply_multi(int n_maps, int k,
                       const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                       const int32_t *src_layers, const int32_t *src_head,
                       const double *W,
                       const uint16_t *src, const int64_t *src_strides, int d_s,
                       uint16_t *out, const int64_t *out_strides, int d_t,
                       int n_seqs, int seq_len, int n_threads) {
    const int P = k * d_s + 1;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        const double *Wm = W + (int64_t)m * P * d_t;
        double *xt = (double *)malloc(sizeof(double) * (size_t)P);
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                for (int i = 0; i < k; ++i) {
                    const uint16_t *xr = src + row_offset(src_strides, src_layers[(int64_t)m * k + i], kv[m], b,
                                                          src_head[m], t);
                    for (int c = 0; c < d_s; ++c) xt[i * d_s + c] = bf16_bits_to_double(xr[c]);
                }
                xt[k * d_s] = 1.0;
                uint16_t *orow = out + row_offset(out_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                for (int j = 0; j < d_t; ++j) {
                    double s = 0.0;
                    for (int p = 0; p < P; ++p) s += xt[p] * Wm[(int64_t)p * d_t + j];
                    orow[j] = oracle_double_to_bf16(s);
                }
            }
        }
        free(xt);
    }
    return 0;
}

/*
 * Multi-layer application with the target's rotary transform (Sec. 3.2
 * feature, Sec. 1 pipeline; Sec. 2.1, Sec. 3.1: the mapped keys receive the
 * target RoPE before decoding).  s = x~ W~ in fp64 as in oracle_apply_multi;
 * for a K map (kv = 0) every channel pair of s (style 0: (i, i + d_t/2),
 * style 1: (2i, 2i + 1)) is turned by the angle pos * theta^(-2 i / d_t),
 * pos = pos_offset + t, in fp64:
 *   (a, b) -> (a cos - b sin, b cos + a sin);
 * then every channel is rounded once to bf16 (RNE).  V maps write
 * RNE_bf16(s).  Returns 0.
 */
int oracle_apply_multi_rope(int n_maps, int k,
                            const int32_t *tgt_layer, const int32_t *tgt_head, const int32_t *kv,
                            const int32_t *src_layers, const int32_t *src_head,
                            const double *W,
                            const uint16_t *src, const int64_t *src_strides, int d_s,
                            uint16_t *out, const int64_t *out_strides, int d_t,
                            int n_seqs, int seq_len, double theta, int style, int pos_offset, int n_threads) {
    const int P = k * d_s + 1;
    const int h = d_t / 2;
    set_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int m = 0; m < n_maps; ++m) {
        const double *Wm = W + (int64_t)m * P * d_t;
        double *xt = (double *)malloc(sizeof(double) * (size_t)P);
        double *s = (double *)malloc(sizeof(double) * (size_t)d_t);
        for (int b = 0; b < n_seqs; ++b) {
            for (int t = 0; t < seq_len; ++t) {
                for (int i = 0; i < k; ++i) {
                    const uint16_t *xr = src + row_offset(src_strides, src_layers[(int64_t)m * k + i], kv[m], b,
                                                          src_head[m], t);
                    for (int c = 0; c < d_s; ++c) xt[i * d_s + c] = bf16_bits_to_double(xr[c]);
                }
                xt[k * d_s] = 1.0;
                for (int j = 0; j < d_t; ++j) {
                    double acc = 0.0;
                    for (int p = 0; p < P; ++p) acc += xt[p] * Wm[(int64_t)p * d_t + j];
                    s[j] = acc;
                }
                if (kv[m] == 0) {
                    const double pos = (double)(pos_offset + t);
                    for (int i = 0; i < h; ++i) {
                        const double ang = pos * pow(theta, -2.0 * i / (double)d_t);
                        const double c = cos(ang), sn = sin(ang);
                        const int ia = style == 0 ? i : 2 * i, ib = style == 0 ? i + h : 2 * i + 1;
                        const double a = s[ia], bb = s[ib];
                        s[ia] = a * c - bb * sn;
                        s[ib] = bb * c + a * sn;
                    }
                }
                uint16_t *orow = out + row_offset(out_strides, tgt_layer[m], kv[m], b, tgt_head[m], t);
                for (int j = 0; j < d_t; ++j) orow[j] = oracle_double_to_bf16(s[j]);
            }
        }
        free(s);
        free(xt);
    }
    return 0;
}

/* Element-wise oracle_double_to_bf16 over n values.  Returns 0. */
int oracle_double_to_bf16_array(int64_t n, const double *v, uint16_t *out) {
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_double_to_bf16(v[i]);
    return 0;
}

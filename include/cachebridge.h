/*
 * cachebridge.h -- C ABI of the MI355X (gfx950) CacheBridge mapper library.
 *
 * The library builds and applies head-local affine ridge maps between the KV
 * caches of a source model and a target model, following CacheBridge
 * ("Efficient Cross-Model KV Cache Transfer"):
 *
 *   cb_stats_accumulate  weighted augmented sufficient statistics
 *                        (Sec. 3.4, Eq. fusedstats; head-local support of
 *                        Sec. 3.2, Eq. localfeature, one source layer per map)
 *   cb_ridge_solve       batched ridge solve (Sec. 3.1, Eq. closedform; Sec. 3.4)
 *   cb_apply             online application of the maps to a sender cache,
 *                        writing a decode-ready target cache (Sec. 1 pipeline;
 *                        Sec. 2.3, Eq. support-cost)
 *
 * and the paper's two-pass centered form of the same fit (Sec. 3.4, Eq.
 * fusedstats; Sec. 3.1, Eq. closedform):
 *
 *   cb_stats_zero_centered, cb_stats_means, cb_stats_accumulate_centered,
 *   cb_ridge_solve_centered (and its one-pass form cb_stats_accumulate_shifted,
 *   cb_stats_shift_finish)
 *
 * and the layer-selection probes of Sec. 3.1 (centered single-source-layer
 * fits ranked by held-in R^2):
 *
 *   cb_probe_r2, cb_select_layers
 *
 * and the attention-aligned calibration weights of Sec. 3.3:
 *
 *   cb_attn_sensitivity, cb_attn_weights
 *
 * and the rotary position transform of cached keys (Sec. 2.1, Sec. 3.1: RoPE
 * removed before fitting, restored after mapping):
 *
 *   cb_rope_table, cb_rope, cb_stats_accumulate_rope and cb_apply_rope (the
 *   rotary transforms folded into the statistics gather and the mapping)
 *
 * and the multi-layer feature of Sec. 3.2 (k selected source layers per map):
 *
 *   cb_plan_create_multi, cb_plan_feature_width, cb_ridge_solve_ws
 *
 * Conventions shared by every call
 * --------------------------------
 * - Row vectors: a map is W~ = [W ; b^T], a P x d_t fp32 matrix with
 *   P = d_s + 1 whose last row is the bias; the mapped row is [x, 1] W~.
 * - Device memory: every data pointer (caches, weights, G, C, maps, info) is a
 *   device pointer on the current HIP device, allocated and owned by the
 *   caller.  The library never frees caller memory.  A plan owns its own
 *   workspace, allocated in cb_plan_create and freed in cb_plan_destroy; no
 *   other call allocates.
 * - Streams: `stream` is a hipStream_t passed as void* (NULL = the null
 *   stream).  Calls enqueue work and return without waiting.
 * - Errors: argument, shape and alignment problems are found on the host,
 *   before anything is enqueued, and returned as a cb_status; cb_last_error()
 *   then returns a message for the calling thread.  A failed launch returns
 *   CB_ERR_DEVICE.  Numerical failure of one ridge system is not a call error:
 *   it is reported per map in `info` (LAPACK style).
 * - Determinism: for a given plan, inputs and sequence of calls, results are
 *   bitwise reproducible (fixed reduction order, no floating-point atomics).
 * - Thread safety: a plan may be used by one thread / stream at a time.
 * - Supported widths: d_s and d_t in {64, 96, 128} (P <= 129).  Cache rows are
 *   bfloat16, channel stride 1, every row 16-byte aligned.
 */
#ifndef CACHEBRIDGE_H
#define CACHEBRIDGE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CB_OK = 0,
    CB_ERR_INVALID_ARGUMENT = 1, /* null pointer, bad index, bad flag, duplicate map */
    CB_ERR_SHAPE = 2,            /* geometry does not match the plan or the call  */
    CB_ERR_MISALIGNED = 3,       /* a pointer or stride breaks 16-byte row alignment */
    CB_ERR_OUT_OF_MEMORY = 4,    /* plan workspace allocation failed               */
    CB_ERR_DEVICE = 5,           /* a HIP call or kernel launch failed             */
    CB_ERR_UNSUPPORTED = 6       /* head width outside {64, 96, 128}, too many tokens */
} cb_status;

/*
 * A KV cache of one model (Sec. 2.1: K and V per layer, token and KV head).
 * Element (layer, kv, seq, head, tok, ch) lives at
 *   data[layer*s_layer + kv*s_kv + seq*s_seq + head*s_head + tok*s_tok + ch]
 * (kv 0 = K, 1 = V; strides in elements; channel stride 1).  The canonical
 * layout is [layer][kv][seq][head][tok][ch].  `data` and every stride must
 * keep each row 16-byte aligned (multiples of 8 elements).  The same struct
 * describes inputs (read) and the output of cb_apply (written).
 */
typedef struct {
    void *data;                 /* device memory, bfloat16 elements            */
    int32_t n_layers;
    int32_t n_heads;            /* KV heads                                     */
    int32_t head_dim;
    int32_t n_seqs;
    int32_t seq_len;
    int64_t s_layer, s_kv, s_seq, s_head, s_tok;
} cb_cache;

/*
 * Mapper support (Sec. 2.1; Sec. 3.2 Eq. localfeature with k = 1): map m
 * predicts target (tgt_layer[m], tgt_head[m], kv[m]) from source
 * (src_layer[m], src_head[m], kv[m]) -- K from K, V from V -- using calibration
 * weight row weight_row[m].  Host arrays of n_maps entries, read during
 * cb_plan_create only.  Map m owns G[m], C[m] and maps[m].  A target (layer,
 * kv, head) may appear in several maps (layer-selection probes fit every
 * candidate source layer); cb_apply needs it at most once.
 */
typedef struct {
    int32_t n_maps;
    const int32_t *tgt_layer;
    const int32_t *tgt_head;
    const int32_t *kv;
    const int32_t *src_layer;
    const int32_t *src_head;
    const int32_t *weight_row;
} cb_head_map;

/*
 * Queries of the target model at the calibration boundaries (Sec. 3.3): the
 * query of head u at boundary k of sequence seq in layer l, element j at
 *   data[l*s_layer + seq*s_seq + k*s_bnd + u*s_head + j]   (bfloat16, j stride 1).
 * Query head u belongs to KV head u / (n_qheads / n_heads) of the target cache.
 * data and every stride must keep each row 16-byte aligned.
 */
typedef struct {
    const void *data;
    int32_t n_layers;
    int32_t n_qheads;
    int32_t head_dim;
    int32_t n_seqs;
    int32_t n_bounds;
    int64_t s_layer, s_seq, s_bnd, s_head;
} cb_queries;

/* Validated head map, its precomputed read plan and workspace (opaque). */
typedef struct cb_plan cb_plan;

/* cb_ridge_solve flags. */
#define CB_LAMBDA_RELATIVE 1u        /* lambda_m = lambda * trace(G_m) / P          */
#define CB_RIDGE_BIAS_UNPENALIZED 2u /* no ridge on the bias row: Eq. closedform    */

/*
 * Turn the head map into the fixed list of work items the statistics kernel
 * walks (Sec. 2.3: the support of every map is known before any fitting, so
 * the reads can be planned once) and allocate the plan's workspace on the
 * current device.
 *   src_geom / tgt_geom: only n_layers, n_heads and head_dim are read.
 *   max_tokens_per_call: upper bound on n_seqs * seq_len of any later
 *     cb_stats_accumulate call (sizes the per-workgroup partial sums).
 * Errors: CB_ERR_INVALID_ARGUMENT (null, index out of range, kv not 0/1,
 * negative weight row), CB_ERR_UNSUPPORTED (head width),
 * CB_ERR_OUT_OF_MEMORY, CB_ERR_DEVICE.  On error *out is set to NULL.
 */
cb_status cb_plan_create(const cb_head_map *map, const cb_cache *src_geom, const cb_cache *tgt_geom,
                         int64_t max_tokens_per_call, cb_plan **out);

/* Free the plan and its workspace (waits for the device).  NULL is accepted. */
cb_status cb_plan_destroy(cb_plan *plan);

/* Number of maps, source width d_s and target width d_t of a plan. */
cb_status cb_plan_shape(const cb_plan *plan, int32_t *n_maps, int32_t *d_s, int32_t *d_t);

/*
 * Set G [n_maps][P][P] and C [n_maps][P][d_t] (fp32, row-major) to zero on
 * `stream`, with a fill kernel (safe under stream capture).
 */
cb_status cb_stats_zero(const cb_plan *plan, float *G, float *C, void *stream);

/*
 * Add one batch of calibration tokens to the statistics (Sec. 3.4, Eq.
 * fusedstats, in the augmented uncentered form that contains A_h, B_h and the
 * weighted means):  for every map m and every token (seq, tok) of the batch,
 *   x~ = [ src(src_layer, kv, seq, src_head, tok) ; 1 ]      (P = d_s + 1)
 *   y  =   tgt(tgt_layer, kv, seq, tgt_head, tok)            (d_t)
 *   w  =   weights[weight_row * w_row_stride + seq * seq_len + tok]   (fp32)
 *   G[m] += w x~ x~^T      C[m] += w x~ y^T
 * src and tgt must have the plan's layers / heads / widths and the same
 * n_seqs and seq_len; n_seqs * seq_len <= max_tokens_per_call; 0 tokens is a
 * no-op.  G is written exactly symmetric.  Weights are non-negative by the
 * paper's definition (Sec. 3.1); NaN propagates.  Accuracy: products are
 * formed from the exact bf16 inputs and an fp32 weight split into two bf16
 * terms, summed in fp32 (relative Frobenius error ~1e-6 against fp64).
 */
cb_status cb_stats_accumulate(cb_plan *plan, const cb_cache *src, const cb_cache *tgt,
                              const float *weights, int64_t w_row_stride,
                              float *G, float *C, void *stream);

/*
 * Batched ridge solve (Sec. 3.1, Eq. closedform; Sec. 3.4):
 *   maps[m] = (G[m] + lambda_m D)^{-1} C[m]
 * G [n_maps][P][P], C [n_maps][P][d_t], maps [n_maps][P][d_t] (fp32,
 * row-major), info [n_maps] (int32, device).  lambda_m = lambda, or
 * lambda * trace(G[m]) / P with CB_LAMBDA_RELATIVE.  D = I by default (the
 * bias row is penalized too); with CB_RIDGE_BIAS_UNPENALIZED the last
 * diagonal entry of D is 0, which equals the paper's centered weighted ridge
 * (weights rescaled to mean one).  G is read in full and must be symmetric
 * (cb_stats_accumulate writes it so).  Gauss-Jordan elimination without
 * pivoting in fp64, one workgroup per system; for the symmetric positive
 * definite G + lambda_m D its pivots are the squared diagonal of the Cholesky
 * factor.  info[m] = 0 on success, else the 1-based index of the first pivot
 * that is not positive and finite (the column where Cholesky would stop), and
 * maps[m] is zero-filled.  P in {65, 97, 129}, d_t in {64, 96, 128}; wider
 * systems return CB_ERR_UNSUPPORTED (use cb_ridge_solve_ws).
 */
cb_status cb_ridge_solve(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C,
                         float lambda, uint32_t flags, float *maps, int32_t *info, void *stream);

/*
 * Two-pass centered statistics (Sec. 3.4, Eq. fusedstats): pass 1 sums the
 * weights and weighted rows over every calibration batch (cb_stats_means),
 * pass 2 revisits the batches and accumulates the moments about the means of
 * pass 1 (cb_stats_accumulate_centered).  Centering before the products keeps
 * A and B accurate when channels carry large means, where the uncentered
 * moments of cb_stats_accumulate lose digits to cancellation.  A multi-layer
 * plan (cb_plan_create_multi) is accepted too: x is then the concatenated
 * feature [x_0; ...; x_{k-1}] of width d_x = k d_s in place of d_s below, the
 * calibration rows are the plan's sampled tokens, sq must be NULL, and the
 * maps are solved with cb_ridge_solve_centered_ws.  Per map m:
 *   sums [n_maps][1 + d_s + d_t] fp64 = (sum w, sum w x, sum w y)
 *   mu_x = (sum w x) / (sum w),  mu_y = (sum w y) / (sum w)   (0 if sum w = 0)
 *   A [n_maps][d_s][d_s] fp32 = sum w (x - mu_x)(x - mu_x)^T
 *   B [n_maps][d_s][d_t] fp32 = sum w (x - mu_x)(y - mu_y)^T
 * with x, y, w read as in cb_stats_accumulate.  All pointers are device
 * pointers owned by the caller; sums is 8-byte aligned.
 *
 * cb_stats_zero_centered: set sums, A, B and, if not NULL, sq (see
 * cb_stats_means) to zero on `stream` (fill kernels).
 */
cb_status cb_stats_zero_centered(const cb_plan *plan, double *sums, double *sq, float *A, float *B, void *stream);

/*
 * Pass 1: sums[m] += (sum w, sum w x, sum w y) over the batch, with the
 * products and sums formed in fp64 (exact products; summation order fixed).
 * If sq is not NULL, also sq[m] += (sum w x_i^2, sum w y_j^2), [n_maps][d_s + d_t]
 * fp64 (8-byte aligned): the sums of squares that cb_probe_r2 needs.
 * Call it on every batch before the first cb_stats_accumulate_centered.
 * Arguments, limits and errors as in cb_stats_accumulate.
 */
cb_status cb_stats_means(cb_plan *plan, const cb_cache *src, const cb_cache *tgt, const float *weights,
                         int64_t w_row_stride, double *sums, double *sq, void *stream);

/*
 * Pass 2: A[m] += sum w (x - mu_x)(x - mu_x)^T and B[m] += sum w (x - mu_x)(y - mu_y)^T
 * over the batch, with the means taken from the complete pass-1 sums (read,
 * not modified; they must not change between the pass-2 calls of one fit).
 * Each product pairs w (x - mu_x), formed in fp32 and split into two bf16
 * terms, with the exact bf16 x or y; the sums run in fp32, and the term
 * (sum w (x - mu_x)) mu^T that the uncentered right operand contributes is
 * subtracted at the end.  A is written exactly symmetric.  Arguments, limits
 * and errors as in cb_stats_accumulate.
 */
cb_status cb_stats_accumulate_centered(cb_plan *plan, const cb_cache *src, const cb_cache *tgt,
                                       const float *weights, int64_t w_row_stride, const double *sums,
                                       float *A, float *B, void *stream);

/*
 * One-pass form of the same centered statistics (Sec. 3.4, Eq. fusedstats:
 * moments about the weighted means).  Pass 1 of the two-pass form reads every
 * calibration row once more only to learn the means; here the moments are
 * formed about the means of a pilot instead (`shift`: the sums that
 * cb_stats_means left for any subset of the data, e.g. the first few
 * sequences; zero sums mean no shift), while the same pass also sums the
 * weights, the residuals and the targets (a multi-layer plan sums the weights
 * and targets in a second, small pass over the call's target rows alone), and
 * cb_stats_shift_finish then moves the moments to the data's own means:
 *   shift [n_maps][1 + d_x + d_t] fp64, read: mu'_x = shift_x / shift_w, mu'_y likewise
 *   accumulate, per batch:  A[m] += sum w (x - mu'_x)(x - mu'_x)^T
 *                           B[m] += sum w (x - mu'_x)(y - mu'_y)^T
 *                           sums[m] += (sum w, sum w (x - mu'_x), sum w y)
 *   finish, once:  with S = sum w, delta = (sum w (x - mu'_x)) / S = mu_x - mu'_x,
 *                  A[m] -= S delta delta^T,  B[m] -= S delta (mu_y - mu'_y)^T  (fp64, rounded once)
 *                  and sums[m] becomes (sum w, sum w x, sum w y)
 * after which sums, A and B are those of the two-pass form (the same exact
 * values; the differences are rounding) and go to cb_ridge_solve_centered or
 * cb_ridge_solve_centered_ws.  The closer the pilot means are to the data's,
 * the smaller the correction: the pilot only has to remove the channels'
 * large common offsets.  Products, splits and fp32 sums as in
 * cb_stats_accumulate_centered; the sums of a single-layer plan run in fp32
 * within a work unit and in fp64 across units and calls (about 1e-7
 * relative; pass 1 is exact), those of a multi-layer plan in fp32 between two
 * flushes (sum w (x - mu')) or in fp64 (sum w, sum w y).  Zero sums, A and B before the first call (cb_stats_zero_centered);
 * shift must not change between the calls of one fit and must not be sums.
 * Single- and multi-layer plans; d_x = d_s or k d_s.  Arguments, limits and
 * errors as in cb_stats_accumulate_centered, plus CB_ERR_INVALID_ARGUMENT
 * when shift is NULL or equals sums.
 */
cb_status cb_stats_accumulate_shifted(cb_plan *plan, const cb_cache *src, const cb_cache *tgt,
                                      const float *weights, int64_t w_row_stride, const double *shift,
                                      double *sums, float *A, float *B, void *stream);
cb_status cb_stats_shift_finish(const cb_plan *plan, const double *shift, double *sums, float *A, float *B,
                                void *stream);

/*
 * Centered ridge solve (Sec. 3.1, Eq. closedform):
 *   W = (A[m] + lambda_m I)^{-1} B[m],   b = mu_y - W^T mu_x,
 * written as maps[m] = [W ; b^T], [n_maps][d_s + 1][d_t] fp32 (the layout of
 * cb_ridge_solve and cb_apply).  The bias is never penalized.  lambda_m =
 * lambda, or with CB_LAMBDA_RELATIVE lambda * (tr A + S |mu_x|^2 + S) / (d_s + 1),
 * S = sum w: the relative lambda of cb_ridge_solve on the uncentered moments
 * of the same data, so both forms solve the same problem
 * (CB_RIDGE_BIAS_UNPENALIZED is accepted and changes nothing).  Gauss-Jordan
 * elimination in fp64, one workgroup per system.  info[m] = 0 on success, else
 * the 1-based index of the first pivot of A + lambda_m I that is not positive
 * and finite, and maps[m] is zero-filled.  d_s, d_t in {64, 96, 128}.
 */
cb_status cb_ridge_solve_centered(int32_t n_maps, int32_t d_s, int32_t d_t, const double *sums, const float *A,
                                  const float *B, float lambda, uint32_t flags, float *maps, int32_t *info,
                                  void *stream);

/*
 * Centered ridge solve for any feature width (Sec. 3.1, Eq. closedform over
 * the multi-layer feature of Sec. 3.2, d_x = k d_s): the arrays, lambda_m,
 * bias and info of cb_ridge_solve_centered with d_x in place of d_s, maps
 * [n_maps][d_x + 1][d_t].  d_x <= 128 runs cb_ridge_solve_centered (the
 * workspace is ignored); otherwise (d_x <= 4096, d_t in {64, 96, 128}) each
 * system A + lambda_m I is factored in fp64 in `workspace` (caller-owned device
 * memory, 8-byte aligned, at least cb_ridge_solve_workspace_bytes(d_x, d_t, 1)
 * bytes) by the blocked Cholesky of cb_ridge_solve_ws, batches as there, and
 * the bias row b = mu_y - W^T mu_x is formed in fp64.  Errors: CB_ERR_SHAPE
 * (workspace too small), else as cb_ridge_solve_centered.
 */
cb_status cb_ridge_solve_centered_ws(int32_t n_maps, int32_t d_x, int32_t d_t, const double *sums, const float *A,
                                     const float *B, float lambda, uint32_t flags, void *workspace,
                                     int64_t workspace_bytes, float *maps, int32_t *info, void *stream);

/*
 * Held-in R^2 of layer-selection probes (Sec. 3.1: for each target layer,
 * centered single-source-layer fits under the same head assignment, scored by
 * held-in R^2).  A probe is an ordinary map of a plan that pairs target heads
 * with candidate source layers; fit it with cb_stats_means (with sq),
 * cb_stats_accumulate_centered and cb_ridge_solve_centered, then
 *   r2[m] = 1 - RSS / TSS,   pooled over the d_t output channels, where
 *   TSS = sum_j (sum w y_j^2 - (sum w y_j)^2 / S),
 *   RSS = sum_t w |y - [x, 1] maps[m]|^2 = TSS - 2 tr(W^T B) + tr(W^T A W)
 * (the bias row of maps is mu_y - W^T mu_x, so the residual has weighted mean
 * zero).  r2[m] = 0 when S = 0 or TSS = 0.  sums, sq: fp64 as written by
 * cb_stats_means; A, B: fp32 as written by cb_stats_accumulate_centered; maps:
 * [n_maps][d_s + 1][d_t] fp32; r2: [n_maps] fp64.  Device pointers; one
 * workgroup per map, fp32 products of A W, fp64 traces.  d_s, d_t in
 * {64, 96, 128}.
 */
cb_status cb_probe_r2(int32_t n_maps, int32_t d_s, int32_t d_t, const double *sums, const double *sq, const float *A,
                      const float *B, const float *maps, double *r2, void *stream);

/*
 * Layer selection (Sec. 3.1), on the host: score[l][j] = the mean of r2 over
 * the maps with target layer l and source layer j (every KV head, K and V);
 * for each target layer the source layers in decreasing score, equal scores in
 * increasing j; the first k of them are selected[l][0..k-1] (S_l).  Pairs
 * without maps get score -HUGE_VAL and are never selected; missing entries
 * are -1.  map: host head map (only n_maps, tgt_layer and src_layer are read);
 * r2: host [n_maps]; selected: host [n_tgt_layers][k]; score: host
 * [n_tgt_layers][n_src_layers] or NULL.  Runs synchronously on the calling
 * thread.  Errors: CB_ERR_INVALID_ARGUMENT (NULL, non-positive counts, a layer
 * outside the given counts).
 */
cb_status cb_select_layers(const cb_head_map *map, const double *r2, int32_t n_tgt_layers, int32_t n_src_layers,
                           int32_t k, int32_t *selected, double *score);

/*
 * Attention-aligned sensitivities (Sec. 3.3, Eq. attentionlinearization and
 * Eq. sensitivity).  For every sequence, target layer l and KV head h of `tgt`
 * (K = kv 0, V = kv 1), every boundary c = boundaries[k] (the position of the
 * first query after the prefix [0, c)) and every query head u of h's group:
 *   a_i = softmax_i(q_u . k_i / sqrt(d)) over the keys i = 0 .. c,  o_u = sum_i a_i v_i,
 * and for the sampled prefix positions E_c = {i < c : i mod sample_stride = 0}
 *   p^V_i = sum_u a_i^2,   p^K_i = sum_u a_i^2 |v_i - o_u|^2 |q_u|^2 / d;
 * every boundary's p^K and p^V are scaled to unit mass over E_c (a boundary
 * with zero mass adds nothing) and the boundaries are summed:
 *   r[((l*2 + z)*H + h) * r_row_stride + seq*seq_len + tok] = r^K (z = 0) or r^V (z = 1),
 * written for every token of the call (0 outside every E_c) -- the row order
 * of the maps of a plan built on all target heads, so weight_row = map index.
 * Sequences are independent: a batch of sequences is one call with r offset
 * to its first column.  tgt: the target cache (head_dim d in {64, 128}); q:
 * n_layers and n_seqs equal to tgt's, n_qheads = G * n_heads with G a power of
 * two <= 32, 1 <= n_bounds <= 64 and n_bounds * G <= 256; boundaries: host
 * array of n_bounds strictly increasing positions in [0, seq_len).  r: device
 * fp32, r_row_stride >= n_seqs * seq_len.  Scores and outputs are fp32 sums of
 * exact bf16 products; a and o enter the products as two bf16 terms each.
 * Errors: CB_ERR_INVALID_ARGUMENT, CB_ERR_SHAPE, CB_ERR_MISALIGNED,
 * CB_ERR_UNSUPPORTED, CB_ERR_DEVICE.
 */
cb_status cb_attn_sensitivity(const cb_cache *tgt, const cb_queries *q, const int32_t *boundaries,
                              int32_t sample_stride, float *r, int64_t r_row_stride, void *stream);

/*
 * Attention-aligned weights (Sec. 3.3): for each of n_rows rows of r (as
 * written by cb_attn_sensitivity over all calibration batches), over the n
 * calibration rows (positions tok with tok mod sample_stride = 0 of all
 * n_seqs sequences):
 *   r_i <- r_i / mean(r)   (all ones if the mean is zero),
 *   CV^2 = mean((r_i - 1)^2),  tau = min(n, 2 p),
 *   alpha = 1 if CV^2 = 0, else min(1, sqrt((n / tau - 1) / CV^2)),
 *   w_i = 1 + alpha (r_i - 1),
 * the largest alpha whose Kish effective sample size n / (1 + alpha^2 CV^2) is
 * at least tau; positions that are not calibration rows get w = 0, so the
 * statistics calls see only the sampled tokens.  p: the map's input width
 * (k d_s).  r, w: device fp32 with row strides >= n_seqs * seq_len; alpha:
 * device fp32 [n_rows].  Sums in fp64, one workgroup per row.
 */
cb_status cb_attn_weights(int32_t n_rows, int32_t n_seqs, int32_t seq_len, int32_t sample_stride, const float *r,
                          int64_t r_row_stride, int32_t p, float *w, int64_t w_row_stride, float *alpha,
                          void *stream);

/* cb_rope styles: which channels of a head form the rotated pairs. */
#define CB_ROPE_HALF_SPLIT 0   /* (i, i + d/2): the split used by Qwen3 and most decoders */
#define CB_ROPE_INTERLEAVED 1  /* (2i, 2i + 1): RoFormer's original pairing               */

/*
 * Rotary frequency table: table[pos][i] = (cos, sin)(pos * theta^(-2 i / d))
 * for 0 <= pos < n_pos and i < d / 2, as fp32 pairs ([n_pos][d/2][2], device,
 * caller-owned).  Angles and sines are formed in fp64.  d even, 2..256.
 */
cb_status cb_rope_table(double theta, int32_t head_dim, int32_t n_pos, float *table, void *stream);

/*
 * A model's rotary transform, as the calls below take it.  The library checks
 * head_dim against the cache it is applied to and n_pos against the positions
 * it needs (CB_ERR_SHAPE), so a table built for another head width or too few
 * positions is refused before anything is enqueued.
 */
typedef struct cb_rope_spec {
    const float *table;     /* cb_rope_table(theta, head_dim, n_pos) output: device, 16-byte aligned */
    int32_t head_dim;       /* the head_dim the table was built for */
    int32_t n_pos;          /* its rows: positions 0 .. n_pos - 1 */
    int32_t style;          /* CB_ROPE_HALF_SPLIT or CB_ROPE_INTERLEAVED */
    int32_t pos_offset;     /* position of token 0 of every sequence (>= 0) */
} cb_rope_spec;

/*
 * Rotary position transform of the keys (Sec. 2.1; Sec. 3.1: the maps act in
 * content coordinates, so source RoPE is removed before fitting and the
 * target's RoPE is applied to the mapped keys).  For every K row (kv = 0) of
 * `in`, at position pos = rope->pos_offset + tok, each channel pair
 * (rope->style) is turned by the table's angle of pos (negated when `inverse`
 * is non-zero):
 *   (a, b) -> (a cos - b sin, b cos + a sin),
 * in fp32 from the exact bf16 values, rounded once to bf16, and written to the
 * same element of `out`.  V rows (kv = 1) carry no position: they are copied
 * when out->data differs from in->data and left alone otherwise.  `out` may be
 * `in` (same data and strides) for an in-place transform; other overlaps are
 * not allowed.  in and out: the same geometry, head_dim a multiple of 16 up to
 * 256 and equal to rope->head_dim; rope->n_pos >= pos_offset + seq_len.
 * cb_stats_accumulate_rope and cb_apply_rope fold the same transform into
 * their reads and writes.
 */
cb_status cb_rope(const cb_cache *in, const cb_cache *out, const cb_rope_spec *rope, int32_t inverse,
                  void *stream);

/*
 * cb_stats_accumulate on keys that carry rotary positions (Sec. 2.1, Sec. 3.1:
 * the maps are fitted in content coordinates, RoPE removed before
 * regression).  For K maps (kv = 0) the source row at position pos =
 * src_rope->pos_offset + tok is turned back by the sender's angle of pos and
 * the target row by the target's angle (tgt_rope), each in fp32 from the
 * exact bf16 values and rounded to bf16 exactly as cb_rope(inverse) writes
 * it; the moments are then those of cb_stats_accumulate on the de-rotated
 * rows (V maps are unchanged).  Either spec may be NULL (that side is not
 * turned).  Checks as cb_stats_accumulate, plus src_rope->head_dim = d_s,
 * tgt_rope->head_dim = d_t and n_pos >= pos_offset + seq_len (CB_ERR_SHAPE).
 * Single-layer plans turn the rows as they land in LDS, inside the moments
 * kernel (d_s = d_t = 64 or 128; other widths CB_ERR_UNSUPPORTED).  A
 * multi-layer plan stages each calibration row many times (once per task of
 * every map that reads it), so there the calibration rows of the K maps are
 * first gathered once, de-rotated, into a compact workspace the plan keeps
 * (every sample_stride-th token only), and the moments kernel reads them
 * from there.
 */
cb_status cb_stats_accumulate_rope(cb_plan *plan, const cb_cache *src, const cb_cache *tgt, const float *weights,
                                   int64_t w_row_stride, float *G, float *C, const cb_rope_spec *src_rope,
                                   const cb_rope_spec *tgt_rope, void *stream);

/*
 * Online mapping (Sec. 1 pipeline; Sec. 2.3 Eq. support-cost): for every map
 * m of the plan and every token of the sender cache,
 *   tgt_out(tgt_layer, kv, seq, tgt_head, tok, :) =
 *       RNE_bf16( [ src(src_layer, kv, seq, src_head, tok) , 1 ] maps[m] )
 * maps [n_maps][P][d_t] fp32 (bias in the last row).  src has the plan's source
 * geometry, tgt_out its target geometry, both with the same n_seqs and
 * seq_len.  Target positions not named by any map are left untouched; a plan
 * that maps some target more than once is rejected (CB_ERR_INVALID_ARGUMENT,
 * before anything is enqueued).  The
 * coefficients are split into two bf16 terms and products accumulate in fp32,
 * then the bias is added and the sum is rounded once to bfloat16.
 */
cb_status cb_apply(cb_plan *plan, const float *maps, const cb_cache *src, const cb_cache *tgt_out,
                   void *stream);

/*
 * Online mapping with the rotary transforms fused (Sec. 1 pipeline; Sec. 2.1,
 * Sec. 3.1: the maps act in content coordinates, so the sender's RoPE is
 * removed from its keys before mapping and the mapped keys receive the target
 * model's RoPE before decoding).  Identical to cb_apply for V maps (kv = 1).
 * For K maps (kv = 0), at position pos = pos_offset + tok:
 *   src_rope (may be NULL): the source row is first turned back by the
 *     sender's angle of pos (inverse transform), in fp32 from the exact bf16
 *     values, and rounded to bf16 as cb_rope(inverse) would write it;
 *   tgt_rope (may be NULL): the fp32 sum s = x W + b has its channel pairs
 *     turned by the target's angle of pos, (a, b) -> (a cos - b sin,
 *     b cos + a sin), in fp32 before the single rounding to bfloat16 (cb_apply
 *     followed by cb_rope rounds twice).
 * src_rope->head_dim must be the plan's d_s and tgt_rope->head_dim its d_t
 * (CB_ERR_SHAPE otherwise, as for a table with fewer than pos_offset +
 * seq_len rows).  Single-layer plans read each source row once and de-rotate
 * it on the way into LDS (d_s = 64 or 128).  A multi-layer plan reads each
 * source row once per map that selects its layer, so there the K rows of the
 * batch are de-rotated once, by a rotation pass into a workspace the plan
 * keeps (sized to the largest batch seen), before the mapping kernel; the
 * target rotation is fused into its epilogue.  Errors as cb_apply, and
 * CB_ERR_UNSUPPORTED for d_s = 96 with a source rotation on a single-layer
 * plan.
 */
cb_status cb_apply_rope(cb_plan *plan, const float *maps, const cb_cache *src, const cb_cache *tgt_out,
                        const cb_rope_spec *src_rope, const cb_rope_spec *tgt_rope, void *stream);

/*
 * Multi-layer mapper support (Sec. 3.2, Eq. localfeature with k selected
 * source layers S_l, chosen for instance by cb_select_layers): map m predicts
 * target (tgt_layer[m], tgt_head[m], kv[m]) from the source rows of layers
 * src_layers[m*k + 0], ..., src_layers[m*k + k-1] (distinct, in that order)
 * at head src_head[m] and the same component, concatenated:
 *   x~ = [ x_0 ; x_1 ; ... ; x_{k-1} ; 1 ]      (P = k d_s + 1)
 * maps[m] is then a P x d_t fp32 matrix whose rows i d_s .. (i+1) d_s - 1 act
 * on x_i and whose last row is the bias.  Host arrays, read by
 * cb_plan_create_multi only.
 */
typedef struct {
    int32_t n_maps;
    int32_t k;
    const int32_t *tgt_layer;
    const int32_t *tgt_head;
    const int32_t *kv;
    const int32_t *src_layers;  /* [n_maps][k] */
    const int32_t *src_head;
    const int32_t *weight_row;
} cb_head_map_multi;

/*
 * Plan for multi-layer maps (1 <= k <= 32, d_s = d_t = 128).  The calibration
 * rows of every cb_stats_accumulate call on this plan are the tokens tok with
 * tok mod sample_stride == 0 of every sequence (Sec. 4.1 samples every fourth
 * token); other tokens are never read.  With such a plan, cb_stats_zero and
 * cb_stats_accumulate compute G [n_maps][P][P] and C [n_maps][P][d_t] for the
 * multi-layer feature, with the arguments, accuracy and symmetry of the
 * single-layer calls and no token limit; the products run on the matrix cores
 * (the work grows as P^2 per row).  G and C must not overlap other buffers of
 * the call.  Solve with cb_ridge_solve_ws.  cb_apply maps a sender cache with
 * the P x d_t maps, every token: out = RNE_bf16([x_0, ..., x_{k-1}, 1] maps[m])
 * (coefficients as two bf16 terms, fp32 sums and bias, one rounding); the
 * rows of one source (layer, kv, head) must span fewer than 4 GiB
 * (2 ((n_seqs - 1) s_seq + (seq_len - 1) s_tok + 128) bytes), else
 * CB_ERR_UNSUPPORTED (apply in smaller batches).  Maps of one (kv, source
 * head) with equal source-layer sets are applied in pairs that read their
 * source rows once.  The two-pass centered calls (cb_stats_means
 * without sq, cb_stats_accumulate_centered) take such a plan too.  Errors
 * as in cb_plan_create, plus CB_ERR_INVALID_ARGUMENT for a source layer
 * selected twice by one map.
 */
cb_status cb_plan_create_multi(const cb_head_map_multi *map, const cb_cache *src_geom, const cb_cache *tgt_geom,
                               int32_t sample_stride, cb_plan **out);

/*
 * Batched ridge solve for any feature width (Sec. 3.1, Eq. closedform; the
 * multi-layer feature of Sec. 3.2 gives P = k d_s + 1):  maps[m] =
 * (G[m] + lambda_m D)^{-1} C[m], with the arrays, flags, lambda_m and info of
 * cb_ridge_solve (G symmetric).  P <= 129 runs cb_ridge_solve and ignores the
 * workspace.  Otherwise (P <= 4097, d_t in {64, 96, 128}) each system is
 * factored in fp64 in `workspace` (device memory owned by the caller, 8-byte
 * aligned, at least cb_ridge_solve_workspace_bytes(P, d_t, 1) bytes): a
 * left-looking blocked Cholesky M = L L^T in 32-column panels, then the
 * forward and back substitutions for the d_t right-hand sides, one workgroup
 * of 256 threads per system; the systems are processed in batches of
 * workspace_bytes / cb_ridge_solve_workspace_bytes(P, d_t, 1).  info[m] = 0, or
 * the 1-based column of the first pivot that is not positive and finite
 * (maps[m] zero-filled).  Errors: CB_ERR_SHAPE (workspace too small), else as
 * cb_ridge_solve.
 */
cb_status cb_ridge_solve_ws(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C, float lambda,
                            uint32_t flags, void *workspace, int64_t workspace_bytes, float *maps, int32_t *info,
                            void *stream);

/* Workspace bytes cb_ridge_solve_ws needs to solve n_systems systems at once (0 for P <= 129). */
int64_t cb_ridge_solve_workspace_bytes(int32_t P, int32_t d_t, int32_t n_systems);

/*
 * Allocation-free wide ridge solve, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the solve of cb_ridge_solve_ws -- same arguments minus
 * the workspace, same arithmetic, identical results -- with the factors in a
 * fixed device array of cb_ridge_solve_noalloc_max_bytes() bytes (128 MiB)
 * that every GPU the library runs on holds until the process ends.  The
 * systems are solved in batches of that size divided by
 * cb_ridge_solve_workspace_bytes(P, d_t, 1).  No call allocates; the first call
 * on a device looks up the array's address there (make it before a graph
 * capture).  The array keeps the last call's contents; calls that overlap on
 * one GPU (several streams or threads) race on it and must be serialized.
 * P <= 129 runs cb_ridge_solve (no scratch).  Errors as cb_ridge_solve_ws, and
 * CB_ERR_UNSUPPORTED when one system needs more than the array holds
 * ((P^2 + P d_t) * 8 bytes: P > 4032 at d_t = 128).
 */
cb_status cb_ridge_solve_noalloc(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C,
                                 float lambda, uint32_t flags, float *maps, int32_t *info, void *stream);

/* Bytes of the fixed device array of cb_ridge_solve_noalloc. */
int64_t cb_ridge_solve_noalloc_max_bytes(void);

/* Feature width P of a plan's maps (d_s + 1, or k d_s + 1) and its k. */
cb_status cb_plan_feature_width(const cb_plan *plan, int32_t *P, int32_t *k);

/* Static name of a status code. */
const char *cb_status_string(cb_status status);

/* Message describing the last error returned to the calling thread ("" if none). */
const char *cb_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CACHEBRIDGE_H */

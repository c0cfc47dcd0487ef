// cb_internal.h -- structures shared by the host library and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cachebridge.h"

namespace cb {

// One unit of the precomputed read plan of the statistics: up to two maps
// that are processed by one workgroup over a token range.  When both maps read
// the same source block (a source layer feeding two target layers) the source
// rows are loaded once ("shared").
struct StatsItem {
    int32_t n_slots;      // 1 or 2
    int32_t shared_x;     // slot 1 reads slot 0's source rows
    int32_t map[2];
    int32_t src_layer[2], src_head[2], kv[2];
    int32_t tgt_layer[2], tgt_head[2], wrow[2];
    int32_t own_y[2];     // this slot's map carries the target sums of its (target block, weight row)
};

// One source block (src_layer, kv, src_head) and up to two target maps that
// read it, for the online application.
struct ApplyGroup {
    int32_t n_slots;
    int32_t src_layer, src_head, kv;
    int32_t map[2];
    int32_t tgt_layer[2], tgt_head[2];
};

struct Strides {
    int64_t layer, kv, seq, head, tok;
};

// Exact unsigned division by a runtime constant d >= 1 (round-up multiplier
// method of Granlund and Montgomery, "Division by invariant integers using
// multiplication", 1994): q = (t + ((n - t) >> sh1)) >> sh2, t = mulhi(m, n).
struct FastDiv {
    uint32_t d, m, sh1, sh2;
};

inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    FastDiv f;
    f.d = d;
    f.m = (uint32_t)((((1ull << 32) * ((1ull << l) - d)) / d) + 1);
    f.sh1 = l > 0 ? 1u : 0u;
    f.sh2 = l > 0 ? l - 1 : 0u;
    return f;
}

struct StatsArgs {
    const uint16_t *src;
    const uint16_t *tgt;
    const float *w;
    Strides ss, ts;
    int64_t w_row_stride;
    uint32_t seq_len;     // tokens per sequence
    FastDiv TPS;          // token tiles per sequence (the last one may be partial)
    int32_t n_tiles;      // token tiles in this call (n_seqs * TPS)
    int32_t chunk_tiles;  // tiles per work unit
    int32_t n_chunks;
    int32_t n_items;
    const StatsItem *items;
    float *partials;      // [n_chunks * n_items][2][slot_floats]
    const void *zero;     // >= 256 zero bytes: source of the weights of absent tokens
    const double *sums;   // centered statistics only: [n_maps][1 + d_s + d_t] = (sum w, sum w x, sum w y)
    int32_t bias_sums;    // centered kernels: 1 = also sum w and w y (the shifted form needs them)
    // Rotary de-rotation of the K rows as they land (the rope variant of the
    // kernel only): tables [n_pos][d/2][2] (cos, sin) of the source and the
    // target (both valid pointers), position of token 0, and which side turns.
    const float *rope_tab[2];
    int32_t rope_pos[2];
    int32_t rope_on[2];
};

struct ReduceArgs {
    const float *partials;
    const int32_t *map_item;  // [n_maps]
    const int32_t *map_slot;  // [n_maps]
    const int32_t *map_yown;  // [n_maps]: the map whose means partial holds this map's target sums
    int32_t n_items, n_chunks, n_maps;
    float *G, *C;         // plain: G [n][P][P], C [n][P][d_t]; centered: A [n][d_s][d_s], B [n][d_s][d_t]
    double *sums;         // centered: read; means: added to.  [n_maps][1 + d_s + d_t] = (sum w, sum w x, sum w y)
    double *sq;           // means only, optional: added to.  [n_maps][d_s + d_t] = (sum w x^2, sum w y^2)
    double *resid;        // centered, optional: added to.  [n_maps][1 + d_s + d_t] = (sum w, sum w (x - mu), sum w y)
};

struct ApplyArgs {
    const uint16_t *src;
    uint16_t *out;
    Strides ss, os;
    FastDiv T;
    int32_t N;            // tokens (n_seqs * seq_len)
    int32_t tile_tokens;  // tokens per workgroup
    int32_t n_tiles;      // per group
    const ApplyGroup *groups;
    const uint16_t *w_hi; // [n_maps][d_t][d_s] bf16, transposed maps
    const uint16_t *w_lo;
    const float *bias;    // [n_maps][d_t]
    const float *rope_table;  // NULL, or the target's (cos, sin) [n_pos][d_t/2][2]: K outputs are rotated
    int32_t rope_style;       // 0: pairs (i, i + d_t/2), 1: pairs (2i, 2i + 1)
    int32_t rope_pos_offset;  // position of token 0 of every sequence
    const float *src_rope_table;  // NULL, or the sender's table [n_pos][d_s/2][2]: K source rows are turned back
    int32_t src_rope_style;
    int32_t src_rope_pos_offset;
};

// Attention-aligned sensitivities of one call (host side of the launch).
struct AttnLaunch {
    const uint16_t *kv;
    Strides ts;
    const uint16_t *q;
    int64_t q_strides[4];     // layer, seq, boundary, query head (elements)
    int32_t n_layers, n_heads, G, n_bounds, seq_len, n_seqs, stride, d;
    const int32_t *bounds;    // host, n_bounds increasing positions
    float *r;
    int64_t r_row_stride;
};

// Rotary transform of one call (host side of the launch).
struct RopeLaunch {
    const uint16_t *in;
    uint16_t *out;
    Strides is, os;
    const float *table;       // [n_pos][d/2][2] (cos, sin)
    int32_t n_layers, n_heads, n_seqs, seq_len, d, style, pos_offset, inverse, copy_v;
    int32_t pos_step;         // token t of a sequence is at position pos_offset + t * pos_step
};

// One workgroup task of the multi-layer statistics (feature x~ = [x_0; ...;
// x_{k-1}; 1], blocks of 128 channels): for map `map`, the products of the
// folded rows of feature blocks rows[0], rows[1] with the exact columns of
// feature blocks cols[0], cols[1] (block k is the target block; it is only
// ever cols[1]), over every calibration row of a call.  Cell (rows[a],
// cols[b]) is written when bit 2a + b of cell_mask is set.  The distinct
// blocks of the task are staged in LDS slots 0..n_lds-1.
struct MultiTask {
    int32_t map, n_lds;
    int32_t flags;            // 1, 2: owns sum w x of rows[0], rows[1]; 4: owns sum w; 8: owns sum w y
    int32_t wrow, kv, tgt_layer, tgt_head, src_head;
    int32_t rows[2], cols[2];
    int32_t row_slot[2], col_slot[2];
    int32_t cell_mask;
    int32_t slot_layer[4];    // source layer staged in each slot, -1: the target block
};

struct MultiArgs {
    const uint16_t *src;
    const uint16_t *tgt;
    const float *w;
    Strides ss, ts;
    int64_t w_row_stride;
    uint32_t seq_len;         // tokens per sequence
    uint32_t stride;          // calibration rows: tokens tok = r * stride
    uint32_t rows_per_seq;    // ceil(seq_len / stride)
    FastDiv TPS;              // row tiles per sequence (the last one may be partial)
    int32_t n_tiles;          // row tiles in this call
    int32_t chunk_tiles;      // tiles between two flushes into G, C
    int32_t n_tasks, per_xcd; // tasks; ceil(n_tasks / 8)
    int32_t k, P, d_t;
    const MultiTask *tasks;
    const void *zero;         // >= 256 zero bytes
    float *G, *C;             // centered: A [n][P-1][P-1], B [n][P-1][d_t]
    const double *sums;       // centered only: [n][P + d_t] = (sum w, sum w x, sum w y)
    double *resid;            // centered, optional: added to.  [n][P + d_t] = (sum w, sum w (x - mu), sum w y)
    // NULL, or compact de-rotated calibration rows of the K maps, [layer][seq][head][row][d]:
    // K tasks read their source / target blocks there (tok stride = one calibration row)
    const uint16_t *srck, *tgtk;
    Strides ssk, tsk;
};


// One map of the multi-layer application.
struct ApplyMultiMap {
    int32_t tgt_layer, tgt_head, kv, src_head;
};

// Pass 1 of the centered multi-layer statistics: per map, sums of w, w x over
// its k source blocks and w y over its target block, on the calibration rows.
struct MeansMultiArgs {
    const uint16_t *src;
    const uint16_t *tgt;
    const float *w;
    Strides ss, ts;
    int64_t w_row_stride;
    int32_t n_seqs, seq_len, stride, rows_per_seq;
    int32_t n_maps, k, d_t;
    const ApplyMultiMap *maps;
    const int32_t *layers;    // [n_maps][k]
    const int32_t *wrow;      // [n_maps]
    double *sums;             // [n_maps][1 + 128 k + d_t], added to
    int32_t tgt_only;         // 1: only sum w and sum w y (the target block)
};

struct ApplyMultiArgs {
    const uint16_t *src;
    uint16_t *out;
    Strides ss, os;
    FastDiv T;                // tokens per sequence
    int64_t N;                // tokens (n_seqs * seq_len)
    int32_t k, n_maps;
    int32_t n_tiles;          // 256-token tiles per map
    int32_t n_tasks;          // n_maps * n_tiles (map, tile) tasks
    int32_t per_xcd;          // tasks per XCD (a contiguous run)
    const ApplyMultiMap *maps;
    const int32_t *order;     // [n_maps] maps in visiting order
    const int32_t *src_layers;// [n_maps][k]
    const uint16_t *wfrag;    // W^T as MFMA fragments, [n_maps][k][8][4][2][64][8] bf16 (hi, lo planes)
    const float *bias;        // [n_maps][128]
    const uint16_t *srck;     // NULL, or the K maps' source view (a de-rotated copy of the sender's keys)
    Strides ssk;              // its strides (kv unused)
    const float *rope_table;  // NULL, or the target's (cos, sin) [n_pos][64][2]: K outputs are rotated
    int32_t rope_style;       // 0: pairs (i, i + 64), with the permuted fragments; 1: pairs (2i, 2i + 1)
    int32_t rope_pos_offset;
    // NULL, or the paired form: tasks are (pair, tile), n_tasks = n_pairs * n_tiles.  Record of a pair
    // (pair_stride int32): [0] map A, [1] map B or -1, [2] staged blocks nb (<= 2k), [3] unused,
    // [4 + j] (j < nb) 4 * source layer + (A uses it) + 2 (B uses it), ascending layers,
    // [4 + 2k + q] (q < k) A's block index of its q-th used block, [4 + 3k + q] the same for B.
    const int32_t *pairs;
    int32_t n_pairs, pair_stride;
};

// Launchers (return hipError_t of the launch).
hipError_t launch_rope_table(int32_t d, int32_t n_pos, double theta, float *table, hipStream_t s);
hipError_t launch_rope(const RopeLaunch &L, hipStream_t s);
hipError_t launch_attn_sensitivity(const AttnLaunch &L, hipStream_t s);
hipError_t launch_attn_weights(int32_t n_rows, int32_t n_seqs, int32_t seq_len, int32_t stride, const float *r,
                               int64_t r_row_stride, int32_t p, float *w, int64_t w_row_stride, float *alpha,
                               hipStream_t s);
hipError_t launch_stats(int d_s, int d_t, const StatsArgs &a, hipStream_t s);
// style: 0 half split, 1 interleaved; d_s = d_t = 64 or 128
hipError_t launch_stats_rope(int d, int style, const StatsArgs &a, hipStream_t s);
hipError_t launch_reduce(int d_s, int d_t, const ReduceArgs &a, hipStream_t s);
hipError_t launch_stats_centered(int d_s, int d_t, const StatsArgs &a, hipStream_t s);
hipError_t launch_reduce_centered(int d_s, int d_t, const ReduceArgs &a, hipStream_t s);
hipError_t launch_means(int d_s, int d_t, const StatsArgs &a, bool sq, hipStream_t s);
hipError_t launch_probe_r2(int32_t n_maps, int32_t d_s, int32_t d_t, const double *sums, const double *sq,
                           const float *A, const float *B, const float *maps, double *r2, hipStream_t s);
hipError_t launch_means_reduce(int d_s, int d_t, const ReduceArgs &a, hipStream_t s);
hipError_t launch_solve_centered(int32_t n_maps, int32_t d_s, int32_t d_t, const double *sums, const float *A,
                                 const float *B, float lambda, uint32_t flags, float *maps, int32_t *info,
                                 hipStream_t s);
hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t s);
// Shifted centered form: turns moments about the shift means into moments
// about the data's means, and the residual sums into (sum w, sum w x, sum w y).
hipError_t launch_shift_finish(int32_t n_maps, int32_t d_x, int32_t d_t, const double *shift, double *sums, float *A,
                               float *B, hipStream_t s);
hipError_t launch_stats_multi(const MultiArgs &a, hipStream_t s);
hipError_t launch_stats_multi_centered(const MultiArgs &a, hipStream_t s);
hipError_t launch_means_multi(const MeansMultiArgs &a, hipStream_t s);
hipError_t launch_split_maps_frag(int32_t n_maps, int32_t k, const float *maps, uint16_t *wfrag, float *bias,
                                  int perm, hipStream_t s);
hipError_t launch_apply_multi(const ApplyMultiArgs &a, int32_t n_cu, hipStream_t s);
int64_t solve_blocked_bytes_per_system(int32_t P, int32_t d_t);
// csums != nullptr: centered systems (A, B of the feature without bias entry,
// sums (sum w, sum w x, sum w y)); maps then get P + 1 rows (W, then the bias).
hipError_t launch_solve_blocked(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C, float lambda,
                                uint32_t flags, void *ws, int64_t ws_bytes, float *maps, int32_t *info,
                                hipStream_t s, const double *csums = nullptr);
constexpr int kMultiTileRows = 16;      // calibration rows per multi-layer tile
constexpr int kMultiFlushTiles = 2046;  // at most 32,736 rows summed in fp32 before a flush (a multiple of 6)
// Size of the fixed device array of the allocation-free blocked solve.
constexpr int64_t kStaticSolveScratchBytes = 128ll << 20;
hipError_t launch_solve_blocked_static(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C,
                                       float lambda, uint32_t flags, float *maps, int32_t *info, hipStream_t s);
hipError_t launch_solve(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C,
                        float lambda, uint32_t flags, float *maps, int32_t *info, hipStream_t s);
hipError_t launch_split_maps(int32_t n_maps, int32_t d_s, int32_t d_t, const float *maps,
                             uint16_t *w_hi, uint16_t *w_lo, float *bias, hipStream_t s);
hipError_t launch_apply(int d_s, int d_t, int n_groups, const ApplyArgs &a, hipStream_t s);

// Geometry of the statistics kernel, shared with the host for workspace sizing.
constexpr int kStatsTileTokens = 32;
inline int64_t stats_slot_floats(int d_s, int d_t) {
    const int rb = d_s / 32, rbt = d_t / 32;
    return (int64_t)(rb * (rb + 1) / 2 + rb * rbt) * 1024 + (int64_t)(rb + rbt + 1) * 64;
}

}  // namespace cb

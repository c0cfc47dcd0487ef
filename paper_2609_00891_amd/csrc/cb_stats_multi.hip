// cb_stats_multi.hip -- weighted augmented moments over the multi-layer
// head-local feature on gfx950.
//
// CacheBridge Sec. 3.2 (Eq. localfeature) feeds target head h of layer l the
// concatenation of its assigned source head from each of the k selected
// source layers S_l.  With x~ = [x_0; ...; x_{k-1}; 1] (P = 128 k + 1) the fit
// needs the augmented moments of Sec. 3.4 (Eq. fusedstats)
//     G = sum_r w_r x~_r x~_r^T      C = sum_r w_r x~_r y_r^T
// over the calibration rows r (every `stride`-th token, Sec. 4.1).  At
// k = 8 that is 2.4 MFLOP per map and row against 256 bytes of target row:
// the work is a dense contraction over rows and runs on the matrix cores.
//
// Decomposition.  The feature splits into blocks of 128 channels: source
// blocks 0..k-1 and the target block k.  The work of a map is the set of
// cells (i, j) of the block matrix with i, j < k (each unordered pair once:
// G is symmetric, so a cell may be computed as (i, j) or as (j, i)) and the
// cells (i, k) of C.  A task is a rectangle: two row blocks times two column
// blocks, four cells (some marked unused when the cells do not pack evenly).
// Every task does the same work, so the tasks of a map, launched together on
// one XCD, move through the rows in step and read each staged row while it
// is still in L2.  One workgroup runs one task over every calibration row of
// the call and adds its fp32 sums into G and C itself (it is the only writer
// of those elements): no partial sums, no reduction pass, no atomics.
//
// Per workgroup: eight waves, two per SIMD.  Wave w owns the 32 rows
// 32 (w mod 4) .. + 31 of row block rows[w / 4] and all eight 32-column
// blocks of the two column blocks: 8 accumulator tiles, 16
// v_mfma_f32_32x32x16_bf16 per 16-row K step.  It folds the fp32 weight
// into its x fragment and splits w x into hi = RNE_bf16(w x) and lo =
// RNE_bf16(w x - hi); the column operands are the exact bf16 rows.  The two
// waves of a SIMD (w and w + 4) take each tile's steps in opposite orders
// (products then fold, fold then products), so one folds while the other
// keeps the matrix core busy.
//
// Staging.  A tile is 16 calibration rows of one sequence.  Its blocks (the
// distinct blocks among its two row and two column blocks) move HBM -> LDS
// by global_load_lds_dwordx4, issued by waves 0..3, through a six-stage
// ring, five tiles ahead; each 16-byte chunk c of row t sits at chunk
// c ^ 4(t mod 4) so the transposed operand reads (ds_read_b64_tr_b16) are
// conflict free.  Rows past the end of a sequence repeat its last row with
// weight zero.
//
// Flush.  Every at most 2,046 tiles (32,736 rows) and at the end of the call
// each wave adds its tiles into G (and C): a tile above the diagonal goes to
// its block and, transposed through LDS, to the mirrored block; a tile on the
// diagonal contributes its upper triangle to both triangles; tiles below the
// diagonal (inside a diagonal block) are dropped.  G stays exactly symmetric.
#include "cb_stats_kernel.h"

namespace cb {
namespace {

struct MCfg {
    static constexpr int KT = kMultiTileRows;      // 16 rows per tile: one K step
    static constexpr int ROW = 256;                // bytes per 128-channel row
    static constexpr int BLK = KT * ROW;           // 4096 bytes per block and stage
    static constexpr int MAXS = 4;                 // LDS slots (two row and two column blocks)
    static constexpr int OFF_W = MAXS * BLK;       // weights of the tile: [KT] fp32
    static constexpr int STAGE = OFF_W + KT * 4;
    static constexpr int NST = 6;                  // ring stages (one per iteration of a loop trip)
    static constexpr int TRS = 33;                 // row stride (floats) of the transpose scratch
    static constexpr int NW = 8;                   // waves: two per SIMD
    static constexpr int OFF_T = NST * STAGE;
    static constexpr int OFF_E = OFF_T + NW * 32 * TRS * 4;  // centered: each wave's row sums e [32]
    static constexpr int LDS = OFF_E + NW * 32 * 4;
    static_assert(KT == 16, "one tile is one MFMA K step");
    static_assert(LDS <= 160 * 1024, "the ring must fit in LDS");
};

// Per-workgroup state that is uniform across the wave.
struct MultiCtx {
    const uint16_t *slot_base[MCfg::MAXS];   // (layer, kv, head) base of each staged block
    int64_t s_row, t_row;                    // elements between calibration rows (source, target view)
    int64_t s_seq, t_seq;                    // elements between sequences
};

// All copies of one tile by one wave, under one save of M0 (and EXEC): NL
// 16-byte copies into consecutive 4 KiB LDS slots starting at m0, then a
// dword copy of the weights by lanes 0..3 into wm0 + 4 lane.  M0 and EXEC are
// restored before the statement ends, so the compiler's use of them is
// unaffected.
template <int NL>
__device__ __forceinline__ void dma_tile(const uint32_t (&voff)[NL], const void *const (&base)[NL], uint32_t m0,
                                         const void *wg, uint32_t wm0) {
    uint32_t keep_m0;
    uint64_t keep_exec;
#define CB_CP(i) "global_load_lds_dwordx4 %" #i "_v, %" #i "_s\n\t"
    if constexpr (NL == 1) {
        asm volatile("s_mov_b32 %[km], m0\n\ts_mov_b32 m0, %[m0]\n\t"
                     "global_load_lds_dwordx4 %[v0], %[s0]\n\t"
                     "s_mov_b32 m0, %[wm]\n\ts_mov_b64 %[ke], exec\n\ts_mov_b64 exec, 15\n\t"
                     "global_load_lds_dword %[wg], off\n\ts_mov_b64 exec, %[ke]\n\ts_mov_b32 m0, %[km]"
                     : [km] "=&s"(keep_m0), [ke] "=&s"(keep_exec)
                     : [m0] "s"(m0), [v0] "v"(voff[0]), [s0] "s"(base[0]), [wm] "s"(wm0), [wg] "v"(wg)
                     : "memory");
    } else if constexpr (NL == 2) {
        asm volatile("s_mov_b32 %[km], m0\n\ts_mov_b32 m0, %[m0]\n\t"
                     "global_load_lds_dwordx4 %[v0], %[s0]\n\ts_add_u32 m0, m0, 0x1000\n\t"
                     "global_load_lds_dwordx4 %[v1], %[s1]\n\t"
                     "s_mov_b32 m0, %[wm]\n\ts_mov_b64 %[ke], exec\n\ts_mov_b64 exec, 15\n\t"
                     "global_load_lds_dword %[wg], off\n\ts_mov_b64 exec, %[ke]\n\ts_mov_b32 m0, %[km]"
                     : [km] "=&s"(keep_m0), [ke] "=&s"(keep_exec)
                     : [m0] "s"(m0), [v0] "v"(voff[0]), [s0] "s"(base[0]), [v1] "v"(voff[1]), [s1] "s"(base[1]),
                       [wm] "s"(wm0), [wg] "v"(wg)
                     : "memory", "scc");
    } else if constexpr (NL == 3) {
        asm volatile("s_mov_b32 %[km], m0\n\ts_mov_b32 m0, %[m0]\n\t"
                     "global_load_lds_dwordx4 %[v0], %[s0]\n\ts_add_u32 m0, m0, 0x1000\n\t"
                     "global_load_lds_dwordx4 %[v1], %[s1]\n\ts_add_u32 m0, m0, 0x1000\n\t"
                     "global_load_lds_dwordx4 %[v2], %[s2]\n\t"
                     "s_mov_b32 m0, %[wm]\n\ts_mov_b64 %[ke], exec\n\ts_mov_b64 exec, 15\n\t"
                     "global_load_lds_dword %[wg], off\n\ts_mov_b64 exec, %[ke]\n\ts_mov_b32 m0, %[km]"
                     : [km] "=&s"(keep_m0), [ke] "=&s"(keep_exec)
                     : [m0] "s"(m0), [v0] "v"(voff[0]), [s0] "s"(base[0]), [v1] "v"(voff[1]), [s1] "s"(base[1]),
                       [v2] "v"(voff[2]), [s2] "s"(base[2]), [wm] "s"(wm0), [wg] "v"(wg)
                     : "memory", "scc");
    } else {
        asm volatile("s_mov_b32 %[km], m0\n\ts_mov_b32 m0, %[m0]\n\t"
                     "global_load_lds_dwordx4 %[v0], %[s0]\n\ts_add_u32 m0, m0, 0x1000\n\t"
                     "global_load_lds_dwordx4 %[v1], %[s1]\n\ts_add_u32 m0, m0, 0x1000\n\t"
                     "global_load_lds_dwordx4 %[v2], %[s2]\n\ts_add_u32 m0, m0, 0x1000\n\t"
                     "global_load_lds_dwordx4 %[v3], %[s3]\n\t"
                     "s_mov_b32 m0, %[wm]\n\ts_mov_b64 %[ke], exec\n\ts_mov_b64 exec, 15\n\t"
                     "global_load_lds_dword %[wg], off\n\ts_mov_b64 exec, %[ke]\n\ts_mov_b32 m0, %[km]"
                     : [km] "=&s"(keep_m0), [ke] "=&s"(keep_exec)
                     : [m0] "s"(m0), [v0] "v"(voff[0]), [s0] "s"(base[0]), [v1] "v"(voff[1]), [s1] "s"(base[1]),
                       [v2] "v"(voff[2]), [s2] "s"(base[2]), [v3] "v"(voff[3]), [s3] "s"(base[3]),
                       [wm] "s"(wm0), [wg] "v"(wg)
                     : "memory", "scc");
    }
#undef CB_CP
}

// Adds the 32 x 32 tile held in the wave's transpose scratch `tr` (row i at
// tr + 33 i) into global memory, two rows per lane group: mode 0 and 2 add it
// at dst (leading dimension ld), mode 2 also adds its transpose at mir, and
// mode 1 (a diagonal tile of G) adds its upper triangle to both triangles.
// The loads of two row pairs are issued before their adds, so the global
// latency is paid 8 times per tile, not 16 (the loop's operand pipeline stays
// live across a flush, which leaves no registers for more).
__device__ __forceinline__ void flush_rows(const float *tr, int lane, int mode, float *dst, float *mir, int64_t ld) {
    constexpr int FB = 2;
    const int jj = lane & 31;
#pragma unroll 1
    for (int i0 = 0; i0 < 16; i0 += FB) {
        float cur[FB], curm[FB];
#pragma unroll
        for (int it = 0; it < FB; ++it) {
            const int ii = 2 * (i0 + it) + (lane >> 5);
            cur[it] = dst[(int64_t)ii * ld + jj];
            curm[it] = mode == 2 ? mir[(int64_t)ii * ld + jj] : 0.f;
        }
#pragma unroll
        for (int it = 0; it < FB; ++it) {
            const int ii = 2 * (i0 + it) + (lane >> 5);
            const float up = tr[ii * MCfg::TRS + jj], dn = tr[jj * MCfg::TRS + ii];
            dst[(int64_t)ii * ld + jj] = cur[it] + (mode == 1 && ii > jj ? dn : up);
            if (mode == 2) mir[(int64_t)ii * ld + jj] = curm[it] + dn;
        }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// NL: blocks staged per tile (distinct blocks of the task).  HASY: the last
// of them is the target block (it is only ever the second column block).
// YS: the task also owns sum w y of its map: waves 0..3 sum w y over 32 of
// the target's channels each.
// CENTER: moments about the map's weighted means (the paper's two-pass form):
// the row operand is w (x - mu), the column operands stay the exact bf16 rows,
// and every flush subtracts e mu^T with e = sum w (x - mu) as multiplied (hi +
// lo); the outputs are A (ld P - 1) and B, with no bias row or column.
template <int NL, bool HASY, bool YS, bool CENTER, bool FOLD_FIRST>
__device__ __forceinline__ void multi_wave(const MultiArgs &a, const MultiTask &tk, const MultiCtx &c,
                                           lds_char_t *lds, int wave, int lane) {
    using K = MCfg;
    constexpr int E = 8;                        // 32-column blocks of every wave
    constexpr int PER_TILE = NL + 1;            // copy instructions per tile of a copying wave
    const int rs = wave >> 2, sub = wave & 3;   // row slot (0: rows[0], 1: rows[1]), 32-row sub-block
    const bool copier = wave < 4;               // waves 0..3 stage the tiles
    const uint32_t lds_base = (uint32_t)(uintptr_t)lds;

    // ---- copy descriptors: copying wave w moves rows 4w..4w+3 of every staged
    // block.  A cursor walks the call's tiles in order (16 rows on, or on to the
    // next sequence); tiles past the end repeat the last one with zero weights.
    const int cw = wave & 3;
    const int crow = 4 * cw + (lane >> 4);
    const uint32_t cchunk = (uint32_t)((lane & 15) ^ (4 * (crow & 3))) * 16u;
    const uint32_t sstep = (uint32_t)(c.s_row * 2);          // bytes between calibration rows
    const uint32_t tstep = (uint32_t)(c.t_row * 2);
    uint32_t voff_full[NL];                     // lane offsets of a full tile
    auto slot_y = [](int s) { return HASY && s == NL - 1; };
#pragma unroll
    for (int s = 0; s < NL; ++s) voff_full[s] = (uint32_t)crow * (slot_y(s) ? tstep : sstep) + cchunk;
    const float *wrow = a.w + (int64_t)tk.wrow * a.w_row_stride;
    const uint32_t wr = 4 * cw + (lane & 3);    // the weight row this lane copies (lanes 0..3)
    struct Cursor {
        int u;                                  // tile index
        uint32_t seq, r0;                       // sequence, first row of the tile
        int64_t soff, toff;                     // element offsets of the tile in the source / target blocks
        const float *wp;                        // weight of the tile's first row
    } cur = {0, 0u, 0u, 0, 0, wrow};
    const int64_t sadv = (int64_t)K::KT * c.s_row, tadv = (int64_t)K::KT * c.t_row;
    auto issue = [&](int st) {
        const bool live = cur.u < a.n_tiles;
        const uint32_t tmax = min((uint32_t)K::KT - 1, a.rows_per_seq - 1 - cur.r0);
        const uint32_t stage = lds_base + st * K::STAGE;
        const uint32_t row = min((uint32_t)crow, tmax);
        uint32_t voff[NL];
        const void *base[NL];
#pragma unroll
        for (int s = 0; s < NL; ++s) {
            voff[s] = tmax == K::KT - 1 ? voff_full[s] : row * (slot_y(s) ? tstep : sstep) + cchunk;
            base[s] = uniform_ptr(c.slot_base[s] + (slot_y(s) ? cur.toff : cur.soff));
        }
        const bool ok = live && wr <= tmax;
        const void *g = ok ? (const void *)(cur.wp + (int64_t)wr * a.stride) : a.zero;
        dma_tile<NL>(voff, base, __builtin_amdgcn_readfirstlane(stage + cw * 1024), g,
                     __builtin_amdgcn_readfirstlane(stage + K::OFF_W + 16 * cw));
        if (cur.u + 1 < a.n_tiles) {
            cur.r0 += K::KT;
            if (cur.r0 >= a.rows_per_seq) {
                cur.r0 = 0;
                cur.seq += 1;
                cur.soff = (int64_t)cur.seq * c.s_seq;
                cur.toff = (int64_t)cur.seq * c.t_seq;
                cur.wp = wrow + (int64_t)cur.seq * a.seq_len;
            } else {
                cur.soff += sadv;
                cur.toff += tadv;
                cur.wp += K::KT * a.stride;
            }
        }
        cur.u += 1;
    };

    // ---- operand geometry (transposed reads; see cb_stats_kernel.h)
    const int g16 = lane >> 4, j16 = lane & 15, aa = j16 & 3, kk = j16 >> 2;
    const int tok_l = 8 * (g16 >> 1) + kk;
    const int cl = 2 * (g16 & 1) + (aa >> 1);
    const uint32_t lrow = tok_l * K::ROW + cl * 16 + (aa & 1) * 8;
    const uint32_t xoff = (uint32_t)tk.row_slot[rs] * K::BLK + lrow + 64u * ((uint32_t)sub ^ (uint32_t)kk);
    uint32_t coff[E];
#pragma unroll
    for (int e = 0; e < E; ++e)
        coff[e] = (uint32_t)tk.col_slot[e >> 2] * K::BLK + lrow + 64u * ((uint32_t)(e & 3) ^ (uint32_t)kk);
    const uint32_t lw = K::OFF_W + (lane >> 5) * 32;
    const bool own_x = (tk.flags >> rs) & 1;
    const bool own_sumx = !CENTER && own_x;
    const bool own_sumw = !CENTER && (tk.flags & 4) && wave == 0;
    // centered: the weighted means of the map (fp64 sums of pass 1, or a pilot's)
    const double *sm = CENTER ? a.sums + (int64_t)tk.map * (a.P + a.d_t) : nullptr;
    const double s_w = CENTER ? sm[0] : 0.0;
    auto mean_of = [&](int ch) { return (CENTER && s_w != 0.0) ? (float)(sm[1 + ch] / s_w) : 0.f; };
    const int rb = tk.rows[rs];                                 // feature block of this wave's rows
    const float mu_row = mean_of(32 * (4 * rb + sub) + (lane & 31));
    // the target block is column block 1 of a YS task: copying wave w sums w y over its window w
    const bool ysum = YS && copier;

    struct Folded {
        bf16x8_t hi, lo;
    };
    f32x16_t acc[E];
    float sumx = 0.f, sumy = 0.f, sumw = 0.f;
    auto zero_acc = [&]() {
#pragma unroll
        for (int t = 0; t < E; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[t][v] = 0.f;
    };
    zero_acc();

    // a = w x for the lane's 8 rows of one channel of the wave's rows, split
    // into hi + lo; sum w x (or, centered, e) and sum w on the side
    auto fold = [&](Folded &f, int st) {
        const lds_char_t *S = lds + st * K::STAGE;
        const bf16x8_t xr = tr_read8(S + xoff, S + xoff + 4 * K::ROW);
        const f32x4_t w0 = *(const lds_f32x4_t *)(S + lw);
        const f32x4_t w1 = *(const lds_f32x4_t *)(S + lw + 16);
        const float w[8] = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
        const uint4 ax = __builtin_bit_cast(uint4, xr);
        const uint32_t xv[4] = {ax.x, ax.y, ax.z, ax.w};
        float av[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (CENTER) {
                av[2 * e] = w[2 * e] * (bf_lo(xv[e]) - mu_row);
                av[2 * e + 1] = w[2 * e + 1] * (bf_hi(xv[e]) - mu_row);
            } else {
                av[2 * e] = w[2 * e] * bf_lo(xv[e]);
                av[2 * e + 1] = w[2 * e + 1] * bf_hi(xv[e]);
            }
        }
        uint32_t hv[4], lv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            hv[e] = pack_bf16(av[2 * e], av[2 * e + 1]);
            lv[e] = pack_bf16(av[2 * e] - bf_lo(hv[e]), av[2 * e + 1] - bf_hi(hv[e]));
        }
        if constexpr (CENTER) {
            // e = sum of the folded operand exactly as multiplied (hi + lo)
            float q[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) q[e] = (bf_lo(hv[e]) + bf_lo(lv[e])) + (bf_hi(hv[e]) + bf_hi(lv[e]));
            sumx += (q[0] + q[1]) + (q[2] + q[3]);
        } else {
            sumx += ((av[0] + av[1]) + (av[2] + av[3])) + ((av[4] + av[5]) + (av[6] + av[7]));
            sumw += ((w[0] + w[1]) + (w[2] + w[3])) + ((w[4] + w[5]) + (w[6] + w[7]));
        }
        f.hi = __builtin_bit_cast(bf16x8_t, make_uint4(hv[0], hv[1], hv[2], hv[3]));
        f.lo = __builtin_bit_cast(bf16x8_t, make_uint4(lv[0], lv[1], lv[2], lv[3]));
    };
    // sum w y over this copying wave's 32 target channels, from the column
    // fragments of the tile (entry 4 + w)
    auto sum_y = [&](const bf16x8_t &yf, int st) {
        const lds_char_t *S = lds + st * K::STAGE;
        const f32x4_t w0 = *(const lds_f32x4_t *)(S + lw);
        const f32x4_t w1 = *(const lds_f32x4_t *)(S + lw + 16);
        const float w[8] = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
        const uint4 yv = __builtin_bit_cast(uint4, yf);
        const uint32_t yy[4] = {yv.x, yv.y, yv.z, yv.w};
        float py[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            py[2 * i] = w[2 * i] * bf_lo(yy[i]);
            py[2 * i + 1] = w[2 * i + 1] * bf_hi(yy[i]);
        }
        sumy += ((py[0] + py[1]) + (py[2] + py[3])) + ((py[4] + py[5]) + (py[6] + py[7]));
    };

    // ---- flush: add the wave's tiles (and bias sums) into G and C
    float *tr = (float *)(lds + K::OFF_T) + wave * 32 * K::TRS;
    float *es = (float *)(lds + K::OFF_E) + wave * 32;       // centered: e of the wave's 32 rows
    const int P = CENTER ? a.P - 1 : a.P;                    // leading dimension of G (or A)
    float *Gm = a.G + (int64_t)tk.map * P * P;
    float *Cm = a.C + (int64_t)tk.map * P * a.d_t;
    auto flush = [&]() {
        const float ex = sumx + __shfl_xor(sumx, 32);         // lanes l and l + 32: the two token halves
        if constexpr (CENTER) {
            if (lane < 32) es[lane] = ex;
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
        const int R = 4 * rb + sub;                          // 32-row block of G
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int cb = e >> 2, win = e & 3;
            if (!((tk.cell_mask >> (2 * rs + cb)) & 1)) continue;      // an unused cell
            const int col = tk.cols[cb];
            const bool is_y = col == a.k;
            const int Cc = 4 * col + win;                    // 32-column block (of G, or of C if is_y)
            if (!is_y && col == rb && Cc < R) continue;      // below the diagonal of a diagonal block
            const f32x16_t &t = acc[e];
            // centered: minus e_i mu_j, mu_j the mean of this lane's column
            const float muc = CENTER ? mean_of(is_y ? 128 * a.k + 32 * win + (lane & 31) : 32 * Cc + (lane & 31))
                                     : 0.f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int i = 8 * (v >> 2) + (v & 3) + 4 * (lane >> 5);
                tr[i * K::TRS + (lane & 31)] = CENTER ? t[v] - es[i] * muc : t[v];
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            // mode 0: cross tile of C; 1: diagonal tile of G; 2: any other tile of G (+ its mirror)
            const int mode = is_y ? 0 : (Cc == R ? 1 : 2);
            float *dst = is_y ? Cm + (int64_t)(32 * R) * a.d_t + 32 * win : Gm + (int64_t)(32 * R) * P + 32 * Cc;
            float *mir = Gm + (int64_t)(32 * Cc) * P + 32 * R;
            const int64_t ld = is_y ? a.d_t : P;
            flush_rows(tr, lane, mode, dst, mir, ld);
        }
        if constexpr (CENTER) {
            if (a.resid && own_x && lane < 32) {
                // shifted form: sum w (x - mu) of the rows, one owner per entry (sum w
                // and sum w y come from the target-block pass of the same call)
                a.resid[(int64_t)tk.map * (a.P + a.d_t) + 1 + 128 * rb + 32 * sub + lane] += (double)ex;
            }
            sumx = 0.f;
            zero_acc();
            return;
        }
        // bias row / column
        if (own_sumx && lane < 32) {
            const int ch = 128 * rb + 32 * sub + lane;
            Gm[(int64_t)ch * P + P - 1] += ex;
            Gm[(int64_t)(P - 1) * P + ch] += ex;
        }
        sumx = 0.f;
        if (ysum) {
            const float sy = sumy + __shfl_xor(sumy, 32);
            if (lane < 32) Cm[(int64_t)(P - 1) * a.d_t + 32 * cw + lane] += sy;
        }
        sumy = 0.f;
        if (own_sumw) {
            const float sw = sumw + __shfl_xor(sumw, 32);
            if (lane == 0) Gm[(int64_t)(P - 1) * P + P - 1] += sw;
        }
        sumw = 0.f;
        zero_acc();
    };

    // ---- pipeline.  Eight waves, two per SIMD: while one wave waits for its
    // operands or folds, the other keeps the matrix core busy.  Iteration t:
    // tile t+1 has landed (the copying waves' wait, then the barrier); tile
    // t+NST-1 is issued into the stage of tile t-1, which every wave finished
    // reading before the barrier; the wave reads tile t's column fragments,
    // runs its 16 MFMAs with tile t's folded rows (folded in iteration t-1),
    // and folds tile t+1.
    if (copier) {
#pragma unroll
        for (int u = 0; u < K::NST - 1; ++u) issue(u);        // tiles 0 .. NST-2 into stages 0 .. NST-2
        wait_vm<(K::NST - 2) * PER_TILE>();                   // tile 0 has landed
    }
    lds_barrier();
    const int n_iter = (a.n_tiles + 5) / 6 * 6;              // padded with zero-weight tiles
    Folded f0, f1;
    fold(f0, 0);
    auto iteration = [&](int t, const Folded &fa, Folded &fb) {
        const int st = t % K::NST, sn = (t + 1) % K::NST, sp = (t + K::NST - 1) % K::NST;
        if (copier) wait_vm<(K::NST - 3) * PER_TILE>();       // tile t+1 has landed
        lds_barrier();
        if (copier) issue(sp);                                // tile t+NST-1 into the stage of tile t-1
        const lds_char_t *S = lds + st * K::STAGE;
        auto products = [&]() __attribute__((always_inline)) {
            bf16x8_t cf[E];
#pragma unroll
            for (int e = 0; e < E; ++e) cf[e] = tr_read8(S + coff[e], S + coff[e] + 4 * K::ROW);
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa.hi, cf[e], acc[e], 0, 0, 0);
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa.lo, cf[e], acc[e], 0, 0, 0);
#pragma unroll
            for (int e = 0; e < E; ++e) {
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);     // the two reads of fragment e
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // its hi product
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
            if (ysum) {
                const bf16x8_t yf = cw == 0 ? cf[4] : cw == 1 ? cf[5] : cw == 2 ? cf[6] : cf[7];
                sum_y(yf, st);
            }
        };
        // the two waves of a SIMD (w and w + 4) take the steps in opposite
        // orders, so one folds while the other keeps the matrix core busy
        if constexpr (FOLD_FIRST) {
            fold(fb, sn);
            products();
        } else {
            products();
            fold(fb, sn);
        }
    };
    for (int c0 = 0; c0 < n_iter; c0 += a.chunk_tiles) {
        const int c1 = min(c0 + a.chunk_tiles, n_iter);
        for (int t = c0; t < c1; t += 2) {
            iteration(t, f0, f1);
            iteration(t + 1, f1, f0);
        }
        flush();
    }
    if (copier) wait_vm<0>();                                 // drain the trailing copies
}

template <bool CENTER>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2)))
void stats_multi_kernel(MultiArgs a) {
    using K = MCfg;
    __shared__ __attribute__((aligned(16))) char lds_raw[K::LDS];
    lds_char_t *lds = (lds_char_t *)lds_raw;
    // Consecutive workgroups go to different XCDs (round robin); this order
    // gives each XCD a contiguous run of tasks, so the tasks of a map and of
    // its neighbours (which share source blocks) meet in one L2.
    const int b = blockIdx.x;
    const int task = (b & 7) * a.per_xcd + (b >> 3);
    if (task >= a.n_tasks) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const MultiTask &tk = a.tasks[task];          // uniform: read with scalar loads
    MultiCtx c;
    // K maps may read compact de-rotated calibration rows (one per row, no sampling stride)
    const bool ks = tk.kv == 0 && a.srck != nullptr, kt = tk.kv == 0 && a.tgtk != nullptr;
    c.s_row = ks ? a.ssk.tok : a.ss.tok * (int64_t)a.stride;
    c.t_row = kt ? a.tsk.tok : a.ts.tok * (int64_t)a.stride;
    c.s_seq = ks ? a.ssk.seq : a.ss.seq;
    c.t_seq = kt ? a.tsk.seq : a.ts.seq;
#pragma unroll
    for (int s = 0; s < K::MAXS; ++s) {
        const int L = tk.slot_layer[s];
        c.slot_base[s] = L < 0 ? (kt ? a.tgtk + tk.tgt_layer * a.tsk.layer + tk.tgt_head * a.tsk.head
                                     : a.tgt + tk.tgt_layer * a.ts.layer + tk.kv * a.ts.kv + tk.tgt_head * a.ts.head)
                               : (ks ? a.srck + L * a.ssk.layer + tk.src_head * a.ssk.head
                                     : a.src + L * a.ss.layer + tk.kv * a.ss.kv + tk.src_head * a.ss.head);
    }
    // variant: staged blocks (1..4), target block staged (HASY), sum w y owned (YS)
    const bool hasy = tk.slot_layer[tk.n_lds - 1] < 0;
    const int var = (tk.n_lds - 1) * 3 + (hasy ? ((!CENTER && (tk.flags & 8)) ? 2 : 1) : 0);
    switch (var) {
#define CB_W(NL_, HY, Y)                                                                            \
    if (wave < 4) multi_wave<NL_, HY, Y, CENTER, false>(a, tk, c, lds, wave, lane);                 \
    else multi_wave<NL_, HY, Y, CENTER, true>(a, tk, c, lds, wave, lane);
#define CB_V(NL_)                                                                                  \
        case (NL_ - 1) * 3 + 0: CB_W(NL_, false, false) break;                                     \
        case (NL_ - 1) * 3 + 1: CB_W(NL_, true, false) break;                                      \
        case (NL_ - 1) * 3 + 2:                                                                     \
            if constexpr (!CENTER) { CB_W(NL_, true, true) }                                        \
            break;
        CB_V(1) CB_V(2) CB_V(3) CB_V(4)
#undef CB_V
#undef CB_W
        default: break;
    }
}

// Pass 1 of the centered form: one workgroup per (map, feature block), 16
// threads per row (16-byte chunks), 16 rows at a time; fp64 sums of w x (and
// of w on the target block), each thread's 8 channels over its rows, then a
// fixed-order sum over the 16 row groups through LDS, added into sums.
__global__ __launch_bounds__(256) void means_multi_kernel(MeansMultiArgs a) {
    __shared__ double red[16][16][9];
    // tgt_only: one workgroup per map, its target block (sum w, sum w y)
    const int m = a.tgt_only ? blockIdx.x : blockIdx.x / (a.k + 1), blk = a.tgt_only ? a.k : blockIdx.x % (a.k + 1);
    const int tid = threadIdx.x, ch = tid & 15, rg = tid >> 4;
    const ApplyMultiMap mp = a.maps[m];
    const bool tgt = blk == a.k;
    const uint16_t *base = tgt ? a.tgt + mp.tgt_layer * a.ts.layer + mp.kv * a.ts.kv + mp.tgt_head * a.ts.head
                               : a.src + a.layers[(int64_t)m * a.k + blk] * a.ss.layer + mp.kv * a.ss.kv +
                                     mp.src_head * a.ss.head;
    const int64_t s_seq = tgt ? a.ts.seq : a.ss.seq, s_tok = tgt ? a.ts.tok : a.ss.tok;
    const float *wr = a.w + (int64_t)a.wrow[m] * a.w_row_stride;
    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0}, accw = 0.0;
    for (int b = 0; b < a.n_seqs; ++b) {
        const uint16_t *rowb = base + (int64_t)b * s_seq + ch * 8;
        const float *wb = wr + (int64_t)b * a.seq_len;
#pragma unroll 4
        for (int r = rg; r < a.rows_per_seq; r += 16) {
            const int tok = r * a.stride;
            const uint4 v = *(const uint4 *)(rowb + (int64_t)tok * s_tok);
            const double w = (double)wb[tok];
            const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc[2 * e] += w * (double)bf_lo(u[e]);
                acc[2 * e + 1] += w * (double)bf_hi(u[e]);
            }
            accw += w;
        }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) red[rg][ch][e] = acc[e];
    red[rg][ch][8] = accw;
    __syncthreads();
    if (tid < 16 * 9) {
        const int c = tid / 9, e = tid % 9;
        double s = 0.0;
        for (int g = 0; g < 16; ++g) s += red[g][c][e];
        double *out = a.sums + (int64_t)m * (1 + 128 * a.k + a.d_t);
        if (e < 8) out[1 + 128 * blk + 8 * c + e] += s;
        else if (tgt && c == 0) out[0] += s;
    }
}

}  // namespace

hipError_t launch_stats_multi(const MultiArgs &a, hipStream_t s) {
    if (a.n_tasks == 0 || a.n_tiles == 0) return hipSuccess;
    hipLaunchKernelGGL(stats_multi_kernel<false>, dim3(8 * a.per_xcd), dim3(512), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_stats_multi_centered(const MultiArgs &a, hipStream_t s) {
    if (a.n_tasks == 0 || a.n_tiles == 0) return hipSuccess;
    hipLaunchKernelGGL(stats_multi_kernel<true>, dim3(8 * a.per_xcd), dim3(512), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_means_multi(const MeansMultiArgs &a, hipStream_t s) {
    if (a.n_maps == 0 || a.n_seqs == 0 || a.rows_per_seq == 0) return hipSuccess;
    hipLaunchKernelGGL(means_multi_kernel, dim3((unsigned)(a.n_maps * (a.tgt_only ? 1 : a.k + 1))), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cb

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
// blocks 0..k-1 and the target block k.  A task is (map, row block i, up to
// four column blocks j >= i, the target block included); the tasks of a map
// cover the upper block triangle of G and the cross block of C once.  One
// workgroup runs one task over every calibration row of the call and adds its
// fp32 sums into G and C itself (it is the only writer of those elements), so
// there are no partial sums, no reduction pass and no atomics.
//
// Per workgroup: four waves, one per SIMD.  Wave (p, q) owns rows 64p..64p+63
// of the row block (two 32-row MFMA blocks) and half q of the task's column
// blocks (2N 32-column blocks for N column blocks): 4N 32x32 accumulator
// tiles.  Per 16-row K step it folds the fp32 weight into its two x
// fragments, splits w x into hi = RNE_bf16(w x) and lo = RNE_bf16(w x - hi),
// and issues 8N v_mfma_f32_32x32x16_bf16 against the exact bf16 columns.
//
// Staging.  A tile is 16 calibration rows of one sequence.  Its blocks (the
// row block and the column blocks other than the diagonal one) move HBM -> LDS
// by global_load_lds_dwordx4 through a six-stage ring, six tiles ahead; each
// 16-byte chunk c of row t sits at chunk c ^ 4(t mod 4) so the transposed
// operand reads (ds_read_b64_tr_b16) are conflict free.  Rows past the end of
// a sequence repeat its last row with weight zero.
//
// Flush.  Every at most 1,020 tiles (16,320 rows) and at the end of the call
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
    static constexpr int MAXS = 5;                 // LDS slots (row block + 4 column blocks)
    static constexpr int OFF_W = MAXS * BLK;       // weights of the tile: [KT] fp32
    static constexpr int STAGE = OFF_W + KT * 4;
    static constexpr int NST = 6;                  // ring stages
    static constexpr int TRS = 33;                 // row stride (floats) of the transpose scratch
    static constexpr int OFF_T = NST * STAGE;
    static constexpr int LDS = OFF_T + 4 * 32 * TRS * 4;
    static_assert(KT == 16, "one tile is one MFMA K step");
    static_assert(LDS <= 160 * 1024, "the ring must fit in LDS");
};

// Per-workgroup state that is uniform across the wave.
struct MultiCtx {
    const uint16_t *slot_base[MCfg::MAXS];   // (layer, kv, head) base of each staged block
    int64_t slot_sseq[MCfg::MAXS], slot_stok[MCfg::MAXS];
};

// Adds the 32 x 32 tile held in the wave's transpose scratch `tr` (row i at
// tr + 33 i) into global memory, two rows per step: mode 0 and 2 add it at
// dst (leading dimension ld), mode 2 also adds its transpose at mir, and mode
// 1 (a diagonal tile of G) adds its upper triangle to both triangles.
__device__ __forceinline__ void flush_rows(const float *tr, int lane, int mode, float *dst, float *mir, int64_t ld) {
    const int jj = lane & 31;
#pragma unroll 1
    for (int it = 0; it < 16; ++it) {
        const int ii = 2 * it + (lane >> 5);
        const float up = tr[ii * MCfg::TRS + jj], dn = tr[jj * MCfg::TRS + ii];
        float *d = dst + (int64_t)ii * ld + jj;
        *d += mode == 1 && ii > jj ? dn : up;
        if (mode == 2) {
            float *dm = mir + (int64_t)ii * ld + jj;
            *dm += dn;
        }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// N: column blocks of the task.  YS: the task owns sum w y of its map (its
// last column block is the target block), so it also sums w y on the VALU.
template <int N, bool YS>
__device__ __forceinline__ void multi_wave(const MultiArgs &a, const MultiTask &tk, const MultiCtx &c,
                                           lds_char_t *lds, int wave, int lane) {
    using K = MCfg;
    constexpr int E = 2 * N;                    // 32-column blocks of this wave
    const int p = wave & 1, q = wave >> 1;
    const uint32_t lds_base = (uint32_t)(uintptr_t)lds;
    const int n_lds = tk.n_lds;

    // ---- copy descriptors: wave w copies rows 4w..4w+3 of every staged block
    const int crow = 4 * wave + (lane >> 4);
    const uint32_t cchunk = (uint32_t)((lane & 15) ^ (4 * (crow & 3))) * 16u;
    uint32_t cstep[K::MAXS];                    // bytes between consecutive calibration rows
#pragma unroll
    for (int s = 0; s < K::MAXS; ++s) cstep[s] = (uint32_t)(c.slot_stok[s] * 2 * (int64_t)a.stride);
    const float *wrow = a.w + (int64_t)tk.wrow * a.w_row_stride;
    const int per_tile = n_lds + 1;             // copy instructions per tile and wave

    struct TilePos {
        uint32_t seq, r0, tmax;                 // sequence, first row, last valid row offset
        bool live;
    };
    auto tile_at = [&](int u) {
        TilePos t;
        t.live = u < a.n_tiles;
        const uint32_t v = (uint32_t)(t.live ? u : a.n_tiles - 1);
        t.seq = fastdiv(v, a.TPS);
        t.r0 = (v - t.seq * a.TPS.d) * K::KT;
        t.tmax = min((uint32_t)K::KT - 1, a.rows_per_seq - 1 - t.r0);
        return t;
    };
    auto issue = [&](int u, int st) {
        const TilePos t = tile_at(u);
        const uint32_t stage = lds_base + st * K::STAGE;
        const uint32_t row = min((uint32_t)crow, t.tmax);
        const int64_t tok0 = (int64_t)t.r0 * a.stride;
#pragma unroll
        for (int s = 0; s < K::MAXS; ++s) {
            if (s < n_lds) {
                const void *base = uniform_ptr(c.slot_base[s] + t.seq * c.slot_sseq[s] + tok0 * c.slot_stok[s]);
                dma16_sbase(row * cstep[s] + cchunk, base,
                            __builtin_amdgcn_readfirstlane(stage + s * K::BLK + wave * 1024));
            }
        }
        const uint32_t wr = 4 * wave + (lane & 3);
        const bool ok = t.live && wr <= t.tmax;
        const void *g = ok ? (const void *)(wrow + (int64_t)t.seq * a.seq_len + (int64_t)(t.r0 + wr) * a.stride)
                           : a.zero;
        dma4_lanes(g, __builtin_amdgcn_readfirstlane(stage + K::OFF_W + 16 * wave), 0xFull);
    };

    // ---- operand geometry (transposed reads; see cb_stats_kernel.h)
    const int g16 = lane >> 4, j16 = lane & 15, aa = j16 & 3, kk = j16 >> 2;
    const int tok_l = 8 * (g16 >> 1) + kk;
    const int cl = 2 * (g16 & 1) + (aa >> 1);
    const uint32_t lrow = tok_l * K::ROW + cl * 16 + (aa & 1) * 8;
    uint32_t xoff[2], coff[E];
#pragma unroll
    for (int r = 0; r < 2; ++r) xoff[r] = lrow + 64u * ((uint32_t)(2 * p + r) ^ (uint32_t)kk);
    bool ecol_y[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int gi = q * E + e, b = gi >> 2, win = gi & 3;
        coff[e] = (uint32_t)tk.col_slot[b] * K::BLK + lrow + 64u * ((uint32_t)win ^ (uint32_t)kk);
        ecol_y[e] = tk.col_blk[b] == a.k;
    }
    const uint32_t lw = K::OFF_W + (lane >> 5) * 32;
    const bool own_sumx = (tk.flags & 1) && q == 0;
    const bool own_sumw = (tk.flags & 4) && wave == 0;
    // entries of this wave that read the target block when it is the task's last column block
    auto ycol = [&](int e) { return YS && q * E + e >= 4 * (N - 1); };

    struct Ops {
        bf16x8_t xr[2], cf[E];
        float w[8];
    };
    struct Folded {
        bf16x8_t hi[2], lo[2];
    };
    f32x16_t acc[2 * E];
    float sumx[2] = {0.f, 0.f}, sumy[E], sumw = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) sumy[e] = 0.f;
    auto zero_acc = [&]() {
#pragma unroll
        for (int t = 0; t < 2 * E; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[t][v] = 0.f;
    };
    zero_acc();

    auto read_ops = [&](Ops &o, int st) {
        const lds_char_t *S = lds + st * K::STAGE;
#pragma unroll
        for (int r = 0; r < 2; ++r) o.xr[r] = tr_read8(S + xoff[r], S + xoff[r] + 4 * K::ROW);
#pragma unroll
        for (int e = 0; e < E; ++e) o.cf[e] = tr_read8(S + coff[e], S + coff[e] + 4 * K::ROW);
        const f32x4_t w0 = *(const lds_f32x4_t *)(S + lw);
        const f32x4_t w1 = *(const lds_f32x4_t *)(S + lw + 16);
        o.w[0] = w0[0]; o.w[1] = w0[1]; o.w[2] = w0[2]; o.w[3] = w0[3];
        o.w[4] = w1[0]; o.w[5] = w1[1]; o.w[6] = w1[2]; o.w[7] = w1[3];
    };
    // a = w x for the lane's 8 rows of one channel of row block r, split into
    // hi + lo; sum w x on the side (kept by every wave: it is branch free and
    // written only by the owner).
    auto fold_row = [&](Folded &f, const Ops &o, int r) {
        const uint4 ax = __builtin_bit_cast(uint4, o.xr[r]);
        const uint32_t xv[4] = {ax.x, ax.y, ax.z, ax.w};
        float av[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            av[2 * e] = o.w[2 * e] * bf_lo(xv[e]);
            av[2 * e + 1] = o.w[2 * e + 1] * bf_hi(xv[e]);
        }
        uint32_t hv[4], lv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            hv[e] = pack_bf16(av[2 * e], av[2 * e + 1]);
            lv[e] = pack_bf16(av[2 * e] - bf_lo(hv[e]), av[2 * e + 1] - bf_hi(hv[e]));
        }
        sumx[r] += ((av[0] + av[1]) + (av[2] + av[3])) + ((av[4] + av[5]) + (av[6] + av[7]));
        f.hi[r] = __builtin_bit_cast(bf16x8_t, make_uint4(hv[0], hv[1], hv[2], hv[3]));
        f.lo[r] = __builtin_bit_cast(bf16x8_t, make_uint4(lv[0], lv[1], lv[2], lv[3]));
    };
    auto sum_w = [&](const Ops &o) {
        sumw += ((o.w[0] + o.w[1]) + (o.w[2] + o.w[3])) + ((o.w[4] + o.w[5]) + (o.w[6] + o.w[7]));
    };
    auto sum_y = [&](const Ops &o) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if (!ycol(e)) continue;
            const uint4 yv = __builtin_bit_cast(uint4, o.cf[e]);
            const uint32_t yy[4] = {yv.x, yv.y, yv.z, yv.w};
            float py[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                py[2 * i] = o.w[2 * i] * bf_lo(yy[i]);
                py[2 * i + 1] = o.w[2 * i + 1] * bf_hi(yy[i]);
            }
            sumy[e] += ((py[0] + py[1]) + (py[2] + py[3])) + ((py[4] + py[5]) + (py[6] + py[7]));
        }
    };
    auto fold = [&](Folded &f, const Ops &o) {
        fold_row(f, o, 0);
        fold_row(f, o, 1);
        sum_w(o);
        sum_y(o);
    };
    auto mma_hi = [&](const Folded &f, const Ops &o) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int e = 0; e < E; ++e)
                acc[r * E + e] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.hi[r], o.cf[e], acc[r * E + e], 0, 0, 0);
    };
    auto mma_lo = [&](const Folded &f, const Ops &o) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int e = 0; e < E; ++e)
                acc[r * E + e] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.lo[r], o.cf[e], acc[r * E + e], 0, 0, 0);
    };

    // ---- flush: add the wave's tiles (and bias sums) into G and C
    float *tr = (float *)(lds + K::OFF_T) + wave * 32 * K::TRS;
    float *Gm = a.G + (int64_t)tk.map * a.P * a.P;
    float *Cm = a.C + (int64_t)tk.map * a.P * a.d_t;
    const int P = a.P;
    auto flush = [&]() {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int R = 4 * tk.row_blk + 2 * p + r;            // 32-row block of G
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int gi = q * E + e, b = gi >> 2, win = gi & 3;
                const bool is_y = ecol_y[e];
                const int Cc = 4 * tk.col_blk[b] + win;          // 32-column block (of G, or of C if is_y)
                if (!is_y && Cc < R) continue;                   // below the diagonal: dropped
                const f32x16_t &t = acc[r * E + e];
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int i = 8 * (v >> 2) + (v & 3) + 4 * (lane >> 5);
                    tr[i * K::TRS + (lane & 31)] = t[v];
                }
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                // mode 0: cross tile of C; 1: diagonal tile of G; 2: tile above the diagonal (+ mirror)
                const int mode = is_y ? 0 : (Cc == R ? 1 : 2);
                float *dst = is_y ? Cm + (int64_t)(32 * R) * a.d_t + 32 * win
                                  : Gm + (int64_t)(32 * R) * P + 32 * Cc;
                float *mir = Gm + (int64_t)(32 * Cc) * P + 32 * R;
                const int64_t ld = is_y ? a.d_t : P;
                flush_rows(tr, lane, mode, dst, mir, ld);
            }
        }
        // bias row / column: lanes l and l + 32 hold the two halves of each K step
        if (own_sumx) {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const float s = sumx[r] + __shfl_xor(sumx[r], 32);
                if (lane < 32) {
                    const int ch = 128 * tk.row_blk + 64 * p + 32 * r + lane;
                    Gm[(int64_t)ch * P + P - 1] += s;
                    Gm[(int64_t)(P - 1) * P + ch] += s;
                }
            }
        }
        sumx[0] = sumx[1] = 0.f;
        if (YS && p == 0) {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                if (!ycol(e)) continue;
                const float s = sumy[e] + __shfl_xor(sumy[e], 32);
                const int win = (q * E + e) & 3;
                if (lane < 32) Cm[(int64_t)(P - 1) * a.d_t + 32 * win + lane] += s;
            }
        }
#pragma unroll
        for (int e = 0; e < E; ++e) sumy[e] = 0.f;
        if (own_sumw) {
            const float s = sumw + __shfl_xor(sumw, 32);
            if (lane == 0) Gm[(int64_t)(P - 1) * P + P - 1] += s;
        }
        sumw = 0.f;
        zero_acc();
    };

    // ---- pipeline.  Tile t's operands are read from LDS two iterations ahead
    // (iteration t-2), folded one iteration ahead (t-1) and multiplied in
    // iteration t, so no LDS latency sits in front of a fold and no fold in
    // front of an MFMA.  Iteration t: tile t+2 has landed (wait + barrier);
    // tile t+6 is issued into the stage of tile t, whose reads finished two
    // iterations ago; the hi MFMAs of tile t run with the fold of row block 0
    // of tile t+1 and half of the reads of tile t+2, the lo MFMAs with the
    // rest (an MFMA keeps the matrix core busy for about as long as the wave
    // needs to issue five other instructions).  Operand sets rotate with
    // period 3, folded sets with period 2: six iterations per loop trip.
#pragma unroll
    for (int u = 0; u < K::NST; ++u) issue(u, u);
    const int n_iter = (a.n_tiles + 5) / 6 * 6;              // padded with zero-weight tiles
    Ops o0, o1, o2;
    Folded f0, f1;
    wait_vm_rt((K::NST - 1) * per_tile);                     // tile 0 has landed
    lds_barrier();
    read_ops(o0, 0);
    wait_vm_rt((K::NST - 2) * per_tile);                     // tile 1 has landed
    lds_barrier();
    read_ops(o1, 1);
    fold(f0, o0);
    auto pin = [&](const Folded &f) {
#pragma unroll
        for (int r = 0; r < 2; ++r) asm volatile("" ::"v"(f.hi[r]), "v"(f.lo[r]));
        asm volatile("" ::"v"(sumx[0]), "v"(sumx[1]), "v"(sumw));
    };
    auto read_half = [&](Ops &o, int st, int half) {
        const lds_char_t *S = lds + st * K::STAGE;
        if (half == 0) {
#pragma unroll
            for (int r = 0; r < 2; ++r) o.xr[r] = tr_read8(S + xoff[r], S + xoff[r] + 4 * K::ROW);
            const f32x4_t w0 = *(const lds_f32x4_t *)(S + lw);
            const f32x4_t w1 = *(const lds_f32x4_t *)(S + lw + 16);
            o.w[0] = w0[0]; o.w[1] = w0[1]; o.w[2] = w0[2]; o.w[3] = w0[3];
            o.w[4] = w1[0]; o.w[5] = w1[1]; o.w[6] = w1[2]; o.w[7] = w1[3];
        }
#pragma unroll
        for (int e = 0; e < E; ++e)
            if ((e < E / 2) == (half == 0)) o.cf[e] = tr_read8(S + coff[e], S + coff[e] + 4 * K::ROW);
    };
    auto iteration = [&](int t, const Ops &oa, const Folded &fa, const Ops &ob, Folded &fb, Ops &oc) {
        wait_vm_rt((K::NST - 3) * per_tile);                 // tile t+2 has landed
        lds_barrier();
        issue(t + K::NST, t % K::NST);
        __builtin_amdgcn_sched_barrier(0);
        read_half(oc, (t + 2) % K::NST, 0);
        mma_hi(fa, oa);
        fold_row(fb, ob, 0);
#pragma unroll
        for (int i = 0; i < 2 * E; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);            // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);            // one LDS read
            __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);            // three VALU
        }
        __builtin_amdgcn_sched_barrier(0);
        read_half(oc, (t + 2) % K::NST, 1);
        fold_row(fb, ob, 1);
        sum_w(ob);
        mma_lo(fa, oa);
        pin(fb);
#pragma unroll
        for (int i = 0; i < 2 * E; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (YS) sum_y(ob);
    };
    for (int c0 = 0; c0 < n_iter; c0 += a.chunk_tiles) {
        const int c1 = min(c0 + a.chunk_tiles, n_iter);
        for (int t = c0; t < c1; t += 6) {
            iteration(t + 0, o0, f0, o1, f1, o2);
            iteration(t + 1, o1, f1, o2, f0, o0);
            iteration(t + 2, o2, f0, o0, f1, o1);
            iteration(t + 3, o0, f1, o1, f0, o2);
            iteration(t + 4, o1, f0, o2, f1, o0);
            iteration(t + 5, o2, f1, o0, f0, o1);
        }
        flush();
    }
    wait_vm<0>();                                            // drain the trailing copies
}

__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
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
#pragma unroll
    for (int s = 0; s < K::MAXS; ++s) {
        const int L = s < tk.n_lds ? tk.slot_layer[s] : tk.slot_layer[0];
        if (L < 0) {
            c.slot_base[s] = a.tgt + tk.tgt_layer * a.ts.layer + tk.kv * a.ts.kv + tk.tgt_head * a.ts.head;
            c.slot_sseq[s] = a.ts.seq;
            c.slot_stok[s] = a.ts.tok;
        } else {
            c.slot_base[s] = a.src + L * a.ss.layer + tk.kv * a.ss.kv + tk.src_head * a.ss.head;
            c.slot_sseq[s] = a.ss.seq;
            c.slot_stok[s] = a.ss.tok;
        }
    }
    const bool ys = (tk.flags & 2) != 0;
    switch (tk.n_cols * 2 + (ys ? 1 : 0)) {
        case 2: multi_wave<1, false>(a, tk, c, lds, wave, lane); break;
        case 3: multi_wave<1, true>(a, tk, c, lds, wave, lane); break;
        case 4: multi_wave<2, false>(a, tk, c, lds, wave, lane); break;
        case 5: multi_wave<2, true>(a, tk, c, lds, wave, lane); break;
        case 6: multi_wave<3, false>(a, tk, c, lds, wave, lane); break;
        case 7: multi_wave<3, true>(a, tk, c, lds, wave, lane); break;
        case 8: multi_wave<4, false>(a, tk, c, lds, wave, lane); break;
        default: multi_wave<4, true>(a, tk, c, lds, wave, lane); break;
    }
}

}  // namespace

hipError_t launch_stats_multi(const MultiArgs &a, hipStream_t s) {
    if (a.n_tasks == 0 || a.n_tiles == 0) return hipSuccess;
    hipLaunchKernelGGL(stats_multi_kernel, dim3(8 * a.per_xcd), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cb

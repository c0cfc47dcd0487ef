// cb_stats.hip -- weighted augmented sufficient statistics on gfx950.
//
// CacheBridge Sec. 3.4 (Eq. fusedstats) needs, per target head and component,
// only weighted means and the weighted (cross-)covariances of the head-local
// feature (Sec. 3.2, Eq. localfeature).  They are all contained in the
// augmented moments
//     G = sum_t w_t [x_t;1][x_t;1]^T      C = sum_t w_t [x_t;1] y_t^T,
// which this file builds in one streaming pass over the caches, without
// materialising any observation panel in HBM.
//
// stats_kernel (one workgroup per (item, token chunk)):
//   * an item is one or two maps; two maps that read the same source block
//     load its rows once;
//   * token tiles stream HBM -> LDS by direct-to-LDS copies through a
//     four-stage ring (see the comment above Cfg);
//   * wave (slot, rb) owns rows rb*32..rb*32+31 of one map: it folds the
//     per-token weight into its x rows in fp32, splits w*x into two bf16 terms
//     (hi = RNE(w x), lo = RNE(w x - hi)) and runs v_mfma_f32_32x32x16_bf16
//     against the exact bf16 x and y columns, accumulating in fp32.  Only the
//     upper-triangle 32x32 tiles of the Gram block are computed;
//   * the bias row/column (sum w, sum w x, sum w y) is summed on the VALU in
//     fp32 from the same operands;
//   * at the end of its token chunk the workgroup writes its fp32 partial to
//     the plan's workspace (plain stores, no atomics).
// reduce_kernel (one workgroup per map) adds the partials of all chunks in a
// fixed order, mirrors the Gram block so G is exactly symmetric, and adds the
// result into the caller's G and C.
#include "cb_internal.h"

namespace cb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

__device__ __forceinline__ uint32_t fastdiv(uint32_t n, const FastDiv &f) {
    const uint32_t t = __umulhi(n, f.m);
    return (t + ((n - t) >> f.sh1)) >> f.sh2;
}

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    f32x2_t v = {lo, hi};
    bf16x2_t p = __builtin_convertvector(v, bf16x2_t);
    return __builtin_bit_cast(uint32_t, p);
}

// ---------------------------------------------------------------------------
// Streaming statistics kernel.
//
// Token tiles of KT = 32 tokens flow through an NST = 4 stage LDS ring.  Each
// stage holds the tile's rows in their natural [token][channel] order:
// x (source) and y (target) rows of the item's one or two maps, plus the two
// weight rows.  The rows are copied HBM -> LDS by global_load_lds_dwordx4
// (direct-to-LDS DMA, no VGPR staging), three tiles ahead of the tile being
// computed.  Every wave issues the same number of DMA instructions per tile
// (tiles past the end load from a zero buffer), so one explicit vmcnt wait
// plus one barrier per tile tells every wave that the tile has landed.
//
// The MFMA operands are read with ds_read_b64_tr_b16, which transposes 16-bit
// elements across each group of 16 lanes: lane j = a + 4k of a group points
// at channels 4a..4a+3 of token k, and output lane i of the group receives
// channel i of the four tokens.  Two such reads give a lane the eight
// consecutive tokens of one channel that v_mfma_f32_32x32x16_bf16 expects,
// for the x operand of the fold and for every B operand alike.
//
// The 16-byte chunk c of token row t is stored at chunk c ^ h(t), h(t) a
// multiple of 4 chunks that depends on t mod 4 only: the four tokens read by
// one 16-lane group fall in different 64-byte windows (no bank conflict), and
// the column-block offset stays a per-lane XOR.
// ---------------------------------------------------------------------------

template <int DS, int DT>
struct Cfg {
    static constexpr int RB = DS / 32, RBT = DT / 32;
    static constexpr int NW = 2 * RB, NT = 64 * NW;            // waves: (slot, row block)
    static constexpr int KT = kStatsTileTokens;                 // tokens per tile
    static constexpr int NST = 4;                               // LDS ring stages
    static constexpr int NCBX = DS / 8, NCBY = DT / 8;          // 16-byte chunks per row
    static constexpr int ROWX = DS * 2, ROWY = DT * 2;          // bytes per row
    static constexpr int CHX = KT * NCBX, CHY = KT * NCBY;      // chunks per tensor tile
    static constexpr int XB = CHX * 16, YB = CHY * 16;
    static constexpr int OFF_W = 2 * XB + 2 * YB;               // weights: [2 slots][KT] fp32
    static constexpr int OFF_DUMMY = OFF_W + 2 * KT * 4;        // 16 bytes no one reads
    static constexpr int STAGE = OFF_DUMMY + 16;
    static constexpr int LDS = NST * STAGE;
    static constexpr int EPW = (2 * KT + NW - 1) / NW;          // weight entries per wave
    static constexpr int LMAX = (2 * CHX + 2 * CHY + NT - 1) / NT;   // DMA loads per wave per tile
    static constexpr int NTG = RB * (RB + 1) / 2, NTC = RB * RBT;
    static constexpr int SUMX = (NTG + NTC) * 1024, SUMY = SUMX + RB * 64, SUMW = SUMY + RBT * 64;
    static constexpr int SLOT = SUMW + 64;
    static_assert(KT == 32, "the transposed-read addressing assumes 32-token tiles");
    static_assert(CHX % 64 == 0 && CHY % 64 == 0, "a DMA instruction must stay inside one tensor");

    __host__ __device__ static constexpr int chunks(int nt) {
        return nt == 2 ? CHX + CHY : nt == 3 ? CHX + 2 * CHY : 2 * CHX + 2 * CHY;
    }
    __host__ __device__ static constexpr int loads(int nt) { return (chunks(nt) + NT - 1) / NT; }
};

// Token-dependent chunk swizzle h(t) (a multiple of 4 chunks), for rows of
// NCB 16-byte chunks.  Depends on t mod 4 only.
template <int NCB>
__device__ __forceinline__ uint32_t swz(uint32_t t) {
    if constexpr (NCB == 16) return 4u * (t & 3u);
    else if constexpr (NCB == 8) return 4u * ((t >> 1) & 1u);
    else return 0u;
}

// Index of accumulator element (row i, col j) of a 32x32 tile stored as
// [v][lane]: v_mfma_f32_32x32x16 leaves D[i][j] in lane j + 32*((i>>2)&1),
// register v = 4*(i>>3) + (i&3).
__device__ __forceinline__ int acc_index(int tile, int i, int j) {
    return tile * 1024 + (4 * (i >> 3) + (i & 3)) * 64 + j + 32 * ((i >> 2) & 1);
}

template <int RB>
__host__ __device__ constexpr int tri_tile(int r, int c) {  // upper-triangle tile id, c >= r
    return r * RB - (r * (r - 1)) / 2 + (c - r);
}

typedef __attribute__((ext_vector_type(4))) short s16x4_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((address_space(3))) f32x4_t lds_f32x4_t;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;
typedef __attribute__((address_space(3))) char lds_char_t;

// HBM -> LDS copies.  The LDS destination of lane l is M0 + 16 l (4 l for the
// dword form).  They are issued through inline assembly so that the compiler
// does not add its own conservative waits between them and the LDS reads of
// other ring stages; completion is tracked with explicit vmcnt waits below.
// M0 is saved and restored around each copy, so the compiler's own use of it
// is unaffected.
__device__ __forceinline__ void dma16(const void *gaddr, uint32_t m0) {
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "v"(gaddr), "s"(m0)
                 : "memory");
}
__device__ __forceinline__ void dma16_sbase(uint32_t voff, const void *sbase, uint32_t m0) {
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\tglobal_load_lds_dwordx4 %1, %2\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "v"(voff), "s"(sbase), "s"(m0)
                 : "memory");
}
__device__ __forceinline__ void dma4(const void *gaddr, uint32_t m0) {
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dword %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "v"(gaddr), "s"(m0)
                 : "memory");
}

// A pointer that is the same in every lane, placed in SGPRs.
__device__ __forceinline__ const void *uniform_ptr(const void *p) {
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (const void *)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// vmcnt wait with a run-time count (the possible counts are small and even).
__device__ __forceinline__ void wait_vm_rt(int n) {
    switch (n) {
        case 0: wait_vm<0>(); break;
        case 2: wait_vm<2>(); break;
        case 4: wait_vm<4>(); break;
        case 6: wait_vm<6>(); break;
        case 8: wait_vm<8>(); break;
        case 10: wait_vm<10>(); break;
        case 12: wait_vm<12>(); break;
        case 14: wait_vm<14>(); break;
        case 16: wait_vm<16>(); break;
        case 18: wait_vm<18>(); break;
        default: wait_vm<0>(); break;
    }
}

__device__ __forceinline__ bf16x8_t tr_read8(const lds_char_t *p0, const lds_char_t *p1) {
    const s16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)p0);
    const s16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)p1);
    typedef __attribute__((ext_vector_type(8))) short s16x8_t;
    const s16x8_t c = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8_t, c);
}

// Per-workgroup context (wave-uniform values).
struct StatsCtx {
    int unit, tok_begin, tok_end, n_tiles, n_slots, nt;
    bool shared_x;
    const uint16_t *tp[4];       // x0, y0, x1, y1 block bases
    const float *wrow[2];
};

// Issue the DMA copies of tile `tile` (any index; tiles past the end copy zeros)
// into ring stage `st`.  Every wave issues exactly loads(nt) + 1 instructions.
template <int DS, int DT>
__device__ __forceinline__ void issue_tile(const StatsArgs &a, const StatsCtx c, lds_char_t *lds, int wave,
                                           int lane, int tile, int st, const uint32_t *fast_off) {
    using K = Cfg<DS, DT>;
    const int t0 = c.tok_begin + tile * K::KT;
    const bool in_range = tile < c.n_tiles;
    const bool fast = a.fast_tiles && in_range && (t0 + K::KT <= c.tok_end);
    const uint32_t stage = (uint32_t)(uintptr_t)(lds + st * K::STAGE);
    const int total = K::chunks(c.nt);
    uint32_t b_tile = 0, tt_tile = 0;
    if (fast) {
        b_tile = fastdiv((uint32_t)t0, a.T);
        tt_tile = (uint32_t)t0 - b_tile * a.T.d;
    }
#pragma unroll
    for (int i = 0; i < K::LMAX; ++i) {
        if (i < K::loads(c.nt)) {
            const int q0 = (i * K::NW + wave) * 64;         // first chunk of this instruction
            const uint32_t m0 = __builtin_amdgcn_readfirstlane(stage + q0 * 16);
            if (q0 < total) {
                // tensor of this instruction (uniform)
                int ten, qs;
                if (q0 < K::CHX) { ten = 0; qs = 0; }
                else if (q0 < K::CHX + K::CHY) { ten = 1; qs = K::CHX; }
                else if (c.nt == 3) { ten = 3; qs = K::CHX + K::CHY; }
                else if (q0 < 2 * K::CHX + K::CHY) { ten = 2; qs = K::CHX + K::CHY; }
                else { ten = 3; qs = 2 * K::CHX + K::CHY; }
                const bool isx = (ten == 0 || ten == 2);
                const uint16_t *tb = ten == 0 ? c.tp[0] : ten == 1 ? c.tp[1] : ten == 2 ? c.tp[2] : c.tp[3];
                const int64_t sseq = isx ? a.ss.seq : a.ts.seq;
                const int64_t stok = isx ? a.ss.tok : a.ts.tok;
                if (fast) {
                    const uint16_t *base = tb + (int64_t)b_tile * sseq + (int64_t)tt_tile * stok;
                    dma16_sbase(fast_off[i], uniform_ptr(base), m0);
                } else {
                    const int ncb = isx ? K::NCBX : K::NCBY;
                    const int q = q0 - qs + lane;
                    const int t = q / ncb, p = q - (q / ncb) * ncb;
                    const uint32_t h = isx ? swz<K::NCBX>(t) : swz<K::NCBY>(t);
                    const int cch = p ^ (int)h;
                    const int tau = t0 + t;
                    const void *g = a.zero;
                    if (in_range && tau < c.tok_end) {
                        const uint32_t b = fastdiv((uint32_t)tau, a.T);
                        const uint32_t tt = (uint32_t)tau - b * a.T.d;
                        g = tb + (int64_t)b * sseq + (int64_t)tt * stok + cch * 8;
                    }
                    dma16(g, m0);
                }
            } else {
                // no chunk left for this instruction: keep the count uniform by
                // copying 16 zero bytes into the stage's unused slot
                const uint32_t md = __builtin_amdgcn_readfirstlane(stage + K::OFF_DUMMY);
                if (lane == 0) dma16(a.zero, md);
            }
        }
    }
    // weights: entries e = lane of [2 slots][KT tokens], this wave's share only
    const uint32_t mw = __builtin_amdgcn_readfirstlane(stage + K::OFF_W);
    const int e = lane;
    if (e >= wave * K::EPW && e < (wave + 1) * K::EPW && e < 2 * K::KT) {
        const int sl = e / K::KT, t = e % K::KT;
        const void *g = a.zero;
        if (in_range && sl < c.n_slots && t0 + t < c.tok_end) g = (sl ? c.wrow[1] : c.wrow[0]) + t0 + t;
        dma4(g, mw);
    } else if (wave * K::EPW >= 2 * K::KT && lane == 0) {
        // waves without weight entries still issue one copy (into the unused slot)
        dma4(a.zero, __builtin_amdgcn_readfirstlane(stage + K::OFF_DUMMY));
    }
}

// Accumulators and MFMA work of row block R of one map.
template <int DS, int DT, int R>
struct RowBlock {
    using K = Cfg<DS, DT>;
    static constexpr int NG = K::RB - R;     // Gram tiles (R, R..RB-1)
    f32x16_t accg[NG];
    f32x16_t accc[K::RBT];
    float sumx;
    float sumy[K::RBT];
    float sumw;

    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int c = 0; c < NG; ++c)
#pragma unroll
            for (int v = 0; v < 16; ++v) accg[c][v] = 0.f;
#pragma unroll
        for (int c = 0; c < K::RBT; ++c)
#pragma unroll
            for (int v = 0; v < 16; ++v) accc[c][v] = 0.f;
        sumx = 0.f;
        sumw = 0.f;
#pragma unroll
        for (int c = 0; c < K::RBT; ++c) sumy[c] = 0.f;
    }

    // One 16-token K step: bx[c] holds x columns (R + c)*32.. (bx[0] is also the
    // A operand's x), by[] the y columns, w the weights of this lane's 8 tokens.
    __device__ __forceinline__ void step(const bf16x8_t *bx, const bf16x8_t *by, const float *w) {
        const uint4 ax = __builtin_bit_cast(uint4, bx[0]);
        const uint32_t xv[4] = {ax.x, ax.y, ax.z, ax.w};
        float av[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            av[2 * e] = w[2 * e] * bf_lo(xv[e]);
            av[2 * e + 1] = w[2 * e + 1] * bf_hi(xv[e]);
        }
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            hi[e] = pack_bf16(av[2 * e], av[2 * e + 1]);
            lo[e] = pack_bf16(av[2 * e] - bf_lo(hi[e]), av[2 * e + 1] - bf_hi(hi[e]));
        }
        float sa = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) sa += av[e];
        sumx += sa;
        if (R == 0) {
            float sw = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) sw += w[e];
            sumw += sw;
        }
#pragma unroll
        for (int c = 0; c < K::RBT; ++c) {
            if (c % K::RB == R) {
                const uint4 yv = __builtin_bit_cast(uint4, by[c]);
                const uint32_t yy[4] = {yv.x, yv.y, yv.z, yv.w};
                float sy = 0.f;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    sy += w[2 * e] * bf_lo(yy[e]);
                    sy += w[2 * e + 1] * bf_hi(yy[e]);
                }
                sumy[c] += sy;
            }
        }
        const bf16x8_t ahi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
        const bf16x8_t alo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
#pragma unroll
        for (int c = 0; c < NG; ++c)
            accg[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi, bx[c], accg[c], 0, 0, 0);
#pragma unroll
        for (int c = 0; c < K::RBT; ++c)
            accc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi, by[c], accc[c], 0, 0, 0);
#pragma unroll
        for (int c = 0; c < NG; ++c)
            accg[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo, bx[c], accg[c], 0, 0, 0);
#pragma unroll
        for (int c = 0; c < K::RBT; ++c)
            accc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo, by[c], accc[c], 0, 0, 0);
    }

    __device__ __forceinline__ void flush(float *P, int lane) const {
#pragma unroll
        for (int c = 0; c < NG; ++c) {
            float *dst = P + tri_tile<K::RB>(R, R + c) * 1024 + lane;
#pragma unroll
            for (int v = 0; v < 16; ++v) dst[v * 64] = accg[c][v];
        }
#pragma unroll
        for (int c = 0; c < K::RBT; ++c) {
            float *dst = P + (K::NTG + R * K::RBT + c) * 1024 + lane;
#pragma unroll
            for (int v = 0; v < 16; ++v) dst[v * 64] = accc[c][v];
        }
        P[K::SUMX + R * 64 + lane] = sumx;
#pragma unroll
        for (int c = 0; c < K::RBT; ++c)
            if (c % K::RB == R) P[K::SUMY + c * 64 + lane] = sumy[c];
        if (R == 0) P[K::SUMW + lane] = sumw;
    }
};

// The token loop of one wave owning row block R of map slot `slot`.
template <int DS, int DT, int R>
__device__ __forceinline__ void stats_wave(const StatsArgs &a, const StatsCtx c, lds_char_t *lds, int wave,
                                           int lane, int slot) {
    using K = Cfg<DS, DT>;
    constexpr int NBX = K::RB - R;
    const bool active = slot < c.n_slots;
    RowBlock<DS, DT, R> blk;
    blk.zero();

    // LDS offsets of this slot's tensors inside a stage
    const int xoff = (slot == 0 || c.nt != 4) ? 0 : K::XB + K::YB;
    const int yoff = slot == 0 ? K::XB : (c.nt == 4 ? 2 * K::XB + K::YB : K::XB + K::YB);
    const int woff = K::OFF_W + slot * K::KT * 4;

    // Transposed-read lane geometry (see the file comment): group g = lane/16,
    // j = a + 4k inside the group.
    const int g = lane >> 4, j = lane & 15, aa = j & 3, kk = j >> 2;
    const int tok_l = 8 * (g >> 1) + kk;                       // token within the 16-token step
    const int cl = 2 * (g & 1) + (aa >> 1);                    // chunk within the 64-byte window
    const uint32_t lx = tok_l * K::ROWX + cl * 16 + (aa & 1) * 8;
    const uint32_t ly = tok_l * K::ROWY + cl * 16 + (aa & 1) * 8;
    const uint32_t hx = swz<K::NCBX>(kk) >> 2, hy = swz<K::NCBY>(kk) >> 2;
    const uint32_t wl = (lane >> 5) * 32;                      // byte offset of this lane's 8 weights

    // Per-lane source offsets of the fast DMA path: chunk (t, p) of the
    // instruction's tensor comes from global chunk p ^ h(t) of token t.
    uint32_t fast_off[K::LMAX];
#pragma unroll
    for (int i = 0; i < K::LMAX; ++i) {
        fast_off[i] = 0;
        if (i < K::loads(c.nt)) {
            const int q0 = (i * K::NW + wave) * 64;
            if (q0 < K::chunks(c.nt)) {
                int qs;
                bool isx;
                if (q0 < K::CHX) { qs = 0; isx = true; }
                else if (q0 < K::CHX + K::CHY) { qs = K::CHX; isx = false; }
                else if (c.nt == 3) { qs = K::CHX + K::CHY; isx = false; }
                else if (q0 < 2 * K::CHX + K::CHY) { qs = K::CHX + K::CHY; isx = true; }
                else { qs = 2 * K::CHX + K::CHY; isx = false; }
                const int ncb = isx ? K::NCBX : K::NCBY;
                const int q = q0 - qs + lane;
                const int t = q / ncb, p = q - (q / ncb) * ncb;
                const uint32_t h = isx ? swz<K::NCBX>(t) : swz<K::NCBY>(t);
                const int64_t stok = isx ? a.ss.tok : a.ts.tok;
                fast_off[i] = (uint32_t)(((int64_t)t * stok + (int64_t)((p ^ (int)h) * 8)) * 2);
            }
        }
    }

    const int vm_per_tile = K::loads(c.nt) + 1;
    // prologue: tiles 0, 1, 2
#pragma unroll
    for (int t = 0; t < K::NST - 1; ++t) issue_tile<DS, DT>(a, c, lds, wave, lane, t, t, fast_off);

    for (int tile = 0; tile < c.n_tiles; ++tile) {
        wait_vm_rt(2 * vm_per_tile);              // this wave's copies of `tile` have landed
        __builtin_amdgcn_s_waitcnt(0xC07F);       // and its LDS reads of the previous tile are done
        __builtin_amdgcn_s_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        issue_tile<DS, DT>(a, c, lds, wave, lane, tile + K::NST - 1, (tile + K::NST - 1) % K::NST, fast_off);
        if (active) {
            const lds_char_t *S = lds + (tile % K::NST) * K::STAGE;
#pragma unroll
            for (int ks = 0; ks < K::KT / 16; ++ks) {
                bf16x8_t bx[NBX], by[K::RBT];
#pragma unroll
                for (int cc = 0; cc < NBX; ++cc) {
                    const lds_char_t *p = S + xoff + lx + 64u * ((uint32_t)(R + cc) ^ hx) + 16 * ks * K::ROWX;
                    bx[cc] = tr_read8(p, p + 4 * K::ROWX);
                }
#pragma unroll
                for (int cc = 0; cc < K::RBT; ++cc) {
                    const lds_char_t *p = S + yoff + ly + 64u * ((uint32_t)cc ^ hy) + 16 * ks * K::ROWY;
                    by[cc] = tr_read8(p, p + 4 * K::ROWY);
                }
                const f32x4_t w0 = *(const lds_f32x4_t *)(S + woff + 64 * ks + wl);
                const f32x4_t w1 = *(const lds_f32x4_t *)(S + woff + 64 * ks + wl + 16);
                const float w[8] = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
                blk.step(bx, by, w);
            }
        }
    }
    wait_vm<0>();                                  // drain the trailing copies before leaving
    if (active) {
        float *P = a.partials + ((int64_t)c.unit * 2 + slot) * K::SLOT;
        blk.flush(P, lane);
    }
}

template <int DS, int DT>
__global__ __attribute__((amdgpu_flat_work_group_size(Cfg<DS, DT>::NT, Cfg<DS, DT>::NT),
                          amdgpu_waves_per_eu(2, 2)))
void stats_kernel(StatsArgs a) {
    using K = Cfg<DS, DT>;
    __shared__ __attribute__((aligned(16))) char lds_raw[K::LDS];
    lds_char_t *lds = (lds_char_t *)lds_raw;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    StatsCtx c;
    c.unit = blockIdx.x;
    const int item_id = c.unit % a.n_items;
    const int chunk = c.unit / a.n_items;
    const StatsItem it = a.items[item_id];
    c.n_slots = it.n_slots;
    c.shared_x = it.shared_x != 0;
    c.nt = c.n_slots == 1 ? 2 : (c.shared_x ? 3 : 4);
    c.tok_begin = chunk * a.chunk_tokens;
    c.tok_end = min(a.N, c.tok_begin + a.chunk_tokens);
    c.n_tiles = c.tok_end > c.tok_begin ? (c.tok_end - c.tok_begin + K::KT - 1) / K::KT : 0;
    c.tp[0] = a.src + it.src_layer[0] * a.ss.layer + it.kv[0] * a.ss.kv + it.src_head[0] * a.ss.head;
    c.tp[1] = a.tgt + it.tgt_layer[0] * a.ts.layer + it.kv[0] * a.ts.kv + it.tgt_head[0] * a.ts.head;
    c.tp[2] = a.src + it.src_layer[1] * a.ss.layer + it.kv[1] * a.ss.kv + it.src_head[1] * a.ss.head;
    c.tp[3] = a.tgt + it.tgt_layer[1] * a.ts.layer + it.kv[1] * a.ts.kv + it.tgt_head[1] * a.ts.head;
    c.wrow[0] = a.w + (int64_t)it.wrow[0] * a.w_row_stride;
    c.wrow[1] = a.w + (int64_t)it.wrow[1] * a.w_row_stride;

    // wave -> (slot, row block).  With four row blocks the two waves sharing a
    // SIMD (w, w + 4) get blocks (0,3) or (1,2), which balances MFMA work.
    int slot, rb;
    if (K::RB == 4) {
        slot = (wave >> 1) & 1;
        const int r = wave & 1;
        rb = wave < 4 ? r : 3 - r;
    } else {
        slot = wave / K::RB;
        rb = wave % K::RB;
    }
    if (rb == 0) stats_wave<DS, DT, 0>(a, c, lds, wave, lane, slot);
    else if (rb == 1) stats_wave<DS, DT, 1>(a, c, lds, wave, lane, slot);
    else if (rb == 2) stats_wave<DS, DT, (K::RB > 2 ? 2 : 0)>(a, c, lds, wave, lane, slot);
    else stats_wave<DS, DT, (K::RB > 3 ? 3 : 0)>(a, c, lds, wave, lane, slot);
}

template <int DS, int DT>
__global__ __launch_bounds__(256) void reduce_kernel(ReduceArgs a) {
    using K = Cfg<DS, DT>;
    constexpr int P = DS + 1;
    const int m = blockIdx.x;
    const int item = a.map_item[m], slot = a.map_slot[m];
    float *G = a.G + (int64_t)m * P * P;
    float *Cm = a.C + (int64_t)m * P * DT;
    const int64_t chunk_stride = (int64_t)a.n_items * 2 * K::SLOT;
    const float *base = a.partials + ((int64_t)item * 2 + slot) * K::SLOT;
    for (int e = threadIdx.x; e < P * P + P * DT; e += blockDim.x) {
        int i0, i1 = -1;
        float *dst;
        if (e < P * P) {
            const int i = e / P, j = e - (e / P) * P;
            const int r = min(i, j), c = max(i, j);
            if (c < DS) {
                i0 = acc_index(tri_tile<K::RB>(r >> 5, c >> 5), r & 31, c & 31);
            } else if (r < DS) {
                i0 = K::SUMX + (r >> 5) * 64 + (r & 31);
                i1 = i0 + 32;
            } else {
                i0 = K::SUMW;
                i1 = K::SUMW + 32;
            }
            dst = G + e;
        } else {
            const int f = e - P * P;
            const int i = f / DT, j = f - (f / DT) * DT;
            if (i < DS) {
                i0 = acc_index(K::NTG + (i >> 5) * K::RBT + (j >> 5), i & 31, j & 31);
            } else {
                i0 = K::SUMY + (j >> 5) * 64 + (j & 31);
                i1 = i0 + 32;
            }
            dst = Cm + f;
        }
        float s = 0.f;
        for (int ch = 0; ch < a.n_chunks; ++ch) {
            const float *p = base + ch * chunk_stride;
            s += p[i0];
            if (i1 >= 0) s += p[i1];
        }
        *dst += s;
    }
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float *p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0.f;
}

template <int DS, int DT>
hipError_t launch_stats_t(const StatsArgs &a, hipStream_t s) {
    using K = Cfg<DS, DT>;
    const int grid = a.n_items * a.n_chunks;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL((stats_kernel<DS, DT>), dim3(grid), dim3(K::NT), 0, s, a);
    return hipGetLastError();
}

template <int DS, int DT>
hipError_t launch_reduce_t(const ReduceArgs &a, hipStream_t s) {
    if (a.n_maps == 0) return hipSuccess;
    hipLaunchKernelGGL((reduce_kernel<DS, DT>), dim3(a.n_maps), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

#define CB_DISPATCH(FN, d_s, d_t, ...)                                        \
    switch ((d_s) * 1000 + (d_t)) {                                          \
        case 64064: return FN<64, 64>(__VA_ARGS__);                          \
        case 64096: return FN<64, 96>(__VA_ARGS__);                          \
        case 64128: return FN<64, 128>(__VA_ARGS__);                         \
        case 96064: return FN<96, 64>(__VA_ARGS__);                          \
        case 96096: return FN<96, 96>(__VA_ARGS__);                          \
        case 96128: return FN<96, 128>(__VA_ARGS__);                         \
        case 128064: return FN<128, 64>(__VA_ARGS__);                        \
        case 128096: return FN<128, 96>(__VA_ARGS__);                        \
        case 128128: return FN<128, 128>(__VA_ARGS__);                       \
        default: return hipErrorInvalidValue;                                \
    }

hipError_t launch_stats(int d_s, int d_t, const StatsArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_stats_t, d_s, d_t, a, s);
}

hipError_t launch_reduce(int d_s, int d_t, const ReduceArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_reduce_t, d_s, d_t, a, s);
}

hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

}  // namespace cb

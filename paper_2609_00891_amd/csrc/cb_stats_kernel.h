// cb_stats_kernel.h -- the statistics kernel template (device code), shared by
// the translation units that instantiate it (cb_stats.hip: plain moments;
// cb_stats_centered.hip: moments about given weighted means).
#pragma once
#include "cb_internal.h"

namespace cb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) short s16x4_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((address_space(3))) f32x4_t lds_f32x4_t;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;
typedef __attribute__((address_space(3))) char lds_char_t;

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
// A tile is KT = 32 consecutive tokens of one sequence (the last tile of a
// sequence may be partial).  Tiles flow through an NST = 4 stage LDS ring.
// Each stage holds the tile's rows in their natural [token][channel] order:
// x (source) and y (target) rows of the item's one or two maps, plus the two
// weight rows.  The rows are copied HBM -> LDS by global_load_lds_dwordx4
// (direct-to-LDS DMA, no VGPR staging), three tiles ahead of the tile being
// read.  Each wave waits for its own copies with an explicit vmcnt wait and
// then meets the others at one barrier per tile.
//
// Tokens past the end of a partial tile are copied from the sequence's last
// token and given weight zero (their weights are copied from a zero buffer),
// so they add exactly nothing; tiles past the end of a chunk likewise repeat
// the chunk's last tile with zero weights, which keeps the pipeline free of
// branches.
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
    static constexpr int NW = 4, NT = 64 * NW;                  // waves: (slot, pair)
    static constexpr int KT = kStatsTileTokens;                 // tokens per tile
    static constexpr int NST = 4;                               // LDS ring stages
    static constexpr int NCBX = DS / 8, NCBY = DT / 8;          // 16-byte chunks per row
    static constexpr int ROWX = DS * 2, ROWY = DT * 2;          // bytes per row
    static constexpr int CHX = KT * NCBX, CHY = KT * NCBY;      // chunks per tensor tile
    static constexpr int XB = CHX * 16, YB = CHY * 16;
    static constexpr int OFF_W = 2 * XB + 2 * YB;               // weights: [2 slots][KT] fp32
    static constexpr int STAGE = OFF_W + 2 * KT * 4;
    static constexpr int LDS = NST * STAGE;
    static constexpr int NTG = RB * (RB + 1) / 2, NTC = RB * RBT;
    static constexpr int SUMX = (NTG + NTC) * 1024, SUMY = SUMX + RB * 64, SUMW = SUMY + RBT * 64;
    static constexpr int SLOT = SUMW + 64;
    static_assert(KT == 32, "the transposed-read addressing assumes 32-token tiles");
    static_assert(CHX % 64 == 0 && CHY % 64 == 0, "a copy instruction must stay inside one tensor");
    static_assert(LDS <= 160 * 1024, "the ring must fit in LDS");

    __host__ __device__ static constexpr int chunks(int nt) {
        return nt == 2 ? CHX + CHY : nt == 3 ? CHX + 2 * CHY : 2 * CHX + 2 * CHY;
    }
};

// Token-dependent chunk swizzle h(t) (a multiple of 4 chunks), for rows of
// NCB 16-byte chunks.  Depends on t mod 4 only.
template <int NCB>
__host__ __device__ __forceinline__ uint32_t swz(uint32_t t) {
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

// What the wave of pair P computes for a map with RB row blocks: its own row
// blocks row[0..NR-1], the x column blocks xc[0..NX-1] it reads (the first NR
// of them are its own rows, the sources of its folded A operands), and its
// Gram tiles g = (row[gr[g]], xc[gx[g]]).  A Gram block G[r][c] (r != c) is
// computed once, by the owner of r or of c; the two pairs together cover the
// RB(RB+1)/2 blocks of one triangle, and each computes NR * RBT cross tiles.
template <int RB, int P> struct Own;
template <> struct Own<4, 0> {
    static constexpr int NR = 2, NX = 3, NG = 5;
    static constexpr int row[2] = {0, 1}, xc[4] = {0, 1, 2, 0};
    static constexpr int gr[5] = {0, 0, 1, 0, 1}, gx[5] = {0, 1, 1, 2, 2};
};
template <> struct Own<4, 1> {
    static constexpr int NR = 2, NX = 4, NG = 5;
    static constexpr int row[2] = {2, 3}, xc[4] = {2, 3, 0, 1};
    static constexpr int gr[5] = {0, 0, 1, 1, 1}, gx[5] = {0, 1, 1, 2, 3};
};
template <> struct Own<3, 0> {
    static constexpr int NR = 2, NX = 2, NG = 3;
    static constexpr int row[2] = {0, 1}, xc[4] = {0, 1, 0, 0};
    static constexpr int gr[5] = {0, 0, 1, 0, 0}, gx[5] = {0, 1, 1, 0, 0};
};
template <> struct Own<3, 1> {
    static constexpr int NR = 1, NX = 3, NG = 3;
    static constexpr int row[2] = {2, 0}, xc[4] = {2, 0, 1, 0};
    static constexpr int gr[5] = {0, 0, 0, 0, 0}, gx[5] = {0, 1, 2, 0, 0};
};
template <> struct Own<2, 0> {
    static constexpr int NR = 1, NX = 2, NG = 2;
    static constexpr int row[2] = {0, 0}, xc[4] = {0, 1, 0, 0};
    static constexpr int gr[5] = {0, 0, 0, 0, 0}, gx[5] = {0, 1, 0, 0, 0};
};
template <> struct Own<2, 1> {
    static constexpr int NR = 1, NX = 1, NG = 1;
    static constexpr int row[2] = {1, 0}, xc[4] = {1, 0, 0, 0};
    static constexpr int gr[5] = {0, 0, 0, 0, 0}, gx[5] = {0, 0, 0, 0, 0};
};

// HBM -> LDS copies.  The LDS destination of lane l is M0 + 16 l (4 l for the
// dword form).  They are issued through inline assembly so that the compiler
// does not add its own conservative waits between them and the LDS reads of
// other ring stages; completion is tracked with explicit vmcnt waits below.
// M0 (and EXEC, where a copy is limited to some lanes) is saved and restored
// inside the statement, so the compiler's own use of them is unaffected.  The
// row copies carry the non-temporal hint: every row is read once per call.
__device__ __forceinline__ void dma16_sbase(uint32_t voff, const void *sbase, uint32_t m0) {
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\tglobal_load_lds_dwordx4 %1, %2 nt\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "v"(voff), "s"(sbase), "s"(m0)
                 : "memory");
}
// Two copies into LDS destinations m0 and m0 + 4096 under one M0 save/restore.
__device__ __forceinline__ void dma16_pair(uint32_t va, const void *sa, uint32_t vb, const void *sb, uint32_t m0) {
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %5\n\tglobal_load_lds_dwordx4 %1, %2 nt\n\t"
                 "s_add_u32 m0, m0, 0x1000\n\tglobal_load_lds_dwordx4 %3, %4 nt\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "v"(va), "s"(sa), "v"(vb), "s"(sb), "s"(m0)
                 : "memory", "scc");
}
// Dword copy by the lanes set in `lanes` only (the wave is otherwise fully active).
__device__ __forceinline__ void dma4_lanes(const void *gaddr, uint32_t m0, uint64_t lanes) {
    uint64_t keep_exec;
    uint32_t keep_m0;
    asm volatile(
        "s_mov_b64 %0, exec\n\t"
        "s_mov_b64 exec, %3\n\t"
        "s_mov_b32 %1, m0\n\t"
        "s_mov_b32 m0, %4\n\t"
        "global_load_lds_dword %2, off\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_mov_b64 exec, %0"
        : "=&s"(keep_exec), "=&s"(keep_m0)
        : "v"(gaddr), "s"(lanes), "s"(m0)
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
// vmcnt wait with a run-time count (0 <= n <= 31).
__device__ __forceinline__ void wait_vm_rt(int n) {
    switch (n) {
#define CB_W(k) case k: wait_vm<k>(); break;
        CB_W(1) CB_W(2) CB_W(3) CB_W(4) CB_W(5) CB_W(6) CB_W(7) CB_W(8) CB_W(9) CB_W(10)
        CB_W(11) CB_W(12) CB_W(13) CB_W(14) CB_W(15) CB_W(16) CB_W(17) CB_W(18) CB_W(19) CB_W(20)
        CB_W(21) CB_W(22) CB_W(23) CB_W(24) CB_W(25) CB_W(26) CB_W(27) CB_W(28) CB_W(29) CB_W(30)
        CB_W(31)
#undef CB_W
        default: wait_vm<0>(); break;
    }
}

// LDS-only barrier: every wave's LDS operations have completed, then s_barrier.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt and expcnt left alone
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Rotary table entries (16 bytes) into registers.  Issued through inline
// assembly like the copies, so the explicit vmcnt waits below account for
// them; the registers are only read after wait_vm_tied has named them.
__device__ __forceinline__ void gload16(f32x4_t &v, const float *p) {
    asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(p) : "memory");
}
// vmcnt wait that also marks the eight table registers as written by it, so
// no read of them can be placed before the wait.
template <int N>
__device__ __forceinline__ void wait_vm_tied(f32x4_t (&v)[2][4]) {
    asm volatile("s_waitcnt vmcnt(%8)"
                 : "+v"(v[0][0]), "+v"(v[0][1]), "+v"(v[0][2]), "+v"(v[0][3]), "+v"(v[1][0]), "+v"(v[1][1]),
                   "+v"(v[1][2]), "+v"(v[1][3])
                 : "n"(N)
                 : "memory");
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
    int unit, tile_begin, tile_end, n_tiles, n_slots;
    const uint16_t *tp[4];       // x0, y0, x1, y1 block bases
};

// Copy schedule of one stage for an item streaming NTEN tensors (2: x0 y0;
// 3: x0 y0 y1 with x shared; 4: x0 y0 x1 y1).  The stage's 16-byte chunks
// form groups of 64 (one copy instruction each); copy i of wave w moves group
// 4 i + w.  When every tensor has a multiple of four groups (row widths 64
// and 128) each copy index i names the same tensor in every wave, and every
// wave issues exactly L copies.
template <int DS, int DT, int NTEN>
struct Copies {
    using K = Cfg<DS, DT>;
    static constexpr int GX = K::CHX / 64, GY = K::CHY / 64;
    static constexpr int NG = NTEN == 2 ? GX + GY : NTEN == 3 ? GX + 2 * GY : 2 * GX + 2 * GY;
    static constexpr bool STATIC = GX % 4 == 0 && GY % 4 == 0;
    static constexpr int L = (NG + K::NW - 1) / K::NW;
    // tensor (index into StatsCtx::tp) and first group of the tensor holding group j
    static constexpr int ten(int j) {
        return j < GX ? 0 : j < GX + GY ? 1 : NTEN == 3 ? 3 : j < 2 * GX + GY ? 2 : 3;
    }
    static constexpr int first(int j) {
        return j < GX ? 0 : j < GX + GY ? GX : NTEN == 3 ? GX + GY : j < 2 * GX + GY ? GX + GY : 2 * GX + GY;
    }
    static constexpr bool isx(int j) { return ten(j) == 0 || ten(j) == 2; }
};

// The token loop of the wave of pair PR of map slot `slot`, for an item
// streaming NTEN tensors.  CENTER: the folded operand is w (x - mu_x) with
// mu_x = (sum w x) / (sum w) of the map, read from args.sums.
//
// RS (rotary de-rotation; 1: pairs (i, i + d/2), 2: pairs (2i, 2i + 1);
// d_s = d_t = 64 or 128): the K rows of a tile are turned back by their
// positions' angles in LDS, by the waves that copied them, before any wave
// reads the tile.  Lane l owns one chunk pair of every tensor tile (token row
// ut, logical chunks uc and uc + d/16 -- the half-split partners), both moved
// by its own wave's copies, so a wave needs only its own vmcnt wait before
// turning them.  Tile t + 2 is turned during iteration t (after that
// iteration's copies), and the next iteration's barrier publishes it.  The
// lane's table entries of a tile are loaded right after the tile's copies,
// into one of two register sets (by tile parity), so waiting for them
// demands no more of the copies than the loop already does.  The products
// are those of cb_rope's inverse transform, rounded once to bf16.
template <int DS, int DT, bool RAGGED, bool CENTER, int NTEN, int PR, int RS>
__device__ __forceinline__ void stats_wave(const StatsArgs &a, const StatsCtx c, const StatsItem &it,
                                           lds_char_t *lds, int wave, int lane) {
    using K = Cfg<DS, DT>;
    using O = Own<K::RB, PR>;
    using CP = Copies<DS, DT, NTEN>;
    constexpr int NR = O::NR, NX = O::NX, NG = O::NG, RBT = K::RBT, L = CP::L;
    const int slot = wave >> 1;
    const uint32_t lds_base = (uint32_t)(uintptr_t)lds;

    // ---- copy descriptors of this wave (loop invariant)
    int n_copies = 0;
    const uint16_t *cbase[L];
    bool cisx[L];
    uint32_t cvo[L], ctok[L], cstk[L];
#pragma unroll
    for (int i = 0; i < L; ++i) {
        const int j = CP::STATIC ? 4 * i : 4 * i + wave;     // group (wave-independent part when static)
        cbase[i] = c.tp[0];
        cisx[i] = true;
        cvo[i] = 0;
        ctok[i] = 0;
        cstk[i] = 0;
        if (CP::STATIC || j < CP::NG) {
            n_copies = i + 1;
            const int ten = CP::ten(j);
            const bool isx = CP::isx(j);
            cbase[i] = ten == 0 ? c.tp[0] : ten == 1 ? c.tp[1] : ten == 2 ? c.tp[2] : c.tp[3];
            cisx[i] = isx;
            const int ncb = isx ? K::NCBX : K::NCBY;
            const int q = (4 * i + wave - CP::first(j)) * 64 + lane;   // chunk within the tensor tile
            const int t = q / ncb, p = q - (q / ncb) * ncb;
            const uint32_t h = isx ? swz<K::NCBX>(t) : swz<K::NCBY>(t);
            const int64_t stok = isx ? a.ss.tok : a.ts.tok;
            ctok[i] = (uint32_t)t;
            cstk[i] = (uint32_t)(stok * 2);
            cvo[i] = (uint32_t)((p ^ (int)h) * 16);            // byte offset of the source chunk
            if (!RAGGED) cvo[i] += (uint32_t)t * cstk[i];
        }
    }
    // weights: wave w copies entries 16 w .. 16 w + 15 of [2 slots][KT tokens]
    const float *wlane = a.w + (int64_t)(lane < 32 ? it.wrow[0] : it.wrow[1]) * a.w_row_stride + (lane & 31);
    const uint64_t wlanes = 0xffffull << (16 * wave);
    const int per_tile = (CP::STATIC ? L : n_copies) + 1;    // copies this wave issues per tile

    // ---- rotary de-rotation (RS != 0): this lane's chunk pair and table entries
    static_assert(RS == 0 || (DS == DT && (DS == 64 || DS == 128) && CP::STATIC && !CENTER),
                  "the rotary variant takes d_s = d_t = 64 or 128");
    constexpr int NP = DS / 16;                              // chunk pairs per row
    constexpr int NTB = 8;                                   // table loads per tile: 2 tables x 4
    constexpr int PT = L + 1 + (RS ? NTB : 0);               // vm instructions per tile
    const int ul = lane & 31;
    const int ut = DS == 128 ? 4 * (lane < 32 ? wave : 4 + wave) + (ul >> 3) : 8 * wave + (ul >> 2);
    const int uc = DS == 128 ? (ul & 7) : (ul & 3);
    const bool ulive = DS == 128 || lane < 32;               // d = 64: 32 chunk pairs per wave
    const uint32_t uh = swz<K::NCBX>((uint32_t)ut);
    const uint32_t offA = (uint32_t)ut * K::ROWX + ((uint32_t)uc ^ uh) * 16u;
    const uint32_t offB = (uint32_t)ut * K::ROWX + ((uint32_t)(uc + NP) ^ uh) * 16u;
    typedef f32x4_t TabSet[2][4];
    auto tab_load = [&](TabSet &tb, const auto &q) __attribute__((always_inline)) {
        const uint32_t tok = q.tt0 + (RAGGED ? min((uint32_t)ut, q.tmax) : (uint32_t)ut);
#pragma unroll
        for (int sd = 0; sd < 2; ++sd) {
            const float *row = a.rope_tab[sd] + (int64_t)(a.rope_pos[sd] + (int)tok) * DS;   // d/2 (cos, sin)
            if constexpr (RS == 1) {
#pragma unroll
                for (int j = 0; j < 4; ++j) gload16(tb[sd][j], row + 16 * uc + 4 * j);
            } else {
                gload16(tb[sd][0], row + 8 * uc);
                gload16(tb[sd][1], row + 8 * uc + 4);
                gload16(tb[sd][2], row + 8 * (uc + NP));
                gload16(tb[sd][3], row + 8 * (uc + NP) + 4);
            }
        }
    };
    // which tensors of the item turn: x0 y0 x1 y1 (x1 only with NTEN = 4, y1 with NTEN >= 3)
    const bool rx0 = a.rope_on[0] && it.kv[0] == 0, ry0 = a.rope_on[1] && it.kv[0] == 0;
    const bool rx1 = NTEN == 4 && a.rope_on[0] && it.kv[1] == 0, ry1 = NTEN >= 3 && a.rope_on[1] && it.kv[1] == 0;
    // inverse rotation of this lane's chunk pair of the tensor tile at p
    auto turn_pair = [&](lds_char_t *p, const f32x4_t (&cs)[4]) __attribute__((always_inline)) {
        const u32x4_t A = *(const lds_u32x4_t *)(p + offA);
        const u32x4_t B = *(const lds_u32x4_t *)(p + offB);
        const uint32_t av[4] = {A[0], A[1], A[2], A[3]}, bv[4] = {B[0], B[1], B[2], B[3]};
        uint32_t oa[4], ob[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (RS == 1) {
                // pairs (8 uc + 2e + h, its partner d/2 further on), frequency 8 uc + 2e + h
                const float c0 = cs[e][0], s0 = cs[e][1], c1 = cs[e][2], s1 = cs[e][3];
                const float x0 = bf_lo(av[e]), x1 = bf_hi(av[e]), y0 = bf_lo(bv[e]), y1 = bf_hi(bv[e]);
                oa[e] = pack_bf16(__builtin_fmaf(x0, c0, y0 * s0), __builtin_fmaf(x1, c1, y1 * s1));
                ob[e] = pack_bf16(__builtin_fmaf(y0, c0, -(x0 * s0)), __builtin_fmaf(y1, c1, -(x1 * s1)));
            } else {
                // pairs (2i, 2i + 1) inside each chunk: frequency 4 uc + e, then 4 (uc + d/16) + e
                const f32x4_t qa = cs[e >> 1], qb = cs[2 + (e >> 1)];
                const float ca = (e & 1) ? qa[2] : qa[0], sa = (e & 1) ? qa[3] : qa[1];
                const float cb = (e & 1) ? qb[2] : qb[0], sb = (e & 1) ? qb[3] : qb[1];
                const float x0 = bf_lo(av[e]), x1 = bf_hi(av[e]), y0 = bf_lo(bv[e]), y1 = bf_hi(bv[e]);
                oa[e] = pack_bf16(__builtin_fmaf(x0, ca, x1 * sa), __builtin_fmaf(x1, ca, -(x0 * sa)));
                ob[e] = pack_bf16(__builtin_fmaf(y0, cb, y1 * sb), __builtin_fmaf(y1, cb, -(y0 * sb)));
            }
        }
        const u32x4_t A2 = {oa[0], oa[1], oa[2], oa[3]}, B2 = {ob[0], ob[1], ob[2], ob[3]};
        *(lds_u32x4_t *)(p + offA) = A2;
        *(lds_u32x4_t *)(p + offB) = B2;
    };
    // turn the K tensors of the tile in ring stage st (its copies and its table entries have landed)
    auto turn_tile = [&](const TabSet &tb, int st) __attribute__((always_inline)) {
        if (!ulive) return;
        lds_char_t *S = lds + st * K::STAGE;
        if (rx0) turn_pair(S, tb[0]);
        if (ry0) turn_pair(S + K::XB, tb[1]);
        if (NTEN == 4 && rx1) turn_pair(S + K::XB + K::YB, tb[0]);
        if (NTEN >= 3 && ry1) turn_pair(S + (NTEN == 4 ? 2 * K::XB + K::YB : K::XB + K::YB), tb[1]);
    };

    // Position of the tile a copy reads.  A cursor walks the chunk's tiles in
    // order (32 tokens on, or to the next sequence); tiles past the chunk
    // repeat its last tile with zero weights.
    struct TilePos {
        int64_t offx, offy, wtok;   // element offsets of the tile in the x / y blocks, token of its weights
        uint32_t seq, tt0;          // sequence and first token of the tile
        uint32_t tmax;              // last valid token of the tile
        int t;                      // relative tile index
        bool live;
    };
    auto tile_at = [&](int t) {
        TilePos q;
        q.t = t;
        q.live = t < c.n_tiles;
        const uint32_t u = (uint32_t)(q.live ? c.tile_begin + t : c.tile_end - 1);
        q.seq = fastdiv(u, a.TPS);
        q.tt0 = (u - q.seq * a.TPS.d) * K::KT;
        q.offx = (int64_t)q.seq * a.ss.seq + (int64_t)q.tt0 * a.ss.tok;
        q.offy = (int64_t)q.seq * a.ts.seq + (int64_t)q.tt0 * a.ts.tok;
        q.wtok = (int64_t)q.seq * a.seq_len + q.tt0;
        q.tmax = RAGGED ? min((uint32_t)K::KT - 1, a.seq_len - 1 - q.tt0) : K::KT - 1;
        return q;
    };
    auto tile_next = [&](TilePos &q) {
        if (q.t + 1 < c.n_tiles) {
            q.tt0 += K::KT;
            if (q.tt0 >= a.seq_len) {
                q.tt0 = 0;
                q.seq += 1;
                q.offx = (int64_t)q.seq * a.ss.seq;
                q.offy = (int64_t)q.seq * a.ts.seq;
                q.wtok = (int64_t)q.seq * a.seq_len;
            } else {
                q.offx += K::KT * a.ss.tok;
                q.offy += K::KT * a.ts.tok;
                q.wtok += K::KT;
            }
            if (RAGGED) q.tmax = min((uint32_t)K::KT - 1, a.seq_len - 1 - q.tt0);
        } else {
            q.live = false;                                  // stays on the chunk's last tile
        }
        q.t += 1;
    };
    // Copies of the tile at `q` into ring stage `st`, part `part` of four: the
    // tensor copies 2 part and 2 part + 1 (all of them in part 0 when the
    // schedule is not static), and the weights in part 3.
    auto issue_part = [&](const TilePos &q, int st, int part) {
        const uint32_t stage = lds_base + st * K::STAGE;
        const uint32_t mw = __builtin_amdgcn_readfirstlane(stage + wave * 1024);
        auto src = [&](int i) { return uniform_ptr(cbase[i] + (cisx[i] ? q.offx : q.offy)); };
        auto voff = [&](int i) { return RAGGED ? min(ctok[i], q.tmax) * cstk[i] + cvo[i] : cvo[i]; };
        if constexpr (CP::STATIC) {
            const int i = 2 * part;
            if (i + 1 < L) dma16_pair(voff(i), src(i), voff(i + 1), src(i + 1), mw + i * 4096);
            else if (i < L) dma16_sbase(voff(i), src(i), mw + i * 4096);
        } else if (part == 0) {
#pragma unroll
            for (int i = 0; i < L; ++i)
                if (i < n_copies) dma16_sbase(voff(i), src(i), mw + i * 4096);
        }
        if (part == 3) {
            const bool ok = q.live && (!RAGGED || (uint32_t)(lane & 31) <= q.tmax);
            const void *g = ok ? (const void *)(wlane + q.wtok) : a.zero;
            dma4_lanes(g, __builtin_amdgcn_readfirstlane(stage + K::OFF_W), wlanes);
        }
    };
    auto issue = [&](const TilePos &q, int st) {
#pragma unroll
        for (int part = 0; part < 4; ++part) issue_part(q, st, part);
    };
    auto wait_tiles = [&](int n) {                           // at most n tiles of this wave's copies in flight
        if constexpr (RS != 0) {
            // tiles t+1 / t+2 / t+3 (and their table entries) follow the one waited for
            if (n == 3) wait_vm<2 * PT>();                   // the prologue waited for tiles 0 and 1 already
            else wait_vm<NTB + 2 * PT>();
        } else if constexpr (CP::STATIC) {
            if (n == 3) wait_vm<3 * (L + 1)>();
            else wait_vm<2 * (L + 1)>();
        } else {
            wait_vm_rt(n * per_tile);
        }
    };

    // prologue: tiles 0..3 fill the ring
    TilePos cur = tile_at(0);
    TabSet tA, tB;                                           // table entries of the even / odd tiles
    if constexpr (RS != 0) {
        // tiles 0 and 1 are turned here, before the loop reads them
        issue(cur, 0);
        tab_load(tA, cur);
        tile_next(cur);
        issue(cur, 1);
        tab_load(tB, cur);
        tile_next(cur);
        wait_vm_tied<0>(tA);
        wait_vm_tied<0>(tB);
        turn_tile(tA, 0);
        turn_tile(tB, 1);
        issue(cur, 2);
        tab_load(tA, cur);
        tile_next(cur);
        issue(cur, 3);
        tab_load(tB, cur);
        tile_next(cur);                                      // ends at tile 4, the first one the loop copies
    } else {
#pragma unroll
        for (int t = 0; t < K::NST; ++t) {
            issue(cur, t);
            tile_next(cur);                                  // ends at tile 4, the first one the loop copies
        }
    }
    // In iteration t, after the copies of tile t + 4: tile t + 2 is turned with
    // its table entries (register set of its parity), whose set then receives
    // the entries of tile t + 4.  Only tile t + 3 and its entries and tile
    // t + 4's copies may still be in flight then.
    auto turn_ahead = [&](TabSet &tb, int t, const TilePos &q4) __attribute__((always_inline)) {
        if constexpr (RS != 0) {
            wait_vm_tied<PT + L + 1>(tb);
            turn_tile(tb, (t + 2) % K::NST);
            tab_load(tb, q4);
        }
    };

    if (slot >= c.n_slots) {
        // A wave without a map (single-map item) only helps with the copies; it
        // meets the same barriers as the computing waves below (one before the
        // loop, one per tile of the loop's even trip count).
        wait_tiles(3);
        lds_barrier();
        for (int t = 0; t < ((c.n_tiles + 1) & ~1); t += 2) {
            wait_tiles(2);
            lds_barrier();
            TilePos q = cur;
            issue(q, t % K::NST);
            tile_next(cur);
            turn_ahead(tA, t, q);
            wait_tiles(2);
            lds_barrier();
            q = cur;
            issue(q, (t + 1) % K::NST);
            tile_next(cur);
            turn_ahead(tB, t + 1, q);
        }
        wait_vm<0>();
        return;
    }
    // LDS offsets of this slot's tensors inside a stage
    const uint32_t xoff = (slot == 0 || NTEN != 4) ? 0 : K::XB + K::YB;
    const uint32_t yoff = slot == 0 ? K::XB : (NTEN == 4 ? 2 * K::XB + K::YB : K::XB + K::YB);
    const uint32_t woff = K::OFF_W + slot * K::KT * 4;

    // Transposed-read lane geometry (see the comment above Cfg): group
    // g = lane/16, j = a + 4k inside the group.
    const int g = lane >> 4, j = lane & 15, aa = j & 3, kk = j >> 2;
    const int tok_l = 8 * (g >> 1) + kk;                       // token within the 16-token step
    const int cl = 2 * (g & 1) + (aa >> 1);                    // chunk within the 64-byte window
    const uint32_t hx = swz<K::NCBX>(kk) >> 2, hy = swz<K::NCBY>(kk) >> 2;
    const uint32_t lx = xoff + tok_l * K::ROWX + cl * 16 + (aa & 1) * 8;
    const uint32_t ly = yoff + tok_l * K::ROWY + cl * 16 + (aa & 1) * 8;
    const uint32_t lw = woff + (lane >> 5) * 32;               // this lane's 8 weights

    struct Ops {
        bf16x8_t xf[NX], yf[RBT];
        float w[8];
    };
    // weighted means of this lane's channel of each own row block (CENTER)
    float mu[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        mu[r] = 0.f;
        if constexpr (CENTER) {
            const double *sm = a.sums + (int64_t)it.map[slot] * (1 + DS + DT);
            const double sw = sm[0];
            mu[r] = sw != 0.0 ? (float)(sm[1 + 32 * O::row[r] + (lane & 31)] / sw) : 0.f;
        }
    }
    struct Half {
        bf16x8_t hi[NR], lo[NR];
    };
    f32x16_t accg[NG], accc[NR * RBT];
    float sumx[NR], sumy[RBT], sumw = 0.f;
#pragma unroll
    for (int k = 0; k < NG; ++k)
#pragma unroll
        for (int v = 0; v < 16; ++v) accg[k][v] = 0.f;
#pragma unroll
    for (int k = 0; k < NR * RBT; ++k)
#pragma unroll
        for (int v = 0; v < 16; ++v) accc[k][v] = 0.f;
#pragma unroll
    for (int r = 0; r < NR; ++r) sumx[r] = 0.f;
#pragma unroll
    for (int k = 0; k < RBT; ++k) sumy[k] = 0.f;

    // Operands of K step ks (16 tokens) of ring stage st.
    auto read_ops = [&](Ops &o, int st, int ks) {
        const lds_char_t *S = lds + st * K::STAGE + 16 * ks * K::ROWX;
        const lds_char_t *SY = lds + st * K::STAGE + 16 * ks * K::ROWY;
#pragma unroll
        for (int cc = 0; cc < NX; ++cc) {
            const lds_char_t *p = S + lx + 64u * ((uint32_t)O::xc[cc] ^ hx);
            o.xf[cc] = tr_read8(p, p + 4 * K::ROWX);
        }
#pragma unroll
        for (int cc = 0; cc < RBT; ++cc) {
            const lds_char_t *p = SY + ly + 64u * ((uint32_t)cc ^ hy);
            o.yf[cc] = tr_read8(p, p + 4 * K::ROWY);
        }
        const lds_char_t *pw = lds + st * K::STAGE + lw + 64 * ks;
        const f32x4_t w0 = *(const lds_f32x4_t *)pw;
        const f32x4_t w1 = *(const lds_f32x4_t *)(pw + 16);
        o.w[0] = w0[0]; o.w[1] = w0[1]; o.w[2] = w0[2]; o.w[3] = w0[3];
        o.w[4] = w1[0]; o.w[5] = w1[1]; o.w[6] = w1[2]; o.w[7] = w1[3];
    };
    // Fold of own row block r for one K step: a = w * x for this lane's 8
    // tokens of one channel, split into hi = RNE_bf16(a), lo = RNE_bf16(a - hi);
    // the row's bias sum on the side.
    auto fold_row = [&](Half &h, const Ops &o, int r) {
        const uint4 ax = __builtin_bit_cast(uint4, o.xf[r]);
        const uint32_t xv[4] = {ax.x, ax.y, ax.z, ax.w};
        float av[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (CENTER) {
                av[2 * e] = o.w[2 * e] * (bf_lo(xv[e]) - mu[r]);
                av[2 * e + 1] = o.w[2 * e + 1] * (bf_hi(xv[e]) - mu[r]);
            } else {
                av[2 * e] = o.w[2 * e] * bf_lo(xv[e]);
                av[2 * e + 1] = o.w[2 * e + 1] * bf_hi(xv[e]);
            }
        }
        uint32_t hv[4], lv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            hv[e] = pack_bf16(av[2 * e], av[2 * e + 1]);
            lv[e] = pack_bf16(av[2 * e] - bf_lo(hv[e]), av[2 * e + 1] - bf_hi(hv[e]));
        }
        if constexpr (CENTER) {
            // e = sum of the folded operand exactly as the MFMA multiplies it
            // (hi + lo): subtracting e mu^T then also cancels the split's
            // rounding against the mean of the uncentered right operand.
            float s[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                s[e] = (bf_lo(hv[e]) + bf_lo(lv[e])) + (bf_hi(hv[e]) + bf_hi(lv[e]));
            sumx[r] += (s[0] + s[1]) + (s[2] + s[3]);
        } else {
            sumx[r] += ((av[0] + av[1]) + (av[2] + av[3])) + ((av[4] + av[5]) + (av[6] + av[7]));
        }
        h.hi[r] = __builtin_bit_cast(bf16x8_t, make_uint4(hv[0], hv[1], hv[2], hv[3]));
        h.lo[r] = __builtin_bit_cast(bf16x8_t, make_uint4(lv[0], lv[1], lv[2], lv[3]));
    };
    // Bias sums of one K step that do not depend on the own rows, in two
    // halves: half k adds sum w y over this pair's k-th y column block (blocks
    // PR, PR + 2), and half 1 also sum w (pair 0 only).
    auto fold_sums = [&](const Ops &o, int half) {
        if constexpr (CENTER) {
            if (!a.bias_sums) return;                        // two-pass form: only sum w (x - mu) is needed
        }
        if (PR == 0 && half == 1)
            sumw += ((o.w[0] + o.w[1]) + (o.w[2] + o.w[3])) + ((o.w[4] + o.w[5]) + (o.w[6] + o.w[7]));
        const int cc = PR + 2 * half;
        if (cc < RBT) {
            const uint4 yv = __builtin_bit_cast(uint4, o.yf[cc]);
            const uint32_t yy[4] = {yv.x, yv.y, yv.z, yv.w};
            float py[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                py[2 * e] = o.w[2 * e] * bf_lo(yy[e]);
                py[2 * e + 1] = o.w[2 * e + 1] * bf_hi(yy[e]);
            }
            sumy[cc] += ((py[0] + py[1]) + (py[2] + py[3])) + ((py[4] + py[5]) + (py[6] + py[7]));
        }
    };
    auto fold = [&](Half &h, const Ops &o) {
#pragma unroll
        for (int r = 0; r < NR; ++r) fold_row(h, o, r);
        fold_sums(o, 0);
        fold_sums(o, 1);
    };
    // MFMA work of one K step, as its hi terms and its lo terms (each a set of
    // independent accumulations, so dependent MFMAs are NG + NR RBT apart).
    auto mma_hi = [&](const Half &h, const Ops &o) {
#pragma unroll
        for (int k = 0; k < NG; ++k)
            accg[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(h.hi[O::gr[k]], o.xf[O::gx[k]], accg[k], 0, 0, 0);
#pragma unroll
        for (int r = 0; r < NR; ++r)
#pragma unroll
            for (int cc = 0; cc < RBT; ++cc)
                accc[r * RBT + cc] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(h.hi[r], o.yf[cc], accc[r * RBT + cc], 0, 0, 0);
    };
    auto mma_lo = [&](const Half &h, const Ops &o) {
#pragma unroll
        for (int k = 0; k < NG; ++k)
            accg[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(h.lo[O::gr[k]], o.xf[O::gx[k]], accg[k], 0, 0, 0);
#pragma unroll
        for (int r = 0; r < NR; ++r)
#pragma unroll
            for (int cc = 0; cc < RBT; ++cc)
                accc[r * RBT + cc] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(h.lo[r], o.yf[cc], accc[r * RBT + cc], 0, 0, 0);
    };

    // Keeps the fold of the next step inside the iteration that computes it
    // (otherwise it may be sunk into the next iteration, past its barrier,
    // where it would no longer overlap this iteration's MFMAs).
    auto pin = [&](const Half &h) {
#pragma unroll
        for (int r = 0; r < NR; ++r) asm volatile("" ::"v"(h.hi[r]), "v"(h.lo[r]));
#pragma unroll
        for (int r = 0; r < NR; ++r) asm volatile("" ::"v"(sumx[r]));
#pragma unroll
        for (int cc = 0; cc < RBT; ++cc)
            if (cc % 2 == PR) asm volatile("" ::"v"(sumy[cc]));
        if (PR == 0) asm volatile("" ::"v"(sumw));
    };

    // Scheduling pattern of one region: its MFMAs evenly spread among the
    // other instructions (one MFMA occupies the matrix core for about as long
    // as the wave takes to issue five to six other instructions).
    auto interleave = [&]() {
        constexpr int NM = NG + NR * RBT;                    // MFMAs in the region
#pragma unroll
        for (int k = 0; k < NM; ++k) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read, if any is left
            __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);   // five VALU
        }
    };

    // Software pipeline over K steps s (two per tile): while the MFMAs of step
    // s run, step s+1 is folded and step s+2 is read from LDS.  Iteration t
    // first waits for tile t+1 (read during the iteration) and refills the
    // stage of tile t, which every wave finished reading in iteration t-1.
    // Iteration t enters with the operands of steps 2t, 2t+1 in (i0, i1) and
    // the folded step 2t in f0, and leaves those of the next tile in (n0, n1),
    // f2.  Two iterations per loop trip swap the register sets instead of
    // copying them.
    //
    // The LDS reads of step 2t+2 are issued first, so that they have landed by
    // the time they are folded.  The rest of the iteration is cut into four
    // scheduling regions of about 13 MFMAs each; every region also holds a
    // quarter of the folds and of the copies of tile t+4, which the compiler
    // interleaves with the MFMAs.  A single wave per SIMD issues all of them,
    // so an even mix keeps the matrix core fed.
    auto iteration = [&](int t, const Ops &i0, const Ops &i1, const Half &f0, Ops &n0, Ops &n1, Half &f2,
                         TabSet &tb) {
        const TilePos q = cur;                               // tile t+4
        tile_next(cur);
        wait_tiles(2);                                       // tile t+1 has landed
        lds_barrier();
        const int sn = (t + 1) % K::NST, st = t % K::NST;
        read_ops(n0, sn, 0);
        __builtin_amdgcn_sched_barrier(0);
        Half f1;
        issue_part(q, st, 0);
        fold_row(f1, i1, 0);
        fold_sums(i1, 0);
        mma_hi(f0, i0);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        issue_part(q, st, 1);
        if (NR > 1) fold_row(f1, i1, NR - 1);
        fold_sums(i1, 1);
        mma_lo(f0, i0);
        pin(f1);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        issue_part(q, st, 2);
        fold_row(f2, n0, 0);
        fold_sums(n0, 0);
        read_ops(n1, sn, 1);
        mma_hi(f1, i1);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        issue_part(q, st, 3);
        turn_ahead(tb, t, q);
        if (NR > 1) fold_row(f2, n0, NR - 1);
        fold_sums(n0, 1);
        mma_lo(f1, i1);
        pin(f2);
        interleave();
    };
    wait_tiles(3);                                           // tile 0 has landed
    lds_barrier();
    Ops a0, a1, b0, b1;
    Half fa, fb;
    read_ops(a0, 0, 0);
    read_ops(a1, 0, 1);
    fold(fa, a0);
    for (int t = 0; t < c.n_tiles; t += 2) {                 // an odd count ends with a zero-weight tile
        iteration(t, a0, a1, fa, b0, b1, fb, tA);
        iteration(t + 1, b0, b1, fb, a0, a1, fa, tB);
    }
    wait_vm<0>();                                            // drain the trailing copies before leaving

    float *P = a.partials + ((int64_t)c.unit * 2 + slot) * K::SLOT;
    constexpr int gbase = PR == 0 ? 0 : Own<K::RB, 0>::NG;
#pragma unroll
    for (int k = 0; k < NG; ++k) {
        float *dst = P + (gbase + k) * 1024 + lane;
#pragma unroll
        for (int v = 0; v < 16; ++v) dst[v * 64] = accg[k][v];
    }
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int cc = 0; cc < RBT; ++cc) {
            float *dst = P + (K::NTG + O::row[r] * RBT + cc) * 1024 + lane;
#pragma unroll
            for (int v = 0; v < 16; ++v) dst[v * 64] = accc[r * RBT + cc][v];
        }
#pragma unroll
    for (int r = 0; r < NR; ++r) P[K::SUMX + O::row[r] * 64 + lane] = sumx[r];
#pragma unroll
    for (int cc = 0; cc < RBT; ++cc)
        if (cc % 2 == PR) P[K::SUMY + cc * 64 + lane] = sumy[cc];
    if (PR == 0) P[K::SUMW + lane] = sumw;
}

template <int DS, int DT, bool RAGGED, bool CENTER, int RS = 0>
__global__ __attribute__((amdgpu_flat_work_group_size(Cfg<DS, DT>::NT, Cfg<DS, DT>::NT),
                          amdgpu_waves_per_eu(1, 1)))
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
    const int nt = c.n_slots == 1 ? 2 : (it.shared_x ? 3 : 4);
    c.tile_begin = chunk * a.chunk_tiles;
    c.tile_end = min(a.n_tiles, c.tile_begin + a.chunk_tiles);
    c.n_tiles = max(c.tile_end - c.tile_begin, 0);
    c.tp[0] = a.src + it.src_layer[0] * a.ss.layer + it.kv[0] * a.ss.kv + it.src_head[0] * a.ss.head;
    c.tp[1] = a.tgt + it.tgt_layer[0] * a.ts.layer + it.kv[0] * a.ts.kv + it.tgt_head[0] * a.ts.head;
    c.tp[2] = a.src + it.src_layer[1] * a.ss.layer + it.kv[1] * a.ss.kv + it.src_head[1] * a.ss.head;
    c.tp[3] = a.tgt + it.tgt_layer[1] * a.ts.layer + it.kv[1] * a.ts.kv + it.tgt_head[1] * a.ts.head;
    if (c.n_tiles == 0) return;

    // wave -> (slot, pair): one wave per SIMD
#define CB_WAVE(NTEN)                                                                               \
    if ((wave & 1) == 0) stats_wave<DS, DT, RAGGED, CENTER, NTEN, 0, RS>(a, c, it, lds, wave, lane); \
    else stats_wave<DS, DT, RAGGED, CENTER, NTEN, 1, RS>(a, c, it, lds, wave, lane);
    if (nt == 4) { CB_WAVE(4) }
    else if (nt == 3) { CB_WAVE(3) }
    else { CB_WAVE(2) }
#undef CB_WAVE
}

}  // namespace
}  // namespace cb

// Host dispatch of a launcher template over the supported (d_s, d_t) pairs.
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

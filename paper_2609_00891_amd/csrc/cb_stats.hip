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
//   * 64-token tiles are loaded with 128-bit global loads (16 lanes cover one
//     256-byte row), transposed in registers to channel-major order and
//     stored in LDS with an XOR swizzle (double buffered, one barrier per
//     tile);
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

// Byte offset of 16-byte token block kb (8 tokens) of channel ch in a
// [channel][64 tokens] bf16 tile.  The block index is XORed with a function of
// the channel so that 16 consecutive channels reading the same block land in
// distinct LDS banks, and channels 8 apart (written together by the
// transposing stores) are spread as well.
__device__ __forceinline__ uint32_t tile_off(uint32_t ch, uint32_t kb) {
    const uint32_t h = ((ch >> 1) ^ (ch >> 3)) & 7u;
    return ch * 128u + ((kb ^ h) << 4);
}

// Per-workgroup context of the statistics kernel (wave-uniform values).
struct StatsCtx {
    int unit, tok_begin, tok_end, n_tiles, n_slots, total_jobs, nj2;
    bool shared_x;
    const uint16_t *tp[4];
    const float *wrow[2];
};

// Every workgroup has four waves, two per map slot, at one wave per SIMD
// (512-VGPR budget).  The two waves of a slot split the row blocks of the
// Gram/cross tiles so that their MFMA work is as even as the widths allow:
// d_s = 128: (0,3) and (1,2), 13 tiles each; d_s = 96: (0,2) and (1);
// d_s = 64: (0) and (1).
template <int DS> struct WaveShape;
template <> struct WaveShape<128> { static constexpr int A1 = 0, A2 = 3, B1 = 1, B2 = 2; };
template <> struct WaveShape<96> { static constexpr int A1 = 0, A2 = 2, B1 = 1, B2 = -1; };
template <> struct WaveShape<64> { static constexpr int A1 = 0, A2 = -1, B1 = 1, B2 = -1; };

template <int DS, int DT>
struct Cfg {
    static constexpr int RB = DS / 32, RBT = DT / 32;
    static constexpr int NW = 4, NT = 64 * NW;
    static constexpr int KT = kStatsTileTokens;               // tokens per tile
    static constexpr int NCGX = DS / 8, NCGY = DT / 8;         // 16-byte channel groups per row
    static constexpr int XB = DS * KT * 2, YB = DT * KT * 2;   // bytes of one tile
    static constexpr int OX0 = 0, OX1 = XB, OY0 = 2 * XB, OY1 = 2 * XB + YB;
    static constexpr int OW0 = 2 * XB + 2 * YB, OW1 = OW0 + KT * 4;
    static constexpr int BUF = OW1 + KT * 4;                   // one LDS buffer
    static constexpr int JX = (KT / 4) * NCGX, JY = (KT / 4) * NCGY;  // load jobs per tensor
    static constexpr int MAXJ = (2 * JX + 2 * JY + NT - 1) / NT;
    static constexpr int NTG = RB * (RB + 1) / 2, NTC = RB * RBT;
    static constexpr int SUMX = (NTG + NTC) * 1024, SUMY = SUMX + RB * 64, SUMW = SUMY + RBT * 64;
    static constexpr int SLOT = SUMW + 64;
    static_assert(KT == 64, "tile_off assumes 64-token tiles");
};

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

// Streaming loader: every thread stages its share of the next tile in
// registers (global -> VGPR), then transposes it into LDS.
template <int DS, int DT>
struct Loader {
    using K = Cfg<DS, DT>;
    uint4 stage[K::MAXJ][4];
    float wstage;

    __device__ __forceinline__ static void decode(const StatsCtx &c, int j, int &t, int &jj) {
        if (j < K::JX) { t = 0; jj = j; }
        else if (j < K::JX + K::JY) { t = 1; jj = j - K::JX; }
        else if (j < K::JX + K::JY + c.nj2) { t = 2; jj = j - K::JX - K::JY; }
        else { t = 3; jj = j - K::JX - K::JY - c.nj2; }
    }

    __device__ __forceinline__ void load(const StatsArgs &a, const StatsCtx &c, int tid, int tile) {
        const int t0 = c.tok_begin + tile * K::KT;
#pragma unroll
        for (int s = 0; s < K::MAXJ; ++s) {
            const int j = tid + s * K::NT;
            if (j < c.total_jobs) {
                int t, jj;
                decode(c, j, t, jj);
                const bool isx = (t == 0 || t == 2);
                const int ncg = isx ? K::NCGX : K::NCGY;
                const int cg = jj % ncg, q = jj / ncg;
                const int64_t sseq = isx ? a.ss.seq : a.ts.seq;
                const int64_t stok = isx ? a.ss.tok : a.ts.tok;
                const int tau = t0 + 4 * q;
                uint32_t b = fastdiv((uint32_t)tau, a.T);
                uint32_t tt = (uint32_t)tau - b * a.T.d;
                const uint16_t *tb = t == 0 ? c.tp[0] : t == 1 ? c.tp[1] : t == 2 ? c.tp[2] : c.tp[3];
                const uint16_t *base = tb + cg * 8;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    uint4 v = make_uint4(0, 0, 0, 0);
                    if (tau + r < c.tok_end)
                        v = *reinterpret_cast<const uint4 *>(base + (int64_t)b * sseq + (int64_t)tt * stok);
                    stage[s][r] = v;
                    if (++tt == a.T.d) { tt = 0; ++b; }
                }
            }
        }
        if (tid < 2 * K::KT) {
            const int ws = tid / K::KT, k = tid % K::KT;
            const int tau = t0 + k;
            wstage = 0.f;
            if (ws < c.n_slots && tau < c.tok_end) wstage = (ws ? c.wrow[1] : c.wrow[0])[tau];
        }
    }

    __device__ __forceinline__ void store(const StatsCtx &c, int tid, char *B) {
#pragma unroll
        for (int s = 0; s < K::MAXJ; ++s) {
            const int j = tid + s * K::NT;
            if (j < c.total_jobs) {
                int t, jj;
                decode(c, j, t, jj);
                const bool isx = (t == 0 || t == 2);
                const int ncg = isx ? K::NCGX : K::NCGY;
                const int cg = jj % ncg, q = jj / ncg;
                const int dst = t == 0 ? K::OX0 : t == 1 ? K::OY0 : t == 2 ? K::OX1 : K::OY1;
                const uint32_t v0[4] = {stage[s][0].x, stage[s][0].y, stage[s][0].z, stage[s][0].w};
                const uint32_t v1[4] = {stage[s][1].x, stage[s][1].y, stage[s][1].z, stage[s][1].w};
                const uint32_t v2[4] = {stage[s][2].x, stage[s][2].y, stage[s][2].z, stage[s][2].w};
                const uint32_t v3[4] = {stage[s][3].x, stage[s][3].y, stage[s][3].z, stage[s][3].w};
#pragma unroll
                for (int ch8 = 0; ch8 < 8; ++ch8) {
                    const int d = ch8 >> 1;
                    const uint32_t sel = (ch8 & 1) ? 0x07060302u : 0x05040100u;
                    uint2 o;
                    o.x = __builtin_amdgcn_perm(v1[d], v0[d], sel);   // tokens 4q, 4q+1
                    o.y = __builtin_amdgcn_perm(v3[d], v2[d], sel);   // tokens 4q+2, 4q+3
                    const uint32_t ch = cg * 8 + ch8;
                    *reinterpret_cast<uint2 *>(B + dst + tile_off(ch, q >> 1) + ((q & 1) << 3)) = o;
                }
            }
        }
        if (tid < 2 * K::KT) {
            const int ws = tid / K::KT, k = tid % K::KT;
            reinterpret_cast<float *>(B + (ws ? K::OW1 : K::OW0))[k] = wstage;
        }
    }
};

// Accumulators and MFMA work of one row block R of one map.
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

    // One 16-token K step.  bx[c] holds x columns c*32.. for c >= RMIN (the
    // smallest row block of this wave), by[] the y columns, w the weights of
    // this lane's 8 tokens.
    template <int RMIN>
    __device__ __forceinline__ void step(const bf16x8_t *bx, const bf16x8_t *by, const float *w) {
        const uint4 ax = __builtin_bit_cast(uint4, bx[R - RMIN]);
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
            accg[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi, bx[R + c - RMIN], accg[c], 0, 0, 0);
#pragma unroll
        for (int c = 0; c < K::RBT; ++c)
            accc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi, by[c], accc[c], 0, 0, 0);
#pragma unroll
        for (int c = 0; c < NG; ++c)
            accg[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo, bx[R + c - RMIN], accg[c], 0, 0, 0);
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

// The whole token loop of one wave whose row blocks are R1 (and R2 >= 0 when
// the wave owns two).  All waves run the same loads, stores and barriers.
template <int DS, int DT, int R1, int R2>
__device__ __forceinline__ void stats_wave(const StatsArgs &a, const StatsCtx &c, char *lds, int tid,
                                           int slot) {
    using K = Cfg<DS, DT>;
    constexpr int RMIN = (R2 >= 0 && R2 < R1) ? R2 : R1;
    constexpr int NBX = K::RB - RMIN;
    const int lane = tid & 63;
    const bool active = slot < c.n_slots;
    RowBlock<DS, DT, R1> blk1;
    RowBlock<DS, DT, (R2 >= 0 ? R2 : R1)> blk2;
    blk1.zero();
    if (R2 >= 0) blk2.zero();

    const int xoff = (slot == 0 || c.shared_x) ? K::OX0 : K::OX1;
    const int yoff = slot == 0 ? K::OY0 : K::OY1;
    const int woff = slot == 0 ? K::OW0 : K::OW1;
    const uint32_t lrow = lane & 31, lhalf = lane >> 5;

    Loader<DS, DT> ld;
    if (c.n_tiles > 0) {
        ld.load(a, c, tid, 0);
        ld.store(c, tid, lds);
        if (c.n_tiles > 1) ld.load(a, c, tid, 1);
        __syncthreads();
        for (int tile = 0; tile < c.n_tiles; ++tile) {
            if (active) {
                const char *B = lds + (tile & 1) * K::BUF;
#pragma unroll 1
                for (int ks = 0; ks < K::KT / 16; ++ks) {
                    const uint32_t kb = 2 * ks + lhalf;
                    bf16x8_t bx[NBX], by[K::RBT];
#pragma unroll
                    for (int cc = 0; cc < NBX; ++cc)
                        bx[cc] = *reinterpret_cast<const bf16x8_t *>(B + xoff + tile_off((RMIN + cc) * 32 + lrow, kb));
#pragma unroll
                    for (int cc = 0; cc < K::RBT; ++cc)
                        by[cc] = *reinterpret_cast<const bf16x8_t *>(B + yoff + tile_off(cc * 32 + lrow, kb));
                    const float4 w0 = *reinterpret_cast<const float4 *>(B + woff + kb * 32);
                    const float4 w1 = *reinterpret_cast<const float4 *>(B + woff + kb * 32 + 16);
                    const float w[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
                    blk1.template step<RMIN>(bx, by, w);
                    if (R2 >= 0) blk2.template step<RMIN>(bx, by, w);
                }
            }
            if (tile + 1 < c.n_tiles) {
                ld.store(c, tid, lds + ((tile + 1) & 1) * K::BUF);
                if (tile + 2 < c.n_tiles) ld.load(a, c, tid, tile + 2);
            }
            __syncthreads();
        }
    }
    if (active) {
        float *P = a.partials + ((int64_t)c.unit * 2 + slot) * K::SLOT;
        blk1.flush(P, lane);
        if (R2 >= 0) blk2.flush(P, lane);
    }
}

template <int DS, int DT>
__global__ __attribute__((amdgpu_flat_work_group_size(Cfg<DS, DT>::NT, Cfg<DS, DT>::NT),
                          amdgpu_waves_per_eu(1, 1)))
void stats_kernel(StatsArgs a) {
    using K = Cfg<DS, DT>;
    __shared__ __attribute__((aligned(16))) char lds[2 * K::BUF];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    StatsCtx c;
    c.unit = blockIdx.x;
    const int item_id = c.unit % a.n_items;
    const int chunk = c.unit / a.n_items;
    const StatsItem it = a.items[item_id];
    c.n_slots = it.n_slots;
    c.shared_x = it.shared_x != 0;
    const bool has_x1 = (c.n_slots == 2) && !c.shared_x;
    c.tok_begin = chunk * a.chunk_tokens;
    c.tok_end = min(a.N, c.tok_begin + a.chunk_tokens);
    c.n_tiles = c.tok_end > c.tok_begin ? (c.tok_end - c.tok_begin + K::KT - 1) / K::KT : 0;
    c.nj2 = has_x1 ? K::JX : 0;
    c.total_jobs = K::JX + K::JY + c.nj2 + (c.n_slots == 2 ? K::JY : 0);
    c.tp[0] = a.src + it.src_layer[0] * a.ss.layer + it.kv[0] * a.ss.kv + it.src_head[0] * a.ss.head;
    c.tp[1] = a.tgt + it.tgt_layer[0] * a.ts.layer + it.kv[0] * a.ts.kv + it.tgt_head[0] * a.ts.head;
    c.tp[2] = a.src + it.src_layer[1] * a.ss.layer + it.kv[1] * a.ss.kv + it.src_head[1] * a.ss.head;
    c.tp[3] = a.tgt + it.tgt_layer[1] * a.ts.layer + it.kv[1] * a.ts.kv + it.tgt_head[1] * a.ts.head;
    c.wrow[0] = a.w + (int64_t)it.wrow[0] * a.w_row_stride;
    c.wrow[1] = a.w + (int64_t)it.wrow[1] * a.w_row_stride;

    using WS = WaveShape<DS>;
    const int slot = wave >> 1;
    if ((wave & 1) == 0) stats_wave<DS, DT, WS::A1, WS::A2>(a, c, lds, tid, slot);
    else stats_wave<DS, DT, WS::B1, WS::B2>(a, c, lds, tid, slot);
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

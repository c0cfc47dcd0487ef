// cb_apply.hip -- online application of the fitted maps (gfx950).
//
// CacheBridge Sec. 1 (online handoff) and Sec. 2.3 (Eq. support-cost): at each
// handoff the deployed affine maps turn the sender's cache into a
// decode-ready target cache, at a cost linear in the prefix length and the
// coefficient count.  Per map m and token t:
//     out[t, :] = RNE_bf16( x_t W_m + b_m )
//
// split_maps_kernel: W (fp32) -> W^T as two bf16 planes, hi = RNE(W) and
//   lo = RNE(W - hi), plus the fp32 bias.  The pair carries ~16 significant
//   bits, so the bf16 MFMA products match an fp32 product to ~2^-17.
// apply_kernel: one workgroup per (source block, token tile).  A copy wave
//   streams the tile's source rows HBM -> LDS in 32-token sub-blocks through
//   a ring of direct-to-LDS copies; wave (slot, rb) keeps its 32 rows of
//   W_hi^T / W_lo^T for its map in registers and computes the 32x32 output
//   tile D = W^T x^T with v_mfma_f32_32x32x16_bf16 (K = source channels),
//   adds the bias and rounds once to bf16; the tile goes through an LDS
//   staging buffer and leaves as whole target rows.  A source block shared by
//   two target maps is read once.
//
// With the sender's rotary transform removed on the way in (Sec. 2.1, Sec.
// 3.1: the maps act on content coordinates), the computing waves turn
// sub-block sb + 1 back in LDS (one chunk pair per lane, in fp32, one
// rounding to bf16) in the iteration of sub-block sb; the next barrier
// publishes it, so the copy wave waits for one more sub-block before each
// barrier.
//
// Angles of the rotations.  A table covers tens of thousands of positions
// (16 MiB at 32,768 x 128), far more than L2, and per-lane reads of each
// token's row would move twice the bytes of the K rows themselves (the two
// maps of a shared source read the same entries).  Both rotations therefore
// form the (cos, sin) of position P = Q + r, Q = P - P mod 32, from the table
// rows of Q and of r by the angle-addition formulas in fp32.  The copy wave
// puts rows 0..31 of each table in LDS once per workgroup and, with every
// sub-block, the one or two rows Q its 32 positions need; the lanes read
// both from LDS.  Only a sub-block whose tokens cross into the next sequence
// reads its rows from global memory.  Those angles carry about 1.5 fp32 ulp
// more error than the table's, which moves a rotated bf16 value by one ulp
// only where it lies within that distance of a rounding boundary.
//
// With the target's rotary transform fused (Sec. 2.1, Sec. 3.1: the mapped
// keys receive the target's RoPE), the K outputs are turned in fp32 before
// the single rounding.  Style (2i, 2i+1) pairs sit in accumulator registers
// v and v+1 of one lane.  For the half split (i, i + d/2) a wave's 32 MFMA
// rows are channel groups rb*16 .. rb*16+15 and d/2 + rb*16 .. +15 instead of
// one 32-channel block, which puts each pair in registers v and v+8 of one
// lane; the stores then write those two 16-channel groups.
#include "cb_internal.h"

namespace cb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// Workgroup barrier for LDS double buffering: waits for this wave's LDS
// operations only (lgkmcnt), not for global loads still in flight, then
// s_barrier.  (A plain __syncthreads() also drains every outstanding global
// load, which would expose the full HBM latency once per tile.)
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // vmcnt = max, expcnt = max, lgkmcnt = 0
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ __forceinline__ uint32_t fastdiv(uint32_t n, const FastDiv &f) {
    const uint32_t t = __umulhi(n, f.m);
    return (t + ((n - t) >> f.sh1)) >> f.sh2;
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    f32x2_t v = {lo, hi};
    bf16x2_t p = __builtin_convertvector(v, bf16x2_t);
    return __builtin_bit_cast(uint32_t, p);
}

__global__ __launch_bounds__(256) void split_maps_kernel(int n_maps, int d_s, int d_t,
                                                         const float *__restrict__ maps,
                                                         uint16_t *__restrict__ w_hi,
                                                         uint16_t *__restrict__ w_lo,
                                                         float *__restrict__ bias) {
    const int P = d_s + 1;
    const int64_t n = (int64_t)n_maps * d_t * d_s;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
        const int k = (int)(e % d_s);
        const int64_t mj = e / d_s;
        const int j = (int)(mj % d_t);
        const int64_t m = mj / d_t;
        const float w = maps[(m * P + k) * d_t + j];
        const uint32_t p = pack_bf16(w, 0.f);
        const float hi = __uint_as_float(p << 16);
        const uint32_t q = pack_bf16(w - hi, 0.f);
        w_hi[e] = (uint16_t)(p & 0xffffu);
        w_lo[e] = (uint16_t)(q & 0xffffu);
        if (k == 0) bias[m * d_t + j] = maps[(m * P + d_s) * d_t + j];
    }
}

template <int DS, int DT, int SR = 0>
struct ACfg {
    static constexpr int KS = DS / 16;              // MFMA K steps over source channels
    static constexpr int RBT = DT / 32;             // 32-row blocks of target channels
    static constexpr int NWC = 2 * RBT;             // computing waves: (slot, rb)
    static constexpr int NW = NWC + 1;              // plus one copy wave
    static constexpr int NT = 64 * NW;
    static constexpr int SB = 32;                   // tokens per sub-block
    static constexpr int NCB = DS / 8;              // 16-byte blocks per source row
    static constexpr int ROWB = DS * 2;             // bytes per source row
    static constexpr int BUFB = SB * ROWB;          // bytes per ring stage
    static constexpr int COPIES = BUFB / 1024;      // copy instructions per stage (64 lanes x 16 B)
    static constexpr int STB = BUFB;                // bytes per ring stage
    static constexpr int NST = 8;                   // ring stages
    static_assert(BUFB % 1024 == 0, "a stage is a whole number of copy instructions");
    static_assert(SR == 0 || DS == 64 || DS == 128, "the source de-rotation takes d_s = 64 or 128");
};

// Lanes l and l ^ 32 trade halves so that each lane owns 8 consecutive channels of its 32-channel
// block (lanes < 32: channels 0-7 and 16-23, lanes >= 32: 8-15 and 24-31).  pk holds the lane's packed
// pairs, its channels 8 g + 4 (lane / 32) + {0 .. 3} in pk[2 g], pk[2 g + 1].  v_permlane32_swap trades
// the upper 32 lanes of its first operand with the lower 32 lanes of its second.
__device__ __forceinline__ void exchange32(const uint32_t (&pk)[8], uint4 (&o)[2]) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const auto x = __builtin_amdgcn_permlane32_swap(pk[4 * p + 0], pk[4 * p + 2], false, false);
        const auto y = __builtin_amdgcn_permlane32_swap(pk[4 * p + 1], pk[4 * p + 3], false, false);
        o[p] = make_uint4(x[0], y[0], x[1], y[1]);
    }
}

// Rotated position of 16-byte block cb of token row t in LDS: 16 consecutive
// tokens reading the same block hit distinct banks (when NCB = 16).
template <int NCB>
__device__ __forceinline__ uint32_t xoff(uint32_t t, uint32_t cb) {
    return t * (NCB * 16) + ((cb + t) % NCB) * 16;
}

// HBM -> LDS copy of 16 bytes per lane to M0 + 16 lane (direct-to-LDS load).
// M0 is saved and restored inside the statement.
__device__ __forceinline__ void dma16(const void *gaddr, uint32_t m0) {
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "v"(gaddr), "s"(m0)
                 : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Rotary style of the fused epilogue: none, pairs (i, i + d/2), pairs (2i, 2i+1).
enum { kRopeNone = 0, kRopeHalf = 1, kRopeInterleaved = 2 };

// Target channel of MFMA row i (0..31) of wave rb.
template <int DT, int RS>
__device__ __forceinline__ int out_channel(int rb, int i) {
    if (RS == kRopeHalf) return i < 16 ? rb * 16 + i : DT / 2 + rb * 16 + (i - 16);
    return rb * 32 + i;
}

// (cos, sin) of position P for frequencies f and f + 1 (float offset 2 f of a
// table row), from the rows of Q = P - P mod 32 and r = P mod 32:
// cos(Q + r) = cos Q cos r - sin Q sin r, sin(Q + r) = sin Q cos r + cos Q sin r,
// in fp32.  Returns (cos f, sin f, cos f+1, sin f+1) like a table read.
__device__ __forceinline__ float4 add_angles(const float4 q, const float4 r) {
    float4 o;
    o.x = __builtin_fmaf(q.x, r.x, -(q.y * r.y));
    o.y = __builtin_fmaf(q.y, r.x, q.x * r.y);
    o.z = __builtin_fmaf(q.z, r.z, -(q.w * r.w));
    o.w = __builtin_fmaf(q.w, r.z, q.z * r.w);
    return o;
}
__device__ __forceinline__ float4 angles2(const float *table, int row_floats, int P, int f) {
    const float4 q = *reinterpret_cast<const float4 *>(table + (int64_t)(P & ~31) * row_floats + 2 * f);
    const float4 r = *reinterpret_cast<const float4 *>(table + (int64_t)(P & 31) * row_floats + 2 * f);
    return add_angles(q, r);
}

// Position run of a 32-token sub-block: the in-sequence position tt0 of its
// first token and whether its stored tokens stay in that sequence (then
// token j sits at tt0 + j).  `last` is the offset of its last stored token.
struct SubRun {
    int tt0;
    int last;
    bool simple;
};

// One workgroup per (group, token tile).  The copy wave streams 32-token
// sub-blocks of the group's source rows HBM -> LDS through an NST-stage ring
// (NST - 1 sub-blocks ahead); since it issues nothing but these copies, its
// vmcnt waits are exact.  One barrier per sub-block publishes the landed
// stage to the computing waves and tells the copy wave that the stage read
// one sub-block earlier is free again.
template <int DS, int DT, int RS, int SR>
__global__ __attribute__((amdgpu_flat_work_group_size(ACfg<DS, DT>::NT, ACfg<DS, DT>::NT))) void apply_kernel(ApplyArgs a) {
    using K = ACfg<DS, DT, SR>;
    __shared__ __attribute__((aligned(16))) char lds[K::NST * K::STB];
    // Without the rotation the outputs go through an LDS staging buffer and
    // leave as whole target rows (16 lanes per row): about 4% faster than
    // each wave storing its 32-channel slices.  With it, the direct stores
    // are faster (the staging costs more than it saves there).
    constexpr bool STAGE = RS == kRopeNone;
    // [buffer][slot][32 tokens][DT bf16], 16-byte chunk c of token j at (c + j) mod NCBT
    constexpr int NCBT = DT / 8;
    constexpr int OBUF = K::SB * DT * 2;
    __shared__ __attribute__((aligned(16))) char obuf[STAGE ? 2 * 2 * OBUF : 16];
    // Rotation angles in LDS (a sub-block whose tokens stay in one sequence):
    // per stage, table rows Q0 and Q0 + 32 of the sub-block's positions
    // (Q0 = first position rounded down to a multiple of 32), one 1 KiB slot
    // per table; per workgroup, table rows 0..31, 16-byte chunk c of row r at
    // chunk (c + r) mod (chunks per row).  Position P's angles are those of
    // Q + (P mod 32) by angle addition, as in the de-rotation below.  Slot 0
    // is the target's table (RS), the last slot the sender's (SR).
    constexpr int NQ = (RS != kRopeNone ? 1 : 0) + (SR != 0 ? 1 : 0);
    constexpr int QSLOT = 1024;
    constexpr int NCHT = DT / 4, NCHS = DS / 4;           // 16-byte chunks per table row
    constexpr int RROWT = RS != kRopeNone ? 32 * DT * 4 : 0;
    constexpr int RROWS = SR != 0 ? 32 * DS * 4 : 0;
    __shared__ __attribute__((aligned(16))) char qbuf[NQ ? K::NST * NQ * QSLOT : 16];
    __shared__ __attribute__((aligned(16))) char rrows[RROWT + RROWS ? RROWT + RROWS : 16];
    constexpr int PER = K::COPIES + NQ;                   // copy instructions per stage

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = blockIdx.x / a.n_tiles;
    const int tile = blockIdx.x % a.n_tiles;
    const ApplyGroup *grp = a.groups + g;                     // read field by field (uniform)
    const int tok0 = tile * a.tile_tokens;
    const int tok1 = min(a.N, tok0 + a.tile_tokens);
    const int n_sb = (tok1 - tok0 + K::SB - 1) / K::SB;
    if (n_sb <= 0) return;
    const int kv = grp->kv;
    const uint16_t *xsrc = a.src + grp->src_layer * a.ss.layer + kv * a.ss.kv + grp->src_head * a.ss.head;

    const bool turn_src = SR != 0 && kv == 0;                 // only keys carry positions
    auto sub_run = [&](int sb) __attribute__((always_inline)) {
        const int tau0 = min(tok0 + sb * K::SB, tok1 - 1);
        const uint32_t b0 = fastdiv((uint32_t)tau0, a.T);
        SubRun u;
        u.tt0 = (int)((uint32_t)tau0 - b0 * a.T.d);
        u.last = min(tau0 + K::SB - 1, tok1 - 1) - tau0;
        u.simple = u.tt0 + u.last < (int)a.T.d;
        return u;
    };
    if (wave == K::NWC) {
        // ---- copy wave: copy i of a stage moves LDS chunks 64 i + lane
        const uint32_t lds_base = (uint32_t)(uintptr_t)lds;
        const uint32_t lds_q = (uint32_t)(uintptr_t)qbuf, lds_r = (uint32_t)(uintptr_t)rrows;
        auto issue = [&](int sb, int st) {
#pragma unroll
            for (int i = 0; i < K::COPIES; ++i) {
                const int q = 64 * i + lane;
                const int t = q / K::NCB, p = q - (q / K::NCB) * K::NCB;
                const int cb = (p + K::NCB - t % K::NCB) % K::NCB;     // inverse of the rotation
                const int tau = min(tok0 + sb * K::SB + t, tok1 - 1);  // past the tile: any valid row
                const uint32_t b = fastdiv((uint32_t)tau, a.T);
                const uint32_t tt = (uint32_t)tau - b * a.T.d;
                const uint16_t *src = xsrc + (int64_t)b * a.ss.seq + (int64_t)tt * a.ss.tok + cb * 8;
                dma16(src, __builtin_amdgcn_readfirstlane(lds_base + st * K::STB + i * 1024));
            }
            if constexpr (NQ != 0) {
                // rows Q0 and Q0 + 32 of each table (Q0 alone when the run ends
                // below Q0 + 32, or when its tokens leave the sequence: then the
                // rows are not used and any valid row will do)
                const SubRun u = sub_run(sb);
                auto qrows = [&](const float *tab, int nch, int off, int qs) __attribute__((always_inline)) {
                    const int p0 = off + u.tt0, q0 = p0 & ~31;
                    const int q1 = (u.simple && q0 + 32 <= p0 + u.last) ? q0 + 32 : q0;
                    const int row = min(lane / nch, 1), ch = min(lane - row * nch, nch - 1);
                    const float *src = tab + (int64_t)(row ? q1 : q0) * (4 * nch) + 4 * ch;
                    dma16(src, __builtin_amdgcn_readfirstlane(lds_q + (st * NQ + qs) * QSLOT));
                };
                if constexpr (RS != kRopeNone) qrows(a.rope_table, NCHT, a.rope_pos_offset, 0);
                if constexpr (SR != 0) qrows(a.src_rope_table, NCHS, a.src_rope_pos_offset, NQ - 1);
            }
        };
        // rows 0..31 of each table (rows past the last position any call
        // reads are clamped to it: they are never used)
        auto rrows_copy = [&](const float *tab, int nch, int off, uint32_t dst) __attribute__((always_inline)) {
            const int maxpos = off + (int)a.T.d - 1;
            for (int i = 0; i < nch / 2; ++i) {
                const int q = 64 * i + lane;
                const int r = q / nch, pch = q - r * nch;
                const int c = (pch - r % nch + nch) % nch;
                dma16(tab + (int64_t)min(r, maxpos) * (4 * nch) + 4 * c, __builtin_amdgcn_readfirstlane(dst + i * 1024));
            }
        };
        if constexpr (RS != kRopeNone) rrows_copy(a.rope_table, NCHT, a.rope_pos_offset, lds_r);
        if constexpr (SR != 0) rrows_copy(a.src_rope_table, NCHS, a.src_rope_pos_offset, lds_r + RROWT);
#pragma unroll
        for (int s = 0; s < K::NST - 1; ++s) issue(s, s);
        if constexpr (SR != 0) {
            wait_vm<(K::NST - 3) * PER>();                     // sub-blocks 0 and 1 have landed
            lds_barrier();
        }
        for (int sb = 0; sb < n_sb; ++sb) {
            // sub-block sb has landed (and, with the de-rotation, sb + 1, which is turned during sb)
            wait_vm<(K::NST - 2 - (SR != 0 ? 1 : 0)) * PER>();
            lds_barrier();
            issue(sb + K::NST - 1, (sb + K::NST - 1) % K::NST);
        }
        if (STAGE) lds_barrier();                              // the computing waves' last store round
        wait_vm<0>();                                          // drain before the LDS is released
        return;
    }

    // ---- computing wave (slot, rb)
    const int slot = wave / K::RBT, rb = wave % K::RBT;
    const bool active = slot < grp->n_slots;
    const int sl = active ? slot : 0;
    const int m = grp->map[sl];
    uint16_t *obase = a.out + grp->tgt_layer[sl] * a.os.layer + kv * a.os.kv + grp->tgt_head[sl] * a.os.head;
    const bool rotate = RS != kRopeNone && kv == 0;            // only keys carry positions

    // coefficients of this wave's 32 target channels, kept in registers
    const uint32_t lrow = lane & 31, lhalf = lane >> 5;
    bf16x8_t ahi[K::KS], alo[K::KS];
    float bias[16];
    {
        const int ch = out_channel<DT, RS>(rb, (int)lrow);
        const uint16_t *wh = a.w_hi + ((int64_t)m * DT + ch) * DS + 8 * lhalf;
        const uint16_t *wl = a.w_lo + ((int64_t)m * DT + ch) * DS + 8 * lhalf;
#pragma unroll
        for (int ks = 0; ks < K::KS; ++ks) {
            ahi[ks] = *reinterpret_cast<const bf16x8_t *>(wh + 16 * ks);
            alo[ks] = *reinterpret_cast<const bf16x8_t *>(wl + 16 * ks);
        }
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            // rows 8 gq + 4 lhalf .. + 3: four consecutive channels
            const float *bp = a.bias + (int64_t)m * DT + out_channel<DT, RS>(rb, 8 * gq + 4 * (int)lhalf);
            const float4 b4 = *reinterpret_cast<const float4 *>(bp);
            bias[4 * gq + 0] = b4.x;
            bias[4 * gq + 1] = b4.y;
            bias[4 * gq + 2] = b4.z;
            bias[4 * gq + 3] = b4.w;
        }
    }
    // channel offsets of the lane's two 16-byte output chunks (after the
    // exchange below: MFMA rows 8 lhalf .. +7 and 16 + 8 lhalf .. +7)
    const int oc0 = out_channel<DT, RS>(rb, 8 * (int)lhalf), oc1 = out_channel<DT, RS>(rb, 16 + 8 * (int)lhalf);

    // ---- de-rotation of a landed sub-block (SR != 0): pair u = 64 wave + lane
    // of its rows, token row t = u / (NCB/2), logical chunks c and c + NCB/2
    constexpr int HP = K::NCB / 2;
    const int tu = (64 * wave + lane) / HP, cu = (64 * wave + lane) % HP;
    const bool ulive = SR != 0 && 64 * wave + lane < K::SB * HP;
    // the lane's (cos, sin) entries for sub-block sb: half split, frequencies
    // 8c .. 8c + 7; interleaved, 4c .. 4c + 3 and 4(c + NCB/2) .. + 3
    auto tab_load = [&](float4 (&cs)[4], int sb) __attribute__((always_inline)) {
        if constexpr (SR != 0) {
            const SubRun u = sub_run(sb);
            if (u.simple) {
                // rows Q0 / Q0 + 32 of the stage and rows 0..31 of the workgroup, in LDS
                const int P = a.src_rope_pos_offset + u.tt0 + (ulive ? tu : 0);   // idle lanes: any row
                const int qi = (P >> 5) - ((a.src_rope_pos_offset + u.tt0) >> 5), r = P & 31;
                const char *Q = qbuf + ((sb % K::NST) * NQ + NQ - 1) * QSLOT + qi * (NCHS * 16);
                const char *R = rrows + RROWT + r * (NCHS * 16);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int ch = SR == 1 ? 4 * cu + j : 2 * (j < 2 ? cu : cu + HP) + (j & 1);   // frequency / 2
                    const float4 q = *reinterpret_cast<const float4 *>(Q + ch * 16);
                    const float4 rr = *reinterpret_cast<const float4 *>(R + ((ch + r) % NCHS) * 16);
                    cs[j] = add_angles(q, rr);
                }
                return;
            }
            const int tau = min(tok0 + sb * K::SB + tu, tok1 - 1);
            const uint32_t tt = (uint32_t)tau - fastdiv((uint32_t)tau, a.T) * a.T.d;
            const int P = a.src_rope_pos_offset + (int)tt;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int f = SR == 1 ? 8 * cu + 2 * j : 4 * (j < 2 ? cu : cu + HP) + 2 * (j & 1);
                cs[j] = angles2(a.src_rope_table, DS, P, f);
            }
        }
    };
    auto turn_sub = [&](int sb, const float4 (&cs)[4]) __attribute__((always_inline)) {
        if constexpr (SR != 0) {
            if (!ulive) return;
            const int t = tu, c = cu;
            char *B = lds + (sb % K::NST) * K::STB;
            char *pa = B + t * (K::NCB * 16) + ((c + t) % K::NCB) * 16;
            char *pb = B + t * (K::NCB * 16) + ((c + HP + t) % K::NCB) * 16;
            const uint4 A = *reinterpret_cast<const uint4 *>(pa);
            const uint4 Bv = *reinterpret_cast<const uint4 *>(pb);
            const uint32_t av[4] = {A.x, A.y, A.z, A.w}, bv[4] = {Bv.x, Bv.y, Bv.z, Bv.w};
            uint32_t oa[4], ob[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float x0 = __uint_as_float(av[e] << 16), x1 = __uint_as_float(av[e] & 0xffff0000u);
                const float y0 = __uint_as_float(bv[e] << 16), y1 = __uint_as_float(bv[e] & 0xffff0000u);
                if constexpr (SR == 1) {
                    // pairs (8c + 2e + h, d/2 further on), frequency 8c + 2e + h: the inverse turn
                    const float c0 = cs[e].x, s0 = cs[e].y, c1 = cs[e].z, s1 = cs[e].w;
                    oa[e] = pack_bf16(__builtin_fmaf(x0, c0, y0 * s0), __builtin_fmaf(x1, c1, y1 * s1));
                    ob[e] = pack_bf16(__builtin_fmaf(y0, c0, -(x0 * s0)), __builtin_fmaf(y1, c1, -(x1 * s1)));
                } else {
                    // pairs (2i, 2i + 1) inside each chunk: frequencies 4c + e and 4(c + NCB/2) + e
                    const float4 qa = cs[e >> 1], qb = cs[2 + (e >> 1)];
                    const float ca = (e & 1) ? qa.z : qa.x, sa = (e & 1) ? qa.w : qa.y;
                    const float cb2 = (e & 1) ? qb.z : qb.x, sb2 = (e & 1) ? qb.w : qb.y;
                    oa[e] = pack_bf16(__builtin_fmaf(x0, ca, x1 * sa), __builtin_fmaf(x1, ca, -(x0 * sa)));
                    ob[e] = pack_bf16(__builtin_fmaf(y0, cb2, y1 * sb2), __builtin_fmaf(y1, cb2, -(y0 * sb2)));
                }
            }
            *reinterpret_cast<uint4 *>(pa) = make_uint4(oa[0], oa[1], oa[2], oa[3]);
            *reinterpret_cast<uint4 *>(pb) = make_uint4(ob[0], ob[1], ob[2], ob[3]);
        }
    };
    if constexpr (SR != 0) {
        lds_barrier();                                         // sub-blocks 0 and 1 have landed
        if (turn_src) {
            float4 cs[4];
            tab_load(cs, 0);
            turn_sub(0, cs);
        }
    }
    // target rotation: (cos, sin) of the lane's eight rotated pairs in a sub-block
    auto tcs_load = [&](float4 (&cs)[4], int sb) __attribute__((always_inline)) {
        if constexpr (RS != kRopeNone) {
            const SubRun u = sub_run(sb);
            if (u.simple) {
                const int P = a.rope_pos_offset + u.tt0 + (int)lrow;
                const int qi = (P >> 5) - ((a.rope_pos_offset + u.tt0) >> 5), r = P & 31;
                const char *Q = qbuf + (sb % K::NST) * NQ * QSLOT + qi * (NCHT * 16);
                const char *R = rrows + r * (NCHT * 16);
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    // chunk = frequency / 2 (as in the table reads below)
                    const int ch = RS == kRopeHalf ? rb * 8 + 4 * (gq >> 1) + 2 * (int)lhalf + (gq & 1)
                                                   : rb * 8 + 2 * gq + (int)lhalf;
                    const float4 q = *reinterpret_cast<const float4 *>(Q + ch * 16);
                    const float4 rr = *reinterpret_cast<const float4 *>(R + ((ch + r) % NCHT) * 16);
                    cs[gq] = add_angles(q, rr);
                }
                return;
            }
            const int tau = min(tok0 + sb * K::SB + (int)lrow, tok1 - 1);
            const uint32_t tt = (uint32_t)tau - fastdiv((uint32_t)tau, a.T) * a.T.d;
            const float *row = a.rope_table + (int64_t)(a.rope_pos_offset + (int)tt) * DT;   // [d/2][2] per position
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                // half split: frequencies rb*16 + 8 (gq/2) + 4 lhalf + 2 (gq%2) + {0, 1}
                // interleaved: frequencies rb*16 + 4 gq + 2 lhalf + {0, 1}
                const int f = RS == kRopeHalf ? rb * 16 + 8 * (gq >> 1) + 4 * (int)lhalf + 2 * (gq & 1)
                                              : rb * 16 + 4 * gq + 2 * (int)lhalf;
                cs[gq] = *reinterpret_cast<const float4 *>(row + 2 * f);
            }
        }
    };

    // With staging, iteration sb stores the rows of sub-block sb - 1 (written to
    // the staging buffer before the barrier), and one more iteration follows.
    for (int sb = 0; sb < n_sb + (STAGE ? 1 : 0); ++sb) {
        lds_barrier();                                         // sub-block sb has landed (and is turned)
        const bool turn_next = SR != 0 && turn_src && sb + 1 < n_sb;
        if (STAGE && active && sb > 0) {
            // 4 DT chunks of 16 bytes: two rounds of the slot's RBT waves
            const char *ob = obuf + (((sb - 1) & 1) * 2 + slot) * OBUF;
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const int q = (r * K::RBT + rb) * 64 + lane;
                const int j = q / NCBT, c = q - (q / NCBT) * NCBT;
                const int tj = tok0 + (sb - 1) * K::SB + j;
                const uint4 val = *reinterpret_cast<const uint4 *>(ob + j * (DT * 2) + ((c + j) % NCBT) * 16);
                if (tj < tok1) {
                    const uint32_t bj = fastdiv((uint32_t)tj, a.T);
                    const uint32_t tq = (uint32_t)tj - bj * a.T.d;
                    *reinterpret_cast<uint4 *>(obase + (int64_t)bj * a.os.seq + (int64_t)tq * a.os.tok + c * 8) = val;
                }
            }
        }
        if (turn_next) {
            // the angles come from LDS (global reads only for a run that leaves its sequence)
            float4 scs[4];
            tab_load(scs, sb + 1);
            turn_sub(sb + 1, scs);
        }
        if (STAGE && sb == n_sb) break;
        if (!active) continue;
        const char *B = lds + (sb % K::NST) * K::STB;
        const int tau = tok0 + sb * K::SB + (int)lrow;
        const uint32_t bseq = fastdiv((uint32_t)min(tau, tok1 - 1), a.T);
        const uint32_t tt = (uint32_t)min(tau, tok1 - 1) - bseq * a.T.d;
        // this sub-block's rotation entries, requested before the products
        float4 cs[4];
        if (RS != kRopeNone && rotate) tcs_load(cs, sb);
        // hi and lo terms in two accumulators: two independent MFMA chains
        f32x16_t acc, acl;
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = acl[v] = 0.f;
#pragma unroll
        for (int ks = 0; ks < K::KS; ++ks) {
            const bf16x8_t bx = *reinterpret_cast<const bf16x8_t *>(B + xoff<K::NCB>(lrow, 2 * ks + lhalf));
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi[ks], bx, acc, 0, 0, 0);
            acl = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo[ks], bx, acl, 0, 0, 0);
        }
        // D[i][t]: t = lane & 31, i = 8*(v/4) + 4*(lane/32) + (v&3)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = acc[v] + acl[v] + bias[v];
        if (RS == kRopeHalf && rotate) {
            // pair (v, v + 8): channels c and c + d/2, frequency c
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                const float4 q = cs[2 * (v >> 2) + ((v & 3) >> 1)];
                const float c = (v & 1) ? q.z : q.x, sn = (v & 1) ? q.w : q.y;
                const float x0 = acc[v], x1 = acc[v + 8];
                acc[v] = __builtin_fmaf(x0, c, -x1 * sn);
                acc[v + 8] = __builtin_fmaf(x1, c, x0 * sn);
            }
        } else if (RS == kRopeInterleaved && rotate) {
            // pair (v, v + 1), v even: channels 2f and 2f + 1
#pragma unroll
            for (int v = 0; v < 16; v += 2) {
                const float4 q = cs[v >> 2];
                const float c = (v & 2) ? q.z : q.x, sn = (v & 2) ? q.w : q.y;
                const float x0 = acc[v], x1 = acc[v + 1];
                acc[v] = __builtin_fmaf(x0, c, -x1 * sn);
                acc[v + 1] = __builtin_fmaf(x1, c, x0 * sn);
            }
        }
        uint32_t pk[8];
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            pk[2 * gq] = pack_bf16(acc[4 * gq + 0], acc[4 * gq + 1]);
            pk[2 * gq + 1] = pack_bf16(acc[4 * gq + 2], acc[4 * gq + 3]);
        }
        uint4 o[2];
        exchange32(pk, o);
        if (STAGE) {
            char *ob = obuf + ((sb & 1) * 2 + slot) * OBUF + lrow * (DT * 2);
            *reinterpret_cast<uint4 *>(ob + ((oc0 / 8 + (int)lrow) % NCBT) * 16) = o[0];
            *reinterpret_cast<uint4 *>(ob + ((oc1 / 8 + (int)lrow) % NCBT) * 16) = o[1];
        } else if (tau < tok1) {
            uint16_t *orow = obase + (int64_t)bseq * a.os.seq + (int64_t)tt * a.os.tok;
            *reinterpret_cast<uint4 *>(orow + oc0) = o[0];
            *reinterpret_cast<uint4 *>(orow + oc1) = o[1];
        }
    }
}

template <int DS, int DT, int SR>
hipError_t launch_apply_sr(int64_t grid, const ApplyArgs &a, hipStream_t s) {
    using K = ACfg<DS, DT>;
    if (!a.rope_table)
        hipLaunchKernelGGL((apply_kernel<DS, DT, kRopeNone, SR>), dim3((unsigned)grid), dim3(K::NT), 0, s, a);
    else if (a.rope_style == 0)
        hipLaunchKernelGGL((apply_kernel<DS, DT, kRopeHalf, SR>), dim3((unsigned)grid), dim3(K::NT), 0, s, a);
    else
        hipLaunchKernelGGL((apply_kernel<DS, DT, kRopeInterleaved, SR>), dim3((unsigned)grid), dim3(K::NT), 0, s, a);
    return hipGetLastError();
}

template <int DS, int DT>
hipError_t launch_apply_t(int n_groups, const ApplyArgs &a, hipStream_t s) {
    const int64_t grid = (int64_t)n_groups * a.n_tiles;
    if (grid == 0) return hipSuccess;
    if (!a.src_rope_table) return launch_apply_sr<DS, DT, 0>(grid, a, s);
    if constexpr (DS == 64 || DS == 128) {
        if (a.src_rope_style == 0) return launch_apply_sr<DS, DT, 1>(grid, a, s);
        return launch_apply_sr<DS, DT, 2>(grid, a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_split_maps(int32_t n_maps, int32_t d_s, int32_t d_t, const float *maps, uint16_t *w_hi,
                             uint16_t *w_lo, float *bias, hipStream_t s) {
    const int64_t n = (int64_t)n_maps * d_t * d_s;
    if (n == 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(split_maps_kernel, dim3((unsigned)blocks), dim3(256), 0, s, n_maps, d_s, d_t, maps, w_hi,
                       w_lo, bias);
    return hipGetLastError();
}

#define CB_DISPATCH_APPLY(d_s, d_t, ...)                                     \
    switch ((d_s) * 1000 + (d_t)) {                                          \
        case 64064: return launch_apply_t<64, 64>(__VA_ARGS__);              \
        case 64096: return launch_apply_t<64, 96>(__VA_ARGS__);              \
        case 64128: return launch_apply_t<64, 128>(__VA_ARGS__);             \
        case 96064: return launch_apply_t<96, 64>(__VA_ARGS__);              \
        case 96096: return launch_apply_t<96, 96>(__VA_ARGS__);              \
        case 96128: return launch_apply_t<96, 128>(__VA_ARGS__);             \
        case 128064: return launch_apply_t<128, 64>(__VA_ARGS__);            \
        case 128096: return launch_apply_t<128, 96>(__VA_ARGS__);            \
        case 128128: return launch_apply_t<128, 128>(__VA_ARGS__);           \
        default: return hipErrorInvalidValue;                                \
    }

hipError_t launch_apply(int d_s, int d_t, int n_groups, const ApplyArgs &a, hipStream_t s) {
    CB_DISPATCH_APPLY(d_s, d_t, n_groups, a, s);
}

}  // namespace cb

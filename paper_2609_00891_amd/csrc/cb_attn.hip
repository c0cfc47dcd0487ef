// cb_attn.hip -- attention-aligned calibration weights on gfx950.
//
// CacheBridge Sec. 3.3 (Eq. attentionlinearization, Eq. sensitivity).  For
// every sequence, target layer l and KV head h, every causal prefix boundary
// c (the position of the first query after the prefix [0, c)) and every query
// head u sharing h,
//     a_i = softmax_i(q_u . k_i / sqrt(d))  over the keys i = 0 .. c,
//     o_u = sum_i a_i v_i,
// and for the sampled prefix positions E_c = {i < c : i mod stride = 0}
//     p^V_i = sum_u a_i^2,   p^K_i = sum_u a_i^2 |v_i - o_u|^2 |q_u|^2 / d.
// Each boundary's p^K and p^V are scaled to unit mass over E_c and the
// boundaries are summed: r^K, r^V.  attn_weights_kernel then normalizes every
// row to mean one over the calibration rows and shrinks it toward uniform
// weights with the largest alpha whose Kish effective sample size reaches
// tau = min(n, 2 p).
//
// attn_sens_kernel: one workgroup of eight waves per (sequence, layer, KV
// head) unit.  The rows are the queries of every boundary and query head
// (row = boundary * G + head), in row tiles of 32.  Row tile t attends the
// keys 0 .. c_hi(t); the lengths grow with t (boundaries are increasing), and
// for log-spaced boundaries the last tile holds half of all the work.  So the
// keys are streamed through LDS in stages of four 32-key tiles, and a long row
// tile is split by key over up to four waves (stage slot s of iteration it
// holds key tile it + s * n_it); short row tiles run first in a pass of their
// own (key tiles 4 it .. 4 it + 3).  The host picks the split (fewest
// lockstep steps).  Two sweeps over the keys:
//   A  S^T = K Q^T (v_mfma_f32_32x32x16_bf16, lane = query): the online
//      softmax maximum m and normalizer l, and with them o~ = sum p v and,
//      over the eligible keys, sum p^2, sum p^2 |v|^2 and sum p^2 v
//      (p = exp(s - m); a tile that raises m rescales the sums by
//      exp(m_old - m_new), the p^2 sums by its square).  p and p^2 enter the
//      matrix products as two bf16 terms each; V^T is read with
//      ds_read_b64_tr_b16 in the key order of the accumulator layout.  The
//      waves sharing a row tile then merge their partial sums (log-sum-exp)
//      through LDS, in wave order; the unit masses of each boundary follow
//      from the merged sums (the K mass, sum a^2 |v - o|^2 |q|^2 / d, expanded).
//   C  S = Q K^T and (o V^T), o as two bf16 terms (lane = key): every
//      eligible (query, key) term, summed over the wave's 32 queries in
//      registers; the waves' per-key sums are added in a fixed order.
// No atomics; results are bitwise reproducible.
#include <algorithm>
#include <cmath>
#include <vector>

#include "cb_stats_kernel.h"

namespace cb {
namespace {

constexpr int kWaves = 8, kThreads = 64 * kWaves, kKT = 32, kSlots = 4, kMaxRounds = 7;

__device__ __forceinline__ f32x16_t mfma(bf16x8_t a, bf16x8_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Eight fp32 values -> hi = RNE_bf16(v), lo = RNE_bf16(v - hi), as MFMA operands.
__device__ __forceinline__ void split8(const float *v, bf16x8_t &hi, bf16x8_t &lo) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        h[e] = pack_bf16(v[2 * e], v[2 * e + 1]);
        l[e] = pack_bf16(v[2 * e] - bf_lo(h[e]), v[2 * e + 1] - bf_hi(h[e]));
    }
    hi = __builtin_bit_cast(bf16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
    lo = __builtin_bit_cast(bf16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
}

// 16 bytes per lane HBM -> LDS at M0 + 16 lane (global_load_lds_dwordx4),
// tracked by vmcnt; M0 is saved and restored inside the statement.
__device__ __forceinline__ void copy16(uint32_t voff, const void *sbase, uint32_t m0) {
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\tglobal_load_lds_dwordx4 %1, %2\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "v"(voff), "s"(sbase), "s"(m0)
                 : "memory");
}

// Key index of accumulator register v in lane half hh of a 32x32 tile whose
// rows are keys: D[i][j] sits in lane j + 32 ((i >> 2) & 1), register
// 4 (i >> 3) + (i & 3).
__device__ __forceinline__ int acc_row(int v, int hh) { return 8 * (v >> 2) + 4 * hh + (v & 3); }

// Work split of one call (the same for every unit: it depends only on the
// boundaries).  Pass "pre": wave w takes row tile pre_tile[w] (-1: none) and
// every slot of stages holding key tiles 4 it .. 4 it + 3.  Pass "main": wave w
// takes row tile main_tile[w] and the slots in main_mask[w] of stages holding
// key tiles it + s * main_it.  Waves sharing a main row tile merge into
// leader[w] in merge rounds of at most three partial records.
struct AttnSched {
    int32_t pre_tile[kWaves];
    int32_t pre_it;
    int32_t main_tile[kWaves];
    int32_t main_mask[kWaves];
    int32_t main_it;
    int32_t leader[kWaves];
    int32_t n_rounds;
    int32_t round_w[kMaxRounds][3];
};

struct AttnArgs {
    const uint16_t *kv;              // target cache (K = kv 0, V = kv 1)
    Strides ts;
    const uint16_t *q;               // boundary queries
    int64_t q_layer, q_seq, q_bnd, q_head;
    int32_t n_layers, n_heads, G, n_bounds, n_rows, seq_len, stride;
    float scale_log2;                // log2(e) / sqrt(d)
    float *r;                        // [(l * 2 + z) * H + h][seq * seq_len + tok]
    int64_t r_row_stride;
    int32_t bounds[64];
    AttnSched s;
};

template <int D>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads), amdgpu_waves_per_eu(2, 2)))
void attn_sens_kernel(AttnArgs a) {
    constexpr int NCH = D / 8, NDT = D / 32, NKS = D / 16;   // 16-byte chunks per row, 32-d tiles, 16-d steps
    constexpr int SW = NCH < 16 ? NCH - 1 : 15;              // chunk swizzle mask
    constexpr int TB = kKT * D * 2;                          // bytes per K or V tile
    constexpr int SLOTB = 2 * TB;                            // a slot: K tile, then V tile
    constexpr int STAGE = kSlots * SLOTB;
    constexpr int IPT = TB / 1024;                           // copy instructions per tile (64 lanes x 16 B)
    constexpr int NCOPY = kSlots * 2 * IPT;                  // copy instructions per stage
    static_assert(NCOPY % kWaves == 0, "every wave issues the same number of copies");
    constexpr int RECF = 4 + 2 * NDT * 16;                   // floats per lane of a partial record
    static_assert(3 * RECF * 64 * 4 <= 2 * STAGE, "three partial records fit the stage buffers");
    static_assert(8 * NKS * 2 * 64 * 16 <= 2 * STAGE, "the final o of eight row tiles fits the stage buffers");
    __shared__ __attribute__((aligned(16))) char lds[2 * STAGE];
    __shared__ __attribute__((aligned(16))) float vvs[kSlots * kKT];         // |v|^2 of the stage's keys
    __shared__ float part[2][kWaves][kSlots][kKT][2];                        // per-key sums of each wave
    __shared__ __attribute__((aligned(16))) float4 ri0[8][32];  // per row: see finish_tile
    __shared__ float ri1[8][32];                                // per row: boundary c (-1: no row)

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int j = lane & 31, hh = lane >> 5;
    const int unit = blockIdx.x;
    const int h = unit % a.n_heads;
    const int l = (unit / a.n_heads) % a.n_layers;
    const int b = unit / (a.n_heads * a.n_layers);
    const uint16_t *Kg = a.kv + l * a.ts.layer + b * a.ts.seq + h * a.ts.head;
    const uint16_t *Vg = Kg + a.ts.kv;
    float *rK = a.r + ((int64_t)(l * 2 + 0) * a.n_heads + h) * a.r_row_stride + (int64_t)b * a.seq_len;
    float *rV = a.r + ((int64_t)(l * 2 + 1) * a.n_heads + h) * a.r_row_stride + (int64_t)b * a.seq_len;
    float *ldsf = (float *)lds;

    // largest boundary of a row tile, and its key tiles in sweep A (keys
    // 0 .. c_hi) and sweep C (keys 0 .. c_hi - 1)
    auto tile_chi = [&](int t) __attribute__((always_inline)) { return a.bounds[min(t * 32 + 31, a.n_rows - 1) / a.G]; };
    auto nt_a = [&](int t) __attribute__((always_inline)) { return t < 0 ? 0 : (tile_chi(t) + kKT) / kKT; };
    auto nt_c = [&](int t) __attribute__((always_inline)) { return t < 0 ? 0 : (tile_chi(t) + kKT - 1) / kKT; };

    // ---- per-wave row state
    bf16x8_t qf[NKS];             // Q[row j][16 s + 8 hh .. +7]: B operand of S^T = K Q^T, A operand of S = Q K^T
    float qq = 0.f;               // |q|^2 of this lane's row
    int c = -1;                   // boundary of this lane's row (-1: no row)
    auto load_q = [&](int t) __attribute__((always_inline)) {
        const int row = t * 32 + j;
        const bool ok = t >= 0 && row < a.n_rows;
        const int kb = ok ? row / a.G : 0;
        c = ok ? a.bounds[kb] : -1;
        const int u = h * a.G + (ok ? row % a.G : 0);
        const uint16_t *qr = a.q + l * a.q_layer + b * a.q_seq + kb * a.q_bnd + u * a.q_head + 8 * hh;
        qq = 0.f;
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (ok) v = *(const uint4 *)(qr + 16 * s);
            const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) qq += bf_lo(w4[e]) * bf_lo(w4[e]) + bf_hi(w4[e]) * bf_hi(w4[e]);
            qf[s] = __builtin_bit_cast(bf16x8_t, v);
        }
        qq += __shfl_xor(qq, 32);
    };

    // ---- stage copies: HBM -> LDS by global_load_lds_dwordx4.  Copy g of a
    // stage (wave w issues g = w, w + 8, ...) moves 64 chunks of one tile:
    // slot g / (2 IPT), tensor (g / IPT) % 2, chunks 64 (g % IPT) + lane.  Chunk
    // q of a tile is stored position q % NCH of key q / NCH and holds the key's
    // global chunk (q % NCH) ^ (key & SW), so the fragment reads below are
    // conflict free.  Keys past the sequence repeat its last token (masked).
    auto issue_stage = [&](int st, int nkt, auto &&kt_of) __attribute__((always_inline)) {
        const uint32_t base = (uint32_t)(uintptr_t)(lds_char_t *)lds + st * STAGE;
#pragma unroll
        for (int i = 0; i < NCOPY / kWaves; ++i) {
            const int g = wave + kWaves * i;
            const int slot = g / (2 * IPT), ten = (g / IPT) % 2, part_ = g % IPT;
            const int kt = kt_of(slot);
            if (kt < 0 || kt >= nkt) continue;
            const int qc = part_ * 64 + lane, key = qc / NCH, cs = qc % NCH;
            const int k0 = kt * kKT;
            const int kk = min(key, a.seq_len - 1 - k0);
            const uint16_t *tb = (ten ? Vg : Kg) + (int64_t)k0 * a.ts.tok;
            const uint32_t voff = (uint32_t)kk * (uint32_t)(a.ts.tok * 2) + (uint32_t)((cs ^ (key & SW)) * 16);
            copy16(voff, uniform_ptr(tb), __builtin_amdgcn_readfirstlane(base + slot * SLOTB + ten * TB + part_ * 1024));
        }
    };
    // |v|^2 of every key of stage st: four threads per key, fixed order
    auto key_norms = [&](int st) __attribute__((always_inline)) {
        const int slot = tid >> 7, key = (tid >> 2) & 31, pq = tid & 3;
        const char *row = lds + st * STAGE + slot * SLOTB + TB + key * D * 2;
        float s2 = 0.f;
#pragma unroll
        for (int cc = 0; cc < NCH / 4; ++cc) {                // chunks rotated by key: no bank conflicts
            const uint4 v = *(const uint4 *)(row + ((pq * (NCH / 4) + cc + key) & (NCH - 1)) * 16);
            const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) s2 += bf_lo(w4[e]) * bf_lo(w4[e]) + bf_hi(w4[e]) * bf_hi(w4[e]);
        }
        s2 += __shfl_xor(s2, 1);
        s2 += __shfl_xor(s2, 2);
        if (pq == 0) vvs[slot * kKT + key] = s2;
    };
    // One pass over n_it stages: body(it, st) on stage st = it & 1 after every
    // wave's copies of it have landed and the key norms are in place; between
    // the two barriers of an iteration, between(it) (the fixed-order reduction
    // of the previous iteration's per-key sums).
    auto sweep = [&](int n_it, int nkt, auto &&kt_of_it, auto &&between, auto &&body) __attribute__((always_inline)) {
        if (n_it <= 0) return;
        issue_stage(0, nkt, [&](int s) __attribute__((always_inline)) { return kt_of_it(0, s); });
        for (int it = 0; it < n_it; ++it) {
            const int st = it & 1;
            wait_vm<0>();
            __syncthreads();                                  // stage it landed; stage it - 1 is free
            key_norms(st);
            between(it);
            __syncthreads();
            if (it + 1 < n_it)
                issue_stage(st ^ 1, nkt, [&](int s) __attribute__((always_inline)) { return kt_of_it(it + 1, s); });
            body(it, st);
        }
        __syncthreads();
        between(n_it);
    };

    // 16-byte fragment s of row j of a K or V tile: channels 16 s + 8 hh .. +7
    // (the swizzled chunk 2 s + hh of the key's row)
    auto kfrag = [&](const char *Ks, int s) __attribute__((always_inline)) {
        return *(const bf16x8_t *)(Ks + j * D * 2 + (((2 * s + hh) ^ (j & SW)) * 16));
    };
    // V^T operand of key step kk of 32-d tile t: d row 32 t + (lane & 31), keys
    // 16 kk + {0..3, 8..11} + 4 hh (the key order of the accumulator layout).
    // Key 16 kk + 8 half + y (y = 4 hh + k4) sits at row offset y, chunk
    // 4 (t' ^ hh) + (z ^ k4) with t' = t ^ (2 half when rows have 16 chunks)
    // and z = 2 ((lane >> 4) & 1) + (a4 >> 1): one lane base for even t', one
    // for odd t', the rest compile-time offsets.
    const int vt_a4 = lane & 3, vt_k4 = (lane >> 2) & 3;
    const int vt_base = (4 * hh + vt_k4) * D * 2 + 16 * ((2 * ((lane >> 4) & 1) + (vt_a4 >> 1)) ^ vt_k4) +
                        8 * (vt_a4 & 1);
    const int vt_even = vt_base + 64 * hh, vt_odd = vt_base - 64 * hh;
    auto vtfrag = [&](const char *Vs, int kk, int t) __attribute__((always_inline)) {
        s16x4_t p4[2];
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int tp = t ^ (NCH == 16 ? 2 * half : 0);
            const char *pp = Vs + (16 * kk + 8 * half) * D * 2 + 64 * tp + ((tp & 1) ? vt_odd : vt_even);
            p4[half] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)pp);
        }
        typedef __attribute__((ext_vector_type(8))) short s16x8_t;
        const s16x8_t v8 = {p4[0][0], p4[0][1], p4[0][2], p4[0][3], p4[1][0], p4[1][1], p4[1][2], p4[1][3]};
        return __builtin_bit_cast(bf16x8_t, v8);
    };

    // ---- sweep A state of this wave's row tile (log2 units)
    float m, lsum, l2, e2v;
    f32x16_t OT[NDT], O2T[NDT];
    bf16x8_t oh[NKS], ol[NKS];                                // o as two bf16 terms: o[row j][16 s + 8 hh .. +7]
    auto reset_a = [&](int t) __attribute__((always_inline)) {
        m = -HUGE_VALF;
        lsum = l2 = e2v = 0.f;
#pragma unroll
        for (int q = 0; q < NDT; ++q) {
            OT[q] = f32x16_t{};
            O2T[q] = f32x16_t{};
        }
#pragma unroll
        for (int q = 0; q < NKS; ++q) oh[q] = ol[q] = bf16x8_t{};     // ends the last pass's o
    };
    // eligible keys of key tile kt (key mod stride == 0) as a bit mask over
    // the tile's 32 keys; wave-uniform
    auto elig_mask = [&](int kt) __attribute__((always_inline)) {
        const int st_ = a.stride;
        if (st_ == 1) return 0xffffffffu;
        const int r0 = (st_ - (kt * kKT) % st_) % st_;
        uint32_t msk = 0u;
        for (int r = r0; r < kKT; r += st_) msk |= 1u << r;
        return (uint32_t)__builtin_amdgcn_readfirstlane(msk);
    };
    // one key tile kt at slot s of stage st
    auto body_a = [&](int st, int s, int kt) __attribute__((always_inline)) {
        const char *Ks = lds + st * STAGE + s * SLOTB, *Vs = Ks + TB;
        f32x16_t S = {};
#pragma unroll
        for (int k = 0; k < NKS; ++k) S = mfma(kfrag(Ks, k), qf[k], S);
        const int kc = c - kt * kKT;                          // keys i <= c of this tile: acc_row <= kc
        const uint32_t em = elig_mask(kt) >> (4 * hh);        // bit acc_row(v, 0) of v's key
        float x[16], tmax = -HUGE_VALF;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            x[v] = acc_row(v, hh) <= kc ? S[v] * a.scale_log2 : -HUGE_VALF;
            tmax = fmaxf(tmax, x[v]);
        }
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        const float mn = fmaxf(m, tmax);                     // -inf only while the row has no key yet
        const float al = m > -HUGE_VALF ? __builtin_amdgcn_exp2f(m - mn) : 0.f;
        const float al2 = al * al;
        float pv[16], ts = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            pv[v] = __builtin_amdgcn_exp2f(x[v] > -HUGE_VALF ? x[v] - mn : -HUGE_VALF);
            ts += pv[v];
        }
        ts += __shfl_xor(ts, 32);
        lsum = lsum * al + ts;
        m = mn;
        if (__ballot(al != 1.f)) {                           // a row's maximum grew: rescale the sums
#pragma unroll
            for (int q = 0; q < NDT; ++q)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    OT[q][v] *= al;
                    O2T[q][v] *= al2;
                }
        }
        const float4 *vv4 = (const float4 *)(vvs + s * kKT);
        float t2 = 0.f, te = 0.f;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            float p2[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int v = 8 * kk + e;
                const bool el = acc_row(v, hh) < kc && ((em >> acc_row(v, 0)) & 1u);
                p2[e] = el ? pv[v] * pv[v] : 0.f;
            }
#pragma unroll
            for (int g2 = 0; g2 < 2; ++g2) {
                const float4 vk = vv4[2 * (2 * kk + g2) + hh];  // |v|^2 of keys 8 (2 kk + g2) + 4 hh .. +3
                t2 += (p2[4 * g2] + p2[4 * g2 + 1]) + (p2[4 * g2 + 2] + p2[4 * g2 + 3]);
                te += (p2[4 * g2] * vk.x + p2[4 * g2 + 1] * vk.y) + (p2[4 * g2 + 2] * vk.z + p2[4 * g2 + 3] * vk.w);
            }
            bf16x8_t ph, pl, qh, ql;
            split8(pv + 8 * kk, ph, pl);
            split8(p2, qh, ql);
#pragma unroll
            for (int q = 0; q < NDT; ++q) {
                const bf16x8_t vf = vtfrag(Vs, kk, q);
                OT[q] = mfma(vf, ph, OT[q]);
                OT[q] = mfma(vf, pl, OT[q]);
                O2T[q] = mfma(vf, qh, O2T[q]);
                O2T[q] = mfma(vf, ql, O2T[q]);
            }
        }
        t2 += __shfl_xor(t2, 32);
        te += __shfl_xor(te, 32);
        l2 = l2 * al2 + t2;
        e2v = e2v * al2 + te;
    };

    // ---- finished row tile: o, the boundary masses, the row data of sweep C.
    // o leaves the accumulator layout (lane half hh holds channels
    // 32 q + 8 g + 4 hh + 0..3) for the operand layout of o V^T (lane half hh
    // holds channels 16 s + 8 hh + 0..7): the halves swap four-channel groups.
    auto split_o = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < NDT; ++q)
#pragma unroll
            for (int sub = 0; sub < 2; ++sub) {
                float own[2][4], oth[2][4];                   // groups g = 2 sub + 0 and 2 sub + 1
#pragma unroll
                for (int gi = 0; gi < 2; ++gi)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        own[gi][e] = OT[q][4 * (2 * sub + gi) + e];
                        oth[gi][e] = __shfl_xor(own[gi][e], 32);
                    }
                // lane half hh takes group 2 sub + hh: channels 0..3 from half 0, 4..7 from half 1
                float ov[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    ov[e] = hh == 0 ? own[0][e] : oth[1][e];
                    ov[4 + e] = hh == 0 ? oth[0][e] : own[1][e];
                }
                split8(ov, oh[2 * q + sub], ol[2 * q + sub]);
            }
    };
    auto finish_tile = [&](int t) __attribute__((always_inline)) {
        const float inv_l = lsum > 0.f ? 1.f / lsum : 0.f;
        float oo = 0.f, oo2 = 0.f;                            // |o|^2 and o . sum p^2 v
#pragma unroll
        for (int k = 0; k < NDT; ++k)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                OT[k][v] *= inv_l;
                oo += OT[k][v] * OT[k][v];
                oo2 += OT[k][v] * O2T[k][v];
            }
        oo += __shfl_xor(oo, 32);
        oo2 += __shfl_xor(oo2, 32);
        split_o();
        const float il2 = inv_l * inv_l;
        float mV = l2 * il2, mK = qq / (float)D * (e2v - 2.f * oo2 + oo * l2) * il2;
        for (int o = 1; o < a.G; o <<= 1) {                   // the G rows of one boundary are adjacent lanes
            mV += __shfl_xor(mV, o);
            mK += __shfl_xor(mK, o);
        }
        // row data: p^2 = exp2(2 s log2e/sqrt(d) - w2) with w2 = 2 (m - log2 inv_l)
        // (+inf for a row without keys), 1/mass_V, (|q|^2/d)/mass_K, that times |o|^2
        const float cK = mK > 0.f ? qq / (float)D / mK : 0.f;
        const float w2 = inv_l > 0.f ? 2.f * (m - __log2f(inv_l)) : HUGE_VALF;
        if (hh == 0) {
            ri0[t][j] = make_float4(w2, mV > 0.f ? 1.f / mV : 0.f, cK, cK * oo);
            ri1[t][j] = (float)c;
        }
    };
    // o of a row tile through LDS: [s][hi, lo][lane] 16-byte fragments
    auto put_o = [&](int t) __attribute__((always_inline)) {
        uint4 *ob = (uint4 *)(lds + t * (NKS * 2 * 64 * 16)) + lane;
#pragma unroll
        for (int q = 0; q < NKS; ++q) {
            ob[(q * 2 + 0) * 64] = __builtin_bit_cast(uint4, oh[q]);
            ob[(q * 2 + 1) * 64] = __builtin_bit_cast(uint4, ol[q]);
        }
    };
    auto get_o = [&](int t) __attribute__((always_inline)) {
        const uint4 *ob = (const uint4 *)(lds + t * (NKS * 2 * 64 * 16)) + lane;
#pragma unroll
        for (int q = 0; q < NKS; ++q) {
            oh[q] = __builtin_bit_cast(bf16x8_t, ob[(q * 2 + 0) * 64]);
            ol[q] = __builtin_bit_cast(bf16x8_t, ob[(q * 2 + 1) * 64]);
        }
    };

    // ---- sweep C: per-key terms of one key tile kt at slot s of stage st
    // (lane = key j of the tile; accumulator rows = the tile's 32 queries)
    auto body_c = [&](int st, int s, int kt, int t, int buf) __attribute__((always_inline)) {
        const char *Ks = lds + st * STAGE + s * SLOTB, *Vs = Ks + TB;
        f32x16_t S = {}, VO = {};
#pragma unroll
        for (int k = 0; k < NKS; ++k) S = mfma(qf[k], kfrag(Ks, k), S);
#pragma unroll
        for (int k = 0; k < NKS; ++k) {
            const bf16x8_t vf = kfrag(Vs, k);                 // V[key j][16 k + 8 hh .. +7]
            VO = mfma(oh[k], vf, VO);
            VO = mfma(ol[k], vf, VO);
        }
        const float vk = vvs[s * kKT + j];
        const float key = (float)(kt * kKT + j);
        const bool key_el = (elig_mask(kt) >> j) & 1u;
        const float s2 = 2.f * a.scale_log2;
        float sK = 0.f, sV = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int qi = acc_row(v, hh);                    // query row within the tile
            const float4 r0 = ri0[t][qi];                     // w2, 1/mass_V, cK, cK |o|^2
            float e = fmaf(S[v], s2, -r0.x);
            e = (key_el && key < ri1[t][qi]) ? e : -HUGE_VALF;    // key < c of the row
            const float p2 = __builtin_amdgcn_exp2f(e);
            sV = fmaf(p2, r0.y, sV);
            const float tk = fmaf(-2.f * r0.z, VO[v], fmaf(r0.z, vk, r0.w));
            sK = fmaf(p2, tk, sK);
        }
        sK += __shfl_xor(sK, 32);
        sV += __shfl_xor(sV, 32);
        if (hh == 0) {
            part[buf][wave][s][j][0] = sK;
            part[buf][wave][s][j][1] = sV;
        }
    };
    auto zero_part = [&](int buf, int s) __attribute__((always_inline)) {
        if (hh == 0) {
            part[buf][wave][s][j][0] = 0.f;
            part[buf][wave][s][j][1] = 0.f;
        }
    };
    // fixed-order sum over the waves of iteration it's per-key sums; `add`:
    // key tiles below it already hold the pre pass's sums in r
    auto reduce_store = [&](int it, auto &&kt_of, int nkt, int add) __attribute__((always_inline)) {
        if (tid < kSlots * 64) {
            const int s = tid >> 6, key = (tid >> 1) & 31, comp = tid & 1;
            const int kt = kt_of(it, s);
            if (kt >= 0 && kt < nkt) {
                float v = 0.f;
                for (int w = 0; w < kWaves; ++w) v += part[it & 1][w][s][key][comp];
                const int tok = kt * kKT + key;
                if (tok < a.seq_len) {
                    float *rr = comp ? rV : rK;
                    if (kt < add) v += rr[tok];
                    rr[tok] = v;
                }
            }
        }
    };

    const AttnSched &S = a.s;
    int cover = 0;                                            // key tiles written by the C sweeps

    // ================= pre pass: short row tiles, one wave each, key tiles 4 it + s
    int pre_c = 0;                                            // key tiles of r the pre pass wrote
    if (S.pre_it > 0) {
        const int t = S.pre_tile[wave];
        int nka = 0;
        for (int w = 0; w < kWaves; ++w) {
            nka = max(nka, nt_a(S.pre_tile[w]));
            pre_c = max(pre_c, nt_c(S.pre_tile[w]));
        }
        const int my_a = nt_a(t), my_c = nt_c(t);
        auto kt_pre = [](int it, int s) __attribute__((always_inline)) { return 4 * it + s; };
        const int n_it_c = (pre_c + kSlots - 1) / kSlots;
        load_q(t);
        reset_a(t);
        sweep(S.pre_it, nka, kt_pre, [](int) __attribute__((always_inline)) {}, [&](int it, int st) __attribute__((always_inline)) {
            for (int s = 0; s < kSlots; ++s) {
                const int kt = kt_pre(it, s);
                if (kt < my_a) body_a(st, s, kt);
            }
        });
        if (t >= 0) finish_tile(t);
        sweep(n_it_c, pre_c, kt_pre,
              [&](int it) __attribute__((always_inline)) { if (it > 0) reduce_store(it - 1, kt_pre, pre_c, 0); },
              [&](int it, int st) __attribute__((always_inline)) {
                  for (int s = 0; s < kSlots; ++s) {
                      const int kt = kt_pre(it, s);
                      if (kt < my_c) body_c(st, s, kt, t, it & 1);
                      else zero_part(it & 1, s);
                  }
              });
        cover = pre_c;
    }

    // ================= main pass: long row tiles split by key over the waves
    if (S.main_it > 0) {
        const int t = S.main_tile[wave];
        const uint32_t mask = (uint32_t)S.main_mask[wave];
        const int n_it = S.main_it;
        int nka = 0, nkc = 0;
        for (int w = 0; w < kWaves; ++w) {
            nka = max(nka, nt_a(S.main_tile[w]));
            nkc = max(nkc, nt_c(S.main_tile[w]));
        }
        const int my_a = nt_a(t), my_c = nt_c(t);
        auto kt_main = [n_it](int it, int s) __attribute__((always_inline)) { return it + s * n_it; };
        load_q(t);
        reset_a(t);
        sweep(n_it, nka, kt_main, [](int) __attribute__((always_inline)) {}, [&](int it, int st) __attribute__((always_inline)) {
            for (int s = 0; s < kSlots; ++s) {
                const int kt = kt_main(it, s);
                if (((mask >> s) & 1u) && kt < my_a) body_a(st, s, kt);
            }
        });
        // merge the partial sums of waves sharing a row tile into its leader
        // (log-sum-exp), in wave order, three records per round
        for (int r = 0; r < S.n_rounds; ++r) {
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                if (S.round_w[r][k] != wave) continue;
                float *rec = ldsf + k * RECF * 64 + lane;
                rec[0] = m;
                rec[64] = lsum;
                rec[128] = l2;
                rec[192] = e2v;
#pragma unroll
                for (int q = 0; q < NDT; ++q)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        rec[(4 + q * 16 + v) * 64] = OT[q][v];
                        rec[(4 + NDT * 16 + q * 16 + v) * 64] = O2T[q][v];
                    }
            }
            __syncthreads();
            for (int k = 0; k < 3; ++k) {
                const int w2 = S.round_w[r][k];
                if (w2 < 0 || w2 == wave || S.leader[w2] != wave) continue;
                const float *rec = ldsf + k * RECF * 64 + lane;
                const float mb = rec[0];
                if (mb == -HUGE_VALF) continue;                       // that part saw no key of this row
                const float mn = fmaxf(m, mb);
                const float al = m > -HUGE_VALF ? __builtin_amdgcn_exp2f(m - mn) : 0.f, be = __builtin_amdgcn_exp2f(mb - mn);
                const float al2 = al * al, be2 = be * be;
                m = mn;
                lsum = al * lsum + be * rec[64];
                l2 = al2 * l2 + be2 * rec[128];
                e2v = al2 * e2v + be2 * rec[192];
#pragma unroll
                for (int q = 0; q < NDT; ++q)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        OT[q][v] = al * OT[q][v] + be * rec[(4 + q * 16 + v) * 64];
                        O2T[q][v] = al2 * O2T[q][v] + be2 * rec[(4 + NDT * 16 + q * 16 + v) * 64];
                    }
            }
            __syncthreads();
        }
        // leaders finish their tiles and publish o; the other waves of a tile take it
        const bool leader = t >= 0 && S.leader[wave] == wave;
        if (leader) {
            finish_tile(t);
            put_o(t);
        }
        __syncthreads();
        if (t >= 0 && !leader) get_o(t);
        __syncthreads();                                       // the stage buffers are free again
        const int add = cover;
        sweep(n_it, nkc, kt_main,
              [&](int it) __attribute__((always_inline)) { if (it > 0) reduce_store(it - 1, kt_main, nkc, add); },
              [&](int it, int st) __attribute__((always_inline)) {
                  for (int s = 0; s < kSlots; ++s) {
                      const int kt = kt_main(it, s);
                      if (((mask >> s) & 1u) && kt < my_c) body_c(st, s, kt, t, it & 1);
                      else zero_part(it & 1, s);
                  }
              });
        cover = max(cover, nkc);
    }

    // positions past the last key tile any C sweep wrote
    for (int tok = cover * kKT + tid; tok < a.seq_len; tok += kThreads) {
        rK[tok] = 0.f;
        rV[tok] = 0.f;
    }
}

// One workgroup per row of r: mean over the calibration rows, CV^2, alpha,
// then w = 1 + alpha (r / mean - 1) on calibration rows and 0 elsewhere.
__global__ __launch_bounds__(256) void attn_weights_kernel(int n_seqs, int seq_len, int stride, const float *r,
                                                           int64_t r_row_stride, int p, float *w,
                                                           int64_t w_row_stride, float *alpha) {
    __shared__ double red[4];
    const int row = blockIdx.x, tid = threadIdx.x;
    const float *rr = r + (int64_t)row * r_row_stride;
    float *ww = w + (int64_t)row * w_row_stride;
    const int per = (seq_len + stride - 1) / stride;          // calibration rows per sequence
    const int64_t n = (int64_t)n_seqs * per;
    auto block_sum = [&](double v) {
        for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
        __syncthreads();
        if ((tid & 63) == 0) red[tid >> 6] = v;
        __syncthreads();
        return (red[0] + red[1]) + (red[2] + red[3]);
    };
    double s = 0.0;
    for (int64_t e = tid; e < n; e += 256) s += (double)rr[(e / per) * seq_len + (e % per) * stride];
    const double mean = n > 0 ? block_sum(s) / (double)n : 0.0;
    double v = 0.0;
    for (int64_t e = tid; e < n; e += 256) {
        const double x = mean > 0.0 ? (double)rr[(e / per) * seq_len + (e % per) * stride] / mean : 1.0;
        v += (x - 1.0) * (x - 1.0);
    }
    const double cv2 = n > 0 ? block_sum(v) / (double)n : 0.0;
    const double tau = (double)(n < 2 * (int64_t)p ? n : 2 * (int64_t)p);
    double al = 1.0;
    if (cv2 > 0.0) al = fmin(1.0, sqrt(((double)n / tau - 1.0) / cv2));
    if (tid == 0) alpha[row] = (float)al;
    for (int64_t i = tid; i < (int64_t)n_seqs * seq_len; i += 256) {
        const int t = (int)(i % seq_len);
        double x = 0.0;
        if (t % stride == 0) x = 1.0 + al * ((mean > 0.0 ? (double)rr[i] / mean : 1.0) - 1.0);
        ww[i] = (float)x;
    }
}

}  // namespace

namespace {

// Work split of a call, chosen on the host (it depends on the boundaries
// only).  nab[t]: key tiles row tile t attends in sweep A.  For every count of
// short tiles sent to the pre pass (the shortest ones), the remaining tiles
// get one wave each, and the spare waves go, one at a time, to the tile whose
// split lowers the cost most; a tile's stage slots are cut into contiguous
// groups, one per wave.  Cost: both sweeps' lockstep steps (per stage, the
// most key tiles any wave handles, plus a fixed cost for the stage's copies
// and barriers) and the merge rounds.  The cheapest choice wins.
AttnSched plan_attn(const std::vector<int> &nab) {
    constexpr double kStage = 0.3, kRound = 0.5;
    const int n_rt = (int)nab.size();
    std::vector<int> order(n_rt);
    for (int t = 0; t < n_rt; ++t) order[t] = t;
    std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return nab[x] > nab[y]; });
    double best = HUGE_VAL;
    AttnSched out = {};
    for (int n_pre = 0; n_pre <= n_rt; ++n_pre) {
        const int n_main = n_rt - n_pre;
        if (n_main > kWaves) continue;
        const std::vector<int> main_t(order.begin(), order.begin() + n_main);
        const std::vector<int> pre_t(order.begin() + n_main, order.end());
        const int main_it = n_main ? (nab[main_t[0]] + kSlots - 1) / kSlots : 0;
        auto slots_of = [&](int i) { return (nab[main_t[i]] + main_it - 1) / main_it; };
        auto mask_of = [&](int i, int g, int k) {
            const int S = slots_of(i), lo = g * S / k, hi = (g + 1) * S / k;
            uint32_t m = 0;
            for (int s = lo; s < hi; ++s) m |= 1u << s;
            return m;
        };
        std::vector<int> k(n_main, 1);
        auto cost_main = [&]() {
            double c = 0.0;
            for (int it = 0; it < main_it; ++it) {
                int mx = 0;
                for (int i = 0; i < n_main; ++i)
                    for (int g = 0; g < k[i]; ++g) {
                        const uint32_t m = mask_of(i, g, k[i]);
                        int cnt = 0;
                        for (int s = 0; s < kSlots; ++s)
                            if (((m >> s) & 1u) && it + s * main_it < nab[main_t[i]]) ++cnt;
                        mx = std::max(mx, cnt);
                    }
                c += mx + kStage;
            }
            return c;
        };
        double cm = cost_main();
        for (int left = kWaves - n_main; left > 0; --left) {
            int bi = -1;
            double bc = cm;
            for (int i = 0; i < n_main; ++i) {
                if (k[i] >= slots_of(i)) continue;
                ++k[i];
                const double c = cost_main();
                --k[i];
                if (c < bc - 1e-9) {
                    bc = c;
                    bi = i;
                }
            }
            if (bi < 0) break;
            ++k[bi];
            cm = bc;
        }
        int pre_it = 0;
        double cp = 0.0;
        if (!pre_t.empty()) {
            int mx = 0;
            for (int t : pre_t) mx = std::max(mx, nab[t]);
            pre_it = (mx + kSlots - 1) / kSlots;
            for (int it = 0; it < pre_it; ++it) {
                int m = 0;
                for (int t : pre_t) m = std::max(m, std::min(kSlots, std::max(0, nab[t] - kSlots * it)));
                cp += m + kStage;
            }
        }
        int extra = 0;
        for (int i = 0; i < n_main; ++i) extra += k[i] - 1;
        const int rounds = (extra + 2) / 3;
        const double total = 2.0 * (cm + cp) + kRound * rounds;
        if (total >= best || rounds > kMaxRounds) continue;
        best = total;
        AttnSched sc;
        for (int w = 0; w < kWaves; ++w) {
            sc.pre_tile[w] = w < (int)pre_t.size() ? pre_t[w] : -1;
            sc.main_tile[w] = -1;
            sc.main_mask[w] = 0;
            sc.leader[w] = w;
        }
        sc.pre_it = pre_it;
        sc.main_it = main_it;
        std::vector<int> writers;
        int w = 0;
        for (int i = 0; i < n_main; ++i) {
            const int lead = w;
            for (int g = 0; g < k[i]; ++g, ++w) {
                sc.main_tile[w] = main_t[i];
                sc.main_mask[w] = (int32_t)mask_of(i, g, k[i]);
                sc.leader[w] = lead;
                if (g > 0) writers.push_back(w);
            }
        }
        sc.n_rounds = rounds;
        for (int r = 0; r < kMaxRounds; ++r)
            for (int q = 0; q < 3; ++q) {
                const size_t idx = (size_t)r * 3 + q;
                sc.round_w[r][q] = idx < writers.size() ? writers[idx] : -1;
            }
        out = sc;
    }
    return out;
}

}  // namespace

hipError_t launch_attn_sensitivity(const AttnLaunch &L, hipStream_t s) {
    AttnArgs a = {};
    a.kv = L.kv;
    a.ts = L.ts;
    a.q = L.q;
    a.q_layer = L.q_strides[0];
    a.q_seq = L.q_strides[1];
    a.q_bnd = L.q_strides[2];
    a.q_head = L.q_strides[3];
    a.n_layers = L.n_layers;
    a.n_heads = L.n_heads;
    a.G = L.G;
    a.n_bounds = L.n_bounds;
    a.n_rows = L.n_bounds * L.G;
    a.seq_len = L.seq_len;
    a.stride = L.stride;
    a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)L.d));
    a.r = L.r;
    a.r_row_stride = L.r_row_stride;
    const int n_rt = (a.n_rows + 31) / 32;
    if (L.n_bounds < 1 || L.n_bounds > 64 || n_rt > 8) return hipErrorInvalidValue;
    std::vector<int> nab(n_rt);
    for (int k = 0; k < L.n_bounds; ++k) a.bounds[k] = L.bounds[k];
    for (int t = 0; t < n_rt; ++t) nab[t] = (a.bounds[std::min(t * 32 + 31, a.n_rows - 1) / a.G] + kKT) / kKT;
    a.s = plan_attn(nab);
    const int64_t units = (int64_t)L.n_seqs * L.n_layers * L.n_heads;
    if (units == 0) return hipSuccess;
    if (L.d == 128) hipLaunchKernelGGL(attn_sens_kernel<128>, dim3((unsigned)units), dim3(kThreads), 0, s, a);
    else if (L.d == 64) hipLaunchKernelGGL(attn_sens_kernel<64>, dim3((unsigned)units), dim3(kThreads), 0, s, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_attn_weights(int32_t n_rows, int32_t n_seqs, int32_t seq_len, int32_t stride, const float *r,
                               int64_t r_row_stride, int32_t p, float *w, int64_t w_row_stride, float *alpha,
                               hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    hipLaunchKernelGGL(attn_weights_kernel, dim3(n_rows), dim3(256), 0, s, n_seqs, seq_len, stride, r, r_row_stride,
                       p, w, w_row_stride, alpha);
    return hipGetLastError();
}

}  // namespace cb

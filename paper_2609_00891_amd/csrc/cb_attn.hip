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
// head).  The queries of all boundaries and query heads of the group are the
// rows (row = boundary * G + head); a wave owns one tile of 32 rows, and SIMD
// s carries tiles s and 7 - s (boundaries increase with the row, so a short
// and a long key range share each SIMD).  Key tiles of 32 rows of K and V are
// streamed into a double-buffered LDS ring (16-byte chunks XOR-swizzled by
// key) by all 512 threads, which also form |v_i|^2; the waves then sweep the
// keys three times:
//   A  S^T = K Q^T (v_mfma_f32_32x32x16_bf16, one lane per query): the
//      online softmax maximum m and normalizer l of every query, and with
//      them o = sum exp(s - m) v / l (the partial o rescaled whenever m
//      grows; exp(s - m) split into two bf16 terms, V^T read with
//      ds_read_b64_tr_b16 in the key order of the accumulator layout);
//   B2 sum a^2 v, sum a^2 and sum a^2 |v|^2 over the eligible keys, then the
//      unit masses of every boundary for both components (the K mass is
//      sum a^2 (|v|^2 - 2 o.v + |o|^2) |q|^2 / d, expanded);
//   C  S = Q K^T and (o V^T) with o split into two bf16 terms (one lane per
//      key): every eligible (query, key) term, summed over the wave's queries
//      in registers; the eight waves' sums are added in a fixed order.
// Separate sweeps keep one set of accumulators live at a time (two waves per
// SIMD leave 256 registers per lane) and make B2 free of rescaling.
#include "cb_internal.h"

namespace cb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) short s16x4_t;
typedef __attribute__((ext_vector_type(8))) short s16x8_t;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

constexpr int kWaves = 8, kThreads = 64 * kWaves, kKT = 32;

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    f32x2_t v = {lo, hi};
    bf16x2_t p = __builtin_convertvector(v, bf16x2_t);
    return __builtin_bit_cast(uint32_t, p);
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

__device__ __forceinline__ f32x16_t mfma(bf16x8_t a, bf16x8_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Key index of accumulator register v in lane half hh of a 32x32 tile whose
// rows are keys: D[i][j] sits in lane j + 32 ((i >> 2) & 1), register
// 4 (i >> 3) + (i & 3).
__device__ __forceinline__ int acc_row(int v, int hh) { return 8 * (v >> 2) + 4 * hh + (v & 3); }

struct AttnArgs {
    const uint16_t *kv;              // target cache (K = kv 0, V = kv 1)
    Strides ts;
    const uint16_t *q;               // boundary queries
    int64_t q_layer, q_seq, q_bnd, q_head;
    int32_t n_layers, n_heads, G, n_bounds, n_rows, n_rtiles, seq_len, stride;
    float scale_log2;                // log2(e) / sqrt(d)
    float *r;                        // [(l * 2 + z) * H + h][seq * seq_len + tok]
    int64_t r_row_stride;
    int32_t bounds[64];
};

template <int D>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads), amdgpu_waves_per_eu(2, 2)))
void attn_sens_kernel(AttnArgs a) {
    constexpr int NCH = D / 8, NDT = D / 32, NKS = D / 16;   // 16-byte chunks per row, 32-d tiles, 16-d steps
    constexpr int SW = NCH < 16 ? NCH - 1 : 15;              // chunk swizzle mask
    constexpr int TB = kKT * D * 2;                          // bytes per K or V tile
    constexpr int PER = D / 64;                              // 16-byte chunks each thread loads per tile
    __shared__ __attribute__((aligned(16))) char lds[2 * 2 * TB];
    __shared__ __attribute__((aligned(16))) float vvs[2][kKT];
    __shared__ __attribute__((aligned(16))) float4 ri0[kWaves][32];   // m, 1/l, |o|^2, (|q|^2/d)/massK
    __shared__ __attribute__((aligned(16))) float2 ri1[kWaves][32];   // 1/massV, query position
    __shared__ float part[2][kWaves][kKT][2];
    __shared__ __attribute__((aligned(16))) char qlds[kWaves][32 * D * 2];    // each wave's 32 query rows

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j = lane & 31, hh = lane >> 5;
    const int unit = blockIdx.x;
    const int h = unit % a.n_heads;
    const int l = (unit / a.n_heads) % a.n_layers;
    const int b = unit / (a.n_heads * a.n_layers);
    const uint16_t *Kg = a.kv + l * a.ts.layer + b * a.ts.seq + h * a.ts.head;
    const uint16_t *Vg = Kg + a.ts.kv;

    // row tile of a wave and the largest query position of a tile
    auto tile_of = [](int w) { return w < 4 ? w : 11 - w; };
    auto tile_chi = [&](int t) {
        if (t >= a.n_rtiles) return -1;
        const int last = min(t * 32 + 31, a.n_rows - 1);
        return a.bounds[last / a.G];
    };
    const int tile = tile_of(wave);
    const int c_hi = tile_chi(tile);                         // -1: idle wave
    const int ntAB = c_hi >= 0 ? (c_hi + kKT) / kKT : 0;     // key tiles of keys 0 .. c_hi
    const int ntC = c_hi > 0 ? (c_hi + kKT - 1) / kKT : 0;   // key tiles of keys 0 .. c_hi - 1

    // this lane's query row (sweeps A and B)
    const int row = tile * 32 + j;
    const bool row_ok = c_hi >= 0 && row < a.n_rows;
    const int kb = row_ok ? row / a.G : 0;
    const int c = row_ok ? a.bounds[kb] : -1;
    const int u = h * a.G + (row_ok ? row % a.G : 0);
    // the wave's query rows go to LDS (chunks swizzled like the K tile); |q|^2 on the way
    float qq = 0.f;
    {
        const uint16_t *qr = a.q + l * a.q_layer + b * a.q_seq + kb * a.q_bnd + u * a.q_head + 8 * hh;
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (row_ok) v = *(const uint4 *)(qr + 16 * s);
            const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) qq += bf_lo(w4[e]) * bf_lo(w4[e]) + bf_hi(w4[e]) * bf_hi(w4[e]);
            *(uint4 *)(qlds[wave] + j * D * 2 + (((2 * s + hh) ^ (j & SW)) * 16)) = v;
        }
        qq += __shfl_xor(qq, 32);
    }
    // Q[row j][16 s + 8 hh .. +7]: B operand of S^T = K Q^T, A operand of S = Q K^T
    auto qfrag = [&](int s) {
        return *(const bf16x8_t *)(qlds[wave] + j * D * 2 + (((2 * s + hh) ^ (j & SW)) * 16));
    };

    // ---- cooperative K/V tile loads: thread chunk g = tid + 512 p of the
    // stage's [K | V] tiles, key-major; keys past the sequence repeat its last
    // token (they are masked everywhere).
    const int cmax = a.bounds[a.n_bounds - 1];
    auto gload = [&](int kt, uint4 (&pre)[PER]) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int g = tid + kThreads * p;
            const int ten = g / (kKT * NCH), rem = g % (kKT * NCH), key = rem / NCH, ch = rem % NCH;
            const int tok = min(kt * kKT + key, a.seq_len - 1);
            pre[p] = *(const uint4 *)((ten ? Vg : Kg) + (int64_t)tok * a.ts.tok + ch * 8);
        }
    };
    auto swrite = [&](int st, const uint4 (&pre)[PER]) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int g = tid + kThreads * p;
            const int ten = g / (kKT * NCH), rem = g % (kKT * NCH), key = rem / NCH, ch = rem % NCH;
            *(uint4 *)(lds + st * 2 * TB + ten * TB + key * D * 2 + ((ch ^ (key & SW)) * 16)) = pre[p];
            if (ten == 1) {                                   // |v|^2 of the key: its NCH chunks are adjacent lanes
                const uint32_t w4[4] = {pre[p].x, pre[p].y, pre[p].z, pre[p].w};
                float s2 = 0.f;
#pragma unroll
                for (int e = 0; e < 4; ++e) s2 += bf_lo(w4[e]) * bf_lo(w4[e]) + bf_hi(w4[e]) * bf_hi(w4[e]);
#pragma unroll
                for (int o = 1; o < NCH; o <<= 1) s2 += __shfl_xor(s2, o);
                if (ch == 0) vvs[st][key] = s2;
            }
        }
    };
    // one sweep over nt key tiles; body(kt, stage)
    auto sweep = [&](int nt, auto &&body) {
        if (nt <= 0) return;
        uint4 pre[PER];
        gload(0, pre);
        swrite(0, pre);
        __syncthreads();
        for (int kt = 0; kt < nt; ++kt) {
            if (kt + 1 < nt) gload(kt + 1, pre);
            body(kt, kt & 1);
            if (kt + 1 < nt) swrite((kt + 1) & 1, pre);
            __syncthreads();
        }
    };
    auto kst = [&](int st) { return lds + st * 2 * TB; };   // stage base: K tile, then V tile
    // A operand of S^T = K Q^T (and B operand of S = Q K^T): K[key j][16 s + 8 hh .. +7]
    auto kfrag = [&](int st, int s) {
        return *(const bf16x8_t *)(kst(st) + j * D * 2 + (((2 * s + hh) ^ (j & SW)) * 16));
    };
    auto s_tile = [&](int st, bool keys_are_rows) {
        f32x16_t acc = {};
#pragma unroll
        for (int s = 0; s < NKS; ++s) acc = keys_are_rows ? mfma(kfrag(st, s), qfrag(s), acc) : mfma(qfrag(s), kfrag(st, s), acc);
        return acc;
    };
    const int ntAll = (cmax + kKT) / kKT;
    const int ntAllC = cmax > 0 ? (cmax + kKT - 1) / kKT : 0;


    float m = -HUGE_VALF, lsum = 0.f, inv_l = 0.f;             // per query row, log2 units
    // V^T operand of key step kk of 32-d tile t: d row 32 t + (lane & 31), keys
    // 16 kk + {0..3, 8..11} + 4 hh (the key order of the accumulator layout)
    auto vtfrag = [&](const char *Vs, int kk, int t) {
        const int j16 = lane & 15, a4 = j16 & 3, k4 = j16 >> 2;
        const int dcol = 32 * t + 16 * ((lane >> 4) & 1) + 4 * a4;
        s16x4_t p4[2];
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int key = 16 * kk + 8 * half + 4 * hh + k4;
            const char *pp = Vs + key * D * 2 + (((dcol >> 3) ^ (key & SW)) * 16) + (dcol & 7) * 2;
            p4[half] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)pp);
        }
        const s16x8_t v8 = {p4[0][0], p4[0][1], p4[0][2], p4[0][3], p4[1][0], p4[1][1], p4[1][2], p4[1][3]};
        return __builtin_bit_cast(bf16x8_t, v8);
    };
    // probabilities a of key step kk of a tile (and, with sq, a^2 on eligible keys)
    auto probs = [&](const f32x16_t &S, int kt, int kk, bool sq, float *out) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int v = 8 * kk + e;
            const int key = kt * kKT + acc_row(v, hh);
            const float p = key <= c ? exp2f(S[v] * a.scale_log2 - m) * inv_l : 0.f;
            out[e] = sq ? ((key < c && key % a.stride == 0) ? p * p : 0.f) : p;
        }
    };

    // ---- sweep A: the softmax maximum m and normalizer l (log2 units) and,
    // online, o = sum_i exp(s_i - m) v_i / l: whenever a tile raises a row's
    // maximum its partial o is rescaled by exp(m_old - m_new), and o is divided
    // by l once every key has been seen.  p = exp(s - m) <= 1 enters the MFMA
    // as two bf16 terms.
    f32x16_t OT[NDT];
#pragma unroll
    for (int t = 0; t < NDT; ++t) OT[t] = f32x16_t{};
    sweep(ntAll, [&](int kt, int st) {
        if (kt >= ntAB) return;
        const f32x16_t S = s_tile(st, true);
        float x[16], tmax = -HUGE_VALF;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int key = kt * kKT + acc_row(v, hh);
            x[v] = key <= c ? S[v] * a.scale_log2 : -HUGE_VALF;
            tmax = fmaxf(tmax, x[v]);
        }
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        const float mn = fmaxf(m, tmax);                     // -inf only while the row has no key yet
        const float alpha = m > -HUGE_VALF ? exp2f(m - mn) : 0.f;
        float pv[16], ts = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            pv[v] = x[v] > -HUGE_VALF ? exp2f(x[v] - mn) : 0.f;
            ts += pv[v];
        }
        ts += __shfl_xor(ts, 32);
        lsum = lsum * alpha + ts;
        m = mn;
#pragma unroll
        for (int t = 0; t < NDT; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) OT[t][v] *= alpha;
        const char *Vs = kst(st) + TB;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            bf16x8_t ph, pl;
            split8(pv + 8 * kk, ph, pl);
#pragma unroll
            for (int t = 0; t < NDT; ++t) {
                const bf16x8_t vf = vtfrag(Vs, kk, t);
                OT[t] = mfma(vf, ph, OT[t]);
                OT[t] = mfma(vf, pl, OT[t]);
            }
        }
    });
    inv_l = lsum > 0.f ? 1.f / lsum : 0.f;
#pragma unroll
    for (int t = 0; t < NDT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) OT[t][v] *= inv_l;
    float oo = 0.f;
    bf16x8_t oh[NDT][2], ol[NDT][2];                          // o as two bf16 terms (the A operand of o V^T)
#pragma unroll
    for (int t = 0; t < NDT; ++t) {
#pragma unroll
        for (int v = 0; v < 16; ++v) oo += OT[t][v] * OT[t][v];
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            float ov[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) ov[e] = OT[t][8 * sub + e];
            split8(ov, oh[t][sub], ol[t][sub]);
        }
    }
    oo += __shfl_xor(oo, 32);

    // ---- sweep B2: sum a^2 v, sum a^2, sum a^2 |v|^2 over the eligible keys
    f32x16_t O2T[NDT];
#pragma unroll
    for (int t = 0; t < NDT; ++t) O2T[t] = f32x16_t{};
    float E2 = 0.f, E2V = 0.f;
    sweep(ntAll, [&](int kt, int st) {
        if (kt >= ntAB) return;
        const f32x16_t S = s_tile(st, true);
        const float4 *vv4 = (const float4 *)vvs[st];
        const char *Vs = kst(st) + TB;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            float a2[8];
            probs(S, kt, kk, true, a2);
#pragma unroll
            for (int g2 = 0; g2 < 2; ++g2) {
                const float4 vk = vv4[2 * (2 * kk + g2) + hh];  // |v|^2 of keys 8 (2 kk + g2) + 4 hh .. +3
                E2 += (a2[4 * g2] + a2[4 * g2 + 1]) + (a2[4 * g2 + 2] + a2[4 * g2 + 3]);
                E2V += (a2[4 * g2] * vk.x + a2[4 * g2 + 1] * vk.y) + (a2[4 * g2 + 2] * vk.z + a2[4 * g2 + 3] * vk.w);
            }
            bf16x8_t qh, ql;
            split8(a2, qh, ql);
#pragma unroll
            for (int t = 0; t < NDT; ++t) {
                const bf16x8_t vf = vtfrag(Vs, kk, t);
                O2T[t] = mfma(vf, qh, O2T[t]);
                O2T[t] = mfma(vf, ql, O2T[t]);
            }
        }
    });

    // ---- per-row sums, boundary masses, row data for sweep C
    E2 += __shfl_xor(E2, 32);
    E2V += __shfl_xor(E2V, 32);
    float oo2 = 0.f;                                          // o . sum a^2 v, with o as its two bf16 terms
#pragma unroll
    for (int t = 0; t < NDT; ++t)
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            const uint4 hv = __builtin_bit_cast(uint4, oh[t][sub]), lv = __builtin_bit_cast(uint4, ol[t][sub]);
            const uint32_t h4[4] = {hv.x, hv.y, hv.z, hv.w}, l4[4] = {lv.x, lv.y, lv.z, lv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                oo2 += (bf_lo(h4[e]) + bf_lo(l4[e])) * O2T[t][8 * sub + 2 * e];
                oo2 += (bf_hi(h4[e]) + bf_hi(l4[e])) * O2T[t][8 * sub + 2 * e + 1];
            }
        }
    oo2 += __shfl_xor(oo2, 32);
    float mV = E2, mK = qq / (float)D * (E2V - 2.f * oo2 + oo * E2);
    for (int o = 1; o < a.G; o <<= 1) {                       // the G rows of one boundary are adjacent lanes
        mV += __shfl_xor(mV, o);
        mK += __shfl_xor(mK, o);
    }
    if (c_hi >= 0 && hh == 0) {
        ri0[wave][j] = make_float4(m, inv_l, oo, mK > 0.f ? qq / (float)D / mK : 0.f);
        ri1[wave][j] = make_float2(mV > 0.f ? 1.f / mV : 0.f, (float)c);
    }
    __syncthreads();

    // ---- sweep C: per-key sums over every eligible query
    float *rK = a.r + ((int64_t)(l * 2 + 0) * a.n_heads + h) * a.r_row_stride + (int64_t)b * a.seq_len;
    float *rV = a.r + ((int64_t)(l * 2 + 1) * a.n_heads + h) * a.r_row_stride + (int64_t)b * a.seq_len;
    auto reduce_store = [&](int kt) {                         // fixed-order sum of the waves' partials
        if (tid < 64) {
            const int key = tid & 31, comp = tid >> 5;
            float s = 0.f;
            for (int w = 0; w < kWaves; ++w) {
                const int cw = tile_chi(tile_of(w));
                const int ntw = cw > 0 ? (cw + kKT - 1) / kKT : 0;
                if (kt < ntw) s += part[kt & 1][w][key][comp];
            }
            const int tok = kt * kKT + key;
            if (tok < a.seq_len) (comp ? rV : rK)[tok] = s;
        }
    };
    sweep(ntAllC, [&](int kt, int st) {
        if (kt > 0) reduce_store(kt - 1);
        if (kt >= ntC) return;
        const f32x16_t S = s_tile(st, false);
        const char *Vs = kst(st) + TB;
        f32x16_t VO = {};
#pragma unroll
        for (int t = 0; t < NDT; ++t)
#pragma unroll
            for (int sub = 0; sub < 2; ++sub) {
                // B operand: V[key j][32 t + 16 sub + 4 hh + {0..3, 8..11}]
                s16x4_t p4[2];
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const int dcol = 32 * t + 16 * sub + 8 * half + 4 * hh;
                    p4[half] = *(const s16x4_t *)(Vs + j * D * 2 + (((dcol >> 3) ^ (j & SW)) * 16) + (dcol & 7) * 2);
                }
                const s16x8_t v8 = {p4[0][0], p4[0][1], p4[0][2], p4[0][3], p4[1][0], p4[1][1], p4[1][2], p4[1][3]};
                const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, v8);
                VO = mfma(oh[t][sub], vf, VO);
                VO = mfma(ol[t][sub], vf, VO);
            }
        const int key = kt * kKT + j;
        const float vk = vvs[st][j];
        float sK = 0.f, sV = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int qi = acc_row(v, hh);                    // query row within the tile
            const float4 r0 = ri0[wave][qi];
            const float2 r1 = ri1[wave][qi];
            const int cq = (int)r1.y;
            if (key < cq && key % a.stride == 0) {
                const float p = exp2f(S[v] * a.scale_log2 - r0.x) * r0.y;
                const float p2 = p * p;
                sV += p2 * r1.x;
                sK += p2 * (vk - 2.f * VO[v] + r0.z) * r0.w;
            }
        }
        sK += __shfl_xor(sK, 32);
        sV += __shfl_xor(sV, 32);
        if (hh == 0) {
            part[kt & 1][wave][j][0] = sK;
            part[kt & 1][wave][j][1] = sV;
        }
    });
    if (ntAllC > 0) reduce_store(ntAllC - 1);
    // positions past the last eligible tile
    for (int tok = ntAllC * kKT + tid; tok < a.seq_len; tok += kThreads) {
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
    a.n_rtiles = (a.n_rows + 31) / 32;
    a.seq_len = L.seq_len;
    a.stride = L.stride;
    a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)L.d));
    a.r = L.r;
    a.r_row_stride = L.r_row_stride;
    if (L.n_bounds < 1 || L.n_bounds > 64 || a.n_rtiles > kWaves) return hipErrorInvalidValue;
    for (int k = 0; k < L.n_bounds; ++k) a.bounds[k] = L.bounds[k];
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

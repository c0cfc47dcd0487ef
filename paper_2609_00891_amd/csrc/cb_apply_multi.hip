// cb_apply_multi.hip -- online application of multi-layer maps (gfx950).
//
// CacheBridge Sec. 1 (online handoff) with the multi-layer feature of Sec. 3.2:
// map m reads the sender's rows of its k selected source layers and writes
//     out[t, :] = RNE_bf16( sum_i x_{i,t} W_{m,i} + b_m )
// where W_{m,i} is rows 128 i .. 128 i + 127 of the map.  At k = 8 that is
// 262 kFLOP per token and map against 256 bytes written: a dense contraction,
// run on the matrix cores.
//
// split_maps_frag_kernel: W (fp32) -> W^T as bf16 MFMA fragments, hi =
//   RNE(W) and lo = RNE(W - hi) (together ~16 significant bits), laid out
//   [map][block i][K step ks][wave w][plane][lane][8]: lane l of wave w holds
//   output channel 32 w + (l mod 32), inputs 128 i + 16 ks + 8 (l / 32) .. + 7.
//   One fragment load is 1 KiB contiguous.  The fp32 bias is kept apart.
//
// Two application kernels share that layout.  apply_pair_kernel (below) takes
// pairs of maps that read the same source blocks, staging each block once for
// both; apply_multi_kernel takes the maps left without such a partner.
//
// apply_multi_kernel: a task is (map, tile of 256 tokens).  The grid is
//   persistent, one workgroup of four waves per compute unit; the workgroups
//   of one XCD walk a contiguous run of tasks (maps in groups of four
//   neighbouring target layers, token tile first within a group, so the
//   group's W^T and the overlapping source windows stay in that XCD's L2).
//   Wave w owns output channels 32 w .. 32 w + 31 of all 256 tokens: eight
//   32 x 32 fp32 accumulator tiles, D = W^T x^T with
//   v_mfma_f32_32x32x16_bf16 (K = source channels), hi and lo products into
//   the same accumulators.
//
//   The work is one stream of source blocks (task, i), eight K steps each,
//   software-pipelined across blocks and tasks:
//     * the 256 x 128 rows of block b+1 are loaded into registers while block
//       b is multiplied, written to the other LDS buffer (16-byte chunk c of
//       token row t at c ^ (t mod 16)) at its last step, then one barrier;
//     * the x fragments of step s+1 are read from LDS during step s;
//     * the W^T fragments are loaded one block ahead, each into the registers
//       its step has just consumed.
//   At the end of a task the bias is added, the sum rounded once to bf16 and
//   stored as 16-byte chunks of target rows.
//
// With the target's rotary transform (Sec. 2.1, Sec. 3.1: the mapped keys
// receive the target's RoPE) the K outputs are turned in fp32 before that one
// rounding.  For the half-split pairing (i, i + 64) the fragments put output
// channels 16 w .. 16 w + 15 and 64 + 16 w .. + 15 on wave w's 32 rows (the
// perm flag of split_maps_frag_kernel), so each pair sits in registers v and
// v + 8 of one lane; the interleaved pairs (2i, 2i + 1) are registers v, v + 1
// in either layout.  K maps may read their source rows from a separate view
// (a de-rotated copy of the sender's keys).
#include "cb_internal.h"

namespace cb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

constexpr int TT = 256;                 // tokens per task
constexpr int ROWB = 256;               // bytes per 128-channel row
constexpr int BUFB = TT * ROWB;         // one staged source block (64 KiB)
constexpr int CPW = BUFB / 1024 / 4;    // 16-byte row chunks per lane and block (16)
constexpr int FRAG = 512;               // bf16 elements of one wave fragment (64 lanes x 8)
constexpr int64_t WBLK = 8 * 4 * 2 * FRAG;  // fragment elements per (map, block)

__device__ __forceinline__ uint32_t fastdiv_u(uint32_t n, const FastDiv &f) {
    const uint32_t t = __umulhi(n, f.m);
    return (t + ((n - t) >> f.sh1)) >> f.sh2;
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    f32x2_t v = {lo, hi};
    bf16x2_t p = __builtin_convertvector(v, bf16x2_t);
    return __builtin_bit_cast(uint32_t, p);
}

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

// This wave's LDS reads and writes have completed, then the workgroup barrier;
// the empty asm keeps the compiler from moving memory operations across it.
__device__ __forceinline__ void lds_sync() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt, expcnt untouched
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Output channel of row r (0..31) of wave w: 32 w + r, or with `perm` the
// half-split layout 16 w + r (r < 16), 64 + 16 w + r - 16.
__host__ __device__ __forceinline__ int frag_channel(int w, int r, bool perm) {
    return perm ? (r < 16 ? 16 * w + r : 64 + 16 * w + (r - 16)) : 32 * w + r;
}

__global__ __launch_bounds__(256) void split_maps_frag_kernel(int n_maps, int k, const float *__restrict__ maps,
                                                              uint16_t *__restrict__ wfrag, float *__restrict__ bias,
                                                              int perm) {
    const int P = 128 * k + 1;
    const int64_t total = (int64_t)n_maps * k * 8 * 4 * 64;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int lane = (int)(e & 63), w = (int)((e >> 6) & 3), ks = (int)((e >> 8) & 7);
        const int64_t mi = e >> 11;                       // map * k + block
        const int64_t m = mi / k;
        const int i = (int)(mi - m * k);
        const int c = frag_channel(w, lane & 31, perm != 0);
        const int K0 = 128 * i + 16 * ks + 8 * (lane >> 5);
        const float *src = maps + (m * P + K0) * 128 + c;
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
            const float v0 = src[j * 128], v1 = src[(j + 1) * 128];
            const uint32_t p = pack_bf16(v0, v1);
            const float h0 = __uint_as_float(p << 16), h1 = __uint_as_float(p & 0xffff0000u);
            hi[j / 2] = p;
            lo[j / 2] = pack_bf16(v0 - h0, v1 - h1);
        }
        uint16_t *dst = wfrag + ((mi * 8 + ks) * 4 + w) * (2 * FRAG) + lane * 8;
        *reinterpret_cast<uint4 *>(dst) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
        *reinterpret_cast<uint4 *>(dst + FRAG) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        if (i == 0 && ks == 0 && lane < 32) bias[m * 128 + c] = maps[(m * P + P - 1) * 128 + c];
    }
}

// Uniform description of one task.
struct Task {
    int32_t m;          // map index
    int64_t tok0;       // first token of the tile
    const uint16_t *x;  // source base of the map's (kv, head), layer 0
    const int32_t *layers;
    int64_t s_layer, s_seq, s_tok;   // strides of the view the map reads
};

__device__ __forceinline__ Task task_of(const ApplyMultiArgs &a, int task) {
    // maps in groups of four (the last group may be smaller), tile-major inside a group
    const int full = a.n_maps & ~3;
    const int64_t in_full = (int64_t)full * a.n_tiles;
    int tile, gm;
    if (task < in_full) {
        const int per = 4 * a.n_tiles;
        const int g = task / per, r = task - g * per;
        tile = r >> 2;
        gm = 4 * g + (r & 3);
    } else {
        const int rem = a.n_maps - full;
        const int r = task - (int)in_full;
        tile = r / rem;
        gm = full + (r - tile * rem);
    }
    Task t;
    t.m = __builtin_amdgcn_readfirstlane(a.order[gm]);
    t.tok0 = (int64_t)tile * TT;
    const ApplyMultiMap mp = a.maps[t.m];
    const bool kview = mp.kv == 0 && a.srck != nullptr;
    const Strides &v = kview ? a.ssk : a.ss;
    t.x = kview ? a.srck + mp.src_head * v.head : a.src + mp.kv * v.kv + mp.src_head * v.head;
    t.s_layer = v.layer;
    t.s_seq = v.seq;
    t.s_tok = v.tok;
    t.layers = a.src_layers + (int64_t)t.m * a.k;
    return t;
}

// RS: target rotation of the K outputs, 0 none, 1 pairs (i, i + 64), 2 pairs (2i, 2i + 1).
template <int RS>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void apply_multi_kernel(ApplyMultiArgs a) {
    __shared__ __attribute__((aligned(16))) char lds[2 * BUFB];
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int per_wg = gridDim.x >> 3;                    // workgroups per XCD (the grid is a multiple of 8)
    const int t_end = min(xcd * a.per_xcd + a.per_xcd, a.n_tasks);
    int task = xcd * a.per_xcd + slot;
    if (task >= t_end) return;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int k = a.k;
    const uint32_t lrow = lane & 31, lhalf = lane >> 5;

    // ---- staging geometry: chunk j of this lane is token row 16 j + 4 wave + lane / 16, chunk lane mod 16,
    // written at LDS chunk position (lane mod 16) ^ (row mod 16), row mod 16 = 4 wave + lane / 16
    const int rsub = 4 * wave + (lane >> 4);
    const uint32_t sdst = (uint32_t)rsub * ROWB + (uint32_t)((lane & 15) ^ rsub) * 16u;
    // element offset of the lane's chunk inside a (layer, kv, head) block (below 2^32: checked on the host)
    uint32_t rowoff[CPW];
    auto set_rows = [&](const Task &tk_) {
#pragma unroll
        for (int j = 0; j < CPW; ++j) {
            int64_t n = tk_.tok0 + 16 * j + rsub;
            if (n >= a.N) n = a.N - 1;                    // rows past the end repeat the last token
            const uint32_t seq = fastdiv_u((uint32_t)n, a.T);
            const uint32_t tk = (uint32_t)n - seq * a.T.d;
            rowoff[j] = (uint32_t)(seq * tk_.s_seq + tk * tk_.s_tok) + (lane & 15) * 8;
        }
    };
    // half h of a block: chunks 8 h .. 8 h + 7 of the lane
    constexpr int HC = CPW / 2;
    auto load_half = [&](u32x4_t (&st)[HC], const uint16_t *xb, int h) {
#pragma unroll
        for (int j = 0; j < HC; ++j) st[j] = *reinterpret_cast<const u32x4_t *>(xb + rowoff[HC * h + j]);
    };
    // a quarter q of the block: chunks 4 q .. 4 q + 3, into st0 (q < 2) or st1
    auto load_quarter = [&](u32x4_t (&st)[HC], const uint16_t *xb, int q) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            st[4 * (q & 1) + j] = *reinterpret_cast<const u32x4_t *>(xb + rowoff[4 * q + j]);
    };
    auto store_half = [&](const u32x4_t (&st)[HC], int buf, int h) {
#pragma unroll
        for (int j = 0; j < HC; ++j)
            *reinterpret_cast<u32x4_t *>(lds + buf * BUFB + (HC * h + j) * 4096 + sdst) = st[j];
    };
    // x fragments of step ks: token row 32 s + lane mod 32, channels 16 ks + 8 (lane / 32) .. + 7
    bf16x8_t xr[2][8];
    auto read_x = [&](bf16x8_t (&x)[8], int buf, int ks) {
        const char *B = lds + buf * BUFB + lrow * ROWB + (((2 * ks + lhalf) ^ (lrow & 15)) * 16);
#pragma unroll
        for (int s = 0; s < 8; ++s) x[s] = *reinterpret_cast<const bf16x8_t *>(B + s * 32 * ROWB);
    };
    // W^T fragments of the eight steps of a block; step ks's registers are refilled with the next block's
    // fragments right after its MFMAs, so every fragment is loaded one block ahead
    bf16x8_t wh[8], wl[8];
    const int64_t wlane = (int64_t)wave * (2 * FRAG) + lane * 8;
    auto wptr = [&](int m, int i) { return a.wfrag + ((int64_t)m * k + i) * WBLK + wlane; };
    auto load_w = [&](int r, const uint16_t *p) {
        wh[r] = *reinterpret_cast<const bf16x8_t *>(p);
        wl[r] = *reinterpret_cast<const bf16x8_t *>(p + FRAG);
    };

    f32x16_t acc[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[s][v] = 0.f;

    // ---- prologue: block 0 of the first task in LDS buffer 0, its W fragments, x of step 0
    Task cur = task_of(a, task);
    set_rows(cur);
    {
        const uint16_t *xb = cur.x + cur.layers[0] * cur.s_layer;
        u32x4_t st0[HC], st1[HC];
        load_half(st0, xb, 0);
        load_half(st1, xb, 1);
        const uint16_t *w0 = wptr(cur.m, 0);
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) load_w(ks, w0 + ks * 8 * FRAG);
        store_half(st0, 0, 0);
        store_half(st1, 0, 1);
    }
    lds_sync();
    read_x(xr[0], 0, 0);
    int buf = 0;

    while (true) {
        Task nxt = cur;
        int next_task = task;
        bool more = true;                                  // is there a block after the current one
        for (int i = 0; i < k; ++i) {
            // ---- the block after (cur, i): (cur, i + 1) or block 0 of the next task
            int ni = i + 1;
            if (ni == k) {
                next_task = task + per_wg;
                more = next_task < t_end;
                if (more) {
                    nxt = task_of(a, next_task);
                    set_rows(nxt);
                }
                ni = 0;
            }
            const uint16_t *nw = more ? wptr(nxt.m, ni) : wptr(cur.m, i);  // past the end: reload valid fragments
            // past the end of the stream the current block is loaded again (and never read)
            const uint16_t *nxb = more ? nxt.x + nxt.layers[ni] * nxt.s_layer : cur.x + cur.layers[i] * cur.s_layer;
            u32x4_t st0[HC], st1[HC];
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                // one step: the next block's rows requested (first step) or published (last two steps), the 16
                // MFMAs with the x reads of the following step interleaved, then the next block's W fragments of
                // this step into the registers just consumed.  In-order completion: a W fragment is waited for
                // one block after its request, and the only slower requests ahead of it (the x rows of its own
                // block) are complete by then.
                __builtin_amdgcn_sched_barrier(0);
                if (ks == 7) {
                    store_half(st1, buf ^ 1, 1);
                    lds_sync();
                }
                if (ks < 4) {
                    if (ks < 2) load_quarter(st0, nxb, ks);
                    else load_quarter(st1, nxb, ks);
                }
                if (ks == 6) store_half(st0, buf ^ 1, 0);
                // at the end of the stream the last read is of a buffer nobody uses any more
                read_x(xr[(ks + 1) & 1], ks < 7 ? buf : buf ^ 1, (ks + 1) & 7);
                const bf16x8_t *x = xr[ks & 1];
#pragma unroll
                for (int s = 0; s < 8; ++s) acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wh[ks], x[s], acc[s], 0, 0, 0);
#pragma unroll
                for (int s = 0; s < 8; ++s) acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wl[ks], x[s], acc[s], 0, 0, 0);
                load_w(ks, nw + ks * 8 * FRAG);
                if (ks < 4) __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);     // x rows of the next block
                if (ks == 6) __builtin_amdgcn_sched_group_barrier(0x200, 8, 0);
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);                 // W of the next block
            }
            buf ^= 1;
        }

        // ---- epilogue of the task: bias, one rounding, 16-byte stores of target rows
        // D[i][t]: t = lane & 31, channel 32 wave + 8 (v / 4) + 4 (lane / 32) + (v & 3)
        {
            const ApplyMultiMap mp = a.maps[cur.m];
            constexpr bool PERM = RS == 1;
            const bool rotate = RS != 0 && mp.kv == 0;
            float bias[16];
#pragma unroll
            for (int v = 0; v < 16; ++v)
                bias[v] = a.bias[(int64_t)cur.m * 128 + frag_channel(wave, 8 * (v >> 2) + 4 * lhalf + (v & 3), PERM)];
            uint16_t *obase = a.out + mp.tgt_layer * a.os.layer + mp.kv * a.os.kv + mp.tgt_head * a.os.head;
            const int oc0 = frag_channel(wave, 8 * lhalf, PERM), oc1 = frag_channel(wave, 16 + 8 * lhalf, PERM);
            // (cos, sin) of the lane's eight pairs at token 32 s + lane mod 32 of the tile,
            // loaded one token group ahead of their use
            auto tok_of = [&](int s) {
                const int64_t n = cur.tok0 + 32 * s + (int64_t)lrow;
                return n < a.N ? n : a.N - 1;
            };
            auto cs_load = [&](float4 (&cs)[4], int s) __attribute__((always_inline)) {
                const int64_t nc = tok_of(s);
                const uint32_t tk = (uint32_t)nc - fastdiv_u((uint32_t)nc, a.T) * a.T.d;
                const float *row = a.rope_table + (int64_t)(a.rope_pos_offset + (int)tk) * 128;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    // half split: frequencies 16 w + 8 (g / 2) + 4 lhalf + 2 (g % 2) + {0, 1}
                    // interleaved: frequencies 16 w + 4 g + 2 lhalf + {0, 1}
                    const int f = RS == 1 ? 16 * wave + 8 * (g >> 1) + 4 * lhalf + 2 * (g & 1)
                                          : 16 * wave + 4 * g + 2 * lhalf;
                    cs[g] = *reinterpret_cast<const float4 *>(row + 2 * f);
                }
            };
            float4 csn[4];
            if (RS != 0 && rotate) cs_load(csn, 0);
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const int64_t n = cur.tok0 + 32 * s + (int64_t)lrow;
                const int64_t nc = tok_of(s);
                const uint32_t seq = fastdiv_u((uint32_t)nc, a.T);
                const uint32_t tk = (uint32_t)nc - seq * a.T.d;
                float o[16];
#pragma unroll
                for (int v = 0; v < 16; ++v) o[v] = acc[s][v] + bias[v];
                if (RS != 0 && rotate) {
                    float4 cs[4];
#pragma unroll
                    for (int g = 0; g < 4; ++g) cs[g] = csn[g];
                    if (s < 7) cs_load(csn, s + 1);
                    if constexpr (RS == 1) {
#pragma unroll
                        for (int v = 0; v < 8; ++v) {          // pair (v, v + 8): channels c and c + 64
                            const float4 q = cs[2 * (v >> 2) + ((v & 3) >> 1)];
                            const float c = (v & 1) ? q.z : q.x, sn = (v & 1) ? q.w : q.y;
                            const float x0 = o[v], x1 = o[v + 8];
                            o[v] = __builtin_fmaf(x0, c, -x1 * sn);
                            o[v + 8] = __builtin_fmaf(x1, c, x0 * sn);
                        }
                    } else {
#pragma unroll
                        for (int v = 0; v < 16; v += 2) {      // pair (v, v + 1): channels 2f and 2f + 1
                            const float4 q = cs[v >> 2];
                            const float c = (v & 2) ? q.z : q.x, sn = (v & 2) ? q.w : q.y;
                            const float x0 = o[v], x1 = o[v + 1];
                            o[v] = __builtin_fmaf(x0, c, -x1 * sn);
                            o[v + 1] = __builtin_fmaf(x1, c, x0 * sn);
                        }
                    }
                }
                uint32_t pk[8];
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    pk[2 * gq] = pack_bf16(o[4 * gq + 0], o[4 * gq + 1]);
                    pk[2 * gq + 1] = pack_bf16(o[4 * gq + 2], o[4 * gq + 3]);
                }
                uint4 ov[2];
                exchange32(pk, ov);
                if (n < a.N) {
                    uint16_t *orow = obase + (int64_t)seq * a.os.seq + (int64_t)tk * a.os.tok;
                    *reinterpret_cast<uint4 *>(orow + oc0) = ov[0];
                    *reinterpret_cast<uint4 *>(orow + oc1) = ov[1];
                }
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[s][v] = 0.f;
            }
        }
        if (!more) break;
        cur = nxt;
        task = next_task;
    }
}


// ---------------------------------------------------------------------------
// The paired form.  A task is (pair of maps, tile of 256 tokens); the two maps
// of a pair read the same k source blocks (one (kv, head) of the sender, the
// same set of layers), so each block is staged once for both: half the staged
// source rows per output.  At k = 8 with L_t > L_s many neighbouring target
// layers select the same source layers.  The pair's record holds its blocks in
// ascending layer order with each map's block index i for them.  Maps without
// such a partner run in apply_multi_kernel.
//
// Four waves, one per SIMD.  Wave w owns output channels 32 w .. 32 w + 31 of
// both maps: sixteen 32 x 32 accumulator tiles (256 registers), so each x
// fragment read from LDS feeds four MFMAs (A hi, B hi, A lo, B lo).  Staged
// blocks move HBM -> LDS with global_load_lds_dwordx4 (no register staging),
// one block ahead through two 64 KiB buffers; each map's W^T fragments run four
// K steps ahead through a ring of four register slots, across blocks and tasks.
typedef __attribute__((address_space(3))) char lds_char_t;
typedef __attribute__((address_space(3))) bf16x8_t lds_bf16x8_t;

constexpr int PG = 4;                   // pairs per tile-major group of the task order

// The pair records are written before the launch and never during it, so they are read through the
// constant address space (scalar loads).
typedef const __attribute__((address_space(4))) int32_t *crec_t;

struct PairTask {
    int32_t mA, mB;
    crec_t rec;                         // the pair's record
    int64_t tok0;
    const uint16_t *x;                  // source view of the pair's (kv, head), layer 0
    int64_t s_layer, s_seq, s_tok;
};

__device__ __forceinline__ PairTask pair_task(const ApplyMultiArgs &a, int task) {
    const int full = a.n_pairs & ~(PG - 1);
    const int in_full = full * a.n_tiles;
    int tile, p;
    if (task < in_full) {
        const int per = PG * a.n_tiles;
        const int g = task / per, r = task - g * per;
        tile = r / PG;
        p = PG * g + (r - tile * PG);
    } else {
        const int rem = a.n_pairs - full;
        const int r = task - in_full;
        tile = r / rem;
        p = full + (r - tile * rem);
    }
    PairTask t;
    t.rec = (crec_t)(a.pairs + (int64_t)p * a.pair_stride);
    t.mA = __builtin_amdgcn_readfirstlane(t.rec[0]);
    t.mB = __builtin_amdgcn_readfirstlane(t.rec[1]);
    t.tok0 = (int64_t)tile * TT;
    const crec_t mp = (crec_t)(a.maps + t.mA);            // tgt_layer, tgt_head, kv, src_head
    const int kv = mp[2], src_head = mp[3];
    const bool kview = kv == 0 && a.srck != nullptr;
    const Strides &v = kview ? a.ssk : a.ss;
    t.x = kview ? a.srck + src_head * v.head : a.src + kv * v.kv + src_head * v.head;
    t.s_layer = v.layer;
    t.s_seq = v.seq;
    t.s_tok = v.tok;
    return t;
}

// Eight 16-byte copies global -> LDS under one save of M0: copy j reads
// base + off[J + j] per lane and writes lane l's chunk at m0 + 1024 j + 16 l.
// The compiler does not count these loads in its own vmcnt waits.
template <int J>
__device__ __forceinline__ void dma8(const uint32_t (&off)[16], const void *base, uint32_t m0) {
    uint32_t keep_m0;
    asm volatile("s_mov_b32 %[km], m0\n\ts_mov_b32 m0, %[m0]\n\t"
                 "global_load_lds_dwordx4 %[v0], %[sb]\n\ts_add_u32 m0, m0, 0x400\n\t"
                 "global_load_lds_dwordx4 %[v1], %[sb]\n\ts_add_u32 m0, m0, 0x400\n\t"
                 "global_load_lds_dwordx4 %[v2], %[sb]\n\ts_add_u32 m0, m0, 0x400\n\t"
                 "global_load_lds_dwordx4 %[v3], %[sb]\n\ts_add_u32 m0, m0, 0x400\n\t"
                 "global_load_lds_dwordx4 %[v4], %[sb]\n\ts_add_u32 m0, m0, 0x400\n\t"
                 "global_load_lds_dwordx4 %[v5], %[sb]\n\ts_add_u32 m0, m0, 0x400\n\t"
                 "global_load_lds_dwordx4 %[v6], %[sb]\n\ts_add_u32 m0, m0, 0x400\n\t"
                 "global_load_lds_dwordx4 %[v7], %[sb]\n\t"
                 "s_mov_b32 m0, %[km]"
                 : [km] "=&s"(keep_m0)
                 : [m0] "s"(m0), [sb] "s"(base), [v0] "v"(off[J + 0]), [v1] "v"(off[J + 1]), [v2] "v"(off[J + 2]),
                   [v3] "v"(off[J + 3]), [v4] "v"(off[J + 4]), [v5] "v"(off[J + 5]), [v6] "v"(off[J + 6]),
                   [v7] "v"(off[J + 7])
                 : "memory", "scc");
}

__device__ __forceinline__ void dma2(uint32_t off0, uint32_t off1, const void *base, uint32_t m0) {
    uint32_t keep_m0;
    asm volatile("s_mov_b32 %[km], m0\n\ts_mov_b32 m0, %[m0]\n\t"
                 "global_load_lds_dwordx4 %[v0], %[sb]\n\ts_add_u32 m0, m0, 0x400\n\t"
                 "global_load_lds_dwordx4 %[v1], %[sb]\n\t"
                 "s_mov_b32 m0, %[km]"
                 : [km] "=&s"(keep_m0)
                 : [m0] "s"(m0), [sb] "s"(base), [v0] "v"(off0), [v1] "v"(off1)
                 : "memory", "scc");
}

template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// A copy of a per-lane value that the compiler cannot see through: values derived from it are rebuilt where
// they are used instead of being held in registers (or spilled) across the whole kernel.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
    asm volatile("" : "+v"(v));
    return v;
}

// RS: target rotation of the K outputs, 0 none, 1 pairs (i, i + 64), 2 pairs (2i, 2i + 1).
template <int RS>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void apply_pair_kernel(ApplyMultiArgs a) {
    __shared__ __attribute__((aligned(16))) char lds_raw[2 * BUFB + 256 * 64];
    lds_char_t *lds = (lds_char_t *)lds_raw;
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int per_wg = gridDim.x >> 3;                    // workgroups per XCD (the grid is a multiple of 8)
    const int t_end = min(xcd * a.per_xcd + a.per_xcd, a.n_tasks);
    int task = xcd * a.per_xcd + slot;
    if (task >= t_end) return;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int k = a.k;
    constexpr int RING = 4;                               // K steps of W^T fragments held ahead
    const uint32_t lrow = lane & 31, lhalf = lane >> 5;

    // ---- copies: instruction i (0..15) of wave w moves token rows 64 w + 4 i + lane / 16; lane l writes LDS
    // position l mod 16 of its row, which holds chunk (l mod 16) ^ (row mod 16) of the row.  The lane's 16
    // source offsets of the copy cursor's task are kept in LDS (its own 64 bytes), not in registers.
    lds_char_t *coff_lds = lds + 2 * BUFB + tid * 64;
    auto set_rows = [&](const PairTask &t) {
        uint32_t o[16];
        const uint32_t ln = opaque((uint32_t)lane);        // (see opaque)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            int64_t n = t.tok0 + (int64_t)(64 * wave + 4 * i + (ln >> 4));
            if (n >= a.N) n = a.N - 1;                    // rows past the end repeat the last token
            const uint32_t seq = fastdiv_u((uint32_t)n, a.T);
            const uint32_t tk = (uint32_t)n - seq * a.T.d;
            const uint32_t r16 = (uint32_t)((4 * i + (ln >> 4)) & 15);
            o[i] = (uint32_t)(2 * ((int64_t)seq * t.s_seq + (int64_t)tk * t.s_tok)) + 16u * ((ln & 15) ^ r16);
        }
#pragma unroll
        for (int i = 0; i < 16; i += 4)
            *(__attribute__((address_space(3))) u32x4_t *)(coff_lds + 4 * i) = u32x4_t{o[i], o[i + 1], o[i + 2], o[i + 3]};
    };
    const uint32_t m0w = (uint32_t)(uintptr_t)lds + (uint32_t)(64 * wave * ROWB);
    PairTask C = pair_task(a, task);                      // the copy cursor: task ctask, staged block cu
    int ctask = task, cu = 0;
    bool cvalid = true;
    set_rows(C);
    auto issue = [&](int b) {
        const int layer = C.rec[4 + cu];
        const uint16_t *base = C.x + (int64_t)layer * C.s_layer;
        uint32_t coff[16];
        uint32_t cbase = (uint32_t)(uintptr_t)coff_lds;
        asm volatile("" : "+v"(cbase));                   // one address register, small constant offsets
#pragma unroll
        for (int i = 0; i < 16; i += 4) {
            const u32x4_t v = *(const __attribute__((address_space(3))) u32x4_t *)(uintptr_t)(cbase + 4 * i);
            coff[i] = v[0];
            coff[i + 1] = v[1];
            coff[i + 2] = v[2];
            coff[i + 3] = v[3];
        }
        dma8<0>(coff, base, m0w + b * BUFB);
        dma8<8>(coff, base, m0w + b * BUFB + 8 * 1024);
    };
    // the same copies in eight pairs, spread over a step's products; each pair's offsets read from LDS
    const uint16_t *pbase = a.wfrag;
    auto prep = [&]() {
        const int layer = C.rec[4 + cu];
        pbase = C.x + (int64_t)layer * C.s_layer;
    };
    auto pair_copy = [&](int j, uint32_t m0) __attribute__((always_inline)) {
        uint32_t cbase = (uint32_t)(uintptr_t)coff_lds;
        asm volatile("" : "+v"(cbase));
        typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;
        const u32x2_t v = *(const __attribute__((address_space(3))) u32x2_t *)(uintptr_t)(cbase + 4 * j);
        dma2(v[0], v[1], pbase, m0);
    };
    auto advance = [&]() {
        if (++cu == k) {
            ctask += per_wg;
            cu = 0;
            cvalid = ctask < t_end;
            if (cvalid) {
                C = pair_task(a, ctask);
                set_rows(C);
            }
        }
    };

    // ---- operands.  The lane's LDS read offsets are rebuilt in every block from an opaque copy of the lane
    // index, so that they are not held in registers across the whole loop.
    uint32_t lrow_b = lrow, lhalf_b = lhalf;
    auto read_x = [&](bf16x8_t &x, int b, int ks, int s) __attribute__((always_inline)) {
        x = *(const lds_bf16x8_t *)(lds + b * BUFB + (s * 32 + (int)lrow_b) * ROWB +
                                    (int)(((2 * ks + lhalf_b) ^ (lrow_b & 15)) * 16));
    };
    auto wptr = [&](int m, int i) {
        return a.wfrag + ((int64_t)m * k + i) * WBLK + wave * (2 * FRAG) + opaque((uint32_t)lane) * 8;
    };
    bf16x8_t whA[RING], wlA[RING], whB[RING], wlB[RING];
    f32x16_t accA[8], accB[8];

    // ---- epilogue of a task: bias, the K outputs' rotation, one rounding, 16-byte stores of target rows.
    // D[i][t]: t = lane & 31, channel 32 wave + 8 (v / 4) + 4 (lane / 32) + (v & 3).  Every load of the
    // epilogue (both maps' bias, the (cos, sin) of the tile's positions, which the two maps share) is issued
    // before its first store: a load issued after a store is waited for only once that store has completed
    // (loads and stores complete in order).
    constexpr bool PERM = RS == 1;
    auto epilogue = [&](const PairTask &t) __attribute__((always_inline)) {
        // the lane's row and half, rebuilt here (see opaque)
        const uint32_t ln = opaque((uint32_t)lane), lr = ln & 31, lh = ln >> 5;
        const int64_t tok0 = t.tok0;
        const crec_t mra = (crec_t)(a.maps + t.mA), mrb = (crec_t)(a.maps + t.mB);
        const bool rotate = RS != 0 && mra[2] == 0;           // both maps of a pair have the same kv
        float bias[2][16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int c = frag_channel(wave, 8 * (v >> 2) + 4 * lh + (v & 3), PERM);
            bias[0][v] = a.bias[(int64_t)t.mA * 128 + c];
            bias[1][v] = a.bias[(int64_t)t.mB * 128 + c];
        }
        auto tok_of = [&](int s) {
            const int64_t n = tok0 + (int64_t)(32 * s + lr);
            return n < a.N ? n : a.N - 1;
        };
        // (cos, sin) of the lane's eight pairs at token 32 s + lane mod 32 of the tile
        float4 csa[8][4];
        if (RS != 0 && rotate) {
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const int64_t nc = tok_of(s);
                const uint32_t tk = (uint32_t)nc - fastdiv_u((uint32_t)nc, a.T) * a.T.d;
                const float *row = a.rope_table + (int64_t)(a.rope_pos_offset + (int)tk) * 128;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    // half split: frequencies 16 w + 8 (g / 2) + 4 lh + 2 (g % 2) + {0, 1}
                    // interleaved: frequencies 16 w + 4 g + 2 lh + {0, 1}
                    const int f = RS == 1 ? 16 * wave + 8 * (g >> 1) + 4 * lh + 2 * (g & 1) : 16 * wave + 4 * g + 2 * lh;
                    csa[s][g] = *reinterpret_cast<const float4 *>(row + 2 * f);
                }
            }
        }
        const int oc0 = frag_channel(wave, 8 * lh, PERM), oc1 = frag_channel(wave, 16 + 8 * lh, PERM);
#pragma unroll
        for (int mi = 0; mi < 2; ++mi) {
            const crec_t mr = mi == 0 ? mra : mrb;          // tgt_layer, tgt_head, kv, src_head
            uint16_t *obase = a.out + mr[0] * a.os.layer + mr[2] * a.os.kv + mr[1] * a.os.head;
            const f32x16_t(&acc)[8] = mi == 0 ? accA : accB;
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                // one token group at a time: its accumulators are read only here
                __builtin_amdgcn_sched_barrier(0);
                const int64_t n = tok0 + (int64_t)(32 * s + lr);
                const int64_t nc = tok_of(s);
                const uint32_t seq = fastdiv_u((uint32_t)nc, a.T);
                const uint32_t tk = (uint32_t)nc - seq * a.T.d;
                float o[16];
#pragma unroll
                for (int v = 0; v < 16; ++v) o[v] = acc[s][v] + bias[mi][v];
                if (RS != 0 && rotate) {
                    const float4(&cs)[4] = csa[s];
                    if constexpr (RS == 1) {
#pragma unroll
                        for (int v = 0; v < 8; ++v) {      // pair (v, v + 8): channels c and c + 64
                            const float4 q = cs[2 * (v >> 2) + ((v & 3) >> 1)];
                            const float c = (v & 1) ? q.z : q.x, sn = (v & 1) ? q.w : q.y;
                            const float x0 = o[v], x1 = o[v + 8];
                            o[v] = __builtin_fmaf(x0, c, -x1 * sn);
                            o[v + 8] = __builtin_fmaf(x1, c, x0 * sn);
                        }
                    } else {
#pragma unroll
                        for (int v = 0; v < 16; v += 2) {  // pair (v, v + 1): channels 2f and 2f + 1
                            const float4 q = cs[v >> 2];
                            const float c = (v & 2) ? q.z : q.x, sn = (v & 2) ? q.w : q.y;
                            const float x0 = o[v], x1 = o[v + 1];
                            o[v] = __builtin_fmaf(x0, c, -x1 * sn);
                            o[v + 1] = __builtin_fmaf(x1, c, x0 * sn);
                        }
                    }
                }
                uint32_t pk[8];
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    pk[2 * gq] = pack_bf16(o[4 * gq + 0], o[4 * gq + 1]);
                    pk[2 * gq + 1] = pack_bf16(o[4 * gq + 2], o[4 * gq + 3]);
                }
                uint4 ov[2];
                exchange32(pk, ov);
                if (n < a.N) {
                    uint16_t *orow = obase + (int64_t)seq * a.os.seq + (int64_t)tk * a.os.tok;
                    *reinterpret_cast<uint4 *>(orow + oc0) = ov[0];
                    *reinterpret_cast<uint4 *>(orow + oc1) = ov[1];
                }
            }
        }
    };

    // ---- prologue: the first staged block in buffer 0
    issue(0);
    advance();
    PairTask T = pair_task(a, task);
    wait_vm<0>();
    lds_sync();

    // the first K steps of both maps' fragments.  Without the rotation the ring runs ahead across blocks and
    // tasks; with it the rotation's epilogue needs the registers, and each task loads its first steps anew.
    constexpr bool CARRY = RS == 0;
    auto first_steps = [&](const PairTask &t) {
        const uint16_t *pa = wptr(t.mA, t.rec[4 + k]);
        const uint16_t *pb = wptr(t.mB, t.rec[4 + 2 * k]);
#pragma unroll
        for (int r = 0; r < RING; ++r) {
            whA[r] = *reinterpret_cast<const bf16x8_t *>(pa + r * 8 * FRAG);
            wlA[r] = *reinterpret_cast<const bf16x8_t *>(pa + r * 8 * FRAG + FRAG);
            whB[r] = *reinterpret_cast<const bf16x8_t *>(pb + r * 8 * FRAG);
            wlB[r] = *reinterpret_cast<const bf16x8_t *>(pb + r * 8 * FRAG + FRAG);
        }
    };
    if constexpr (CARRY) first_steps(T);
    bool has_next = task + per_wg < t_end;
    PairTask NT = T;
    if (has_next) NT = pair_task(a, task + per_wg);
    int buf = 0;
    while (true) {
        if constexpr (!CARRY) first_steps(T);
        // the task's accumulators live only from here to its epilogue; zeroed by products of zeros so that
        // they are born in the accumulation registers
        {
            const bf16x8_t z8 = {};
            const f32x16_t z16 = {};
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                accA[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(z8, z8, z16, 0, 0, 0);
                accB[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(z8, z8, z16, 0, 0, 0);
            }
        }
        for (int u = 0; u < k; ++u) {
            // this block's fragments, requested during the last block (or at the task's start), are waited
            // for before the copies: the compiler's own waits do not count the copies, so a wait for a load
            // issued before them, placed after them, would also wait for the copies
            asm volatile("" ::"v"(whA[0]), "v"(wlA[0]), "v"(whB[0]), "v"(wlB[0]), "v"(whA[1]), "v"(wlA[1]),
                         "v"(whB[1]), "v"(wlB[1]), "v"(whA[2]), "v"(wlA[2]), "v"(whB[2]), "v"(wlB[2]),
                         "v"(whA[3]), "v"(wlA[3]), "v"(whB[3]), "v"(wlB[3]));
            // the block after this one goes, in eight pairs of copies spread over step 0's products, into
            // the other buffer, which every wave finished reading before the last barrier
            const bool issued = cvalid;
            if (cvalid) prep();
            const uint32_t pm0 = m0w + (buf ^ 1) * BUFB;
            // fragments: this block's, and the first steps of the next block (of this task, else of the next
            // task; past the last task, or with the rotation, this block's again, never used)
            const uint16_t *wcurA = wptr(T.mA, T.rec[4 + k + u]);
            const uint16_t *wcurB = wptr(T.mB, T.rec[4 + 2 * k + u]);
            const uint16_t *wnextA = wcurA, *wnextB = wcurB;
            if (u + 1 < k) {
                wnextA = wptr(T.mA, T.rec[4 + k + u + 1]);
                wnextB = wptr(T.mB, T.rec[4 + 2 * k + u + 1]);
            } else if (CARRY && has_next) {
                wnextA = wptr(NT.mA, NT.rec[4 + k]);
                wnextB = wptr(NT.mB, NT.rec[4 + 2 * k]);
            }
            // eight K steps; per x fragment A hi, B hi, A lo, B lo; after step ks each map refills its ring slot
            // ks mod 4 with step ks + 4 (this block's, or the next block's first four)
            lrow_b = lrow;
            lhalf_b = lhalf;
            asm volatile("" : "+v"(lrow_b), "+v"(lhalf_b));
            bf16x8_t xr[4];
            read_x(xr[0], buf, 0, 0);
            read_x(xr[1], buf, 0, 1);
            read_x(xr[2], buf, 0, 2);
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                const int r = ks % RING;
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int s = 0; s < 8; ++s) {
                    const int f = 8 * ks + s;
                    if (f + 3 < 64) read_x(xr[(f + 3) & 3], buf, (f + 3) >> 3, (f + 3) & 7);
                    const bf16x8_t x = xr[f & 3];
                    accA[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(whA[r], x, accA[s], 0, 0, 0);
                    accB[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(whB[r], x, accB[s], 0, 0, 0);
                    accA[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wlA[r], x, accA[s], 0, 0, 0);
                    accB[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wlB[r], x, accB[s], 0, 0, 0);
                    if (ks == 0 && issued) pair_copy(2 * s, pm0 + 2 * s * 1024);
                }
                {
                    const uint16_t *pa = ks + RING < 8 ? wcurA + (ks + RING) * 8 * FRAG : wnextA + (ks + RING - 8) * 8 * FRAG;
                    const uint16_t *pb = ks + RING < 8 ? wcurB + (ks + RING) * 8 * FRAG : wnextB + (ks + RING - 8) * 8 * FRAG;
                    whA[r] = *reinterpret_cast<const bf16x8_t *>(pa);
                    wlA[r] = *reinterpret_cast<const bf16x8_t *>(pa + FRAG);
                    whB[r] = *reinterpret_cast<const bf16x8_t *>(pb);
                    wlB[r] = *reinterpret_cast<const bf16x8_t *>(pb + FRAG);
                }
                // one x read ahead of each fragment's products, the ring loads after the step
#pragma unroll
                for (int s = 0; s < 8; ++s) {
                    if (8 * ks + s + 3 < 64) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
            if (issued) advance();                        // the copy cursor moves on (to the next task: its rows)
            // this wave's copies of the next block have landed (loads complete in order and this block's 32
            // ring loads were issued after them); the barrier publishes every wave's
            wait_vm<32>();
            lds_sync();
            buf ^= 1;
        }
        epilogue(T);
        if (!has_next) break;
        task += per_wg;
        T = NT;
        has_next = task + per_wg < t_end;
        if (has_next) NT = pair_task(a, task + per_wg);
    }
}

}  // namespace

hipError_t launch_split_maps_frag(int32_t n_maps, int32_t k, const float *maps, uint16_t *wfrag, float *bias,
                                  int perm, hipStream_t s) {
    const int64_t n = (int64_t)n_maps * k * 8 * 4 * 64;
    if (n == 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(split_maps_frag_kernel, dim3((unsigned)blocks), dim3(256), 0, s, n_maps, k, maps, wfrag, bias,
                       perm);
    return hipGetLastError();
}

hipError_t launch_apply_multi(const ApplyMultiArgs &a, int32_t n_cu, hipStream_t s) {
    if (a.n_tasks == 0) return hipSuccess;
    // one workgroup per compute unit, a multiple of 8 so every XCD gets the same count
    int per_xcd_wg = n_cu / 8 > 0 ? n_cu / 8 : 1;
    if (per_xcd_wg > a.per_xcd) per_xcd_wg = a.per_xcd;
    if (a.pairs) {
        if (!a.rope_table)
            hipLaunchKernelGGL(apply_pair_kernel<0>, dim3(8 * per_xcd_wg), dim3(256), 0, s, a);
        else if (a.rope_style == 0)
            hipLaunchKernelGGL(apply_pair_kernel<1>, dim3(8 * per_xcd_wg), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL(apply_pair_kernel<2>, dim3(8 * per_xcd_wg), dim3(256), 0, s, a);
        return hipGetLastError();
    }
    if (!a.rope_table)
        hipLaunchKernelGGL(apply_multi_kernel<0>, dim3(8 * per_xcd_wg), dim3(256), 0, s, a);
    else if (a.rope_style == 0)
        hipLaunchKernelGGL(apply_multi_kernel<1>, dim3(8 * per_xcd_wg), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(apply_multi_kernel<2>, dim3(8 * per_xcd_wg), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cb

// cb_apply_multi.hip -- online application of multi-layer maps (gfx950).
//
// CacheBridge Sec. 1 (online handoff) with the multi-layer feature of Sec. 3.2:
// map m reads the sender's rows of its k selected source layers and writes
//     out[t, :] = RNE_bf16( sum_i x_{i,t} W_{m,i} + b_m )
// where W_{m,i} is rows 128 i .. 128 i + 127 of the map.  The maps arrive
// split as W^T in two bf16 planes (hi = RNE(W), lo = RNE(W - hi)) and an fp32
// bias, as for the single-layer apply.
//
// One workgroup per (map, tile of 256 tokens), four waves; wave w owns output
// channels 32 w .. 32 w + 31.  For each of the k source blocks the tile's 256
// rows are copied HBM -> LDS (direct-to-LDS, 16-byte chunk c of token row t at
// position c ^ (t mod 16), double buffered: block i+1 streams in while block i
// is multiplied), the wave loads its W^T hi/lo fragments for the block from
// global memory, and accumulates D = W^T x^T (channels x tokens, K = the
// block's 128 channels) with v_mfma_f32_32x32x16_bf16, hi and lo products into
// the same fp32 accumulators.  Then the bias is added, the sum rounded once to
// bf16 and stored as 16-byte chunks of target rows.
//
// Workgroup order: maps in groups of four neighbouring target layers (same K/V
// component and head); within a group the tiles are visited token-tile first,
// so the four maps' W^T stays in L2 and their overlapping source windows
// share the staged rows.
#include "cb_internal.h"

namespace cb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

constexpr int TT = 256;                 // tokens per workgroup
constexpr int ROWB = 256;               // bytes per 128-channel row
constexpr int BUFB = TT * ROWB;         // one staged source block (64 KiB)
constexpr int CPW = BUFB / 1024 / 4;    // copy instructions per wave and block (16)

__device__ __forceinline__ uint32_t fastdiv_u(uint32_t n, const FastDiv &f) {
    const uint32_t t = __umulhi(n, f.m);
    return (t + ((n - t) >> f.sh1)) >> f.sh2;
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    f32x2_t v = {lo, hi};
    bf16x2_t p = __builtin_convertvector(v, bf16x2_t);
    return __builtin_bit_cast(uint32_t, p);
}

// HBM -> LDS copy of 16 bytes per lane to M0 + 16 lane; M0 restored inside.
__device__ __forceinline__ void dma16(const void *gaddr, uint32_t m0) {
    uint32_t keep;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(keep)
                 : "v"(gaddr), "s"(m0)
                 : "memory");
}

__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void apply_multi_kernel(ApplyMultiArgs a) {
    __shared__ __attribute__((aligned(16))) char lds[2 * BUFB];
    const int b = blockIdx.x;
    const int task = (b & 7) * a.per_xcd + (b >> 3);       // a contiguous run of tasks per XCD
    if (task >= a.n_tasks) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // task -> (group of maps, token tile, map in group)
    const int per_group = a.n_tiles * a.group;
    const int grp = task / per_group, rem = task - grp * per_group;
    const int tile = rem / a.group;
    const int gm = grp * a.group + rem % a.group;
    if (gm >= a.n_maps) return;
    const int m = a.order[gm];
    const ApplyMultiMap &mp = a.maps[m];
    const int k = a.k, Pm1 = 128 * k;
    const int64_t tok0 = (int64_t)tile * TT;

    // ---- copy geometry: instruction j of this wave covers token rows 4 c .. 4 c + 3, c = wave + 4 j
    const int ch = lane & 15;
    int64_t rowoff[CPW];                                  // element offset of the lane's token row in a block
    uint32_t cpos[CPW];                                   // source chunk of the lane (swizzled position ch)
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
        const int t = 4 * (wave + 4 * j) + (lane >> 4);
        int64_t n = tok0 + t;
        if (n >= a.N) n = a.N - 1;                        // rows past the end repeat the last token
        const uint32_t seq = fastdiv_u((uint32_t)n, a.T);
        const uint32_t tk = (uint32_t)n - seq * a.T.d;
        rowoff[j] = (int64_t)seq * a.ss.seq + (int64_t)tk * a.ss.tok;
        cpos[j] = (uint32_t)(ch ^ (t & 15)) * 8u;         // elements
    }
    const uint32_t lds_base = (uint32_t)(uintptr_t)lds;
    auto issue = [&](int i, int buf) {
        const int L = a.src_layers[(int64_t)m * k + i];
        const uint16_t *blk = a.src + L * a.ss.layer + mp.kv * a.ss.kv + mp.src_head * a.ss.head;
#pragma unroll
        for (int j = 0; j < CPW; ++j)
            dma16(blk + rowoff[j] + cpos[j],
                  __builtin_amdgcn_readfirstlane(lds_base + buf * BUFB + (wave + 4 * j) * 1024));
    };

    // ---- W^T fragments of this wave for block i: 8 K steps x (hi, lo)
    const int c = 32 * wave + (lane & 31);                // output channel of the A operand row
    const uint16_t *whi = a.w_hi + ((int64_t)m * a.d_t + c) * Pm1 + 8 * (lane >> 5);
    const uint16_t *wlo = a.w_lo + ((int64_t)m * a.d_t + c) * Pm1 + 8 * (lane >> 5);
    struct WF {
        bf16x8_t hi[8], lo[8];
    };
    auto load_w = [&](WF &f, int i) {
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            f.hi[ks] = *reinterpret_cast<const bf16x8_t *>(whi + 128 * i + 16 * ks);
            f.lo[ks] = *reinterpret_cast<const bf16x8_t *>(wlo + 128 * i + 16 * ks);
        }
    };

    f32x16_t acc[TT / 32];
#pragma unroll
    for (int s = 0; s < TT / 32; ++s)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[s][v] = 0.f;
    // B operand (x^T): lane holds token row 32 s + (lane & 31), channels 16 ks + 8 (lane >> 5) .. + 7
    const uint32_t lrow = lane & 31, lhalf = lane >> 5;
    auto compute = [&](const WF &f, int buf) {
        const char *B = lds + buf * BUFB;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            bf16x8_t x[TT / 32];
#pragma unroll
            for (int s = 0; s < TT / 32; ++s) {
                const uint32_t t = 32 * s + lrow;
                x[s] = *reinterpret_cast<const bf16x8_t *>(B + t * ROWB + (((2 * ks + lhalf) ^ (t & 15)) * 16));
            }
#pragma unroll
            for (int s = 0; s < TT / 32; ++s) acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.hi[ks], x[s], acc[s], 0, 0, 0);
#pragma unroll
            for (int s = 0; s < TT / 32; ++s) acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.lo[ks], x[s], acc[s], 0, 0, 0);
        }
    };

    // ---- blocks: i+1 streams in (copies and W fragments) while i is multiplied
    WF wa, wb;
    load_w(wa, 0);
    issue(0, 0);
    for (int i = 0; i < k; i += 2) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // block i (and its W) has landed
        __syncthreads();
        if (i + 1 < k) {
            load_w(wb, i + 1);
            issue(i + 1, 1);
        }
        compute(wa, 0);
        if (i + 1 < k) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            if (i + 2 < k) {
                load_w(wa, i + 2);
                issue(i + 2, 0);
            }
            compute(wb, 1);
        }
    }

    // ---- bias, one rounding, 16-byte stores of target rows
    // D[i][t]: t = lane & 31, channel 32 wave + 8 (v / 4) + 4 (lane / 32) + (v & 3)
    float bias[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) bias[v] = a.bias[(int64_t)m * a.d_t + 32 * wave + 8 * (v >> 2) + 4 * lhalf + (v & 3)];
    uint16_t *obase = a.out + mp.tgt_layer * a.os.layer + mp.kv * a.os.kv + mp.tgt_head * a.os.head + 32 * wave;
#pragma unroll
    for (int s = 0; s < TT / 32; ++s) {
        uint32_t pk[8];
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            pk[2 * gq] = pack_bf16(acc[s][4 * gq + 0] + bias[4 * gq + 0], acc[s][4 * gq + 1] + bias[4 * gq + 1]);
            pk[2 * gq + 1] = pack_bf16(acc[s][4 * gq + 2] + bias[4 * gq + 2], acc[s][4 * gq + 3] + bias[4 * gq + 3]);
        }
        // exchange with lane ^ 32 so that each lane owns 8 consecutive channels:
        // lanes < 32 get channels 0-7 and 16-23, lanes >= 32 get 8-15 and 24-31
        uint4 o[2];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const uint32_t s0 = lhalf ? pk[4 * p + 0] : pk[4 * p + 2];
            const uint32_t s1 = lhalf ? pk[4 * p + 1] : pk[4 * p + 3];
            const uint32_t r0 = (uint32_t)__shfl_xor((int)s0, 32);
            const uint32_t r1 = (uint32_t)__shfl_xor((int)s1, 32);
            o[p] = lhalf ? make_uint4(r0, r1, pk[4 * p + 2], pk[4 * p + 3])
                         : make_uint4(pk[4 * p + 0], pk[4 * p + 1], r0, r1);
        }
        const int64_t n = tok0 + 32 * s + (int64_t)lrow;
        if (n < a.N) {
            const uint32_t seq = fastdiv_u((uint32_t)n, a.T);
            const uint32_t tk = (uint32_t)n - seq * a.T.d;
            uint16_t *orow = obase + (int64_t)seq * a.os.seq + (int64_t)tk * a.os.tok + 8 * lhalf;
            *reinterpret_cast<uint4 *>(orow) = o[0];
            *reinterpret_cast<uint4 *>(orow + 16) = o[1];
        }
    }
}

}  // namespace

hipError_t launch_apply_multi(const ApplyMultiArgs &a, hipStream_t s) {
    if (a.n_tasks == 0) return hipSuccess;
    hipLaunchKernelGGL(apply_multi_kernel, dim3(8 * a.per_xcd), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cb

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
// apply_kernel: one workgroup per (source block, token tile).  The tile's
//   source rows are staged in LDS in 32-token sub-blocks (one 128-bit load per
//   thread, double buffered); wave (slot, rb) keeps its 32 rows of
//   W_hi^T / W_lo^T for its map in registers and computes the 32x32 output
//   tile D = W^T x^T with v_mfma_f32_32x32x16_bf16 (K = source channels),
//   adds the bias, rounds once to bf16 and stores 16-byte chunks of target
//   rows.  A source block shared by two target maps is read once.
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

template <int DS, int DT>
struct ACfg {
    static constexpr int KS = DS / 16;              // MFMA K steps over source channels
    static constexpr int RBT = DT / 32;             // 32-row blocks of target channels
    static constexpr int NW = 2 * RBT, NT = 64 * NW;
    static constexpr int SB = 32;                   // tokens per sub-block
    static constexpr int NCB = DS / 8;              // 16-byte blocks per source row
    static constexpr int ROWB = DS * 2;             // bytes per source row
    static constexpr int BUFB = SB * ROWB;          // bytes per sub-block buffer
    static constexpr int LOADS = SB * NCB;          // 16-byte loads per sub-block
    static constexpr int LPT = (LOADS + NT - 1) / NT;
};

// Rotated position of 16-byte block cb of token row t in LDS: 16 consecutive
// tokens reading the same block hit distinct banks (when NCB = 16).
template <int NCB>
__device__ __forceinline__ uint32_t xoff(uint32_t t, uint32_t cb) {
    return t * (NCB * 16) + ((cb + t) % NCB) * 16;
}

template <int DS, int DT>
__global__ __attribute__((amdgpu_flat_work_group_size(ACfg<DS, DT>::NT, ACfg<DS, DT>::NT),
                          amdgpu_waves_per_eu(2, 2)))
void apply_kernel(ApplyArgs a) {
    using K = ACfg<DS, DT>;
    __shared__ __attribute__((aligned(16))) char lds[2 * K::BUFB];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int slot = wave / K::RBT, rb = wave % K::RBT;
    const int g = blockIdx.x / a.n_tiles;
    const int tile = blockIdx.x % a.n_tiles;
    const ApplyGroup grp = a.groups[g];
    const bool active = slot < grp.n_slots;
    const int tok0 = tile * a.tile_tokens;
    const int tok1 = min(a.N, tok0 + a.tile_tokens);
    const int n_sb = (tok1 - tok0 + K::SB - 1) / K::SB;

    const uint16_t *xsrc = a.src + grp.src_layer * a.ss.layer + grp.kv * a.ss.kv + grp.src_head * a.ss.head;
    const int m = grp.map[slot < grp.n_slots ? slot : 0];
    uint16_t *obase = a.out + grp.tgt_layer[slot < grp.n_slots ? slot : 0] * a.os.layer + grp.kv * a.os.kv +
                      grp.tgt_head[slot < grp.n_slots ? slot : 0] * a.os.head + rb * 32;

    // coefficients of this wave's 32 target channels, kept in registers
    const uint32_t lrow = lane & 31, lhalf = lane >> 5;
    bf16x8_t ahi[K::KS], alo[K::KS];
    float bias[16];
    if (active) {
        const uint16_t *wh = a.w_hi + ((int64_t)m * DT + rb * 32 + lrow) * DS + 8 * lhalf;
        const uint16_t *wl = a.w_lo + ((int64_t)m * DT + rb * 32 + lrow) * DS + 8 * lhalf;
#pragma unroll
        for (int ks = 0; ks < K::KS; ++ks) {
            ahi[ks] = *reinterpret_cast<const bf16x8_t *>(wh + 16 * ks);
            alo[ks] = *reinterpret_cast<const bf16x8_t *>(wl + 16 * ks);
        }
        const float *bp = a.bias + (int64_t)m * DT + rb * 32 + 4 * lhalf;
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            const float4 b4 = *reinterpret_cast<const float4 *>(bp + 8 * gq);
            bias[4 * gq + 0] = b4.x;
            bias[4 * gq + 1] = b4.y;
            bias[4 * gq + 2] = b4.z;
            bias[4 * gq + 3] = b4.w;
        }
    }

    uint4 stage[K::LPT];
    auto load_sb = [&](int sb) {
        const int t0 = tok0 + sb * K::SB;
#pragma unroll
        for (int s = 0; s < K::LPT; ++s) {
            const int i = tid + s * K::NT;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (i < K::LOADS) {
                const int t = i / K::NCB, cb = i % K::NCB;
                const int tau = t0 + t;
                if (tau < tok1) {
                    const uint32_t b = fastdiv((uint32_t)tau, a.T);
                    const uint32_t tt = (uint32_t)tau - b * a.T.d;
                    v = *reinterpret_cast<const uint4 *>(xsrc + (int64_t)b * a.ss.seq + (int64_t)tt * a.ss.tok + cb * 8);
                }
            }
            stage[s] = v;
        }
    };
    auto store_sb = [&](int buf) {
        char *B = lds + buf * K::BUFB;
#pragma unroll
        for (int s = 0; s < K::LPT; ++s) {
            const int i = tid + s * K::NT;
            if (i < K::LOADS) {
                const int t = i / K::NCB, cb = i % K::NCB;
                *reinterpret_cast<uint4 *>(B + xoff<K::NCB>(t, cb)) = stage[s];
            }
        }
    };

    if (n_sb > 0) {
        load_sb(0);
        store_sb(0);
        lds_barrier();
        for (int sb = 0; sb < n_sb; ++sb) {
            if (sb + 1 < n_sb) load_sb(sb + 1);
            if (active) {
                const char *B = lds + (sb & 1) * K::BUFB;
                f32x16_t acc;
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
                for (int ks = 0; ks < K::KS; ++ks) {
                    const bf16x8_t bx = *reinterpret_cast<const bf16x8_t *>(B + xoff<K::NCB>(lrow, 2 * ks + lhalf));
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi[ks], bx, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo[ks], bx, acc, 0, 0, 0);
                }
                // D[i][t]: t = lane & 31, i = 8*(v/4) + 4*(lane/32) + (v&3)
                uint32_t pk[8];
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    pk[2 * gq] = pack_bf16(acc[4 * gq + 0] + bias[4 * gq + 0], acc[4 * gq + 1] + bias[4 * gq + 1]);
                    pk[2 * gq + 1] = pack_bf16(acc[4 * gq + 2] + bias[4 * gq + 2], acc[4 * gq + 3] + bias[4 * gq + 3]);
                }
                // Exchange with lane ^ 32 so that each lane owns 8 consecutive
                // channels: lanes < 32 get channels 0-7 and 16-23, lanes >= 32
                // get 8-15 and 24-31 of the 32-channel block.
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
                const int tau = tok0 + sb * K::SB + (int)lrow;
                if (tau < tok1) {
                    const uint32_t b = fastdiv((uint32_t)tau, a.T);
                    const uint32_t tt = (uint32_t)tau - b * a.T.d;
                    uint16_t *orow = obase + (int64_t)b * a.os.seq + (int64_t)tt * a.os.tok + 8 * lhalf;
                    *reinterpret_cast<uint4 *>(orow) = o[0];
                    *reinterpret_cast<uint4 *>(orow + 16) = o[1];
                }
            }
            if (sb + 1 < n_sb) store_sb((sb + 1) & 1);
            lds_barrier();
        }
    }
}

template <int DS, int DT>
hipError_t launch_apply_t(int n_groups, const ApplyArgs &a, hipStream_t s) {
    using K = ACfg<DS, DT>;
    const int64_t grid = (int64_t)n_groups * a.n_tiles;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL((apply_kernel<DS, DT>), dim3((unsigned)grid), dim3(K::NT), 0, s, a);
    return hipGetLastError();
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

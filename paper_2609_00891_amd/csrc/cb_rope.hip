// cb_rope.hip -- rotary position transform of cached keys on gfx950.
//
// CacheBridge Sec. 2.1 and Sec. 3.1: the maps act in content coordinates --
// source RoPE is removed from the keys before fitting and the target's RoPE
// is applied to the mapped keys, which makes the handed-off cache
// decode-ready.  With frequencies f_i = theta^(-2 i / d), i < d/2, the K row of
// position pos has its channel pairs (i, i + d/2) (half split) or (2i, 2i + 1)
// (interleaved) turned by the angle pos * f_i:
//     (a, b) -> (a cos - b sin, b cos + a sin),   the angle negated to invert.
//
// rope_table_kernel: (cos, sin) of pos * f_i for every position and
//   frequency, the angle and the sines in fp64 (positions in the tens of
//   thousands need the extra bits), stored as fp32.
// rope_kernel: one thread per (sequence, token, pair of 16-byte chunks) --
//   channels 8c .. 8c+7 and the chunk d/16 further on, which holds their
//   half-split partners -- and a group of 16 (layer, head) rows that share the
//   token's angles; fp32 products from the exact bf16 values and the fp32
//   table, one rounding to bf16.  V rows are copied when out is not in.
//   HBM-bound.  A position step other than one turns a strided selection of
//   tokens (every sample_stride-th, gathered into a compact copy).
#include "cb_internal.h"

namespace cb {
namespace {

typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    f32x2_t v = {lo, hi};
    bf16x2_t p = __builtin_convertvector(v, bf16x2_t);
    return __builtin_bit_cast(uint32_t, p);
}

__global__ __launch_bounds__(256) void rope_table_kernel(int d, int n_pos, double theta, float2 *__restrict__ table) {
    const int h = d / 2;
    const int64_t n = (int64_t)n_pos * h;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) {
        const int i = (int)(e % h);
        const double pos = (double)(e / h);
        const double ang = pos * pow(theta, -2.0 * i / (double)d);
        double s, c;
        sincos(ang, &s, &c);
        table[e] = make_float2((float)c, (float)s);
    }
}

struct RopeArgs {
    const uint16_t *in;
    uint16_t *out;
    Strides is, os;
    const float2 *table;      // [n_pos][d/2]
    int32_t n_layers, n_heads, n_seqs, seq_len, d, style, pos_offset, pos_step;
    float sign;               // +1 rotate, -1 de-rotate
    int32_t copy_v;           // out is not in: V rows are copied
};

// One thread per (sequence, token, chunk pair) and group of kRows (layer,
// head) rows: the token's table entries are loaded once and serve every row
// of the group, so the table costs a fraction of the cache traffic.
constexpr int kRows = 16;

__global__ __launch_bounds__(256) void rope_kernel(RopeArgs a) {
    const int NC2 = a.d / 16;                                // chunk pairs per row
    const int h = a.d / 2;
    const int LH = a.n_layers * a.n_heads;                   // (layer, head) rows per token and component
    const int n_rg = (LH + kRows - 1) / kRows;
    const int64_t n = (int64_t)a.n_seqs * a.seq_len * NC2 * n_rg;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) {
        const int c = (int)(e % NC2);
        int64_t r = e / NC2;
        const int t = (int)(r % a.seq_len);
        r /= a.seq_len;
        const int b = (int)(r % a.n_seqs);
        const int rg = (int)(r / a.n_seqs);
        // this token's angles for the thread's 8 channel pairs
        const float2 *cs = a.table + (int64_t)(a.pos_offset + (int64_t)t * a.pos_step) * h;
        float cw[8], sw[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int f = a.style == 0 ? 8 * c + q : (q < 4 ? 4 * c + q : 4 * (c + NC2) + q - 4);
            const float2 w = cs[f];
            cw[q] = w.x;
            sw[q] = a.sign * w.y;
        }
        const int lh1 = min(LH, (rg + 1) * kRows);
        for (int lh = rg * kRows; lh < lh1; ++lh) {
            const int l = lh / a.n_heads, g = lh - (lh / a.n_heads) * a.n_heads;
#pragma unroll
            for (int z = 0; z < 2; ++z) {
                if (z == 1 && !a.copy_v) continue;           // values carry no position
                const uint16_t *xr = a.in + l * a.is.layer + z * a.is.kv + b * a.is.seq + g * a.is.head + t * a.is.tok;
                uint16_t *yr = a.out + l * a.os.layer + z * a.os.kv + b * a.os.seq + g * a.os.head + t * a.os.tok;
                const uint4 p0 = *(const uint4 *)(xr + 8 * c);
                const uint4 p1 = *(const uint4 *)(xr + 8 * (c + NC2));
                if (z == 1) {
                    *(uint4 *)(yr + 8 * c) = p0;
                    *(uint4 *)(yr + 8 * (c + NC2)) = p1;
                    continue;
                }
                const uint32_t u0[4] = {p0.x, p0.y, p0.z, p0.w}, u1[4] = {p1.x, p1.y, p1.z, p1.w};
                uint32_t o0[4], o1[4];
                if (a.style == 0) {
                    // pairs (8c + k, 8c + k + d/2), frequency 8c + k
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float x0 = bf_lo(u0[q]), x1 = bf_hi(u0[q]), y0 = bf_lo(u1[q]), y1 = bf_hi(u1[q]);
                        const float c0 = cw[2 * q], c1 = cw[2 * q + 1], s0 = sw[2 * q], s1 = sw[2 * q + 1];
                        o0[q] = pack_bf16(__builtin_fmaf(x0, c0, -y0 * s0), __builtin_fmaf(x1, c1, -y1 * s1));
                        o1[q] = pack_bf16(__builtin_fmaf(y0, c0, x0 * s0), __builtin_fmaf(y1, c1, x1 * s1));
                    }
                } else {
                    // pairs (2i, 2i + 1) inside each chunk, frequency i
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float x0 = bf_lo(u0[q]), x1 = bf_hi(u0[q]), y0 = bf_lo(u1[q]), y1 = bf_hi(u1[q]);
                        const float c0 = cw[q], s0 = sw[q], c1 = cw[4 + q], s1 = sw[4 + q];
                        o0[q] = pack_bf16(__builtin_fmaf(x0, c0, -x1 * s0), __builtin_fmaf(x1, c0, x0 * s0));
                        o1[q] = pack_bf16(__builtin_fmaf(y0, c1, -y1 * s1), __builtin_fmaf(y1, c1, y0 * s1));
                    }
                }
                *(uint4 *)(yr + 8 * c) = make_uint4(o0[0], o0[1], o0[2], o0[3]);
                *(uint4 *)(yr + 8 * (c + NC2)) = make_uint4(o1[0], o1[1], o1[2], o1[3]);
            }
        }
    }
}

}  // namespace

hipError_t launch_rope_table(int32_t d, int32_t n_pos, double theta, float *table, hipStream_t s) {
    const int64_t n = (int64_t)n_pos * (d / 2);
    if (n == 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)blocks), dim3(256), 0, s, d, n_pos, theta, (float2 *)table);
    return hipGetLastError();
}

hipError_t launch_rope(const RopeLaunch &L, hipStream_t s) {
    RopeArgs a = {};
    a.in = L.in;
    a.out = L.out;
    a.is = L.is;
    a.os = L.os;
    a.table = (const float2 *)L.table;
    a.n_layers = L.n_layers;
    a.n_heads = L.n_heads;
    a.n_seqs = L.n_seqs;
    a.seq_len = L.seq_len;
    a.d = L.d;
    a.style = L.style;
    a.pos_offset = L.pos_offset;
    a.pos_step = L.pos_step > 0 ? L.pos_step : 1;
    a.sign = L.inverse ? -1.f : 1.f;
    a.copy_v = L.copy_v;
    const int64_t n_rg = ((int64_t)L.n_layers * L.n_heads + kRows - 1) / kRows;
    const int64_t n = (int64_t)L.n_seqs * L.seq_len * (L.d / 16) * n_rg;
    if (n == 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(rope_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cb

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
// stats_kernel (one workgroup of four waves per (item, tile chunk)):
//   * an item is one or two maps; two maps that read the same source block
//     load its rows once;
//   * token tiles stream HBM -> LDS by direct-to-LDS copies through a
//     four-stage ring (see the comment above Cfg);
//   * wave (slot, pair) runs on a SIMD of its own and owns one or two 32-row
//     blocks of one map: it folds the per-token weight into its x rows in
//     fp32, splits w*x into two bf16 terms (hi = RNE(w x), lo = RNE(w x - hi))
//     and runs v_mfma_f32_32x32x16_bf16 against the exact bf16 x and y
//     columns, accumulating in fp32.  Only one 32x32 tile of each pair of
//     mirrored Gram blocks is computed;
//   * the bias row/column (sum w, sum w x, sum w y) is summed on the VALU in
//     fp32 from the same operands;
//   * at the end of its chunk the workgroup writes its fp32 partial to the
//     plan's workspace (plain stores, no atomics).
// reduce_kernel (one workgroup per map) adds the partials of all chunks in a
// fixed order, mirrors the Gram block so G is exactly symmetric, and adds the
// result into the caller's G and C.
#include <algorithm>

#include "cb_stats_kernel.h"

namespace cb {
namespace {

// Block (a, b) of Gram tile slot k in the partial layout (pair 0's tiles,
// then pair 1's).
template <int RB>
__device__ __forceinline__ void gram_block(int k, int &a, int &b) {
    using O0 = Own<RB, 0>;
    using O1 = Own<RB, 1>;
    a = b = 0;
#pragma unroll
    for (int g = 0; g < O0::NG; ++g)
        if (k == g) { a = O0::row[O0::gr[g]]; b = O0::xc[O0::gx[g]]; }
#pragma unroll
    for (int g = 0; g < O1::NG; ++g)
        if (k == O0::NG + g) { a = O1::row[O1::gr[g]]; b = O1::xc[O1::gx[g]]; }
}

// One workgroup per (map, job): jobs 0 .. NTG-1 are the Gram tiles, NTG ..
// NTG+NTC-1 the cross tiles, the last one the bias sums.  A tile's partials
// are summed over the chunks in a fixed order (coalesced reads of the [v][lane]
// accumulator layout) and added into G / C; an off-diagonal Gram tile is also
// added, transposed through LDS, into the mirrored block, and a diagonal one
// only contributes its upper triangle (mirrored), so G is exactly symmetric.
//
// CENTER: the partials hold sum w u_i x_j and sum w u_i y_j with the folded
// operand u = x - mu_x, and the bias partials hold e = sum w u.  Subtracting
// e_i mu_j turns them into sum w u_i (x_j - mu_j), that is the centered
// moments A = sum w u u^T and B = sum w u (y - mu_y)^T of Sec. 3.4, written
// without a bias row or column ([d_s][d_s] and [d_s][d_t]).
template <int DS, int DT, bool CENTER>
__global__ __launch_bounds__(256) void reduce_kernel(ReduceArgs a) {
    using K = Cfg<DS, DT>;
    constexpr int P = DS + 1;
    constexpr int GS = CENTER ? DS : P;                       // row stride of the Gram output
    __shared__ float tile[32][33];
    __shared__ float ev[32], mv[32];
    const int m = blockIdx.x, job = blockIdx.y;
    const int tid = threadIdx.x;
    const int item = a.map_item[m], slot = a.map_slot[m];
    float *G = a.G + (int64_t)m * GS * GS;
    float *Cm = a.C + (int64_t)m * GS * DT;
    const int64_t chunk_stride = (int64_t)a.n_items * 2 * K::SLOT;
    const float *base = a.partials + ((int64_t)item * 2 + slot) * K::SLOT;

    if (job < K::NTG + K::NTC) {
        int ba, bb;                                           // folded row block, column block
        if (job >= K::NTG) {
            const int c = job - K::NTG;
            ba = c / K::RBT;
            bb = c - ba * K::RBT;
        } else {
            gram_block<K::RB>(job, ba, bb);
        }
        if constexpr (CENTER) {
            if (tid < 32) {
                float e = 0.f;
                for (int ch = 0; ch < a.n_chunks; ++ch) {
                    const float *pp = base + ch * chunk_stride + K::SUMX + ba * 64 + tid;
                    e += pp[0];
                    e += pp[32];
                }
                ev[tid] = e;
            } else if (tid < 64) {
                const double *sm = a.sums + (int64_t)m * (1 + DS + DT);
                const double sw = sm[0];
                const int ch = job >= K::NTG ? DS + 32 * bb + (tid - 32) : 32 * bb + (tid - 32);
                mv[tid - 32] = sw != 0.0 ? (float)(sm[1 + ch] / sw) : 0.f;
            }
        }
        float sum[4];
        int ii[4], jj[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int f = tid + 256 * q;                      // [v][lane] position in the tile
            const int v = f >> 6, l = f & 63;
            ii[q] = 8 * (v >> 2) + 4 * (l >> 5) + (v & 3);
            jj[q] = l & 31;
            float acc = 0.f;
            for (int ch = 0; ch < a.n_chunks; ++ch) acc += base[ch * chunk_stride + job * 1024 + f];
            sum[q] = acc;
        }
        if constexpr (CENTER) {
            __syncthreads();
#pragma unroll
            for (int q = 0; q < 4; ++q) sum[q] -= ev[ii[q]] * mv[jj[q]];
        }
        if (job >= K::NTG) {
#pragma unroll
            for (int q = 0; q < 4; ++q) Cm[(ba * 32 + ii[q]) * DT + bb * 32 + jj[q]] += sum[q];
            return;
        }
        if (ba == bb) {
            // upper triangle of the diagonal block and its mirror
#pragma unroll
            for (int q = 0; q < 4; ++q) tile[ii[q]][jj[q]] = sum[q];
            __syncthreads();
            for (int e = tid; e < 1024; e += 256) {
                const int i = e >> 5, j = e & 31;
                const float val = i <= j ? tile[i][j] : tile[j][i];
                G[(ba * 32 + i) * GS + ba * 32 + j] += val;
            }
            return;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            G[(ba * 32 + ii[q]) * GS + bb * 32 + jj[q]] += sum[q];
            tile[jj[q]][ii[q]] = sum[q];
        }
        __syncthreads();
        for (int e = tid; e < 1024; e += 256) {
            const int i = e >> 5, j = e & 31;               // row bb*32 + i, column ba*32 + j
            G[(bb * 32 + i) * GS + ba * 32 + j] += tile[i][j];
        }
        return;
    }
    if constexpr (CENTER) {
        // no bias row / column; the shifted form adds the batch's (sum w,
        // sum w (x - mu), sum w y) to resid, summed over the chunks in fp64
        if (!a.resid) return;
        double *rs = a.resid + (int64_t)m * (1 + DS + DT);
        for (int e = tid; e < DS + DT + 1; e += 256) {
            int i0;
            if (e == 0) i0 = K::SUMW;
            else if (e <= DS) i0 = K::SUMX + ((e - 1) >> 5) * 64 + ((e - 1) & 31);
            else i0 = K::SUMY + ((e - 1 - DS) >> 5) * 64 + ((e - 1 - DS) & 31);
            double acc = 0.0;
            for (int ch = 0; ch < a.n_chunks; ++ch) {
                const float *pp = base + ch * chunk_stride;
                acc += (double)pp[i0] + (double)pp[i0 + 32];
            }
            rs[e] += acc;
        }
        return;
    }

    // bias sums: row / column P-1 of G and row P-1 of C (two lane halves each)
    for (int e = tid; e < DS + DT + 1; e += 256) {
        int i0;
        if (e < DS) i0 = K::SUMX + (e >> 5) * 64 + (e & 31);
        else if (e < DS + DT) i0 = K::SUMY + ((e - DS) >> 5) * 64 + ((e - DS) & 31);
        else i0 = K::SUMW;
        float acc = 0.f;
        for (int ch = 0; ch < a.n_chunks; ++ch) {
            const float *pp = base + ch * chunk_stride;
            acc += pp[i0];
            acc += pp[i0 + 32];
        }
        if (e < DS) {
            G[(int64_t)(P - 1) * P + e] += acc;
            G[(int64_t)e * P + (P - 1)] += acc;
        } else if (e < DS + DT) {
            Cm[(int64_t)(P - 1) * DT + (e - DS)] += acc;
        } else {
            G[(int64_t)(P - 1) * P + (P - 1)] += acc;
        }
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
    if (a.seq_len % K::KT == 0)
        hipLaunchKernelGGL((stats_kernel<DS, DT, false, false>), dim3(grid), dim3(K::NT), 0, s, a);
    else
        hipLaunchKernelGGL((stats_kernel<DS, DT, true, false>), dim3(grid), dim3(K::NT), 0, s, a);
    return hipGetLastError();
}

template <int DS, int DT>
hipError_t launch_reduce_t(const ReduceArgs &a, hipStream_t s) {
    if (a.n_maps == 0) return hipSuccess;
    using K = Cfg<DS, DT>;
    hipLaunchKernelGGL((reduce_kernel<DS, DT, false>), dim3(a.n_maps, K::NTG + K::NTC + 1), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int DS, int DT>
hipError_t launch_reduce_centered_t(const ReduceArgs &a, hipStream_t s) {
    if (a.n_maps == 0) return hipSuccess;
    using K = Cfg<DS, DT>;
    hipLaunchKernelGGL((reduce_kernel<DS, DT, true>), dim3(a.n_maps, K::NTG + K::NTC + (a.resid ? 1 : 0)), dim3(256), 0,
                       s, a);
    return hipGetLastError();
}

// Shifted centered form, last step.  The moments were formed about the means
// mu' of `shift` (a pilot's sums), resid holds (S, e = sum w (x - mu'), sum w y)
// of all the data.  With delta = e / S = mu - mu' and mu_y = (sum w y) / S:
//     sum w (x - mu)(x - mu)^T = A' - S delta delta^T
//     sum w (x - mu)(y - mu_y)^T = B' - S delta (mu_y - mu'_y)^T
// (fp64, rounded once to fp32), then sum w x = e + S mu' replaces e.
__device__ __forceinline__ double mean_of(const double *sm, int i) { return sm[0] != 0.0 ? sm[1 + i] / sm[0] : 0.0; }

__global__ __launch_bounds__(256) void shift_moments_kernel(int32_t n_maps, int32_t d_x, int32_t d_t,
                                                            const double *__restrict__ shift,
                                                            const double *__restrict__ sums, float *__restrict__ A,
                                                            float *__restrict__ B) {
    const int64_t na = (int64_t)d_x * d_x, per = na + (int64_t)d_x * d_t, n = per * n_maps;
    for (int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x; g < n; g += (int64_t)gridDim.x * 256) {
        const int64_t m = g / per, e = g - m * per;
        const double *sh = shift + m * (1 + d_x + d_t);
        const double *su = sums + m * (1 + d_x + d_t);
        const double S = su[0];
        if (S == 0.0) continue;                               // no data: nothing to move
        if (e < na) {
            const int i = (int)(e / d_x), j = (int)(e - (int64_t)i * d_x);
            const double di = su[1 + i] / S, dj = su[1 + j] / S;
            float *p = A + m * na + e;
            *p = (float)((double)*p - S * (di * dj));           // the same value at (j, i): A stays symmetric
        } else {
            const int64_t f = e - na;
            const int i = (int)(f / d_t), j = (int)(f - (int64_t)i * d_t);
            const double di = su[1 + i] / S;
            const double dy = su[1 + d_x + j] / S - mean_of(sh, d_x + j);
            float *p = B + m * (int64_t)d_x * d_t + f;
            *p = (float)((double)*p - S * di * dy);
        }
    }
}

__global__ __launch_bounds__(256) void shift_sums_kernel(int32_t n_maps, int32_t d_x, int32_t d_t,
                                                         const double *__restrict__ shift, double *__restrict__ sums) {
    const int64_t n = (int64_t)n_maps * d_x;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) {
        const int64_t m = e / d_x;
        const int i = (int)(e - m * d_x);
        const double *sh = shift + m * (1 + d_x + d_t);
        double *su = sums + m * (1 + d_x + d_t);
        su[1 + i] += su[0] * mean_of(sh, i);
    }
}

}  // namespace

hipError_t launch_shift_finish(int32_t n_maps, int32_t d_x, int32_t d_t, const double *shift, double *sums, float *A,
                               float *B, hipStream_t s) {
    if (n_maps == 0) return hipSuccess;
    const int64_t tot = (int64_t)n_maps * d_x * (d_x + d_t);
    const unsigned bx = (unsigned)std::min<int64_t>((tot + 255) / 256, 16384);
    hipLaunchKernelGGL(shift_moments_kernel, dim3(bx), dim3(256), 0, s, n_maps, d_x, d_t, shift, sums, A, B);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)n_maps * d_x;
    const unsigned g = (unsigned)std::min<int64_t>((n + 255) / 256, 8192);
    hipLaunchKernelGGL(shift_sums_kernel, dim3(g), dim3(256), 0, s, n_maps, d_x, d_t, shift, sums);
    return hipGetLastError();
}

hipError_t launch_stats(int d_s, int d_t, const StatsArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_stats_t, d_s, d_t, a, s);
}

hipError_t launch_reduce(int d_s, int d_t, const ReduceArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_reduce_t, d_s, d_t, a, s);
}

hipError_t launch_reduce_centered(int d_s, int d_t, const ReduceArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_reduce_centered_t, d_s, d_t, a, s);
}

hipError_t launch_fill_zero(float *p, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

}  // namespace cb

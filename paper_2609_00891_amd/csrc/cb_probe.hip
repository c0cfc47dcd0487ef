// cb_probe.hip -- held-in R^2 of layer-selection probes on gfx950.
//
// CacheBridge Sec. 3.1 ranks the source layers of every target layer by the
// held-in R^2 of centered single-source-layer probes, averaged over KV heads
// and K/V.  The probes are ordinary maps of a plan whose head map pairs every
// target head with every candidate source layer; their statistics and solve
// are the centered ones.  With the probe's centered moments A, B, its fitted
// map [W ; b] (b = mu_y - W^T mu_x, so the residual has weighted mean zero),
// the weighted sums and the per-channel sums of squares,
//     TSS = sum_j (sum w y_j^2 - (sum w y_j)^2 / S),
//     RSS = TSS - 2 tr(W^T B) + tr(W^T A W),      R^2 = 1 - RSS / TSS,
// which needs no further pass over the tokens.
//
// probe_r2_kernel: one workgroup of 256 threads per map.  W and A are staged
// in LDS (fp32; A with a padded row stride so that the 32 rows read by a wave
// fall in different banks).  Thread (i, h) forms row i of A W over column
// half h in fp32 and its share of both traces in fp64; the workgroup adds the
// shares in a fixed order.
#include "cb_internal.h"

namespace cb {
namespace {

constexpr int kMaxD = 128;

__global__ __launch_bounds__(256) void probe_r2_kernel(int d_s, int d_t, const double *__restrict__ sums,
                                                       const double *__restrict__ sq, const float *__restrict__ A,
                                                       const float *__restrict__ B, const float *__restrict__ maps,
                                                       double *__restrict__ r2) {
    __shared__ __attribute__((aligned(16))) float Ws[kMaxD * kMaxD];       // W [d_s][d_t]
    __shared__ float As[kMaxD * (kMaxD + 1)];                              // A [d_s][d_s + 1]
    __shared__ double red[2][256 / 64];
    const int m = blockIdx.x, tid = threadIdx.x;
    const float *Am = A + (int64_t)m * d_s * d_s;
    const float *Bm = B + (int64_t)m * d_s * d_t;
    const float *Wm = maps + (int64_t)m * (d_s + 1) * d_t;                  // rows 0..d_s-1 = W
    const double *sm = sums + (int64_t)m * (1 + d_s + d_t);
    const double *qm = sq + (int64_t)m * (d_s + d_t);
    for (int e = tid; e < d_s * d_t; e += 256) Ws[e] = Wm[e];
    for (int e = tid; e < d_s * d_s; e += 256) As[(e / d_s) * (kMaxD + 1) + e % d_s] = Am[e];
    __syncthreads();

    // row i of A W over the column half h (d_t / 2 consecutive columns)
    const int i = tid >> 1, h = tid & 1, half = d_t / 2, j0 = h * half;
    double t1 = 0.0, t2 = 0.0;                                             // tr(W^T B), tr(W^T A W) shares
    if (i < d_s) {
        float aw[kMaxD / 2];
#pragma unroll
        for (int q = 0; q < kMaxD / 2; ++q) aw[q] = 0.f;
        for (int k = 0; k < d_s; ++k) {
            const float a = As[i * (kMaxD + 1) + k];
            const float4 *wr = (const float4 *)(Ws + k * d_t + j0);
#pragma unroll
            for (int q4 = 0; q4 < kMaxD / 8; ++q4) {
                if (4 * q4 < half) {
                    const float4 w = wr[q4];
                    aw[4 * q4] = __builtin_fmaf(a, w.x, aw[4 * q4]);
                    aw[4 * q4 + 1] = __builtin_fmaf(a, w.y, aw[4 * q4 + 1]);
                    aw[4 * q4 + 2] = __builtin_fmaf(a, w.z, aw[4 * q4 + 2]);
                    aw[4 * q4 + 3] = __builtin_fmaf(a, w.w, aw[4 * q4 + 3]);
                }
            }
        }
#pragma unroll
        for (int q = 0; q < kMaxD / 2; ++q) {
            if (q < half) {
                const double w = Ws[i * d_t + j0 + q];
                t1 += w * (double)Bm[(int64_t)i * d_t + j0 + q];
                t2 += w * (double)aw[q];
            }
        }
    }
    // fixed-order block sums (wave shuffles, then one value per wave)
    for (int o = 32; o > 0; o >>= 1) {
        t1 += __shfl_xor(t1, o);
        t2 += __shfl_xor(t2, o);
    }
    if ((tid & 63) == 0) {
        red[0][tid >> 6] = t1;
        red[1][tid >> 6] = t2;
    }
    __syncthreads();
    if (tid == 0) {
        double tr1 = 0.0, tr2 = 0.0;
        for (int w = 0; w < 256 / 64; ++w) {
            tr1 += red[0][w];
            tr2 += red[1][w];
        }
        const double S = sm[0];
        double tss = 0.0;
        if (S != 0.0)
            for (int j = 0; j < d_t; ++j) tss += qm[d_s + j] - sm[1 + d_s + j] * (sm[1 + d_s + j] / S);
        r2[m] = tss > 0.0 ? 1.0 - (tss - 2.0 * tr1 + tr2) / tss : 0.0;
    }
}

}  // namespace

hipError_t launch_probe_r2(int32_t n_maps, int32_t d_s, int32_t d_t, const double *sums, const double *sq,
                           const float *A, const float *B, const float *maps, double *r2, hipStream_t s) {
    if (n_maps == 0) return hipSuccess;
    if (d_s > kMaxD || d_t > kMaxD || d_t % 8 != 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL(probe_r2_kernel, dim3(n_maps), dim3(256), 0, s, d_s, d_t, sums, sq, A, B, maps, r2);
    return hipGetLastError();
}

}  // namespace cb

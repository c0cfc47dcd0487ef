// cb_solve.hip -- batched ridge solve, one workgroup per system (gfx950).
//
// CacheBridge Sec. 3.1 (Eq. closedform) and Sec. 3.4: the maps are the ridge
// solutions W~ = (G + lambda D)^{-1} C of the augmented moments.  For each map
// the workgroup
//   1. copies the lower triangle of G into LDS as packed fp64 and adds
//      lambda_m on the diagonal (lambda_m = lambda or lambda * tr(G) / P;
//      the last diagonal entry is skipped when the bias is not penalized),
//   2. factors M = L L^T column by column (left-looking; two lanes per row
//      share each dot product, one barrier per phase),
//   3. solves L Z = C and L^T W~ = Z on 64-column panels of C held in LDS as
//      fp64, four lanes per column,
//   4. writes W~ in fp32 and the per-map status info (0, or the 1-based index
//      of the first pivot that is not positive and finite; W~ is then zero).
#include "cb_internal.h"

namespace cb {
namespace {

constexpr int kMaxP = 129;
constexpr int kPanel = 64;
constexpr int kPackedMax = kMaxP * (kMaxP + 1) / 2;
constexpr int kZStride = kPanel + 1;   // fp64 elements per panel row (padded)

__device__ __forceinline__ int pk(int i, int j) { return i * (i + 1) / 2 + j; }  // j <= i

__global__ __launch_bounds__(256) void ridge_solve_kernel(int P, int d_t, const float *__restrict__ G,
                                                          const float *__restrict__ C, float lambda,
                                                          uint32_t flags, float *__restrict__ maps,
                                                          int32_t *__restrict__ info) {
    __shared__ double L[kPackedMax];
    __shared__ double Z[kMaxP * kZStride];
    __shared__ double red[256];
    __shared__ int fail;

    const int m = blockIdx.x;
    const int tid = threadIdx.x;
    const float *Gm = G + (int64_t)m * P * P;
    const float *Cm = C + (int64_t)m * P * d_t;
    float *Wm = maps + (int64_t)m * P * d_t;

    // 1. lower triangle of G -> LDS (fp64), trace
    double tr = 0.0;
    for (int idx = tid; idx < P * P; idx += 256) {
        const int i = idx / P, j = idx - (idx / P) * P;
        if (j <= i) {
            const double g = (double)Gm[idx];
            L[pk(i, j)] = g;
            if (i == j) tr += g;
        }
    }
    red[tid] = tr;
    if (tid == 0) fail = 0;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (tid < s) red[tid] += red[tid + s];
        __syncthreads();
    }
    const double lam = (flags & CB_LAMBDA_RELATIVE) ? (double)lambda * red[0] / (double)P : (double)lambda;
    const int n_pen = (flags & CB_RIDGE_BIAS_UNPENALIZED) ? P - 1 : P;
    for (int i = tid; i < n_pen; i += 256) L[pk(i, i)] += lam;
    __syncthreads();

    // 2. Cholesky, left-looking: column j of L from rows i >= j.  Thread t
    //    takes rows j + t/2 and j + t/2 + 128 (P <= 129), lane pairs split k.
    const int half = tid & 1;
    for (int j = 0; j < P; ++j) {
        double v[2];
#pragma unroll
        for (int rr = 0; rr < 2; ++rr) {
            const int i = j + (tid >> 1) + 128 * rr;
            double s = 0.0;
            if (i < P) {
                const double *Li = L + pk(i, 0);
                const double *Lj = L + pk(j, 0);
                for (int k = half; k < j; k += 2) s += Li[k] * Lj[k];
            }
            s += __shfl_xor(s, 1);
            v[rr] = (i < P) ? L[pk(i, j)] - s : 0.0;
        }
        __syncthreads();                       // all reads of column-j inputs done
        if (tid == 0) {
            if (!(v[0] > 0.0) || !isfinite(v[0])) fail = j + 1;
            else L[pk(j, j)] = sqrt(v[0]);
        }
        __syncthreads();
        if (fail) break;
        if (half == 0) {
            const double d = L[pk(j, j)];
#pragma unroll
            for (int rr = 0; rr < 2; ++rr) {
                const int i = j + (tid >> 1) + 128 * rr;
                if (i > j && i < P) L[pk(i, j)] = v[rr] / d;
            }
        }
        __syncthreads();
    }

    if (fail) {
        for (int idx = tid; idx < P * d_t; idx += 256) Wm[idx] = 0.f;
        if (tid == 0) info[m] = fail;
        return;
    }

    // 3. triangular solves on 64-column panels; lane q of each quad sums the
    //    k == q (mod 4) terms, every lane of the quad writes the result.
    const int q = tid & 3, col = tid >> 2;
    for (int p0 = 0; p0 < d_t; p0 += kPanel) {
        const int ncol = min(kPanel, d_t - p0);
        __syncthreads();
        for (int idx = tid; idx < P * kPanel; idx += 256) {
            const int i = idx / kPanel, c = idx - (idx / kPanel) * kPanel;
            Z[i * kZStride + c] = c < ncol ? (double)Cm[(int64_t)i * d_t + p0 + c] : 0.0;
        }
        __syncthreads();
        // forward: L z = c
        for (int i = 0; i < P; ++i) {
            double s = 0.0;
            const double *Li = L + pk(i, 0);
            for (int k = q; k < i; k += 4) s += Li[k] * Z[k * kZStride + col];
            s += __shfl_xor(s, 1);
            s += __shfl_xor(s, 2);
            Z[i * kZStride + col] = (Z[i * kZStride + col] - s) / Li[i];
        }
        // backward: L^T w = z
        for (int i = P - 1; i >= 0; --i) {
            double s = 0.0;
            for (int k = i + 1 + q; k < P; k += 4) s += L[pk(k, i)] * Z[k * kZStride + col];
            s += __shfl_xor(s, 1);
            s += __shfl_xor(s, 2);
            Z[i * kZStride + col] = (Z[i * kZStride + col] - s) / L[pk(i, i)];
        }
        __syncthreads();
        for (int idx = tid; idx < P * ncol; idx += 256) {
            const int i = idx / ncol, c = idx - (idx / ncol) * ncol;
            Wm[(int64_t)i * d_t + p0 + c] = (float)Z[i * kZStride + c];
        }
    }
    if (tid == 0) info[m] = 0;
}

}  // namespace

hipError_t launch_solve(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C,
                        float lambda, uint32_t flags, float *maps, int32_t *info, hipStream_t s) {
    if (n_maps == 0) return hipSuccess;
    hipLaunchKernelGGL(ridge_solve_kernel, dim3(n_maps), dim3(256), 0, s, P, d_t, G, C, lambda, flags,
                       maps, info);
    return hipGetLastError();
}

}  // namespace cb

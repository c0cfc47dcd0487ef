// cb_solve.hip -- batched ridge solve, one workgroup per system (gfx950).
//
// CacheBridge Sec. 3.1 (Eq. closedform) and Sec. 3.4: the maps are the ridge
// solutions W~ = (G + lambda D)^{-1} C of the augmented moments.  For each map
// the workgroup holds the augmented matrix [M | C], M = G + lambda_m D, in
// registers as fp64 (512 threads, a cyclic 16 x 32 thread grid, up to 9 x 9
// elements each) and runs Gauss-Jordan elimination without pivoting:
//   step k publishes row k and column k through LDS (double buffered, one
//   barrier per step), and every thread subtracts (A[i][k] / A[k][k]) A[k][j]
//   from its elements of the other rows.
// M is symmetric positive definite, for which elimination in the natural
// order is stable and the pivot of step k is the k-th squared diagonal
// entry of the Cholesky factor; a pivot that is not positive and finite
// stops the system with info = k + 1 (1-based) and zero maps, the failure
// the Cholesky factorization would report at the same column.  At the end
// row i of the C part divided by the pivot of row i is row i of W~.
//   lambda_m = lambda, or lambda * tr(G) / P with CB_LAMBDA_RELATIVE; with
//   CB_RIDGE_BIAS_UNPENALIZED the last (bias) diagonal entry gets no lambda.
//
// Centered form (Sec. 3.1, Eq. closedform as written): the system is
// (A + lambda_m I) W = B of size d_s with the centered moments A, B, and the
// bias row is b = mu_y - W^T mu_x, formed in fp64 from the unrounded W.  The
// relative lambda uses the trace of the augmented matrix the same data would
// give, tr(A) + S |mu_x|^2 + S (S = sum w), so that both forms solve the same
// problem.
#include "cb_internal.h"

namespace cb {
namespace {

constexpr int kTR = 16, kTC = 32;                 // thread grid: rows x columns
constexpr int kThreads = kTR * kTC;
constexpr int kMaxP = 129, kMaxCols = 129 + 128;  // M and C columns
constexpr int kRA = (kMaxP + kTR - 1) / kTR;      // rows per thread (9)
constexpr int kCB = (kMaxCols + kTC - 1) / kTC;   // columns per thread (9)

// P: size of the system (plain: d_s + 1 with the bias row; centered: d_s).
// Plain: G [P][P], C [P][d_t] -> maps [P][d_t].  Centered: G = A [d_s][d_s],
// C = B [d_s][d_t], sums [1 + d_s + d_t] -> maps [d_s + 1][d_t].
template <bool CENTERED>
__global__ __launch_bounds__(kThreads) void ridge_solve_kernel(int P, int d_t, const float *__restrict__ G,
                                                               const float *__restrict__ C,
                                                               const double *__restrict__ sums, float lambda,
                                                               uint32_t flags, float *__restrict__ maps,
                                                               int32_t *__restrict__ info) {
    __shared__ double rowbuf[2][kCB * kTC];
    __shared__ double colbuf[2][kRA * kTR];
    __shared__ double red[kThreads / 64];

    const int m = blockIdx.x;
    const int tid = threadIdx.x;
    const int r = tid / kTC, c = tid % kTC;       // element (i, j): i = r + kTR a, j = c + kTC b
    const int NC = P + d_t;
    const int PW = CENTERED ? P + 1 : P;          // rows of the written map
    const float *Gm = G + (int64_t)m * P * P;
    const float *Cm = C + (int64_t)m * P * d_t;
    float *Wm = maps + (int64_t)m * PW * d_t;
    const double *sm = CENTERED ? sums + (int64_t)m * (1 + P + d_t) : nullptr;
    const double S = CENTERED ? sm[0] : 0.0;

    // load [G | C] (fp32 -> fp64) and sum the diagonal of G (centered: of
    // the augmented matrix of the same data)
    double A[kRA][kCB];
    double trp = 0.0;
#pragma unroll
    for (int a = 0; a < kRA; ++a) {
        const int i = r + kTR * a;
#pragma unroll
        for (int b = 0; b < kCB; ++b) {
            const int j = c + kTC * b;
            double v = 0.0;
            if (i < P && j < NC) v = j < P ? (double)Gm[(int64_t)i * P + j] : (double)Cm[(int64_t)i * d_t + (j - P)];
            A[a][b] = v;
            if (i == j && i < P) {
                trp += v;
                if (CENTERED && S != 0.0) trp += sm[1 + i] * (sm[1 + i] / S);
            }
        }
    }
    // block sum of the trace parts (wave shuffles, then one value per wave)
    for (int o = 32; o > 0; o >>= 1) trp += __shfl_xor(trp, o);
    if ((tid & 63) == 0) red[tid >> 6] = trp;
    __syncthreads();
    double tr = CENTERED ? S : 0.0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) tr += red[w];
    const double lam = (flags & CB_LAMBDA_RELATIVE) ? (double)lambda * tr / (double)PW : (double)lambda;
    const int n_pen = (!CENTERED && (flags & CB_RIDGE_BIAS_UNPENALIZED)) ? P - 1 : P;
#pragma unroll
    for (int a = 0; a < kRA; ++a)
#pragma unroll
        for (int b = 0; b < kCB; ++b) {
            const int i = r + kTR * a, j = c + kTC * b;
            if (i == j && i < n_pen) A[a][b] += lam;
        }

    // Gauss-Jordan elimination
    int fail = 0;
    for (int k = 0; k < P; ++k) {
        double *rb = rowbuf[k & 1];
        double *cb = colbuf[k & 1];
#pragma unroll
        for (int a = 0; a < kRA; ++a)
            if (r + kTR * a == k) {
#pragma unroll
                for (int b = 0; b < kCB; ++b) rb[c + kTC * b] = A[a][b];
            }
#pragma unroll
        for (int b = 0; b < kCB; ++b)
            if (c + kTC * b == k) {
#pragma unroll
                for (int a = 0; a < kRA; ++a) cb[r + kTR * a] = A[a][b];
            }
        __syncthreads();
        const double p = rb[k];
        if (!(p > 0.0) || !isfinite(p)) {       // same value in every thread
            fail = k + 1;
            break;
        }
        const double inv = 1.0 / p;
        double f[kRA], rv[kCB];
#pragma unroll
        for (int a = 0; a < kRA; ++a) {
            const int i = r + kTR * a;
            f[a] = (i == k || i >= P) ? 0.0 : cb[i] * inv;
        }
#pragma unroll
        for (int b = 0; b < kCB; ++b) rv[b] = rb[c + kTC * b];
#pragma unroll
        for (int a = 0; a < kRA; ++a)
#pragma unroll
            for (int b = 0; b < kCB; ++b) A[a][b] = __builtin_fma(-f[a], rv[b], A[a][b]);
    }

    if (fail) {
        for (int idx = tid; idx < PW * d_t; idx += kThreads) Wm[idx] = 0.f;
        if (tid == 0) info[m] = fail;
        return;
    }

    // W~[i][:] = C part of row i / pivot of row i (the pivots sit on the
    // diagonal of the eliminated M part; colbuf is free again)
    __syncthreads();
#pragma unroll
    for (int a = 0; a < kRA; ++a)
#pragma unroll
        for (int b = 0; b < kCB; ++b) {
            const int i = r + kTR * a, j = c + kTC * b;
            if (i == j && i < P) colbuf[0][i] = 1.0 / A[a][b];
        }
    __syncthreads();
    double bpart[kCB];                            // centered: sum over this thread's rows of mu_x,i W_ij
#pragma unroll
    for (int b = 0; b < kCB; ++b) bpart[b] = 0.0;
#pragma unroll
    for (int a = 0; a < kRA; ++a) {
        const int i = r + kTR * a;
        if (i >= P) continue;
        const double inv = colbuf[0][i];
        const double mui = CENTERED && S != 0.0 ? sm[1 + i] / S : 0.0;
#pragma unroll
        for (int b = 0; b < kCB; ++b) {
            const int j = c + kTC * b;
            if (j >= P && j < NC) {
                const double wv = A[a][b] * inv;
                Wm[(int64_t)i * d_t + (j - P)] = (float)wv;
                if (CENTERED) bpart[b] = __builtin_fma(mui, wv, bpart[b]);
            }
        }
    }
    if constexpr (CENTERED) {
        // b_j = mu_y,j - sum_i mu_x,i W_ij: the 16 row partials of each column
        // are combined through LDS in a fixed order.
        __shared__ double bred[kTR][kCB * kTC];
#pragma unroll
        for (int b = 0; b < kCB; ++b) bred[r][c + kTC * b] = bpart[b];
        __syncthreads();
        for (int j = tid; j < d_t; j += kThreads) {
            double s = 0.0;
            for (int rr = 0; rr < kTR; ++rr) s += bred[rr][P + j];
            const double muy = S != 0.0 ? sm[1 + P + j] / S : 0.0;
            Wm[(int64_t)P * d_t + j] = (float)(muy - s);
        }
    }
    if (tid == 0) info[m] = 0;
}

}  // namespace

hipError_t launch_solve(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C,
                        float lambda, uint32_t flags, float *maps, int32_t *info, hipStream_t s) {
    if (n_maps == 0) return hipSuccess;
    if (P > kMaxP || P + d_t > kMaxCols) return hipErrorInvalidValue;
    hipLaunchKernelGGL(ridge_solve_kernel<false>, dim3(n_maps), dim3(kThreads), 0, s, P, d_t, G, C,
                       (const double *)nullptr, lambda, flags, maps, info);
    return hipGetLastError();
}

hipError_t launch_solve_centered(int32_t n_maps, int32_t d_s, int32_t d_t, const double *sums, const float *A,
                                 const float *B, float lambda, uint32_t flags, float *maps, int32_t *info,
                                 hipStream_t s) {
    if (n_maps == 0) return hipSuccess;
    if (d_s + 1 > kMaxP || d_s + d_t > kMaxCols) return hipErrorInvalidValue;
    hipLaunchKernelGGL(ridge_solve_kernel<true>, dim3(n_maps), dim3(kThreads), 0, s, d_s, d_t, A, B, sums, lambda,
                       flags, maps, info);
    return hipGetLastError();
}

}  // namespace cb

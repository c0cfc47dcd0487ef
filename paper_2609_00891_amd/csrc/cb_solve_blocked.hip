// cb_solve_blocked.hip -- batched ridge solve for wide features (P > 129).
//
// CacheBridge Sec. 3.1 (Eq. closedform) with the multi-layer feature of
// Sec. 3.2 (P = k d_s + 1, 1025 at k = 8): the systems no longer fit in one
// workgroup's registers or LDS, so each one is factored in the caller's
// workspace.  One workgroup of 256 threads per system, all arithmetic fp64:
//
//   M = G + lambda_m D  (lambda_m = lambda, or lambda tr(G) / P; D = I, or
//                        diag(1, .., 1, 0) with CB_RIDGE_BIAS_UNPENALIZED)
//   1. left-looking blocked Cholesky M = L L^T in panels of 32 columns:
//      panel = M[c0:, c0:c0+32] - L[c0:, :c0] L[c0:c0+32, :c0]^T (LDS-tiled),
//      the 32 x 32 diagonal block factored in LDS, the rows below solved
//      against it (one thread per row);
//   2. forward substitution L Z = C by 32-row panels;
//   3. back substitution L^T W~ = Z by 32-row panels, in place of Z;
//   4. maps = (float) W~.
// A pivot that is not positive and finite stops the system: info = its
// 1-based column, maps zero-filled (the report of the register solver).
//
// Workspace per system: L (P x P fp64, lower triangle used) and Z (P x d_t
// fp64).  Systems are solved in batches that fit the workspace.
#include <algorithm>

#include "cb_internal.h"

namespace cb {
namespace {

constexpr int NB = 32;          // panel width
constexpr int TRW = 64;         // rows per GEMM tile of the factorization
constexpr int KC = 32;          // inner-dimension chunk
constexpr int NT = 256;
constexpr int LP = 33;          // padded LDS row (doubles)
constexpr int DTMAX = 128;
constexpr int ZP = DTMAX + 1;

__global__ __launch_bounds__(NT) void chol_solve_kernel(int32_t P, int32_t d_t, const float *__restrict__ G,
                                                        const float *__restrict__ C, float lambda, uint32_t flags,
                                                        double *__restrict__ ws, int64_t ws_stride, int32_t m0,
                                                        float *__restrict__ maps, int32_t *__restrict__ info) {
    __shared__ double sA[TRW * LP];        // row tile chunk (factorization) / L panel chunk (solves)
    __shared__ double sB[KC * ZP];         // panel rows chunk (factorization) / Z rows chunk (solves)
    __shared__ double sD[NB * LP];         // the factored diagonal block
    __shared__ double sR[NB * ZP];         // right-hand sides of one panel (solves)
    __shared__ double sInv[NB];
    __shared__ double red[NT / 64];
    __shared__ int s_bad;

    const int m = m0 + blockIdx.x;
    const int tid = threadIdx.x;
    double *L = ws + (int64_t)blockIdx.x * ws_stride;
    double *Z = L + (int64_t)P * P;
    const float *Gm = G + (int64_t)m * P * P;
    const float *Cm = C + (int64_t)m * P * d_t;
    float *Wm = maps + (int64_t)m * P * d_t;

    // ---- lambda_m
    double tr = 0.0;
    for (int i = tid; i < P; i += NT) tr += (double)Gm[(int64_t)i * P + i];
    for (int o = 32; o > 0; o >>= 1) tr += __shfl_xor(tr, o);
    if ((tid & 63) == 0) red[tid >> 6] = tr;
    if (tid == 0) s_bad = 0;
    __syncthreads();
    const double trace = (red[0] + red[1]) + (red[2] + red[3]);
    const double lam = (flags & CB_LAMBDA_RELATIVE) ? (double)lambda * trace / (double)P : (double)lambda;
    const int lam_last = (flags & CB_RIDGE_BIAS_UNPENALIZED) ? P - 1 : P;   // diagonal entries < lam_last get lambda

    // ================= 1. blocked Cholesky
    for (int c0 = 0; c0 < P; c0 += NB) {
        const int nb = min(NB, P - c0);
        // panel = M[c0:, c0:c0+nb] - L[c0:, :c0] L[c0:c0+nb, :c0]^T, into L
        const int i0 = tid >> 3, j0 = (tid & 7) * 4;
        for (int rt = c0; rt < P; rt += TRW) {
            double acc[2][4] = {{0, 0, 0, 0}, {0, 0, 0, 0}};
            for (int k0 = 0; k0 < c0; k0 += KC) {
                for (int e = tid; e < TRW * KC; e += NT) {
                    const int i = e / KC, kk = e % KC;
                    sA[i * LP + kk] = rt + i < P ? L[(int64_t)(rt + i) * P + k0 + kk] : 0.0;
                }
                for (int e = tid; e < NB * KC; e += NT) {
                    const int j = e / KC, kk = e % KC;
                    sB[j * LP + kk] = j < nb ? L[(int64_t)(c0 + j) * P + k0 + kk] : 0.0;
                }
                __syncthreads();
#pragma unroll 8
                for (int kk = 0; kk < KC; ++kk) {
                    const double a0 = sA[i0 * LP + kk], a1 = sA[(i0 + 32) * LP + kk];
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        const double bv = sB[(j0 + b) * LP + kk];
                        acc[0][b] = fma(a0, bv, acc[0][b]);
                        acc[1][b] = fma(a1, bv, acc[1][b]);
                    }
                }
                __syncthreads();
            }
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                const int r = rt + i0 + 32 * a;
                if (r >= P) continue;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int c = c0 + j0 + b;
                    if (j0 + b >= nb) continue;
                    double v = (double)Gm[(int64_t)r * P + c];
                    if (r == c && c < lam_last) v += lam;
                    L[(int64_t)r * P + c] = v - acc[a][b];
                }
            }
        }
        __syncthreads();
        // factor the diagonal block in LDS
        for (int e = tid; e < NB * NB; e += NT) {
            const int i = e / NB, j = e % NB;
            sD[i * LP + j] = (i < nb && j < nb && j <= i) ? L[(int64_t)(c0 + i) * P + c0 + j] : 0.0;
        }
        __syncthreads();
        for (int j = 0; j < nb; ++j) {
            if (tid == 0) {
                const double d = sD[j * LP + j];
                if (!(d > 0.0) || !isfinite(d)) {
                    s_bad = c0 + j + 1;
                } else {
                    const double s = sqrt(d);
                    sD[j * LP + j] = s;
                    sInv[j] = 1.0 / s;
                }
            }
            __syncthreads();
            if (s_bad) break;
            if (tid > j && tid < nb) sD[tid * LP + j] *= sInv[j];
            __syncthreads();
            for (int e = tid; e < NB * NB; e += NT) {
                const int i = e / NB, l = e % NB;
                if (i > j && l > j && l <= i && i < nb) sD[i * LP + l] -= sD[i * LP + j] * sD[l * LP + j];
            }
            __syncthreads();
        }
        if (s_bad) break;
        for (int e = tid; e < NB * NB; e += NT) {
            const int i = e / NB, j = e % NB;
            if (i < nb && j <= i) L[(int64_t)(c0 + i) * P + c0 + j] = sD[i * LP + j];
        }
        // rows below: L[r][c0:c0+32] = panel row solved against the diagonal block
        for (int r = c0 + NB + tid; r < P; r += NT) {
            asm volatile("" ::: "memory");              // keeps the block's LDS reads inside the row loop
            double x[NB];
#pragma unroll
            for (int j = 0; j < NB; ++j) x[j] = L[(int64_t)r * P + c0 + j];
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                double s = x[j];
#pragma unroll
                for (int i = 0; i < j; ++i) s -= x[i] * sD[j * LP + i];
                x[j] = s * sInv[j];
            }
#pragma unroll
            for (int j = 0; j < NB; ++j) L[(int64_t)r * P + c0 + j] = x[j];
        }
        __syncthreads();
    }
    if (s_bad) {
        if (tid == 0) info[m] = s_bad;
        for (int64_t e = tid; e < (int64_t)P * d_t; e += NT) Wm[e] = 0.f;
        return;
    }

    // ================= 2. forward substitution L Z = C
    const int ri = tid >> 4, cj = (tid & 15) * 8;          // GEMM outputs: rows ri, ri+16; cols cj..cj+7
    for (int c0 = 0; c0 < P; c0 += NB) {
        const int nb = min(NB, P - c0);
        double acc[2][8];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 8; ++b) acc[a][b] = 0.0;
        for (int k0 = 0; k0 < c0; k0 += KC) {
            for (int e = tid; e < NB * KC; e += NT) {
                const int i = e / KC, kk = e % KC;
                sA[i * LP + kk] = i < nb ? L[(int64_t)(c0 + i) * P + k0 + kk] : 0.0;
            }
            for (int e = tid; e < KC * DTMAX; e += NT) {
                const int kk = e / DTMAX, c = e % DTMAX;
                sB[kk * ZP + c] = c < d_t ? Z[(int64_t)(k0 + kk) * d_t + c] : 0.0;
            }
            __syncthreads();
#pragma unroll 4
            for (int kk = 0; kk < KC; ++kk) {
                const double a0 = sA[ri * LP + kk], a1 = sA[(ri + 16) * LP + kk];
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                    const double zv = sB[kk * ZP + cj + b];
                    acc[0][b] = fma(a0, zv, acc[0][b]);
                    acc[1][b] = fma(a1, zv, acc[1][b]);
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                const int i = ri + 16 * a, c = cj + b;
                sR[i * ZP + c] = (i < nb && c < d_t) ? (double)Cm[(int64_t)(c0 + i) * d_t + c] - acc[a][b] : 0.0;
            }
        for (int e = tid; e < NB * NB; e += NT) {
            const int i = e / NB, j = e % NB;
            sD[i * LP + j] = (i < nb && j <= i) ? L[(int64_t)(c0 + i) * P + c0 + j] : 0.0;
        }
        __syncthreads();
        if (tid < d_t) {
            double z[NB];
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                double s = sR[i * ZP + tid];
#pragma unroll
                for (int l = 0; l < i; ++l) s -= sD[i * LP + l] * z[l];
                z[i] = i < nb ? s / sD[i * LP + i] : 0.0;
            }
#pragma unroll
            for (int i = 0; i < NB; ++i)
                if (i < nb) Z[(int64_t)(c0 + i) * d_t + tid] = z[i];
        }
        __syncthreads();
    }

    // ================= 3. back substitution L^T W~ = Z (W~ overwrites Z)
    const int last = ((P - 1) / NB) * NB;
    for (int c0 = last; c0 >= 0; c0 -= NB) {
        const int nb = min(NB, P - c0), c1 = c0 + nb;
        double acc[2][8];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 8; ++b) acc[a][b] = 0.0;
        for (int k0 = c1; k0 < P; k0 += KC) {
            // L[k][c0 + i] for k in the chunk, stored as sA[i][kk]
            for (int e = tid; e < KC * NB; e += NT) {
                const int kk = e / NB, i = e % NB;
                sA[i * LP + kk] = (k0 + kk < P) ? L[(int64_t)(k0 + kk) * P + c0 + i] : 0.0;
            }
            for (int e = tid; e < KC * DTMAX; e += NT) {
                const int kk = e / DTMAX, c = e % DTMAX;
                sB[kk * ZP + c] = (k0 + kk < P && c < d_t) ? Z[(int64_t)(k0 + kk) * d_t + c] : 0.0;
            }
            __syncthreads();
#pragma unroll 4
            for (int kk = 0; kk < KC; ++kk) {
                const double a0 = sA[ri * LP + kk], a1 = sA[(ri + 16) * LP + kk];
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                    const double zv = sB[kk * ZP + cj + b];
                    acc[0][b] = fma(a0, zv, acc[0][b]);
                    acc[1][b] = fma(a1, zv, acc[1][b]);
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                const int i = ri + 16 * a, c = cj + b;
                sR[i * ZP + c] = (i < nb && c < d_t) ? Z[(int64_t)(c0 + i) * d_t + c] - acc[a][b] : 0.0;
            }
        for (int e = tid; e < NB * NB; e += NT) {
            const int i = e / NB, j = e % NB;
            sD[i * LP + j] = (i < nb && j <= i) ? L[(int64_t)(c0 + i) * P + c0 + j] : 0.0;
        }
        __syncthreads();
        if (tid < d_t) {
            double w[NB];
#pragma unroll
            for (int i = NB - 1; i >= 0; --i) {
                double s = sR[i * ZP + tid];
#pragma unroll
                for (int l = i + 1; l < NB; ++l) s -= sD[l * LP + i] * w[l];
                w[i] = i < nb ? s / sD[i * LP + i] : 0.0;
            }
#pragma unroll
            for (int i = 0; i < NB; ++i)
                if (i < nb) Z[(int64_t)(c0 + i) * d_t + tid] = w[i];
        }
        __syncthreads();
    }

    // ================= 4. maps
    for (int64_t e = tid; e < (int64_t)P * d_t; e += NT) Wm[e] = (float)Z[e];
    if (tid == 0) info[m] = 0;
}

}  // namespace

int64_t solve_blocked_bytes_per_system(int32_t P, int32_t d_t) {
    return ((int64_t)P * P + (int64_t)P * d_t) * (int64_t)sizeof(double);
}

hipError_t launch_solve_blocked(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C, float lambda,
                                uint32_t flags, void *ws, int64_t ws_bytes, float *maps, int32_t *info,
                                hipStream_t s) {
    if (n_maps == 0) return hipSuccess;
    if (d_t > DTMAX || P < 2) return hipErrorInvalidValue;
    const int64_t per = solve_blocked_bytes_per_system(P, d_t);
    const int64_t stride = per / (int64_t)sizeof(double);
    const int64_t batch = ws_bytes / per;
    if (batch < 1) return hipErrorInvalidValue;
    for (int32_t m0 = 0; m0 < n_maps; m0 += (int32_t)std::min<int64_t>(batch, n_maps)) {
        const int32_t nb = (int32_t)std::min<int64_t>(batch, n_maps - m0);
        hipLaunchKernelGGL(chol_solve_kernel, dim3(nb), dim3(NT), 0, s, P, d_t, G, C, lambda, flags, (double *)ws,
                           stride, m0, maps, info);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace cb

// cb_solve_blocked.hip -- batched ridge solve for wide features (P > 129).
//
// CacheBridge Sec. 3.1 (Eq. closedform) with the multi-layer feature of
// Sec. 3.2 (P = k d_s + 1, 1025 at k = 8): the systems no longer fit in one
// workgroup's registers or LDS, so each one is factored in the caller's
// workspace.  One workgroup of 256 threads per system, all arithmetic fp64:
//
//   M = G + lambda_m D  (lambda_m = lambda, or lambda tr(G) / P; D = I, or
//                        diag(1, .., 1, 0) with CB_RIDGE_BIAS_UNPENALIZED)
//   1. left-looking blocked Cholesky M = L L^T in panels of 32 columns.  The
//      panel M[c0:, c0:c0+32] - L[c0:, :c0] L[c0:c0+32, :c0]^T is a product on
//      the fp64 matrix cores (v_mfma_f64_16x16x4: wave w owns the 16-row tiles
//      w, w + 4, ... of a pass of up to 192 rows), its inner dimension in
//      16-wide chunks double-buffered through LDS so the next chunk's global
//      loads overlap this chunk's products.  The diagonal block's 32 rows go
//      first; one wave factors the block and forms its inverse V in
//      registers (lane i holds row i; the other rows' entries arrive by
//      readlane) and V is kept, transposed, in the block's unused upper half.
//      Each later pass then stores (M - L L^T) V^T for its rows, a second
//      matrix-core product on its LDS copy of M - L L^T;
//   2. forward substitution L Z = C by 32-row panels: the panel product on
//      the matrix cores (16-wide chunks through LDS), then the panel's rows
//      times the kept inverse of its diagonal block (4 x 4 outputs per thread);
//   3. back substitution L^T W~ = Z by 32-row panels, in place of Z;
//   4. maps = (float) W~.
// A pivot that is not positive and finite stops the system: info = its
// 1-based column, maps zero-filled (the report of the register solver).
//
// Workspace per system: L (P x P fp64: the lower triangle, plus the inverse
// diagonal blocks in the upper halves of the diagonal blocks) and Z (P x d_t
// fp64).  Systems are solved in batches that fit the workspace.
#include <algorithm>
#include <mutex>
#include <type_traits>

#include "cb_internal.h"

namespace cb {
namespace {

constexpr int NT = 256;
constexpr int NB = 32;          // panel width
constexpr int KC = 16;          // inner-dimension chunk
constexpr int KP = KC + 1;      // padded LDS row of a chunk (doubles)
constexpr int TR = 192;         // rows per GEMM pass of the factorization
static_assert(TR == 6 * 32, "the pass dispatch below covers 1 .. 6 groups of 32 rows");
constexpr int KS = 16;          // inner-dimension chunk of the substitutions
constexpr int KSP = KS + 1;
constexpr int DP = NB + 1;      // padded row of the diagonal block
constexpr int RP = NB + 1;      // padded row of a pass's M - acc (solved rows below the diagonal block)
constexpr int DTMAX = 128;
constexpr int ZP = DTMAX + 1;   // padded row of a right-hand-side chunk

// LDS (doubles): factorization: A chunks [2][TR][KP], B chunks [2][NB][KP];
// substitutions: L chunks [2][NB][KSP], Z chunks [2][KS][ZP]; the panel rhs [NB][ZP] reuses the chunks'
// space once a panel's products are done.
// About 78 KB in all, so two systems share a compute unit (with at most
// 256 registers per lane: two waves per SIMD).
constexpr int OFF_A = 0;
constexpr int OFF_B = OFF_A + 2 * TR * KP;
constexpr int OFF_L = 0;
constexpr int OFF_Z = OFF_L + 2 * NB * KSP;
constexpr int OFF_R = 0;
constexpr int LQ = NB * KS / NT, ZQ = KS * DTMAX / NT;   // operand elements per thread and chunk
static_assert(LQ * NT == NB * KS && ZQ * NT == KS * DTMAX, "substitution chunks split evenly over the threads");
constexpr int SH_WORK = std::max(OFF_B + 2 * NB * KP, std::max(OFF_Z + 2 * KS * ZP, OFF_R + NB * ZP));

typedef __attribute__((ext_vector_type(4))) double f64x4_t;

// fp64 matrix-core product D += A B of a 16 x 4 by 4 x 16 block: lane l
// supplies A[l % 16][l / 16] and B[l / 16][l % 16] and holds D[l / 16 + 4 i][l % 16]
// in element i.
__device__ __forceinline__ f64x4_t mfma_f64(double a, double b, f64x4_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// Lane l's value of v, read by every lane (l uniform).
__device__ __forceinline__ double readlane_f64(double v, int l) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, l), hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), l);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ void wave_sync_lds() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

// csums != nullptr: the centered form (Sec. 3.1, Eq. closedform as written).
// G and C are then A [P][P] and B [P][d_t] of the feature x (no bias entry),
// csums [n][1 + P + d_t] holds (sum w, sum w x, sum w y); every diagonal entry
// gets lambda_m, lambda_m = lambda (tr A + S |mu_x|^2 + S) / (P + 1) when
// relative (the trace of the augmented matrix of the same data), and each map
// gets P + 1 rows: W, then the bias b = mu_y - W^T mu_x.
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2))) void chol_solve_kernel(int32_t P, int32_t d_t, const float *__restrict__ G,
                                                        const float *__restrict__ C, float lambda, uint32_t flags,
                                                        double *__restrict__ ws, int64_t ws_stride, int32_t m0,
                                                        float *__restrict__ maps, int32_t *__restrict__ info,
                                                        const double *__restrict__ csums) {
    __shared__ double sh[SH_WORK];
    __shared__ double sD[NB * DP];         // the diagonal block of the current panel
    __shared__ double sInv[NB];            // reciprocals of its diagonal
    __shared__ double sV[NB * DP];         // the inverse of the diagonal block
    __shared__ double red[NT / 64];
    __shared__ int s_bad;

    const int m = m0 + blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double *L = ws + (int64_t)blockIdx.x * ws_stride;
    double *Z = L + (int64_t)P * P;
    const float *Gm = G + (int64_t)m * P * P;
    const float *Cm = C + (int64_t)m * P * d_t;
    const int out_rows = csums ? P + 1 : P;
    float *Wm = maps + (int64_t)m * out_rows * d_t;
    const double *sm = csums ? csums + (int64_t)m * (1 + P + d_t) : nullptr;
    const double sw = sm ? sm[0] : 0.0;

    // ---- lambda_m
    double tr = 0.0;
    for (int i = tid; i < P; i += NT) {
        tr += (double)Gm[(int64_t)i * P + i];
        if (sm && sw != 0.0) tr += sm[1 + i] * (sm[1 + i] / sw);       // S mu_i^2
    }
    for (int o = 32; o > 0; o >>= 1) tr += __shfl_xor(tr, o);
    if (lane == 0) red[wave] = tr;
    if (tid == 0) s_bad = 0;
    __syncthreads();
    const double trace = (red[0] + red[1]) + (red[2] + red[3]) + sw;
    const double lam = (flags & CB_LAMBDA_RELATIVE) ? (double)lambda * trace / (double)(sm ? P + 1 : P)
                                                    : (double)lambda;
    const int lam_last = (!sm && (flags & CB_RIDGE_BIAS_UNPENALIZED)) ? P - 1 : P;   // entries < lam_last get lambda

    // Loads the inverse V of the 32 x 32 diagonal block at (c0, c0) into sV
    // (lower triangular, zero outside the nb x nb block): its diagonal is
    // 1 / L[c0+i][c0+i], its strictly lower part was stored transposed in the
    // (otherwise unused) strictly upper part of the block by the factorization.
    auto load_inv = [&](int c0, int nb) {
        for (int e = tid; e < NB * NB; e += NT) {
            const int i = e / NB, c = e % NB;
            double v = 0.0;
            if (i < nb && c < nb) {
                if (c == i) v = 1.0 / L[(int64_t)(c0 + i) * P + c0 + i];
                else if (c < i) v = L[(int64_t)(c0 + c) * P + c0 + i];
            }
            sV[i * DP + c] = v;
        }
    };

    // ================= 1. blocked Cholesky
    double *sA = sh + OFF_A, *sB = sh + OFF_B;
    for (int c0 = 0; c0 < P; c0 += NB) {
        const int nb = min(NB, P - c0);
        const int nch = c0 / KC;                        // c0 is a multiple of 32
        // rows c0 .. P-1 in passes of up to TR rows; a pass of NI 32-row groups
        // (the last one may be shorter) is compiled for its NI so that no FMA is
        // spent on rows past P
        // SOLVE: rows below the diagonal block, whose panel entries are
        // x = (M - acc) L_dd^-T = (M - acc) V^T: the pass puts M - acc in LDS
        // and multiplies it by V^T on the matrix cores before storing it.
        auto gemm_pass = [&](auto NIc, auto SOLVEc, int rt) {
            constexpr int NI = decltype(NIc)::value;
            constexpr bool SOLVE = decltype(SOLVEc)::value;
            constexpr int NRT = 2 * NI;                 // 16-row tiles of the pass
            constexpr int MAXT = (NRT + 3) / 4;         // tiles of one wave (wave w: w, w + 4, ...)
            f64x4_t acc[MAXT][2];
#pragma unroll
            for (int j = 0; j < MAXT; ++j)
#pragma unroll
                for (int ct = 0; ct < 2; ++ct) acc[j][ct] = f64x4_t{0.0, 0.0, 0.0, 0.0};
            double pa[2 * NI], pb[2];
            auto fetch = [&](int ch) {                  // chunk ch of L[rt:rt+32NI, :] and L[c0:c0+32, :]
                const int k0 = ch * KC, kk = tid & 15;
#pragma unroll
                for (int q = 0; q < 2 * NI; ++q) {
                    const int r = rt + (tid >> 4) + 16 * q;
                    pa[q] = r < P ? L[(int64_t)r * P + k0 + kk] : 0.0;
                }
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const int j = (tid >> 4) + 16 * q;
                    pb[q] = j < nb ? L[(int64_t)(c0 + j) * P + k0 + kk] : 0.0;
                }
            };
            auto stash = [&](int buf) {
                const int kk = tid & 15;
#pragma unroll
                for (int q = 0; q < 2 * NI; ++q) sA[buf * TR * KP + ((tid >> 4) + 16 * q) * KP + kk] = pa[q];
#pragma unroll
                for (int q = 0; q < 2; ++q) sB[buf * NB * KP + ((tid >> 4) + 16 * q) * KP + kk] = pb[q];
            };
            const int lr = lane & 15, lk = lane >> 4;   // fragment row / column, inner index
            if (nch > 0) fetch(0);
            for (int ch = 0; ch < nch; ++ch) {
                stash(ch & 1);
                __syncthreads();
                if (ch + 1 < nch) fetch(ch + 1);
                const double *a = sA + (ch & 1) * TR * KP, *b = sB + (ch & 1) * NB * KP;
#pragma unroll
                for (int s4 = 0; s4 < KC / 4; ++s4) {
                    const int kk = 4 * s4 + lk;
                    const double b0 = b[lr * KP + kk], b1 = b[(16 + lr) * KP + kk];
#pragma unroll
                    for (int j = 0; j < MAXT; ++j) {
                        const int t = wave + 4 * j;
                        if (t < NRT) {
                            const double av = a[(16 * t + lr) * KP + kk];
                            acc[j][0] = mfma_f64(av, b0, acc[j][0]);
                            acc[j][1] = mfma_f64(av, b1, acc[j][1]);
                        }
                    }
                }
            }
            if constexpr (SOLVE) {
                // R = M - acc of this wave's rows, [16 t + row][RP] over the chunk buffers
                __syncthreads();                        // every wave is done with the chunks
#pragma unroll
                for (int j = 0; j < MAXT; ++j) {
                    const int t = wave + 4 * j;
                    if (t >= NRT) continue;
#pragma unroll
                    for (int ct = 0; ct < 2; ++ct) {
                        const int cc = 16 * ct + lr;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int rl = 16 * t + lk + 4 * i, r = rt + rl;
                            const double g = (r < P && cc < nb) ? (double)Gm[(int64_t)r * P + c0 + cc] : 0.0;
                            sA[rl * RP + cc] = (r < P && cc < nb) ? g - acc[j][ct][i] : 0.0;
                        }
                    }
                }
                wave_sync_lds();                        // a wave reads back only its own rows
#pragma unroll
                for (int j = 0; j < MAXT; ++j) {
                    const int t = wave + 4 * j;
                    if (t >= NRT) continue;
                    f64x4_t x0 = {0.0, 0.0, 0.0, 0.0}, x1 = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
                    for (int s4 = 0; s4 < NB / 4; ++s4) {
                        const int kk = 4 * s4 + lk;
                        const double av = sA[(16 * t + lr) * RP + kk];
                        x0 = mfma_f64(av, sV[lr * DP + kk], x0);            // V^T[k][c] = V[c][k]
                        x1 = mfma_f64(av, sV[(16 + lr) * DP + kk], x1);
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = rt + 16 * t + lk + 4 * i;
                        if (r >= P) continue;
                        if (lr < nb) L[(int64_t)r * P + c0 + lr] = x0[i];
                        if (16 + lr < nb) L[(int64_t)r * P + c0 + 16 + lr] = x1[i];
                    }
                }
            } else {
#pragma unroll
                for (int j = 0; j < MAXT; ++j) {
                    const int t = wave + 4 * j;
                    if (t >= NRT) continue;
#pragma unroll
                    for (int ct = 0; ct < 2; ++ct) {
                        const int cc = 16 * ct + lr;
                        if (cc >= nb) continue;
                        const int c = c0 + cc;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int r = rt + 16 * t + lk + 4 * i;
                            if (r >= P) continue;
                            double v = (double)Gm[(int64_t)r * P + c];
                            if (r == c && c < lam_last) v += lam;
                            L[(int64_t)r * P + c] = v - acc[j][ct][i];
                        }
                    }
                }
            }
            __syncthreads();
        };
        // the diagonal block's rows first: it is factored before the rows below
        gemm_pass(std::integral_constant<int, 1>(), std::false_type(), c0);
        // Factor the diagonal block and invert it: one wave, in registers.  Lane
        // i (and its mirror i + 32) holds row i of the block in a[] and, after
        // the factorization, row i of V = L_dd^-1 in v[]; the entries of other
        // rows that a step needs arrive by readlane.  Right-looking: step j
        // scales column j and subtracts its outer product from the columns to
        // its right.  (Entries right of the diagonal collect junk that no step
        // reads; they are dropped when the rows are stored.)
        if (wave == 0) {
            const int i = lane & 31;
            double a[NB];
#pragma unroll
            for (int c = 0; c < NB; ++c) a[c] = (i < nb && c <= i) ? L[(int64_t)(c0 + i) * P + c0 + c] : 0.0;
            int bad = 0;
            double dinv = 0.0;                          // 1 / L[i][i]
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                // (no break: a fixed trip count keeps the loop unrolled and a[] in registers)
                if (j < nb && !bad) {
                    const double d = readlane_f64(a[j], j);
                    if (!(d > 0.0) || !isfinite(d)) {
                        bad = c0 + j + 1;
                    } else {
                        const double sq = sqrt(d), inv = 1.0 / sq;
                        if (i == j) dinv = inv;
                        a[j] = i > j ? a[j] * inv : (i == j ? sq : 0.0);
#pragma unroll
                        for (int l = j + 1; l < NB; ++l) a[l] = fma(-a[j], readlane_f64(a[j], l), a[l]);
                    }
                }
            }
            if (lane == 0) s_bad = bad;
            if (!bad) {
                if (lane < NB) {
#pragma unroll
                    for (int c = 0; c < NB; ++c) sD[i * DP + c] = (i < nb && c < nb && c <= i) ? a[c] : 0.0;
                    sInv[i] = i < nb ? dinv : 0.0;
                }
                wave_sync_lds();
                // V = L_dd^-1 by forward elimination on the identity: step j
                // scales row j by 1 / L[j][j] and removes L[i][j] times it from
                // the rows i > j (L[i][j] read back from LDS, so only v[] stays
                // in registers)
                double v[NB];
#pragma unroll
                for (int c = 0; c < NB; ++c) v[c] = i == c ? 1.0 : 0.0;
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    if (j < nb) {
                        const double m = i > j ? sD[i * DP + j] : 0.0;
                        const double sj = i == j ? sInv[i] : 1.0;
#pragma unroll
                        for (int c = 0; c <= j; ++c) {
                            v[c] *= sj;
                            v[c] = fma(-m, readlane_f64(v[c], j), v[c]);
                        }
                    }
                }
                if (lane < NB) {
#pragma unroll
                    for (int c = 0; c < NB; ++c) sV[i * DP + c] = (i < nb && c < nb && c <= i) ? v[c] : 0.0;
                }
            }
        }
        __syncthreads();
        if (s_bad) break;
        for (int e = tid; e < NB * NB; e += NT) {
            const int i = e / NB, j = e % NB;
            if (i < nb && j <= i) L[(int64_t)(c0 + i) * P + c0 + j] = sD[i * DP + j];
            if (i < nb && j < i) L[(int64_t)(c0 + j) * P + c0 + i] = sV[i * DP + j];   // V, transposed, above
        }
        // rows below, solved against the diagonal block inside their passes
        for (int rt = c0 + NB; rt < P; rt += TR) {
            switch (min((P - rt + 31) / 32, TR / 32)) {
                case 1: gemm_pass(std::integral_constant<int, 1>(), std::true_type(), rt); break;
                case 2: gemm_pass(std::integral_constant<int, 2>(), std::true_type(), rt); break;
                case 3: gemm_pass(std::integral_constant<int, 3>(), std::true_type(), rt); break;
                case 4: gemm_pass(std::integral_constant<int, 4>(), std::true_type(), rt); break;
                case 5: gemm_pass(std::integral_constant<int, 5>(), std::true_type(), rt); break;
                default: gemm_pass(std::integral_constant<int, TR / 32>(), std::true_type(), rt); break;
            }
        }
    }
    if (s_bad) {
        if (tid == 0) info[m] = s_bad;
        for (int64_t e = tid; e < (int64_t)out_rows * d_t; e += NT) Wm[e] = 0.f;
        return;
    }

    // ================= 2., 3. substitutions (Z then W~ in Z)
    double *sL = sh + OFF_L, *sZ = sh + OFF_Z, *sR = sh + OFF_R;
    const int ri = tid >> 5, cj = tid & 31;            // apply_inv: rows ri + 8 q, columns cj + 32 n
    // The panel products on the matrix cores: wave w owns columns 32 w .. 32 w + 31
    // (two 16-column tiles) of both 16-row tiles; element e of acc[rt][ct] is
    // row 16 rt + lane / 16 + 4 e, column 32 w + 16 ct + lane % 16.
    const int lr = lane & 15, lk = lane >> 4;
    auto out_row = [&](int rt, int e) { return 16 * rt + lk + 4 * e; };
    auto out_col = [&](int ct) { return 32 * wave + 16 * ct + lr; };
    // acc = sum over k in [k_lo, k_hi) of Lop(i, k) Z[k][c], where
    // Lop(i, k) = L[c0 + i][k] (forward) or L[k][c0 + i] (backward).
    auto panel_gemm = [&](f64x4_t (&acc)[2][2], int c0, int nb, int k_lo, int k_hi, bool backward) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) acc[rt][ct] = f64x4_t{0.0, 0.0, 0.0, 0.0};
        const int nch = (k_hi - k_lo + KS - 1) / KS;
        double pl[LQ], pz[ZQ];
        auto fetch = [&](int ch) {
            const int k0 = k_lo + ch * KS;
#pragma unroll
            for (int q = 0; q < LQ; ++q) {              // 32 x KS operand: (i, kk)
                const int e = tid + NT * q;
                int i, kk;
                if (backward) { kk = e / NB; i = e % NB; } else { i = e / KS; kk = e % KS; }
                const int k = k0 + kk;
                pl[q] = (i < nb && k < k_hi) ? (backward ? L[(int64_t)k * P + c0 + i] : L[(int64_t)(c0 + i) * P + k])
                                             : 0.0;
            }
#pragma unroll
            for (int q = 0; q < ZQ; ++q) {              // KS x 128 operand: (kk, c)
                const int e = tid + NT * q;
                const int kk = e / DTMAX, c = e % DTMAX;
                const int k = k0 + kk;
                pz[q] = (k < k_hi && c < d_t) ? Z[(int64_t)k * d_t + c] : 0.0;
            }
        };
        auto stash = [&](int buf) {
#pragma unroll
            for (int q = 0; q < LQ; ++q) {
                const int e = tid + NT * q;
                int i, kk;
                if (backward) { kk = e / NB; i = e % NB; } else { i = e / KS; kk = e % KS; }
                sL[buf * NB * KSP + i * KSP + kk] = pl[q];
            }
#pragma unroll
            for (int q = 0; q < ZQ; ++q) {
                const int e = tid + NT * q;
                sZ[buf * KS * ZP + (e / DTMAX) * ZP + e % DTMAX] = pz[q];
            }
        };
        if (nch > 0) fetch(0);
        for (int ch = 0; ch < nch; ++ch) {
            stash(ch & 1);
            __syncthreads();
            if (ch + 1 < nch) fetch(ch + 1);
            const double *a = sL + (ch & 1) * NB * KSP, *b = sZ + (ch & 1) * KS * ZP;
#pragma unroll
            for (int s4 = 0; s4 < KS / 4; ++s4) {
                const int kk = 4 * s4 + lk;
                const double a0 = a[lr * KSP + kk], a1 = a[(16 + lr) * KSP + kk];
                const double b0 = b[kk * ZP + out_col(0)], b1 = b[kk * ZP + out_col(1)];
                acc[0][0] = mfma_f64(a0, b0, acc[0][0]);
                acc[0][1] = mfma_f64(a0, b1, acc[0][1]);
                acc[1][0] = mfma_f64(a1, b0, acc[1][0]);
                acc[1][1] = mfma_f64(a1, b1, acc[1][1]);
            }
        }
        __syncthreads();                                // the chunks' space becomes the panel rhs
    };

    // Z[c0 + i][c] = sum_k V[i][k] R[k][c]  (forward, V = L_dd^-1), or
    //               sum_k V[k][i] R[k][c]  (backward, V^T = L_dd^-T), R the panel
    // right-hand sides in sR; 4 x 4 outputs per thread.
    auto apply_inv = [&](int c0, int nb, bool transposed) {
        double acc[4][4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int n = 0; n < 4; ++n) acc[q][n] = 0.0;
#pragma unroll 4
        for (int k = 0; k < NB; ++k) {
            double av[4], bv[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) av[q] = transposed ? sV[k * DP + ri + 8 * q] : sV[(ri + 8 * q) * DP + k];
#pragma unroll
            for (int n = 0; n < 4; ++n) bv[n] = sR[k * ZP + cj + 32 * n];
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int n = 0; n < 4; ++n) acc[q][n] = fma(av[q], bv[n], acc[q][n]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int n = 0; n < 4; ++n) {
                const int i = ri + 8 * q, c = cj + 32 * n;
                if (i < nb && c < d_t) Z[(int64_t)(c0 + i) * d_t + c] = acc[q][n];
            }
    };
    // forward: Z[c0:c1] = L_dd^-1 (C[c0:c1] - L[c0:c1, :c0] Z[:c0])
    for (int c0 = 0; c0 < P; c0 += NB) {
        const int nb = min(NB, P - c0);
        f64x4_t acc[2][2];
        panel_gemm(acc, c0, nb, 0, c0, false);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int i = out_row(rt, e), c = out_col(ct);
                    sR[i * ZP + c] = (i < nb && c < d_t) ? (double)Cm[(int64_t)(c0 + i) * d_t + c] - acc[rt][ct][e] : 0.0;
                }
        load_inv(c0, nb);
        __syncthreads();
        apply_inv(c0, nb, false);
        __syncthreads();
    }
    // backward: W[c0:c1] = L_dd^-T (Z[c0:c1] - L[c1:, c0:c1]^T W[c1:])
    const int last = ((P - 1) / NB) * NB;
    for (int c0 = last; c0 >= 0; c0 -= NB) {
        const int nb = min(NB, P - c0), c1 = c0 + nb;
        f64x4_t acc[2][2];
        panel_gemm(acc, c0, nb, c1, P, true);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int ct = 0; ct < 2; ++ct)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int i = out_row(rt, e), c = out_col(ct);
                    sR[i * ZP + c] = (i < nb && c < d_t) ? Z[(int64_t)(c0 + i) * d_t + c] - acc[rt][ct][e] : 0.0;
                }
        load_inv(c0, nb);
        __syncthreads();
        apply_inv(c0, nb, true);
        __syncthreads();
    }

    // ================= 4. maps (and, centered, the bias row b = mu_y - W^T mu_x in fp64)
    for (int64_t e = tid; e < (int64_t)P * d_t; e += NT) Wm[e] = (float)Z[e];
    if (sm) {
        for (int c = tid; c < d_t; c += NT) {
            double b = sw != 0.0 ? sm[1 + P + c] / sw : 0.0;
            if (sw != 0.0)
                for (int i = 0; i < P; ++i) b -= Z[(int64_t)i * d_t + c] * (sm[1 + i] / sw);
            Wm[(int64_t)P * d_t + c] = (float)b;
        }
    }
    if (tid == 0) info[m] = 0;
}

}  // namespace

int64_t solve_blocked_bytes_per_system(int32_t P, int32_t d_t) {
    return ((int64_t)P * P + (int64_t)P * d_t) * (int64_t)sizeof(double);
}

hipError_t launch_solve_blocked(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C, float lambda,
                                uint32_t flags, void *ws, int64_t ws_bytes, float *maps, int32_t *info,
                                hipStream_t s, const double *csums) {
    if (n_maps == 0) return hipSuccess;
    if (d_t > DTMAX || P < 2) return hipErrorInvalidValue;
    const int64_t per = solve_blocked_bytes_per_system(P, d_t);
    const int64_t stride = per / (int64_t)sizeof(double);
    const int64_t batch = ws_bytes / per;
    if (batch < 1) return hipErrorInvalidValue;
    for (int32_t m0 = 0; m0 < n_maps; m0 += (int32_t)std::min<int64_t>(batch, n_maps)) {
        const int32_t nb = (int32_t)std::min<int64_t>(batch, n_maps - m0);
        hipLaunchKernelGGL(chol_solve_kernel, dim3(nb), dim3(NT), 0, s, P, d_t, G, C, lambda, flags, (double *)ws,
                           stride, m0, maps, info, csums);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Allocation-free variant: the factors live in `scratch`, a fixed device array
// that the code object carries (every GPU the library runs on holds its own
// copy until the process ends).  Its device address is looked up once per
// device, with that device current, on the first call there; host code never
// passes the array's name itself to a kernel (on the host it only names the
// variable).  Calls that overlap on one GPU share the array and race.
static __device__ __align__(256) double scratch[kStaticSolveScratchBytes / sizeof(double)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t static_solve_scratch(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

hipError_t launch_solve_blocked_static(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C,
                                       float lambda, uint32_t flags, float *maps, int32_t *info, hipStream_t s) {
    void *ws = nullptr;
    const hipError_t e = static_solve_scratch(&ws);
    if (e != hipSuccess) return e;
    return launch_solve_blocked(n_maps, P, d_t, G, C, lambda, flags, ws, kStaticSolveScratchBytes, maps, info, s);
}

}  // namespace cb

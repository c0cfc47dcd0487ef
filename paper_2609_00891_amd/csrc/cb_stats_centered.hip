// cb_stats_centered.hip -- two-pass centered statistics on gfx950.
//
// CacheBridge Sec. 3.4 (Eq. fusedstats) forms its moments in two passes:
// weighted means first, then the centered moments
//     A = sum_t w_t (x_t - mu_x)(x_t - mu_x)^T,
//     B = sum_t w_t (x_t - mu_x)(y_t - mu_y)^T.
// Centering before the products keeps A and B accurate when channels carry
// large means, where forming them from uncentered moments cancels.
//
// means_kernel (pass 1, one workgroup per (item, tile chunk), the units of
// the statistics kernel): every thread owns one 16-byte chunk (8 channels)
// of one of the item's rows and a strided set of the chunk's tokens, and
// sums w and w * value in fp64 (the products of a bf16 value and an fp32
// weight are exact in fp64).  The rows of the workgroup are combined through
// LDS and the unit's fp64 partial is written to the plan's workspace;
// means_reduce_kernel adds the partials of all chunks, in a fixed order, into
// the caller's fp64 sums.  The pass reads every cache row of the call once.
//
// stats_kernel<..., CENTER = true> (pass 2) is the streaming moments kernel
// with the folded operand w (x - mu_x); the reduction then subtracts
// e mu^T with e = sum w (x - mu_x), which leaves A and B (see reduce_kernel).
#include "cb_stats_kernel.h"

namespace cb {
namespace {

template <int DS, int DT>
struct MCfg {
    static constexpr int NCBX = DS / 8, NCBY = DT / 8;          // 16-byte chunks per row
    static constexpr int NS = 1 + DS + DT;                      // sums per map
    static constexpr int MAXR = 256 / (NCBX + NCBY);            // token rows of an item with one map
    static constexpr int SLOTD = Cfg<DS, DT>::SLOT / 2;         // workspace slot in doubles
    static_assert(Cfg<DS, DT>::SLOT % 2 == 0 && SLOTD >= NS, "an fp64 partial must fit a workspace slot");
};

// Pass 1 for one (item, chunk) unit.  Columns of a token: the 16-byte chunks
// of x0 and y0, then y1 (x shared by both maps) or x1 and y1.  Thread
// (row, col) sums the chunk's tokens row, row + R, row + 2R, ... of column
// col.  A shared x chunk is summed with both maps' weights.
template <int DS, int DT>
__global__ __launch_bounds__(256) void means_kernel(StatsArgs a) {
    using M = MCfg<DS, DT>;
    constexpr int NCBX = M::NCBX, NCBY = M::NCBY, NS = M::NS;
    __shared__ double red[M::MAXR][2 * NS];

    const int tid = threadIdx.x;
    const int unit = blockIdx.x;
    const int item_id = unit % a.n_items, chunk = unit / a.n_items;
    const StatsItem *it = a.items + item_id;
    const int n_slots = it->n_slots;
    const int nt = n_slots == 1 ? 2 : (it->shared_x ? 3 : 4);
    const int ncol = nt == 2 ? NCBX + NCBY : nt == 3 ? NCBX + 2 * NCBY : 2 * NCBX + 2 * NCBY;
    const int R = 256 / ncol;
    const int col = tid % ncol, row = tid / ncol;
    const int tile_begin = chunk * a.chunk_tiles;
    const int n_tiles = min(a.n_tiles, tile_begin + a.chunk_tiles) - tile_begin;
    if (n_tiles <= 0) return;                                  // the same in every thread

    // column -> tensor (0 x0, 1 y0, 2 x1, 3 y1) and chunk within its row
    int ten, cc;
    if (col < NCBX) { ten = 0; cc = col; }
    else if (col < NCBX + NCBY) { ten = 1; cc = col - NCBX; }
    else if (nt == 3) { ten = 3; cc = col - NCBX - NCBY; }
    else if (col < 2 * NCBX + NCBY) { ten = 2; cc = col - NCBX - NCBY; }
    else { ten = 3; cc = col - 2 * NCBX - NCBY; }
    const int slot = ten >> 1;
    const bool isx = (ten & 1) == 0;
    const bool dual = nt == 3 && ten == 0;                     // x0 also feeds map slot 1
    const Strides &st = isx ? a.ss : a.ts;
    const uint16_t *base = isx ? a.src + it->src_layer[slot] * st.layer + it->kv[slot] * st.kv + it->src_head[slot] * st.head
                               : a.tgt + it->tgt_layer[slot] * st.layer + it->kv[slot] * st.kv + it->tgt_head[slot] * st.head;
    base += 8 * cc;
    const float *wp = a.w + (int64_t)it->wrow[slot] * a.w_row_stride;
    const float *wq = a.w + (int64_t)it->wrow[1] * a.w_row_stride;

    double acc[8], acc2[8], sw = 0.0;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = acc2[e] = 0.0;
    const int nq = n_tiles * kStatsTileTokens;
    if (row < R) {
        for (int q0 = row; q0 < nq; q0 += 4 * R) {
            uint4 v[4];
            float wa[4], wb[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int q = q0 + k * R;
                const uint32_t u = (uint32_t)(tile_begin + (q >> 5));
                const uint32_t seq = fastdiv(u, a.TPS);
                const uint32_t tok = (u - seq * a.TPS.d) * kStatsTileTokens + (uint32_t)(q & 31);
                const bool ok = q < nq && tok < a.seq_len;       // absent tokens read the zero buffer
                const int64_t widx = (int64_t)seq * a.seq_len + tok;
                const uint4 *px = ok ? (const uint4 *)(base + (int64_t)seq * st.seq + (int64_t)tok * st.tok)
                                     : (const uint4 *)a.zero;
                v[k] = *px;
                wa[k] = ok ? wp[widx] : 0.f;
                wb[k] = (ok && dual) ? wq[widx] : 0.f;
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t xv[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
                const double w0 = wa[k], w1 = wb[k];
                sw += w0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[2 * e] = __builtin_fma(w0, (double)bf_lo(xv[e]), acc[2 * e]);
                    acc[2 * e + 1] = __builtin_fma(w0, (double)bf_hi(xv[e]), acc[2 * e + 1]);
                }
                if (dual) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        acc2[2 * e] = __builtin_fma(w1, (double)bf_lo(xv[e]), acc2[2 * e]);
                        acc2[2 * e + 1] = __builtin_fma(w1, (double)bf_hi(xv[e]), acc2[2 * e + 1]);
                    }
                }
            }
        }
        // this thread's entries of the unit's sums (slot, index)
        const int off = slot * NS + (isx ? 1 + 8 * cc : 1 + DS + 8 * cc);
#pragma unroll
        for (int e = 0; e < 8; ++e) red[row][off + e] = acc[e];
        if (dual) {
#pragma unroll
            for (int e = 0; e < 8; ++e) red[row][NS + 1 + 8 * cc + e] = acc2[e];
        }
        if (!isx && cc == 0) red[row][slot * NS] = sw;        // sum w of the slot, once per slot
    }
    __syncthreads();
    double *dst = (double *)a.partials + (int64_t)unit * 2 * M::SLOTD;
    for (int idx = tid; idx < n_slots * NS; idx += 256) {
        double s = 0.0;
        for (int r = 0; r < R; ++r) s += red[r][idx];
        const int sl = idx >= NS ? 1 : 0;
        dst[sl * M::SLOTD + (idx - sl * NS)] = s;
    }
}

// sums[m] += the fp64 partials of map m over all chunks, in chunk order.
template <int DS, int DT>
__global__ __launch_bounds__(256) void means_reduce_kernel(ReduceArgs a) {
    using M = MCfg<DS, DT>;
    const int m = blockIdx.x;
    const int item = a.map_item[m], slot = a.map_slot[m];
    const double *part = (const double *)a.partials + ((int64_t)item * 2 + slot) * M::SLOTD;
    const int64_t chunk_stride = (int64_t)a.n_items * 2 * M::SLOTD;
    for (int e = threadIdx.x; e < M::NS; e += 256) {
        double s = 0.0;
        for (int ch = 0; ch < a.n_chunks; ++ch) s += part[ch * chunk_stride + e];
        a.sums[(int64_t)m * M::NS + e] += s;
    }
}

template <int DS, int DT>
hipError_t launch_means_t(const StatsArgs &a, hipStream_t s) {
    const int grid = a.n_items * a.n_chunks;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL((means_kernel<DS, DT>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int DS, int DT>
hipError_t launch_means_reduce_t(const ReduceArgs &a, hipStream_t s) {
    if (a.n_maps == 0) return hipSuccess;
    hipLaunchKernelGGL((means_reduce_kernel<DS, DT>), dim3(a.n_maps), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int DS, int DT>
hipError_t launch_stats_centered_t(const StatsArgs &a, hipStream_t s) {
    using K = Cfg<DS, DT>;
    const int grid = a.n_items * a.n_chunks;
    if (grid == 0) return hipSuccess;
    if (a.seq_len % K::KT == 0)
        hipLaunchKernelGGL((stats_kernel<DS, DT, false, true>), dim3(grid), dim3(K::NT), 0, s, a);
    else
        hipLaunchKernelGGL((stats_kernel<DS, DT, true, true>), dim3(grid), dim3(K::NT), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_means(int d_s, int d_t, const StatsArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_means_t, d_s, d_t, a, s);
}

hipError_t launch_means_reduce(int d_s, int d_t, const ReduceArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_means_reduce_t, d_s, d_t, a, s);
}

hipError_t launch_stats_centered(int d_s, int d_t, const StatsArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_stats_centered_t, d_s, d_t, a, s);
}

}  // namespace cb

// cb_stats_centered.hip -- two-pass centered statistics on gfx950.
//
// CacheBridge Sec. 3.4 (Eq. fusedstats) forms its moments in two passes:
// weighted means first, then the centered moments
//     A = sum_t w_t (x_t - mu_x)(x_t - mu_x)^T,
//     B = sum_t w_t (x_t - mu_x)(y_t - mu_y)^T.
// Centering before the products keeps A and B accurate when channels carry
// large means, where forming them from uncentered moments cancels.
//
// means_kernel (pass 1, one workgroup per (item, tile chunk)): every thread
// owns one 16-byte chunk (8 channels) of one of the item's rows and a strided
// set of each tile's tokens, and sums w and w * value in fp64 (the products of
// a bf16 value and an fp32 weight are exact in fp64).  The rows of the
// workgroup are combined through LDS and the unit's fp64 partial is written to
// the plan's workspace; means_reduce_kernel adds the partials of all chunks, in
// a fixed order, into the caller's fp64 sums.  The pass reads every cache row
// of the call once.
//
// stats_kernel<..., CENTER = true> (pass 2) is the streaming moments kernel
// with the folded operand w (x - mu_x); the reduction then subtracts
// e mu^T with e = sum w (x - mu_x), which leaves A and B (see reduce_kernel).
#include "cb_stats_kernel.h"

namespace cb {
namespace {

// SQ: also the per-channel sums of squares (sum w x^2, sum w y^2).
template <int DS, int DT, bool SQ>
struct MCfg {
    static constexpr int NCBX = DS / 8, NCBY = DT / 8;          // 16-byte chunks per row
    static constexpr int NS = 1 + DS + DT;                      // sums per map
    static constexpr int NQ = SQ ? DS + DT : 0;                 // sums of squares per map
    static constexpr int NE = NS + NQ;                          // partial entries per map
    static constexpr int MAXR = 256 / (NCBX + NCBY);            // token rows of an item with one map
};

// Geometry of pass 1 for an item of NSL maps: NCOL 16-byte chunks per token
// (x0 y0, or x0 y0 x1 y1; x0, or x0 x1, when YS is false because none of the
// item's maps carries target sums), R token rows per workgroup pass (at most
// the rows of the reduction buffer), J loads per thread per 32-token tile.
template <int DS, int DT, int NSL, bool YS>
struct MGeo {
    static constexpr int NCBX = DS / 8, NCBY = DT / 8;
    static constexpr int NCOL = NSL * (YS ? NCBX + NCBY : NCBX);
    static constexpr int R = 256 / NCOL < 256 / (NCBX + NCBY) ? 256 / NCOL : 256 / (NCBX + NCBY);
    static constexpr int J = (kStatsTileTokens + R - 1) / R;
};

// Pass 1 for one (item, chunk) unit.  Thread (row, col) owns 16-byte chunk
// col of the token's concatenated rows [x0 | y0 | x1 | y1] and tokens row,
// row + R, ... of every tile.  When both maps read one source block, x1 is x0
// again: its chunks are loaded by the same wave instruction as x0's, so the
// repeated lines do not reach HBM twice.  Tiles are whole 32-token runs of
// one sequence, so their position is computed once per tile (the same in
// every thread).
template <int DS, int DT, bool SQ, int NSL, bool YS>
__device__ __forceinline__ void means_unit(const StatsArgs &a, const StatsItem *it, int tile_begin, int n_tiles,
                                           double (*red)[2 * MCfg<DS, DT, SQ>::NE]) {
    using M = MCfg<DS, DT, SQ>;
    using Gm = MGeo<DS, DT, NSL, YS>;
    constexpr int NCBX = M::NCBX, NCBY = M::NCBY, NS = M::NS, NE = M::NE, R = Gm::R, J = Gm::J;
    const int tid = threadIdx.x;
    const int col = tid % Gm::NCOL, row = tid / Gm::NCOL;
    if (row >= R) return;

    // column -> map slot, x or y row, and chunk within the row
    constexpr int NPS = YS ? NCBX + NCBY : NCBX;                 // columns per slot
    const int slot = col / NPS;
    const int cs = col - slot * NPS;
    const bool isx = cs < NCBX;
    const int cc = isx ? cs : cs - NCBX;
    const Strides st = isx ? a.ss : a.ts;
    const uint16_t *base = isx ? a.src + it->src_layer[slot] * st.layer + it->kv[slot] * st.kv + it->src_head[slot] * st.head
                               : a.tgt + it->tgt_layer[slot] * st.layer + it->kv[slot] * st.kv + it->tgt_head[slot] * st.head;
    base += 8 * cc + (int64_t)row * st.tok;
    const float *wp = a.w + (int64_t)it->wrow[slot] * a.w_row_stride + row;
    const bool load = isx || it->own_y[slot];                   // target rows: the owner map's item only
    const int64_t jstep = (int64_t)R * st.tok;                  // elements between a thread's tokens

    double acc[8], acq[8], sw = 0.0;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = acq[e] = 0.0;
    for (int t = 0; t < n_tiles; ++t) {
        const uint32_t u = (uint32_t)(tile_begin + t);
        const uint32_t seq = fastdiv(u, a.TPS);
        const uint32_t tt0 = (u - seq * a.TPS.d) * kStatsTileTokens;
        const int nvalid = (int)min((uint32_t)kStatsTileTokens, a.seq_len - tt0);
        const uint16_t *p = base + (int64_t)seq * st.seq + (int64_t)tt0 * st.tok;
        const int64_t w0 = (int64_t)seq * a.seq_len + tt0;
        uint4 v[J];
        float wa[J];
#pragma unroll
        for (int j = 0; j < J; ++j) {
            v[j] = make_uint4(0u, 0u, 0u, 0u);
            wa[j] = 0.f;
            if (row + j * R < nvalid) {
                if (load) v[j] = *(const uint4 *)(p + j * jstep);
                wa[j] = wp[w0 + j * R];
            }
        }
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const uint32_t xv[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
            const double ww = wa[j];
            sw += ww;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const double v0 = (double)bf_lo(xv[e]), v1 = (double)bf_hi(xv[e]);
                if constexpr (SQ) {
                    const double t0 = ww * v0, t1 = ww * v1;        // exact: 24 + 8 significant bits
                    acc[2 * e] += t0;
                    acc[2 * e + 1] += t1;
                    acq[2 * e] = __builtin_fma(t0, v0, acq[2 * e]);   // exact product, rounded sum
                    acq[2 * e + 1] = __builtin_fma(t1, v1, acq[2 * e + 1]);
                } else {
                    acc[2 * e] = __builtin_fma(ww, v0, acc[2 * e]);
                    acc[2 * e + 1] = __builtin_fma(ww, v1, acc[2 * e + 1]);
                }
            }
        }
    }
    // this thread's entries of the unit's partial: per slot [sums (NS) | squares (NQ)]
    const int off = slot * NE + (isx ? 1 + 8 * cc : 1 + DS + 8 * cc);
#pragma unroll
    for (int e = 0; e < 8; ++e) red[row][off + e] = acc[e];
    if constexpr (SQ) {
        const int offq = slot * NE + NS + (isx ? 8 * cc : DS + 8 * cc);
#pragma unroll
        for (int e = 0; e < 8; ++e) red[row][offq + e] = acq[e];
    }
    if (!isx && cc == 0) red[row][slot * NE] = sw;            // sum w of the slot, once per slot
}

// One workgroup per (item, chunk) unit: the unit's rows are combined through
// LDS in a fixed order and written as an fp64 partial [unit][2][NE].
template <int DS, int DT, bool SQ>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(SQ ? 2 : 4)))
void means_kernel(StatsArgs a) {
    using M = MCfg<DS, DT, SQ>;
    constexpr int NE = M::NE;
    __shared__ double red[M::MAXR][2 * NE];
    const int unit = blockIdx.x;
    const int item_id = unit % a.n_items, chunk = unit / a.n_items;
    const StatsItem *it = a.items + item_id;
    const int n_slots = it->n_slots;
    const int tile_begin = chunk * a.chunk_tiles;
    const int n_tiles = min(a.n_tiles, tile_begin + a.chunk_tiles) - tile_begin;
    if (n_tiles <= 0) return;                                  // the same in every thread
    int R;
    const bool ys = it->own_y[0] || (n_slots == 2 && it->own_y[1]);   // the same in every thread
    if (n_slots == 1) {
        if (ys) { means_unit<DS, DT, SQ, 1, true>(a, it, tile_begin, n_tiles, red); R = MGeo<DS, DT, 1, true>::R; }
        else { means_unit<DS, DT, SQ, 1, false>(a, it, tile_begin, n_tiles, red); R = MGeo<DS, DT, 1, false>::R; }
    } else {
        if (ys) { means_unit<DS, DT, SQ, 2, true>(a, it, tile_begin, n_tiles, red); R = MGeo<DS, DT, 2, true>::R; }
        else { means_unit<DS, DT, SQ, 2, false>(a, it, tile_begin, n_tiles, red); R = MGeo<DS, DT, 2, false>::R; }
    }
    __syncthreads();
    double *dst = (double *)a.partials + (int64_t)unit * 2 * NE;
    for (int idx = threadIdx.x; idx < n_slots * NE; idx += 256) {
        double s = 0.0;
        for (int r = 0; r < R; ++r) s += red[r][idx];
        dst[idx] = s;
    }
}

// sums[m] (and sq[m]) += the fp64 partials of map m over all chunks, in chunk order.
template <int DS, int DT, bool SQ>
__global__ __launch_bounds__(256) void means_reduce_kernel(ReduceArgs a) {
    using M = MCfg<DS, DT, SQ>;
    const int m = blockIdx.x;
    const int item = a.map_item[m], slot = a.map_slot[m];
    const int o = a.map_yown[m];                               // carries the target sums
    const double *part = (const double *)a.partials + ((int64_t)item * 2 + slot) * M::NE;
    const double *opart = (const double *)a.partials + ((int64_t)a.map_item[o] * 2 + a.map_slot[o]) * M::NE;
    const int64_t chunk_stride = (int64_t)a.n_items * 2 * M::NE;
    for (int e = threadIdx.x; e < M::NE; e += 256) {
        // sum w and the target sums come from the map that carries them (same weight row and target)
        const bool ysum = e == 0 || (e >= 1 + DS && e < M::NS) || e >= M::NS + DS;
        const double *src = ysum ? opart : part;
        double s = 0.0;
        for (int ch = 0; ch < a.n_chunks; ++ch) s += src[ch * chunk_stride + e];
        if (e < M::NS) a.sums[(int64_t)m * M::NS + e] += s;
        else a.sq[(int64_t)m * M::NQ + (e - M::NS)] += s;
    }
}

template <int DS, int DT>
hipError_t launch_means_t(const StatsArgs &a, bool sq, hipStream_t s) {
    const int grid = a.n_items * a.n_chunks;
    if (grid == 0) return hipSuccess;
    if (sq) hipLaunchKernelGGL((means_kernel<DS, DT, true>), dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((means_kernel<DS, DT, false>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int DS, int DT>
hipError_t launch_means_reduce_t(const ReduceArgs &a, hipStream_t s) {
    if (a.n_maps == 0) return hipSuccess;
    if (a.sq) hipLaunchKernelGGL((means_reduce_kernel<DS, DT, true>), dim3(a.n_maps), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((means_reduce_kernel<DS, DT, false>), dim3(a.n_maps), dim3(256), 0, s, a);
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

hipError_t launch_means(int d_s, int d_t, const StatsArgs &a, bool sq, hipStream_t s) {
    CB_DISPATCH(launch_means_t, d_s, d_t, a, sq, s);
}

hipError_t launch_means_reduce(int d_s, int d_t, const ReduceArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_means_reduce_t, d_s, d_t, a, s);
}

hipError_t launch_stats_centered(int d_s, int d_t, const StatsArgs &a, hipStream_t s) {
    CB_DISPATCH(launch_stats_centered_t, d_s, d_t, a, s);
}

}  // namespace cb

// cb_stats_rope.hip -- the statistics kernel with the rotary de-rotation of
// the keys folded into its gather (CacheBridge Sec. 2.1, Sec. 3.1: the maps
// are fitted in content coordinates, so RoPE is removed from the source and
// target keys before regression).  The K rows of each tile are turned back in
// LDS as they land, by the waves that copied them (see stats_wave in
// cb_stats_kernel.h); V rows and the moments are exactly those of the plain
// kernel.  Instantiated for d_s = d_t = 64 and 128, both pairings.
#include "cb_stats_kernel.h"

namespace cb {
namespace {

template <int D, int RS>
hipError_t launch_stats_rope_t(const StatsArgs &a, hipStream_t s) {
    using K = Cfg<D, D>;
    const int grid = a.n_items * a.n_chunks;
    if (grid == 0) return hipSuccess;
    if (a.seq_len % K::KT == 0)
        hipLaunchKernelGGL((stats_kernel<D, D, false, false, RS>), dim3(grid), dim3(K::NT), 0, s, a);
    else
        hipLaunchKernelGGL((stats_kernel<D, D, true, false, RS>), dim3(grid), dim3(K::NT), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_stats_rope(int d, int style, const StatsArgs &a, hipStream_t s) {
    if (d == 128) return style == 0 ? launch_stats_rope_t<128, 1>(a, s) : launch_stats_rope_t<128, 2>(a, s);
    if (d == 64) return style == 0 ? launch_stats_rope_t<64, 1>(a, s) : launch_stats_rope_t<64, 2>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace cb

// stats.hip -- block summaries: prefill build and streaming append (Sections 4.1, 4.2; Appendix E.1).
//
// One workgroup computes one block's summary with wg_block_stats (block_stats.h): the prefill strides
// over every (unit, block), the append recomputes each unit's active block after storing the new row.
// Build, append and the fused decode step share that routine, so an appended block's summary is
// bit-identical to the prefill one.
#include "block_stats.h"

namespace compkv {
namespace {

// Grid-stride over (unit, block); the workgroup summarizes one block per iteration.
template <int D>
__global__ __launch_bounds__(kThreads) void build_stats_kernel(Geom g, StatsArgs a) {
    __shared__ BlockStatsLds<D> L;
    const int xmax = g.xmax();
    for (int flat = blockIdx.x; flat < xmax * g.units(); flat += gridDim.x) {
        const int u = flat / xmax, b = flat % xmax;
        const int n = clamp_len(a.seq_lens[u / g.hkv], g.max_seq);
        const int X = (n + g.B - 1) / g.B;
        if (b >= X) continue;  // workgroup-uniform
        const int nb = min(g.B, n - b * g.B);
        const size_t row0 = (size_t)u * g.cap + (size_t)b * g.B;
        const size_t blk = (size_t)u * g.xcap + b;
        wg_block_stats<D>(a.K + row0 * D, a.V + row0 * D, nb, nullptr, nullptr, -1, g.r, g.layout,
                          a.kmean + blk * D, a.dvar + blk * g.r, a.vmean + blk * D, L);
    }
}

// grid = (units): workgroup u recomputes block n / B with the new row n = seq_lens (before the append)
// taken from k_new / v_new, then stores that row in the cache.
template <int D>
__global__ __launch_bounds__(kThreads) void append_stats_kernel(Geom g, StatsArgs a) {
    __shared__ BlockStatsLds<D> L;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int u = blockIdx.x;
    const int n = a.seq_lens[u / g.hkv];
    if (n < 0 || n >= g.cap) return;  // workgroup-uniform
    const int blk_id = n / g.B;
    const int nb = n - blk_id * g.B + 1;
    const uint16_t* kn = a.k_new + (size_t)u * D;
    const uint16_t* vn = a.v_new + (size_t)u * D;
    const size_t row0 = (size_t)u * g.cap + (size_t)blk_id * g.B;
    const size_t blk = (size_t)u * g.xcap + blk_id;
    wg_block_stats<D>(a.K + row0 * D, a.V + row0 * D, nb, kn, vn, nb - 1, g.r, g.layout, a.kmean + blk * D,
                      a.dvar + blk * g.r, a.vmean + blk * D, L);
    if (wave == 0) {  // the cache row (the summary above read it from k_new / v_new)
        const size_t row = (size_t)u * g.cap + n;
        for (int i = lane; i < D / 8; i += 64) {
            reinterpret_cast<uint4*>(a.K_out + row * D)[i] = reinterpret_cast<const uint4*>(kn)[i];
            reinterpret_cast<uint4*>(a.V_out + row * D)[i] = reinterpret_cast<const uint4*>(vn)[i];
        }
    }
}

}  // namespace

hipError_t launch_build_stats(const Geom& g, const StatsArgs& a, hipStream_t s) {
    const long long total = (long long)g.xmax() * g.units();
    dim3 grid(total < 4096 ? (unsigned)total : 4096u);
    if (g.D == 128)
        build_stats_kernel<128><<<grid, kThreads, 0, s>>>(g, a);
    else
        build_stats_kernel<64><<<grid, kThreads, 0, s>>>(g, a);
    return hipGetLastError();
}

hipError_t launch_append_stats(const Geom& g, const StatsArgs& a, hipStream_t s) {
    dim3 grid(g.units());
    if (g.D == 128)
        append_stats_kernel<128><<<grid, kThreads, 0, s>>>(g, a);
    else
        append_stats_kernel<64><<<grid, kThreads, 0, s>>>(g, a);
    return hipGetLastError();
}

}  // namespace compkv

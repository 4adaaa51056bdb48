// stats.hip -- block summaries: prefill build and streaming append (Sections 4.1, 4.2; Appendix E.1).
//
// One wave64 computes one block's summary. A key row of d bf16 is read as d/8 lanes x 16 bytes, so a
// wave covers 64/(d/8) rows per load (4 rows for d = 128) and the loads of consecutive lanes are
// contiguous. Each lane accumulates its 8 coordinates over the rows it visits; the row groups are then
// combined with cross-lane adds. Rows are loaded in batches of 8 load steps (32 rows for d = 128), all
// loads of a batch issued before use. Two passes (mean, then squared deviations) keep the variance
// numerically stable; a block that fits in one batch is still in registers for the second pass, a
// larger one is re-read from L1/L2. Per-coordinate sums of squared deviations go through LDS to form
// the r group averages.
//
// build and append share wave_block_stats with the same lane-to-row mapping, so an appended block's
// summary is bit-identical to the prefill one.
#include "block_stats.h"

namespace compkv {
namespace {

// Grid-stride over (unit, group of four blocks) with a capped grid; wave w of a group summarizes its
// block w.
template <int D>
__global__ __launch_bounds__(kThreads) void build_stats_kernel(Geom g, StatsArgs a) {
    __shared__ float m2s[4][D];
    const int wave = threadIdx.x >> 6;
    const int quads = (g.xmax() + 3) / 4;
    for (int flat = blockIdx.x; flat < quads * g.units(); flat += gridDim.x) {
    const int u = flat / quads;
    const int b = (flat % quads) * 4 + wave;
    const int n = clamp_len(a.seq_lens[u / g.hkv], g.max_seq);
    const int X = (n + g.B - 1) / g.B;
    const bool active = b < X;
    const int nb = active ? min(g.B, n - b * g.B) : 0;
    const size_t row0 = (size_t)u * g.cap + (size_t)b * g.B;
    const size_t blk = (size_t)u * g.xcap + b;
    wave_block_stats<D>(a.K + row0 * D, a.V + row0 * D, nb, nullptr, nullptr, -1, g.r, g.layout,
                        a.kmean + blk * D, a.dvar + blk * g.r, a.vmean + blk * D, m2s[wave], active);
    }
}

// grid = (ceil(units / 4)); wave w of workgroup x appends to unit 4x + w.
template <int D>
__global__ __launch_bounds__(kThreads) void append_stats_kernel(Geom g, StatsArgs a) {
    __shared__ float m2s[4][D];
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int u = blockIdx.x * 4 + wave;
    const bool in_grid = u < g.units();
    const int n = in_grid ? a.seq_lens[u / g.hkv] : g.cap;
    const bool active = in_grid && n >= 0 && n < g.cap;
    int nb = 0, blk_id = 0;
    const uint16_t* kn = nullptr;
    const uint16_t* vn = nullptr;
    size_t row0 = 0;
    if (active) {
        blk_id = n / g.B;
        nb = n - blk_id * g.B + 1;
        kn = a.k_new + (size_t)u * D;
        vn = a.v_new + (size_t)u * D;
        row0 = (size_t)u * g.cap + (size_t)blk_id * g.B;
        // write the new row into the cache (the summary below reads it from k_new / v_new)
        const size_t row = (size_t)u * g.cap + n;
        for (int i = lane; i < D / 8; i += 64) {
            reinterpret_cast<uint4*>(a.K_out + row * D)[i] = reinterpret_cast<const uint4*>(kn)[i];
            reinterpret_cast<uint4*>(a.V_out + row * D)[i] = reinterpret_cast<const uint4*>(vn)[i];
        }
    }
    const size_t blk = (size_t)u * g.xcap + blk_id;
    wave_block_stats<D>(a.K + row0 * D, a.V + row0 * D, nb, kn, vn, nb - 1, g.r, g.layout,
                        a.kmean + blk * D, a.dvar + blk * g.r, a.vmean + blk * D, m2s[wave], active);
}

}  // namespace

hipError_t launch_build_stats(const Geom& g, const StatsArgs& a, hipStream_t s) {
    const int total = (g.xmax() + 3) / 4 * g.units();
    dim3 grid(total < 2048 ? total : 2048);
    if (g.D == 128)
        build_stats_kernel<128><<<grid, kThreads, 0, s>>>(g, a);
    else
        build_stats_kernel<64><<<grid, kThreads, 0, s>>>(g, a);
    return hipGetLastError();
}

hipError_t launch_append_stats(const Geom& g, const StatsArgs& a, hipStream_t s) {
    dim3 grid((g.units() + 3) / 4);
    if (g.D == 128)
        append_stats_kernel<128><<<grid, kThreads, 0, s>>>(g, a);
    else
        append_stats_kernel<64><<<grid, kThreads, 0, s>>>(g, a);
    return hipGetLastError();
}

}  // namespace compkv

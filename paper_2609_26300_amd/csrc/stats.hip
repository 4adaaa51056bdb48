// stats.hip -- block summaries: prefill build and streaming append (Sections 4.1, 4.2; Appendix E.1).
//
// One workgroup computes one block's summary with wg_block_stats (block_stats.h): the prefill strides
// over every (unit, block) (blocks of up to 32 rows at d = 128: one wave per block, same arithmetic),
// the append recomputes each unit's active block after storing the new row.
// Build, append and the fused decode step share that routine, so an appended block's summary is
// bit-identical to the prefill one.
#include "block_stats.h"

namespace compkv {
namespace {

// Grid-stride over (unit, block); the workgroup summarizes one block per iteration and requests the
// next block's rows before computing the current one.
template <int D>
__global__ __launch_bounds__(kThreads) void build_stats_kernel(Geom g, StatsArgs a) {
    __shared__ BlockStatsLds<D> L;
    const int xmax = g.xmax();
    const int total = xmax * g.units();
    struct Item {
        BlockSrc src;
        size_t blk;
        bool valid;
    };
    auto item = [&](int flat) {
        Item it{};
        it.valid = false;
        if (flat >= total) return it;
        const int u = flat / xmax, b = flat % xmax;
        const int n = clamp_len(a.seq_lens[u / g.hkv], g.max_seq);
        if (b >= (n + g.B - 1) / g.B) return it;
        const size_t row0 = (size_t)block_row0(g, u, b);
        it.src = BlockSrc{a.K + row0 * D, a.V + row0 * D, nullptr, nullptr, min(g.B, n - b * g.B), -1};
        it.blk = (size_t)u * g.xcap + b;
        it.valid = true;
        return it;
    };
    int flat = blockIdx.x;
    Item cur = item(flat);
    BlockRows rc;
    if (cur.valid) load_block_rows<D>(cur.src, 0, rc);
    while (flat < total) {  // workgroup-uniform
        const int nf = flat + gridDim.x;
        const Item nxt = item(nf);
        BlockRows rn;
        if (nxt.valid) load_block_rows<D>(nxt.src, 0, rn);
        if (cur.valid)
            block_stats_from<D>(cur.src, rc, g.r, g.layout, a.kmean + cur.blk * D, a.dvar + cur.blk * g.r,
                                a.vmean + cur.blk * D, L);
        cur = nxt;
        rc = rn;
        flat = nf;
    }
}

// Blocks of at most wave_stats_max_rows<D>() rows: each wave summarizes whole blocks on its own (no
// barrier, no LDS; bit-identical to the workgroup routine), consecutive waves taking consecutive
// blocks, every row of a block requested at once.
template <int D>
__global__ __launch_bounds__(kThreads) void build_stats_wave_kernel(Geom g, StatsArgs a) {
    constexpr int WPG = kThreads / 64;
    const int xmax = g.xmax();
    const int total = xmax * g.units();
    const int nwaves = gridDim.x * WPG;
    for (int flat = blockIdx.x * WPG + (threadIdx.x >> 6); flat < total; flat += nwaves) {  // wave-uniform
        const int u = flat / xmax, b = flat % xmax;
        const int n = clamp_len(a.seq_lens[u / g.hkv], g.max_seq);
        if (b >= (n + g.B - 1) / g.B) continue;
        const size_t row0 = (size_t)block_row0(g, u, b);
        const BlockSrc src{a.K + row0 * D, a.V + row0 * D, nullptr, nullptr, min(g.B, n - b * g.B), -1};
        const size_t blk = (size_t)u * g.xcap + b;
        wave_block_stats<D>(src, g.r, g.layout, a.kmean + blk * D, a.dvar + blk * g.r, a.vmean + blk * D);
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
    const size_t row0 = (size_t)block_row0(g, u, blk_id);
    const size_t blk = (size_t)u * g.xcap + blk_id;
    wg_block_stats<D>(a.K + row0 * D, a.V + row0 * D, nb, kn, vn, nb - 1, g.r, g.layout, a.kmean + blk * D,
                      a.dvar + blk * g.r, a.vmean + blk * D, L);
    if (wave == 0) {  // the cache row (the summary above read it from k_new / v_new)
        const size_t row = row0 + (n - blk_id * g.B);
        for (int i = lane; i < D / 8; i += 64) {
            reinterpret_cast<uint4*>(a.K_out + row * D)[i] = reinterpret_cast<const uint4*>(kn)[i];
            reinterpret_cast<uint4*>(a.V_out + row * D)[i] = reinterpret_cast<const uint4*>(vn)[i];
        }
    }
}

}  // namespace

template <int D>
void launch_build_d(const Geom& g, const StatsArgs& a, hipStream_t s) {
    const long long total = (long long)g.xmax() * g.units();
    if (g.B <= wave_stats_max_rows<D>()) {  // one wave per block
        const long long wgs = (total + kThreads / 64 - 1) / (kThreads / 64);
        const long long slots = resident_slots(build_stats_wave_kernel<D>);  // one resident round
        build_stats_wave_kernel<D><<<dim3((unsigned)(wgs < slots ? wgs : slots)), kThreads, 0, s>>>(g, a);
        return;
    }
    const long long slots = resident_slots(build_stats_kernel<D>);  // one resident round, grid-stride
    build_stats_kernel<D><<<dim3((unsigned)(total < slots ? total : slots)), kThreads, 0, s>>>(g, a);
}

hipError_t launch_build_stats(const Geom& g, const StatsArgs& a, hipStream_t s) {
    if (g.D == 128)
        launch_build_d<128>(g, a, s);
    else
        launch_build_d<64>(g, a, s);
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

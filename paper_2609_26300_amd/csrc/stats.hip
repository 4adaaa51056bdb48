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
#include "internal.h"

namespace compkv {
namespace {

// Sum the coordinates of group t (Appendix A.4) from a per-coordinate array in LDS.
__device__ float group_sum(const float* m2, int t, int D, int r, int layout) {
    float s = 0.0f;
    if (r == D) return m2[t];
    const int w = (D / 2) / r;  // frequency pairs per group
    if (layout == 0) {          // rotate-half: pair f = (f, f + D/2)
        for (int f = t * w; f < (t + 1) * w; ++f) s += m2[f] + m2[f + D / 2];
    } else {  // interleaved: pair f = (2f, 2f + 1)
        for (int i = 2 * t * w; i < 2 * (t + 1) * w; ++i) s += m2[i];
    }
    return s;
}

// Summary of one block of nb rows (row j at Kb + j*D). Row new_j (if >= 0) is read from k_new / v_new
// instead of the cache. m2s: D floats of LDS private to this wave. Called by whole waves; every wave
// of the workgroup must reach the trailing __syncthreads() the same number of times.
template <int D>
__device__ void wave_block_stats(const uint16_t* __restrict__ Kb, const uint16_t* __restrict__ Vb, int nb,
                                 const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
                                 int new_j, int r, int layout, float* __restrict__ km_out,
                                 float* __restrict__ dv_out, float* __restrict__ vm_out, float* m2s,
                                 bool active) {
    constexpr int LPR = D / 8;     // lanes per row
    constexpr int RPS = 64 / LPR;  // rows per load step
    constexpr int NS = 8;          // load steps held in registers (32 rows for d = 128)
    constexpr int BATCH = NS * RPS;
    const int lane = threadIdx.x & 63;
    const int ro = lane / LPR, li = lane % LPR;
    auto krow = [&](int j) { return (j == new_j) ? k_new : Kb + (size_t)j * D; };
    auto vrow = [&](int j) { return (j == new_j) ? v_new : Vb + (size_t)j * D; };
    float mk[8], mv[8], m2[8];
    if (active) {
        float sk[8] = {0, 0, 0, 0, 0, 0, 0, 0}, sv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        uint4 kw[NS];
        for (int j0 = 0; j0 < nb; j0 += BATCH) {
            uint4 vw[NS];
#pragma unroll
            for (int st = 0; st < NS; ++st) {  // every load of the batch before any use
                const int j = j0 + st * RPS + ro;
                kw[st] = j < nb ? *reinterpret_cast<const uint4*>(krow(j) + li * 8) : make_uint4(0, 0, 0, 0);
                vw[st] = j < nb ? *reinterpret_cast<const uint4*>(vrow(j) + li * 8) : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int st = 0; st < NS; ++st) {
                float kf[8], vf[8];
                unpack_bf16x8(kw[st], kf);
                unpack_bf16x8(vw[st], vf);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    sk[e] += kf[e];
                    sv[e] += vf[e];
                }
            }
        }
#pragma unroll
        for (int off = LPR; off < 64; off <<= 1)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                sk[e] += __shfl_xor(sk[e], off);
                sv[e] += __shfl_xor(sv[e], off);
            }
        const float fn = (float)nb;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            mk[e] = sk[e] / fn;
            mv[e] = sv[e] / fn;
            m2[e] = 0.0f;
        }
        // squared deviations; a block of one batch is still in registers
        for (int j0 = 0; j0 < nb; j0 += BATCH) {
            if (nb > BATCH) {
#pragma unroll
                for (int st = 0; st < NS; ++st) {
                    const int j = j0 + st * RPS + ro;
                    kw[st] = j < nb ? *reinterpret_cast<const uint4*>(krow(j) + li * 8) : make_uint4(0, 0, 0, 0);
                }
            }
#pragma unroll
            for (int st = 0; st < NS; ++st) {
                if (j0 + st * RPS + ro >= nb) continue;
                float kf[8];
                unpack_bf16x8(kw[st], kf);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float dev = kf[e] - mk[e];
                    m2[e] += dev * dev;
                }
            }
        }
#pragma unroll
        for (int off = LPR; off < 64; off <<= 1)
#pragma unroll
            for (int e = 0; e < 8; ++e) m2[e] += __shfl_xor(m2[e], off);
        if (ro == 0) {
            float4* kmo = reinterpret_cast<float4*>(km_out + li * 8);
            float4* vmo = reinterpret_cast<float4*>(vm_out + li * 8);
            kmo[0] = make_float4(mk[0], mk[1], mk[2], mk[3]);
            kmo[1] = make_float4(mk[4], mk[5], mk[6], mk[7]);
            vmo[0] = make_float4(mv[0], mv[1], mv[2], mv[3]);
            vmo[1] = make_float4(mv[4], mv[5], mv[6], mv[7]);
#pragma unroll
            for (int e = 0; e < 8; ++e) m2s[li * 8 + e] = m2[e];
        }
    }
    __syncthreads();
    if (active) {
        const float denom = (float)nb * (float)(D / r);
        for (int t = lane; t < r; t += 64) dv_out[t] = group_sum(m2s, t, D, r, layout) / denom;
    }
    __syncthreads();
}

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

// block_stats.h -- the block summary routine shared by the prefill, the append and the fused decode
// step (private to libcompkv). Every caller runs the same workgroup-wide routine, so a summary does not
// depend on which of them computed it (Section 4.2: an appended block's summary equals a rebuild).
#pragma once

#include "internal.h"

namespace compkv {

template <int D>
struct BlockStatsLds {
    float part[4][2][D];  // per-wave partial sums (key, value), later (squared deviations)
    alignas(16) float km[D];
    alignas(16) float vm[D];
    float dv[D];
};

// Summary of one block of nb >= 1 rows (row j at Kb + j*D; row new_j, if >= 0, is read from k_new /
// v_new instead of the cache): mean key, mean value and the r grouped population variances of
// Section 4.1 (Appendix A.4 groups). Called by all four waves of the workgroup with uniform arguments.
//
// A row of d bf16 is d/8 lanes x 16 bytes; a wave covers 64/(d/8) rows per load step and the workgroup
// four times that. Wave w takes rows 16s + 4w + (lane / 16) (for d = 128) of each step s, up to four
// steps per batch with every load of a batch issued before use. Per-lane sums over the rows, then
// cross-lane sums within the wave, then the four waves in a fixed order. Two passes (mean, then
// squared deviations from the mean) keep the variance stable; a block of at most one batch per wave
// (64 rows for d = 128) is still in registers for the second pass. On return the results are written
// to km_out / vm_out / dv_out and their copies in L.km / L.vm / L.dv are visible to the workgroup.
//
// The first batch's loads are separate (BlockRows / load_block_rows) so that a caller can request the
// next block's rows before computing the current one.
constexpr int kStatsSteps = 4;  // load steps per batch held in registers

struct BlockSrc {
    const uint16_t* Kb;
    const uint16_t* Vb;
    const uint16_t* k_new;
    const uint16_t* v_new;
    int nb, new_j;
};

struct BlockRows {
    uint4 kw[kStatsSteps], vw[kStatsSteps];
};

template <int D>
__device__ __forceinline__ int stats_row(int st) {
    constexpr int LPR = D / 8, RPW = 64 / LPR, RPG = 4 * RPW;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    return st * RPG + wave * RPW + lane / LPR;
}

template <int D>
__device__ __forceinline__ const uint16_t* stats_krow(const BlockSrc& b, int j) {
    return (j == b.new_j) ? b.k_new : b.Kb + (size_t)j * D;
}
template <int D>
__device__ __forceinline__ const uint16_t* stats_vrow(const BlockSrc& b, int j) {
    return (j == b.new_j) ? b.v_new : b.Vb + (size_t)j * D;
}

// rows of the batch starting at step s0 (branch-free: a row past the block reloads row 0, unused)
template <int D>
__device__ __forceinline__ void load_block_rows(const BlockSrc& b, int s0, BlockRows& R, bool values = true) {
    const int li = (threadIdx.x & 63) % (D / 8);
#pragma unroll
    for (int st = 0; st < kStatsSteps; ++st) {
        const int j = stats_row<D>(s0 + st);
        const int jj = j < b.nb ? j : 0;
        R.kw[st] = *reinterpret_cast<const uint4*>(stats_krow<D>(b, jj) + li * 8);
        if (values) R.vw[st] = *reinterpret_cast<const uint4*>(stats_vrow<D>(b, jj) + li * 8);
    }
}

// The summary from the rows of the first batch (already requested into R) and the rest of the block.
// In a workgroup larger than four waves only waves 0-3 work (`active`); every thread reaches the
// barriers.
template <int D>
__device__ void block_stats_from(const BlockSrc& b, BlockRows& R, int r, int layout, float* __restrict__ km_out,
                                 float* __restrict__ dv_out, float* __restrict__ vm_out, BlockStatsLds<D>& L,
                                 bool active = true) {
    constexpr int LPR = D / 8;     // lanes per row
    constexpr int RPW = 64 / LPR;  // rows per wave step
    constexpr int RPG = 4 * RPW;   // rows per workgroup step
    constexpr int NS = kStatsSteps;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ro = lane / LPR, li = lane % LPR;
    const int nb = b.nb;
    const int nsteps = (nb + RPG - 1) / RPG;

    float sk[8] = {0, 0, 0, 0, 0, 0, 0, 0}, sv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int s0 = 0; active && s0 < nsteps; s0 += NS) {
        if (s0 > 0) load_block_rows<D>(b, s0, R);
#pragma unroll
        for (int st = 0; st < NS; ++st) {
            const bool ok = stats_row<D>(s0 + st) < nb;
            float kf[8], vf[8];
            unpack_bf16x8(R.kw[st], kf);
            unpack_bf16x8(R.vw[st], vf);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                sk[e] += ok ? kf[e] : 0.0f;
                sv[e] += ok ? vf[e] : 0.0f;
            }
        }
    }
    if (active) {
#pragma unroll
        for (int off = LPR; off < 64; off <<= 1)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                sk[e] = xor_add(sk[e], off);
                sv[e] = xor_add(sv[e], off);
            }
    }
    if (active && ro == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            L.part[wave][0][li * 8 + e] = sk[e];
            L.part[wave][1][li * 8 + e] = sv[e];
        }
    }
    __syncthreads();
    const float fn = (float)nb;
    for (int i = tid; i < D; i += kThreads) {
        const float mk = ((L.part[0][0][i] + L.part[1][0][i]) + (L.part[2][0][i] + L.part[3][0][i])) / fn;
        const float mv = ((L.part[0][1][i] + L.part[1][1][i]) + (L.part[2][1][i] + L.part[3][1][i])) / fn;
        L.km[i] = mk;
        L.vm[i] = mv;
        km_out[i] = mk;
        vm_out[i] = mv;
    }
    __syncthreads();
    float mk[8], m2[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        mk[e] = L.km[li * 8 + e];
        m2[e] = 0.0f;
    }
    for (int s0 = 0; active && s0 < nsteps; s0 += NS) {
        if (nsteps > NS) load_block_rows<D>(b, s0, R, false);  // larger blocks: reload (L1/L2 hits)
#pragma unroll
        for (int st = 0; st < NS; ++st) {
            const bool ok = stats_row<D>(s0 + st) < nb;
            float kf[8];
            unpack_bf16x8(R.kw[st], kf);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float dev = kf[e] - mk[e];
                m2[e] += ok ? __fmul_rn(dev, dev) : 0.0f;  // (no fused multiply-add: same bits everywhere)
            }
        }
    }
    if (active) {
#pragma unroll
        for (int off = LPR; off < 64; off <<= 1)
#pragma unroll
            for (int e = 0; e < 8; ++e) m2[e] = xor_add(m2[e], off);
    }
    if (active && ro == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) L.part[wave][0][li * 8 + e] = m2[e];
    }
    __syncthreads();
    auto m2_of = [&](int i) { return (L.part[0][0][i] + L.part[1][0][i]) + (L.part[2][0][i] + L.part[3][0][i]); };
    if (r == D) {
        for (int t = tid; t < D; t += kThreads) {
            const float dv = m2_of(t) / fn;
            L.dv[t] = dv;
            dv_out[t] = dv;
        }
    } else if (wave == 0) {
        // group t = a run of (d/2)/r consecutive frequency pairs (Appendix A.4); lane f holds pair f
        const bool in = lane < D / 2;
        const int f = in ? lane : 0;
        const int ia = layout == 0 ? f : 2 * f, ib = layout == 0 ? f + D / 2 : 2 * f + 1;
        float e = in ? m2_of(ia) + m2_of(ib) : 0.0f;
        const int w = (D / 2) / r;
        for (int off = 1; off < w; off <<= 1) e = xor_add(e, off);
        if (in && lane % w == 0) {
            const float dv = e / (fn * (float)(D / r));
            L.dv[lane / w] = dv;
            dv_out[lane / w] = dv;
        }
    }
    __syncthreads();
}

// The same summary computed by ONE wave (no barrier, no LDS), for blocks of at most two workgroup load
// steps (nb <= 2 * 4 * 64/(d/8): 32 rows at d = 128, 64 at d = 64). The wave plays the four waves of the
// workgroup routine in turn (virtual wave v takes the rows the real wave v takes there) and adds in
// exactly the same order: per lane over the steps, the butterflies over the row groups, the four waves'
// sums as (w0 + w1) + (w2 + w3), the pair sums and the group butterflies over lanes = pairs. So its
// results are bit-identical to block_stats_from's, which the append and the fused step keep using.
template <int D>
constexpr int wave_stats_max_rows() {
    return 2 * 4 * (64 / (D / 8));
}

template <int D>
__device__ void wave_block_stats(const BlockSrc& b, int r, int layout, float* __restrict__ km_out,
                                 float* __restrict__ dv_out, float* __restrict__ vm_out) {
    constexpr int LPR = D / 8;     // lanes per row
    constexpr int RPW = 64 / LPR;  // rows per wave step
    constexpr int RPG = 4 * RPW;   // rows per workgroup step
    const int lane = threadIdx.x & 63, ro = lane / LPR, li = lane % LPR;
    const int nb = b.nb;
    // every row of the block (two workgroup steps x four virtual waves), requested at once
    uint4 kw[2][4], vw[2][4];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = st * RPG + v * RPW + ro;
            const int jj = j < nb ? j : 0;
            kw[st][v] = *reinterpret_cast<const uint4*>(stats_krow<D>(b, jj) + li * 8);
            vw[st][v] = *reinterpret_cast<const uint4*>(stats_vrow<D>(b, jj) + li * 8);
        }
    // per virtual wave: the lane's sums over its rows (step order), then over the row groups
    float tk[8], tv[8], ak[8], av[8];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        float sk[8] = {0, 0, 0, 0, 0, 0, 0, 0}, sv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int st = 0; st < 2; ++st) {
            const bool ok = st * RPG + v * RPW + ro < nb;
            float kf[8], vf[8];
            unpack_bf16x8(kw[st][v], kf);
            unpack_bf16x8(vw[st][v], vf);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                sk[e] += ok ? kf[e] : 0.0f;
                sv[e] += ok ? vf[e] : 0.0f;
            }
        }
        // (the workgroup routine's later steps add +0 for rows past the block: no change)
#pragma unroll
        for (int off = LPR; off < 64; off <<= 1)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                sk[e] = xor_add(sk[e], off);
                sv[e] = xor_add(sv[e], off);
            }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (v == 0 || v == 2) {
                tk[e] = sk[e];
                tv[e] = sv[e];
            } else if (v == 1) {
                ak[e] = tk[e] + sk[e];
                av[e] = tv[e] + sv[e];
            } else {
                ak[e] = ak[e] + (tk[e] + sk[e]);
                av[e] = av[e] + (tv[e] + sv[e]);
            }
        }
    }
    const float fn = (float)nb;
    float mk[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        mk[e] = ak[e] / fn;
        av[e] = av[e] / fn;
    }
    if (ro == 0) {
        float4* ko = reinterpret_cast<float4*>(km_out + li * 8);
        float4* vo = reinterpret_cast<float4*>(vm_out + li * 8);
        ko[0] = make_float4(mk[0], mk[1], mk[2], mk[3]);
        ko[1] = make_float4(mk[4], mk[5], mk[6], mk[7]);
        vo[0] = make_float4(av[0], av[1], av[2], av[3]);
        vo[1] = make_float4(av[4], av[5], av[6], av[7]);
    }
    // squared deviations, the same way
    float m2[8];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        float s2[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int st = 0; st < 2; ++st) {
            const bool ok = st * RPG + v * RPW + ro < nb;
            float kf[8];
            unpack_bf16x8(kw[st][v], kf);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float dev = kf[e] - mk[e];
                s2[e] += ok ? __fmul_rn(dev, dev) : 0.0f;
            }
        }
#pragma unroll
        for (int off = LPR; off < 64; off <<= 1)
#pragma unroll
            for (int e = 0; e < 8; ++e) s2[e] = xor_add(s2[e], off);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (v == 0 || v == 2) tk[e] = s2[e];
            else if (v == 1) m2[e] = tk[e] + s2[e];
            else m2[e] = m2[e] + (tk[e] + s2[e]);
        }
    }
    if (r == D) {
        if (ro == 0) {
#pragma unroll
            for (int e = 0; e < 8; ++e) dv_out[li * 8 + e] = m2[e] / fn;
        }
        return;
    }
    // lane f = pair f: its two coordinates' totals, fetched from the lanes that hold them
    auto coord = [&](int c) {  // every lane active; the value of coordinate c (lane c / 8, element c % 8)
        float x = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float y = __shfl(m2[e], c / 8);
            x = (c % 8 == e) ? y : x;
        }
        return x;
    };
    const bool in = lane < D / 2;
    const int f = in ? lane : 0;
    const int ia = layout == 0 ? f : 2 * f, ib = layout == 0 ? f + D / 2 : 2 * f + 1;
    const float xa = coord(ia), xb = coord(ib);
    float e2 = in ? xa + xb : 0.0f;
    const int w = (D / 2) / r;
    for (int off = 1; off < w; off <<= 1) e2 = xor_add(e2, off);
    if (in && lane % w == 0) dv_out[lane / w] = e2 / (fn * (float)(D / r));
}

template <int D>
__device__ void wg_block_stats(const uint16_t* __restrict__ Kb, const uint16_t* __restrict__ Vb, int nb,
                               const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new, int new_j,
                               int r, int layout, float* __restrict__ km_out, float* __restrict__ dv_out,
                               float* __restrict__ vm_out, BlockStatsLds<D>& L) {
    const BlockSrc b{Kb, Vb, k_new, v_new, nb, new_j};
    BlockRows R;
    load_block_rows<D>(b, 0, R);
    block_stats_from<D>(b, R, r, layout, km_out, dv_out, vm_out, L);
}

}  // namespace compkv

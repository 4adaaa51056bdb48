// block_stats.h -- the one-wave block summary routine shared by the prefill, the append and the fused
// decode step (private to libcompkv). Every caller uses the same lane-to-row mapping and reduction
// order, so a summary does not depend on which of them computed it.
#pragma once

#include "internal.h"

namespace compkv {

// Sum the coordinates of group t (Appendix A.4) from a per-coordinate array in LDS.
__device__ inline float group_sum(const float* m2, int t, int D, int r, int layout) {
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
// instead of the cache. m2s: D floats of LDS private to this wave. km_lds / dv_lds / vm_lds (optional)
// receive a copy of the result in LDS. Called by whole waves; every wave
// of the workgroup must reach the trailing __syncthreads() the same number of times.
template <int D>
__device__ inline void wave_block_stats(const uint16_t* __restrict__ Kb, const uint16_t* __restrict__ Vb, int nb,
                                 const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
                                 int new_j, int r, int layout, float* __restrict__ km_out,
                                 float* __restrict__ dv_out, float* __restrict__ vm_out, float* m2s,
                                 bool active, float* km_lds = nullptr, float* dv_lds = nullptr,
                                 float* vm_lds = nullptr) {
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
            if (km_lds) {  // optional LDS copy of the result for the caller's workgroup
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    km_lds[li * 8 + e] = mk[e];
                    vm_lds[li * 8 + e] = mv[e];
                }
            }
        }
    }
    __syncthreads();
    if (active) {
        const float denom = (float)nb * (float)(D / r);
        for (int t = lane; t < r; t += 64) {
            const float dv = group_sum(m2s, t, D, r, layout) / denom;
            dv_out[t] = dv;
            if (dv_lds) dv_lds[t] = dv;
        }
    }
    __syncthreads();
}

}  // namespace compkv

// exact.h -- exact attention over a list of selected blocks on the matrix cores (private to
// libcompkv): the tile loop of an exact item and the combination of its waves' softmax states. Used by
// the sparse decode's exact items and by the fused selection + exact kernel.
//
// One 16-token tile per wave and round. The logits are formed as S^T = K Q^T with
// v_mfma_f32_16x16x32_bf16 (A = 16 key rows, B = the unit's query heads as columns, zero-padded to 16):
// lane l then holds the logits of head l%16 for tokens 4(l/16)..4(l/16)+3, which is exactly the
// A-operand layout of v_mfma_f32_16x16x16bf16_1k, so the probabilities feed the P.V product without any
// data movement. For P.V the value row of each of the lane's 4 tokens is loaded as one contiguous chunk
// of d/16 coordinates (coordinate (d/16)*(l%16) + j goes to output block j), so every load is a
// contiguous piece of a row. P.V runs as v_mfma_f32_16x16x16bf16_1k per tile, with P split into three
// bf16 terms (three MFMAs), which keeps P within 2^-27 of its fp32 value (two terms, 2^-17, are not
// enough for outputs that cancel to near zero); products with the bf16 values are exact and accumulate
// in fp32. The softmax max is taken per tile.
//
// In the fused step the compensation partials already hold the pseudo-token of every block (logit
// log|b| + zbar_b, value vmean_b), so an exact item takes its own blocks' pseudo-tokens back out. As
// |b| e^{zbar_b} vmean_b = sum over the block's tokens of e^{zbar_b} v_j, this is a per-token weight
// p'_j = e^{zbar_b - m}: the item multiplies V by p_j - p'_j in the same MFMAs, and by Jensen's
// inequality each block's sum of these weights is non-negative.
#pragma once

#include "internal.h"

namespace compkv {

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf16 __attribute__((ext_vector_type(8)));
typedef float v4f32 __attribute__((ext_vector_type(4)));

constexpr int kMaxEb = 128;  // selected blocks per exact item, upper bound

// The softmax states of NW waves and the fused step's block-logit table.
template <int D, int G, int NW>
struct ExactLds {
    float m[NW][G], l[NW][G];
    float f[NW][G];  // each wave's rescale factor exp(m_w - M) per head
    float fx[G];     // the same for an absorbed partial (finish_exact's xm, xl, xacc)
    float M[G], L[G];
    alignas(16) float acc[NW][G][D];
    float zb[G][kMaxEb];  // fused step: the block logits of the item's selected blocks
};

// Stores and loads coherent across the device (relaxed atomics at agent scope: they bypass the
// non-coherent cached copies), for partials that another workgroup of the same launch merges.
__device__ __forceinline__ void st_agent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
    return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent_i32(int32_t* p, int32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t ld_agent_i32(const int32_t* p) {
    return __hip_atomic_load(const_cast<int32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent_u32(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_agent_u32(const uint32_t* p) {
    return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// 8 and 16 bytes (8-byte aligned): one or two 64-bit accesses
__device__ __forceinline__ float2 ld_agent2(const float* p) {
    const unsigned long long w =
        __hip_atomic_load(reinterpret_cast<unsigned long long*>(const_cast<float*>(p)), __ATOMIC_RELAXED,
                          __HIP_MEMORY_SCOPE_AGENT);
    return make_float2(__uint_as_float((uint32_t)w), __uint_as_float((uint32_t)(w >> 32)));
}
__device__ __forceinline__ float4 ld_agent4(const float* p) {
    const float2 a = ld_agent2(p), b = ld_agent2(p + 2);
    return make_float4(a.x, a.y, b.x, b.y);
}
__device__ __forceinline__ void st_agent_u64(void* p, unsigned long long v) {
    __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ short f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (short)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float bf16_bits_to_f32(short h) { return __uint_as_float(uint32_t((unsigned short)h) << 16); }

// Virtual token v of an item -> absolute cache row, or -1 if v is past the item's tokens / the block's
// length. Sparse items: rowbase[k] is the row of token 0 of the item's k-th selected block. Dense
// items (tokens t0 .. t1 - 1): contiguous caches give rowbase[0] = the row of token t0; paged caches
// (page tokens per page) give rowbase[i] = the row of token 0 of logical page pg0 + i.
struct TokenMap {
    const int32_t* sel;      // sparse: the item's selected ids (first entry of the item)
    const int32_t* rowbase;  // see above (LDS)
    int nblk, B, n, X;       // sparse
    float invB;
    int t0, t1;              // dense: token range
    int page, pg0;           // dense, paged: tokens per page, first logical page of the item
    float invP;
    bool dense;
    __device__ int row(int v) const {
        if (dense) {
            const int j = t0 + v;
            if (j >= t1) return -1;
            if (page == 0) return rowbase[0] + v;
            const int lp = div_small(j, page, invP);
            return rowbase[lp - pg0] + (j - lp * page);
        }
        const int k = div_small(v, B, invB);
        if (k >= nblk) return -1;
        const int blk = sel[k];
        const int off = v - k * B;
        if (blk < 0 || blk >= X || off >= min(B, n - blk * B)) return -1;
        return rowbase[k] + off;
    }
    __device__ int count() const { return dense ? max(0, t1 - t0) : nblk * B; }
};

// Exact tokens of one item with MFMA. Leaves this wave's (m, l) for head lane%16 (lanes with the same
// lane%16 agree) and acc[j][i] = sum over the wave's tokens of p * v for head 4(lane/16)+i at
// coordinate (D/16)*(lane%16) + j. With lg (the fused step: the unit's block logits, lg[g * lstride +
// b] for head g and block b; sparse items only) every token's weight is p_j - p'_j with
// p'_j = e^{zbar_b - m} for its block b; the item's block logits are staged in zt (LDS, [G][kMaxEb]).
// Ku / Vu are the cache bases (tm.row gives absolute rows). Loads are requested in the order of their
// use (they return in that order): the block logits, the query, then the first tiles' keys and values.
template <int D, int G, int NW>
__device__ void exact_tokens(const TokenMap& tm, const uint16_t* __restrict__ Ku, const uint16_t* __restrict__ Vu,
                             const uint16_t* __restrict__ qh, const float* lg, size_t lstride, float (*zt)[kMaxEb],
                             float scale, float& m, float& l, v4f32 (&acc)[D / 16]) {
    static_assert(NW * 64 >= kMaxEb, "one block logit per thread and head");
    constexpr int KS = D / 32;   // k-steps of the logit MFMA
    constexpr int CPL = D / 16;  // value coordinates per lane (= output blocks)
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;
    m = -INFINITY;
    l = 0.0f;
#pragma unroll
    for (int j = 0; j < CPL; ++j) acc[j] = v4f32{0.0f, 0.0f, 0.0f, 0.0f};
    // the block logits of the item's blocks (thread k < nblk: block k, every head)
    const bool stage = lg != nullptr && !tm.dense;  // (workgroup-uniform)
    float zv[G];
    if (stage && tid < tm.nblk) {
        const int b = tm.sel[tid];
        const int bb = b >= 0 && b < tm.X ? b : 0;
#pragma unroll
        for (int g = 0; g < G; ++g) zv[g] = lg[(size_t)g * lstride + bb];
    }
    // B operand of the logit product: query head `col` (zero for padding heads)
    v8bf16 qb[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        uint4 w = make_uint4(0, 0, 0, 0);
        if (col < G) w = *reinterpret_cast<const uint4*>(qh + col * D + 32 * ks + 8 * grp);
        qb[ks] = __builtin_bit_cast(v8bf16, w);
    }
    const int ntiles = (tm.count() + 15) / 16;
    const bool pseudo = stage && col < G;
    uint4 kreg[KS];
    uint4 vreg[4];
    bool vvalid[4];
    bool kvalid;
    // every load of a tile is issued first (branch-free: a row past the item's tokens loads row 0 of
    // the unit and is zeroed after)
    // (lane l < 16 maps token l of the tile to its row; the value rows come from those lanes)
    auto issue = [&](int t) {
        const int base = t * 16;
        const int rk = t < ntiles ? tm.row(base + col) : -1;  // the key row of token `col`
        kvalid = rk >= 0;
        const uint16_t* kp = Ku + (size_t)(rk >= 0 ? rk : 0) * D + 8 * grp;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kreg[ks] = *reinterpret_cast<const uint4*>(kp + 32 * ks);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int rv = __shfl(rk, 4 * grp + e);  // the row of token 4*grp + e
            vvalid[e] = rv >= 0;
            const uint16_t* vp = Vu + (size_t)(rv >= 0 ? rv : 0) * D + CPL * col;
            if constexpr (CPL == 8) {
                vreg[e] = *reinterpret_cast<const uint4*>(vp);
            } else {
                const uint2 hv = *reinterpret_cast<const uint2*>(vp);
                vreg[e] = make_uint4(hv.x, hv.y, 0, 0);
            }
        }
    };
    issue(wave);
    if (stage) {  // (the logits were requested first: this waits for them alone)
        if (tid < tm.nblk) {
#pragma unroll
            for (int g = 0; g < G; ++g) zt[g][tid] = zv[g];
        }
        __syncthreads();
    }
    for (int t = wave; t < ntiles; t += NW) {
        if (t != wave) issue(t);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kreg[ks] = kvalid ? kreg[ks] : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) vreg[e] = vvalid[e] ? vreg[e] : make_uint4(0, 0, 0, 0);
        // logits: lane holds head `col`, tokens 4*grp + i of the tile; the pseudo-logits join the max so
        // that both weights stay at most 1
        auto zpseudo = [&](int i) {
            return (pseudo && vvalid[i]) ? zt[col][div_small(t * 16 + 4 * grp + i, tm.B, tm.invB)] : -INFINITY;
        };
        v4f32 sv = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            sv = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf16, kreg[ks]), qb[ks], sv, 0, 0, 0);
        float z[4], zp[4];
        float rmax = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            z[i] = vvalid[i] ? scale * sv[i] : -INFINITY;
            zp[i] = zpseudo(i);
            rmax = fmaxf(rmax, fmaxf(z[i], zp[i]));
        }
        rmax = fmaxf(rmax, __shfl_xor(rmax, 16));
        rmax = fmaxf(rmax, __shfl_xor(rmax, 32));
        const float m_new = fmaxf(m, rmax);
        if (m_new == -INFINITY) continue;  // nothing valid for this head yet (uniform per wave-round)
        if (m != -INFINITY) {  // a later round: rescale the running state
            const float c = __expf(m - m_new);
            l *= c;
            // accumulator row i holds head 4*grp + i, whose factor lives in lane 4*grp + i
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float ci = __shfl(c, 4 * grp + i);
#pragma unroll
                for (int j = 0; j < CPL; ++j) acc[j][i] *= ci;
            }
        }
        m = m_new;
        // P.V with v_mfma_f32_16x16x16bf16_1k: k-index 4*grp + e is token 4*grp + e in both operands.
        // The weight is split into three bf16 terms (hi + mid + lo equals it to within 2^-27 relative).
        v4i16 pa[3];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float p = (z[i] == -INFINITY ? 0.0f : __expf(z[i] - m)) - (zp[i] == -INFINITY ? 0.0f : __expf(zp[i] - m));
            l += p;
            const short hi = f32_to_bf16_rne(p);
            const float r1 = p - bf16_bits_to_f32(hi);
            const short md = f32_to_bf16_rne(r1);
            const short lo = f32_to_bf16_rne(r1 - bf16_bits_to_f32(md));
            pa[0][i] = hi;
            pa[1][i] = md;
            pa[2][i] = lo;
        }
        const uint32_t* w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = reinterpret_cast<const uint32_t*>(&vreg[e]);
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            // B operand for output block j: element 4*grp + e = coordinate CPL*col + j of token 4*grp + e
            const int wi = j >> 1;
            uint32_t pk0, pk1;
            if ((j & 1) == 0) {
                pk0 = (w[0][wi] & 0xFFFFu) | (w[1][wi] << 16);
                pk1 = (w[2][wi] & 0xFFFFu) | (w[3][wi] << 16);
            } else {
                pk0 = (w[0][wi] >> 16) | (w[1][wi] & 0xFFFF0000u);
                pk1 = (w[2][wi] >> 16) | (w[3][wi] & 0xFFFF0000u);
            }
            const v4i16 bv = __builtin_bit_cast(v4i16, make_uint2(pk0, pk1));
#pragma unroll
            for (int k = 0; k < 3; ++k) acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa[k], bv, acc[j], 0, 0, 0);
        }
    }
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
}

// Combine the NW waves' exact states in LDS and write the item's partial: the per-head maximum M
// over the waves and each wave's factor exp(m_w - M) first, then every coordinate as a plain sum of
// the waves' scaled accumulators in wave order. kCoherent: the partial is stored with device-coherent
// stores (merged by another workgroup of the same launch). With xm non-null, one more partial in LDS
// (per head: max xm[g], sum xl[g], weighted sums xacc[g * xstride + i]) is absorbed after the waves.
template <int D, int G, int NW, bool kCoherent = false>
__device__ void finish_exact(float m, float l, const v4f32 (&acc)[D / 16], ExactLds<D, G, NW>& sh, float* part,
                             const float* xm = nullptr, const float* xl = nullptr, const float* xacc = nullptr,
                             int xstride = 0) {
    constexpr int CPL = D / 16;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;
    if (grp == 0 && col < G) {
        sh.m[wave][col] = m;
        sh.l[wave][col] = l;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int g = 4 * grp + i;
        if (g < G) {  // coordinates CPL*col .. CPL*col + CPL - 1 of head g, contiguous
#pragma unroll
            for (int j = 0; j < CPL; j += 4)
                *reinterpret_cast<float4*>(&sh.acc[wave][g][CPL * col + j]) =
                    make_float4(acc[j][i], acc[j + 1][i], acc[j + 2][i], acc[j + 3][i]);
        }
    }
    __syncthreads();
    if (tid < G) {
        const int g = tid;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < NW; ++w) M = fmaxf(M, sh.m[w][g]);
        if (xm) M = fmaxf(M, xm[g]);
        float L = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const float fw = sh.m[w][g] == -INFINITY ? 0.0f : __expf(sh.m[w][g] - M);
            sh.f[w][g] = fw;
            L += fw * sh.l[w][g];
        }
        if (xm) {
            const float fx = xm[g] == -INFINITY ? 0.0f : __expf(xm[g] - M);
            sh.fx[g] = fx;
            L += fx * xl[g];
        }
        sh.M[g] = M;
        sh.L[g] = L;
    }
    __syncthreads();
    for (int idx = tid; idx < G * D; idx += 64 * NW) {
        const int g = idx / D, i = idx % D;
        float aa = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) aa += sh.f[w][g] * sh.acc[w][g][i];
        if (xm) aa += sh.fx[g] * xacc[(size_t)g * xstride + i];
        float* p = part + (size_t)g * (D + 2);
        if constexpr (kCoherent) {
            if (i == 0) {
                st_agent(p, sh.M[g]);
                st_agent(p + 1, sh.L[g]);
            }
            st_agent(p + 2 + i, aa);
        } else {
            if (i == 0) {
                p[0] = sh.M[g];
                p[1] = sh.L[g];
            }
            p[2 + i] = aa;
        }
    }
}

}  // namespace compkv

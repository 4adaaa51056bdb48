// decode.hip -- compensated sparse decode and dense decode (Eq. compkv-output; Section 3.1).
//
// grid = (items, units). Every item produces one softmax partial per query head of its unit: the
// running max m, the sum of weights l and the weighted value sum acc[d] (flash-decoding split-K).
//   * exact items (sparse): the tokens of up to `eb` consecutive entries of the selected-id list;
//   * compensation items (sparse): the unselected blocks of a range of `cb` block ids, each entering
//     once as a pseudo-token with logit log|b| + zbar_b and value vmean_b;
//   * dense items: a contiguous range of `eb` tokens.
// The last item of a unit to arrive (atomic ticket) merges all partials of that unit in item order,
// so the result does not depend on scheduling. Nothing waits on another workgroup.
//
// Exact tokens: d/8 lanes share a token, each holding 8 coordinates (one 16-byte load of the bf16
// row), so a wave reads 4 rows (d = 128) per load. Logits are reduced across those lanes; every token
// slot keeps its own online softmax state, and the slots are merged at the end of the item.
// Compensation: d/4 lanes share a block's fp32 mean-value row (one float4 each).
#include "internal.h"

namespace compkv {
namespace {

constexpr int kMaxItems = 256;  // partials per unit, upper bound (checked by the host)
constexpr int kCbMax = 2048;    // blocks per compensation item, upper bound

template <int G, int CPL>
struct SoftmaxState {
    float m[G], l[G], acc[G][CPL];
    __device__ void init() {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            m[g] = -INFINITY;
            l[g] = 0.0f;
#pragma unroll
            for (int e = 0; e < CPL; ++e) acc[g][e] = 0.0f;
        }
    }
    // add one term with logit z[g] and value vals[e] (same value row for every head)
    __device__ void add(const float (&z)[G], const float (&vals)[CPL]) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const float mn = fmaxf(m[g], z[g]);
            const float c = (m[g] == -INFINITY) ? 0.0f : __expf(m[g] - mn);
            const float w = __expf(z[g] - mn);
            l[g] = l[g] * c + w;
#pragma unroll
            for (int e = 0; e < CPL; ++e) acc[g][e] = acc[g][e] * c + w * vals[e];
            m[g] = mn;
        }
    }
    // merge with the state of the lane `off` away (xor), for lanes holding the same coordinates
    __device__ void merge_xor(int off) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const float mo = __shfl_xor(m[g], off);
            const float lo = __shfl_xor(l[g], off);
            float mn, ca, cb;
            merge_scales(m[g], mo, mn, ca, cb);
            l[g] = l[g] * ca + lo * cb;
#pragma unroll
            for (int e = 0; e < CPL; ++e) {
                const float ao = __shfl_xor(acc[g][e], off);
                acc[g][e] = acc[g][e] * ca + ao * cb;
            }
            m[g] = mn;
        }
    }
};

template <int D, int G>
struct DecodeShared {
    float m[4][G], l[4][G];
    float acc[4][G][D];
    unsigned char flag[kCbMax];
    float pm[G][kMaxItems], pc[G][kMaxItems];
    float M[G], L[G];
    int last;
};

// Reduce the per-slot states of the workgroup (LPS lanes per slot, CPL coordinates per lane at
// coordinate li*CPL) and write the item's partial. Called by all threads.
template <int D, int G, int CPL, int LPS>
__device__ void finish_item(SoftmaxState<G, CPL>& st, DecodeShared<D, G>& sh, float* part) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane % LPS;
#pragma unroll
    for (int off = LPS; off < 64; off <<= 1) st.merge_xor(off);
    if (lane < LPS) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            if (li == 0) {
                sh.m[wave][g] = st.m[g];
                sh.l[wave][g] = st.l[g];
            }
#pragma unroll
            for (int e = 0; e < CPL; ++e) sh.acc[wave][g][li * CPL + e] = st.acc[g][e];
        }
    }
    __syncthreads();
    for (int idx = tid; idx < G * D; idx += kThreads) {
        const int g = idx / D, i = idx % D;
        float m = -INFINITY, l = 0.0f, acc = 0.0f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            float mn, ca, cb;
            merge_scales(m, sh.m[w][g], mn, ca, cb);
            l = l * ca + sh.l[w][g] * cb;
            acc = acc * ca + sh.acc[w][g][i] * cb;
            m = mn;
        }
        float* p = part + (size_t)g * (D + 2);
        if (i == 0) {
            p[0] = m;
            p[1] = l;
        }
        p[2 + i] = acc;
    }
}

template <int D, int G>
__global__ __launch_bounds__(kThreads) void decode_kernel(Geom geo, DecodeArgs a) {
    __shared__ DecodeShared<D, G> sh;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u = blockIdx.y, item = blockIdx.x, nitems = gridDim.x;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int n = clamp_len(a.seq_lens[bseq], geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    float* part = a.ws_part + ((size_t)u * nitems + item) * G * (D + 2);
    const bool comp_item = !a.dense && item >= a.n_exact;

    if (!comp_item) {
        // ---------------- exact tokens
        constexpr int LPT = D / 8, SPW = 64 / LPT, SLOTS = 4 * SPW;
        const int li = lane % LPT, slot = wave * SPW + lane / LPT;
        const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
        float qreg[G][8];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float qf[8];
            unpack_bf16x8(*reinterpret_cast<const uint4*>(qh + g * D + li * 8), qf);
#pragma unroll
            for (int e = 0; e < 8; ++e) qreg[g][e] = a.scale * qf[e];
        }
        SoftmaxState<G, 8> st;
        st.init();
        const uint16_t* Ku = a.K + (size_t)u * geo.cap * D;
        const uint16_t* Vu = a.V + (size_t)u * geo.cap * D;
        int t0, t1;  // virtual token range
        const int32_t* selu = a.sel + (size_t)u * a.sel_stride;
        int nsel = 0, e0 = 0;
        if (a.dense) {
            t0 = item * a.eb;
            t1 = min(t0 + a.eb, n);
        } else {
            nsel = min(a.n_sel[u], a.sel_stride);
            e0 = item * a.eb;
            t0 = 0;
            t1 = max(0, min(a.eb, nsel - e0)) * geo.B;
        }
        for (int t = t0 + slot; t < t1; t += SLOTS) {
            int row;
            if (a.dense) {
                row = t;
            } else {
                const int blk = selu[e0 + t / geo.B];
                const int off = t % geo.B;
                if (blk < 0 || blk >= X || off >= min(geo.B, n - blk * geo.B)) continue;
                row = blk * geo.B + off;
            }
            float kf[8], vf[8];
            unpack_bf16x8(*reinterpret_cast<const uint4*>(Ku + (size_t)row * D + li * 8), kf);
            unpack_bf16x8(*reinterpret_cast<const uint4*>(Vu + (size_t)row * D + li * 8), vf);
            float z[G];
#pragma unroll
            for (int g = 0; g < G; ++g) {
                float acc = 0.0f;
#pragma unroll
                for (int e = 0; e < 8; ++e) acc += qreg[g][e] * kf[e];
                z[g] = acc;
            }
#pragma unroll
            for (int off = 1; off < LPT; off <<= 1)
#pragma unroll
                for (int g = 0; g < G; ++g) z[g] += __shfl_xor(z[g], off);
            st.add(z, vf);
        }
        finish_item<D, G, 8, LPT>(st, sh, part);
    } else {
        // ---------------- compensation pseudo-tokens of unselected blocks
        constexpr int LPB = D / 4, BPW = 64 / LPB, CSLOTS = 4 * BPW;
        const int li = lane % LPB, cslot = wave * BPW + lane / LPB;
        const int c0 = (item - a.n_exact) * a.cb;
        const int c1 = min(c0 + a.cb, X);
        const int nsel = min(a.n_sel[u], a.sel_stride);
        const int32_t* selu = a.sel + (size_t)u * a.sel_stride;
        for (int i = tid; i < a.cb; i += kThreads) sh.flag[i] = 0;
        __syncthreads();
        for (int k = tid; k < nsel; k += kThreads) {
            const int sb = selu[k];
            if (sb >= c0 && sb < c1) sh.flag[sb - c0] = 1;
        }
        __syncthreads();
        SoftmaxState<G, 4> st;
        st.init();
        const float* lg = a.blk_logit + (size_t)u * G * geo.xcap;
        for (int lb = cslot; lb < c1 - c0; lb += CSLOTS) {
            if (sh.flag[lb]) continue;
            const int b = c0 + lb;
            const float lnb = logf((float)min(geo.B, n - b * geo.B));
            float z[G];
#pragma unroll
            for (int g = 0; g < G; ++g) z[g] = lnb + lg[(size_t)g * geo.xcap + b];
            const float4 v4 = reinterpret_cast<const float4*>(a.vmean + ((size_t)u * geo.xcap + b) * D)[li];
            const float vals[4] = {v4.x, v4.y, v4.z, v4.w};
            st.add(z, vals);
        }
        finish_item<D, G, 4, LPB>(st, sh, part);
    }

    // ---------------- arrival ticket; the last item of the unit merges
    __threadfence();
    __syncthreads();
    if (tid == 0) sh.last = (atomicAdd(&a.counters[u], 1u) == (unsigned)(nitems - 1));
    __syncthreads();
    if (!sh.last) return;
    __threadfence();

    const float* pu = a.ws_part + (size_t)u * nitems * G * (D + 2);
    for (int idx = tid; idx < G * nitems; idx += kThreads) {
        const int g = idx / nitems, it = idx % nitems;
        const float* p = pu + ((size_t)it * G + g) * (D + 2);
        sh.pm[g][it] = p[0];
        sh.pc[g][it] = p[1];
    }
    __syncthreads();
    if (tid < G) {
        const int g = tid;
        float M = -INFINITY;
        for (int it = 0; it < nitems; ++it) M = fmaxf(M, sh.pm[g][it]);
        float L = 0.0f;
        for (int it = 0; it < nitems; ++it) {
            const float c = (sh.pm[g][it] == -INFINITY) ? 0.0f : __expf(sh.pm[g][it] - M);
            L += c * sh.pc[g][it];
            sh.pc[g][it] = c;  // reuse as the item's rescale factor
        }
        sh.M[g] = M;
        sh.L[g] = L;
    }
    __syncthreads();
    for (int idx = tid; idx < G * D; idx += kThreads) {
        const int g = idx / D, i = idx % D;
        float A = 0.0f;
        for (int it = 0; it < nitems; ++it) {
            const float c = sh.pc[g][it];
            if (c != 0.0f) A += c * pu[((size_t)it * G + g) * (D + 2) + 2 + i];
        }
        const float L = sh.L[g];
        const size_t o = (size_t)bseq * geo.hq + (size_t)h * G + g;
        a.out[o * D + i] = L > 0.0f ? A / L : 0.0f;
        if (i == 0 && a.lse) a.lse[o] = L > 0.0f ? sh.M[g] + logf(L) : -INFINITY;
    }
    if (tid == 0) a.counters[u] = 0u;
}

template <int D>
hipError_t dispatch_g(const Geom& g, const DecodeArgs& a, hipStream_t s, dim3 grid) {
    switch (g.G) {
        case 1: decode_kernel<D, 1><<<grid, kThreads, 0, s>>>(g, a); break;
        case 2: decode_kernel<D, 2><<<grid, kThreads, 0, s>>>(g, a); break;
        case 4: decode_kernel<D, 4><<<grid, kThreads, 0, s>>>(g, a); break;
        case 8: decode_kernel<D, 8><<<grid, kThreads, 0, s>>>(g, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const Geom& g, const DecodeArgs& a, hipStream_t s) {
    const int items = a.dense ? a.n_exact : a.n_exact + a.n_comp;
    if (items < 1 || items > kMaxItems || (!a.dense && a.cb > kCbMax)) return hipErrorInvalidValue;
    dim3 grid(items, g.units());
    return g.D == 128 ? dispatch_g<128>(g, a, s, grid) : dispatch_g<64>(g, a, s, grid);
}

}  // namespace compkv

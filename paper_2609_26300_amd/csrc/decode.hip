// decode.hip -- compensated sparse decode and dense decode (Eq. compkv-output; Section 3.1).
//
// One-dimensional grid of items * units workgroups, mapped by xcd_unit_work so that (when the units
// fill whole rounds of eight) all items of unit u run on XCD u % 8. Every item produces one softmax
// partial per query head of its unit: the
// max m, the sum of weights l and the weighted value sum acc[d] (flash-decoding split-K).
//   * exact items (sparse): the tokens of up to `eb` consecutive entries of the selected-id list;
//   * compensation items (sparse): the unselected blocks among `cb` consecutive block ids, each
//     entering once as a pseudo-token with logit log|b| + zbar_b and value vmean_b;
//   * dense items: `eb` consecutive tokens.
// A second launch, grid = (units, G), merges each unit's partials in item order, so the result does
// not depend on scheduling; the kernel boundary makes the partials visible (no cross-workgroup fences).
//
// Item workgroups have eight waves (kItemThreads); an exact item runs the tile loop of exact.h, one
// 16-token tile per wave and round, so a 128-token item is one round of the eight waves (256-token
// items, two rounds, when the 128-token items would not all be resident at once).
//
// Compensation items are plain fp32 streaming on the vector ALUs: the mean-value rows (d/4 lanes x
// float4 per row, 16 rows per thread in flight) are requested first; meanwhile the item marks its
// selected blocks, forms the pseudo-logits of the others and their per-head max; then the weighted
// rows are summed.
#include "exact.h"

namespace compkv {
namespace {

constexpr int kMaxItems = 256;     // items per unit and launch, upper bound (checked by the host)
constexpr int kMaxPartials = 2048;  // partials per unit in a merge, upper bound
constexpr int kCbMax = 512;     // blocks per compensation item, upper bound
constexpr int kMaxRowBase = 1024;  // row bases per item: selected blocks, or pages of a dense item
constexpr int kItemWaves = 8;  // waves of an item workgroup
constexpr int kItemThreads = 64 * kItemWaves;

template <int D, int G>
struct DecodeShared {
    ExactLds<D, G, kItemWaves> ex;  // exact items; compensation items use ex.acc for their wave sums
    float w[G][kCbMax];  // compensation weights
    float M[G], L[G];
    unsigned char flag[kCbMax];
    int sel[kMaxEb];  // the exact item's selected ids
    int rowbase[kMaxRowBase];  // cache row of token 0 of each selected block (sparse) or page (dense)
};

// Pseudo-logits log|b| + zbar of the unselected blocks in [c0, c0 + nb) recomputed from the mean keys
// (no block logits given): zbar_g = s q_g . kmean_b. The scaled query goes to LDS (in the exact items'
// accumulator area, unused here); each wave then takes blocks in turn, four mean-key rows in flight per
// lane, the G dot products summed over the wave. Selected blocks (sh.flag) get -inf.
template <int D, int G>
__device__ void block_logits_from_kmean(const DecodeArgs& a, const Geom& geo, int u, int n, int c0, int nb,
                                        DecodeShared<D, G>& sh) {
    constexpr int CPL = D / 64;  // mean-key coordinates per lane
    constexpr int RIF = 4;       // rows in flight per wave
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    float (*qs)[D] = sh.ex.acc[0];  // [G][D] scaled query
    const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    for (int idx = tid; idx < G * D; idx += kItemThreads) qs[idx / D][idx % D] = a.scale * bf16_at(qh + idx);
    __syncthreads();
    float qv[G][CPL];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int c = 0; c < CPL; ++c) qv[g][c] = qs[g][lane * CPL + c];
    const float* km = a.kmean + ((size_t)u * geo.xcap + c0) * D + lane * CPL;
    for (int lb0 = wave * RIF; lb0 < nb; lb0 += kItemWaves * RIF) {  // wave-uniform
        float k[RIF][CPL];
#pragma unroll
        for (int e = 0; e < RIF; ++e) {  // branch-free: rows past the range reload row 0, unused
            const int lb = lb0 + e < nb ? lb0 + e : 0;
#pragma unroll
            for (int c = 0; c < CPL; ++c) k[e][c] = km[(size_t)lb * D + c];
        }
#pragma unroll
        for (int e = 0; e < RIF; ++e) {
            const int lb = lb0 + e;
            if (lb >= nb) break;  // wave-uniform
            const int b = c0 + lb;
            const float lnb = logf((float)min(geo.B, n - b * geo.B));
#pragma unroll
            for (int g = 0; g < G; ++g) {
                float z = 0.0f;
#pragma unroll
                for (int c = 0; c < CPL; ++c) z += qv[g][c] * k[e][c];
                z = wave_sum(z);
                if (lane == 0) sh.w[g][lb] = sh.flag[lb] ? -INFINITY : lnb + z;
            }
        }
    }
}

// Pseudo-tokens of the unselected blocks in [c0, c1).
template <int D, int G>
__device__ void compensation(const DecodeArgs& a, const Geom& geo, int u, int n, int X, int c0, int c1,
                             DecodeShared<D, G>& sh, float* part) {
    constexpr int LPB = D / 4;          // lanes per mean-value row (one float4 each)
    constexpr int RPS = kItemThreads / LPB;  // rows per workgroup step
    constexpr int ROWS = 8;                  // rows in flight per thread
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nb = max(0, c1 - c0);
    const int li = tid % LPB, slot = tid / LPB;
    // issue this thread's first ROWS mean-value rows before anything else (rows of selected blocks
    // are fetched too and then weighted by zero)
    const float4* vm = reinterpret_cast<const float4*>(a.vmean + ((size_t)u * geo.xcap + c0) * D) + li;
    float4 v[ROWS];
#pragma unroll
    for (int k = 0; k < ROWS; ++k) {  // branch-free: a slot past the item reloads row 0, weighted by zero
        const int lb = slot + k * RPS;
        v[k] = vm[(size_t)(lb < nb ? lb : 0) * (D / 4)];
    }
    const int nsel = min(a.n_sel[u], a.sel_stride);
    const int32_t* selu = a.sel + (size_t)u * a.sel_stride;
    for (int i = tid; i < nb; i += kItemThreads) sh.flag[i] = 0;
    __syncthreads();
    for (int k = tid; k < nsel; k += kItemThreads) {
        const int sb = selu[k];
        if (sb >= c0 && sb < c1) sh.flag[sb - c0] = 1;
    }
    __syncthreads();
    // pseudo-logits log|b| + zbar and their per-head max
    if (a.blk_logit) {  // workgroup-uniform: zbar as written by the scoring call
        const float* lg = a.blk_logit + (size_t)u * G * geo.xcap;
        for (int idx = tid; idx < G * nb; idx += kItemThreads) {
            const int g = idx / nb, lb = idx % nb, b = c0 + lb;
            sh.w[g][lb] = sh.flag[lb] ? -INFINITY
                                      : logf((float)min(geo.B, n - b * geo.B)) + lg[(size_t)g * geo.xcap + b];
        }
    } else {
        block_logits_from_kmean<D, G>(a, geo, u, n, c0, nb, sh);
    }
    __syncthreads();
    for (int g = wave; g < G; g += kItemWaves) {
        float mx = -INFINITY;
        for (int lb = lane; lb < nb; lb += 64) mx = fmaxf(mx, sh.w[g][lb]);
        mx = wave_max(mx);
        float sum = 0.0f;
        for (int lb = lane; lb < nb; lb += 64) {
            const float wv = (mx == -INFINITY || sh.w[g][lb] == -INFINITY) ? 0.0f : __expf(sh.w[g][lb] - mx);
            sh.w[g][lb] = wv;
            sum += wv;
        }
        sum = wave_sum(sum);
        if (lane == 0) {
            sh.M[g] = mx;
            sh.L[g] = sum;
        }
    }
    __syncthreads();
    // weighted mean values; lane li of a row slot holds coordinates 4li..4li+3
    float acc[G][4];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g][0] = acc[g][1] = acc[g][2] = acc[g][3] = 0.0f;
    for (int lb0 = slot; lb0 < nb; lb0 += RPS * ROWS) {
        if (lb0 != slot) {
#pragma unroll
            for (int k = 0; k < ROWS; ++k) {
                const int lb = lb0 + k * RPS;
                v[k] = vm[(size_t)(lb < nb ? lb : 0) * (D / 4)];
            }
        }
#pragma unroll
        for (int k = 0; k < ROWS; ++k) {
            const int lb = lb0 + k * RPS;
            if (lb >= nb) break;
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const float wv = sh.w[g][lb];
                acc[g][0] += wv * v[k].x;
                acc[g][1] += wv * v[k].y;
                acc[g][2] += wv * v[k].z;
                acc[g][3] += wv * v[k].w;
            }
        }
    }
    // reduce over row slots: lanes li and li + LPB of a wave, then the waves in order
#pragma unroll
    for (int off = LPB; off < 64; off <<= 1)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[g][e] += __shfl_xor(acc[g][e], off);
    if (lane < LPB) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e) sh.ex.acc[wave][g][4 * li + e] = acc[g][e];
    }
    __syncthreads();
    for (int idx = tid; idx < G * D; idx += kItemThreads) {
        const int g = idx / D, i = idx % D;
        float* p = part + (size_t)g * (D + 2);
        if (i == 0) {
            p[0] = sh.M[g];
            p[1] = sh.L[g];
        }
        float tot = 0.0f;
#pragma unroll
        for (int w = 0; w < kItemWaves; ++w) tot += sh.ex.acc[w][g][i];
        p[2 + i] = tot;
    }
}

// Two workgroups per CU (at most 128 registers per lane).
template <int D, int G>
__global__ __launch_bounds__(kItemThreads) __attribute__((amdgpu_waves_per_eu(4))) void decode_items_kernel(
    Geom geo, DecodeArgs a, int nitems) {
    __shared__ DecodeShared<D, G> sh;
    const int tid = threadIdx.x;
    // the items of unit u all on XCD u % kXcds, like the unit's selection before and merge after them
    int u, item;
    xcd_unit_work(blockIdx.x, geo.units(), nitems, u, item);
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int n = clamp_len(a.seq_lens[bseq], geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    float* part = a.ws_part + ((size_t)u * a.part_count + a.part_base + item) * G * (D + 2);

    if (a.dense || item < a.n_exact) {
        TokenMap tm;
        tm.dense = a.dense != 0;
        tm.B = geo.B;
        tm.invB = 1.0f / (float)geo.B;
        tm.n = n;
        tm.X = X;
        tm.rowbase = sh.rowbase;
        tm.page = 0;
        tm.pg0 = 0;
        tm.invP = 0.0f;
        if (tm.dense) {
            tm.t0 = item * a.eb;
            tm.t1 = min(tm.t0 + a.eb, n);
            tm.sel = nullptr;
            tm.nblk = 0;
            if (geo.bpp == 0) {
                if (tid == 0) sh.rowbase[0] = u * geo.cap + tm.t0;
            } else {  // the item's logical pages (the host bounds their count by kMaxRowBase)
                tm.page = geo.bpp * geo.B;
                tm.invP = 1.0f / (float)tm.page;
                tm.pg0 = tm.t0 / tm.page;
                const int npg = tm.t1 > tm.t0 ? (tm.t1 - 1) / tm.page - tm.pg0 + 1 : 0;
                for (int i = tid; i < npg; i += kItemThreads) sh.rowbase[i] = block_row0(geo, u, (tm.pg0 + i) * geo.bpp);
            }
            __syncthreads();
        } else {
            const int nsel = a.sel_padded ? a.sel_stride : min(a.n_sel[u], a.sel_stride);
            const int e0 = item * a.eb;
            tm.nblk = max(0, min(a.eb, nsel - e0));
            const int32_t* selu = a.sel + (size_t)u * a.sel_stride + e0;
            for (int k = tid; k < tm.nblk; k += kItemThreads) {
                const int b = selu[k];
                sh.sel[k] = b;
                sh.rowbase[k] = block_row0(geo, u, b >= 0 && b < X ? b : 0);
            }
            __syncthreads();
            tm.sel = sh.sel;
            tm.t0 = tm.t1 = 0;
        }
        float m, l;
        v4f32 acc[D / 16];
        const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
        // fused step: the block logits of the item's blocks (their pseudo-terms are taken back out)
        const bool pseudo = a.neg_pseudo && !tm.dense;
        exact_tokens<D, G, kItemWaves>(tm, a.K, a.V, qh, pseudo ? a.blk_logit + (size_t)u * G * geo.xcap : nullptr,
                                       geo.xcap, sh.ex.zb, a.scale, m, l, acc);
        finish_exact<D, G, kItemWaves>(m, l, acc, sh.ex, part);
    } else {
        const int c0 = (item - a.n_exact) * a.cb;
        compensation<D, G>(a, geo, u, n, X, c0, min(c0 + a.cb, X), sh, part);
    }
}

// Merge of one (unit, query head): the item partials in item order. grid = (units, G); thread (s, i)
// sums items s, s + S, ... for coordinate i, then the S partial sums are added in LDS in a fixed order.
// The partial maxima/sums and this thread's first R partial values are all requested at the start,
// so the usual merge costs one memory round trip.
template <int D, int G>
__global__ __launch_bounds__(kThreads) void decode_merge_kernel(Geom geo, DecodeArgs a, int nitems) {
    constexpr int S = kThreads / D;  // item subsets
    constexpr int R = 32;            // partial values per thread requested up front
    constexpr int UNR = 16;          // later batches
    __shared__ float pm[kMaxPartials], pc[kMaxPartials];
    __shared__ float part_acc[S][D];
    __shared__ float sM, sL;
    const int tid = threadIdx.x, lane = tid & 63;
    const int u = blockIdx.x, g = blockIdx.y;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const size_t stride = (size_t)G * (D + 2);
    const float* pu = a.ws_part + (size_t)u * a.part_count * stride + (size_t)g * (D + 2);
    const int i = tid % D, sub = tid / D;
    const float* pi = pu + 2 + i;
    const float2 mc = tid < nitems ? *reinterpret_cast<const float2*>(pu + tid * stride) : make_float2(0.0f, 0.0f);
    float x[R];
#pragma unroll
    for (int k = 0; k < R; ++k) {  // branch-free: past nitems reloads item 0, unused
        const int it = sub + k * S;
        x[k] = pi[(size_t)(it < nitems ? it : 0) * stride];
    }
    if (tid < nitems) {
        pm[tid] = mc.x;
        pc[tid] = mc.y;
    }
    for (int it = tid + kThreads; it < nitems; it += kThreads) {
        const float2 t = *reinterpret_cast<const float2*>(pu + it * stride);
        pm[it] = t.x;
        pc[it] = t.y;
    }
    __syncthreads();
    if (tid < 64) {
        float M = -INFINITY;
        for (int it = lane; it < nitems; it += 64) M = fmaxf(M, pm[it]);
        M = wave_max(M);
        float L = 0.0f;
        for (int it = lane; it < nitems; it += 64) {
            const float c = (pm[it] == -INFINITY) ? 0.0f : __expf(pm[it] - M);
            L += c * pc[it];
            pc[it] = c;  // from here on: the partial's rescale factor
        }
        L = wave_sum(L);
        if (lane == 0) {
            sM = M;
            sL = L;
        }
    }
    __syncthreads();
    float A = 0.0f;
#pragma unroll
    for (int k = 0; k < R; ++k) {
        const int it = sub + k * S;
        if (it < nitems) A += pc[it] * x[k];
    }
    for (int it0 = sub + R * S; it0 < nitems; it0 += UNR * S) {
        float y[UNR];
#pragma unroll
        for (int k = 0; k < UNR; ++k) {
            const int it = it0 + k * S;
            y[k] = pi[(size_t)(it < nitems ? it : 0) * stride];
        }
#pragma unroll
        for (int k = 0; k < UNR; ++k) {
            const int it = it0 + k * S;
            if (it < nitems) A += pc[it] * y[k];
        }
    }
    part_acc[sub][i] = A;
    __syncthreads();
    if (sub == 0) {
        float tot = 0.0f;
#pragma unroll
        for (int k = 0; k < S; ++k) tot += part_acc[k][i];
        const float L = sL;
        const size_t o = (size_t)bseq * geo.hq + (size_t)h * G + g;
        a.out[o * D + i] = L > 0.0f ? tot / L : 0.0f;
        if (i == 0 && a.lse) a.lse[o] = L > 0.0f ? sM + logf(L) : -INFINITY;
    }
}

template <int D, int G>
hipError_t items_g(const Geom& g, const DecodeArgs& a, int items, hipStream_t s) {
    decode_items_kernel<D, G><<<dim3(items * g.units()), kItemThreads, 0, s>>>(g, a, items);
    return hipGetLastError();
}

template <int D, int G>
hipError_t merge_g(const Geom& g, const DecodeArgs& a, int nitems, hipStream_t s) {
    decode_merge_kernel<D, G><<<dim3(g.units(), G), kThreads, 0, s>>>(g, a, nitems);
    return hipGetLastError();
}

template <int D>
hipError_t items_d(const Geom& g, const DecodeArgs& a, int items, hipStream_t s) {
    switch (g.G) {
        case 1: return items_g<D, 1>(g, a, items, s);
        case 2: return items_g<D, 2>(g, a, items, s);
        case 4: return items_g<D, 4>(g, a, items, s);
        case 8: return items_g<D, 8>(g, a, items, s);
        default: return hipErrorInvalidValue;
    }
}

template <int D>
hipError_t merge_d(const Geom& g, const DecodeArgs& a, int nitems, hipStream_t s) {
    switch (g.G) {
        case 1: return merge_g<D, 1>(g, a, nitems, s);
        case 2: return merge_g<D, 2>(g, a, nitems, s);
        case 4: return merge_g<D, 4>(g, a, nitems, s);
        case 8: return merge_g<D, 8>(g, a, nitems, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

int decode_max_items() { return kMaxItems; }
int decode_max_partials() { return kMaxPartials; }
int decode_max_cb() { return kCbMax; }
int decode_max_eb() { return kMaxEb; }
int decode_max_row_bases() { return kMaxRowBase; }

template <int D>
int item_slots_d(const Geom& g) {
    switch (g.G) {
        case 1: return resident_slots(decode_items_kernel<D, 1>, kItemThreads);
        case 2: return resident_slots(decode_items_kernel<D, 2>, kItemThreads);
        case 4: return resident_slots(decode_items_kernel<D, 4>, kItemThreads);
        default: return resident_slots(decode_items_kernel<D, 8>, kItemThreads);
    }
}
int decode_item_slots(const Geom& g) { return g.D == 128 ? item_slots_d<128>(g) : item_slots_d<64>(g); }

hipError_t launch_decode_items(const Geom& g, const DecodeArgs& a, int items, hipStream_t s) {
    if (items < 1 || a.part_base + items > a.part_count || a.part_count > kMaxPartials ||
        (!a.dense && (a.cb > kCbMax || a.eb > kMaxEb)) ||
        (a.dense && g.bpp > 0 && a.eb / (g.bpp * g.B) + 2 > kMaxRowBase))
        return hipErrorInvalidValue;
    return g.D == 128 ? items_d<128>(g, a, items, s) : items_d<64>(g, a, items, s);
}

hipError_t launch_decode_merge(const Geom& g, const DecodeArgs& a, int nitems, hipStream_t s) {
    if (nitems < 1 || nitems > a.part_count || a.part_count > kMaxPartials) return hipErrorInvalidValue;
    return g.D == 128 ? merge_d<128>(g, a, nitems, s) : merge_d<64>(g, a, nitems, s);
}

// A whole sparse or dense decode call: items, then the merge.
hipError_t launch_decode(const Geom& g, const DecodeArgs& a0, hipStream_t s) {
    DecodeArgs a = a0;
    const int items = a.dense ? a.n_exact : a.n_exact + a.n_comp;
    a.part_count = items;
    a.part_base = 0;
    a.neg_pseudo = 0;
    hipError_t e = launch_decode_items(g, a, items, s);
    if (e != hipSuccess) return e;
    return launch_decode_merge(g, a, items, s);
}

}  // namespace compkv

// select.hip -- block scoring and Top-K selection in one launch (Sections 4.1, 4.2; Appendix E.1).
//
// Two launches. Phase 1, grid = (nchunks, units): each workgroup streams the fp32 summaries (mean key, grouped
// variances) of `bpc` consecutive blocks of one unit. Eight lanes share a block: lane i of the eight
// reads float4 i, i+8, ... of the mean-key row (the eight lanes read 128 contiguous bytes per load) and
// the variance groups t = i, i+8, .... Every load of a thread is issued before any arithmetic. For
// each of the unit's G query heads it forms the block-mean logit zbar = s q.kmean, the projected
// variance sig2 = s^2 sum_t Q_t dvar_t and the log weight estimate a = log|b| + zbar + sig2/2 (the log
// of the numerator of Eq. compkv-mass-estimate), stages them in LDS, stores them with coalesced
// writes, and writes the chunk's per-head (max a, sum exp(a - max)).
//
// Phase 2, grid = (units): one workgroup per unit, in a second launch so that the kernel boundary
// makes every chunk's results visible (no cross-workgroup fences or atomics). It merges the chunk partials into each head's log normalizer, forms
// S_b = sum_g exp(a - lse_g) sig2 (Eq. compkv-score) into LDS, finds the (K-|F|)-th largest score among
// the non-mandatory blocks with a three-pass radix select on the score bits (scores are >= 0, so their
// IEEE bit patterns order like the values), and writes the selected ids in ascending order. Equal
// scores are taken in ascending id order: the stable Top-K of the paper.
#include "internal.h"

namespace compkv {
namespace {

constexpr int kBpcMax = 128;  // blocks per chunk, upper bound
constexpr int kPMax = kBpcMax / 32;
constexpr int kHistBins = 2048;

// all-reduce over aligned groups of 8 lanes
__device__ __forceinline__ float sum8(float x) {
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));  // xor 1
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));  // xor 2
    x += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), 0x101F));                    // xor 4
    return x;
}

__device__ __forceinline__ bool mandatory(int b, int X, int n_sink, int n_recent) {
    return b < n_sink || b >= X - n_recent;
}

__device__ __forceinline__ int lanes_below(unsigned long long mask) {
    const int lane = threadIdx.x & 63;
    return __popcll(mask & ((1ull << lane) - 1ull));
}

template <int D, int G>
struct SelectShared {
    float q[G][D];     // scaled query
    float Qv[G][D];    // s^2 * sum of q^2 over each group (first r entries)
    float z[G][kBpcMax];
    float v[G][kBpcMax];
    float lse[G];
    int hist[kHistBins];
    int cnt[4], cnt2[4];
    int scan[4];
    int digit, above, last;
};

template <int D, int G>
__global__ __launch_bounds__(kThreads) void score_chunks_kernel(Geom geo, ScoreArgs a) {
    constexpr int NF4 = D / 32;  // float4 of the mean-key row per lane
    __shared__ SelectShared<D, G> sh;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u = blockIdx.y, chunk = blockIdx.x;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int n = clamp_len(a.seq_lens[bseq], geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    const int xmax = geo.xmax();
    const float s = a.scale;
    const int chunk0 = chunk * a.bpc;
    const int P = a.bpc / 32;
    const int li = tid & 7, grp = tid >> 3;

    // ---- phase 1: issue the summary loads of this thread's blocks
    float4 kv[kPMax][NF4];
    float dv0[kPMax];
#pragma unroll
    for (int p = 0; p < kPMax; ++p) {
        const int b = chunk0 + p * 32 + grp;
        const bool valid = p < P && b < X;
        const size_t blk = (size_t)u * geo.xcap + b;
        const float4* kp = reinterpret_cast<const float4*>(a.kmean + blk * D);
#pragma unroll
        for (int m = 0; m < NF4; ++m) kv[p][m] = valid ? kp[li + 8 * m] : make_float4(0, 0, 0, 0);
        dv0[p] = (valid && li < geo.r) ? a.dvar[blk * geo.r + li] : 0.0f;
    }
    const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    for (int idx = tid; idx < G * D; idx += kThreads) sh.q[idx / D][idx % D] = s * bf16_at(qh + idx);
    for (int idx = tid; idx < G * geo.r; idx += kThreads) {
        const int g = idx / geo.r, t = idx % geo.r;
        // Q_{g,t}: sum of q^2 over group t (Appendix A.4), times s^2
        float acc = 0.0f;
        if (geo.r == D) {
            const float qv = bf16_at(qh + g * D + t);
            acc = qv * qv;
        } else {
            const int w = (D / 2) / geo.r;
            for (int k = 0; k < 2 * w; ++k) {
                const int i = geo.layout == 0 ? (k < w ? t * w + k : D / 2 + t * w + (k - w)) : 2 * t * w + k;
                const float qv = bf16_at(qh + g * D + i);
                acc += qv * qv;
            }
        }
        sh.Qv[g][t] = s * s * acc;
    }
    __syncthreads();

#pragma unroll
    for (int p = 0; p < kPMax; ++p) {
        if (p >= P) break;
        const int lb = p * 32 + grp;
        const int b = chunk0 + lb;
        const bool valid = b < X;
        float z[G], v[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float acc = 0.0f;
#pragma unroll
            for (int m = 0; m < NF4; ++m) {
                const float* qq = &sh.q[g][4 * (li + 8 * m)];
                acc += qq[0] * kv[p][m].x + qq[1] * kv[p][m].y + qq[2] * kv[p][m].z + qq[3] * kv[p][m].w;
            }
            z[g] = acc;
            v[g] = li < geo.r ? sh.Qv[g][li] * dv0[p] : 0.0f;
        }
        if (geo.r > 8 && valid) {
            const size_t blk = (size_t)u * geo.xcap + b;
            for (int t = li + 8; t < geo.r; t += 8) {
                const float dv = a.dvar[blk * geo.r + t];
#pragma unroll
                for (int g = 0; g < G; ++g) v[g] += sh.Qv[g][t] * dv;
            }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
            z[g] = sum8(z[g]);
            v[g] = sum8(v[g]);
        }
        if (li == 0) {
#pragma unroll
            for (int g = 0; g < G; ++g) {
                sh.z[g][lb] = valid ? z[g] : 0.0f;
                sh.v[g][lb] = valid ? v[g] : 0.0f;
            }
        }
    }
    __syncthreads();
    // coalesced stores of the chunk's rows, and the chunk's per-head (max, sum exp)
    const int nvalid = max(0, min(a.bpc, X - chunk0));
    for (int idx = tid; idx < G * nvalid; idx += kThreads) {
        const int g = idx / nvalid, lb = idx % nvalid, b = chunk0 + lb;
        const float lnb = logf((float)min(geo.B, n - b * geo.B));
        const float av = lnb + sh.z[g][lb] + 0.5f * sh.v[g][lb];
        a.ws_a[((size_t)u * G + g) * xmax + b] = av;
        a.ws_v[((size_t)u * G + g) * xmax + b] = sh.v[g][lb];
        a.blk_logit[((size_t)u * G + g) * geo.xcap + b] = sh.z[g][lb];
    }
    for (int g = wave; g < G; g += 4) {
        float m = -INFINITY;
        float av[kBpcMax / 64];
#pragma unroll
        for (int k = 0; k < kBpcMax / 64; ++k) {
            const int lb = lane + 64 * k;
            av[k] = -INFINITY;
            if (lb < nvalid) {
                const int b = chunk0 + lb;
                av[k] = logf((float)min(geo.B, n - b * geo.B)) + sh.z[g][lb] + 0.5f * sh.v[g][lb];
            }
            m = fmaxf(m, av[k]);
        }
        m = wave_max(m);
        float ssum = 0.0f;
        if (m != -INFINITY) {
#pragma unroll
            for (int k = 0; k < kBpcMax / 64; ++k) ssum += (av[k] == -INFINITY) ? 0.0f : expf(av[k] - m);
        }
        ssum = wave_sum(ssum);
        if (lane == 0) {
            float* pp = a.ws_part + (((size_t)u * a.nchunks + chunk) * G + g) * 2;
            pp[0] = m;
            pp[1] = ssum;
        }
    }

}

// Phase 2: one workgroup per unit, after every chunk of the unit has been written.
template <int D, int G>
__global__ __launch_bounds__(kThreads) void select_finalize_kernel(Geom geo, ScoreArgs a) {
    __shared__ SelectShared<D, G> sh;
    extern __shared__ uint32_t dyn[];  // chunk partials, then score bits
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u = blockIdx.x;
    const int bseq = u / geo.hkv;
    const int n = clamp_len(a.seq_lens[bseq], geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    const int xmax = geo.xmax();

    // ---- phase 2a: per-head log normalizer over every block
    float* part = reinterpret_cast<float*>(dyn);
    const float* pu = a.ws_part + (size_t)u * a.nchunks * G * 2;
    for (int idx = tid; idx < a.nchunks * G * 2; idx += kThreads) part[idx] = pu[idx];
    __syncthreads();
    for (int g = wave; g < G; g += 4) {
        float m = -INFINITY;
        for (int c = lane; c < a.nchunks; c += 64) m = fmaxf(m, part[(c * G + g) * 2]);
        m = wave_max(m);
        float l = 0.0f;
        for (int c = lane; c < a.nchunks; c += 64) {
            const float pm = part[(c * G + g) * 2];
            if (pm != -INFINITY) l += part[(c * G + g) * 2 + 1] * expf(pm - m);
        }
        l = wave_sum(l);
        if (lane == 0) sh.lse[g] = m + logf(l);
    }
    __syncthreads();

    // ---- phase 2b: scores S_b and their bits
    uint32_t* keys = a.keys_in_lds ? dyn : a.ws_key + (size_t)u * xmax;
    for (int b = tid; b < X; b += kThreads) {
        float av[G], vv[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const size_t o = ((size_t)u * G + g) * xmax + b;
            av[g] = a.ws_a[o];
            vv[g] = a.ws_v[o];
        }
        float S = 0.0f;
#pragma unroll
        for (int g = 0; g < G; ++g) S += expf(av[g] - sh.lse[g]) * vv[g];
        if (a.scores) a.scores[(size_t)u * geo.xcap + b] = S;
        keys[b] = __float_as_uint(S);
    }
    __syncthreads();

    // ---- phase 2c: threshold of the Top-(K-|F|) among non-mandatory blocks
    const int K = a.K;
    const bool take_all = K >= X;
    int n_mand;
    {
        const int sink = min(a.n_sink, X);
        const int rec_lo = max(X - a.n_recent, 0);
        n_mand = sink + (X - rec_lo) - max(0, sink - rec_lo);
    }
    const int kk = take_all ? 0 : K - n_mand;  // >= 0: the host checks K >= n_sink + n_recent
    uint32_t thr = 0xFFFFFFFFu;                // keys above thr are taken; keys equal to thr up to need_eq
    int need_eq = 0;
    if (!take_all && kk > 0) {
        uint32_t prefix = 0, pmask = 0;
        int remaining = kk;
#pragma unroll
        for (int pass = 0; pass < 3; ++pass) {
            const int shft = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
            const uint32_t dmask = pass == 2 ? 0x3FFu : 0x7FFu;
            for (int i = tid; i < kHistBins; i += kThreads) sh.hist[i] = 0;
            __syncthreads();
            for (int b = tid; b < X; b += kThreads) {
                if (mandatory(b, X, a.n_sink, a.n_recent)) continue;
                const uint32_t key = keys[b];
                if ((key & pmask) == prefix) atomicAdd(&sh.hist[(key >> shft) & dmask], 1);
            }
            __syncthreads();
            // suffix counts: thread t owns bins [8t, 8t + 8)
            int local = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e) local += sh.hist[tid * 8 + e];
            int incl = local;  // inclusive suffix sum within the wave (higher lanes own higher bins)
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int o = __shfl_down(incl, off);
                if (lane + off < 64) incl += o;
            }
            if (lane == 0) sh.scan[wave] = incl;
            __syncthreads();
            int cum = incl - local;
            for (int w = wave + 1; w < 4; ++w) cum += sh.scan[w];
            for (int e = 7; e >= 0; --e) {
                const int c = sh.hist[tid * 8 + e];
                if (cum < remaining && cum + c >= remaining) {
                    sh.digit = tid * 8 + e;
                    sh.above = cum;
                }
                cum += c;
            }
            __syncthreads();
            remaining -= sh.above;
            prefix |= (uint32_t)sh.digit << shft;
            pmask |= dmask << shft;
            __syncthreads();
        }
        thr = prefix;
        need_eq = remaining;
    }

    // ---- phase 2d: mark and compact in ascending id order; wave w scans its own id segment
    const int seg = ((X + 3) / 4 + 63) / 64 * 64;
    const int s0 = min(X, wave * seg), s1 = min(X, s0 + seg);
    const bool ranked = !take_all && kk > 0;
    int cnt_eq = 0;
    for (int base = s0; base < s1; base += 64) {
        const int b = base + lane;
        const bool eq = ranked && b < s1 && !mandatory(b, X, a.n_sink, a.n_recent) && keys[b] == thr;
        cnt_eq += __popcll(__ballot(eq));
    }
    if (lane == 0) sh.cnt[wave] = cnt_eq;
    __syncthreads();
    int eq_run = 0;
    for (int w = 0; w < wave; ++w) eq_run += sh.cnt[w];
    const int eq_before = eq_run;
    int cnt_take = 0;
    for (int base = s0; base < s1; base += 64) {
        const int b = base + lane;
        const bool in = b < s1;
        const bool mand = in && mandatory(b, X, a.n_sink, a.n_recent);
        const uint32_t key = in ? keys[b] : 0u;
        const bool cand = in && !mand && ranked;
        const bool eq = cand && key == thr;
        const unsigned long long em = __ballot(eq);
        const bool take = in && (take_all || mand || (cand && (key > thr || (eq && eq_run + lanes_below(em) < need_eq))));
        eq_run += __popcll(em);
        cnt_take += __popcll(__ballot(take));
    }
    if (lane == 0) sh.cnt2[wave] = cnt_take;
    __syncthreads();
    int pos = 0;
    for (int w = 0; w < wave; ++w) pos += sh.cnt2[w];
    int total = 0;
    for (int w = 0; w < 4; ++w) total += sh.cnt2[w];
    eq_run = eq_before;
    int32_t* sel = a.sel + (size_t)u * K;
    for (int base = s0; base < s1; base += 64) {
        const int b = base + lane;
        const bool in = b < s1;
        const bool mand = in && mandatory(b, X, a.n_sink, a.n_recent);
        const uint32_t key = in ? keys[b] : 0u;
        const bool cand = in && !mand && ranked;
        const bool eq = cand && key == thr;
        const unsigned long long em = __ballot(eq);
        const bool take = in && (take_all || mand || (cand && (key > thr || (eq && eq_run + lanes_below(em) < need_eq))));
        eq_run += __popcll(em);
        const unsigned long long tm = __ballot(take);
        const int p = pos + lanes_below(tm);
        if (take && p < K) sel[p] = b;
        pos += __popcll(tm);
    }
    for (int k = total + tid; k < K; k += kThreads) sel[k] = -1;
    if (tid == 0) a.n_sel[u] = min(total, K);
}

template <int D, int G>
hipError_t launch_pair(const Geom& g, const ScoreArgs& a, hipStream_t s, size_t dyn) {
    score_chunks_kernel<D, G><<<dim3(a.nchunks, g.units()), kThreads, 0, s>>>(g, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    select_finalize_kernel<D, G><<<dim3(g.units()), kThreads, dyn, s>>>(g, a);
    return hipGetLastError();
}

template <int D>
hipError_t dispatch_g(const Geom& g, const ScoreArgs& a, hipStream_t s, size_t dyn) {
    switch (g.G) {
        case 1: return launch_pair<D, 1>(g, a, s, dyn);
        case 2: return launch_pair<D, 2>(g, a, s, dyn);
        case 4: return launch_pair<D, 4>(g, a, s, dyn);
        case 8: return launch_pair<D, 8>(g, a, s, dyn);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

int select_max_bpc() { return kBpcMax; }

size_t select_dyn_lds(const Geom& g, const ScoreArgs& a) {
    const size_t part = (size_t)a.nchunks * g.G * 2 * sizeof(float);
    const size_t keys = a.keys_in_lds ? (size_t)g.xmax() * sizeof(uint32_t) : 0;
    return part > keys ? part : keys;
}

hipError_t launch_score_select(const Geom& g, ScoreArgs a, hipStream_t s) {
    if (a.bpc % 32 != 0 || a.bpc > kBpcMax || a.bpc < 32) return hipErrorInvalidValue;
    constexpr size_t kDynBudget = 32768;  // LDS beyond the static part, per workgroup
    a.keys_in_lds = (size_t)g.xmax() * sizeof(uint32_t) <= kDynBudget;
    const size_t dyn = select_dyn_lds(g, a);
    if (dyn > kDynBudget) return hipErrorInvalidValue;
    return g.D == 128 ? dispatch_g<128>(g, a, s, dyn) : dispatch_g<64>(g, a, s, dyn);
}

}  // namespace compkv

// select.hip -- block scoring and Top-K selection in one launch (Sections 4.1, 4.2; Appendix E.1).
//
// grid = (nchunks, units). Phase 1: each workgroup streams the fp32 summaries (mean key, grouped
// variances) of `bpc` consecutive blocks of one unit. Eight lanes share a block: lane i of the eight
// reads float4 i, i+8, ... of the mean-key row, so the eight lanes read 128 contiguous bytes per load,
// and lane i also takes the variance groups t = i, i+8, .... For each of the unit's G query heads it
// forms the block-mean logit zbar = s q.kmean, the projected variance sig2 = s^2 sum_t Q_t dvar_t and
// the log weight estimate a = log|b| + zbar + sig2/2 (Eq. compkv-mass-estimate's numerator), stores
// them, and writes the chunk's per-head (max a, sum exp(a - max)).
//
// Phase 2 runs in the last workgroup of the unit to arrive (an atomic ticket; no workgroup ever waits
// for another): it merges the chunk partials in chunk order into each head's log normalizer, forms
// S_b = sum_g exp(a - lse_g) sig2 (Eq. compkv-score), finds the (K-|F|)-th largest score among the
// non-mandatory blocks with a three-pass radix select on the score bits (scores are >= 0, so their
// IEEE bit patterns order like the values), and writes the selected ids in ascending order. Equal
// scores are taken in ascending id order, which is the stable Top-K the paper specifies.
#include "internal.h"

namespace compkv {
namespace {

constexpr int kBpcMax = 256;   // blocks per chunk, upper bound
constexpr int kHistBins = 2048;

struct ScanShared {
    int wave_cnt[4];
    int digit, above;
};

// Exclusive count of `flag` over threads of the workgroup (in thread order) and the total.
__device__ __forceinline__ int block_exclusive_count(bool flag, int* total, int* sh_cnt) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const unsigned long long mask = __ballot(flag);
    const int before = __popcll(mask & ((1ull << lane) - 1ull));
    if (lane == 0) sh_cnt[wave] = __popcll(mask);
    __syncthreads();
    int base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const int c = sh_cnt[w];
        base += (w < wave) ? c : 0;
        tot += c;
    }
    __syncthreads();
    *total = tot;
    return base + before;
}

__device__ __forceinline__ bool mandatory(int b, int X, int n_sink, int n_recent) {
    return b < n_sink || b >= X - n_recent;
}

template <int D, int G>
__global__ __launch_bounds__(kThreads) void score_select_kernel(Geom geo, ScoreArgs a) {
    constexpr int NF4 = D / 32;  // float4 of the mean-key row per lane
    __shared__ float sh_q[G][D];
    __shared__ float sh_Qv[G][D];
    __shared__ float sh_a[G][kBpcMax];
    __shared__ float sh_lse[G];
    __shared__ int sh_hist[kHistBins];
    __shared__ int sh_cnt[4];
    __shared__ int sh_scan[4];
    __shared__ int sh_digit, sh_above, sh_last;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u = blockIdx.y, chunk = blockIdx.x;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int n = clamp_len(a.seq_lens[bseq], geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    const int xmax = geo.xmax();
    const float s = a.scale;

    // ---- phase 1: block statistics of this chunk
    const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    for (int idx = tid; idx < G * D; idx += kThreads) sh_q[idx / D][idx % D] = s * bf16_at(qh + idx);
    __syncthreads();
    for (int idx = tid; idx < G * geo.r; idx += kThreads) {
        const int g = idx / geo.r, t = idx % geo.r;
        // Q_{g,t} = sum of q^2 over group t (Appendix A.4), times s^2
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
        sh_Qv[g][t] = s * s * acc;
    }
    __syncthreads();

    const int li = tid & 7;
    float qreg[G][NF4][4];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int m = 0; m < NF4; ++m)
#pragma unroll
            for (int e = 0; e < 4; ++e) qreg[g][m][e] = sh_q[g][4 * (li + 8 * m) + e];

    const int chunk0 = chunk * a.bpc;
    for (int pass = 0; pass < a.bpc / 32; ++pass) {
        const int lb = pass * 32 + (tid >> 3);
        const int b = chunk0 + lb;
        const bool valid = b < X;
        float z[G], v[G];
#pragma unroll
        for (int g = 0; g < G; ++g) z[g] = v[g] = 0.0f;
        if (valid) {
            const size_t blk = (size_t)u * geo.xcap + b;
            const float4* kp = reinterpret_cast<const float4*>(a.kmean + blk * D);
#pragma unroll
            for (int m = 0; m < NF4; ++m) {
                const float4 k4 = kp[li + 8 * m];
#pragma unroll
                for (int g = 0; g < G; ++g)
                    z[g] += qreg[g][m][0] * k4.x + qreg[g][m][1] * k4.y + qreg[g][m][2] * k4.z +
                            qreg[g][m][3] * k4.w;
            }
            for (int t = li; t < geo.r; t += 8) {
                const float dv = a.dvar[blk * geo.r + t];
#pragma unroll
                for (int g = 0; g < G; ++g) v[g] += sh_Qv[g][t] * dv;
            }
        }
#pragma unroll
        for (int off = 1; off < 8; off <<= 1)
#pragma unroll
            for (int g = 0; g < G; ++g) {
                z[g] += __shfl_xor(z[g], off);
                v[g] += __shfl_xor(v[g], off);
            }
        const float lnb = valid ? logf((float)min(geo.B, n - b * geo.B)) : 0.0f;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            if ((g & 7) != li) continue;
            if (valid) {
                const float av = lnb + z[g] + 0.5f * v[g];
                a.ws_a[((size_t)u * G + g) * xmax + b] = av;
                a.ws_v[((size_t)u * G + g) * xmax + b] = v[g];
                a.blk_logit[((size_t)u * G + g) * geo.xcap + b] = z[g];
                sh_a[g][lb] = av;
            } else {
                sh_a[g][lb] = -INFINITY;
            }
        }
    }
    __syncthreads();
    for (int g = wave; g < G; g += 4) {
        float m = -INFINITY;
        for (int i = lane; i < a.bpc; i += 64) m = fmaxf(m, sh_a[g][i]);
        m = wave_max(m);
        float ssum = 0.0f;
        if (m != -INFINITY)
            for (int i = lane; i < a.bpc; i += 64) ssum += (sh_a[g][i] == -INFINITY) ? 0.0f : expf(sh_a[g][i] - m);
        ssum = wave_sum(ssum);
        if (lane == 0) {
            float* p = a.ws_part + (((size_t)u * a.nchunks + chunk) * G + g) * 2;
            p[0] = m;
            p[1] = ssum;
        }
    }

    // ---- arrival ticket: the last chunk of the unit finishes the selection
    __threadfence();
    __syncthreads();
    if (tid == 0) sh_last = (atomicAdd(&a.counters[u], 1u) == (unsigned)(gridDim.x - 1));
    __syncthreads();
    if (!sh_last) return;
    __threadfence();

    // ---- phase 2a: per-head log normalizer over every block (chunk order)
    if (tid < G) {
        float m = -INFINITY, l = 0.0f;
        for (int c = 0; c < a.nchunks; ++c) {
            const float* p = a.ws_part + (((size_t)u * a.nchunks + c) * G + tid) * 2;
            const float pm = p[0], pl = p[1];
            if (pm == -INFINITY) continue;
            if (pm > m) {
                l = l * expf(m - pm) + pl;
                m = pm;
            } else {
                l += pl * expf(pm - m);
            }
        }
        sh_lse[tid] = m + logf(l);
    }
    __syncthreads();

    // ---- phase 2b: scores S_b and their bits
    uint32_t* keys = a.ws_key + (size_t)u * xmax;
    for (int b = tid; b < X; b += kThreads) {
        float S = 0.0f;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const size_t o = ((size_t)u * G + g) * xmax + b;
            S += expf(a.ws_a[o] - sh_lse[g]) * a.ws_v[o];
        }
        if (a.scores) a.scores[(size_t)u * geo.xcap + b] = S;
        keys[b] = __float_as_uint(S);
    }
    __syncthreads();

    // ---- phase 2c: threshold of the Top-(K-|F|) among non-mandatory blocks
    const int K = a.K;
    const bool take_all = K >= X;
    int n_mand = 0;
    {
        const int sink = min(a.n_sink, X);
        const int rec_lo = max(X - a.n_recent, 0);
        n_mand = sink + (X - rec_lo) - max(0, sink - rec_lo);
    }
    const int kk = take_all ? 0 : K - n_mand;  // >= 0: the host checks K >= n_sink + n_recent
    uint32_t thr = 0xFFFFFFFFu;                // keys > thr are taken; keys == thr up to need_eq
    int need_eq = 0;
    if (!take_all && kk > 0) {
        uint32_t prefix = 0, pmask = 0;
        int remaining = kk;
        const int shifts[3] = {21, 10, 0};
        const int widths[3] = {11, 11, 10};
        for (int pass = 0; pass < 3; ++pass) {
            const int sh = shifts[pass];
            const uint32_t dmask = (1u << widths[pass]) - 1u;
            for (int i = tid; i < kHistBins; i += kThreads) sh_hist[i] = 0;
            __syncthreads();
            for (int b = tid; b < X; b += kThreads) {
                if (mandatory(b, X, a.n_sink, a.n_recent)) continue;
                const uint32_t key = keys[b];
                if ((key & pmask) == prefix) atomicAdd(&sh_hist[(key >> sh) & dmask], 1);
            }
            __syncthreads();
            // suffix counts: thread t owns bins [8t, 8t + 8)
            int local = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e) local += sh_hist[tid * 8 + e];
            int incl = local;  // inclusive suffix sum within the wave (higher lanes own higher bins)
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int o = __shfl_down(incl, off);
                if (lane + off < 64) incl += o;
            }
            if (lane == 0) sh_scan[wave] = incl;
            __syncthreads();
            int above = incl - local;
            for (int w = wave + 1; w < 4; ++w) above += sh_scan[w];
            int cum = above;
            for (int e = 7; e >= 0; --e) {
                const int c = sh_hist[tid * 8 + e];
                if (cum < remaining && cum + c >= remaining) {
                    sh_digit = tid * 8 + e;
                    sh_above = cum;
                }
                cum += c;
            }
            __syncthreads();
            remaining -= sh_above;
            prefix |= (uint32_t)sh_digit << sh;
            pmask |= dmask << sh;
            __syncthreads();
        }
        thr = prefix;
        need_eq = remaining;
    }

    // ---- phase 2d: mark and compact in ascending id order
    int32_t* sel = a.sel + (size_t)u * K;
    int run_eq = 0, run_sel = 0;
    for (int base = 0; base < X; base += kThreads) {
        const int b = base + tid;
        const bool valid = b < X;
        const bool mand = valid && mandatory(b, X, a.n_sink, a.n_recent);
        const uint32_t key = valid ? keys[b] : 0u;
        const bool cand = valid && !mand && !take_all && kk > 0;
        const bool eq = cand && key == thr;
        int tot_eq;
        const int eq_rank = block_exclusive_count(eq, &tot_eq, sh_cnt);
        const bool take = valid && (take_all || mand || (cand && (key > thr || (eq && run_eq + eq_rank < need_eq))));
        int tot_take;
        const int pos = block_exclusive_count(take, &tot_take, sh_cnt);
        if (take && run_sel + pos < K) sel[run_sel + pos] = b;
        run_eq += tot_eq;
        run_sel += tot_take;
    }
    for (int k = run_sel + tid; k < K; k += kThreads) sel[k] = -1;
    if (tid == 0) {
        a.n_sel[u] = run_sel;
        a.counters[u] = 0u;  // leave the counter ready for the next call
    }
}

template <int D>
hipError_t dispatch_g(const Geom& g, const ScoreArgs& a, hipStream_t s, dim3 grid) {
    switch (g.G) {
        case 1: score_select_kernel<D, 1><<<grid, kThreads, 0, s>>>(g, a); break;
        case 2: score_select_kernel<D, 2><<<grid, kThreads, 0, s>>>(g, a); break;
        case 4: score_select_kernel<D, 4><<<grid, kThreads, 0, s>>>(g, a); break;
        case 8: score_select_kernel<D, 8><<<grid, kThreads, 0, s>>>(g, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_score_select(const Geom& g, const ScoreArgs& a, hipStream_t s) {
    if (a.bpc % 32 != 0 || a.bpc > kBpcMax) return hipErrorInvalidValue;
    dim3 grid(a.nchunks, g.units());
    return g.D == 128 ? dispatch_g<128>(g, a, s, grid) : dispatch_g<64>(g, a, s, grid);
}

}  // namespace compkv

// select_core.h -- pieces of the scoring, selection and fused decode kernels shared by select.hip and
// step.hip (private to libcompkv): query preparation, score kinds, the Top-K selection of one unit
// from chunk partials, the compensation stream of mean values and the in-launch merge of partials.
#pragma once

#include "block_stats.h"
#include "exact.h"

#include <type_traits>

namespace compkv {
namespace {

constexpr int kBpcMax = 128;  // blocks per chunk, upper bound
constexpr int kHistBins = 2048;
constexpr size_t kDynBudget = 32768;  // dynamic LDS of the finalize launch
constexpr int kUnitTerms = 8192;      // G * xmax bound of the one-workgroup-per-unit path (64 KB of LDS)

// The query enters through frequency pairs (Appendix A.4): lane f of wave w holds pair f of heads
// g = w, w + 4, ... (coordinates f, f + d/2 for rotate-half; 2f, 2f + 1 interleaved). The loads are
// issued before the summaries' so that waiting for them never waits for the summaries.
template <int D, int G>
struct QueryPairs {
    static constexpr int J = (G + 3) / 4;
    uint16_t xa[J], xb[J];
};

__device__ __forceinline__ int pair_a(int f, int layout) { return layout == 0 ? f : 2 * f; }
__device__ __forceinline__ int pair_b(int f, int layout, int D) { return layout == 0 ? f + D / 2 : 2 * f + 1; }

template <int D, int G>
__device__ __forceinline__ void load_query_pairs(const uint16_t* qh, int layout, QueryPairs<D, G>& qp) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int f = lane < D / 2 ? lane : 0;
#pragma unroll
    for (int j = 0; j < QueryPairs<D, G>::J; ++j) {
        const int g = wave + 4 * j < G ? wave + 4 * j : 0;  // branch-free: unused when past G
        qp.xa[j] = qh[g * D + pair_a(f, layout)];
        qp.xb[j] = qh[g * D + pair_b(f, layout, D)];
    }
}

// From the loaded pairs: the scaled query s q into q (nullable) and s^2 Q_{g,t} -- the squared scaled
// coordinates summed over group t -- into Qv[g][t]. A group is a run of (d/2)/r consecutive pairs,
// summed by butterflies; with r == d every coordinate is its own group.
template <int D, int G>
__device__ __forceinline__ void store_query(const QueryPairs<D, G>& qp, float s, int r, int layout, float (*q)[D],
                                            float (*Qv)[D]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const bool in = lane < D / 2;
    const int ia = pair_a(in ? lane : 0, layout), ib = pair_b(in ? lane : 0, layout, D);
#pragma unroll
    for (int j = 0; j < QueryPairs<D, G>::J; ++j) {
        const int g = wave + 4 * j;
        if (g >= G) break;  // wave-uniform
        const float xa = s * bf16_at(&qp.xa[j]), xb = s * bf16_at(&qp.xb[j]);
        if (q && in) {
            q[g][ia] = xa;
            q[g][ib] = xb;
        }
        if (r == D) {
            if (in) {
                Qv[g][ia] = xa * xa;
                Qv[g][ib] = xb * xb;
            }
            continue;
        }
        float e = in ? xa * xa + xb * xb : 0.0f;
        const int w = (D / 2) / r;
        for (int off = 1; off < w; off <<= 1) e = xor_add(e, off);
        if (in && lane % w == 0) Qv[g][lane / w] = e;
    }
}

// Score kinds (the ablations of Section 5.4): the log weight of a block is
// log|b| + zbar + half * sig2 (half = 1/2, or 0 for the first-order mass estimate), and its score
// term is p-hat * sig2, or p-hat alone for the mass-only score.
__device__ __forceinline__ float kind_half(int kind) { return kind == 2 ? 0.0f : 0.5f; }
__device__ __forceinline__ float kind_term(int kind, float sig2) { return kind == 1 ? 1.0f : sig2; }

constexpr int kFinThreads = 1024;  // threads of the selection workgroup (one per unit)
constexpr int kFinWaves = kFinThreads / 64;
constexpr int kKeysPerThread = 8;  // fast path: up to 8192 keys in registers
constexpr int kBitmapWords = kKeysPerThread * kFinThreads / 32;
constexpr int kCandCap = 1024;     // candidates ranked by brute force on the fast path
constexpr int kHistTail = 255;     // distance bins counted on the fast path (bin 255 = everything farther)

struct FinalShared {
    float qv[8 * 4];  // logit terms: s^2 Q_{g,t} (G <= 8 heads, r = 4 groups)
    float lse[8];     // logit terms: each head's log normalizer
    int hist[kHistBins];
    uint32_t wmax[kFinWaves];
    int cnt[kFinWaves], cnt2[kFinWaves];
    int digit, above, beta, ncand;
    unsigned long long cand[kCandCap];
    uint32_t bitmap[kBitmapWords];
};

// bits [lo, hi) of the 32-bit word holding ids base .. base + 31
__device__ __forceinline__ uint32_t range_bits(int lo, int hi, int base) {
    const int l = max(lo - base, 0), r = min(hi - base, 32);
    if (l >= r) return 0u;
    const uint32_t upto = r == 32 ? 0xFFFFFFFFu : ((1u << r) - 1u);
    return upto & ~((1u << l) - 1u);
}

// score terms of block b (G floats, contiguous). kCoh: device-coherent loads (terms written by other
// workgroups of the same launch).
template <int G, bool kCoh = false>
__device__ __forceinline__ void load_terms(const float* wu, int b, float (&w)[G]) {
    if constexpr (G % 4 == 0) {
#pragma unroll
        for (int g4 = 0; g4 < G; g4 += 4) {
            const float* tp = wu + (size_t)b * G + g4;
            const float4 t4 = kCoh ? ld_agent4(tp) : *reinterpret_cast<const float4*>(tp);
            w[g4] = t4.x;
            w[g4 + 1] = t4.y;
            w[g4 + 2] = t4.z;
            w[g4 + 3] = t4.w;
        }
    } else {
#pragma unroll
        for (int g = 0; g < G; ++g) w[g] = kCoh ? ld_agent(wu + (size_t)b * G + g) : wu[(size_t)b * G + g];
    }
}

// Selection shared by the workgroups that rank one unit's blocks (kFinThreads threads, keys as in
// select_finalize_kernel).
struct SelectCtx {
    int X, K, kk, sink, rec_lo, n_sink, n_recent;
    bool take_all, ranked;
    int32_t* sel;    // this unit's row of selected ids
    int32_t* n_sel;  // this unit's count
    uint32_t* keys;  // [X] score bits, for the radix path
};

__device__ inline SelectCtx make_select_ctx(int X, int K, int n_sink, int n_recent, int32_t* sel, int32_t* n_sel,
                                            uint32_t* keys) {
    SelectCtx c;
    c.X = X;
    c.K = K;
    c.n_sink = n_sink;
    c.n_recent = n_recent;
    c.take_all = K >= X;
    c.sink = min(n_sink, X);
    c.rec_lo = max(X - n_recent, 0);
    const int n_mand = c.sink + (X - c.rec_lo) - max(0, c.sink - c.rec_lo);
    c.kk = c.take_all ? 0 : K - n_mand;  // >= 0: the host checks K >= n_sink + n_recent
    c.ranked = !c.take_all && c.kk > 0;
    c.sel = sel;
    c.n_sel = n_sel;
    c.keys = keys;
    return c;
}

// before the first barrier that precedes select_fast (any workgroup of at least 256 threads)
__device__ inline void select_init(FinalShared& sh) {
    const int tid = threadIdx.x;
    if (tid < kBitmapWords) sh.bitmap[tid] = 0u;
    if (tid <= kHistTail) sh.hist[tid] = 0;
    if (tid == 0) {
        sh.beta = kHistTail;
        sh.ncand = 0;
    }
}

// Fast path: the keys ck (each non-zero key held by exactly one thread; zero = no key) and this
// thread's largest score bits mx. Returns false when too many keys tie around the cut: their bits are
// then in c.keys and select_radix finishes.
template <int KPT, int FT = kFinThreads>
__device__ bool select_fast(const SelectCtx& ctx, const unsigned long long (&ck)[KPT], uint32_t mx, FinalShared& sh) {
    static_assert(FT >= kBitmapWords && FT <= kFinThreads && KPT * FT <= 32 * kBitmapWords, "selection shape");
    constexpr int NW = FT / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int X = ctx.X, K = ctx.K, kk = ctx.kk, sink = ctx.sink, rec_lo = ctx.rec_lo;
    const bool take_all = ctx.take_all, ranked = ctx.ranked;
    int32_t* sel = ctx.sel;
    uint32_t* keys = ctx.keys;
    int m = 0;  // candidates ranked exactly
    if (ranked) {
        mx = wave_max_u32(mx);
        if (lane == 0) sh.wmax[wave] = mx;
        __syncthreads();
        uint32_t smax = 0u;
#pragma unroll
        for (int w2 = 0; w2 < NW; ++w2) smax = max(smax, sh.wmax[w2]);
        // histogram of the keys' distance below the largest score, in bins of 2^19 float ulps (1/16
        // of an octave); keys more than 255 bins below are not counted
        uint32_t bin[KPT];
#pragma unroll
        for (int k = 0; k < KPT; ++k) {
            const uint32_t bits = (uint32_t)(ck[k] >> 32);
            bin[k] = ck[k] ? min((smax - bits) >> 19, (uint32_t)kHistTail) : 0xFFFFFFFFu;
            if (bin[k] < (uint32_t)kHistTail) atomicAdd(&sh.hist[bin[k]], 1);
        }
        __syncthreads();
        // every wave: prefix over the counted bins (four per lane); the bin reaching kk holds the cut (at
        // most one lane finds it; none: the cut lies below the counted range, beta = kHistTail)
        uint32_t beta;
        {
            int c[4], tot = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int bi = 4 * lane + e;
                c[e] = bi < kHistTail ? sh.hist[bi] : 0;
                tot += c[e];
            }
            int run = wave_incl_scan(tot) - tot;
            int cut = kHistTail;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (run < kk && run + c[e] >= kk) cut = 4 * lane + e;
                run += c[e];
            }
            const unsigned long long found = __ballot(cut != kHistTail);
            beta = found ? (uint32_t)__builtin_amdgcn_readlane(cut, (int)__builtin_ctzll(found)) : (uint32_t)kHistTail;
        }
        // candidates: keys in the cut's bin or above; each wave reserves its slots with one atomic
        int mine = 0;
#pragma unroll
        for (int k = 0; k < KPT; ++k) mine += bin[k] <= beta;
        const int incl = wave_incl_scan(mine);
        int base = 0;
        if (lane == 63) base = atomicAdd(&sh.ncand, incl);
        int off = __builtin_amdgcn_readlane(base, 63) + incl - mine;
#pragma unroll
        for (int k = 0; k < KPT; ++k) {
            if (bin[k] <= beta) {
                if (off < kCandCap) sh.cand[off] = ck[k];
                ++off;
            }
        }
        __syncthreads();
        m = sh.ncand;
        if (m <= kCandCap) {
            // exact rank among the candidates (order-independent); the kk best are selected. With
            // few candidates the four lanes of a quad share one.
            const int share = m <= FT / 4 ? 4 : 1;
            const int part = tid % share;
            for (int i = tid / share; i < m; i += FT / share) {  // quad-uniform
                const unsigned long long ci = sh.cand[i];
                int r = 0;
                int j = part;
                for (; j + 7 * share < m; j += 8 * share) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) r += sh.cand[j + e * share] > ci;
                }
                for (; j < m; j += share) r += sh.cand[j] > ci;
                if (share == 4) {
                    r += dpp_i<0xB1>(r, r);
                    r += dpp_i<0x4E>(r, r);
                }
                if (part == 0 && r < kk) {
                    const uint32_t b = 0xFFFFFFFFu - (uint32_t)(ci & 0xFFFFFFFFull);
                    atomicOr(&sh.bitmap[b >> 5], 1u << (b & 31));
                }
            }
        } else {
            // too many ties around the threshold: keep the bits for the radix path below
#pragma unroll
            for (int k = 0; k < KPT; ++k)
                if (ck[k]) keys[0xFFFFFFFFu - (uint32_t)(ck[k] & 0xFFFFFFFFull)] = (uint32_t)(ck[k] >> 32);
        }
        __syncthreads();
    }
    if (m <= kCandCap) {  // block-uniform
        // thread t < 256 owns ids 32t .. 32t+31: selected, mandatory (or every block when K >= X)
        uint32_t word = 0u;
        if (tid < kBitmapWords) {
            word = take_all ? range_bits(0, X, 32 * tid)
                            : (sh.bitmap[tid] | range_bits(0, sink, 32 * tid) | range_bits(rec_lo, X, 32 * tid));
        }
        const int c = __popc(word);
        const int incl = wave_incl_scan(c);
        if (lane == 63) sh.cnt[wave] = incl;
        __syncthreads();
        int pos = incl - c, total = 0;
#pragma unroll
        for (int w2 = 0; w2 < kBitmapWords / 64; ++w2) {
            pos += w2 < wave ? sh.cnt[w2] : 0;
            total += sh.cnt[w2];
        }
        while (word) {
            const int bit = __ffs(word) - 1;
            word &= word - 1;
            if (pos < K) sel[pos] = 32 * tid + bit;
            ++pos;
        }
        for (int k = total + tid; k < K; k += FT) sel[k] = -1;
        if (tid == 0) *ctx.n_sel = min(total, K);
        return true;
    }
    return false;
}

// General path: radix select on the key bits of blocks [0, X), then ascending compaction.
template <int FT = kFinThreads>
__device__ void select_radix(const SelectCtx& c, FinalShared& sh) {
    constexpr int NW = FT / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int X = c.X, K = c.K, kk = c.kk;
    const bool take_all = c.take_all, ranked = c.ranked;
    int32_t* sel = c.sel;
    const uint32_t* keys = c.keys;
    struct {
        int n_sink, n_recent;
    } a{c.n_sink, c.n_recent};
    __syncthreads();

    // ---- threshold of the Top-(K-|F|) among non-mandatory blocks (radix select on the score bits)
    uint32_t thr = 0xFFFFFFFFu;  // keys above thr are taken; keys equal to thr up to need_eq
    int need_eq = 0;
    if (ranked) {
        uint32_t prefix = 0, pmask = 0;
        int remaining = kk;
#pragma unroll
        for (int pass = 0; pass < 3; ++pass) {
            const int shft = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
            const uint32_t dmask = pass == 2 ? 0x3FFu : 0x7FFu;
            for (int i = tid; i < kHistBins; i += FT) sh.hist[i] = 0;
            __syncthreads();
            for (int b = tid; b < X; b += FT) {
                if (mandatory(b, X, a.n_sink, a.n_recent)) continue;
                const uint32_t key = keys[b];
                if ((key & pmask) == prefix) atomicAdd(&sh.hist[(key >> shft) & dmask], 1);
            }
            __syncthreads();
            // suffix counts: thread t < 256 owns bins [8t, 8t + 8)
            int local = 0;
            if (tid < kHistBins / 8) {
#pragma unroll
                for (int e = 0; e < 8; ++e) local += sh.hist[tid * 8 + e];
            }
            const int pre = wave_incl_scan(local);
            const int wtot = __builtin_amdgcn_readlane(pre, 63);
            const int incl = wtot - pre + local;  // over this lane and the higher ones (higher bins)
            if (lane == 0) sh.cnt[wave] = wtot;
            __syncthreads();
            if (tid < kHistBins / 8) {
                int cum = incl - local;
                for (int w2 = wave + 1; w2 < kHistBins / 8 / 64; ++w2) cum += sh.cnt[w2];
                for (int e = 7; e >= 0; --e) {
                    const int c = sh.hist[tid * 8 + e];
                    if (cum < remaining && cum + c >= remaining) {
                        sh.digit = tid * 8 + e;
                        sh.above = cum;
                    }
                    cum += c;
                }
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

    // ---- mark and compact in ascending id order; wave w scans its own id segment
    const int seg = ((X + NW - 1) / NW + 63) / 64 * 64;
    const int s0 = min(X, wave * seg), s1 = min(X, s0 + seg);
    int cnt_eq = 0;
    for (int base = s0; base < s1; base += 64) {
        const int b = base + lane;
        const bool eq = ranked && b < s1 && !mandatory(b, X, a.n_sink, a.n_recent) && keys[b] == thr;
        cnt_eq += __popcll(__ballot(eq));
    }
    if (lane == 0) sh.cnt[wave] = cnt_eq;
    __syncthreads();
    int eq_run = 0;
    for (int w2 = 0; w2 < wave; ++w2) eq_run += sh.cnt[w2];
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
    for (int w2 = 0; w2 < wave; ++w2) pos += sh.cnt2[w2];
    int total = 0;
    for (int w2 = 0; w2 < NW; ++w2) total += sh.cnt2[w2];
    eq_run = eq_before;
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
    for (int k = total + tid; k < K; k += FT) sel[k] = -1;
    if (tid == 0) *c.n_sel = min(total, K);
}

// The selection of unit u from the chunk partials (kFinThreads threads): per-head log normalizers,
// scores (written to a.scores when write_scores) and the stable Top-K into sel_out / nsel_out (global
// or LDS). dyn: [np][G] partial maxima, then factors; [np][G] sums; [xmax] key bits (keys_in_lds).
// kCoh: the partials and terms were written by other workgroups of the same launch (device-coherent
// loads; the values of blocks past the unit's, loaded only to keep the loads in flight fixed, go unused).
// FT threads holding up to KPT keys each (the terms of the first eight requested up front, the rest
// once the normalizers are formed).
// kLogits (a.logit_terms, G >= 4, r = 4, at most 4096 blocks): block b's terms are formed here from
// zbar (a.zlog), its variances (dvar) and the query's group sums (a.ws_qv): sig2_{g,b} = sum_t
// s^2 Q_{g,t} D_{b,t}, a_{g,b} = log|b| + zbar_{g,b} + half * sig2_{g,b}, and S_b = sum_g
// exp(a_{g,b} - lse_g) * term(sig2_{g,b}), with lse_g from the chunk partials as above.
template <int G, bool kCoh = false, int FT = kFinThreads, int KPT = kKeysPerThread, bool kLogits = false>
__device__ void finalize_select(const Geom& geo, const ScoreArgs& a, int u, FinalShared& sh, float* dyn,
                                int32_t* sel_out, int32_t* nsel_out, bool write_scores) {
    static_assert(!kLogits || (G >= 4 && G <= 8 && !kCoh && KPT <= 4), "logit terms: four to eight heads, one "
                                                                         "launch apart, at most 4096 blocks");
    constexpr int KB = KPT < 8 ? KPT : 8;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bseq = u / geo.hkv;
    const int xmax = geo.xmax();
    const int nc = a.nchunks, np = nc + 1;  // partial nc: the last block's
    const float* wu = a.ws_w + (size_t)u * xmax * G;
    const bool fast = xmax <= KPT * FT;

    // ---- loads in the order of their use: the length, the partials, this thread's score terms. Every
    // load is issued, also where its value goes unused (a clamped address instead), so that the count
    // of loads in flight is fixed and each wait below is for the loads it needs.
    int n_raw = a.seq_lens[bseq];
    float* fac = dyn;
    float* sums = dyn + np * G;
    const bool one_pass = np * G <= FT;  // usual case: one partial per thread
    float2 pv = make_float2(0.0f, 0.0f);
    if (one_pass) {  // (workgroup-uniform)
        const float* pp = a.ws_part + ((size_t)u * np * G + (tid < np * G ? tid : 0)) * 2;
        pv = kCoh ? ld_agent2(pp) : *reinterpret_cast<const float2*>(pp);
    }
    float qv = 0.0f;
    if constexpr (kLogits) qv = a.ws_qv[(size_t)u * G * 4 + (tid < G * 4 ? tid : 0)];
    __asm__ volatile("" ::: "memory");
    // score terms (or, kLogits, zbar of each head and the block's four variances)
    float w[KB][G];
    float4 dvk[kLogits ? KB : 1];
#pragma unroll
    for (int k = 0; k < KB; ++k) {  // ids past xmax load block 0, unused
        const int b = tid + k * FT;
        const int bb = b < xmax ? b : 0;
        if constexpr (kLogits) {
            const float* zu = a.zlog + (size_t)u * G * a.zstride + bb;
#pragma unroll
            for (int g = 0; g < G; ++g) w[k][g] = zu[(size_t)g * a.zstride];
            dvk[k] = *reinterpret_cast<const float4*>(a.dvar + ((size_t)u * geo.xcap + bb) * 4);
        } else {
            load_terms<G, kCoh>(wu, bb, w[k]);
        }
    }
    // the length is read only now (a value made uniform early would wait for every load above)
    __asm__ volatile("" : "+v"(n_raw));
    const int n = clamp_len(n_raw, geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    if (one_pass && tid < np * G) {
        fac[tid] = pv.x;
        sums[tid] = pv.y;
    }
    if (kLogits && tid < G * 4) sh.qv[tid] = qv;
    if (!one_pass) {
        for (int idx = tid; idx < np * G; idx += FT) {
            const float* pp = a.ws_part + ((size_t)u * np * G + idx) * 2;
            const float2 t = kCoh ? ld_agent2(pp) : *reinterpret_cast<const float2*>(pp);
            fac[idx] = t.x;
            sums[idx] = t.y;
        }
    }
    select_init(sh);
    __syncthreads();
    COMPKV_MARK(a.trace, 2);  // the selection's loads are in
    // ---- wave g: head g's log normalizer over every block, then each partial's factor exp(m_c - lse)
    if (wave < G) {
        const int g = wave;
        float m = -INFINITY;
        for (int c = lane; c < np; c += 64) m = fmaxf(m, fac[c * G + g]);
        m = wave_max(m);
        float l = 0.0f;
        for (int c = lane; c < np; c += 64) {
            const float pm = fac[c * G + g];
            if (pm != -INFINITY) l += sums[c * G + g] * expf(pm - m);
        }
        l = wave_sum(l);  // (every lane's reads above are complete)
        const float lse = m + logf(l);
        if (kLogits && lane == 0) sh.lse[g] = lse;
        for (int c = lane; c < np; c += 64) {
            const float pm = fac[c * G + g];
            fac[c * G + g] = pm == -INFINITY ? 0.0f : expf(pm - lse);
        }
    }
    __syncthreads();

    const SelectCtx sc = make_select_ctx(X, a.K, a.n_sink, a.n_recent, sel_out, nsel_out,
                                         a.keys_in_lds ? reinterpret_cast<uint32_t*>(dyn + 2 * np * G)
                                                       : a.ws_key + (size_t)u * xmax);
    const int bpc_log2 = __builtin_ctz((unsigned)a.bpc);  // the chunk size is a power of two (32, 64, 128)
    auto score_of = [&](int b, const float (&wt)[G]) {
        const float* f = fac + (b == X - 1 ? nc : b >> bpc_log2) * G;
        float S = 0.0f;
#pragma unroll
        for (int g = 0; g < G; ++g) S += f[g] * wt[g];
        return S;
    };

    // ---- fast path. Block b's key is (bits of S_b) << 32 | ~b: unique, and ordered exactly like
    // (S_b descending, b ascending). Thread t keeps the keys of blocks t + 1024k in registers.
    if (fast) {
        unsigned long long ck[KPT];
        uint32_t mx = 0u;
        const float half = kind_half(a.score_kind);
        const float logB = logf((float)geo.B), lnlast = logf((float)max(1, n - (X - 1) * geo.B));
        auto key = [&](int k, const float (&wt)[G]) {
            const int b = tid + k * FT;
            ck[k] = 0ull;
            if (b < X) {
                float S;
                if constexpr (kLogits) {  // wt: zbar of each head
                    const float4 dv = dvk[k];
                    const float lnb = b == X - 1 ? lnlast : logB;
                    S = 0.0f;
#pragma unroll
                    for (int g = 0; g < G; ++g) {
                        const float v = sh.qv[4 * g] * dv.x + sh.qv[4 * g + 1] * dv.y + sh.qv[4 * g + 2] * dv.z +
                                        sh.qv[4 * g + 3] * dv.w;
                        S += __expf(lnb + wt[g] + half * v - sh.lse[g]) * kind_term(a.score_kind, v);
                    }
                } else {
                    S = score_of(b, wt);
                }
                if (write_scores && a.scores) a.scores[(size_t)u * geo.xcap + b] = S;
                if (!mandatory(b, X, a.n_sink, a.n_recent)) {
                    ck[k] = ((unsigned long long)__float_as_uint(S) << 32) | (0xFFFFFFFFu - (uint32_t)b);
                    mx = max(mx, __float_as_uint(S));
                }
            }
        };
#pragma unroll
        for (int k = 0; k < KB; ++k) key(k, w[k]);
        if constexpr (KPT > KB) {
            float w2[KPT - KB][G];
#pragma unroll
            for (int k = KB; k < KPT; ++k) {
                if (k * FT >= xmax) {  // (workgroup-uniform)
#pragma unroll
                    for (int g = 0; g < G; ++g) w2[k - KB][g] = 0.0f;
                } else {
                    const int b = tid + k * FT;
                    load_terms<G, kCoh>(wu, b < xmax ? b : 0, w2[k - KB]);
                }
            }
#pragma unroll
            for (int k = KB; k < KPT; ++k) key(k, w2[k - KB]);
        }
        COMPKV_MARK(a.trace, 3);  // normalizers and keys formed
        if (select_fast<KPT, FT>(sc, ck, mx, sh)) return;
    } else {
        // ---- general path (more than 8192 blocks): scores and their bits into the key array
        for (int b = tid; b < X; b += FT) {
            float wt[G];
            load_terms<G, kCoh>(wu, b, wt);
            const float S = score_of(b, wt);
            if (write_scores && a.scores) a.scores[(size_t)u * geo.xcap + b] = S;
            sc.keys[b] = __float_as_uint(S);
        }
    }
    __syncthreads();
    select_radix<FT>(sc, sh);
}

constexpr int kSxWaves = kFinThreads / 64;
constexpr int kSelLdsMax = 1024;  // budget limit of the fused kernel (ids held in LDS)
constexpr int kStepCbMax = 1024;  // blocks per compensation workgroup of the fused launch

// LDS of a workgroup of NW waves that selects, attends exactly, streams mean values (at most CB blocks)
// or merges.
template <int D, int G, int CB, int NW = kSxWaves>
struct SelExactLdsT {
    union {
        FinalShared fin;
        ExactLds<D, G, NW> ex;  // (compensation workgroups: their wave sums in ex.acc)
    } u;
    int32_t sel[kSelLdsMax];
    int32_t rowbase[kMaxEb];  // cache row of token 0 of each of the item's blocks
    int32_t nsel;
    float cw[G][CB];          // compensation workgroups: pseudo-logits, then their weights
    float cm[G], cl[G];
    int32_t last;             // this workgroup arrived last for its unit (it merges the partials)
};
template <int D, int G>
using SelExactLds = SelExactLdsT<D, G, kStepCbMax>;

// Partials per unit that the in-launch merge handles (their maxima and factors live in the selection's
// LDS area).
constexpr int kMergeMaxTerms = (int)(sizeof(FinalShared) / (2 * sizeof(float)));

// After a workgroup has stored what another workgroup of the same launch reads (device-coherent
// stores): count its arrival on `counter`; true (workgroup-uniform) for the last of `arrivals`.
// `last` is an LDS word.
__device__ inline bool arrive_last(uint32_t* counter, int arrivals, int32_t& last) {
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's stores are complete
    __syncthreads();
    if (threadIdx.x == 0)
        last = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               (uint32_t)(arrivals - 1);
    __syncthreads();
    return last != 0;
}

// The merge of unit u's d.part_count partials (the result does not depend on which workgroup runs it):
// per head the maximum M, the sum L of exp(m_p - M) l_p and of exp(m_p - M) acc_p, then out = acc / L
// and lse = M + log L (NaN when `poison`). SPLIT = FT / (G d) threads share a coordinate: thread h of
// a coordinate adds partials h, h + SPLIT, ... in that order (RB of them requested per round, the first
// round with the maxima and sums), then the SPLIT sums are added in h order (in the compensation
// weights' LDS, free by then), so a unit of up to SPLIT RB partials costs one memory round trip.
template <int D, int G, typename Lds, int FT = kFinThreads>
__device__ void merge_unit(const Geom& geo, const DecodeArgs& d, int u, Lds& L, bool poison = false) {
    constexpr int GD = G * D;
    constexpr int SPLIT = GD >= FT ? 1 : FT / GD;
    static_assert(SPLIT == 1 || SPLIT * GD <= (int)(sizeof(L.cw) / sizeof(float)), "split sums fit in LDS");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int np = d.part_count;
    constexpr int RB = 16;  // partial values requested per round and thread
    const float* pu = d.ws_part + (size_t)u * np * G * (D + 2);
    float* pm = reinterpret_cast<float*>(&L.u.fin);  // [np][G] maxima, then factors
    float* pl = pm + np * G;                         // [np][G] sums
    float* part_sum = &L.cw[0][0];                   // [SPLIT][G d]
    const int h = SPLIT > 1 ? tid / GD : 0;          // this thread's share of a coordinate's partials
    const int idx0 = SPLIT > 1 ? tid - h * GD : tid;
    // the first round of this thread's first coordinate, requested with the maxima and sums
    float x[RB];
    {
        const int g = idx0 / D, i = idx0 - g * D;
        const float* pi = pu + (size_t)g * (D + 2) + 2 + i;
#pragma unroll
        for (int k = 0; k < RB; ++k) {
            const int p = h + SPLIT * k;
            x[k] = (idx0 < GD && p < np) ? ld_agent(pi + (size_t)p * G * (D + 2)) : 0.0f;
        }
    }
    for (int t = tid; t < np * G; t += FT) {
        const float* q = pu + (size_t)t * (D + 2);
        pm[t] = ld_agent(q);
        pl[t] = ld_agent(q + 1);
    }
    __syncthreads();
    if (wave < G) {
        float M = -INFINITY;
        for (int p = lane; p < np; p += 64) M = fmaxf(M, pm[p * G + wave]);
        M = wave_max(M);
        float S = 0.0f;
        for (int p = lane; p < np; p += 64) {
            const float mp = pm[p * G + wave];
            const float f = mp == -INFINITY ? 0.0f : __expf(mp - M);
            S += f * pl[p * G + wave];
            pm[p * G + wave] = f;
        }
        S = wave_sum(S);
        if (lane == 0) {
            L.cm[wave] = M;
            L.cl[wave] = S;
        }
    }
    __syncthreads();
    const int bseq = u / geo.hkv, hk = u - bseq * geo.hkv;
    auto emit = [&](int idx, float A) {  // coordinate idx of the unit's output
        const int g = idx / D, i = idx - g * D;
        const size_t o = (size_t)bseq * geo.hq + (size_t)hk * G + g;
        const float S = L.cl[g];
        d.out[o * D + i] = poison ? __int_as_float(0x7FC00000) : (S > 0.0f ? A / S : 0.0f);
        if (i == 0 && d.lse) d.lse[o] = poison ? __int_as_float(0x7FC00000) : (S > 0.0f ? L.cm[g] + logf(S) : -INFINITY);
    };
    // coordinate idx of head g: this thread's partials in order, RB requested at a time
    for (int idx = idx0; idx < GD; idx += SPLIT > 1 ? GD : FT) {
        const int g = idx / D, i = idx - g * D;
        const float* pi = pu + (size_t)g * (D + 2) + 2 + i;
        float A = 0.0f;
        for (int p0 = 0; p0 < np; p0 += SPLIT * RB) {
            if (p0 > 0 || idx != idx0) {
#pragma unroll
                for (int k = 0; k < RB; ++k) {
                    const int p = p0 + h + SPLIT * k;
                    x[k] = p < np ? ld_agent(pi + (size_t)p * G * (D + 2)) : 0.0f;
                }
            }
#pragma unroll
            for (int k = 0; k < RB; ++k) {
                const int p = p0 + h + SPLIT * k;
                if (p < np) A += pm[p * G + g] * x[k];
            }
        }
        if constexpr (SPLIT > 1)
            part_sum[h * GD + idx] = A;
        else
            emit(idx, A);
    }
    if constexpr (SPLIT > 1) {
        __syncthreads();
        for (int idx = tid; idx < GD; idx += FT) {
            float A = 0.0f;
#pragma unroll
            for (int s = 0; s < SPLIT; ++s) A += part_sum[s * GD + idx];
            emit(idx, A);
        }
    }
}

// The fused selection/exact launch: count the arrival; the unit's last workgroup merges.
template <int D, int G, typename Lds, int FT = kFinThreads>
__device__ void arrive_and_merge(const Geom& geo, const DecodeArgs& d, int u, Lds& L) {
    if (arrive_last(d.arrive + u, d.part_count, L.last)) {
        COMPKV_MARK(d.trace, 10);  // this workgroup merges
        merge_unit<D, G, Lds, FT>(geo, d, u, L);
    }
}

// The mean-value stream of one compensation range of unit u: blocks [c0, c1) (at most kStepCbMax, within
// the unit's xmax; blocks past the sequence's last contribute nothing), each a pseudo-token with logit
// log|b| + zbar_b (the block logits the chunk launch wrote) and value vmean_b, reduced to one softmax
// partial per head. In steps, so that a caller can place the requests:
//   request_logits()  the block logits of the range (ZR per thread and head);
//   request_rows()    the first two batches of mean-value rows (NT / (D / 4) * ROWS rows each, two
//                     register buffers of ROWS rows per thread);
//   weigh(...)        the pseudo-logits and their per-head weights (in LDS), then every batch, each
//                     requested two batches ahead of its use so that one batch is in flight while
//                     another is weighed; the per-wave sums are left in L.u.ex.acc;
//   store(...) / keep(...)  the partial to memory (device-coherent) / to LDS (L.cm, L.cl, L.cw[g][0, D)).
// Every batch is requested, also past the range (then the range's first row again, weighted by zero):
// the number of loads in flight stays fixed, so each wait is for one batch, never for all of them.
struct NoPoll {
    __device__ void operator()() const {}
};

// One compensation workgroup of a fused launch: blocks [c0, c1) (at most kStepCbMax, within the unit's
// xmax; the blocks past the sequence's last contribute nothing) of unit u, whose sequence length n_raw
// was requested before the call and is read only once the loads below are requested (a value made
// uniform right away would wait for its load). The block logits zbar are requested first (loads return
// in order, so they arrive ahead of the mean values); then the mean-value rows in batches of
// NT / (D / 4) * ROWS rows, each batch
// requested two batches ahead of its use (two register buffers of ROWS rows per thread), so that a
// batch is in flight while another is weighed. While the first two batches are in flight: the pseudo-
// logits log|b| + zbar and their per-head softmax weights (in LDS). `after` runs once the last mean
// values have arrived, before the partial is reduced (loads it issues are not queued behind mean values);
// `poll` runs once, right after the last batch is requested (a load whose value the caller uses after the
// call: it returns with the last mean values instead of a round trip after them). The partial is stored
// to `part` (device-coherent), or with kKeep left in LDS for the workgroup's exact partial to absorb:
// per head its max in L.cm, its sum in L.cl and its weighted sums in L.cw[g][0, D) (the weights are
// no longer needed by then).
template <int D, int G, int ROWS, typename Lds, int NT = kFinThreads, bool kKeep = false, typename After,
          typename Poll = NoPoll>
__device__ void step_compensation(const Geom& geo, const DecodeArgs& d, int u, int n_raw, int c0, int c1, Lds& L,
                                  float* part, After&& after, Poll&& poll = Poll()) {
    constexpr int LPB = D / 4;     // lanes per mean-value row (one float4 each)
    constexpr int RPS = NT / LPB;  // rows per workgroup step
    constexpr int BATCH = RPS * ROWS;
    constexpr int ZR = (kStepCbMax + NT - 1) / NT;  // block logits per thread and head
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nb = max(0, min(c1 - c0, kStepCbMax));
    const int li = tid % LPB, slot = tid / LPB;
    const float* lg = d.blk_logit + (size_t)u * G * geo.xcap + c0;
    float zl[G][ZR];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int k = 0; k < ZR; ++k) {
            const int lb = tid + k * NT;
            zl[g][k] = lb < nb ? lg[(size_t)g * geo.xcap + lb] : 0.0f;
        }
    // (an empty range reads row 0 of the unit, unused)
    const float4* vm = reinterpret_cast<const float4*>(d.vmean + ((size_t)u * geo.xcap + (nb > 0 ? c0 : 0)) * D) + li;
    float4 va[ROWS], vb[ROWS];
    // branch-free within a batch: a row past the range reloads the range's first row, weighted by zero
    auto issue = [&](int base, float4 (&v)[ROWS]) {
#pragma unroll
        for (int k = 0; k < ROWS; ++k) {
            const int lb = base + slot + k * RPS;
            v[k] = vm[(size_t)(lb < nb ? lb : 0) * (D / 4)];
        }
    };
    // every wave's block logits are requested before any wave's mean values (a barrier that waits for
    // no load): the returns of a CU come back in request order, so the logits then arrive first
    __builtin_amdgcn_s_barrier();
    // every batch is requested, also past the range (then row 0 again): the number of loads in flight
    // stays fixed, so each wait below is for one batch, never for all of them
    issue(0, va);
    issue(BATCH, vb);
    __asm__ volatile("" : "+v"(n_raw));
    const int n = clamp_len(n_raw, geo.max_seq);
    const int nv = max(0, min(nb, (n + geo.B - 1) / geo.B - c0));  // blocks of the range in the sequence
    // pseudo-logits log|b| + zbar, then per head (wave g) their max and the weights exp(. - max)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int k = 0; k < ZR; ++k) {
            const int lb = tid + k * NT, b = c0 + lb;
            if (lb < nv) L.cw[g][lb] = logf((float)min(geo.B, n - b * geo.B)) + zl[g][k];
        }
    __syncthreads();
    if (wave < G) {
        const int g = wave;
        float mx = -INFINITY;
        for (int lb = lane; lb < nv; lb += 64) mx = fmaxf(mx, L.cw[g][lb]);
        mx = wave_max(mx);
        float sum = 0.0f;
        for (int lb = lane; lb < nv; lb += 64) {
            const float wv = __expf(L.cw[g][lb] - mx);
            L.cw[g][lb] = wv;
            sum += wv;
        }
        sum = wave_sum(sum);
        if (lane == 0) {
            L.cm[g] = mx;
            L.cl[g] = sum;
        }
    }
    __syncthreads();
    COMPKV_MARK(d.trace, 5);  // weights formed
    // weighted mean values; lane li of a row slot holds coordinates 4 li .. 4 li + 3
    float acc[G][4];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g][0] = acc[g][1] = acc[g][2] = acc[g][3] = 0.0f;
    auto weigh = [&](int base, const float4 (&v)[ROWS]) {
#pragma unroll
        for (int k = 0; k < ROWS; ++k) {
            const int lb = base + slot + k * RPS;
            if (lb < nv) {
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const float wv = L.cw[g][lb];
                    acc[g][0] += wv * v[k].x;
                    acc[g][1] += wv * v[k].y;
                    acc[g][2] += wv * v[k].z;
                    acc[g][3] += wv * v[k].w;
                }
            }
        }
    };
    int base = 0;
    for (; base + 2 * BATCH < nv; base += 2 * BATCH) {  // workgroup-uniform
        weigh(base, va);
        issue(base + 2 * BATCH, va);
        weigh(base + BATCH, vb);
        issue(base + 3 * BATCH, vb);
    }
    poll();  // (after the last requests)
    weigh(base, va);
    weigh(base + BATCH, vb);
    COMPKV_MARK(d.trace, 6);  // the last mean values weighed
    after();
    // the row slots of a wave (lanes li, li + LPB, ...), then the waves in order
#pragma unroll
    for (int off = LPB; off < 64; off <<= 1)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[g][e] = xor_add(acc[g][e], off);
    if (lane < LPB) {
#pragma unroll
        for (int g = 0; g < G; ++g)
            *reinterpret_cast<float4*>(&L.u.ex.acc[wave][g][4 * li]) = make_float4(acc[g][0], acc[g][1], acc[g][2], acc[g][3]);
    }
    __syncthreads();
    if constexpr (kKeep) {
        static_assert(D <= (int)(sizeof(L.cw[0]) / sizeof(float)), "the sums fit the weights' rows");
        constexpr int PT = (G * D + NT - 1) / NT;
        float tot[PT];
#pragma unroll
        for (int k = 0; k < PT; ++k) {
            const int idx = tid + k * NT;
            tot[k] = 0.0f;
            if (idx < G * D) {
                const int g = idx / D, i = idx - g * D;
#pragma unroll
                for (int w = 0; w < NT / 64; ++w) tot[k] += L.u.ex.acc[w][g][i];
            }
        }
        __syncthreads();  // (every wave sum read: the exact path reuses L.u.ex)
#pragma unroll
        for (int k = 0; k < PT; ++k) {
            const int idx = tid + k * NT;
            if (idx < G * D) L.cw[idx / D][idx % D] = tot[k];
        }
    } else {
        for (int idx = tid; idx < G * D; idx += NT) {
            const int g = idx / D, i = idx - g * D;
            float* p = part + (size_t)g * (D + 2);
            if (i == 0) {
                st_agent(p, L.cm[g]);
                st_agent(p + 1, L.cl[g]);
            }
            float tot = 0.0f;
#pragma unroll
            for (int w = 0; w < NT / 64; ++w) tot += L.u.ex.acc[w][g][i];
            st_agent(p + 2 + i, tot);
        }
    }
}

size_t finalize_dyn_lds(const Geom& g, const ScoreArgs& a) {
    return ((size_t)2 * (a.nchunks + 1) * g.G + (a.keys_in_lds ? (size_t)g.xmax() : 0)) * sizeof(float);
}

}  // namespace
}  // namespace compkv

// step.hip -- the decode step (Section 4.2, Appendix E.1) in two launches: append and refresh, block
// scores, selection, the mean-value compensation stream, exact attention over the selected blocks and
// the merge of the partials.
//
// Launch 1 (step_score_kernel): first the last block X - 1 of each unit: the new token's cache row is
// stored and the block's summary recomputed (the append's routine, bit-identical), the block is scored
// and its compensation partial written. Then the scores of every completed block, blocks [0, X - 1),
// whose summaries the step does not change. Persistent 512-thread workgroups take groups of 128
// consecutive blocks of one unit (one to four scoring chunks of the chunked path) grid-stride, and
// request the next group's query, mean keys and first variance groups before computing the current
// one, so each compute unit streams its share in order with about two groups in flight. Per block and
// query head it forms the block-mean logit zbar = s q.kmean, the projected variance
// sig2 = s^2 sum_t Q_t dvar_t and the log weight a = log|b| + zbar + sig2 / 2 (Eqs.
// grouped-variance-metadata, compkv-mass-estimate); per chunk and head the (max, sum of exp(a - max))
// partial and per block the score terms exp(a - max) sig2 (Eq. compkv-score) -- the arithmetic of the
// chunked path, so the scores and selections are bit-identical to compkv_score_select's.
//
// Launch 2 (step_stream_kernel), one-dimensional grid of 1024-thread workgroups in three segments:
//  1. one selector per unit: forms the per-head normalizers and the scores, ranks the blocks (the stable
//     Top-K with the mandatory set, Eq. compkv-selected-set) and publishes the ids;
//  2. compensation, n_comp per unit: stream the mean values of cb blocks short of the last and reduce
//     their pseudo-tokens (logit log|b| + zbar, value vmean) to one softmax partial per head, with the
//     next rows requested before the current ones are weighted. Every such block is counted here
//     (selected ones included); the exact workgroups take the selected blocks' pseudo-tokens back out
//     (Eq. compkv-output regrouped);
//  3. exact, n_exact per unit: once the unit's ids are published, exact attention on the matrix cores
//     over eb selected blocks (exact.h), one partial.
// The selectors and the compensation fill the first round of workgroups, so the mean values stream
// while the selections run; the exact workgroups take the compute units they free. The last
// compensation or exact workgroup of a unit to arrive merges the unit's partials in index order and
// returns the unit's words to zero.
//
// Handoffs inside launch 2 use device-coherent stores and loads (relaxed atomics at agent scope: they
// bypass the per-XCD caches), each thread's stores completed before its workgroup's arrival is
// counted or the ids are published. The only wait (an exact workgroup for its unit's ids) is on a
// selector, which has a lower id and never waits, so under the in-order dispatch of workgroups every
// wait ends; it is also bounded: on a timeout the unit is marked, its outputs become NaN and the
// unit's timeout word counts it, so the launch always drains.
#include "select_core.h"

namespace compkv {
namespace {

constexpr int kStepGroup = 128;    // blocks per scoring group (eight lanes per block, 1024 threads)
constexpr uint32_t kSelected = 2u, kFailed = 4u;
constexpr int kSpinLimit = 1 << 17;  // polls of a wait (each a memory round trip): well over 50 ms

template <int D, int G>
struct StepScoreLds {
    float q[G][D];   // scaled query of the group's unit
    float Qv[G][D];  // s^2 * sum of q^2 over each group (first r entries)
    float z[G][kStepGroup];
    float v[G][kStepGroup];
    float m[kStepGroup / 32][G];  // per chunk of the group
};

template <int D, int G>
struct StepTailLds {
    BlockStatsLds<D> bs;  // the last block's summary
    float q[G][D];
    float Qv[G][D];
    float z[G], v[G];
};

template <int D, int G>
struct StepLds {
    union {
        SelExactLdsT<D, G, kStepCbMax> sx;
    } u;
    int32_t last;
};

// Wait (thread 0 polls, the workgroup then meets at a barrier) until the unit's phase word has `bit`.
// On a timeout the unit is marked failed and its timeout word counts it.
__device__ void wait_phase(uint32_t* st, uint32_t bit) {
    if (threadIdx.x == 0) {
        uint32_t v = ld_agent_u32(st + 2);
        for (int spins = 0; !(v & bit) && spins < kSpinLimit; ++spins) {
            __builtin_amdgcn_s_sleep(2);
            v = ld_agent_u32(st + 2);
        }
        if (!(v & bit)) {
            __hip_atomic_fetch_or(st + 2, kFailed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_fetch_add(st + 3, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __syncthreads();
}

// ---------------------------------------------------------------- launch 1: scoring

constexpr int kScoreThreads = 512;  // eight waves; two block slots of eight lanes per thread
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kLenCache = 64;       // sequence lengths of a workgroup's next groups, held in LDS

// One thread's share of a group's loads: its unit's query pairs (waves 0-3), the mean keys of block
// slots tid / 8 and tid / 8 + 64 and their first variance groups (a block id past the allocated range
// loads block 0; unused).
template <int D, int G>
struct GroupLoads {
    QueryPairs<D, G> qp;
    float4 kv[2][D / 32];
    float dv0[2];
};

template <int D, int G>
__device__ __forceinline__ void issue_group(const Geom& geo, const ScoreArgs& a, int gpu, int gi,
                                            GroupLoads<D, G>& L) {
    const int tid = threadIdx.x, wave = tid >> 6, li = tid & 7;
    const int u = gi / gpu, grp0 = (gi - u * gpu) * kStepGroup;
    const int bseq = u / geo.hkv, h = u - bseq * geo.hkv;
    if (wave < 4) load_query_pairs<D, G>(a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D, geo.layout, L.qp);
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const int b = grp0 + 64 * p + (tid >> 3);
        const size_t blk = (size_t)u * geo.xcap + (b < geo.xmax() ? b : 0);
        const float4* kp = reinterpret_cast<const float4*>(a.kmean + blk * D);
#pragma unroll
        for (int m = 0; m < D / 32; ++m) L.kv[p][m] = kp[li + 8 * m];
        L.dv0[p] = a.dvar[blk * geo.r + min(li, geo.r - 1)];
    }
}

// Group gi: blocks [(gi % gpu) 128, + 128) of unit gi / gpu with n tokens, short of the unit's last
// block.
template <int D, int G>
__device__ void score_group(const Geom& geo, const ScoreArgs& a, int gpu, int gi, int n_raw,
                            const GroupLoads<D, G>& L, StepScoreLds<D, G>& sh) {
    constexpr int NF4 = D / 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = tid & 7;
    const int u = gi / gpu, grp0 = (gi - u * gpu) * kStepGroup;
    const int bpc = a.bpc, cpg = kStepGroup / bpc;  // chunks per group
    const int n = clamp_len(n_raw, geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    const int xs = X - 1;  // the last block is scored by the unit's tail task
    __syncthreads();  // the previous group's reads of the LDS rows are done
    if (wave < 4) store_query<D, G>(L.qp, a.scale, geo.r, geo.layout, sh.q, sh.Qv);
    __syncthreads();
    // per slot: projected variances, then the block-mean logits one head at a time
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const int lb = 64 * p + (tid >> 3);
        const int b = grp0 + lb;
        float v[G];
#pragma unroll
        for (int g = 0; g < G; ++g) v[g] = (li < geo.r ? sh.Qv[g][li] : 0.0f) * L.dv0[p];
        if (geo.r > 8 && b < xs) {
            const size_t blk = (size_t)u * geo.xcap + b;
            for (int t = li + 8; t < geo.r; t += 8) {
                const float dv = a.dvar[blk * geo.r + t];
#pragma unroll
                for (int g = 0; g < G; ++g) v[g] += sh.Qv[g][t] * dv;
            }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
            v[g] = sum8_lead(v[g]);
            if (li == 0) sh.v[g][lb] = v[g];
        }
#pragma unroll 1
        for (int g = 0; g < G; ++g) {  // one head's query slice in registers at a time
            float4 qq[NF4];
#pragma unroll
            for (int m = 0; m < NF4; ++m) qq[m] = *reinterpret_cast<const float4*>(&sh.q[g][4 * (li + 8 * m)]);
            float z = 0.0f;
#pragma unroll
            for (int m = 0; m < NF4; ++m)
                z += qq[m].x * L.kv[p][m].x + qq[m].y * L.kv[p][m].y + qq[m].z * L.kv[p][m].z +
                     qq[m].w * L.kv[p][m].w;
            z = sum8_lead(z);
            if (li == 0) sh.z[g][lb] = z;
        }
    }
    __syncthreads();
    const float half = kind_half(a.score_kind);
    auto logw = [&](int g, int j) {  // j: block slot of the group
        return logf((float)min(geo.B, n - (grp0 + j) * geo.B)) + sh.z[g][j] + half * sh.v[g][j];
    };
    // per chunk q and head g (one wave each): the chunk's max of a and sum of exp(a - max), with the
    // chunk's blocks on the lanes as in the chunked path (block j of the chunk on lane j % 64)
    const int c_first = grp0 / bpc;
    for (int qg = wave; qg < cpg * G; qg += kScoreWaves) {
        const int q = qg / G, g = qg - q * G;
        const int c = c_first + q;
        const int nvalid = max(0, min(bpc, xs - c * bpc));
        float av[2];
        float m = -INFINITY;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int j = lane + 64 * k;
            av[k] = (j < bpc && j < nvalid) ? logw(g, q * bpc + j) : -INFINITY;
            m = fmaxf(m, av[k]);
        }
        m = wave_max(m);
        float ssum = 0.0f;
        if (m != -INFINITY) {
#pragma unroll
            for (int k = 0; k < 2; ++k) ssum += (av[k] == -INFINITY) ? 0.0f : expf(av[k] - m);
        }
        ssum = wave_sum(ssum);
        if (lane == 0) {
            sh.m[q][g] = m;
            if (c < a.nchunks) {
                float* pp = a.ws_part + (((size_t)u * (a.nchunks + 1) + c) * G + g) * 2;
                pp[0] = m;
                pp[1] = ssum;
            }
        }
    }
    __syncthreads();
    // block logits [g][b] and score terms [b][g]
    const int nval = max(0, min(kStepGroup, xs - grp0));
    for (int idx = tid; idx < G * nval; idx += kScoreThreads) {
        const int g = idx / nval, j = idx - g * nval;
        a.blk_logit[((size_t)u * G + g) * geo.xcap + grp0 + j] = sh.z[g][j];
    }
    for (int idx = tid; !a.logit_terms && idx < G * nval; idx += kScoreThreads) {
        const int j = idx / G, g = idx - j * G;
        a.ws_w[((size_t)u * geo.xmax() + grp0 + j) * G + g] =
            expf(logw(g, j) - sh.m[j / bpc][g]) * kind_term(a.score_kind, sh.v[g][j]);
    }
}

// The last block X - 1 of unit u: refreshed first when the step appends (the new row is read from
// k_new / v_new, the cache row stored at the end), then scored as a chunk of one block (partial
// a.nchunks), with its own compensation partial (decode partial 0) under Mean.
template <int D, int G, int NT>
__device__ void step_score_tail(const Geom& geo, const ScoreArgs& a, const DecodeArgs& d, int u,
                                StepTailLds<D, G>& ts) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int nc = a.nchunks;
    const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    QueryPairs<D, G> qp;
    if (wave < 4) load_query_pairs<D, G>(qh, geo.layout, qp);
    const int n_raw = a.seq_lens[bseq];
    const int n = clamp_len(n_raw, geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    float* pp = a.ws_part + ((size_t)u * (nc + 1) + nc) * G * 2;
    float* cp = d.neg_pseudo ? d.ws_part + (size_t)u * d.part_count * G * (D + 2) : nullptr;
    if (X == 0) {  // empty sequence: neutral partials
        for (int g = tid; g < G; g += NT) {
            st_agent(pp + 2 * g, -INFINITY);
            st_agent(pp + 2 * g + 1, 0.0f);
        }
        if (cp)
            for (int idx = tid; idx < G * (D + 2); idx += NT)
                st_agent(cp + idx, (idx % (D + 2) == 0) ? -INFINITY : 0.0f);
        return;
    }
    const int b = X - 1, nb = n - b * geo.B;
    const size_t blk = (size_t)u * geo.xcap + b;
    // a length beyond max_seq_len appends nothing (as in the other paths)
    const bool append = a.k_new && n_raw <= geo.max_seq;
    if (append) {
        const size_t row0 = (size_t)block_row0(geo, u, b);
        const BlockSrc src{a.Kc + row0 * D, a.Vc + row0 * D, a.k_new + (size_t)u * D, a.v_new + (size_t)u * D, nb,
                           nb - 1};
        BlockRows rows;
        if (wave < 4) {
            load_block_rows<D>(src, 0, rows);
            store_query<D, G>(qp, a.scale, geo.r, geo.layout, ts.q, ts.Qv);  // while the rows are in flight
        }
        block_stats_from<D>(src, rows, geo.r, geo.layout, a.kmean_w + blk * D, a.dvar_w + blk * geo.r,
                            a.vmean + blk * D, ts.bs, wave < 4);  // (its barriers also publish ts.q / ts.Qv)
    } else {
        for (int i = tid; i < D; i += NT) {
            ts.bs.km[i] = a.kmean[blk * D + i];
            ts.bs.vm[i] = a.vmean[blk * D + i];
        }
        for (int t = tid; t < geo.r; t += NT) ts.bs.dv[t] = a.dvar[blk * geo.r + t];
        if (wave < 4) store_query<D, G>(qp, a.scale, geo.r, geo.layout, ts.q, ts.Qv);
        __syncthreads();
    }
    for (int g = wave; g < G; g += NT / 64) {
        float z = 0.0f, v = 0.0f;
        for (int i = lane; i < D; i += 64) z += ts.q[g][i] * ts.bs.km[i];
        for (int t = lane; t < geo.r; t += 64) v += ts.Qv[g][t] * ts.bs.dv[t];
        z = wave_sum(z);
        v = wave_sum(v);
        if (lane == 0) {
            ts.z[g] = z;
            ts.v[g] = v;
        }
    }
    __syncthreads();
    const float lnb = logf((float)nb);
    for (int g = tid; g < G; g += NT) {
        const float z = ts.z[g], v = ts.v[g];
        st_agent(a.blk_logit + ((size_t)u * G + g) * geo.xcap + b, z);
        st_agent(pp + 2 * g, lnb + z + kind_half(a.score_kind) * v);  // one block: max a, sum 1
        st_agent(pp + 2 * g + 1, 1.0f);
        if (!a.logit_terms) st_agent(a.ws_w + ((size_t)u * geo.xmax() + b) * G + g, kind_term(a.score_kind, v));
    }
    if (a.logit_terms)  // the query's group sums for the selection (r = 4)
        for (int idx = tid; idx < G * 4; idx += NT) a.ws_qv[(size_t)u * G * 4 + idx] = ts.Qv[idx / 4][idx % 4];
    if (cp) {
        for (int idx = tid; idx < G * D; idx += NT) {
            const int g = idx / D, i = idx - g * D;
            float* p = cp + (size_t)g * (D + 2);
            if (i == 0) {
                st_agent(p, lnb + ts.z[g]);
                st_agent(p + 1, 1.0f);
            }
            st_agent(p + 2 + i, ts.bs.vm[i]);
        }
    }
    if (append && wave == 0) {  // the new token's cache row (read by the unit's exact workgroups)
        const size_t row = (size_t)block_row0(geo, u, b) + (n - 1 - b * geo.B);
        const unsigned long long* kn = reinterpret_cast<const unsigned long long*>(a.k_new + (size_t)u * D);
        const unsigned long long* vn = reinterpret_cast<const unsigned long long*>(a.v_new + (size_t)u * D);
        for (int i = lane; i < D / 4; i += 64) {
            st_agent_u64(reinterpret_cast<unsigned long long*>(a.Kc + row * D) + i, kn[i]);
            st_agent_u64(reinterpret_cast<unsigned long long*>(a.Vc + row * D) + i, vn[i]);
        }
    }
}


// ---------------------------------------------------------------- launch 1: the kernel

template <int D, int G>
__global__ __launch_bounds__(kScoreThreads) void step_score_kernel(Geom geo, ScoreArgs a, DecodeArgs d, int gpu) {
    __shared__ union {
        StepScoreLds<D, G> sc;
        StepTailLds<D, G> tl;
    } lds;
    __shared__ int len[kLenCache];
    StepScoreLds<D, G>& sh = lds.sc;
    const int tid = threadIdx.x;
    const int total = geo.units() * gpu;
    const int stride = gridDim.x;
    // the last blocks first
    for (int u = blockIdx.x; u < geo.units(); u += stride) {
        step_score_tail<D, G, kScoreThreads>(geo, a, d, u, lds.tl);
        __syncthreads();
    }
    int gi = blockIdx.x;
    if (gi >= total) return;  // workgroup-uniform
    // the lengths of this workgroup's groups (the host sizes the grid for at most kLenCache each), so
    // that no group waits on a length load queued behind the next group's mean keys
    if (tid < kLenCache) {
        const int k = gi + tid * stride;
        len[tid] = k < total ? a.seq_lens[(k / gpu) / geo.hkv] : 0;
    }
    __syncthreads();
    // groups grid-stride, two per turn, each one's loads requested before the other is computed
    GroupLoads<D, G> A, B;
    issue_group<D, G>(geo, a, gpu, gi, A);
    for (int k = 0;; k += 2) {
        int gn = gi + stride;
        if (gn < total) issue_group<D, G>(geo, a, gpu, gn, B);
        score_group<D, G>(geo, a, gpu, gi, len[k], A, sh);
        gi = gn;
        if (gi >= total) break;
        gn = gi + stride;
        if (gn < total) issue_group<D, G>(geo, a, gpu, gn, A);
        score_group<D, G>(geo, a, gpu, gi, len[k + 1], B, sh);
        gi = gn;
        if (gi >= total) break;
    }
}

// ---------------------------------------------------------------- launch 2: selectors

// The selector of unit u: the selection of the chunked path from the partials and terms of launch 1,
// then the ids are published.
template <int D, int G>
__device__ void step_select(const Geom& geo, const ScoreArgs& a, const DecodeArgs& d, int u, uint32_t* st,
                            StepLds<D, G>& L, float* dyn) {
    const int tid = threadIdx.x;
    SelExactLdsT<D, G, kStepCbMax>& S = L.u.sx;
    bool done = false;
    if constexpr (G >= 4) {
        if (a.logit_terms) {  // (workgroup-uniform)
            finalize_select<G, false, kFinThreads, 4, true>(geo, a, u, S.u.fin, dyn, S.sel, &S.nsel, true);
            done = true;
        }
    }
    if (!done) finalize_select<G>(geo, a, u, S.u.fin, dyn, S.sel, &S.nsel, true);
    __syncthreads();
    for (int k = tid; k < a.K; k += kFinThreads) st_agent_i32(a.sel + (size_t)u * a.K + k, S.sel[k]);
    if (tid == 0) st_agent_i32(a.n_sel + u, S.nsel);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the ids are stored
    __syncthreads();
    if (tid == 0) __hip_atomic_fetch_or(st + 2, kSelected, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- launch 2: compensation

// Blocks [c0, c1) of unit u with n tokens: pseudo-logits log|b| + zbar and their per-head softmax
// weights first (in LDS), then the mean-value rows in batches of 128 (D = 128; ROWS rows per thread),
// each batch requested one batch ahead.
template <int D, int G, int ROWS>
__device__ void stream_compensation(const Geom& geo, const DecodeArgs& d, int u, int n, int c0, int c1,
                                    SelExactLdsT<D, G, kStepCbMax>& L, float* part) {
    constexpr int NT = kFinThreads;
    constexpr int LPB = D / 4;     // lanes per mean-value row (one float4 each)
    constexpr int RPS = NT / LPB;  // rows per workgroup step
    constexpr int BATCH = RPS * ROWS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nb = max(0, c1 - c0);
    const int li = tid % LPB, slot = tid / LPB;
    const float4* vm = reinterpret_cast<const float4*>(d.vmean + ((size_t)u * geo.xcap + c0) * D) + li;
    float4 va[ROWS], vb[ROWS];
    // branch-free within a batch: a row past the range reloads the range's first row, weighted by zero
    auto issue = [&](int base, float4 (&v)[ROWS]) {
#pragma unroll
        for (int k = 0; k < ROWS; ++k) {
            const int lb = base + slot + k * RPS;
            v[k] = vm[(size_t)(lb < nb ? lb : 0) * (D / 4)];
        }
    };
    issue(0, va);
    if (BATCH < nb) issue(BATCH, vb);
    const float* lg = d.blk_logit + (size_t)u * G * geo.xcap;
    for (int idx = tid; idx < G * nb; idx += NT) {
        const int g = idx / nb, lb = idx - g * nb, b = c0 + lb;
        L.cw[g][lb] = logf((float)min(geo.B, n - b * geo.B)) + lg[(size_t)g * geo.xcap + b];
    }
    __syncthreads();
    if (wave < G) {
        const int g = wave;
        float mx = -INFINITY;
        for (int lb = lane; lb < nb; lb += 64) mx = fmaxf(mx, L.cw[g][lb]);
        mx = wave_max(mx);
        float sum = 0.0f;
        for (int lb = lane; lb < nb; lb += 64) {
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
    float acc[G][4];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g][0] = acc[g][1] = acc[g][2] = acc[g][3] = 0.0f;
    auto weigh = [&](int base, const float4 (&v)[ROWS]) {
#pragma unroll
        for (int k = 0; k < ROWS; ++k) {
            const int lb = base + slot + k * RPS;
            if (lb < nb) {
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
    for (int base = 0; base < nb; base += 2 * BATCH) {  // workgroup-uniform
        weigh(base, va);
        if (base + 2 * BATCH < nb) issue(base + 2 * BATCH, va);
        if (base + BATCH < nb) {
            weigh(base + BATCH, vb);
            if (base + 3 * BATCH < nb) issue(base + 3 * BATCH, vb);
        }
    }
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
    for (int idx = tid; idx < G * D; idx += NT) {
        const int g = idx / D, i = idx - g * D;
        float* p = part + (size_t)g * (D + 2);
        if (i == 0) {
            st_agent(p, L.cm[g]);
            st_agent(p + 1, L.cl[g]);
        }
        float tot = 0.0f;
#pragma unroll
        for (int w = 0; w < kSxWaves; ++w) tot += L.u.ex.acc[w][g][i];
        st_agent(p + 2 + i, tot);
    }
}

// ---------------------------------------------------------------- launch 2: exact workgroups

// Item `item` of unit u: selected blocks [item eb, (item + 1) eb) of the published ids.
template <int D, int G>
__device__ void step_exact(const Geom& geo, const ScoreArgs& a, const DecodeArgs& d, int u, int item,
                           uint32_t* st, SelExactLdsT<D, G, kStepCbMax>& L) {
    const int tid = threadIdx.x;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int n = clamp_len(d.seq_lens[bseq], geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    const int e0 = item * d.eb;
    wait_phase(st, kSelected);
    for (int k = tid; k < d.eb; k += kFinThreads)
        L.sel[k] = e0 + k < a.K ? ld_agent_i32(a.sel + (size_t)u * a.K + e0 + k) : -1;
    if (tid == 0) L.nsel = ld_agent_i32(a.n_sel + u);
    __syncthreads();
    TokenMap tm;
    tm.dense = false;
    tm.B = geo.B;
    tm.invB = 1.0f / (float)geo.B;
    tm.n = n;
    tm.X = X;
    tm.nblk = max(0, min(d.eb, L.nsel - e0));
    tm.sel = L.sel;
    tm.t0 = tm.t1 = 0;
    tm.page = tm.pg0 = 0;
    tm.invP = 0.0f;
    tm.rowbase = L.rowbase;
    for (int k = tid; k < tm.nblk; k += kFinThreads) {
        const int b = tm.sel[k];
        L.rowbase[k] = block_row0(geo, u, b >= 0 && b < X ? b : 0);
    }
    __syncthreads();
    float m, l;
    v4f32 acc[D / 16];
    const uint16_t* qh = d.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    const bool pseudo = d.neg_pseudo != 0;  // Mean: the compensation counted every block's pseudo-token
    exact_tokens<D, G, kSxWaves>(tm, d.K, d.V, qh, pseudo ? d.blk_logit + (size_t)u * G * geo.xcap : nullptr,
                                 geo.xcap, L.u.ex.zb, d.scale, m, l, acc);
    float* part = d.ws_part + ((size_t)u * d.part_count + d.part_base + item) * G * (D + 2);
    finish_exact<D, G, kSxWaves, true>(m, l, acc, L.u.ex, part);
}


// After a compensation or exact workgroup stored its partial: the unit's last one merges (NaN outputs
// if a wait of the unit timed out) and returns the unit's words to zero.
template <int D, int G>
__device__ void step_arrive(const Geom& geo, const DecodeArgs& d, int u, uint32_t* st, StepLds<D, G>& L) {
    if (!arrive_last(st + 1, d.n_comp + d.n_exact, L.last)) return;
    const bool poison = (ld_agent_u32(st + 2) & kFailed) != 0;  // (workgroup-uniform)
    merge_unit<D, G>(geo, d, u, L.u.sx, poison);
    if (threadIdx.x == 0) {
        __hip_atomic_store(st + 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(st + 2, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <int D, int G>
__global__ __launch_bounds__(kFinThreads) void step_stream_kernel(Geom geo, ScoreArgs a, DecodeArgs d,
                                                                  uint32_t* state) {
    __shared__ StepLds<D, G> L;
    extern __shared__ float dyn[];  // the selection's partial factors and key bits
    const int units = geo.units();
    int w = blockIdx.x;
    if (w < units) {  // selector (workgroup-uniform branches throughout)
        step_select<D, G>(geo, a, d, w, state + 4 * w, L, dyn);
        return;
    }
    w -= units;
    if (w < units * d.n_comp) {  // compensation
        const int u = w / d.n_comp, j = w - u * d.n_comp;
        const int n = clamp_len(d.seq_lens[u / geo.hkv], geo.max_seq);
        const int xs = max(0, (n + geo.B - 1) / geo.B - 1);
        const int c0 = min(j * d.cb, xs), c1 = min(c0 + d.cb, xs);
        constexpr int ROWS = 128 / (kFinThreads / (D / 4));  // batches of 128 rows
        stream_compensation<D, G, ROWS>(geo, d, u, n, c0, c1, L.u.sx,
                                        d.ws_part + ((size_t)u * d.part_count + 1 + j) * G * (D + 2));
        step_arrive<D, G>(geo, d, u, state + 4 * u, L);
        return;
    }
    w -= units * d.n_comp;
    const int u = w / d.n_exact, item = w - u * d.n_exact;
    step_exact<D, G>(geo, a, d, u, item, state + 4 * u, L.u.sx);
    step_arrive<D, G>(geo, d, u, state + 4 * u, L);
}

template <int D, int G>
int score_slots() {
    return resident_slots(step_score_kernel<D, G>, kScoreThreads);
}

template <int D, int G>
hipError_t launch_stream(const Geom& g, const ScoreArgs& a, const DecodeArgs& d, uint32_t* state, hipStream_t s) {
    const int gpu = (g.xmax() + kStepGroup - 1) / kStepGroup;  // scoring groups per unit
    const long long groups = (long long)g.units() * gpu;
    // one resident round of workgroups (more only when one would hold more than kLenCache groups)
    long long grid1 = std::min<long long>(std::max<long long>(groups, g.units()), score_slots<D, G>());
    grid1 = std::max(grid1, (groups + kLenCache - 1) / kLenCache);
    step_score_kernel<D, G><<<dim3((unsigned)std::max(1LL, grid1)), kScoreThreads, 0, s>>>(g, a, d, gpu);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const long long grid2 = (long long)g.units() * (1 + d.n_comp + d.n_exact);
    step_stream_kernel<D, G><<<dim3((unsigned)grid2), kFinThreads, step_stream_dyn_lds(g, a.nchunks), s>>>(g, a, d, state);
    return hipGetLastError();
}

template <int D>
hipError_t stream_g(const Geom& g, const ScoreArgs& a, const DecodeArgs& d, uint32_t* state, hipStream_t s) {
    switch (g.G) {
        case 1: return launch_stream<D, 1>(g, a, d, state, s);
        case 2: return launch_stream<D, 2>(g, a, d, state, s);
        case 4: return launch_stream<D, 4>(g, a, d, state, s);
        case 8: return launch_stream<D, 8>(g, a, d, state, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

int step_stream_max_cb() { return kStepCbMax; }
int step_stream_max_budget() { return kSelLdsMax; }
int step_stream_merge_terms() { return kMergeMaxTerms; }
size_t step_stream_dyn_lds(const Geom& g, int nchunks) {
    return ((size_t)2 * (nchunks + 1) * g.G + (size_t)g.xmax()) * sizeof(float);
}

hipError_t launch_step_stream(const Geom& g, ScoreArgs a, const DecodeArgs& d, uint32_t* state, hipStream_t s) {
    a.keys_in_lds = 1;  // the fast path's tie fallback keeps its key bits in LDS
    const int np = d.part_count;
    if (g.xmax() > kFinThreads * kKeysPerThread || a.K > kSelLdsMax || (a.bpc != 32 && a.bpc != 64 && a.bpc != 128) ||
        (long long)a.nchunks * a.bpc < g.xmax() || d.eb < 1 || d.eb > kMaxEb || d.eb > kSelLdsMax ||
        d.n_exact < 1 || (long long)d.n_exact * d.eb < std::min(a.K, g.xmax()) ||
        (d.neg_pseudo && (d.n_comp < 1 || d.cb < 1 || d.cb > kStepCbMax || (long long)d.n_comp * d.cb < g.xmax() ||
                          d.part_base != 1 + d.n_comp)) ||
        (!d.neg_pseudo && (d.n_comp != 0 || d.part_base != 0)) || np != d.part_base + d.n_exact ||
        np * g.G > kMergeMaxTerms || step_stream_dyn_lds(g, a.nchunks) > kDynBudget || !state || !a.blk_logit ||
        !logit_terms_ok(g, a) || (a.logit_terms && a.zlog != a.blk_logit))
        return hipErrorInvalidValue;
    return g.D == 128 ? stream_g<128>(g, a, d, state, s) : stream_g<64>(g, a, d, state, s);
}

}  // namespace compkv

// select.hip -- block scoring and Top-K selection (Sections 4.1, 4.2; Appendix E.1), and the decode
// step's fused selection/exact launch.
//
// Launch 1, grid = units * (nchunks + 1), one-dimensional. Chunk workgroups stream the fp32 summaries
// (mean key, grouped variances) of `bpc` consecutive blocks of one unit. Eight lanes share a block: lane
// i of the eight reads float4 i, i+8, ... of the mean-key row (the eight lanes read 128 contiguous bytes
// per load) and the variance groups t = i, i+8, .... The sequence length and the query are requested
// first and the query is in LDS before any mean key is requested (a CU returns loads in request order,
// so a query requested after the other workgroups' mean keys would wait behind them); then two slots of
// 32 blocks are in flight, slot p + 2 requested once slot p is computed (block ids are clamped to the
// allocated range and masked afterwards). For each of the unit's G query heads a workgroup forms the
// block-mean logit zbar = s q.kmean, the projected variance sig2 = s^2 sum_t Q_t dvar_t and the log
// weight estimate a = log|b| + zbar + sig2/2 (the log of the numerator of Eq. compkv-mass-estimate). It
// writes zbar (block logits, reused by the decode), the chunk's per-head (max m_c of a, sum of
// exp(a - m_c)), and per block the G terms w_g = exp(a_g - m_c) sig2_g, stored contiguously so one
// vector load fetches a block's terms. The last block of each unit (the one a decode step appends to) is
// scored by one extra workgroup per unit, which writes its own partial; the chunks skip it. When every
// workgroup is resident at once these lead the grid (dispatched first, they are no longer the last to
// finish); otherwise they trail it, so that the chunks (the long pole) all start at once.
//
// Fused decode step (kStep): the extra workgroup first stores the new row and recomputes the last
// block's summary with the append's routine (bit-identical), so no chunk waits for it, and zeroes the
// unit's words for the fused selection/exact launch. On the chunked shape every workgroup also forms the
// compensation partial of its blocks (pseudo-logits log|b| + zbar, weights exp(. - max), weighted mean
// values); on the chunked-exact shape the fused launch streams the mean values instead.
//
// Launch 2 (chunked shape), grid = units: the kernel boundary makes every partial visible. One
// workgroup per unit merges the partials into each head's log normalizer lse_g and forms
// S_b = sum_g exp(m_c - lse_g) w_g (= Eq. compkv-score). Block b is ranked by the 64-bit key
// (bits of S_b) << 32 | ~b: scores are >= 0, so their IEEE bit patterns order like the values, and the
// keys are unique and order exactly like (S_b descending, b ascending), the stable Top-K of the paper.
// Up to 8192 blocks the keys stay in registers (eight per thread of 1024). One histogram of each key's
// distance below the largest score (bins of 1/16 octave on the float bits; keys farther than 255 bins
// are not counted) locates the bin that holds the (K-|F|)-th largest key; only the keys in that bin or
// above are ranked exactly, by brute force, and a bitmap of the selected and mandatory blocks is
// compacted into ascending ids. Larger inputs, or ties that leave too many keys at or above the cut's
// bin, go through a three-pass radix select on the score bits instead. Wave-level reductions and prefix
// sums use DPP lane moves. (select_core.h holds this selection, shared with the fused launches.)
//
// The chunked-exact shape replaces launch 2 and the decode's launches by one fused selection/exact
// launch in one of two forms (below): item workgroups that each select and attend, beside compensation
// workgroups that stream the mean values; or one selector per unit whose ids the unit's other
// workgroups take from a mailbox after streaming their share of the mean values. Either form merges the
// unit's partials in the launch (its last workgroup).
#include "select_core.h"

namespace compkv {
namespace {

// Per-block LDS rows of a chunk of 32 PMAX blocks: at least one wave's width, since the per-head passes
// give every lane of a wave a slot. Sizing them by the chunk (not the largest one) keeps the 64-block
// chunks of G = 8 at five workgroups per CU.
template <int PMAX>
constexpr int chunk_slots() {
    return 32 * PMAX < 64 ? 64 : 32 * PMAX;
}

template <int D, int G, int NB>
struct ChunkShared {
    float q[G][D];   // scaled query
    float Qv[G][D];  // s^2 * sum of q^2 over each group (first r entries)
    float z[G][NB];
    float v[G][NB];  // (a block's log weight is formed from z and v where it is needed)
    float m[G];
};

// Compensation state of the fused decode step.
template <int D, int G, int NB>
struct CompShared {
    float cw[G][NB];
    float cm[G], cl[G];
    alignas(16) float acc[4][G][D];
};
struct NoComp {};

template <int D, int G>
struct TailShared {
    BlockStatsLds<D> bs;  // the last block's summary (km, vm, dv)
    float q[G][D];
    float Qv[G][D];
    float z[G], v[G];
};

// A chunk workgroup and a last-block workgroup share one LDS allocation.
template <int D, int G, bool kStep, int NB>
union ChunkLds {
    struct {
        ChunkShared<D, G, NB> sh;
        std::conditional_t<kStep, CompShared<D, G, NB>, NoComp> st;
    } c;
    TailShared<D, G> t;
};

// The extra workgroup of unit u: the last block X - 1 (refreshed first when the step appends).
template <int D, int G, bool kStep>
__device__ void score_tail(const Geom& geo, const ScoreArgs& a, int u, TailShared<D, G>& ts) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int nc = a.nchunks;
    const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    QueryPairs<D, G> qp;
    load_query_pairs<D, G>(qh, geo.layout, qp);  // consumed only after the block's own loads are issued
    const int n_raw = a.seq_lens[bseq];
    const int n = clamp_len(n_raw, geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    float* pp = a.ws_part + ((size_t)u * (nc + 1) + nc) * G * 2;
    if (a.arrive_zero) {  // for the launch that merges after this one
        if (tid == 0) {
            a.arrive_zero[u] = 0u;
            a.arrive_zero[geo.units() + u] = 0u;
        }
        uint32_t* mbox = a.arrive_zero + 2 * (size_t)geo.units() + (size_t)u * a.K;
        for (int k = tid; k < a.K; k += kThreads) mbox[k] = 0u;
    }
    // fused step with Mean compensation: this workgroup's compensation partial
    float* cp = (kStep && a.comp_part) ? a.comp_part + ((size_t)u * a.part_count + nc) * G * (D + 2) : nullptr;
    if (X == 0) {  // empty sequence: neutral partials
        for (int g = tid; g < G; g += kThreads) {
            pp[2 * g] = -INFINITY;
            pp[2 * g + 1] = 0.0f;
        }
        if (cp)
            for (int idx = tid; idx < G * (D + 2); idx += kThreads) cp[idx] = (idx % (D + 2) == 0) ? -INFINITY : 0.0f;
        return;
    }
    const int b = X - 1, nb = n - b * geo.B;
    const size_t blk = (size_t)u * geo.xcap + b;
    // a length beyond max_seq_len appends nothing (row n - 1 would lie past the sized range): the unit
    // is scored over max_seq_len tokens from its stored summaries, as in the separate calls
    const bool append = kStep && a.k_new && n_raw <= geo.max_seq;
    if (append) {  // the summary reads row n - 1 from k_new / v_new; the cache row is stored at the end
        const size_t row0 = (size_t)block_row0(geo, u, b);
        const BlockSrc src{a.Kc + row0 * D, a.Vc + row0 * D, a.k_new + (size_t)u * D, a.v_new + (size_t)u * D, nb,
                           nb - 1};
        BlockRows rows;
        load_block_rows<D>(src, 0, rows);
        store_query<D, G>(qp, a.scale, geo.r, geo.layout, ts.q, ts.Qv);  // while the rows are in flight
        block_stats_from<D>(src, rows, geo.r, geo.layout, a.kmean_w + blk * D, a.dvar_w + blk * geo.r,
                            a.vmean + blk * D, ts.bs);  // (its barriers also publish ts.q / ts.Qv)
    } else {
        for (int i = tid; i < D; i += kThreads) {
            ts.bs.km[i] = a.kmean[blk * D + i];
            if constexpr (kStep) ts.bs.vm[i] = a.vmean[blk * D + i];
        }
        for (int t = tid; t < geo.r; t += kThreads) ts.bs.dv[t] = a.dvar[blk * geo.r + t];
        store_query<D, G>(qp, a.scale, geo.r, geo.layout, ts.q, ts.Qv);
        __syncthreads();
    }
    for (int g = wave; g < G; g += 4) {
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
    for (int g = tid; g < G; g += kThreads) {
        const float z = ts.z[g], v = ts.v[g];
        if (a.zlog) a.zlog[((size_t)u * G + g) * a.zstride + b] = z;
        pp[2 * g] = lnb + z + kind_half(a.score_kind) * v;  // the partial of one block: max a, sum exp(a - a) = 1
        pp[2 * g + 1] = 1.0f;
        if (!a.logit_terms) a.ws_w[((size_t)u * geo.xmax() + b) * G + g] = kind_term(a.score_kind, v);
    }
    if (a.logit_terms)  // the query's group sums for the selection (r = 4)
        for (int idx = tid; idx < G * 4; idx += kThreads) a.ws_qv[(size_t)u * G * 4 + idx] = ts.Qv[idx / 4][idx % 4];
    if (cp) {
        for (int idx = tid; idx < G * D; idx += kThreads) {
            const int g = idx / D, i = idx % D;
            float* p = cp + (size_t)g * (D + 2);
            if (i == 0) {
                p[0] = lnb + ts.z[g];
                p[1] = 1.0f;
            }
            p[2 + i] = ts.bs.vm[i];
        }
    }
    if (append && wave == 0) {  // the new token's cache row
        const size_t row = (size_t)block_row0(geo, u, b) + (n - 1 - b * geo.B);
        const uint4* kn = reinterpret_cast<const uint4*>(a.k_new + (size_t)u * D);
        const uint4* vn = reinterpret_cast<const uint4*>(a.v_new + (size_t)u * D);
        for (int i = lane; i < D / 8; i += 64) {
            reinterpret_cast<uint4*>(a.Kc + row * D)[i] = kn[i];
            reinterpret_cast<uint4*>(a.Vc + row * D)[i] = vn[i];
        }
    }
}

// PMAX = bpc / 32: block slots per thread (the chunk is 32 PMAX blocks). Phase-trace slots: 0 start,
// 1 role (1 chunk, 2 last block), 2 query in LDS, 3 first slot computed, 4 every slot computed,
// 6 stores begin, 15 end.
template <int D, int G, bool kStep, int PMAX>
__global__ __launch_bounds__(kThreads) void score_chunks_kernel(Geom geo, ScoreArgs a) {
    constexpr int NB = chunk_slots<PMAX>();
    static_assert(NB % 64 == 0 && NB >= 32 * PMAX, "per-block rows must cover the chunk and whole waves");
    __shared__ ChunkLds<D, G, kStep, NB> lds;
    const int units = geo.units();
    COMPKV_TRACE_START();
    const int tail = a.tail_first ? (int)blockIdx.x : (int)blockIdx.x - units * a.nchunks;
    if (tail >= 0 && tail < units) {
        COMPKV_MARK_VALUE(a.trace, 1, 2);
        score_tail<D, G, kStep>(geo, a, tail, lds.t);
        COMPKV_TRACE_END(a.trace);
        return;
    }
    COMPKV_MARK_VALUE(a.trace, 1, 1);
    const int ck = a.tail_first ? (int)blockIdx.x - units : (int)blockIdx.x;
    constexpr int NF4 = D / 32;           // float4 of the mean-key row per lane
    constexpr int LPB = D / 4;            // compensation: lanes per mean-value row (one float4 each)
    constexpr int RPS = kThreads / LPB;   // mean-value rows per workgroup step
    constexpr int VROWS = kStep ? 32 * PMAX / RPS : 1;
    ChunkShared<D, G, NB>& sh = lds.c.sh;
    auto& st = lds.c.st;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // every chunk of unit u (like its last-block workgroup) on XCD u % kXcds, the XCD whose L2 the
    // unit's selection then reads the chunks' outputs through (the chunks' linear ids start at 0 or at
    // units, a multiple of kXcds whenever the mapping applies)
    int u, chunk;
    xcd_unit_work(ck, units, a.nchunks, u, chunk);
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int xmax = geo.xmax();
    const float s = a.scale;
    const int chunk0 = chunk * a.bpc;
    const int li = tid & 7, grp = tid >> 3;
    const int vli = tid % LPB, vslot = tid / LPB;
    const bool comp = kStep && a.comp_part != nullptr;  // fused step with Mean compensation (uniform)
    const float half = kind_half(a.score_kind);

    // The sequence length and the query pairs first, on their own: loads return in order per compute
    // unit, so requesting the mean keys only once the query is in LDS keeps the query (and the first
    // slots' keys) from queueing behind the mean keys of the other workgroups on the CU. Then per slot
    // the mean key and first variance group (the mean values follow once the keys are consumed, which
    // halves the registers held). Block ids past the allocated range load block 0 of the unit; values
    // of blocks that turn out invalid are never used (every result below is selected by validity).
    const int n_raw = a.seq_lens[bseq];
    const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    QueryPairs<D, G> qp;
    load_query_pairs<D, G>(qh, geo.layout, qp);
    store_query<D, G>(qp, s, geo.r, geo.layout, sh.q, sh.Qv);
    const int n = clamp_len(n_raw, geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    const int xs = X - 1;  // blocks [0, X - 1) are scored here (all full); the last one by the extra workgroup
    const float logB = logf((float)geo.B);
    __syncthreads();
    COMPKV_MARK(a.trace, 2);  // the query in LDS
    // a rolling window of two slots: slot p + 2 is requested once slot p is computed
    float4 kv[2][NF4];
    float dv0[2];
    auto issue = [&](int p, int w) {
        const int b = chunk0 + p * 32 + grp;
        const size_t blk = (size_t)u * geo.xcap + (b < xmax ? b : 0);
        const float4* kp = reinterpret_cast<const float4*>(a.kmean + blk * D);
#pragma unroll
        for (int m = 0; m < NF4; ++m) kv[w][m] = kp[li + 8 * m];
        dv0[w] = a.dvar[blk * geo.r + min(li, geo.r - 1)];
    };
    issue(0, 0);
    if (PMAX > 1) issue(1, 1);
    float4 vrow[VROWS];

    // slot by slot, in the order the slots' loads return: the projected variances (the lead lane of
    // each block keeps them in LDS), then the block-mean logits one pair of heads at a time, the pair's
    // query slice read from LDS into registers
    float qv[G];
#pragma unroll
    for (int g = 0; g < G; ++g) qv[g] = li < geo.r ? sh.Qv[g][li] : 0.0f;
    constexpr int GB = G < 2 ? G : 2;
#pragma unroll
    for (int p = 0; p < PMAX; ++p) {
        const int w = p & 1;
        const int lb = p * 32 + grp;
        const int b = chunk0 + lb;
        const bool valid = b < xs;
        const float lnb = valid ? logB : 0.0f;
        float v[G];
#pragma unroll
        for (int g = 0; g < G; ++g) v[g] = qv[g] * dv0[w];
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
            v[g] = sum8_lead(v[g]);
            if (li == 0) sh.v[g][lb] = v[g];
        }
#pragma unroll 1
        for (int g0 = 0; g0 < G; g0 += GB) {
            float4 qq[GB][NF4];
#pragma unroll
            for (int gb = 0; gb < GB; ++gb)
#pragma unroll
                for (int m = 0; m < NF4; ++m) qq[gb][m] = *reinterpret_cast<const float4*>(&sh.q[g0 + gb][4 * (li + 8 * m)]);
#pragma unroll
            for (int gb = 0; gb < GB; ++gb) {
                float z = 0.0f;
#pragma unroll
                for (int m = 0; m < NF4; ++m)
                    z += qq[gb][m].x * kv[w][m].x + qq[gb][m].y * kv[w][m].y + qq[gb][m].z * kv[w][m].z +
                         qq[gb][m].w * kv[w][m].w;
                z = sum8_lead(z);
                if (li == 0) {
                    const int g = g0 + gb;
                    sh.z[g][lb] = z;
                    if constexpr (kStep) st.cw[g][lb] = valid ? lnb + z : -INFINITY;  // pseudo-logit
                }
            }
        }
        if (p + 2 < PMAX) issue(p + 2, w);
        if (p == 0) COMPKV_MARK(a.trace, 3);  // the first slot computed
    }
    COMPKV_MARK(a.trace, 4);  // every slot computed
    if (comp) {  // mean-value rows, requested once the mean keys are consumed
        const float4* vm = reinterpret_cast<const float4*>(a.vmean + (size_t)u * geo.xcap * D) + vli;
#pragma unroll
        for (int k = 0; k < VROWS; ++k) {
            const int b = chunk0 + vslot + k * RPS;
            vrow[k] = vm[(size_t)(b < xmax ? b : 0) * (D / 4)];
        }
    }
    __syncthreads();
    // log weight a = log|b| + zbar + half * sig2 of valid block lb of the chunk
    auto logw = [&](int g, int lb) {  // (every block of a chunk is full: |b| = B)
        return logB + sh.z[g][lb] + half * sh.v[g][lb];
    };
    // the chunk's per-head max and sum of exp(a - max) (and, fused, of the pseudo-logits)
    const int nvalid = max(0, min(a.bpc, xs - chunk0));
    for (int g = wave; g < G; g += 4) {
        float av[NB / 64];
        float m = -INFINITY;
#pragma unroll
        for (int k = 0; k < NB / 64; ++k) {
            const int lb = lane + 64 * k;
            av[k] = lb < nvalid ? logw(g, lb) : -INFINITY;
            m = fmaxf(m, av[k]);
        }
        m = wave_max(m);
        float ssum = 0.0f;
        if (m != -INFINITY) {
#pragma unroll
            for (int k = 0; k < NB / 64; ++k) ssum += (av[k] == -INFINITY) ? 0.0f : expf(av[k] - m);
        }
        ssum = wave_sum(ssum);
        if (lane == 0) {
            sh.m[g] = m;
            float* pp = a.ws_part + (((size_t)u * (a.nchunks + 1) + chunk) * G + g) * 2;
            pp[0] = m;
            pp[1] = ssum;
        }
        if constexpr (kStep) if (comp) {
            float cv[NB / 64];
            float cm = -INFINITY;
#pragma unroll
            for (int k = 0; k < NB / 64; ++k) {
                const int lb = lane + 64 * k;
                cv[k] = lb < nvalid ? st.cw[g][lb] : -INFINITY;
                cm = fmaxf(cm, cv[k]);
            }
            cm = wave_max(cm);
            float csum = 0.0f;
#pragma unroll
            for (int k = 0; k < NB / 64; ++k) {
                const int lb = lane + 64 * k;
                const float wv = (cv[k] == -INFINITY) ? 0.0f : __expf(cv[k] - cm);
                st.cw[g][lb] = wv;
                csum += wv;
            }
            csum = wave_sum(csum);
            if (lane == 0) {
                st.cm[g] = cm;
                st.cl[g] = csum;
            }
        }
    }
    __syncthreads();
    COMPKV_MARK(a.trace, 6);  // the chunk's partials formed: stores
    // coalesced stores: block logits [g][b] (when requested) and score terms [b][g]
    for (int idx = tid; a.zlog && idx < G * nvalid; idx += kThreads) {
        const int g = idx / nvalid, lb = idx % nvalid;
        a.zlog[((size_t)u * G + g) * a.zstride + chunk0 + lb] = sh.z[g][lb];
    }
    for (int idx = tid; !a.logit_terms && idx < G * nvalid; idx += kThreads) {
        const int lb = idx / G, g = idx % G;
        a.ws_w[((size_t)u * xmax + chunk0 + lb) * G + g] =
            expf(logw(g, lb) - sh.m[g]) * kind_term(a.score_kind, sh.v[g][lb]);
    }
    if constexpr (kStep) if (comp) {
        // weighted mean values; lane vli of a row slot holds coordinates 4 vli .. 4 vli + 3
        float acc[G][4];
#pragma unroll
        for (int g = 0; g < G; ++g) acc[g][0] = acc[g][1] = acc[g][2] = acc[g][3] = 0.0f;
#pragma unroll
        for (int k = 0; k < VROWS; ++k) {
            const int lb = vslot + k * RPS;
            if (lb < nvalid) {
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const float wv = st.cw[g][lb];
                    acc[g][0] += wv * vrow[k].x;
                    acc[g][1] += wv * vrow[k].y;
                    acc[g][2] += wv * vrow[k].z;
                    acc[g][3] += wv * vrow[k].w;
                }
            }
        }
#pragma unroll
        for (int off = LPB; off < 64; off <<= 1)
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[g][e] = xor_add(acc[g][e], off);
        if (lane < LPB) {
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int e = 0; e < 4; ++e) st.acc[wave][g][4 * vli + e] = acc[g][e];
        }
        __syncthreads();
        float* cp = a.comp_part + ((size_t)u * a.part_count + chunk) * G * (D + 2);
        for (int idx = tid; idx < G * D; idx += kThreads) {
            const int g = idx / D, i = idx % D;
            float* p = cp + (size_t)g * (D + 2);
            if (i == 0) {
                p[0] = st.cm[g];
                p[1] = st.cl[g];
            }
            p[2 + i] = st.acc[0][g][i] + st.acc[1][g][i] + st.acc[2][g][i] + st.acc[3][g][i];
        }
    }
    COMPKV_TRACE_END(a.trace);
}

template <int G, bool kLogits = false>
__global__ __launch_bounds__(kFinThreads) void select_finalize_kernel(Geom geo, ScoreArgs a) {
    __shared__ FinalShared sh;
    extern __shared__ float dyn[];
    const int u = blockIdx.x;
    finalize_select<G, false, kFinThreads, kLogits ? 4 : kKeysPerThread, kLogits>(
        geo, a, u, sh, dyn, a.sel + (size_t)u * a.K, a.n_sel + u, true);
}


// ---------------------------------------------------------------- one workgroup per unit
// For units with few blocks (G * xmax <= kUnitTerms) one 1024-thread workgroup per unit refreshes the
// active block (fused step), forms every block's block-mean logits, projected variances and log
// weight estimates (kept in LDS), the per-head log normalizers over every block, the scores and the
// selection: one launch, no partials. The summaries are read in batches of passes of 128 blocks (8
// lanes per block, as in the chunk kernel), each batch's loads issued before its arithmetic.
constexpr int kUnitBatch = 2;  // passes whose summaries a thread requests at once

template <int D, int G>
struct UnitShared {
    float q[G][D];
    float Qv[G][D];
    BlockStatsLds<D> bs;
    float lse[G];
};

template <int D, int G, bool kStep>
__global__ __launch_bounds__(kFinThreads) void unit_select_kernel(Geom geo, ScoreArgs a) {
    constexpr int FT = kFinThreads, KPT = kKeysPerThread, NF4 = D / 32, PB = kUnitBatch;
    constexpr int GPP = FT / 8;  // blocks per pass
    __shared__ FinalShared sh;
    __shared__ UnitShared<D, G> us;
    extern __shared__ float dyn[];  // [xmax][G] log weights (later the key bits), [xmax][G] projected variances
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u = blockIdx.x, bseq = u / geo.hkv, h = u % geo.hkv;
    const int xmax = geo.xmax();
    const int li = tid & 7, grp = tid >> 3;
    float* A = dyn;
    float* Vp = dyn + (size_t)xmax * G;
    const float s = a.scale;

    // loads in the order of their use: query pairs, the refreshed block's rows, the first batch
    const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    QueryPairs<D, G> qp;
    if (wave < 4) load_query_pairs<D, G>(qh, geo.layout, qp);
    __asm__ volatile("" ::: "memory");
    const int n_raw = a.seq_lens[bseq];
    const int n = clamp_len(n_raw, geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    const int npass = (X + GPP - 1) / GPP;
    // workgroup-uniform; a length beyond max_seq_len appends nothing (as in the chunked path)
    const bool refresh = kStep && a.k_new && X >= 1 && n_raw <= geo.max_seq;
    const int lastb = X - 1;
    const size_t blk_last = (size_t)u * geo.xcap + (lastb >= 0 ? lastb : 0);
    BlockSrc src{};
    BlockRows rows;
    if (refresh) {
        const size_t row0 = (size_t)block_row0(geo, u, lastb);
        const int nb = n - lastb * geo.B;
        src = BlockSrc{a.Kc + row0 * D, a.Vc + row0 * D, a.k_new + (size_t)u * D, a.v_new + (size_t)u * D, nb, nb - 1};
        if (wave < 4) load_block_rows<D>(src, 0, rows);
    }
    float4 kv[PB][NF4];
    float dv0[PB];
    auto issue = [&](int p0) {  // branch-free: ids past xmax load block 0, unused
#pragma unroll
        for (int p = 0; p < PB; ++p) {
            const int b = (p0 + p) * GPP + grp;
            const size_t blk = (size_t)u * geo.xcap + (b < xmax ? b : 0);
            const float4* kp = reinterpret_cast<const float4*>(a.kmean + blk * D);
#pragma unroll
            for (int m = 0; m < NF4; ++m) kv[p][m] = kp[li + 8 * m];
            dv0[p] = a.dvar[blk * geo.r + min(li, geo.r - 1)];
        }
    };
    issue(0);
    if (wave < 4) store_query<D, G>(qp, s, geo.r, geo.layout, us.q, us.Qv);
    select_init(sh);
    if (refresh)  // (its barriers also publish the query)
        block_stats_from<D>(src, rows, geo.r, geo.layout, a.kmean_w + blk_last * D, a.dvar_w + blk_last * geo.r,
                            a.vmean + blk_last * D, us.bs, wave < 4);
    else
        __syncthreads();

    // every block: zbar, sig2 and a = log|b| + zbar + sig2 / 2 per head. A block's sig2 goes to LDS
    // first; the lane that wrote it reads it back for a.
    constexpr int GB = G < 2 ? G : 2;
    float qv0[G];
#pragma unroll
    for (int g = 0; g < G; ++g) qv0[g] = li < geo.r ? us.Qv[g][li] : 0.0f;
    for (int p0 = 0; p0 < npass; p0 += PB) {  // workgroup-uniform
        if (p0 > 0) issue(p0);
        if (refresh) {
#pragma unroll
            for (int p = 0; p < PB; ++p) {
                if ((p0 + p) * GPP + grp == lastb) {  // the refreshed summary
#pragma unroll
                    for (int m = 0; m < NF4; ++m) kv[p][m] = *reinterpret_cast<const float4*>(&us.bs.km[4 * (li + 8 * m)]);
                    dv0[p] = us.bs.dv[min(li, geo.r - 1)];
                }
            }
        }
#pragma unroll
        for (int p = 0; p < PB; ++p) {
            const int b = (p0 + p) * GPP + grp;
            const bool valid = b < X;
            float v[G];
#pragma unroll
            for (int g = 0; g < G; ++g) v[g] = qv0[g] * dv0[p];
            if (geo.r > 8 && valid) {
                const size_t blk = (size_t)u * geo.xcap + b;
                for (int t = li + 8; t < geo.r; t += 8) {
                    const float dv = (refresh && b == lastb) ? us.bs.dv[t] : a.dvar[blk * geo.r + t];
#pragma unroll
                    for (int g = 0; g < G; ++g) v[g] += us.Qv[g][t] * dv;
                }
            }
#pragma unroll
            for (int g = 0; g < G; ++g) {
                v[g] = sum8_lead(v[g]);
                if (li == 0 && valid) Vp[b * G + g] = v[g];
            }
        }
#pragma unroll 1
        for (int g0 = 0; g0 < G; g0 += GB) {  // (not unrolled: one head pair's query in registers at a time)
            float4 qq[GB][NF4];
#pragma unroll
            for (int gb = 0; gb < GB; ++gb)
#pragma unroll
                for (int m = 0; m < NF4; ++m) qq[gb][m] = *reinterpret_cast<const float4*>(&us.q[g0 + gb][4 * (li + 8 * m)]);
#pragma unroll
            for (int p = 0; p < PB; ++p) {
                const int b = (p0 + p) * GPP + grp;
                const bool valid = b < X;
#pragma unroll
                for (int gb = 0; gb < GB; ++gb) {
                    float z = 0.0f;
#pragma unroll
                    for (int m = 0; m < NF4; ++m)
                        z += qq[gb][m].x * kv[p][m].x + qq[gb][m].y * kv[p][m].y + qq[gb][m].z * kv[p][m].z +
                             qq[gb][m].w * kv[p][m].w;
                    z = sum8_lead(z);
                    if (li == 0 && valid) {
                        const int g = g0 + gb;
                        const float lnb = logf((float)min(geo.B, n - b * geo.B));
                        A[b * G + g] = lnb + z + kind_half(a.score_kind) * Vp[b * G + g];
                        if (a.zlog) a.zlog[((size_t)u * G + g) * a.zstride + b] = z;
                    }
                }
            }
        }
    }
    if (refresh && wave == 4) {  // the new token's cache row (the refresh read it from k_new / v_new)
        const size_t row = (size_t)block_row0(geo, u, lastb) + (n - 1 - lastb * geo.B);
        const uint4* kn = reinterpret_cast<const uint4*>(a.k_new + (size_t)u * D);
        const uint4* vn = reinterpret_cast<const uint4*>(a.v_new + (size_t)u * D);
        for (int i = lane; i < D / 8; i += 64) {
            reinterpret_cast<uint4*>(a.Kc + row * D)[i] = kn[i];
            reinterpret_cast<uint4*>(a.Vc + row * D)[i] = vn[i];
        }
    }
    __syncthreads();
    // wave g: head g's log normalizer over every block
    if (wave < G) {
        const int g = wave;
        float m = -INFINITY;
        for (int b = lane; b < X; b += 64) m = fmaxf(m, A[b * G + g]);
        m = wave_max(m);
        float l = 0.0f;
        for (int b = lane; b < X; b += 64) l += expf(A[b * G + g] - m);
        l = wave_sum(l);
        if (lane == 0) us.lse[g] = m + logf(l);
    }
    __syncthreads();
    // scores and keys; thread t holds blocks t + 1024k
    unsigned long long ck[KPT];
    uint32_t mx = 0u;
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
        const int b = tid + k * FT;
        ck[k] = 0ull;
        if (b < X) {
            float S = 0.0f;
#pragma unroll
            for (int g = 0; g < G; ++g) S += expf(A[b * G + g] - us.lse[g]) * kind_term(a.score_kind, Vp[b * G + g]);
            if (a.scores) a.scores[(size_t)u * geo.xcap + b] = S;
            if (!mandatory(b, X, a.n_sink, a.n_recent)) {
                ck[k] = ((unsigned long long)__float_as_uint(S) << 32) | (0xFFFFFFFFu - (uint32_t)b);
                mx = max(mx, __float_as_uint(S));
            }
        }
    }
    // (the key bits of the radix path overwrite the log weights, which every thread has read by then)
    const SelectCtx sc = make_select_ctx(X, a.K, a.n_sink, a.n_recent, a.sel + (size_t)u * a.K, a.n_sel + u,
                                         reinterpret_cast<uint32_t*>(A));
    if (select_fast<KPT>(sc, ck, mx, sh)) return;
    __syncthreads();
    select_radix(sc, sh);
}

// ---------------------------------------------------------------- selection + exact items, fused
// Form 1 of the fused step's selection/exact launch: a one-dimensional grid of (items + n_comp) * units
// workgroups of kSxThreads threads, mapped by xcd_unit_work so that (when the units fill whole rounds
// of eight) all workgroups of unit u run on XCD u % 8. Every item workgroup of a unit repeats the unit's
// selection from the chunk partials (the same computation as select_finalize_kernel, so all of them
// hold the same ids) into LDS; item 0 also writes the selection outputs. Then the sixteen waves attend
// exactly over the item's blocks (exact.h, one 16-token tile per wave and round) and write the item's
// partial. The unit's last workgroup to arrive merges its partials (merge_unit), so the step needs no
// further launch. The launch pays off while every workgroup is resident at once (one per CU).
//
// Compensation workgroups (the fused step with Mean compensation and the chunk launch scoring only):
// the same launch also holds n_comp workgroups per unit, after the item workgroups in the grid, that
// stream the mean values of every block while the item workgroups select. Workgroup c of unit u takes
// blocks [c cb, (c + 1) cb): the pseudo-token of each (logit log|b| + zbar_b from the block logits the
// chunk launch wrote, value vmean_b), reduced to one softmax partial per head (max, sum of weights,
// weighted mean values). The exact items take their selected blocks' pseudo-tokens back out, so the
// compensation needs no selection and the mean values stream while the HBM would otherwise idle.
// threads of the fused selection/exact launch's workgroups and keys per thread
constexpr int kSxThreads = 1024;
constexpr int kSxKeys = 8192 / kSxThreads;
// mean-value rows per thread and batch of a compensation workgroup (two batches in flight: 32 KB at
// d = 128). While nearly every CU streams, that suffices for the HBM rate, and less data queued at the
// memory keeps the latency of the selections' and the exact items' loads short.
constexpr int kCompRows = 1;

// Exact attention of unit u over nblk selected blocks whose ids are in LDS (ids; -1 or an id past the
// unit's blocks contributes nothing) into decode partial `part` of the unit (device-coherent stores).
// Under Mean compensation every token's weight is p_j - p'_j (the chunk launch's block logits).
// absorb: the workgroup's compensation partial (step_compensation with kKeep) joins the stored partial.
template <int D, int G, int NW, typename Lds>
__device__ void sx_exact(const Geom& geo, const DecodeArgs& d, int u, int n, const int32_t* ids, int nblk,
                         int part, Lds& L, bool absorb = false) {
    constexpr int FT = NW * 64;
    const int tid = threadIdx.x;
    const int bseq = u / geo.hkv, h = u % geo.hkv;
    const int X = (n + geo.B - 1) / geo.B;
    TokenMap tm;
    tm.dense = false;
    tm.B = geo.B;
    tm.invB = 1.0f / (float)geo.B;
    tm.n = n;
    tm.X = X;
    tm.nblk = nblk;
    tm.sel = ids;
    tm.t0 = tm.t1 = 0;
    tm.page = tm.pg0 = 0;
    tm.invP = 0.0f;
    tm.rowbase = L.rowbase;
    for (int k = tid; k < nblk; k += FT) {
        const int b = ids[k];
        L.rowbase[k] = block_row0(geo, u, b >= 0 && b < X ? b : 0);
    }
    __syncthreads();
    float m, l;
    v4f32 acc[D / 16];
    const uint16_t* qh = d.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    const bool pseudo = d.neg_pseudo != 0;  // Mean: the compensation added every block's pseudo-token
    exact_tokens<D, G, NW>(tm, d.K, d.V, qh, pseudo ? d.blk_logit + (size_t)u * G * geo.xcap : nullptr, geo.xcap,
                           L.u.ex.zb, d.scale, m, l, acc);
    COMPKV_MARK(d.trace, 8);  // this wave 0's tiles attended
    constexpr int kCwStride = (int)(sizeof(L.cw[0]) / sizeof(float));
    finish_exact<D, G, NW, true>(m, l, acc, L.u.ex, d.ws_part + ((size_t)u * d.part_count + part) * G * (D + 2),
                                 absorb ? L.cm : nullptr, L.cl, &L.cw[0][0], kCwStride);
    COMPKV_MARK(d.trace, 9);  // partial stored
}

template <int D, int G, int FT, int KPT, bool kLogits = false>
__global__ __launch_bounds__(FT) void select_exact_kernel(Geom geo, ScoreArgs a, DecodeArgs d, int items) {
    constexpr int NW = FT / 64;
    using Lds = SelExactLdsT<D, G, kStepCbMax, NW>;
    __shared__ Lds L;
    extern __shared__ float dyn[];
    const int tid = threadIdx.x;
    const int units = geo.units();
    COMPKV_TRACE_START();
    int u, item;
    if ((int)blockIdx.x >= items * units) {  // a compensation workgroup (workgroup-uniform)
        COMPKV_MARK_VALUE(d.trace, 1, 2);
        int c;
        xcd_unit_work((int)blockIdx.x - items * units, units, d.n_comp, u, c);
        const int xmax = geo.xmax();
        const int c0 = min(c * d.cb, xmax), c1 = min(c0 + d.cb, xmax);
        step_compensation<D, G, kCompRows, Lds, FT>(geo, d, u, d.seq_lens[u / geo.hkv], c0, c1, L,
                                                          d.ws_part + ((size_t)u * d.part_count + c) * G * (D + 2),
                                                          [] {});
        COMPKV_MARK(d.trace, 9);
        if (d.arrive) arrive_and_merge<D, G, Lds, FT>(geo, d, u, L);
        COMPKV_TRACE_END(d.trace);
        return;
    }
    COMPKV_MARK_VALUE(d.trace, 1, 1);
    // the items of unit u all on XCD u % kXcds: the unit's selection inputs are fetched once into
    // that XCD's L2
    xcd_unit_work(blockIdx.x, units, items, u, item);
    finalize_select<G, false, FT, KPT, kLogits>(geo, a, u, L.u.fin, dyn, L.sel, &L.nsel, item == 0);
    __syncthreads();
    COMPKV_MARK(d.trace, 4);  // selected
    const int n = clamp_len(d.seq_lens[u / geo.hkv], geo.max_seq);
    const int nsel = L.nsel;
    if (item == 0) {  // the selection outputs (the ids past n_sel hold -1)
        for (int k = tid; k < a.K; k += FT) a.sel[(size_t)u * a.K + k] = L.sel[k];
        if (tid == 0) a.n_sel[u] = nsel;
    }
    const int e0 = item * d.eb;
    sx_exact<D, G, NW>(geo, d, u, n, L.sel + e0, max(0, min(d.eb, nsel - e0)), d.part_base + item, L);
    if (d.arrive) arrive_and_merge<D, G, Lds, FT>(geo, d, u, L);
    COMPKV_TRACE_END(d.trace);
}

// ---------------------------------------------------------------- selection + exact, one selector
// The same step when every workgroup of the launch is resident at once: per unit one selector and
// P - 1 workers (grid units * P, the selectors first; xcd_unit_work keeps a unit's workgroups on one
// XCD). The selector ranks the unit's blocks and posts every id slot k < K to the unit's mailbox
// (id ^ kPosted, device-coherent; the chunk launch zeroed the mailbox, and no posted value is zero),
// then attends exactly over the first eb ids. Worker w (1 .. P - 1) first streams its share of the
// mean values (compensation blocks [(w - 1) cb, w cb)), requesting its slots [w eb, (w + 1) eb) of the
// mailbox once the last mean values are in; a slot still zero is polled until posted (a bounded wait:
// the selector started before any worker and never waits itself; past the bound the unit's outputs
// become NaN and its timeout word counts it). Then it attends exactly over those ids, and its
// compensation partial (kept in LDS) joins its exact partial: workgroup w stores partial w, and the
// unit's last workgroup of P merges the P partials. The HBM streams from the start on every CU but the
// selectors', and the selection runs once per unit.
// Phase-trace slots (both forms of the fused launch): 0 start, 1 role (1 selects, 2 streams mean values
// first), 2 the selection's loads in, 3 keys formed, 4 selected, 5 compensation weights formed, 6 mean
// values weighed, 7 ids in hand (worker), 8 wave 0's tiles attended, 9 partial stored, 10 merges, 15 end.
constexpr uint32_t kPosted = 0x80000000u;  // mailbox value of id b: b ^ kPosted (-1 gives 0x7FFFFFFF)
constexpr uint32_t kSelFailed = 1u;        // selection word: a worker's wait timed out
constexpr int kSelSpinLimit = 1 << 17;     // polls of a wait (each a memory round trip): well over 50 ms

// KPT: keys per thread of the selection (xmax <= KPT kSxThreads); kLogits: a.logit_terms
template <int D, int G, int KPT, bool kLogits = false>
__global__ __launch_bounds__(kSxThreads) void select_work_kernel(Geom geo, ScoreArgs a, DecodeArgs d, int P) {
    constexpr int FT = kSxThreads, NW = FT / 64;
    using Lds = SelExactLdsT<D, G, kStepCbMax, NW>;
    __shared__ Lds L;
    extern __shared__ float dyn[];
    const int tid = threadIdx.x;
    const int units = geo.units();
    COMPKV_TRACE_START();
    int u, w;
    if ((int)blockIdx.x < units) {
        u = blockIdx.x;  // (XCD blockIdx % 8 = u % 8)
        w = 0;
    } else {
        xcd_unit_work((int)blockIdx.x - units, units, P - 1, u, w);
        ++w;
    }
    uint32_t* word = d.sel_word + u;
    uint32_t* mbox = d.mailbox + (size_t)u * a.K;
    COMPKV_MARK_VALUE(d.trace, 1, w == 0 ? 1 : 2);
    if (w == 0) {
        finalize_select<G, false, FT, KPT, kLogits>(geo, a, u, L.u.fin, dyn, L.sel, &L.nsel, true);
        __syncthreads();
        COMPKV_MARK(d.trace, 4);  // selected
        for (int k = tid; k < a.K; k += FT) {
            const int32_t b = L.sel[k];
            st_agent_u32(mbox + k, (uint32_t)b ^ kPosted);
            a.sel[(size_t)u * a.K + k] = b;
        }
        if (tid == 0) a.n_sel[u] = L.nsel;
        const int n = clamp_len(d.seq_lens[u / geo.hkv], geo.max_seq);
        sx_exact<D, G, NW>(geo, d, u, n, L.sel, max(0, min(d.eb, L.nsel)), 0, L);
    } else {
        const int n_raw = d.seq_lens[u / geo.hkv];
        const int e0 = w * d.eb;
        const int nblk = max(0, min(d.eb, a.K - e0));  // (the ids past n_sel are -1)
        uint32_t mv = 0u;
        auto request = [&] { mv = ld_agent_u32(mbox + (tid < nblk ? e0 + tid : 0)); };
        const bool comp = d.n_comp > 0;  // (workgroup-uniform)
        if (comp) {  // its compensation partial stays in LDS for the exact partial to absorb
            const int xmax = geo.xmax();
            const int c0 = min((w - 1) * d.cb, xmax), c1 = min(c0 + d.cb, xmax);
            // the slots are polled once the last mean values are requested: if the selector has posted
            // them by then, they return with those values; else they are requested once more after them
            step_compensation<D, G, kCompRows, Lds, FT, true>(
                geo, d, u, n_raw, c0, c1, L, nullptr, [&] { if (__any(mv == 0u)) request(); }, request);
        } else {
            request();
        }
        const int n = clamp_len(n_raw, geo.max_seq);
        bool ok = true;
        if (tid < nblk) {
            for (int spins = 0; mv == 0u && spins < kSelSpinLimit; ++spins) {
                __builtin_amdgcn_s_sleep(2);
                mv = ld_agent_u32(mbox + e0 + tid);
            }
            ok = mv != 0u;
            L.sel[tid] = ok ? (int32_t)(mv ^ kPosted) : -1;
        }
        if (!ok) {
            __hip_atomic_fetch_or(word, kSelFailed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (d.timeouts) __hip_atomic_fetch_add(d.timeouts + 4 * u + 3, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();
        COMPKV_MARK(d.trace, 7);  // the ids in hand
        sx_exact<D, G, NW>(geo, d, u, n, L.sel, nblk, w, L, comp);
    }
    if (arrive_last(d.arrive + u, P, L.last)) {
        COMPKV_MARK(d.trace, 10);  // this workgroup merges
        const bool failed = (ld_agent_u32(word) & kSelFailed) != 0;  // (workgroup-uniform)
        merge_unit<D, G, Lds, FT>(geo, d, u, L, failed);
    }
    COMPKV_TRACE_END(d.trace);
}

template <int D, int G, bool kStep, int PMAX>
void launch_chunks_p(const Geom& g, ScoreArgs a, hipStream_t s) {
    const int grid = (a.nchunks + 1) * g.units();
    a.tail_first = grid <= resident_slots(score_chunks_kernel<D, G, kStep, PMAX>);
    score_chunks_kernel<D, G, kStep, PMAX><<<dim3(grid), kThreads, 0, s>>>(g, a);
}

template <int D, int G, bool kStep>
void launch_chunks(const Geom& g, const ScoreArgs& a, hipStream_t s) {
    switch (a.bpc / 32) {
        case 1: launch_chunks_p<D, G, kStep, 1>(g, a, s); break;
        case 2: launch_chunks_p<D, G, kStep, 2>(g, a, s); break;
        default: launch_chunks_p<D, G, kStep, 4>(g, a, s); break;
    }
}

template <int D, int G>
hipError_t launch_pair(const Geom& g, const ScoreArgs& a, hipStream_t s) {
    if (a.one_group) {
        const size_t dyn = (size_t)2 * g.xmax() * G * sizeof(float);
        if (a.k_new)
            unit_select_kernel<D, G, true><<<dim3(g.units()), kFinThreads, dyn, s>>>(g, a);
        else
            unit_select_kernel<D, G, false><<<dim3(g.units()), kFinThreads, dyn, s>>>(g, a);
        return hipGetLastError();
    }
    if (a.comp_part || a.k_new)  // fused step: the refresh and / or the compensation partials
        launch_chunks<D, G, true>(g, a, s);
    else
        launch_chunks<D, G, false>(g, a, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.chunks_only) return e;
    if constexpr (G >= 4) {
        if (a.logit_terms) {
            select_finalize_kernel<G, true><<<dim3(g.units()), kFinThreads, finalize_dyn_lds(g, a), s>>>(g, a);
            return hipGetLastError();
        }
    }
    select_finalize_kernel<G><<<dim3(g.units()), kFinThreads, finalize_dyn_lds(g, a), s>>>(g, a);
    return hipGetLastError();
}

template <int D>
hipError_t dispatch_g(const Geom& g, const ScoreArgs& a, hipStream_t s) {
    switch (g.G) {
        case 1: return launch_pair<D, 1>(g, a, s);
        case 2: return launch_pair<D, 2>(g, a, s);
        case 4: return launch_pair<D, 4>(g, a, s);
        case 8: return launch_pair<D, 8>(g, a, s);
        default: return hipErrorInvalidValue;
    }
}

template <int D, int G>
hipError_t launch_sx(const Geom& g, const ScoreArgs& a, const DecodeArgs& d, int items, hipStream_t s) {
    const dim3 grid((items + d.n_comp) * g.units());
    const size_t dyn = finalize_dyn_lds(g, a);
    if constexpr (G >= 4) {
        if (a.logit_terms) {  // (at most 4096 blocks: checked by the launcher)
            if (g.xmax() <= kSxThreads)
                select_exact_kernel<D, G, kSxThreads, 1, true><<<grid, kSxThreads, dyn, s>>>(g, a, d, items);
            else
                select_exact_kernel<D, G, kSxThreads, 4, true><<<grid, kSxThreads, dyn, s>>>(g, a, d, items);
            return hipGetLastError();
        }
    }
    // keys per thread for the unit's blocks (as in launch_work)
    if (g.xmax() <= kSxThreads)
        select_exact_kernel<D, G, kSxThreads, 1><<<grid, kSxThreads, dyn, s>>>(g, a, d, items);
    else if (g.xmax() <= 4 * kSxThreads)
        select_exact_kernel<D, G, kSxThreads, 4><<<grid, kSxThreads, dyn, s>>>(g, a, d, items);
    else
        select_exact_kernel<D, G, kSxThreads, kSxKeys><<<grid, kSxThreads, dyn, s>>>(g, a, d, items);
    return hipGetLastError();
}

template <int D, int G>
hipError_t launch_work(const Geom& g, const ScoreArgs& a, const DecodeArgs& d, int P, hipStream_t s) {
    const dim3 grid(P * g.units());
    const size_t dyn = finalize_dyn_lds(g, a);
    if constexpr (G >= 4) {
        if (a.logit_terms) {  // (at most 4096 blocks: checked by the launcher)
            if (g.xmax() <= kSxThreads)
                select_work_kernel<D, G, 1, true><<<grid, kSxThreads, dyn, s>>>(g, a, d, P);
            else
                select_work_kernel<D, G, 4, true><<<grid, kSxThreads, dyn, s>>>(g, a, d, P);
            return hipGetLastError();
        }
    }
    // keys per thread for the unit's blocks: fewer loads and keys where the blocks are few
    if (g.xmax() <= kSxThreads)
        select_work_kernel<D, G, 1><<<grid, kSxThreads, dyn, s>>>(g, a, d, P);
    else if (g.xmax() <= 4 * kSxThreads)
        select_work_kernel<D, G, 4><<<grid, kSxThreads, dyn, s>>>(g, a, d, P);
    else
        select_work_kernel<D, G, kSxKeys><<<grid, kSxThreads, dyn, s>>>(g, a, d, P);
    return hipGetLastError();
}

template <int D>
hipError_t work_g(const Geom& g, const ScoreArgs& a, const DecodeArgs& d, int P, hipStream_t s) {
    switch (g.G) {
        case 1: return launch_work<D, 1>(g, a, d, P, s);
        case 2: return launch_work<D, 2>(g, a, d, P, s);
        case 4: return launch_work<D, 4>(g, a, d, P, s);
        case 8: return launch_work<D, 8>(g, a, d, P, s);
        default: return hipErrorInvalidValue;
    }
}

template <int D>
hipError_t sx_g(const Geom& g, const ScoreArgs& a, const DecodeArgs& d, int items, hipStream_t s) {
    switch (g.G) {
        case 1: return launch_sx<D, 1>(g, a, d, items, s);
        case 2: return launch_sx<D, 2>(g, a, d, items, s);
        case 4: return launch_sx<D, 4>(g, a, d, items, s);
        case 8: return launch_sx<D, 8>(g, a, d, items, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

int select_max_bpc() { return kBpcMax; }
int select_exact_max_budget() { return kSelLdsMax; }
int select_exact_waves() { return kSxThreads / 64; }
int select_exact_max_cb() { return kStepCbMax; }
int select_exact_merge_terms() { return kMergeMaxTerms; }

// Resident workgroups of the one-selector fused launch on the current device with `dyn` bytes of
// dynamic LDS each.
template <int D, int G>
int sx_slots(size_t dyn) {
    int per_cu = 0, cus = 0, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, select_work_kernel<D, G, kSxKeys>, kSxThreads, dyn) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    return per_cu * cus;
}
template <int D>
int sx_slots_d(const Geom& g, size_t dyn) {
    switch (g.G) {
        case 1: return sx_slots<D, 1>(dyn);
        case 2: return sx_slots<D, 2>(dyn);
        case 4: return sx_slots<D, 4>(dyn);
        default: return sx_slots<D, 8>(dyn);
    }
}
int select_exact_slots(const Geom& g, size_t dyn) { return g.D == 128 ? sx_slots_d<128>(g, dyn) : sx_slots_d<64>(g, dyn); }

// the selection's logit-terms input (ScoreArgs::logit_terms) within its limits
bool logit_terms_ok(const Geom& g, const ScoreArgs& a) {
    return !a.logit_terms || (g.r == 4 && g.G >= 4 && g.G <= 8 && g.xmax() <= 4 * kFinThreads && a.zlog && a.ws_qv);
}

hipError_t launch_select_exact(const Geom& g, ScoreArgs a, const DecodeArgs& d, int items, hipStream_t s) {
    // the keys of the fast path's tie fallback stay in LDS: no workgroup writes global scratch
    a.keys_in_lds = 1;
    if (!logit_terms_ok(g, a)) return hipErrorInvalidValue;
    if (a.bpc < 1 || (a.bpc & (a.bpc - 1)) != 0 || g.xmax() > kFinThreads * kKeysPerThread || a.K > kSelLdsMax ||
        d.eb > kMaxEb ||
        finalize_dyn_lds(g, a) > kDynBudget || (d.n_comp > 0 && (d.cb < 1 || d.cb > kStepCbMax)) ||
        (long long)d.n_comp * d.cb < (d.n_comp > 0 ? g.xmax() : 0) || d.part_base + items > d.part_count ||
        (d.arrive && (d.part_count != d.n_comp + items || d.part_count * g.G > kMergeMaxTerms)))
        return hipErrorInvalidValue;
    return g.D == 128 ? sx_g<128>(g, a, d, items, s) : sx_g<64>(g, a, d, items, s);
}
hipError_t launch_select_work(const Geom& g, ScoreArgs a, const DecodeArgs& d, int P, hipStream_t s) {
    a.keys_in_lds = 1;
    if (!logit_terms_ok(g, a)) return hipErrorInvalidValue;
    const int keff = std::max(1, std::min(a.K, g.xmax()));
    if (P < 2 || a.bpc < 1 || (a.bpc & (a.bpc - 1)) != 0 || g.xmax() > kFinThreads * kKeysPerThread || a.K > kSelLdsMax || d.eb < 1 || d.eb > kMaxEb ||
        (long long)P * d.eb < keff || finalize_dyn_lds(g, a) > kDynBudget || !d.arrive || !d.sel_word || !d.mailbox ||
        (d.n_comp != 0 && (d.n_comp != P - 1 || d.cb < 1 || d.cb > kStepCbMax || (long long)d.n_comp * d.cb < g.xmax())) ||
        d.part_base != 0 || d.part_count != P || d.part_count * g.G > kMergeMaxTerms)
        return hipErrorInvalidValue;
    return g.D == 128 ? work_g<128>(g, a, d, P, s) : work_g<64>(g, a, d, P, s);
}
int select_one_group_terms() { return kUnitTerms; }
int select_one_group_auto_blocks() { return kUnitBatch * kFinThreads / 8; }
int select_max_chunk_heads() { return (int)(kDynBudget / (2 * sizeof(float))); }

hipError_t launch_score_select(const Geom& g, ScoreArgs a, hipStream_t s) {
    if (!logit_terms_ok(g, a) || (a.logit_terms && a.one_group)) return hipErrorInvalidValue;
    if (a.one_group) {
        if (g.G * g.xmax() > kUnitTerms) return hipErrorInvalidValue;
        return g.D == 128 ? dispatch_g<128>(g, a, s) : dispatch_g<64>(g, a, s);
    }
    if (a.bpc != 32 && a.bpc != 64 && a.bpc != 128) return hipErrorInvalidValue;
    a.keys_in_lds = 0;
    a.keys_in_lds = finalize_dyn_lds(g, a) + (size_t)g.xmax() * sizeof(float) <= kDynBudget;
    if (finalize_dyn_lds(g, a) > kDynBudget) return hipErrorInvalidValue;
    return g.D == 128 ? dispatch_g<128>(g, a, s) : dispatch_g<64>(g, a, s);
}

}  // namespace compkv

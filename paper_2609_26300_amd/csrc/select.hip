// select.hip -- block scoring and Top-K selection (Sections 4.1, 4.2; Appendix E.1). Two launches.
//
// Launch 1, grid = (nchunks, units): each workgroup streams the fp32 summaries (mean key, grouped
// variances) of `bpc` consecutive blocks of one unit. Eight lanes share a block: lane i of the eight
// reads float4 i, i+8, ... of the mean-key row (the eight lanes read 128 contiguous bytes per load) and
// the variance groups t = i, i+8, .... Every load of a thread is issued before any arithmetic. For
// each of the unit's G query heads it forms the block-mean logit zbar = s q.kmean, the projected
// variance sig2 = s^2 sum_t Q_t dvar_t and the log weight estimate a = log|b| + zbar + sig2/2 (the log
// of the numerator of Eq. compkv-mass-estimate). It writes zbar (block logits, reused by the decode),
// the chunk's per-head (max m_c of a, sum of exp(a - m_c)), and per block the G terms
// w_g = exp(a_g - m_c) sig2_g, stored contiguously so one vector load fetches a block's terms.
//
// Launch 2, grid = (units): the kernel boundary makes every chunk's results visible (no
// cross-workgroup fences or atomics). One workgroup per unit merges the chunk partials into each
// head's log normalizer lse_g and forms S_b = sum_g exp(m_c - lse_g) w_g (= Eq. compkv-score). Block b
// is ranked by the 64-bit key (bits of S_b) << 32 | ~b: scores are >= 0, so their IEEE bit patterns order
// like the values, and the keys are unique and order exactly like (S_b descending, b ascending), the
// stable Top-K of the paper. Up to 8192 blocks the keys stay in registers (32 per thread). One
// histogram of each key's distance below the largest score (bins of 1/16 octave on the float bits; keys
// farther than 255 bins are not counted) locates the bin that holds the (K-|F|)-th largest key; only the
// keys in that bin or above are ranked exactly, by brute force, and a bitmap of the selected and
// mandatory blocks is compacted into ascending ids. Larger inputs, or ties that leave too many keys at
// or above the cut's bin, go through a three-pass radix select on the score bits instead.
#include "block_stats.h"

#include <type_traits>

namespace compkv {
namespace {

constexpr int kBpcMax = 128;  // blocks per chunk, upper bound
constexpr int kPMax = kBpcMax / 32;
constexpr int kHistBins = 2048;
constexpr size_t kDynBudget = 32768;  // dynamic LDS of the finalize launch

template <int D, int G>
struct ChunkShared {
    float q[G][D];   // scaled query
    float Qv[G][D];  // s^2 * sum of q^2 over each group (first r entries)
    float z[G][kBpcMax];
    float v[G][kBpcMax];
    float a[G][kBpcMax];
    float m[G];
};

// Extra state of the fused decode step: the refreshed summary of the active block, the compensation
// weights and the per-wave compensation sums.
template <int D, int G>
struct StepShared {
    alignas(16) float km[D];
    alignas(16) float vm[D];
    float dv[D], m2s[D];
    float cw[G][kBpcMax];
    float cm[G], cl[G];
    alignas(16) float acc[4][G][D];
};
struct NoStep {};

// kStep (fused decode step): before scoring, the workgroup whose chunk holds the active block stores the
// new row and recomputes that block's summary (the append's routine, so bit-identical), then scores the
// block from the LDS copy. After scoring, every chunk also forms the compensation partial of all its
// blocks: pseudo-logits log|b| + zbar_g,b, weights exp(. - chunk max), weighted mean values.
template <int D, int G, bool kStep>
__global__ __launch_bounds__(kThreads) void score_chunks_kernel(Geom geo, ScoreArgs a) {
    constexpr int NF4 = D / 32;  // float4 of the mean-key row per lane
    constexpr int LPB = D / 4;             // compensation: lanes per mean-value row (one float4 each)
    constexpr int RPS = kThreads / LPB;    // mean-value rows per workgroup step
    constexpr int VROWS = kStep ? kBpcMax / RPS : 1;
    __shared__ ChunkShared<D, G> sh;
    __shared__ std::conditional_t<kStep, StepShared<D, G>, NoStep> st;
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
    const int vli = tid % LPB, vslot = tid / LPB;

    int ab = -1;  // active block refreshed by this workgroup
    if constexpr (kStep) {
        if (a.k_new && n >= 1 && (n - 1) / geo.B / a.bpc == chunk) {  // uniform over the workgroup
            ab = (n - 1) / geo.B;
            const int nb = n - ab * geo.B;
            const uint16_t* kn = a.k_new + (size_t)u * D;
            const uint16_t* vn = a.v_new + (size_t)u * D;
            if (wave == 0) {
                const size_t row = (size_t)u * geo.cap + (n - 1);
                for (int i = lane; i < D / 8; i += 64) {
                    reinterpret_cast<uint4*>(a.Kc + row * D)[i] = reinterpret_cast<const uint4*>(kn)[i];
                    reinterpret_cast<uint4*>(a.Vc + row * D)[i] = reinterpret_cast<const uint4*>(vn)[i];
                }
            }
            const size_t row0 = (size_t)u * geo.cap + (size_t)ab * geo.B;
            const size_t blk = (size_t)u * geo.xcap + ab;
            wave_block_stats<D>(a.Kc + row0 * D, a.Vc + row0 * D, nb, kn, vn, nb - 1, geo.r, geo.layout,
                                a.kmean_w + blk * D, a.dvar_w + blk * geo.r, a.vmean + blk * D, st.m2s, wave == 0,
                                st.km, st.dv, st.vm);
        }
    }

    // issue the summary loads of this thread's blocks first
    float4 kv[kPMax][NF4];
    float dv0[kPMax];
    // (branch-free: an invalid slot loads block 0 of the unit, always allocated, and is zeroed after)
#pragma unroll
    for (int p = 0; p < kPMax; ++p) {
        const int b = chunk0 + p * 32 + grp;
        const bool valid = p < P && b < X;
        const size_t blk = (size_t)u * geo.xcap + (valid ? b : 0);
        const float4* kp = reinterpret_cast<const float4*>(a.kmean + blk * D);
#pragma unroll
        for (int m = 0; m < NF4; ++m) kv[p][m] = kp[li + 8 * m];
        dv0[p] = a.dvar[blk * geo.r + min(li, geo.r - 1)];
    }
    float4 vrow[VROWS];
    if constexpr (kStep) {
        const float4* vm = reinterpret_cast<const float4*>(a.vmean + (size_t)u * geo.xcap * D) + vli;
#pragma unroll
        for (int k = 0; k < VROWS; ++k) {
            if (k * RPS >= a.bpc) break;
            const int b = chunk0 + vslot + k * RPS;
            vrow[k] = vm[(size_t)(b < X ? b : 0) * (D / 4)];
        }
    }
#pragma unroll
    for (int p = 0; p < kPMax; ++p) {
        const int b = chunk0 + p * 32 + grp;
        const bool valid = p < P && b < X;
#pragma unroll
        for (int m = 0; m < NF4; ++m) kv[p][m] = valid ? kv[p][m] : make_float4(0, 0, 0, 0);
        dv0[p] = (valid && li < geo.r) ? dv0[p] : 0.0f;
        if constexpr (kStep) {
            if (b == ab) {  // the refreshed summary (the global copy may predate the refresh)
#pragma unroll
                for (int m = 0; m < NF4; ++m) kv[p][m] = *reinterpret_cast<const float4*>(&st.km[4 * (li + 8 * m)]);
                dv0[p] = li < geo.r ? st.dv[li] : 0.0f;
            }
        }
    }
    if constexpr (kStep) {
#pragma unroll
        for (int k = 0; k < VROWS; ++k)
            if (chunk0 + vslot + k * RPS == ab) vrow[k] = *reinterpret_cast<const float4*>(&st.vm[4 * vli]);
    }
    const uint16_t* qh = a.q + ((size_t)bseq * geo.hq + (size_t)h * G) * D;
    for (int idx = tid; idx < G * D; idx += kThreads) sh.q[idx / D][idx % D] = s * bf16_at(qh + idx);
    __syncthreads();
    for (int idx = tid; idx < G * geo.r; idx += kThreads) {
        // s^2 Q_{g,t}: squared (scaled) query coordinates summed over group t (Appendix A.4)
        const int g = idx / geo.r, t = idx % geo.r;
        float acc = 0.0f;
        if (geo.r == D) {
            acc = sh.q[g][t] * sh.q[g][t];
        } else {
            const int w = (D / 2) / geo.r;
            for (int k = 0; k < 2 * w; ++k) {
                const int i = geo.layout == 0 ? (k < w ? t * w + k : D / 2 + t * w + (k - w)) : 2 * t * w + k;
                acc += sh.q[g][i] * sh.q[g][i];
            }
        }
        sh.Qv[g][t] = acc;
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
                const float4 qq = *reinterpret_cast<const float4*>(&sh.q[g][4 * (li + 8 * m)]);
                acc += qq.x * kv[p][m].x + qq.y * kv[p][m].y + qq.z * kv[p][m].z + qq.w * kv[p][m].w;
            }
            z[g] = acc;
            v[g] = li < geo.r ? sh.Qv[g][li] * dv0[p] : 0.0f;
        }
        if (geo.r > 8 && valid) {
            const size_t blk = (size_t)u * geo.xcap + b;
            for (int t = li + 8; t < geo.r; t += 8) {
                float dv = a.dvar[blk * geo.r + t];
                if constexpr (kStep) dv = (b == ab) ? st.dv[t] : dv;
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
            const float lnb = valid ? logf((float)min(geo.B, n - b * geo.B)) : 0.0f;
#pragma unroll
            for (int g = 0; g < G; ++g) {
                sh.z[g][lb] = z[g];
                sh.v[g][lb] = v[g];
                sh.a[g][lb] = valid ? lnb + z[g] + 0.5f * v[g] : -INFINITY;
                if constexpr (kStep) st.cw[g][lb] = valid ? lnb + z[g] : -INFINITY;  // pseudo-logit
            }
        }
    }
    __syncthreads();
    // the chunk's per-head max and sum of exp(a - max)
    const int nvalid = max(0, min(a.bpc, X - chunk0));
    for (int g = wave; g < G; g += 4) {
        float av[kBpcMax / 64];
        float m = -INFINITY;
#pragma unroll
        for (int k = 0; k < kBpcMax / 64; ++k) {
            const int lb = lane + 64 * k;
            av[k] = lb < nvalid ? sh.a[g][lb] : -INFINITY;
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
            sh.m[g] = m;
            float* pp = a.ws_part + (((size_t)u * a.nchunks + chunk) * G + g) * 2;
            pp[0] = m;
            pp[1] = ssum;
        }
        if constexpr (kStep) {  // compensation weights of every block of the chunk
            float cv[kBpcMax / 64];
            float cm = -INFINITY;
#pragma unroll
            for (int k = 0; k < kBpcMax / 64; ++k) {
                const int lb = lane + 64 * k;
                cv[k] = lb < nvalid ? st.cw[g][lb] : -INFINITY;
                cm = fmaxf(cm, cv[k]);
            }
            cm = wave_max(cm);
            float csum = 0.0f;
#pragma unroll
            for (int k = 0; k < kBpcMax / 64; ++k) {
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
    // coalesced stores: block logits [g][b] and score terms [b][g]
    for (int idx = tid; idx < G * nvalid; idx += kThreads) {
        const int g = idx / nvalid, lb = idx % nvalid;
        a.blk_logit[((size_t)u * G + g) * geo.xcap + chunk0 + lb] = sh.z[g][lb];
    }
    for (int idx = tid; idx < G * nvalid; idx += kThreads) {
        const int lb = idx / G, g = idx % G;
        a.ws_w[((size_t)u * xmax + chunk0 + lb) * G + g] = expf(sh.a[g][lb] - sh.m[g]) * sh.v[g][lb];
    }
    if constexpr (kStep) {
        // weighted mean values; lane vli of a row slot holds coordinates 4 vli .. 4 vli + 3
        float acc[G][4];
#pragma unroll
        for (int g = 0; g < G; ++g) acc[g][0] = acc[g][1] = acc[g][2] = acc[g][3] = 0.0f;
#pragma unroll
        for (int k = 0; k < VROWS; ++k) {
            const int lb = vslot + k * RPS;
            if (k * RPS >= a.bpc) break;
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
                for (int e = 0; e < 4; ++e) acc[g][e] += __shfl_xor(acc[g][e], off);
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
}

constexpr int kRegKeys = 32;    // score keys one thread keeps in registers (fast path: X <= 8192)
constexpr int kCandCap = 1024;  // candidates ranked by brute force on the fast path
constexpr int kHistTail = 255;  // distance bins counted on the fast path (bin 255 = everything farther)

struct FinalShared {
    float lse[8];
    int hist[kHistBins];
    int cnt[4], cnt2[4];
    int scan[4];
    int digit, above;
    unsigned long long cand[kCandCap];
    uint32_t bitmap[kThreads];
    int ncand, beta;
};

template <int G>
__global__ __launch_bounds__(kThreads) void select_finalize_kernel(Geom geo, ScoreArgs a) {
    constexpr int NBATCH = 8;  // blocks whose score terms one thread loads at once
    __shared__ FinalShared sh;
    extern __shared__ float dyn[];  // [nchunks][G] factors, [nchunks][G] sums, then [xmax] score bits
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u = blockIdx.x;
    const int bseq = u / geo.hkv;
    const int n = clamp_len(a.seq_lens[bseq], geo.max_seq);
    const int X = (n + geo.B - 1) / geo.B;
    const int xmax = geo.xmax();
    const int nc = a.nchunks;

    // ---- per-head log normalizer over every block, then each chunk's factor exp(m_c - lse)
    float* fac = dyn;
    float* sums = dyn + nc * G;
    const float* pu = a.ws_part + (size_t)u * nc * G * 2;
    for (int idx = tid; idx < nc * G; idx += kThreads) {
        fac[idx] = pu[2 * idx];
        sums[idx] = pu[2 * idx + 1];
    }
    __syncthreads();
    for (int g = wave; g < G; g += 4) {
        float m = -INFINITY;
        for (int c = lane; c < nc; c += 64) m = fmaxf(m, fac[c * G + g]);
        m = wave_max(m);
        float l = 0.0f;
        for (int c = lane; c < nc; c += 64) {
            const float pm = fac[c * G + g];
            if (pm != -INFINITY) l += sums[c * G + g] * expf(pm - m);
        }
        l = wave_sum(l);
        if (lane == 0) sh.lse[g] = m + logf(l);
    }
    __syncthreads();
    for (int idx = tid; idx < nc * G; idx += kThreads) {
        const float pm = fac[idx];
        fac[idx] = pm == -INFINITY ? 0.0f : expf(pm - sh.lse[idx % G]);
    }
    __syncthreads();

    const int K = a.K;
    const bool take_all = K >= X;
    int n_mand;
    {
        const int sink = min(a.n_sink, X);
        const int rec_lo = max(X - a.n_recent, 0);
        n_mand = sink + (X - rec_lo) - max(0, sink - rec_lo);
    }
    const int kk = take_all ? 0 : K - n_mand;  // >= 0: the host checks K >= n_sink + n_recent
    int32_t* sel = a.sel + (size_t)u * K;
    uint32_t* keys = a.keys_in_lds ? reinterpret_cast<uint32_t*>(dyn + 2 * nc * G) : a.ws_key + (size_t)u * xmax;
    const float* wu = a.ws_w + (size_t)u * xmax * G;

    // ---- fast path. Block b's key is (bits of S_b) << 32 | ~b: unique, and ordered exactly like
    // (S_b descending, b ascending). Thread t keeps the keys of blocks t + 256k in registers.
    if (X <= kRegKeys * kThreads) {
        unsigned long long ck[kRegKeys];
#pragma unroll
        for (int k0 = 0; k0 < kRegKeys; k0 += NBATCH) {
            float w[NBATCH][G];
#pragma unroll
            for (int k = 0; k < NBATCH; ++k) {
                const int b = tid + (k0 + k) * kThreads;
                const size_t bs = (size_t)(b < X ? b : 0) * G;  // branch-free; unused when b >= X
                if constexpr (G % 4 == 0) {
#pragma unroll
                    for (int g4 = 0; g4 < G; g4 += 4) {
                        const float4 t4 = *reinterpret_cast<const float4*>(wu + bs + g4);
                        w[k][g4] = t4.x;
                        w[k][g4 + 1] = t4.y;
                        w[k][g4 + 2] = t4.z;
                        w[k][g4 + 3] = t4.w;
                    }
                } else {
#pragma unroll
                    for (int g = 0; g < G; ++g) w[k][g] = wu[bs + g];
                }
            }
#pragma unroll
            for (int k = 0; k < NBATCH; ++k) {
                const int b = tid + (k0 + k) * kThreads;
                ck[k0 + k] = 0ull;
                if (b < X) {
                    const float* f = fac + (b / a.bpc) * G;
                    float S = 0.0f;
#pragma unroll
                    for (int g = 0; g < G; ++g) S += f[g] * w[k][g];
                    if (a.scores) a.scores[(size_t)u * geo.xcap + b] = S;
                    if (!mandatory(b, X, a.n_sink, a.n_recent))
                        ck[k0 + k] = ((unsigned long long)__float_as_uint(S) << 32) | (0xFFFFFFFFu - (uint32_t)b);
                }
            }
        }
        // histogram of the keys' distance below the largest score, in bins of 2^19 float ulps (1/16 of
        // an octave); keys more than 255 bins below are not counted
        uint32_t mx = 0u;
#pragma unroll
        for (int k = 0; k < kRegKeys; ++k) mx = ck[k] ? max(mx, (uint32_t)(ck[k] >> 32)) : mx;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
        if (lane == 0) sh.scan[wave] = (int)mx;
        sh.hist[tid] = 0;
        sh.bitmap[tid] = 0u;
        if (tid == 0) {
            sh.beta = kHistTail;
            sh.ncand = 0;
        }
        __syncthreads();
        if (!take_all && kk > 0) {
            const uint32_t smax = max(max((uint32_t)sh.scan[0], (uint32_t)sh.scan[1]),
                                      max((uint32_t)sh.scan[2], (uint32_t)sh.scan[3]));
            uint32_t bin[kRegKeys];
#pragma unroll
            for (int k = 0; k < kRegKeys; ++k) {
                const uint32_t bits = (uint32_t)(ck[k] >> 32);
                bin[k] = ck[k] ? min((smax - bits) >> 19, (uint32_t)kHistTail) : 0xFFFFFFFFu;
                if (bin[k] < (uint32_t)kHistTail) atomicAdd(&sh.hist[bin[k]], 1);
            }
            __syncthreads();
            // inclusive prefix over bins (thread t holds bin t); the bin reaching kk holds the cut
            const int c = sh.hist[tid];
            int incl = c;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int o = __shfl_up(incl, off);
                if (lane >= off) incl += o;
            }
            if (lane == 63) sh.cnt[wave] = incl;
            __syncthreads();
            for (int w = 0; w < wave; ++w) incl += sh.cnt[w];
            if (tid < kHistTail && incl - c < kk && incl >= kk) sh.beta = tid;
            __syncthreads();
            const uint32_t beta = (uint32_t)sh.beta;  // kHistTail: the cut lies below the counted range
#pragma unroll
            for (int k = 0; k < kRegKeys; ++k) {
                const bool cnd = bin[k] <= beta;
                const unsigned long long mask = __ballot(cnd);
                if (mask == 0ull) continue;
                const int first = __ffsll((long long)mask) - 1;
                int base = 0;
                if (lane == first) base = atomicAdd(&sh.ncand, __popcll(mask));
                base = __shfl(base, first);
                const int pos = base + lanes_below(mask);
                if (cnd && pos < kCandCap) sh.cand[pos] = ck[k];
            }
            __syncthreads();
            const int m = sh.ncand;
            if (m <= kCandCap) {
                // exact rank among the candidates; the kk best are selected
                for (int i = tid; i < m; i += kThreads) {
                    const unsigned long long ci = sh.cand[i];
                    int r = 0;
                    int j = 0;
                    for (; j + 16 <= m; j += 16) {
#pragma unroll
                        for (int e = 0; e < 16; ++e) r += sh.cand[j + e] > ci;
                    }
                    for (; j < m; ++j) r += sh.cand[j] > ci;
                    if (r < kk) {
                        const uint32_t b = 0xFFFFFFFFu - (uint32_t)(ci & 0xFFFFFFFFull);
                        atomicOr(&sh.bitmap[b >> 5], 1u << (b & 31));
                    }
                }
            } else {
                // too many ties around the threshold: keep the bits for the radix path below
#pragma unroll
                for (int k = 0; k < kRegKeys; ++k) {
                    const int b = tid + k * kThreads;
                    if (b < X) keys[b] = (uint32_t)(ck[k] >> 32);
                }
            }
            if (m > kCandCap) goto radix_path;  // block-uniform (every thread read the same m)
        }
        // mandatory blocks (or every block when K >= X); thread t owns ids 32t .. 32t+31
        {
            __syncthreads();  // every selected bit is set
            uint32_t word = sh.bitmap[tid];
#pragma unroll
            for (int bit = 0; bit < 32; ++bit) {
                const int b = 32 * tid + bit;
                if (b < X && (take_all || mandatory(b, X, a.n_sink, a.n_recent))) word |= 1u << bit;
            }
            const int c = __popc(word);
            int incl = c;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int o = __shfl_up(incl, off);
                if (lane >= off) incl += o;
            }
            if (lane == 63) sh.scan[wave] = incl;
            __syncthreads();
            int pos = incl - c, total = 0;
            for (int w = 0; w < 4; ++w) {
                pos += w < wave ? sh.scan[w] : 0;
                total += sh.scan[w];
            }
            while (word) {
                const int bit = __ffs(word) - 1;
                word &= word - 1;
                if (pos < K) sel[pos] = 32 * tid + bit;
                ++pos;
            }
            for (int k = total + tid; k < K; k += kThreads) sel[k] = -1;
            if (tid == 0) a.n_sel[u] = min(total, K);
        }
        return;
    }

    // ---- general path (more than 8192 blocks): scores and their bits into the key array
    for (int b0 = tid; b0 < X; b0 += NBATCH * kThreads) {
        float w[NBATCH][G];
#pragma unroll
        for (int k = 0; k < NBATCH; ++k) {
            const int b = b0 + k * kThreads;
#pragma unroll
            for (int g = 0; g < G; ++g) w[k][g] = b < X ? wu[(size_t)b * G + g] : 0.0f;
        }
#pragma unroll
        for (int k = 0; k < NBATCH; ++k) {
            const int b = b0 + k * kThreads;
            if (b >= X) break;
            const float* f = fac + (b / a.bpc) * G;
            float S = 0.0f;
#pragma unroll
            for (int g = 0; g < G; ++g) S += f[g] * w[k][g];
            if (a.scores) a.scores[(size_t)u * geo.xcap + b] = S;
            keys[b] = __float_as_uint(S);
        }
    }
radix_path:
    __syncthreads();

    // ---- threshold of the Top-(K-|F|) among non-mandatory blocks (radix select on the score bits)
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

    // ---- mark and compact in ascending id order; wave w scans its own id segment
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

size_t finalize_dyn_lds(const Geom& g, const ScoreArgs& a) {
    return ((size_t)2 * a.nchunks * g.G + (a.keys_in_lds ? (size_t)g.xmax() : 0)) * sizeof(float);
}

template <int D, int G>
hipError_t launch_pair(const Geom& g, const ScoreArgs& a, hipStream_t s) {
    if (a.comp_part)
        score_chunks_kernel<D, G, true><<<dim3(a.nchunks, g.units()), kThreads, 0, s>>>(g, a);
    else
        score_chunks_kernel<D, G, false><<<dim3(a.nchunks, g.units()), kThreads, 0, s>>>(g, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    select_finalize_kernel<G><<<dim3(g.units()), kThreads, finalize_dyn_lds(g, a), s>>>(g, a);
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

}  // namespace

int select_max_bpc() { return kBpcMax; }
int select_max_chunk_heads() { return (int)(kDynBudget / (2 * sizeof(float))); }

hipError_t launch_score_select(const Geom& g, ScoreArgs a, hipStream_t s) {
    if (a.bpc % 32 != 0 || a.bpc > kBpcMax || a.bpc < 32) return hipErrorInvalidValue;
    a.keys_in_lds = 0;
    a.keys_in_lds = finalize_dyn_lds(g, a) + (size_t)g.xmax() * sizeof(float) <= kDynBudget;
    if (finalize_dyn_lds(g, a) > kDynBudget) return hipErrorInvalidValue;
    return g.D == 128 ? dispatch_g<128>(g, a, s) : dispatch_g<64>(g, a, s);
}

}  // namespace compkv

// internal.h -- private declarations shared by libcompkv's translation units (not installed).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace compkv {

constexpr int kThreads = 256;  // every kernel runs 256-thread workgroups (4 wave64)

// Shape of one call after host validation. The K/V cache is either contiguous per unit
// ([units][cap][D], bpp == 0) or paged: [npages][hkv][bpp * B][D] with table[bseq][pps] mapping a
// sequence's logical page to a physical page (bpp blocks per page). Row indices below are absolute
// rows of the cache (the host checks that every row index fits in int32).
struct Geom {
    int batch, hq, hkv, G, D, B, r, layout, cap, xcap, max_seq;
    int bpp, pps, npages;  // paged cache (bpp == 0: contiguous)
    float inv_bpp;
    const int32_t* table;
    __host__ __device__ int units() const { return batch * hkv; }
    __host__ __device__ int xmax() const { return (max_seq + B - 1) / B; }
};

// ------------------------------------------------------------------ launch parameter blocks

struct StatsArgs {
    const uint16_t* K;
    const uint16_t* V;
    const uint16_t* k_new;  // append only
    const uint16_t* v_new;  // append only
    uint16_t* K_out;        // append only: cache rows written
    uint16_t* V_out;
    const int32_t* seq_lens;
    float* kmean;
    float* dvar;
    float* vmean;
};

// Phase trace (a library built with -DCOMPKV_PHASE_TRACE; the marks compile to nothing otherwise):
// thread 0 of workgroup w of a traced launch stores the 100 MHz real-time counter at the phase
// boundaries into trace[w * kTraceSlots + slot] (slots per kernel: the kernel's own comment), and a
// role or count into the value slots. Only the fused step's two launches are traced.
constexpr int kTraceSlots = 16;
#ifdef COMPKV_PHASE_TRACE
#define COMPKV_MARK(buf, slot)                                                                           \
    do {                                                                                                 \
        if ((buf) != nullptr && threadIdx.x == 0)                                                        \
            (buf)[(size_t)blockIdx.x * ::compkv::kTraceSlots + (slot)] = __builtin_amdgcn_s_memrealtime(); \
    } while (0)
#define COMPKV_MARK_VALUE(buf, slot, v)                                                                  \
    do {                                                                                                 \
        if ((buf) != nullptr && threadIdx.x == 0)                                                        \
            (buf)[(size_t)blockIdx.x * ::compkv::kTraceSlots + (slot)] = (unsigned long long)(v);        \
    } while (0)
// the start stamp is held (scalar registers) and stored with the end stamp: a store at the very start
// would keep the first loads from being scheduled ahead of it
#define COMPKV_TRACE_START() const unsigned long long compkv_trace_t0_ = __builtin_amdgcn_s_memrealtime()
// slot 14: where the workgroup ran (XCC id << 32 | the HW_ID register: CU, SIMD, wave slot)
#define COMPKV_TRACE_END(buf)                                                          \
    do {                                                                               \
        unsigned compkv_hw_ = 0, compkv_xcc_ = 0;                                      \
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(compkv_hw_));        \
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(compkv_xcc_));      \
        COMPKV_MARK_VALUE(buf, 14, ((unsigned long long)compkv_xcc_ << 32) | compkv_hw_); \
        COMPKV_MARK_VALUE(buf, 0, compkv_trace_t0_);                                   \
        COMPKV_MARK(buf, 15);                                                          \
    } while (0)
#else
#define COMPKV_TRACE_START() \
    do {                     \
    } while (0)
#define COMPKV_TRACE_END(buf) \
    do {                      \
    } while (0)
#define COMPKV_MARK(buf, slot) \
    do {                       \
    } while (0)
#define COMPKV_MARK_VALUE(buf, slot, v) \
    do {                                \
    } while (0)
#endif

struct ScoreArgs {
    const uint16_t* q;
    const float* kmean;
    const float* dvar;
    const int32_t* seq_lens;
    int32_t* sel;
    int32_t* n_sel;
    float* blk_logit;
    float* scores;     // nullable
    float* ws_part;    // [units][nchunks][G][2]  (chunk max m_c, chunk sum of exp(a - m_c))
    float* ws_w;       // [units][xmax][G]       exp(a - m_c) * projected variance (unless logit_terms)
    float* zlog;       // where the chunk launch stores zbar, [units][G][zstride] (blk_logit, or with
    int zstride;       // logit_terms and no blk_logit the ws_w region with stride xmax); null: nowhere
    float* ws_qv;      // [units][G][4]: s^2 Q_{g,t} of the step's query (logit_terms)
    int logit_terms;   // set by the host (r = 4, G >= 4, chunked selection of up to 4096 blocks): the
                       // selection forms each block's terms from zbar (zlog) and its variances (dvar)
                       // instead of reading score terms the chunk launch wrote
    uint32_t* ws_key;  // [units][xmax]          score bits (when they do not fit in LDS)
    int bpc;          // blocks per chunk (multiple of 32)
    int nchunks;      // grid.x
    int keys_in_lds;  // set by the launcher: score bits kept in LDS (else in ws_key)
    int K, n_sink, n_recent;
    float scale;
    // fused decode step only (comp_part == nullptr otherwise)
    const uint16_t* k_new;  // nullable: [units][D] row n - 1 to store; its block's summary is refreshed first
    const uint16_t* v_new;
    uint16_t* Kc;           // caches: row n - 1 written, the active block's rows read
    uint16_t* Vc;
    float* kmean_w;         // writable views of kmean / dvar (the active block only)
    float* dvar_w;
    float* vmean;           // [units][xcap][D]: read by the compensation; the active block written
    float* comp_part;       // [units][part_count][G][D + 2]: chunk c writes compensation partial c
    int part_count;
    int one_group;          // 1: one workgroup per unit scores and selects (no chunks, no partials)
    int score_kind;         // COMPKV_SCORE_*: CompKV score, mass only, or first-order mass estimate
    int chunks_only;        // chunked path: launch the chunk scoring without the selection
    int tail_first;         // set by the launcher: the last-block workgroups lead the grid (else trail)
    uint32_t* arrive_zero;  // nullable: [2][units] words (arrivals, selection words), then [units][K]
                            // (mailbox), that the last-block workgroups zero
    unsigned long long* trace;  // phase-trace build only: [grid][kTraceSlots] timestamps, or null
};

struct DecodeArgs {
    const uint16_t* q;
    const uint16_t* K;
    const uint16_t* V;
    const float* vmean;
    const float* blk_logit;  // with vmean: null for the Drop decode (no compensation items)
    const float* kmean;      // Mean decode without blk_logit: the block-mean logits are recomputed
    const int32_t* seq_lens;
    const int32_t* sel;
    const int32_t* n_sel;
    float* out;
    float* lse;      // nullable
    float* ws_part;  // [units][items][G][D + 2]
    int sel_stride;
    int n_exact;  // exact items per unit
    int eb;       // selected blocks per exact item (sparse) / tokens per item (dense)
    int n_comp;   // compensation items per unit (sparse)
    int cb;       // blocks per compensation item
    int dense;    // 1: every item is a token range of the dense decode
    float scale;
    int part_count;  // partials per unit in ws_part (row stride of the partial array)
    int part_base;   // partial index of this launch's item 0
    int neg_pseudo;  // exact items subtract the pseudo-terms of their selected blocks (fused step)
    int sel_padded;  // the id slots past n_sel hold -1 (written by this library's selection): exact
                     // items read their ids without waiting for n_sel
    uint32_t* arrive;  // fused selection/exact launch: per-unit arrival counters (zeroed by the chunk
                       // launch); the unit's last workgroup merges its partials (null: a merge launch
                       // follows)
    uint32_t* sel_word;  // one-selector fused launch: per-unit selection words (zeroed by the chunk launch)
    uint32_t* mailbox;   // one-selector fused launch: [units][K] posted ids (zeroed by the chunk launch)
    uint32_t* timeouts;  // per-unit words [units][4] at the start of the workspace (word 3 counts timeouts)
    unsigned long long* trace;  // phase-trace build only: [grid][kTraceSlots] timestamps, or null
};

// ------------------------------------------------------------------ launchers (one per kernel family)

hipError_t launch_build_stats(const Geom& g, const StatsArgs& a, hipStream_t s);
hipError_t launch_append_stats(const Geom& g, const StatsArgs& a, hipStream_t s);
hipError_t launch_score_select(const Geom& g, ScoreArgs a, hipStream_t s);
// ScoreArgs::logit_terms within its limits (r = 4, 4 <= G <= 8, at most 4096 blocks, zlog and ws_qv set)
bool logit_terms_ok(const Geom& g, const ScoreArgs& a);
int select_max_bpc();
int select_max_chunk_heads();  // nchunks * G limit of the selection's partial merge
int select_one_group_terms();  // G * xmax limit of the one-workgroup-per-unit selection
int select_one_group_auto_blocks();  // xmax up to which the automatic choice takes that selection
int decode_max_items();
int decode_max_partials();
int decode_max_cb();
int decode_max_eb();
int decode_item_slots(const Geom& g);  // item workgroups resident at once on the current device
int decode_max_row_bases();  // row bases an item holds (dense items of a paged cache: their pages)
hipError_t launch_decode(const Geom& g, const DecodeArgs& a, hipStream_t s);
hipError_t launch_decode_items(const Geom& g, const DecodeArgs& a, int items, hipStream_t s);
// fused step: the selection (from the chunk partials) and the exact items in one launch, `items`
// workgroups of select_exact_waves() waves per unit, plus d.n_comp compensation workgroups per unit of
// d.cb blocks each (partials 0 .. n_comp - 1; the items' from d.part_base); hipErrorInvalidValue outside
// its limits
hipError_t launch_select_exact(const Geom& g, ScoreArgs a, const DecodeArgs& d, int items, hipStream_t s);
// the same step with one selector per unit and P - 1 workers (compensation share d.cb, then exact share
// d.eb once the selection word is set): P workgroups per unit, all resident at once (checked by the
// caller with select_exact_slots); one partial per workgroup (d.part_count = P, d.part_base = 0: a
// worker's compensation partial joins its exact one); hipErrorInvalidValue outside its limits
hipError_t launch_select_work(const Geom& g, ScoreArgs a, const DecodeArgs& d, int P, hipStream_t s);
int select_exact_max_budget();
int select_exact_waves();
int select_exact_max_cb();  // blocks per compensation workgroup of the fused launch
int select_exact_slots(const Geom& g, size_t dyn);  // one-selector launch: workgroups resident at once
int select_exact_merge_terms();  // partials x heads limit of its in-launch merge
hipError_t launch_decode_merge(const Geom& g, const DecodeArgs& a, int nitems, hipStream_t s);

// The decode step in two launches (step.hip): the scores of every completed block (the chunked path's
// chunks of a.bpc blocks), then per unit one selector (the last block, the selection), d.n_comp
// compensation workgroups of d.cb blocks and d.n_exact exact workgroups of d.eb selected blocks,
// ordered through `state` ([units][4] words: unused, final arrivals, phase bits, timeouts; zero on
// entry, returned to zero except the timeout count). The decode partials are [last block's
// compensation][n_comp compensation][n_exact exact] (Mean) or the exact ones alone (Drop);
// d.part_base is the first exact partial. hipErrorInvalidValue outside its limits.
hipError_t launch_step_stream(const Geom& g, ScoreArgs a, const DecodeArgs& d, uint32_t* state, hipStream_t s);
int step_stream_max_cb();  // blocks per compensation workgroup, upper bound
int step_stream_max_budget();
int step_stream_merge_terms();  // partials x heads limit of the in-launch merge
size_t step_stream_dyn_lds(const Geom& g, int nchunks);

// Resident workgroups of `kern` (`threads` each, no dynamic LDS) on the current device, cached per
// (kernel, device). Not thread-safe on first use per kernel; a race only repeats the same query.
template <typename Kern>
int resident_slots(Kern kern, int threads = kThreads) {
    constexpr int kSlots = 64;
    static const void* key_fn[kSlots];
    static int key_dev[kSlots], value[kSlots];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    const void* fn = reinterpret_cast<const void*>(kern);
    for (int i = 0; i < kSlots; ++i)
        if (key_fn[i] == fn && key_dev[i] == dev && value[i] > 0) return value[i];
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, 0) != hipSuccess || per_cu < 1)
        per_cu = 1;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 1;
    for (int i = 0; i < kSlots; ++i)
        if (key_fn[i] == nullptr) {
            key_fn[i] = fn;
            key_dev[i] = dev;
            value[i] = per_cu * cus;
            break;
        }
    return per_cu * cus;
}

// ------------------------------------------------------------------ device helpers

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_at(const uint16_t* p) { return __uint_as_float(uint32_t(*p) << 16); }

__device__ __forceinline__ void unpack_bf16x8(const uint4 w, float f[8]) {
    f[0] = bf16_lo(w.x);
    f[1] = bf16_hi(w.x);
    f[2] = bf16_lo(w.y);
    f[3] = bf16_hi(w.y);
    f[4] = bf16_lo(w.z);
    f[5] = bf16_hi(w.z);
    f[6] = bf16_lo(w.w);
    f[7] = bf16_hi(w.w);
}

__device__ __forceinline__ int clamp_len(int n, int cap) { return n < 0 ? 0 : (n > cap ? cap : n); }

// The dispatcher deals the workgroups of a launch to the XCDs (accelerator complex dies, each with its
// own L2) in turn by linear id. For a one-dimensional grid of units x per workgroups, work item w of
// unit u is given linear id kXcds * (per * (u / kXcds) + w) + u % kXcds when the units fill whole
// rounds of kXcds, so all of a unit's workgroups run on XCD u % kXcds (where the workgroups before
// and after it for that unit run too); otherwise unit-major order. A bijection either way.
constexpr int kXcds = 8;
__device__ __forceinline__ void xcd_unit_work(int lin, int units, int per, int& u, int& w) {
    if (units % kXcds == 0) {
        const int s = lin / kXcds;
        u = lin % kXcds + kXcds * (s / per);
        w = s % per;
    } else {
        u = lin / per;
        w = lin % per;
    }
}

// floor(v / B) for 0 <= v < 2^23: the float quotient is within one of it, and one step corrects it
__device__ __forceinline__ int div_small(int v, int B, float invB) {
    int k = (int)((float)v * invB);
    const int r = v - k * B;
    return k + (r >= B ? 1 : 0) - (r < 0 ? 1 : 0);
}

// Absolute cache row of the first token of logical block blk (0 <= blk < xcap) of unit u; a block's
// rows are consecutive. Paged: one table read; a page id outside [0, npages) is clamped, so a bad table
// entry reads the wrong page but never outside the cache.
__device__ __forceinline__ int block_row0(const Geom& g, int u, int blk) {
    if (g.bpp == 0) return u * g.cap + blk * g.B;
    const int bseq = u / g.hkv, h = u - bseq * g.hkv;
    const int lp = div_small(blk, g.bpp, g.inv_bpp);
    int pg = g.table[(size_t)bseq * g.pps + lp];
    pg = pg < 0 ? 0 : (pg >= g.npages ? g.npages - 1 : pg);
    return ((pg * g.hkv + h) * g.bpp + (blk - lp * g.bpp)) * g.B;
}

// Cross-lane moves with DPP (data-parallel primitives): `old` is kept by lanes whose source is outside
// the row or whose row/bank is masked off.
template <int CTRL, int ROW_MASK = 0xF, int BANK_MASK = 0xF>
__device__ __forceinline__ int dpp_i(int old, int x) {
    return __builtin_amdgcn_update_dpp(old, x, CTRL, ROW_MASK, BANK_MASK, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(x), __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float readlane_f(float x, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

// Wave64 all-reductions (every lane of the wave must be active; the result is wave-uniform). Within
// each 16-lane row: xor 1 and xor 2 (quad permutes), then rotations by 4 and 8; the four row results
// are combined in a fixed order.
__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, dpp_f<0xB1>(v));
    v = fmaxf(v, dpp_f<0x4E>(v));
    v = fmaxf(v, dpp_f<0x124>(v));
    v = fmaxf(v, dpp_f<0x128>(v));
    return fmaxf(fmaxf(readlane_f(v, 0), readlane_f(v, 16)), fmaxf(readlane_f(v, 32), readlane_f(v, 48)));
}

__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f<0xB1>(v);
    v += dpp_f<0x4E>(v);
    v += dpp_f<0x124>(v);
    v += dpp_f<0x128>(v);
    return (readlane_f(v, 0) + readlane_f(v, 16)) + (readlane_f(v, 32) + readlane_f(v, 48));
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    auto mx = [](uint32_t a, uint32_t b) { return a > b ? a : b; };
    v = mx(v, (uint32_t)dpp_i<0xB1>((int)v, (int)v));
    v = mx(v, (uint32_t)dpp_i<0x4E>((int)v, (int)v));
    v = mx(v, (uint32_t)dpp_i<0x124>((int)v, (int)v));
    v = mx(v, (uint32_t)dpp_i<0x128>((int)v, (int)v));
    const uint32_t r0 = __builtin_amdgcn_readlane((int)v, 0), r1 = __builtin_amdgcn_readlane((int)v, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane((int)v, 32), r3 = __builtin_amdgcn_readlane((int)v, 48);
    return mx(mx(r0, r1), mx(r2, r3));
}

// Inclusive prefix sum over the 64 lanes (row shifts by 1, 2, 4, 8, then the row-15 and row-31
// broadcasts carry row totals upward).
__device__ __forceinline__ int wave_incl_scan(int x) {
    x += dpp_i<0x111>(0, x);
    x += dpp_i<0x112>(0, x);
    x += dpp_i<0x114>(0, x);
    x += dpp_i<0x118>(0, x);
    x += dpp_i<0x142, 0xA>(0, x);
    x += dpp_i<0x143, 0xC>(0, x);
    return x;
}

// x + (x of lane ^ off), for a power of two off < 64
__device__ __forceinline__ float xor_add(float x, int off) {
    switch (off) {
        case 1: return x + dpp_f<0xB1>(x);
        case 2: return x + dpp_f<0x4E>(x);
        case 4: return x + __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), 0x101F));
        case 8: return x + dpp_f<0x128>(x);
        case 16: {  // gfx950 lane swaps (VALU, no LDS crossbar): the lower and upper rows of each half
            const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
            return __uint_as_float(r[0]) + __uint_as_float(r[1]);
        }
        case 32: {  // the two halves of the wave
            const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
            return __uint_as_float(r[0]) + __uint_as_float(r[1]);
        }
        default: return x + __shfl_xor(x, off);
    }
}

// Sum over each aligned group of 8 lanes, valid in the group's first four lanes (xor 1 and xor 2 quad
// permutes, then a row shift left by 4: lane i adds lane i + 4).
__device__ __forceinline__ float sum8_lead(float x) {
    x += dpp_f<0xB1>(x);
    x += dpp_f<0x4E>(x);
    x += dpp_f<0x104>(x);
    return x;
}

// block b is mandatory: one of the first n_sink or last n_recent blocks (Section 4.2)
__device__ __forceinline__ bool mandatory(int b, int X, int n_sink, int n_recent) {
    return b < n_sink || b >= X - n_recent;
}

// number of set bits of a wave mask below this lane
__device__ __forceinline__ int lanes_below(unsigned long long mask) {
    const int lane = threadIdx.x & 63;
    return __popcll(mask & ((1ull << lane) - 1ull));
}

// Merge two softmax partials (max m, sum l, accumulators) into the first.
__device__ __forceinline__ void merge_scales(float m_a, float m_b, float& m, float& ca, float& cb) {
    m = fmaxf(m_a, m_b);
    ca = (m_a == -INFINITY) ? 0.0f : __expf(m_a - m);
    cb = (m_b == -INFINITY) ? 0.0f : __expf(m_b - m);
}

}  // namespace compkv

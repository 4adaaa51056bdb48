// api.hip -- host side of the C ABI declared in include/compkv.h: argument validation, workspace
// layout and launch shapes. Never touches device memory from the host.
#include "compkv.h"
#include "internal.h"

#include <algorithm>
#include <initializer_list>
#include <mutex>

using compkv::Geom;

// Scratch of the allocation-free decode step: a fixed device array in place of the caller's
// workspace. Every GPU the library runs on holds its own copy until the process ends. In host code
// `scratch` names a host-side stand-in, never a device address: its device address is looked up per
// device (hipGetSymbolAddress with that device current) and only that address reaches the kernels.
static constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int ceil_div(int a, int b) { return (a + b - 1) / b; }

bool valid_r(int d, int r) { return r >= 1 && (r == d || (d % 2 == 0 && (d / 2) % r == 0)); }

// Validate dims; fill geom. Returns COMPKV_OK or a status.
int check_dims(const compkv_dims* dm, Geom* g) {
    if (!dm) return COMPKV_EINVAL;
    if (dm->batch < 1 || dm->n_q_heads < 1 || dm->n_kv_heads < 1 || dm->n_q_heads % dm->n_kv_heads != 0)
        return COMPKV_EINVAL;
    if (dm->capacity_tokens < 1 || dm->max_seq_len < 1 || dm->max_seq_len > dm->capacity_tokens)
        return COMPKV_EINVAL;
    const int G = dm->n_q_heads / dm->n_kv_heads;
    if (dm->head_dim != 64 && dm->head_dim != 128) return COMPKV_EUNSUPPORTED;
    if (G != 1 && G != 2 && G != 4 && G != 8) return COMPKV_EUNSUPPORTED;
    if (dm->block_size < 1 || dm->block_size > 1024) return COMPKV_EUNSUPPORTED;
    if (!valid_r(dm->head_dim, dm->n_var_groups)) return COMPKV_EUNSUPPORTED;
    if (dm->group_layout != COMPKV_GROUPS_ROTATE_HALF && dm->group_layout != COMPKV_GROUPS_INTERLEAVED)
        return COMPKV_EUNSUPPORTED;
    const long long units = (long long)dm->batch * dm->n_kv_heads;
    if (units > 65535) return COMPKV_EUNSUPPORTED;  // grid.y limit
    // cache rows are addressed with 32-bit indices
    if (dm->page_tokens < 0) return COMPKV_EINVAL;
    if (dm->page_tokens == 0) {
        if (units * dm->capacity_tokens >= (1LL << 31)) return COMPKV_EUNSUPPORTED;
        g->bpp = g->pps = g->npages = 0;
        g->inv_bpp = 0.0f;
        g->table = nullptr;
    } else {
        if (dm->num_pages < 1 || dm->pages_per_seq < 1 || !dm->block_table) return COMPKV_EINVAL;
        if ((long long)dm->pages_per_seq * dm->page_tokens != dm->capacity_tokens) return COMPKV_EINVAL;
        if (dm->page_tokens % dm->block_size != 0) return COMPKV_EUNSUPPORTED;
        if ((long long)dm->num_pages * dm->n_kv_heads * dm->page_tokens >= (1LL << 31)) return COMPKV_EUNSUPPORTED;
        g->bpp = dm->page_tokens / dm->block_size;
        g->pps = dm->pages_per_seq;
        g->npages = dm->num_pages;
        g->inv_bpp = 1.0f / (float)g->bpp;
        g->table = dm->block_table;
    }
    g->batch = dm->batch;
    g->hq = dm->n_q_heads;
    g->hkv = dm->n_kv_heads;
    g->G = G;
    g->D = dm->head_dim;
    g->B = dm->block_size;
    g->r = dm->n_var_groups;
    g->layout = dm->group_layout;
    g->cap = dm->capacity_tokens;
    g->xcap = ceil_div(dm->capacity_tokens, dm->block_size);
    g->max_seq = dm->max_seq_len;
    return COMPKV_OK;
}

// ---------------------------------------------------------------- launch shapes

struct ScoreShape {
    int bpc, nchunks;
};

ScoreShape score_shape(const Geom& g) {
    const int xmax = g.xmax();
    int bpc = 32;
    // widen chunks while the grid keeps >= 1024 workgroups (fewer partials to merge)
    while (bpc < compkv::select_max_bpc() && (long long)g.units() * ceil_div(xmax, bpc * 2) >= 1024) bpc *= 2;
    return {bpc, ceil_div(xmax, bpc)};
}

struct SparseShape {
    int eb, n_exact, cb, n_comp;
};

SparseShape sparse_shape(const Geom& g, int K) {
    const int xmax = g.xmax();
    const int keff = std::max(1, std::min(K, xmax));
    int eb = std::max(1, 128 / g.B);         // one round of 128 exact tokens per item
    eb = std::max(eb, ceil_div(keff, 128));  // at most 128 exact items
    // when the items would take more than one resident round, items of two rounds each (one
    // workgroup's prologue and merge of its waves instead of two)
    if ((long long)g.units() * ceil_div(keff, eb) > compkv::decode_item_slots(g))
        eb = std::max(eb, std::min(compkv::decode_max_eb(), std::max(1, 256 / g.B)));
    const int n_exact = ceil_div(keff, eb);
    int cb = 128;                            // mean-value rows per compensation item
    cb = std::max(cb, ceil_div(xmax, compkv::decode_max_items() - n_exact));
    const int n_comp = ceil_div(xmax, cb);
    return {eb, n_exact, cb, n_comp};
}

struct DenseShape {
    int te, items;
};

DenseShape dense_shape(const Geom& g) {
    // items of up to 1024 tokens (eight rounds of the eight waves: fewer workgroup prologues and wave
    // merges; measured 37.0 -> 33.7 us at 32K) while a unit keeps at least 32 of them, and at most 128
    // items per unit
    int te = std::max(128, std::min(1024, ceil_div(g.max_seq, 32)));
    te = std::max(te, ceil_div(g.max_seq, 128));
    te = ceil_div(te, 128) * 128;  // whole rounds of 128 tokens
    return {te, ceil_div(g.max_seq, te)};
}

// ---------------------------------------------------------------- workspace layout


size_t score_ws(const Geom& g) {
    const ScoreShape sh = score_shape(g);
    const size_t units = g.units(), xmax = g.xmax();
    return align_up(units * (sh.nchunks + 1) * g.G * 2 * sizeof(float)) +
           align_up(units * xmax * g.G * sizeof(float)) + align_up(units * xmax * sizeof(uint32_t)) +
           align_up(units * g.G * 4 * sizeof(float));
}

size_t sparse_ws(const Geom& g, int K) {
    const SparseShape sh = sparse_shape(g, K);
    return align_up((size_t)g.units() * (sh.n_exact + sh.n_comp) * g.G * (g.D + 2) * sizeof(float));
}

size_t dense_ws(const Geom& g) {
    const DenseShape sh = dense_shape(g);
    return align_up((size_t)g.units() * sh.items * g.G * (g.D + 2) * sizeof(float));
}

// phase-trace build: the record arrays of the fused step's two launches (null: not traced)
unsigned long long* g_trace_chunks = nullptr;
unsigned long long* g_trace_fused = nullptr;

struct SxShape {  // the fused step's selection + exact launch (sx_shape below)
    int eb, n_exact;
    int cb, n_comp;  // its compensation workgroups: blocks each, workgroups per unit
    bool fits;       // within the kernel's limits
    bool one_round;  // every workgroup of the chosen form resident at once (one per CU)
    bool work;       // the one-selector form (below) is chosen
    int P, web, wcb;  // one-selector form: workgroups per unit, exact blocks each, compensation blocks
                      // per worker
};
SxShape sx_shape(const Geom& g, int nchunks, int K);

struct StreamShape {  // the two-launch step (stream_shape below)
    int n_comp, cb;    // compensation workgroups per unit, blocks each (0 under Drop)
    int n_exact, eb;   // exact workgroups per unit, selected blocks each
    int parts;         // decode partials per unit
    bool fits;         // within the kernel's limits
};

size_t step_part_bytes(const Geom& g, int parts) {
    return align_up((size_t)g.units() * parts * g.G * (g.D + 2) * sizeof(float));
}

// fused step: the score region, then [units][parts][G][D + 2] decode partials. Chunked path: the
// compensation of each chunk and of the last block, then each exact item's (nchunks + 1 + n_exact);
// fused selection/exact launch: each compensation workgroup's, then each exact item's (n_comp +
// n_exact), or in its one-selector form one per workgroup (P). Sized for the largest.
int step_partials(const Geom& g, int K) {
    const int nchunks = score_shape(g).nchunks;
    const SxShape sx = sx_shape(g, nchunks, K);
    return std::max(std::max(nchunks + 1 + sparse_shape(g, K).n_exact, sx.fits ? sx.n_comp + sx.n_exact : 0),
                    sx.work ? sx.P : 0);
}

// fused step: the arrival counters of the fused selection/exact launch's in-launch merge and the
// selection words of its one-selector form (one each per unit), then that form's mailbox of posted ids
// ([units][K]), follow the partials
size_t step_ws(const Geom& g, int K) {
    return score_ws(g) + step_part_bytes(g, step_partials(g, K)) +
           align_up((size_t)g.units() * (2 + (size_t)K) * sizeof(uint32_t));
}

StreamShape stream_shape(const Geom& g, int K, bool mean);
size_t stream_ws(const Geom& g, int K);

// Every workspace starts with the per-unit words of the two-launch step (final
// arrivals, phase bits, timeouts): zero before a workspace's first compkv_decode_step call, returned to
// zero by every step (the timeout count aside), never written by the other calls.
size_t state_bytes(const Geom& g) { return align_up((size_t)g.units() * 4 * sizeof(uint32_t)); }

size_t ws_bytes(const Geom& g, int K, int which) {
    size_t body = 0;
    if (which == COMPKV_WS_ALL || which == COMPKV_WS_DECODE_STEP)  // either selection path
        body = std::max(body, std::max(step_ws(g, K), sparse_ws(g, K)));
    if (which == COMPKV_WS_ALL || which == COMPKV_WS_SCORE_SELECT) body = std::max(body, score_ws(g));
    if (which == COMPKV_WS_ALL || which == COMPKV_WS_SPARSE_DECODE) body = std::max(body, sparse_ws(g, K));
    if (which == COMPKV_WS_ALL || which == COMPKV_WS_DENSE_DECODE) body = std::max(body, dense_ws(g));
    if (which == COMPKV_WS_ALL || which == COMPKV_WS_DECODE_STEP) body = std::max(body, stream_ws(g, K));
    return state_bytes(g) + body;
}

// select_path of the call: true for the one-workgroup-per-unit selection; *st receives the status
bool one_group_path(const Geom& g, int path, int* st) {
    *st = COMPKV_OK;
    if (path < COMPKV_SELECT_AUTO || path > COMPKV_SELECT_STREAM) {
        *st = COMPKV_EINVAL;
        return false;
    }
    const bool fits = (long long)g.G * g.xmax() <= compkv::select_one_group_terms();
    if (path == COMPKV_SELECT_ONE_GROUP && !fits) *st = COMPKV_EUNSUPPORTED;
    if (path == COMPKV_SELECT_AUTO)  // one workgroup reads at most one batch of summaries per unit
        return fits && g.xmax() <= compkv::select_one_group_auto_blocks();
    return path == COMPKV_SELECT_ONE_GROUP && fits;
}

// Shape of the fused step's selection + exact launch: items of up to select_exact_waves() tiles of 16
// tokens.
SxShape sx_shape(const Geom& g, int nchunks, int K) {
    const int xmax = g.xmax();
    const int keff = std::max(1, std::min(K, xmax));
    int cus = 0, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        cus = 0;
    // one resident round of workgroups (two per CU): up to half of a unit's share goes to compensation
    // workgroups (of at least 128 and at most select_exact_max_cb() blocks each: few partials to merge)
    // and the rest to exact items, the smallest of at least 64 tokens that fit it (an item of more
    // tiles than the workgroup has waves takes several rounds of its waves), so that each CU streams
    // mean values while its item workgroup selects
    const size_t dyn = ((size_t)2 * (nchunks + 1) * g.G + (size_t)xmax) * sizeof(float);
    const int resident = compkv::select_exact_slots(g, dyn);
    const int per = std::max(1, resident / std::max(1, g.units()));
    const int cbmax = compkv::select_exact_max_cb();
    int n_comp = std::max(1, std::min(per / 2, ceil_div(xmax, 128)));
    n_comp = std::max(n_comp, ceil_div(xmax, cbmax));
    const int cb = ceil_div(xmax, n_comp);
    const int slots = std::max(1, per - n_comp);
    const int eb = std::max(std::max(1, 64 / g.B), ceil_div(keff, slots));
    const int n_exact = ceil_div(keff, eb);
    const bool fits = K <= compkv::select_exact_max_budget() && xmax <= 8192 && dyn <= 32768 &&
                      eb <= compkv::decode_max_eb() && n_exact <= compkv::decode_max_items() && cb <= cbmax &&
                      n_comp + n_exact <= compkv::decode_max_partials() &&
                      (n_comp + n_exact) * g.G <= compkv::select_exact_merge_terms();
    // one-selector launch: per unit one selector and P - 1 workers, compensation shares of at least 128
    // blocks, every workgroup resident at once
    int P = std::min(per, 1 + ceil_div(xmax, 128));
    P = std::max(P, 1 + ceil_div(xmax, cbmax));
    P = std::max(P, ceil_div(keff, compkv::decode_max_eb()));
    const int wcb = ceil_div(xmax, std::max(1, P - 1));
    const int web = ceil_div(keff, P);
    const bool work_fits = cus > 0 && P >= 2 && (long long)g.units() * P <= resident &&
                           K <= compkv::select_exact_max_budget() && xmax <= 8192 && dyn <= 32768 &&
                           web <= compkv::decode_max_eb() && wcb <= cbmax &&
                           P * g.G <= compkv::select_exact_merge_terms();
    const bool items_round = fits && cus > 0 && (long long)g.units() * (n_exact + n_comp) <= resident;
    // the one-selector form where a unit's selected tokens are at least its mean-value rows (both 4 d
    // bytes each): spread over all of the unit's workgroups, the exact share then outweighs the repeated
    // selections it saves. Where the mean values dominate, the form with compensation workgroups that
    // stream from the start while the item workgroups select is faster (measured: 128K layer 26.9 vs
    // 28.6 us; wide GQA 33.3 vs 29.9 us; 32K layer 18.3 vs 18.5 us)
    const bool work = work_fits && ((long long)xmax <= (long long)keff * g.B || !items_round);
    return {eb, n_exact, cb, n_comp, fits, work || items_round, work, P, web, wcb};
}

// Shape of the two-launch step: the chunked path's scoring chunks; one round of selectors and
// compensation workgroups (one per compute unit, at least 32 and at most step_stream_max_cb() blocks
// each) so that the mean values stream while the selections run; exact workgroups of one round of the
// sixteen waves (256 tokens).
StreamShape stream_shape(const Geom& g, int K, bool mean) {
    const int xmax = g.xmax();
    const int keff = std::max(1, std::min(K, xmax));
    int cus = 0, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        cus = 256;
    const int units = g.units();
    int n_comp = 0, cb = 0;
    if (mean) {
        n_comp = std::max(1, (cus - units) / units);
        n_comp = std::min(n_comp, std::max(1, ceil_div(xmax, 32)));
        n_comp = std::max(n_comp, ceil_div(xmax, compkv::step_stream_max_cb()));
        cb = ceil_div(xmax, n_comp);
    }
    const int eb = std::max(1, std::min(keff, 256 / g.B));
    const int n_exact = ceil_div(keff, eb);
    const int parts = (mean ? 1 + n_comp : 0) + n_exact;
    const ScoreShape sc = score_shape(g);
    const bool fits = K <= compkv::step_stream_max_budget() && xmax <= 8192 && eb <= compkv::decode_max_eb() &&
                      (long long)parts * g.G <= compkv::step_stream_merge_terms() &&
                      compkv::step_stream_dyn_lds(g, sc.nchunks) <= 32768;
    return {n_comp, cb, n_exact, eb, parts, fits};
}

// the two-launch step: the score region, then [units][parts][G][D + 2] decode partials (Mean's shape,
// the larger)
size_t stream_ws(const Geom& g, int K) {
    const StreamShape sh = stream_shape(g, K, true);
    return score_ws(g) + step_part_bytes(g, sh.parts);
}

bool use_select_exact(int path, const SxShape& sx) {
    return (path == COMPKV_SELECT_CHUNKED_EXACT && (sx.fits || sx.work)) || (path == COMPKV_SELECT_AUTO && sx.one_round);
}

// The fused step's choice of the one-group path: as for the scoring call, except that AUTO prefers the
// fused selection/exact launch whenever all of its workgroups are resident at once (one launch fewer
// than the one-group decode; measured faster at 4K-8K on 2 and 8 units)
bool step_one_group(const Geom& g, const compkv_select_params* params, int* st) {
    const bool one = one_group_path(g, params->select_path, st);
    if (!one || params->select_path != COMPKV_SELECT_AUTO) return one;
    return !sx_shape(g, score_shape(g).nchunks, params->budget_blocks).one_round;
}

// The launch shape of compkv_decode_step (a COMPKV_SELECT_* value other than AUTO); *st receives the
// status. STREAM takes the two-launch step whenever it fits (AUTO does not: it measured slower);
// otherwise as CHUNKED.
int step_path(const Geom& g, const compkv_select_params* params, int* st) {
    const bool one = step_one_group(g, params, st);
    if (*st != COMPKV_OK) return 0;
    const int path = params->select_path;
    if (path == COMPKV_SELECT_STREAM &&
        stream_shape(g, params->budget_blocks, params->compensation == COMPKV_COMP_MEAN).fits)
        return COMPKV_SELECT_STREAM;
    if (one) return COMPKV_SELECT_ONE_GROUP;
    return use_select_exact(path, sx_shape(g, score_shape(g).nchunks, params->budget_blocks))
               ? COMPKV_SELECT_CHUNKED_EXACT
               : COMPKV_SELECT_CHUNKED;
}

// arrays the kernels read with 16-byte vector loads: null (checked separately) or 16-byte aligned
bool vec_aligned(std::initializer_list<const void*> ps) {
    for (const void* p : ps)
        if ((reinterpret_cast<uintptr_t>(p) & 15u) != 0) return false;
    return true;
}

int check_ws(const Geom& g, void* ws, size_t bytes, size_t need) {
    if (!ws || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0 || bytes < need) return COMPKV_EWORKSPACE;
    (void)g;
    return COMPKV_OK;
}

int launch_status(hipError_t e) { return e == hipSuccess ? COMPKV_OK : COMPKV_EHIP; }

// Scoring arguments with the score region at the start of the workspace.
compkv::ScoreArgs score_args(const Geom& g, const compkv_select_params* params, const void* q, const float* kmean,
                             const float* dvar, const int32_t* seq_lens, int32_t* sel, int32_t* n_sel,
                             float* blk_logit, float* scores, void* workspace) {
    const ScoreShape sh = score_shape(g);
    const size_t units = g.units(), xmax = g.xmax();
    compkv::ScoreArgs a{};
    char* p = static_cast<char*>(workspace);
    a.ws_part = reinterpret_cast<float*>(p);
    p += align_up(units * (sh.nchunks + 1) * g.G * 2 * sizeof(float));
    a.ws_w = reinterpret_cast<float*>(p);
    p += align_up(units * xmax * g.G * sizeof(float));
    a.ws_key = reinterpret_cast<uint32_t*>(p);
    p += align_up(units * xmax * sizeof(uint32_t));
    a.ws_qv = reinterpret_cast<float*>(p);
    a.zlog = blk_logit;
    a.zstride = g.xcap;
    a.q = static_cast<const uint16_t*>(q);
    a.kmean = kmean;
    a.dvar = dvar;
    a.seq_lens = seq_lens;
    a.sel = sel;
    a.n_sel = n_sel;
    a.blk_logit = blk_logit;
    a.scores = scores;
    a.bpc = sh.bpc;
    a.nchunks = sh.nchunks;
    a.K = params->budget_blocks;
    a.n_sink = params->n_sink;
    a.n_recent = params->n_recent;
    a.scale = params->scale;
    a.score_kind = params->score_kind;
    return a;
}

// The selection forms its score terms from zbar and the variances where these are fewer than the
// terms (r = 4 variances against G = 8 terms per block) and the keys fit the four-per-thread selection:
// the scoring launch then writes zbar alone (to blk_logit, or without it to the terms' region,
// [units][G][xmax]) and the query's group sums. (At G = 4 the reads would not shrink, and forming the
// terms in the selection lengthens it: measured 128K +1.8 us, 32K +1.1 us.)
void use_logit_terms(const Geom& g, compkv::ScoreArgs& a) {
    if (a.one_group || g.r != 4 || g.G != 8 || g.xmax() > 4096) return;
    a.logit_terms = 1;
    if (!a.zlog) {
        a.zlog = a.ws_w;
        a.zstride = g.xmax();
    }
}

constexpr int kMaxDevices = 64;
std::mutex scratch_mutex;
void* scratch_ptr[kMaxDevices];

// The current device's scratch address (nullptr: no device, too many devices, or the lookup failed).
void* device_scratch() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(scratch_mutex);
    if (!scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
            (void)hipGetLastError();
            return nullptr;
        }
        scratch_ptr[dev] = ptr;
    }
    return scratch_ptr[dev];
}

}  // namespace

extern "C" {

int compkv_version(void) { return 100; }

const char* compkv_status_string(int status) {
    switch (status) {
        case COMPKV_OK: return "COMPKV_OK";
        case COMPKV_EINVAL: return "COMPKV_EINVAL: null pointer or inconsistent dims";
        case COMPKV_EUNSUPPORTED: return "COMPKV_EUNSUPPORTED: head_dim, group size, block size or r not supported";
        case COMPKV_EBUDGET: return "COMPKV_EBUDGET: budget smaller than the mandatory set";
        case COMPKV_EWORKSPACE: return "COMPKV_EWORKSPACE: workspace null, misaligned or too small";
        case COMPKV_EHIP: return "COMPKV_EHIP: kernel launch failed";
        case COMPKV_ESCRATCH:
            return "COMPKV_ESCRATCH: the step needs more scratch than compkv_decode_step_noalloc holds "
                   "(use compkv_decode_step with a workspace)";
        default: return "unknown compkv status";
    }
}

size_t compkv_workspace_bytes(const compkv_dims* dims, int32_t budget_blocks, int32_t which) {
    Geom g;
    if (check_dims(dims, &g) != COMPKV_OK || budget_blocks < 1 || which < 0 || which > 4) return 0;
    return ws_bytes(g, budget_blocks, which);
}

int compkv_build_stats(const compkv_dims* dims, const void* k_cache, const void* v_cache,
                       const int32_t* seq_lens, float* kmean, float* dvar, float* vmean, void* stream) {
    Geom g;
    int st = check_dims(dims, &g);
    if (st != COMPKV_OK) return st;
    if (!k_cache || !v_cache || !seq_lens || !kmean || !dvar || !vmean) return COMPKV_EINVAL;
    if (!vec_aligned({k_cache, v_cache, kmean, dvar, vmean})) return COMPKV_EINVAL;
    compkv::StatsArgs a{};
    a.K = static_cast<const uint16_t*>(k_cache);
    a.V = static_cast<const uint16_t*>(v_cache);
    a.seq_lens = seq_lens;
    a.kmean = kmean;
    a.dvar = dvar;
    a.vmean = vmean;
    return launch_status(compkv::launch_build_stats(g, a, static_cast<hipStream_t>(stream)));
}

int compkv_append_stats(const compkv_dims* dims, void* k_cache, void* v_cache, const void* k_new,
                        const void* v_new, const int32_t* seq_lens, float* kmean, float* dvar,
                        float* vmean, void* stream) {
    Geom g;
    int st = check_dims(dims, &g);
    if (st != COMPKV_OK) return st;
    if (!k_cache || !v_cache || !k_new || !v_new || !seq_lens || !kmean || !dvar || !vmean) return COMPKV_EINVAL;
    if (!vec_aligned({k_cache, v_cache, k_new, v_new, kmean, dvar, vmean})) return COMPKV_EINVAL;
    compkv::StatsArgs a{};
    a.K = static_cast<const uint16_t*>(k_cache);
    a.V = static_cast<const uint16_t*>(v_cache);
    a.K_out = static_cast<uint16_t*>(k_cache);
    a.V_out = static_cast<uint16_t*>(v_cache);
    a.k_new = static_cast<const uint16_t*>(k_new);
    a.v_new = static_cast<const uint16_t*>(v_new);
    a.seq_lens = seq_lens;
    a.kmean = kmean;
    a.dvar = dvar;
    a.vmean = vmean;
    return launch_status(compkv::launch_append_stats(g, a, static_cast<hipStream_t>(stream)));
}

int compkv_score_select(const compkv_dims* dims, const compkv_select_params* params, const void* q,
                        const float* kmean, const float* dvar, const int32_t* seq_lens, int32_t* sel,
                        int32_t* n_sel, float* blk_logit, float* scores, void* workspace,
                        size_t workspace_bytes, void* stream) {
    Geom g;
    int st = check_dims(dims, &g);
    if (st != COMPKV_OK) return st;
    if (!params || !q || !kmean || !dvar || !seq_lens || !sel || !n_sel) return COMPKV_EINVAL;
    if (!vec_aligned({q, kmean, dvar})) return COMPKV_EINVAL;
    if (params->budget_blocks < 1 || params->n_sink < 0 || params->n_recent < 0) return COMPKV_EINVAL;
    if (params->budget_blocks < params->n_sink + params->n_recent) return COMPKV_EBUDGET;
    if (params->score_kind < COMPKV_SCORE_COMPKV || params->score_kind > COMPKV_SCORE_FIRST_ORDER) return COMPKV_EINVAL;
    const bool one = one_group_path(g, params->select_path, &st);
    if (st != COMPKV_OK) return st;
    if (!one && (score_shape(g).nchunks + 1) * g.G > compkv::select_max_chunk_heads()) return COMPKV_EUNSUPPORTED;
    const size_t need = ws_bytes(g, params->budget_blocks, COMPKV_WS_SCORE_SELECT);
    st = check_ws(g, workspace, workspace_bytes, need);
    if (st != COMPKV_OK) return st;
    void* body = static_cast<char*>(workspace) + state_bytes(g);
    compkv::ScoreArgs a = score_args(g, params, q, kmean, dvar, seq_lens, sel, n_sel, blk_logit, scores, body);
    a.one_group = one;
    use_logit_terms(g, a);
    return launch_status(compkv::launch_score_select(g, a, static_cast<hipStream_t>(stream)));
}

int compkv_sparse_decode(const compkv_dims* dims, float scale, const void* q, const void* k_cache,
                         const void* v_cache, const float* kmean, const float* vmean, const float* blk_logit,
                         const int32_t* seq_lens, const int32_t* sel, const int32_t* n_sel,
                         int32_t sel_stride, float* out, float* lse, void* workspace,
                         size_t workspace_bytes, void* stream) {
    Geom g;
    int st = check_dims(dims, &g);
    if (st != COMPKV_OK) return st;
    if (!q || !k_cache || !v_cache || !seq_lens || !sel || !n_sel || !out) return COMPKV_EINVAL;
    if (!vec_aligned({q, k_cache, v_cache, kmean, vmean})) return COMPKV_EINVAL;
    // Mean: vmean with blk_logit or kmean (zbar recomputed); Drop: vmean and blk_logit both null
    if (vmean ? (!blk_logit && !kmean) : blk_logit != nullptr) return COMPKV_EINVAL;
    if (sel_stride < 1) return COMPKV_EINVAL;
    const size_t need = ws_bytes(g, sel_stride, COMPKV_WS_SPARSE_DECODE);
    st = check_ws(g, workspace, workspace_bytes, need);
    if (st != COMPKV_OK) return st;
    const SparseShape sh = sparse_shape(g, sel_stride);
    if (sh.cb > compkv::decode_max_cb() || sh.eb > compkv::decode_max_eb()) return COMPKV_EUNSUPPORTED;
    char* base = static_cast<char*>(workspace) + state_bytes(g);
    compkv::DecodeArgs a{};
    a.ws_part = reinterpret_cast<float*>(base);
    a.q = static_cast<const uint16_t*>(q);
    a.K = static_cast<const uint16_t*>(k_cache);
    a.V = static_cast<const uint16_t*>(v_cache);
    a.vmean = vmean;
    a.blk_logit = blk_logit;
    a.kmean = kmean;
    a.seq_lens = seq_lens;
    a.sel = sel;
    a.n_sel = n_sel;
    a.out = out;
    a.lse = lse;
    a.sel_stride = sel_stride;
    a.n_exact = sh.n_exact;
    a.eb = sh.eb;
    a.n_comp = vmean ? sh.n_comp : 0;
    a.cb = sh.cb;
    a.dense = 0;
    a.scale = scale;
    return launch_status(compkv::launch_decode(g, a, static_cast<hipStream_t>(stream)));
}

int compkv_dense_decode(const compkv_dims* dims, float scale, const void* q, const void* k_cache,
                        const void* v_cache, const int32_t* seq_lens, float* out, float* lse,
                        void* workspace, size_t workspace_bytes, void* stream) {
    Geom g;
    int st = check_dims(dims, &g);
    if (st != COMPKV_OK) return st;
    if (!q || !k_cache || !v_cache || !seq_lens || !out) return COMPKV_EINVAL;
    if (!vec_aligned({q, k_cache, v_cache})) return COMPKV_EINVAL;
    const size_t need = ws_bytes(g, 1, COMPKV_WS_DENSE_DECODE);
    st = check_ws(g, workspace, workspace_bytes, need);
    if (st != COMPKV_OK) return st;
    const DenseShape sh = dense_shape(g);
    if (g.bpp > 0 && sh.te / (g.bpp * g.B) + 2 > compkv::decode_max_row_bases()) return COMPKV_EUNSUPPORTED;
    char* base = static_cast<char*>(workspace) + state_bytes(g);
    compkv::DecodeArgs a{};
    a.ws_part = reinterpret_cast<float*>(base);
    a.q = static_cast<const uint16_t*>(q);
    a.K = static_cast<const uint16_t*>(k_cache);
    a.V = static_cast<const uint16_t*>(v_cache);
    a.seq_lens = seq_lens;
    a.out = out;
    a.lse = lse;
    a.n_exact = sh.items;
    a.eb = sh.te;
    a.dense = 1;
    a.scale = scale;
    return launch_status(compkv::launch_decode(g, a, static_cast<hipStream_t>(stream)));
}

int compkv_host_cache_pointer(const void* host_ptr, void** device_ptr) {
    if (!host_ptr || !device_ptr) return COMPKV_EINVAL;
    *device_ptr = nullptr;
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, const_cast<void*>(host_ptr), 0) != hipSuccess || !d) {
        (void)hipGetLastError();  // clear the sticky error of the failed query
        return COMPKV_EINVAL;
    }
    *device_ptr = d;
    return COMPKV_OK;
}

int compkv_decode_step_path(const compkv_dims* dims, const compkv_select_params* params) {
    Geom g;
    int st = check_dims(dims, &g);
    if (st != COMPKV_OK) return st;
    if (!params) return COMPKV_EINVAL;
    const int path = step_path(g, params, &st);
    return st != COMPKV_OK ? st : path;
}

int compkv_decode_step(const compkv_dims* dims, const compkv_select_params* params, const void* q, void* k_cache,
                       void* v_cache, const void* k_new, const void* v_new, const int32_t* seq_lens, float* kmean,
                       float* dvar, float* vmean, int32_t* sel, int32_t* n_sel, float* blk_logit, float* scores,
                       float* out, float* lse, void* workspace, size_t workspace_bytes, void* stream) {
    Geom g;
    int st = check_dims(dims, &g);
    if (st != COMPKV_OK) return st;
    if (!params || !q || !k_cache || !v_cache || !seq_lens || !kmean || !dvar || !vmean || !sel || !n_sel ||
        !blk_logit || !out)
        return COMPKV_EINVAL;
    if ((k_new == nullptr) != (v_new == nullptr)) return COMPKV_EINVAL;
    if (!vec_aligned({q, k_cache, v_cache, k_new, v_new, kmean, dvar, vmean})) return COMPKV_EINVAL;
    if (params->budget_blocks < 1 || params->n_sink < 0 || params->n_recent < 0) return COMPKV_EINVAL;
    if (params->budget_blocks < params->n_sink + params->n_recent) return COMPKV_EBUDGET;
    if (params->score_kind < COMPKV_SCORE_COMPKV || params->score_kind > COMPKV_SCORE_FIRST_ORDER) return COMPKV_EINVAL;
    if (params->compensation != COMPKV_COMP_MEAN && params->compensation != COMPKV_COMP_DROP) return COMPKV_EINVAL;
    const bool drop = params->compensation == COMPKV_COMP_DROP;
    const int K = params->budget_blocks;
    const int path = step_path(g, params, &st);
    if (st != COMPKV_OK) return st;
    const bool one = path == COMPKV_SELECT_ONE_GROUP;
    const SparseShape sp = sparse_shape(g, K);
    const ScoreShape sc = score_shape(g);
    const int parts = step_partials(g, K);
    if (path != COMPKV_SELECT_STREAM) {
        if (sp.eb > compkv::decode_max_eb() || sp.n_exact > compkv::decode_max_items()) return COMPKV_EUNSUPPORTED;
        if (one ? sp.cb > compkv::decode_max_cb()
                : (parts > compkv::decode_max_partials() || (sc.nchunks + 1) * g.G > compkv::select_max_chunk_heads()))
            return COMPKV_EUNSUPPORTED;
    }
    st = check_ws(g, workspace, workspace_bytes, ws_bytes(g, K, COMPKV_WS_DECODE_STEP));
    if (st != COMPKV_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t* state = static_cast<uint32_t*>(workspace);
    void* wsb = static_cast<char*>(workspace) + state_bytes(g);
    const size_t wsb_bytes = workspace_bytes - state_bytes(g);

    compkv::ScoreArgs a = score_args(g, params, q, kmean, dvar, seq_lens, sel, n_sel, blk_logit, scores, wsb);
    a.k_new = static_cast<const uint16_t*>(k_new);
    a.v_new = static_cast<const uint16_t*>(v_new);
    a.Kc = static_cast<uint16_t*>(k_cache);
    a.Vc = static_cast<uint16_t*>(v_cache);
    a.kmean_w = kmean;
    a.dvar_w = dvar;
    a.vmean = vmean;
    a.one_group = one;
    compkv::DecodeArgs d{};
    d.q = static_cast<const uint16_t*>(q);
    d.K = static_cast<const uint16_t*>(k_cache);
    d.V = static_cast<const uint16_t*>(v_cache);
    d.vmean = vmean;
    d.blk_logit = blk_logit;
    d.seq_lens = seq_lens;
    d.sel = sel;
    d.n_sel = n_sel;
    d.out = out;
    d.lse = lse;
    d.sel_stride = K;
    d.scale = params->scale;
    d.sel_padded = 1;
    if (path == COMPKV_SELECT_STREAM) {
        // everything in one launch: scoring (with the append), selection, compensation stream, exact
        // items and merge, ordered by the per-unit words at the start of the workspace
        const StreamShape sh = stream_shape(g, K, !drop);
        if (!sh.fits || score_ws(g) + step_part_bytes(g, sh.parts) > wsb_bytes) return COMPKV_EWORKSPACE;  // sizing invariant
        d.ws_part = reinterpret_cast<float*>(static_cast<char*>(wsb) + score_ws(g));
        d.n_exact = sh.n_exact;
        d.eb = sh.eb;
        d.n_comp = sh.n_comp;
        d.cb = sh.cb;
        d.part_count = sh.parts;
        d.part_base = drop ? 0 : 1 + sh.n_comp;
        d.neg_pseudo = drop ? 0 : 1;
        use_logit_terms(g, a);
        return launch_status(compkv::launch_step_stream(g, a, d, state, s));
    }
    if (one) {
        // one workgroup per unit refreshes, scores and selects; then the compensated sparse decode
        // (exact and compensation items, merge) with its partials at the start of the workspace
        hipError_t e = compkv::launch_score_select(g, a, s);
        if (e != hipSuccess) return COMPKV_EHIP;
        d.ws_part = static_cast<float*>(wsb);
        d.q = static_cast<const uint16_t*>(q);
        d.K = static_cast<const uint16_t*>(k_cache);
        d.V = static_cast<const uint16_t*>(v_cache);
        d.vmean = vmean;
        d.blk_logit = blk_logit;
        d.seq_lens = seq_lens;
        d.sel = sel;
        d.n_sel = n_sel;
        d.out = out;
        d.lse = lse;
        d.sel_stride = K;
        d.n_exact = sp.n_exact;
        d.eb = sp.eb;
        d.n_comp = drop ? 0 : sp.n_comp;
        d.cb = sp.cb;
        d.dense = 0;
        d.scale = params->scale;
        d.sel_padded = 1;
        return launch_status(compkv::launch_decode(g, d, s));
    }
    // chunked scoring; then either the selection and the exact items as two launches, or
    // (CHUNKED_EXACT, or AUTO when every item workgroup is resident at once) one fused launch
    use_logit_terms(g, a);
    const SxShape sx = sx_shape(g, sc.nchunks, K);
    const bool use_sx = use_select_exact(params->select_path, sx);
    if (use_sx) {
        // the chunks score from the mean keys and variances alone; the fused launch's compensation
        // workgroups stream the mean values while its item workgroups select, and the last of each
        // unit's workgroups merges the unit's partials
        // (all workgroups resident at once: one selector per unit, the others stream the mean values
        // and then attend over their share of its ids)
        float* dpart = reinterpret_cast<float*>(static_cast<char*>(wsb) + score_ws(g));
        const bool work = sx.work;
        const int n_comp = drop ? 0 : (work ? sx.P - 1 : sx.n_comp);
        const int nparts = work ? sx.P : n_comp + sx.n_exact;
        const size_t part_bytes = step_part_bytes(g, step_partials(g, K));
        uint32_t* arrive = reinterpret_cast<uint32_t*>(static_cast<char*>(wsb) + score_ws(g) + part_bytes);
        if (step_part_bytes(g, nparts) > part_bytes || step_ws(g, K) > wsb_bytes)
            return COMPKV_EWORKSPACE;  // sizing invariant
        a.arrive_zero = arrive;
        a.trace = g_trace_chunks;
        a.comp_part = nullptr;
        a.part_count = nparts;
        a.chunks_only = 1;
        hipError_t e = compkv::launch_score_select(g, a, s);
        if (e != hipSuccess) return COMPKV_EHIP;
        d.ws_part = dpart;
        d.q = static_cast<const uint16_t*>(q);
        d.K = static_cast<const uint16_t*>(k_cache);
        d.V = static_cast<const uint16_t*>(v_cache);
        d.vmean = vmean;
        d.blk_logit = blk_logit;
        d.seq_lens = seq_lens;
        d.sel = sel;
        d.n_sel = n_sel;
        d.out = out;
        d.lse = lse;
        d.sel_stride = K;
        d.n_exact = work ? sx.P : sx.n_exact;
        d.eb = work ? sx.web : sx.eb;
        d.n_comp = n_comp;
        d.cb = work ? sx.wcb : sx.cb;
        d.dense = 0;
        d.scale = params->scale;
        d.part_count = nparts;
        d.part_base = work ? 0 : n_comp;
        d.neg_pseudo = drop ? 0 : 1;
        d.sel_padded = 1;
        d.arrive = arrive;
        d.sel_word = arrive + g.units();
        d.mailbox = arrive + 2 * (size_t)g.units();
        d.timeouts = state;
        d.trace = g_trace_fused;
        a.trace = g_trace_fused;  // (the selection's marks, in the fused launch's records)
        if (work) return launch_status(compkv::launch_select_work(g, a, d, sx.P, s));
        return launch_status(compkv::launch_select_exact(g, a, d, sx.n_exact, s));
    }
    // separate selection and exact items. Mean: the chunks' compensation partials, then the exact
    // items' partials; Drop: exact items only
    const int n_ex = sp.n_exact;
    float* dpart = reinterpret_cast<float*>(static_cast<char*>(wsb) + score_ws(g));
    const int nparts = drop ? n_ex : sc.nchunks + 1 + n_ex;
    if (score_ws(g) + step_part_bytes(g, nparts) > wsb_bytes) return COMPKV_EWORKSPACE;  // sizing invariant
    a.comp_part = drop ? nullptr : dpart;
    a.part_count = nparts;
    a.chunks_only = 0;
    hipError_t e = compkv::launch_score_select(g, a, s);
    if (e != hipSuccess) return COMPKV_EHIP;

    d.ws_part = dpart;
    d.q = static_cast<const uint16_t*>(q);
    d.K = static_cast<const uint16_t*>(k_cache);
    d.V = static_cast<const uint16_t*>(v_cache);
    d.vmean = vmean;
    d.blk_logit = blk_logit;
    d.seq_lens = seq_lens;
    d.sel = sel;
    d.n_sel = n_sel;
    d.out = out;
    d.lse = lse;
    d.sel_stride = K;
    d.n_exact = n_ex;
    d.eb = sp.eb;
    d.n_comp = 0;
    d.cb = 0;
    d.dense = 0;
    d.scale = params->scale;
    d.part_count = nparts;
    d.part_base = drop ? 0 : sc.nchunks + 1;
    d.neg_pseudo = drop ? 0 : 1;
    d.sel_padded = 1;
    e = compkv::launch_decode_items(g, d, n_ex, s);
    if (e != hipSuccess) return COMPKV_EHIP;
    return launch_status(compkv::launch_decode_merge(g, d, nparts, s));
}

int compkv_phase_trace_set(void* chunk_records, void* fused_records) {
#ifdef COMPKV_PHASE_TRACE
    g_trace_chunks = static_cast<unsigned long long*>(chunk_records);
    g_trace_fused = static_cast<unsigned long long*>(fused_records);
    return COMPKV_OK;
#else
    (void)chunk_records;
    (void)fused_records;
    return COMPKV_EUNSUPPORTED;
#endif
}

size_t compkv_decode_step_noalloc_limit(void) { return kScratchBytes; }

int compkv_decode_step_noalloc(const compkv_dims* dims, const compkv_select_params* params, const void* q,
                               void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                               const int32_t* seq_lens, float* kmean, float* dvar, float* vmean, int32_t* sel,
                               int32_t* n_sel, float* blk_logit, float* scores, float* out, float* lse,
                               void* stream) {
    Geom g;
    int st = check_dims(dims, &g);
    if (st != COMPKV_OK) return st;
    if (!params || params->budget_blocks < 1) return COMPKV_EINVAL;
    if (ws_bytes(g, params->budget_blocks, COMPKV_WS_DECODE_STEP) > kScratchBytes) return COMPKV_ESCRATCH;
    void* ws = device_scratch();
    if (!ws) return COMPKV_EHIP;
    return compkv_decode_step(dims, params, q, k_cache, v_cache, k_new, v_new, seq_lens, kmean, dvar, vmean, sel,
                              n_sel, blk_logit, scores, out, lse, ws, kScratchBytes, stream);
}

}  // extern "C"

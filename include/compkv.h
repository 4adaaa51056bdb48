/*
 * compkv.h -- C ABI of the MI355X (gfx950) CompKV decode-step attention library (libcompkv.so).
 *
 * CompKV (compensation-aware KV selection) decodes one token per sequence. Each KV head of each
 * sequence (a "unit") is shared by G = n_q_heads / n_kv_heads query heads (Section 3.1). The cache is
 * split into contiguous blocks of block_size tokens from the first token; the last block may be
 * partial (Section 3.1). For every block the library keeps a summary: mean key, mean value and r
 * grouped key variances (Sections 4.1 and 4.2). A decode step scores every block from the summaries
 * (Eqs. grouped-variance-metadata, compkv-mass-estimate, compkv-score), selects the mandatory blocks
 * plus the best-scoring others up to the budget (Eq. compkv-selected-set), then attends exactly over
 * the selected blocks and through one mean pseudo-token per omitted block (Eq. compkv-output).
 *
 * Conventions shared by every call:
 *  - Every pointer argument is a DEVICE pointer allocated and owned by the caller. The library never
 *    allocates, frees or synchronizes, and never reads device memory from the host. Every call only
 *    validates its host-side arguments and enqueues work on `stream` (a hipStream_t; NULL means the
 *    default stream). Results are ready when the stream reaches that point.
 *  - Layouts (row-major, innermost last). d = head_dim, Xcap = ceil(capacity_tokens / block_size):
 *      k_cache, v_cache  bf16 [batch][n_kv_heads][capacity_tokens][d] (or paged, see compkv_dims)
 *      q                 bf16 [batch][n_q_heads][d]; query head hq uses KV head hq / G
 *      kmean, vmean      fp32 [batch][n_kv_heads][Xcap][d]
 *      dvar              fp32 [batch][n_kv_heads][Xcap][n_var_groups]
 *      seq_lens          int32 [batch]: tokens present per sequence (device memory). Values above
 *                        max_seq_len are treated as max_seq_len and values below 0 as 0, so a bad
 *                        length can never address memory outside the buffers described here
 *      sel               int32 [batch][n_kv_heads][budget_blocks], n_sel int32 [batch][n_kv_heads]
 *      blk_logit         fp32 [batch][n_kv_heads][G][Xcap]: block-mean logits s q_g . kmean_b
 *      scores            fp32 [batch][n_kv_heads][Xcap]
 *      out               fp32 [batch][n_q_heads][d]; lse fp32 [batch][n_q_heads] (natural log)
 *  - bf16 values are passed as their 16-bit patterns. Inputs must be finite.
 *  - q, k_cache, v_cache, k_new, v_new, kmean, dvar and vmean are read with 16-byte vector loads: each
 *    must be 16-byte aligned (any device allocation is); a misaligned one is COMPKV_EINVAL.
 *  - workspace: device scratch of at least compkv_workspace_bytes(...) bytes, 256-byte aligned. Its
 *    first 16 * batch * n_kv_heads bytes, rounded up to 256, are per-unit words of the STREAM step
 *    (below): they must be zero before a workspace's first compkv_decode_step on that path (zero the
 *    whole workspace once after allocating it); every such step leaves them zero, and no other call
 *    writes them. The rest needs no initial contents. Each call that takes one enqueues two kernels
 *    (compkv_decode_step: up to four), each reading what the previous one wrote there. Calls that may
 *    run concurrently need distinct workspaces.
 *  - Return value: COMPKV_OK (0) or a negative status; compkv_status_string() names it. On error
 *    nothing has been enqueued, except for COMPKV_EHIP (a launch failed).
 *
 * Supported shapes: head_dim in {64, 128}; G in {1, 2, 4, 8}; 1 <= block_size <= 1024; n_var_groups
 * r dividing head_dim / 2, or r == head_dim.
 */
#ifndef COMPKV_H
#define COMPKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define COMPKV_OK 0
#define COMPKV_EINVAL (-1)      /* null required pointer, inconsistent dims or sizes */
#define COMPKV_EUNSUPPORTED (-2) /* head_dim, G, block_size or n_var_groups outside the supported set */
#define COMPKV_EBUDGET (-3)     /* budget smaller than the mandatory set n_sink + n_recent */
#define COMPKV_EWORKSPACE (-4)  /* workspace null, misaligned or too small */
#define COMPKV_EHIP (-5)        /* a kernel launch failed */
#define COMPKV_ESCRATCH (-6)    /* compkv_decode_step_noalloc: the step needs more than its fixed scratch */

/* Coordinate groups of the grouped key variance (Appendix A.4): the d coordinates form d/2 RoPE
 * frequency pairs, cut into r equal consecutive groups with both coordinates of a pair together.
 * ROTATE_HALF pairs coordinate f with f + d/2 (the layout of the paper's models); INTERLEAVED pairs
 * 2f with 2f + 1. With r == d every coordinate is its own group t = {t}. */
#define COMPKV_GROUPS_ROTATE_HALF 0
#define COMPKV_GROUPS_INTERLEAVED 1

typedef struct compkv_dims {
    int32_t batch;           /* sequences */
    int32_t n_q_heads;       /* query heads per sequence */
    int32_t n_kv_heads;      /* KV heads per sequence; must divide n_q_heads */
    int32_t head_dim;        /* d */
    int32_t block_size;      /* B, tokens per block (Section 3.1) */
    int32_t n_var_groups;    /* r, grouped variances per block (Section 4.1) */
    int32_t group_layout;    /* COMPKV_GROUPS_* */
    int32_t capacity_tokens; /* cache rows per unit (row stride of k_cache / v_cache) */
    int32_t max_seq_len;     /* host-side upper bound of seq_lens, 1..capacity_tokens; sizes grids */
    /* Paged cache (all zero: the contiguous layout above). With page_tokens > 0, a multiple of
     * block_size, k_cache and v_cache are bf16 [num_pages][n_kv_heads][page_tokens][d], and token j of
     * sequence b lives in page block_table[b][j / page_tokens] at row j % page_tokens. block_table is a
     * device int32 [batch][pages_per_seq] (entries outside [0, num_pages) are clamped, so a bad table
     * reads the wrong page but never outside the cache); capacity_tokens must equal
     * pages_per_seq * page_tokens. Summaries, selections and outputs keep their per-sequence layouts. */
    int32_t page_tokens;
    int32_t num_pages;
    int32_t pages_per_seq;
    const int32_t* block_table;
} compkv_dims;

typedef struct compkv_select_params {
    int32_t budget_blocks; /* K: blocks read exactly per unit, mandatory blocks included (Eq. compkv-selected-set) */
    int32_t n_sink;        /* leading blocks always selected (the paper uses 1; Section 4.2) */
    int32_t n_recent;      /* most recent blocks always selected (the paper uses 2; Section 4.2) */
    float scale;           /* logit scale s; the paper's 1/sqrt(d) (Section 3.1) */
    int32_t select_path;   /* COMPKV_SELECT_*: how the scores are formed and ranked (0 = automatic) */
    int32_t score_kind;    /* COMPKV_SCORE_*: the block score (0 = the CompKV score) */
    int32_t compensation;  /* COMPKV_COMP_*: what stands in for the omitted blocks in
                              compkv_decode_step (0 = Mean compensation) */
} compkv_select_params;

/*
 * Block scores (compkv_select_params.score_kind): the paper's score and the variants of its
 * ablations (Section 5.4). p-hat is normalized per query head over every block in all three.
 *   COMPKV:      S_b = sum_g p-hat_{g,b} sigma-hat^2_{g,b}, p-hat from log|b| + zbar + sigma-hat^2/2
 *                (Eqs. compkv-mass-estimate, compkv-score).
 *   MASS:        S_b = sum_g p-hat_{g,b} (the second-order mass estimate alone).
 *   FIRST_ORDER: S_b = sum_g p-hat_{g,b} sigma-hat^2_{g,b} with p-hat from log|b| + zbar alone.
 * Decoding of the omitted blocks (compkv_select_params.compensation):
 *   MEAN: one pseudo-token per omitted block (Eq. compkv-output).
 *   DROP: omitted blocks are left out; attention is renormalized over the selected tokens
 *         (Appendix A.5).
 */
#define COMPKV_SCORE_COMPKV 0
#define COMPKV_SCORE_MASS 1
#define COMPKV_SCORE_FIRST_ORDER 2
#define COMPKV_COMP_MEAN 0
#define COMPKV_COMP_DROP 1

/*
 * Scoring / selection launch shapes (compkv_select_params.select_path). Both compute the same
 * quantities; their floating-point sums run in different orders, so scores may differ in the last
 * bits and selections only among blocks whose scores tie within that rounding.
 *   CHUNKED:   chunks of blocks spread over many workgroups, then one workgroup per unit merges the
 *              per-chunk normalizers and selects (two launches).
 *   ONE_GROUP: one workgroup per unit scores every block and selects (one launch); needs
 *              G * ceil(max_seq_len / block_size) <= 8192, else COMPKV_EUNSUPPORTED.
 *   CHUNKED_EXACT: CHUNKED scoring; in compkv_decode_step the selection and the exact attention over
 *              the selected blocks then run as one launch (each of a unit's workgroups repeats the
 *              unit's selection and attends over its share of the blocks), when the budget is at most
 *              1024 blocks and a unit at most 8192 blocks; otherwise, and in compkv_score_select, as
 *              CHUNKED.
 *   STREAM:    in compkv_decode_step, two launches: the scoring of every completed block (the
 *              CHUNKED chunks, bit-identical scores) with the refreshed last block, then one launch in
 *              which one selector per unit ranks the blocks while compensation workgroups stream the
 *              mean values, and exact workgroups wait for their unit's ids (a bounded wait on a
 *              per-unit word of the workspace; a wait that times out makes the unit's outputs NaN);
 *              the unit's last workgroup merges. When the budget is at most 1024 blocks and a unit at
 *              most 8192 blocks; otherwise, and in compkv_score_select, as CHUNKED.
 *   AUTO:      in compkv_score_select, ONE_GROUP when a unit holds at most 256 blocks (one workgroup
 *              then reads every summary in a single round of loads), else CHUNKED. In
 *              compkv_decode_step, CHUNKED_EXACT when all of its workgroups are resident at once (at
 *              most one per compute unit), else ONE_GROUP when a unit holds at most 256 blocks, else
 *              CHUNKED.
 */
#define COMPKV_SELECT_AUTO 0
#define COMPKV_SELECT_CHUNKED 1
#define COMPKV_SELECT_ONE_GROUP 2
#define COMPKV_SELECT_CHUNKED_EXACT 3
#define COMPKV_SELECT_STREAM 4

/* Which call a workspace is sized for (compkv_workspace_bytes). */
#define COMPKV_WS_ALL 0
#define COMPKV_WS_SCORE_SELECT 1
#define COMPKV_WS_SPARSE_DECODE 2
#define COMPKV_WS_DENSE_DECODE 3
#define COMPKV_WS_DECODE_STEP 4

/*
 * Block summaries of the first seq_lens[b] tokens of every unit (prefill). Section 4.1, Eq.
 * grouped-variance-metadata, and Section 4.2: for block b with |b| tokens,
 *   kmean[b] = mean key, vmean[b] = mean value,
 *   dvar[b][t] = (1 / (|b| |G_t|)) sum_{j in b} sum_{i in G_t} (k_{j,i} - kmean[b][i])^2
 * (population variances, Appendix E.1). Blocks at or past ceil(seq_lens[b] / B) are not written.
 */
int compkv_build_stats(const compkv_dims* dims, const void* k_cache, const void* v_cache,
                       const int32_t* seq_lens, float* kmean, float* dvar, float* vmean, void* stream);

/*
 * Streaming append (Section 4.2, Appendix E.1): writes the new token's key and value (bf16
 * [batch][n_kv_heads][d] each) into cache row n = seq_lens[b] -- the length BEFORE the append;
 * seq_lens is not modified -- and refreshes the summary of the active block n / B only (completed
 * blocks never change). The refreshed summary is bit-identical to what compkv_build_stats computes
 * for n + 1 tokens. Units whose n is not below capacity_tokens are left untouched.
 */
int compkv_append_stats(const compkv_dims* dims, void* k_cache, void* v_cache, const void* k_new,
                        const void* v_new, const int32_t* seq_lens, float* kmean, float* dvar,
                        float* vmean, void* stream);

/*
 * Scoring and selection (Sections 4.1 and 4.2). Per unit and block b, with s = params->scale:
 *   zbar[g][b] = s q_g . kmean_b,   sig2[g][b] = s^2 sum_t (sum_{i in G_t} q_{g,i}^2) dvar[b][t],
 *   phat[g][b] = |b| exp(zbar + sig2/2) / sum_c |c| exp(zbar_c + sig2_c/2)   (per query head, all blocks)
 *   S_b = sum_g phat[g][b] sig2[g][b]
 * then S = F u TopK_{K-|F|}{S_b : b not in F}, F = first n_sink and last n_recent blocks (overlap
 * counted once). Ties rank the lower block id first; sel lists the ids in ascending order and
 * n_sel[u] = min(K, X); slots past n_sel are set to -1. If K >= X every block is selected.
 * blk_logit (nullable) receives zbar, which compkv_sparse_decode can take instead of recomputing it;
 * scores (nullable) receives S_b for every block. q is bf16 [batch][n_q_heads][d]. Returns COMPKV_EBUDGET if K < n_sink + n_recent and
 * COMPKV_EUNSUPPORTED when a unit can hold more than 128 * (4096 / G - 1) blocks
 * (ceil(max_seq_len / block_size)).
 */
int compkv_score_select(const compkv_dims* dims, const compkv_select_params* params, const void* q,
                        const float* kmean, const float* dvar, const int32_t* seq_lens, int32_t* sel,
                        int32_t* n_sel, float* blk_logit, float* scores, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * Compensated sparse decode (Eq. compkv-output). For every unit and query head g:
 *   out_g = [ sum_{b in S} sum_{j in b} e^{z_{g,j}} v_j + sum_{b not in S} |b| e^{zbar_{g,b}} vmean_b ]
 *         / [ sum_{b in S} sum_{j in b} e^{z_{g,j}}     + sum_{b not in S} |b| e^{zbar_{g,b}} ]
 * with z_{g,j} = scale q_g . k_j, S = sel[u][0 .. n_sel[u]) (ascending, unique ids below X; entries
 * outside [0, X) are ignored) and zbar_{g,b} = scale q_g . kmean_b. zbar is read from blk_logit as
 * written by compkv_score_select when blk_logit is given; with blk_logit NULL it is recomputed from
 * kmean (then required). sel_stride is the row stride of sel (the budget K). lse (nullable) receives
 * the log of the denominator, i.e. of the compensated normalizer. With vmean and blk_logit both NULL
 * the omitted blocks are left out (the Drop decode of Appendix A.5: out_g is attention over the
 * selected tokens alone; kmean is ignored); a unit with nothing selected then gets out = 0 and
 * lse = -inf. COMPKV_EINVAL: vmean given without blk_logit or kmean, or blk_logit without vmean.
 */
int compkv_sparse_decode(const compkv_dims* dims, float scale, const void* q, const void* k_cache,
                         const void* v_cache, const float* kmean, const float* vmean, const float* blk_logit,
                         const int32_t* seq_lens, const int32_t* sel, const int32_t* n_sel,
                         int32_t sel_stride, float* out, float* lse, void* workspace,
                         size_t workspace_bytes, void* stream);

/*
 * Dense decode over every cached token (full attention of Section 3.1, the speedup baseline):
 * out_g = softmax_j(scale q_g . k_j) V, lse_g = log sum_j e^{z_{g,j}} (lse nullable).
 */
int compkv_dense_decode(const compkv_dims* dims, float scale, const void* q, const void* k_cache,
                        const void* v_cache, const int32_t* seq_lens, float* out, float* lse,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * One whole decode step of one layer (Section 4.2 and Appendix E.1 in a single call): optional
 * streaming append, scoring, selection and compensated sparse decode, with the results of the
 * separate calls:
 *  - seq_lens holds the lengths AFTER the new token (n = seq_lens[b] >= 1 per sequence). If k_new and
 *    v_new are given (bf16 [batch][n_kv_heads][d], both or neither), row n - 1 of every unit is
 *    stored from them and the summary of its block (n - 1) / B is refreshed, bit-identical to
 *    compkv_append_stats with length n - 1. Units with n == 0 append nothing, and so do units with
 *    n > max_seq_len (their cache rows and summaries are left untouched; like every call, the step
 *    then scores and decodes them over max_seq_len tokens).
 *  - sel, n_sel, blk_logit and scores (nullable) are bit-identical to compkv_score_select on the
 *    refreshed summaries (sel has row stride params->budget_blocks).
 *  - out and lse (nullable) follow Eq. compkv-output as in compkv_sparse_decode (same tolerance, not
 *    bitwise: on the chunked path the pseudo-token sum is formed over all blocks while the summaries
 *    are streamed, and the selected blocks' pseudo-terms are then taken back out). With
 *    params->compensation == COMPKV_COMP_DROP they are the Drop decode of compkv_sparse_decode.
 *  - params->score_kind and params->select_path as for compkv_score_select.
 * Enqueues four kernels on the chunked path, three on the one-group and chunked-exact paths. Workspace:
 * compkv_workspace_bytes(dims, budget, COMPKV_WS_DECODE_STEP). Returns COMPKV_EUNSUPPORTED for shapes
 * whose partial count exceeds the merge limit (then use the separate calls), COMPKV_EINVAL for an
 * unknown compensation, otherwise the statuses of compkv_score_select.
 */
int compkv_decode_step(const compkv_dims* dims, const compkv_select_params* params, const void* q,
                       void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                       const int32_t* seq_lens, float* kmean, float* dvar, float* vmean, int32_t* sel,
                       int32_t* n_sel, float* blk_logit, float* scores, float* out, float* lse,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * compkv_decode_step for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same step, arguments and results, with
 * no workspace argument. Its scratch is a fixed device array of compkv_decode_step_noalloc_limit()
 * bytes (32 MiB) inside the library, one per GPU, held until the process ends; the call allocates and
 * frees nothing. Returns COMPKV_ESCRATCH when compkv_workspace_bytes(dims, budget,
 * COMPKV_WS_DECODE_STEP) exceeds that size (use compkv_decode_step with a workspace then), and
 * COMPKV_EHIP when the scratch's device address cannot be obtained. The scratch needs no initial
 * contents and keeps whatever the last call left; every call on one GPU uses the same scratch, so
 * calls that may overlap on one GPU (concurrent streams or threads) race and must be serialized by
 * the caller.
 */
int compkv_decode_step_noalloc(const compkv_dims* dims, const compkv_select_params* params, const void* q,
                               void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                               const int32_t* seq_lens, float* kmean, float* dvar, float* vmean, int32_t* sel,
                               int32_t* n_sel, float* blk_logit, float* scores, float* out, float* lse,
                               void* stream);

/* Bytes of the fixed scratch behind compkv_decode_step_noalloc. */
size_t compkv_decode_step_noalloc_limit(void);

/*
 * Phase trace of compkv_decode_step (for measurement; a library built with -DCOMPKV_PHASE_TRACE, which
 * paper_2609_26300_amd/build.py writes as libcompkv_trace.so): on the chunked-exact launch shape, thread 0
 * of every workgroup of the chunk-scoring launch and of the fused selection/exact launch stores the GPU's
 * 100 MHz real-time counter at its phase boundaries, and its role, into 16 64-bit words per workgroup
 * (workgroup w at words 16 w .. 16 w + 15; the slot meanings are listed beside each kernel). chunk_records
 * and fused_records are device arrays of at least 16 words per workgroup of the respective launch, written
 * by every later compkv_decode_step until this is called again with null pointers (which stops the
 * trace). The caller owns the arrays and keeps them alive while traced steps run. Returns COMPKV_OK, or
 * COMPKV_EUNSUPPORTED from a library built without the trace (its kernels hold no marks).
 */
int compkv_phase_trace_set(void* chunk_records, void* fused_records);

/* The launch shape compkv_decode_step takes for these dims and params on the current device:
 * COMPKV_SELECT_ONE_GROUP, COMPKV_SELECT_CHUNKED or COMPKV_SELECT_CHUNKED_EXACT (params->select_path
 * resolved), or a negative status (invalid dims or path). Enqueues nothing. */
int compkv_decode_step_path(const compkv_dims* dims, const compkv_select_params* params);

/*
 * Offload tier (Appendix E.1 keeps the cache in host memory): k_cache and v_cache may live in pinned,
 * device-mapped host memory (hipHostMalloc). This returns the device address of such an allocation in
 * *device_ptr, to be passed as k_cache / v_cache to any call; the kernels then read the rows they need
 * (the selected blocks, the active block) and write appended rows across the host link, with no
 * staging copy. The summaries (kmean, dvar, vmean) may be placed there the same way (the paper keeps
 * both in host memory); every step then also streams them across the link. Selections, outputs and
 * workspace stay in device memory. Returns COMPKV_EINVAL for null arguments or memory that is not
 * pinned and mapped.
 */
int compkv_host_cache_pointer(const void* host_ptr, void** device_ptr);

/* Workspace bytes needed by `which` (COMPKV_WS_*; COMPKV_WS_ALL = enough for every call) for these
 * dims and budget. The fused step's launch shape follows the compute-unit count of the current device:
 * query with the device that runs the calls current (a call given too small a workspace returns
 * COMPKV_EWORKSPACE). Returns 0 if dims are invalid. */
size_t compkv_workspace_bytes(const compkv_dims* dims, int32_t budget_blocks, int32_t which);

/* Static string naming a status code. */
const char* compkv_status_string(int status);

/* Library ABI version (major * 100 + minor). */
int compkv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* COMPKV_H */

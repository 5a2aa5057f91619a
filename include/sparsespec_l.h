/*
 * sparsespec_l.h -- C ABI of the MI355X (gfx950) hot path of SparseSpec-L's
 * self-speculative decode step ("A Sparse Glimpse of the Whole: Train-Free
 * Self-Speculative Decoding").
 *
 * One decode iteration of the method (Sec. 3.1) drafts tokens with attention
 * over a sparse, recallable view of the KV cache and verifies them with one
 * dense attention pass whose attention weights are recycled into per-head
 * importance scores.  For one layer this library provides:
 *
 *   ssl_verify_attn   dense verify attention of the k+1 verify rows over the
 *                     whole cache, emitting the Eq. 3 importance scores in the
 *                     same call (Sec. 3.1, Sec. 3.2 Eq. 3);
 *   ssl_select_topb   the Eq. 4 index set: sink, top-K_mid of the middle span
 *                     by score, recent (Sec. 3.2);
 *   ssl_draft_attn    draft-step attention over the K/V rows the index set
 *                     names, gathered on the fly (Sec. 3.2 Eq. 5);
 *   ssl_ctrl_*        the host-side adaptive speculation-length controller
 *                     (Sec. 3.3 Eq. 6-8); scalar, never touches the GPU.
 *
 * Conventions shared by every GPU entry point
 * -------------------------------------------
 *  - Tensors are caller-owned device buffers.  Element types: bf16 for q, k,
 *    v and q_draft; fp32 for scores; int32 for indices; outputs bf16 or fp32
 *    (ssl_params.out_fp32).
 *  - Layouts (row-major, innermost last; head_dim must be 128):
 *      q        [batch][max_q][n_q_heads][128]   verify rows of each sequence
 *      k, v     [batch][n_kv_heads][max_ctx][128] dense cache, head-major
 *      out      [batch][max_q][n_q_heads][128]   verify output
 *      scores   [batch][n_kv_heads][max_ctx]     Eq. 3 importance
 *      idx      [batch][n_kv_heads][budget]      Eq. 4 index sets
 *      n_idx    [batch]
 *      q_draft  [batch][n_q_heads][128], draft out the same
 *  - ctx_len[b] counts the cached tokens of sequence b *including* its
 *    q_len[b] verify rows, which occupy positions ctx_len-q_len .. ctx_len-1.
 *    Verify row j attends to keys 0 .. ctx_len-q_len+j (causal, bottom-right
 *    aligned).  Query head h reads KV head h / (n_q_heads / n_kv_heads).
 *  - Scores are kept per KV head: the attention probability a key receives,
 *    summed over the query heads sharing that KV head and over the last
 *    min(window, q_len) verify rows.  Rows of each sequence therefore sum to
 *    min(window, q_len) * (n_q_heads / n_kv_heads).
 *  - Host arrays (ctx_len, q_len, n_idx_host) are read during the call only.
 *  - The workspace is caller-allocated device memory of at least the size the
 *    matching *_workspace function reports; its contents need no
 *    initialization.  Every workspace layout starts with the same 64 KiB of
 *    exchange epochs (8192 words, one per exchange group: KV-head unit or
 *    logit row), which calls made under graph capture keep between replays
 *    and only ever advance; no call stores anything else there, so calls may
 *    share a workspace, captured or not.
 *  - Calls are asynchronous on `stream`; the library allocates nothing and
 *    synchronizes only in ssl_exchange_status.  Two calls that share a
 *    workspace must be ordered on one stream.
 *  - Process state kept by the library: a 64-bit call-tag sequence (host),
 *    per device the CU count, the one-sweep verify kernel's raised LDS limit
 *    and its occupancy (host, read once), the CU budget of ssl_set_cu_budget
 *    and the settings of ssl_test_exchange_faults (host), and one exchange
 *    status word per device (device memory, see ssl_exchange_status).
 *  - Calls may be captured in a HIP graph and the graph replayed any number
 *    of times, also with new contents in the captured input buffers: a call
 *    that finds its stream capturing has its kernels' cross-workgroup
 *    exchanges take a new tag on every replay from the workspace's epochs.
 *    A captured call with more than 8192 exchange groups is refused
 *    (SSL_ERR_UNSUPPORTED).  No call records a memset or an allocation.
 *  - Kernels whose workgroups exchange partial results (one-sweep verify,
 *    one-kernel select, draft and draft steps, logit statistics) wait for
 *    each other with bounded polls.  The plans keep every group that must be
 *    resident at once within half of what the device's CUs hold (see
 *    ssl_set_cu_budget).  A wait that still gives up (e.g. because other work
 *    held CUs) leaves that call's results unspecified and raises a bit of the
 *    device's exchange status word (ssl_exchange_status); under capture it
 *    also marks the group's epoch, and every later captured call on that
 *    workspace then gives up at once (raising the bit again) until the
 *    workspace is filled with zeros.
 *  - Every argument check happens on the host before any HIP call, so a
 *    rejected call has no effect on the device.  Device-side data (scores,
 *    idx) is not validated: index values outside [0, max_ctx) are clamped
 *    (results are then meaningless but memory stays in bounds).
 *  - Limits: head_dim 128; 1 <= batch <= 64; max_q <= 64; group <= 64 for
 *    verify (more than 64 rows per KV head, q_len * group > 64, run the
 *    two-sweep schedule once per block of 64 / group positions);
 *    n_q_heads / n_kv_heads <= 16 for the draft call.
 */
#ifndef SPARSESPEC_L_H
#define SPARSESPEC_L_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes: every entry point returns one; no exception crosses the ABI. */
enum {
    SSL_OK = 0,
    SSL_ERR_NULL = -1,        /* a required pointer is NULL */
    SSL_ERR_SHAPE = -2,       /* inconsistent sizes (see each call) */
    SSL_ERR_UNSUPPORTED = -3, /* valid request outside the limits the library is built for */
    SSL_ERR_BUDGET = -4,      /* budget < 1, k_sink/k_recent < 0 or k_sink + k_recent > budget */
    SSL_ERR_ALIGN = -5,       /* device pointer not 16-byte (tensors) / 4-byte (int, fp32) aligned */
    SSL_ERR_WORKSPACE = -6,   /* workspace NULL or smaller than required */
    SSL_ERR_HIP = -7          /* a HIP call failed (ssl_last_hip_error names it) */
};

typedef struct {
    int32_t batch;       /* sequences */
    int32_t n_q_heads;   /* query heads; a multiple of n_kv_heads */
    int32_t n_kv_heads;  /* KV heads */
    int32_t head_dim;    /* must be 128 */
    int32_t max_ctx;     /* token capacity of each (sequence, KV head) cache row */
    int32_t max_q;       /* verify-row capacity of q and out per sequence */
} ssl_shape;

typedef struct {
    float sm_scale;      /* logit scale, usually 1/sqrt(head_dim) */
    int32_t window;      /* W of Eq. 3 (the paper uses 16); >= 1 */
    int32_t k_sink;      /* K_sink of Eq. 4; >= 0 */
    int32_t k_recent;    /* K_recent of Eq. 4; >= 0 */
    int32_t budget;      /* K_total = K_sink + K_mid + K_recent of Eq. 4 */
    int32_t out_fp32;    /* 1: outputs are fp32, 0: bf16 (round to nearest even) */
    int32_t verify_mode; /* SSL_VERIFY_AUTO, SSL_VERIFY_TWO_SWEEP or SSL_VERIFY_ONE_SWEEP */
    int32_t per_head;    /* 0: importance and index sets per KV head (Eq. 3 summed over the
                          *    query heads of the group);
                          * 1: per query head (Sec. 3.2 keeps importance for every attention
                          *    head): verify writes scores [batch][Hq][max_ctx] (each head's
                          *    own window rows), select builds one index set per query head
                          *    (scores, idx [batch][Hq][...]), and draft gives each query
                          *    head its own set idx[b][h] over the rows of KV head h / group.
                          *    Two-sweep verify needs the group to be 1, 2, 4, 8 or 16
                          *    (SSL_ERR_UNSUPPORTED otherwise); the draft-round calls take
                          *    idx [batch][Hq][budget] and k_sel / v_sel
                          *    [batch][Hq][budget][128], each query head attending over the
                          *    fixed rows of its own set and the shared slid window.  Other
                          *    values: SSL_ERR_SHAPE. */
} ssl_params;

/* How ssl_verify_attn schedules its work (results agree to rounding):
 *  AUTO       a one-sweep schedule where one fits and a KV head has at most
 *             32 verify rows, or more when its chunks run in one round of
 *             workgroups, or up to 48 when the persistent form runs (their
 *             measured sweet spots), else the two-sweep one;
 *  TWO_SWEEP  a K-only pass for the row statistics, then a K+V pass;
 *  ONE_SWEEP  a single K+V pass whose chunks of one (sequence, KV head)
 *             exchange row statistics while resident together: one
 *             workgroup per chunk when every chunk of the call runs in one
 *             round of workgroups (a (sequence, KV head) may then span at most
 *             128 chunks of at most 2048 / 1024 / 640 / 512 keys for up to
 *             16 / 32 / 48 / 64 verify rows per KV head), else, for up to 48
 *             rows, a persistent grid of what the device holds at once (see
 *             ssl_set_cu_budget), each workgroup taking every grid-th chunk
 *             and keeping two chunks' probabilities in 16-bit form (relative
 *             error 2^-11; probabilities below 2^-54 of the row's running
 *             maximum count as 0); SSL_ERR_UNSUPPORTED when neither fits.
 * ssl_verify_plan reports the persistent form as
 * SSL_VERIFY_ONE_SWEEP_PERSISTENT (an output only, not a request). */
enum {
    SSL_VERIFY_AUTO = 0,
    SSL_VERIFY_TWO_SWEEP = 1,
    SSL_VERIFY_ONE_SWEEP = 2,
    SSL_VERIFY_ONE_SWEEP_PERSISTENT = 3
};

/* Human-readable text of a status code (static storage). */
const char *ssl_status_string(int status);

/* An identifier of the sources this library was built from (a hash of the
 * kernel, ABI and build sources; static storage), so that a caller can tell a
 * stale build from a current one. */
const char *ssl_build_id(void);

/*
 * Exchange health (see the conventions above).  Bits of the status word, one
 * per kernel family whose bounded cross-workgroup wait gave up since the word
 * was last read:
 */
enum {
    SSL_EXCHANGE_VERIFY = 1,  /* one-sweep ssl_verify_attn / _paged */
    SSL_EXCHANGE_SELECT = 2,  /* one-kernel ssl_select_topb */
    SSL_EXCHANGE_DRAFT = 4,   /* ssl_draft_attn / _paged, ssl_draft_step */
    SSL_EXCHANGE_LOGITS = 8   /* ssl_logit_stats, ssl_greedy_accept */
};
/* Reads and clears the current device's status word in the order of
 * `stream` (after the work queued before it), waits for `stream`, and stores
 * the bits in *flags_out (0: every exchange since the last read completed).
 * It synchronizes, so it may not be captured (SSL_ERR_UNSUPPORTED while
 * `stream` captures).  Bits raised by work on other streams that is still
 * running may be reported by a later read.  Errors: SSL_ERR_NULL,
 * SSL_ERR_HIP. */
int ssl_exchange_status(hipStream_t stream, uint32_t *flags_out);

/* The name of the HIP error (hipGetErrorName) behind the calling thread's
 * last SSL_ERR_HIP; "hipSuccess" if it has had none.  A static string. */
const char *ssl_last_hip_error(void);

/* The CU count that verify and select plans count on (process-wide; 0, the
 * default, uses the device's own count).  A caller that runs other kernels
 * beside these calls can lower it so that the one-sweep verify and the
 * one-kernel select are chosen only where their exchange groups fit in the
 * CUs left to them.  It also sizes the one-sweep chunks and is read by
 * ssl_verify_plan and the *_workspace calls, also without a GPU.  Errors:
 * SSL_ERR_SHAPE if n_cu < 0. */
int ssl_set_cu_budget(int32_t n_cu);

/* Testing the give-up path, process-wide: spin_limit > 0 bounds every
 * exchange wait to that many polls (0 restores the default), and
 * mismatch_tags = 1 makes every workgroup publish tags that no wait accepts,
 * so that every exchange of later calls gives up, raises its status bit and
 * leaves its outputs unwritten (all kernels still finish).  Errors:
 * SSL_ERR_SHAPE on a negative limit or mismatch_tags not 0 or 1. */
int ssl_test_exchange_faults(int32_t spin_limit, int32_t mismatch_tags);

/* Number of indices Eq. 4 yields for T positions:
 * min(k_sink,T) + min(K_mid, |middle span|) + |recent span|, where the recent
 * span is [max(T - k_recent, min(k_sink, T)), T).  Equals T when T <= budget.
 * Returns SSL_ERR_BUDGET / SSL_ERR_SHAPE (T < 1) on bad arguments. */
int32_t ssl_index_count(int32_t T, int32_t k_sink, int32_t k_recent, int32_t budget);

/*
 * Verify attention with importance scores (Sec. 3.1; Sec. 3.2 Eq. 3).
 *
 * For each sequence b, verify row j < q_len[b], query head h (KV head c):
 *   out[b,j,h]  = softmax_i(sm_scale * q[b,j,h].k[b,c,i]) . v[b,c,i],
 *                 over keys i <= ctx_len[b] - q_len[b] + j;
 *   scores[b,c,i] = sum over the last min(window, q_len[b]) rows j and the
 *                 query heads of c of those probabilities, 0 <= i < ctx_len[b].
 * Probabilities are computed in fp32 from bf16 inputs with fp32 accumulation;
 * the value product uses the probabilities rounded to bf16.
 * Writes out rows j < q_len[b] and scores entries i < ctx_len[b] only.
 * Errors: SSL_ERR_SHAPE if n_q_heads % n_kv_heads, q_len < 1,
 * q_len > ctx_len, ctx_len > max_ctx, q_len > max_q, max_q > 64, window < 1,
 * sm_scale not positive and finite, or verify_mode unknown;
 * SSL_ERR_UNSUPPORTED if head_dim != 128, batch > 64, group > 64, or a
 * one-sweep request that does not fit (including any with q_len * group >
 * 64).  When a KV head has more than 64 verify rows (e.g. Eq. 3 seeded over
 * the last W = 16 prompt positions of a group of 8), the call runs the
 * two-sweep schedule once per block of 64 / group positions, last positions
 * first, and adds the later blocks' scores to the first's.  The workspace
 * size covers both schedules.
 */
int ssl_verify_workspace(const ssl_shape *shape, const ssl_params *params,
                         const int32_t *ctx_len_host, const int32_t *q_len_host,
                         size_t *bytes_out);
/*
 * ssl_verify_attn for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops and harnesses that forbid allocation): the
 * same computation, arguments, limits and errors, with no workspace argument.
 * Its workspace is a 128 MiB device array the library holds on each GPU it
 * runs on until the process ends (it fits every workspace of the five
 * workloads the library is measured on; the largest needs 105 MiB).  The call
 * itself allocates nothing.  SSL_ERR_WORKSPACE if ssl_verify_workspace reports
 * more than 128 MiB for these arguments; SSL_ERR_HIP if the array's address
 * cannot be found on the current device.  Every call on one GPU shares that
 * GPU's array: calls that overlap in time on one GPU (concurrent streams,
 * threads, or graphs replayed concurrently) race and give unspecified results.
 * The array needs no initial contents; an eager call re-arms the exchange
 * epochs of the units it covers, lifting the mark that a captured call whose
 * exchange gave up may have left.
 */
int ssl_verify_attn_static(const ssl_shape *shape, const ssl_params *params,
                           const int32_t *ctx_len_host, const int32_t *q_len_host,
                           const void *q, const void *k_cache, const void *v_cache,
                           void *out, float *scores, hipStream_t stream);

/* The schedule ssl_verify_attn would use for these arguments: *schedule_out
 * = SSL_VERIFY_ONE_SWEEP, SSL_VERIFY_ONE_SWEEP_PERSISTENT or
 * SSL_VERIFY_TWO_SWEEP, *chunk_out = keys per work item, *items_out = work
 * items (each one workgroup, or, persistent, one chunk of a workgroup's
 * sequence).  Host only. */
int ssl_verify_plan(const ssl_shape *shape, const ssl_params *params,
                    const int32_t *ctx_len_host, const int32_t *q_len_host,
                    int32_t *schedule_out, int32_t *chunk_out, int32_t *items_out);
int ssl_verify_attn(const ssl_shape *shape, const ssl_params *params,
                    const int32_t *ctx_len_host, const int32_t *q_len_host,
                    const void *q, const void *k_cache, const void *v_cache,
                    void *out, float *scores,
                    void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Recallable index construction (Sec. 3.2 Eq. 4).
 *
 * For each (b, c) with T = ctx_len_host[b] (the committed length; scores
 * entries 0..T-1 are read):
 *   sink    [0, min(k_sink, T))
 *   recent  [max(T - k_recent, min(k_sink, T)), T)
 *   TopK    the min(K_mid, |middle|) middle positions of highest score,
 *           K_mid = budget - k_sink - k_recent; equal scores go to the lower
 *           position.  Scores must be non-negative and finite (as verify
 *           writes them); comparison is exact on their fp32 values.
 * idx[b,c,0..n) receives sink U TopK U recent in ascending order and
 * n_idx[b] = n = ssl_index_count(T, ...); slots past n are not written.
 *
 * Workspace: ssl_select_workspace gives its size for these context lengths
 * (at most 25 bytes per position of the longest context, per (b, c)); device
 * memory, 16-byte aligned, owned by the caller, no initial contents needed.
 * A call uses it until the call's work on `stream` ends; calls that overlap
 * in time must not share one workspace.
 * Errors: SSL_ERR_BUDGET; SSL_ERR_SHAPE if ctx_len < 1 or > max_ctx;
 * SSL_ERR_UNSUPPORTED if the longest context exceeds 2^21 positions;
 * SSL_ERR_WORKSPACE if the workspace is missing or too small.
 */
int ssl_select_workspace(const ssl_shape *shape, const ssl_params *params,
                         const int32_t *ctx_len_host, size_t *bytes_out);
/* The schedule ssl_select_topb would use: *one_kernel_out = 1 when the
 * partitions of every unit exchange inside one kernel (calls of at most 256
 * partitions whose units' partitions fit in half of what the device holds at
 * once), 0 for the three-kernel schedule; *part_out = positions per
 * partition, *parts_out = partitions of the longest context.  Host only. */
int ssl_select_plan(const ssl_shape *shape, const ssl_params *params,
                    const int32_t *ctx_len_host, int32_t *one_kernel_out, int32_t *part_out,
                    int32_t *parts_out);
int ssl_select_topb(const ssl_shape *shape, const ssl_params *params,
                    const int32_t *ctx_len_host, const float *scores,
                    int32_t *idx, int32_t *n_idx,
                    void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Draft attention over the gathered sparse view (Sec. 3.2 Eq. 5).
 *
 * For each b and query head h (KV head c), with n = n_idx_host[b] and
 * I = idx[b,c,0..n):
 *   out[b,h] = softmax_t(sm_scale * q_draft[b,h].k[b,c,I_t]) . v[b,c,I_t].
 * K/V rows are read in place from the dense cache (never copied).  Same
 * arithmetic as verify.  Errors: SSL_ERR_SHAPE if n < 1 or n > budget;
 * SSL_ERR_UNSUPPORTED if the group exceeds 16.
 */
int ssl_draft_workspace(const ssl_shape *shape, const ssl_params *params,
                        const int32_t *n_idx_host, size_t *bytes_out);
int ssl_draft_attn(const ssl_shape *shape, const ssl_params *params,
                   const int32_t *n_idx_host, const void *q_draft,
                   const void *k_cache, const void *v_cache, const int32_t *idx,
                   void *out, void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Select and the first draft step in one call (Sec. 3.2: Eq. 4 builds the
 * recallable set, Eq. 5 attends over it): ssl_select_topb, then
 * ssl_draft_attn over the index sets it builds (n_idx = ssl_index_count at
 * T = ctx_len_host[b]), with the same arguments, layouts and results (the
 * draft's sums may be ordered differently).  Where select runs as one kernel
 * (ssl_select_plan; partitions of at most 4096 positions, at most 16 query
 * heads per unit) that kernel also runs the draft step: each partition
 * attends over the rows it selected and the partitions' partial results are
 * merged inside the kernel, so the index sets are never read back.  Otherwise
 * the two calls run one after the other on `stream`.  The workspace size comes
 * from ssl_select_draft_workspace.  Errors: those of the two calls.  When an
 * exchange gives up (SSL_EXCHANGE_SELECT raised), the one-kernel form writes
 * neither index sets nor draft outputs for the unit; the two-call form then
 * drafts over idx as it stood (indices are clamped into [0, max_ctx), so no
 * access leaves the cache) and the draft output is meaningless.
 */
int ssl_select_draft_workspace(const ssl_shape *shape, const ssl_params *params,
                               const int32_t *ctx_len_host, size_t *bytes_out);
int ssl_select_draft(const ssl_shape *shape, const ssl_params *params,
                     const int32_t *ctx_len_host, const float *scores, int32_t *idx,
                     int32_t *n_idx, const void *q_draft, const void *k_cache,
                     const void *v_cache, void *out, void *workspace, size_t workspace_bytes,
                     hipStream_t stream);

/*
 * One decode step of the hot path in one call (Sec. 3.1: verify the drafted
 * tokens against the dense cache; Sec. 3.2: Eq. 3 scores from that pass, the
 * Eq. 4 recallable set, the Eq. 5 sparse draft step over it):
 * ssl_verify_attn, then ssl_select_draft on the scores it writes, with the
 * arguments and results of those two calls (q_draft, draft_out and idx/n_idx
 * as there; draft_out has the verify output's dtype).  Where verify takes one
 * sweep (ssl_verify_plan) in a single round of workgroups (every chunk of the
 * call resident at once) with chunks of at least 512 keys, params->per_head
 * is 0 and a KV head has at most 16 query heads, ONE kernel runs the whole
 * step: every chunk workgroup of a
 * (sequence, KV head) is also that unit's select partition over the scores it
 * has just computed and drafts over the rows it selected, so neither the
 * scores nor the index sets are read back.  Otherwise the calls run one after
 * the other on `stream`.  ssl_decode_step_plan reports which (one_kernel_out
 * = 1 or 0).  The workspace size comes from ssl_decode_step_workspace.
 * Errors: those of the two calls.  When an exchange gives up, the status word
 * holds SSL_EXCHANGE_VERIFY or SSL_EXCHANGE_SELECT and the outputs that
 * depended on it are not written (see ssl_select_draft for the two-call form).
 */
int ssl_decode_step_workspace(const ssl_shape *shape, const ssl_params *params,
                              const int32_t *ctx_len_host, const int32_t *q_len_host,
                              size_t *bytes_out);
int ssl_decode_step_plan(const ssl_shape *shape, const ssl_params *params,
                         const int32_t *ctx_len_host, const int32_t *q_len_host,
                         int32_t *one_kernel_out);
int ssl_decode_step(const ssl_shape *shape, const ssl_params *params, const int32_t *ctx_len_host,
                    const int32_t *q_len_host, const void *q, const void *k_cache,
                    const void *v_cache, void *out, float *scores, int32_t *idx, int32_t *n_idx,
                    const void *q_draft, void *draft_out, void *workspace, size_t workspace_bytes,
                    hipStream_t stream);

/*
 * Paged KV cache, as serving engines keep it: the same calls with K and V in
 * page pools instead of one contiguous row per (sequence, KV head).
 *
 * k_pages / v_pages: [n_pages][Hkv][page_size][128] bf16, 16-byte aligned;
 * block_table: device int32 [batch][max_blocks]; key t of sequence b, KV head
 * c is row t % page_size of head c in page block_table[b][t / page_size].
 * page_size must be a multiple of 32.  Page ids are not checked: every entry
 * the call reads must name a page of the pool.  Everything else (shapes, q,
 * out, scores, idx, workspaces and their sizes, errors) is as in
 * ssl_verify_attn / ssl_draft_attn; in addition SSL_ERR_SHAPE if page_size
 * is not a positive multiple of 32, or the pages cannot hold a context
 * (verify: ctx_len[b] > page_size * max_blocks; draft: max_ctx >
 * page_size * max_blocks, since the indices may name any key below max_ctx).
 */
int ssl_verify_attn_paged(const ssl_shape *shape, const ssl_params *params,
                          const int32_t *ctx_len_host, const int32_t *q_len_host,
                          const void *q, const void *k_pages, const void *v_pages,
                          const int32_t *block_table, int32_t page_size, int32_t max_blocks,
                          void *out, float *scores, void *workspace, size_t workspace_bytes,
                          hipStream_t stream);
int ssl_draft_attn_paged(const ssl_shape *shape, const ssl_params *params,
                         const int32_t *n_idx_host, const void *q_draft, const void *k_pages,
                         const void *v_pages, const int32_t *block_table, int32_t page_size,
                         int32_t max_blocks, const int32_t *idx, void *out, void *workspace,
                         size_t workspace_bytes, hipStream_t stream);

/*
 * Draft round (Sec. 3.1: the target model drafts k tokens one after another
 * over the sparse view of Sec. 3.2 Eq. 5).
 *
 * The index set idx[b,c,0..n) was built by ssl_select_topb at
 * T = ctx_len_host[b] (n = ssl_index_count(T, ...)).  Its sink and TopK part,
 * F = the entries below r_T = max(T - k_recent, min(k_sink, T)) (the first
 * n_F = n - (T - r_T) entries), stays for the whole round; the recent window
 * slides.  After i drafted tokens, cur = cur_len_host[b] = T + i with their
 * K/V rows written to the cache, a step attends over F and
 *   W = [max(r_T, cur - k_recent), cur)
 * (so every drafted token lies in W; the entry count stays n when T is long):
 *   out[b,h] = softmax_{t in F u W}(sm_scale * q_draft[b,h].k[b,c,t]) . v[b,c,t].
 * Needs T <= cur <= min(T + k_recent, max_ctx) (else SSL_ERR_SHAPE).
 *
 * ssl_draft_step reads W from the cache and F either through idx (k_sel and
 * v_sel NULL) or from k_sel / v_sel (idx may then be NULL): caller-owned
 * device buffers of [batch][Hkv][budget][128] bf16 that ssl_draft_materialize
 * fills once per round (row e of (b, c) = cache row idx[b,c,e], e < n_F;
 * other rows are not written).  shape->max_q is not used.  Steps use a
 * workspace as ssl_draft_attn does (size from ssl_draft_step_workspace); idx,
 * k_sel and v_sel must not change during a round.  Errors as ssl_draft_attn,
 * plus SSL_ERR_SHAPE for cur_len out of range.
 */
int ssl_draft_materialize(const ssl_shape *shape, const ssl_params *params,
                          const int32_t *ctx_len_host, const void *k_cache,
                          const void *v_cache, const int32_t *idx, void *k_sel, void *v_sel,
                          hipStream_t stream);
int ssl_draft_step_workspace(const ssl_shape *shape, const ssl_params *params,
                             const int32_t *ctx_len_host, const int32_t *cur_len_host,
                             size_t *bytes_out);
int ssl_draft_step(const ssl_shape *shape, const ssl_params *params,
                   const int32_t *ctx_len_host, const int32_t *cur_len_host,
                   const void *q_draft, const void *k_cache, const void *v_cache,
                   const int32_t *idx, const void *k_sel, const void *v_sel, void *out,
                   void *workspace, size_t workspace_bytes, hipStream_t stream);
/* The draft round over a paged cache (pages and block table as in
 * ssl_verify_attn_paged; the drafted tokens' rows written to their pages):
 * the same calls and results, every cache row (sink, TopK and window) read
 * through the block table; materialized rows stay a dense per-unit copy.
 * Workspaces as ssl_draft_step_workspace.  In addition SSL_ERR_NULL without a
 * block table and SSL_ERR_SHAPE if page_size is not a positive multiple of
 * 32 or max_ctx > page_size * max_blocks. */
int ssl_draft_materialize_paged(const ssl_shape *shape, const ssl_params *params,
                                const int32_t *ctx_len_host, const void *k_pages,
                                const void *v_pages, const int32_t *block_table, int32_t page_size,
                                int32_t max_blocks, const int32_t *idx, void *k_sel, void *v_sel,
                                hipStream_t stream);
int ssl_draft_step_paged(const ssl_shape *shape, const ssl_params *params,
                         const int32_t *ctx_len_host, const int32_t *cur_len_host,
                         const void *q_draft, const void *k_pages, const void *v_pages,
                         const int32_t *block_table, int32_t page_size, int32_t max_blocks,
                         const int32_t *idx, const void *k_sel, const void *v_sel, void *out,
                         void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Around the path: token statistics of logit rows.
 *
 * Sec. 3.3 drives the length controller with the entropy H_i of the
 * drafter's output distribution for each drafted token (the ssl_ctrl_* calls
 * below take them in nats); the verification stage (Sec. 2.1) keeps the
 * longest prefix of drafted tokens the target model agrees with and adds one
 * token of its own.  The paper does not spell out the acceptance rule; these
 * calls implement the greedy one, and ssl_spec_accept below the speculative
 * sampling one.
 *
 * Logit rows: logits[r][0..row_stride) of n_rows rows, bf16 (SSL_DT_BF16) or
 * fp32 (SSL_DT_F32); entries [0, vocab) are the logits, the rest is padding
 * that is never read.  row_stride * element size must be a multiple of 16
 * bytes and logits 16-byte aligned; 1 <= vocab <= row_stride, vocab <= 524288.
 * Logits must be finite.
 *
 * ssl_logit_stats: for each row, with p = softmax(logits[r][0..vocab)):
 *   entropy[r] = -sum_i p_i ln p_i (nats, fp32), argmax[r] = the lowest index
 *   of the largest logit.  Either output may be NULL, not both.
 * ssl_greedy_accept: sequence b drafted k = k_len_host[b] <= max_k <= 63
 *   tokens draft_tokens[b][0..k) (layout [batch][max_k]); its verify pass gave
 *   the k + 1 rows logits[b][0..k] (layout [batch][max_k + 1][row_stride]; row j
 *   scores the token after drafted token j - 1; rows past k are not read).
 *   With t_j = argmax of row j:
 *     n_accepted[b] = the largest m <= k with draft_tokens[b][j] == t_j, j < m;
 *     next_token[b] = t_m (the corrected token, or the bonus one when m = k).
 * Both use a caller workspace (size from the *_workspace calls, no initial
 * contents needed; calls that overlap in time must not share one).  Errors:
 * SSL_ERR_NULL, SSL_ERR_SHAPE (counts or sizes out of range, unknown dtype),
 * SSL_ERR_UNSUPPORTED (vocab > 524288, batch > 64), SSL_ERR_ALIGN,
 * SSL_ERR_WORKSPACE.
 */
enum { SSL_DT_BF16 = 0, SSL_DT_F32 = 1 };

int ssl_logit_stats_workspace(int32_t n_rows, int32_t vocab, size_t *bytes_out);
int ssl_logit_stats(const void *logits, int32_t dtype, int32_t n_rows, int32_t vocab,
                    int32_t row_stride, float *entropy, int32_t *argmax, void *workspace,
                    size_t workspace_bytes, hipStream_t stream);
int ssl_greedy_accept_workspace(int32_t batch, int32_t max_k, int32_t vocab, size_t *bytes_out);
int ssl_greedy_accept(const void *logits, int32_t dtype, int32_t batch, int32_t max_k,
                      const int32_t *k_len_host, int32_t vocab, int32_t row_stride,
                      const int32_t *draft_tokens, int32_t *n_accepted, int32_t *next_token,
                      void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Speculative sampling: the verification rule that keeps the target model's
 * output distribution (Sec. 1 and Sec. 2.1 rely on it; the paper does not
 * print it).  Sequence b drafted k = k_len_host[b] <= max_k <= 63 tokens
 * x_j = draft_tokens[b][j] ([batch][max_k]) from the drafter's logit rows
 * draft_logits[b][j] ([batch][max_k][row_stride]); its verify pass gave the
 * target rows target_logits[b][0..k] ([batch][max_k + 1][row_stride]).  With
 * p_j = softmax(target row j / temperature), q_j = softmax(drafter row j /
 * temperature) and the caller's uniforms in [0, 1), u_accept[b][j]
 * ([batch][max_k]) and u_sample[b] ([batch]):
 *   drafted token j passes when u_accept[b][j] * q_j(x_j) < p_j(x_j);
 *   n_accepted[b] = m, the number that pass before the first that fails;
 *   next_token[b] = the smallest x whose cumulative mass (index order)
 *   exceeds u_sample[b] times the total, of max(0, p_m - q_m) when m < k
 *   (of p_m if that has no mass), of p_k when all k passed.
 * Both logit tensors have the dtype and layout rules of ssl_logit_stats; rows
 * past a sequence's k (+1 for the target) are not read.  The arithmetic is
 * fp32: decisions within fp32 rounding of a boundary may go either way.
 * temperature must be finite and > 0 (greedy verification is
 * ssl_greedy_accept).  Token ids are clamped into [0, vocab).  Errors as
 * ssl_greedy_accept, plus SSL_ERR_SHAPE for the temperature.
 */
int ssl_spec_accept_workspace(int32_t batch, int32_t max_k, int32_t vocab, size_t *bytes_out);
int ssl_spec_accept(const void *target_logits, const void *draft_logits, int32_t dtype,
                    int32_t batch, int32_t max_k, const int32_t *k_len_host, int32_t vocab,
                    int32_t row_stride, const int32_t *draft_tokens, float temperature,
                    const float *u_accept, const float *u_sample, int32_t *n_accepted,
                    int32_t *next_token, void *workspace, size_t workspace_bytes,
                    hipStream_t stream);

/*
 * Adaptive speculation length (Sec. 3.3), host only.
 *
 * State: the class-mean entropies of accepted and rejected drafts, tracked by
 * exponential moving averages with coefficient beta (Eq. 6).  Each class mean
 * starts at its first observation.  Entropies are in nats.
 */
typedef struct ssl_ctrl ssl_ctrl;

/* k_cands: the candidate set (values >= 0, copied); k_default is returned by
 * ssl_ctrl_choose_k until both classes have been observed.  NULL on bad
 * arguments (beta outside [0,1], n_cands < 1 or > 256, a negative candidate). */
ssl_ctrl *ssl_ctrl_create(double beta, const int32_t *k_cands, int32_t n_cands,
                          int32_t k_default);
void ssl_ctrl_destroy(ssl_ctrl *ctrl);

/* Eq. 6 update after one verification: H[0..n_drafted) are the draft
 * entropies in drafting order, the first n_accepted were accepted.  The
 * accepted class observes the mean of H[0..n_accepted), the rejected class
 * the mean of the rest; a class with no tokens is not updated. */
int ssl_ctrl_observe(ssl_ctrl *ctrl, const double *H, int32_t n_drafted, int32_t n_accepted);

/* Eq. 7: soft acceptance probability of a draft with entropy H (0.5 while a
 * class is still unobserved). */
double ssl_ctrl_accept_prob(const ssl_ctrl *ctrl, double H);

/* Eq. 8 over the first n draft entropies: the candidate k <= n maximizing
 * (1 + sum_{m<=k} prod_{i<=m} p_i) / (k*c_draft + c_verify), ties to the
 * smaller k.  Returns k_default before both classes are observed, and
 * SSL_ERR_SHAPE if no candidate is <= n, n < 0, or the costs are not finite
 * with c_draft >= 0 and c_verify > 0 (a negative return is always an error:
 * candidates are >= 0). */
int32_t ssl_ctrl_choose_k(const ssl_ctrl *ctrl, const double *H, int32_t n,
                          double c_draft, double c_verify);

/* State access: out[0..4) = {h_acc, h_rej, seen_acc, seen_rej}. */
int ssl_ctrl_get_state(const ssl_ctrl *ctrl, double *out4);
int ssl_ctrl_set_state(ssl_ctrl *ctrl, const double *in4);

#ifdef __cplusplus
}
#endif

#endif /* SPARSESPEC_L_H */

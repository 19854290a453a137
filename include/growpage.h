/*
 * growpage.h -- C ABI of the GrowPage decode-step library for MI355X (gfx950).
 *
 * GrowPage ("On-Demand KV Budgeting for Efficient LLM Reasoning Serving",
 * arXiv 2609.03494) decides, each time a request's last KV page fills, whether
 * to compress its cache in place or to grow it by one page.  This library runs
 * the per-decode-step path on one GPU:
 *
 *   gp_update_summaries  every step: the two EMA query summaries (Sec. 3.2)
 *   gp_decode_attention  every step: paged GQA decode attention (Sec. 3.1)
 *   gp_boundary_score    at boundaries: calibrated, rotated summaries scored
 *                        against the cached keys, top-p working sets (Sec. 3.2,
 *                        App. E.1) and token importance (Sec. 3.3)
 *   gp_boundary_apply    at boundaries: demand trend, decision, page allocation,
 *                        block-local + global selection and in-place compaction
 *                        (Sec. 3.2, 3.3, 4.2, App. E.2)
 *
 * Conventions shared by every call
 *  - Every data pointer is DEVICE memory owned by the caller.  Structs passed
 *    by pointer (gp_kv_layer_t, gp_page_state_t, gp_params_t) live in HOST
 *    memory and are read during the call only.
 *  - The library allocates and frees nothing, never synchronises the stream
 *    and keeps no global state: every call only enqueues kernels on `stream`
 *    and returns.  Results are valid once the stream has reached them.  (One
 *    exception: gp_decode_attention_noalloc keeps its partials in a static
 *    8 MiB device array, one per device, and caches that array's address.)
 *  - Host-side validation returns a status without launching anything.  A
 *    launch failure returns GP_ERR_HIP.  Device-side state that breaks the
 *    layout contract (page ids out of range, seq_len above the pages held) is
 *    never read out of bounds but gives unspecified results.
 *  - Workspaces (`ws`) are caller-owned device buffers of at least
 *    gp_workspace_bytes() bytes, one per operation.  A workspace must be
 *    zero-filled once after allocation; every call leaves its counters at
 *    zero on completion, so it can be reused without clearing.  Two calls
 *    that run concurrently must not share a workspace.
 *  - Page size b is 16 tokens; head_dim is 64 or 128; num_q_heads is 1, 2, 4
 *    or 8 times num_kv_heads.  Decode attention takes page tables up to 8192
 *    pages wide (131072 tokens per request), the boundary calls up to 4096
 *    pages.  Other shapes return GP_ERR_UNSUPPORTED.
 *
 * Layout
 *  K and V pools     [pool_pages][num_kv_heads][page_size][head_dim], float32
 *                    or bfloat16; token i of a request lives in page
 *                    page_table[r][i / page_size], slot i % page_size.
 *  page_table        [num_reqs][max_pages] int32 physical page ids.
 *  num_pages, seq_lens  [num_reqs] int32: pages held P_r and resident tokens
 *                    m_r (m_r <= P_r * page_size).  A request is at a capacity
 *                    boundary when m_r == P_r * page_size (Sec. 3.3).
 *                    seq_lens[r] < 0 marks a HELD request (App. E.3: its
 *                    compaction is still running): it stands for
 *                    m_r = -seq_lens[r] - 1, and the request is out of the
 *                    step's batch -- decode attention writes no output for
 *                    it, the step prologue gives it no token, and the boundary
 *                    calls treat it as not at a boundary.  Only
 *                    gp_boundary_decide(hold = 1) creates held requests and
 *                    gp_release_held() ends them.
 *  refcount          [pool_pages] int32 references from page tables (pages
 *                    shared by a common prefix have refcount > 1, App. E.2).
 *  free_list, free_count  stack of free page ids; the top is
 *                    free_list[*free_count - 1].
 *  qstate            [num_slots][2][num_q_heads][head_dim] float32 summary
 *                    pool (view 0 = short-timescale S, 1 = long-timescale L),
 *                    the per-layer slice of the paper's query-state pool
 *                    (App. E.1, query-cache layout).
 *  q_pre, q_post     [num_reqs][num_q_heads][head_dim] in the KV dtype: the
 *                    current query before and after RoPE.
 */
#ifndef GROWPAGE_H
#define GROWPAGE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GP_OK = 0,
    GP_ERR_INVALID = 1,      /* null pointer, negative size, inconsistent shapes */
    GP_ERR_UNSUPPORTED = 2,  /* page size, head_dim or GQA ratio not built       */
    GP_ERR_WORKSPACE = 3,    /* ws_bytes below gp_workspace_bytes()              */
    GP_ERR_HIP = 4,          /* a kernel launch failed                           */
    GP_ERR_SCRATCH = 5       /* beyond the static scratch of a no-allocation call */
} gp_status_t;

typedef enum { GP_F32 = 0, GP_BF16 = 1 } gp_dtype_t;

/* Per-request decisions written by gp_boundary_apply (Sec. 3.3, 4.2). */
enum {
    GP_COMPRESS = 0,      /* Compress & Hold: one page of tokens evicted in place  */
    GP_GROW = 1,          /* Grow by One Page: a free page appended to the table   */
    GP_FALLBACK = 2,      /* wanted to grow, no page could be granted: compressed  */
    GP_PREEMPT = 3,       /* neither possible; state untouched (scheduler decides) */
    GP_NOT_BOUNDARY = 4,  /* m_r != P_r * page_size; state untouched               */
    GP_SHRINK = 5         /* GP_POLICY_SHRINK only: two pages of tokens evicted,   */
                          /* the last page returned, P_r - 1 pages kept            */
};

/* Capacity-control policies (the paper's appendix on alternative
 * capacity-control policies).  GP_POLICY_GROWPAGE is the method itself. */
enum {
    GP_POLICY_GROWPAGE = 0,  /* grow iff Delta > tau, else Compress & Hold         */
    GP_POLICY_FIXED = 1,     /* grow while P_r < fixed_pages, compress after that  */
    GP_POLICY_RANDOM = 2,    /* compress iff draws[i] < compress_prob, else grow   */
    GP_POLICY_INVERSE = 3,   /* grow iff Delta <= tau, else compress               */
    GP_POLICY_SHRINK = 4     /* Delta < shrink_threshold: shrink (if P_r - 1 >=     */
                             /* max(min_capacity_pages, 2)); Delta > tau: grow;    */
                             /* otherwise compress                                 */
};

/* Demand metric behind K^x (Sec. 3.2; the signal ablation). */
enum {
    GP_METRIC_TOP_P = 0,     /* min k whose k largest weights reach p              */
    GP_METRIC_ENTROPY = 1    /* exp(-sum a ln a) rounded to the nearest integer    */
};

/* Where compaction puts the survivors (Sec. 3.3).  SHIFT is the paper's
 * stable compaction: kept tokens in slot order, then the protected page.
 * FILL leaves every survivor below T (the resident length after the event)
 * in place and moves the survivors at or above T, in slot order, into the
 * evicted slots below T, in slot order: O(b) rows per KV head instead of the
 * whole cache.  Attention does not depend on token order; later boundary
 * events see pages that mix old and recent tokens. */
enum {
    GP_LAYOUT_SHIFT = 0,
    GP_LAYOUT_FILL = 1
};

/* Which workspace gp_workspace_bytes() sizes. */
enum { GP_OP_DECODE = 0, GP_OP_SCORE = 1, GP_OP_APPLY = 2 };

typedef struct {
    void *k;                 /* [pool_pages][num_kv_heads][page_size][head_dim] */
    void *v;                 /* same layout as k                                */
    int32_t pool_pages;
    int32_t num_kv_heads;
    int32_t page_size;       /* must be 16                                      */
    int32_t head_dim;        /* 64 or 128                                       */
    gp_dtype_t dtype;
} gp_kv_layer_t;

typedef struct {
    int32_t *page_table;     /* [num_reqs][max_pages]                           */
    int32_t *num_pages;      /* [num_reqs] P_r                                  */
    int32_t *seq_lens;       /* [num_reqs] m_r                                  */
    int32_t *refcount;       /* [pool_pages]                                    */
    int32_t *free_list;      /* [pool_pages] stack                              */
    int32_t *free_count;     /* [1] stack height                                */
    int32_t num_reqs;
    int32_t max_pages;
    int32_t pool_pages;
} gp_page_state_t;

/* Method constants.  Paper defaults: beta_s 0.9, beta_l 0.999 (Sec. 3.2),
 * p 0.99 (Sec. 3.2), tau 0 (Sec. 3.2), k_loc a quarter of a block (App. D.2
 * uses 64 of 256; 4 of 16 here), scale 1/sqrt(head_dim), rope_theta 1e6
 * (half-split rotary pairs, as in Qwen3).  reserve_pages: a grow is granted
 * only while more than this many pages are free (Sec. 4.2, "safely").
 * The remaining fields select a policy variant and the demand metric; all
 * zero is the method itself.  Appendix values: fixed_pages 256 (4096
 * tokens), compress_prob 0.7, shrink_threshold -0.005, min_capacity_pages 64
 * (1024 tokens).  draws: DEVICE [num_bnd] float32 uniform in [0, 1), one per
 * boundary request, read by GP_POLICY_RANDOM only (may be NULL otherwise).
 * layout: GP_LAYOUT_SHIFT (0, the method) or GP_LAYOUT_FILL.
 * select_skip_grows: nonzero tells gp_boundary_select that k_counts are
 * final when it runs (see the split calls below). */
typedef struct {
    float beta_s, beta_l;
    float p;
    float tau;
    float scale;
    float rope_theta;
    int32_t k_loc;
    int32_t reserve_pages;
    int32_t policy;              /* GP_POLICY_*                                 */
    int32_t metric;              /* GP_METRIC_*                                 */
    int32_t fixed_pages;
    int32_t min_capacity_pages;
    float compress_prob;
    float shrink_threshold;
    const float *draws;
    int32_t layout;              /* GP_LAYOUT_*                                 */
    int32_t select_skip_grows;   /* gp_boundary_select only, see there          */
} gp_params_t;

/* Dual-timescale summaries (Sec. 3.2, EMA equation; App. E.1).
 * For each request r with slot s = slot_ids[r]: if init[r] != 0 both views of
 * slot s become q_pre[r] (a new owner overwrites whatever the slot held);
 * otherwise qbar_x <- beta_x * qbar_x + (1 - beta_x) * q_pre[r] for x in {S, L}.
 * Arithmetic is fp64, rounded once to float32.  Requests with a slot outside
 * [0, num_slots) are skipped.  q_pre: [num_reqs][num_q_heads][head_dim] in
 * `dtype`; slot_ids [num_reqs] int32; init [num_reqs] uint8; qstate updated
 * in place.  Slots must be distinct across requests. */
gp_status_t gp_update_summaries(const void *q_pre, gp_dtype_t dtype, int32_t num_reqs,
                                int32_t num_q_heads, int32_t head_dim,
                                const int32_t *slot_ids, const uint8_t *init,
                                float *qstate, int32_t num_slots,
                                float beta_s, float beta_l, hipStream_t stream);

/* Paged decode attention (Sec. 3.1, attention-output equation):
 * out[r][g] = sum_{i < m_r} softmax_i(scale * q_post[r][g] . k_i) v_i, with
 * k_i, v_i read from KV head g / (num_q_heads / num_kv_heads) through the page
 * table.  fp32 accumulation; output in the KV dtype.  A request with m_r == 0
 * gets a zero output; a held request (seq_lens[r] < 0) gets none (its rows of
 * out are not written, and gp_decode_step leaves its summaries alone).  Page slots at or beyond m_r are never used, whatever
 * they hold.  out: [num_reqs][num_q_heads][head_dim]. */
gp_status_t gp_decode_attention(const gp_kv_layer_t *kv, const gp_page_state_t *ps,
                                const void *q_post, int32_t num_q_heads, float scale,
                                void *out, void *ws, size_t ws_bytes, hipStream_t stream);

/* Decode attention over batches whose requests share a common prefix of
 * pages (App. E.2: a shared prefix sits in reference-counted blocks that every
 * request holding it reads; Sec. 3.1 attention-output equation).  Same
 * arguments and outputs as gp_decode_attention, plus prefix groups (HOST
 * array, read during the call): requests [first_req, first_req + num_reqs)
 * share the first prefix_pages pages of request first_req's table.  The
 * shared pages are read once per block of 8 * 16 / G requests of a group
 * (not once per request), in a prefix pass on the matrix cores; each
 * request's private pages follow in the usual split pass, and the two
 * partial results are merged.  Whether a request reads the prefix pass is
 * decided on the device: it must not be held, hold at least prefix_pages
 * pages and prefix_pages * page_size tokens, and have the leader's page ids
 * on all prefix pages; any other member (e.g. one whose shared pages a
 * compaction has replaced by private copies, App. E.2) is served like a
 * request of no group, so the groups only decide the speed, never the
 * result.  The outputs equal gp_decode_attention's to float32 rounding of the
 * sums (P.V of the prefix runs in another order; the bf16 output may differ
 * in its last bit).  Groups: at most 16, in order of first_req, disjoint;
 * bfloat16 pools only (GP_ERR_UNSUPPORTED otherwise).  Takes the decode
 * workspace.
 * `stages` (any non-empty combination of GP_DECODE_PREFIX, GP_DECODE_CHUNKS,
 * GP_DECODE_MERGE; all three = the whole call, run in that order) lets a
 * caller overlap the two passes: PREFIX (the shared pages, on the matrix
 * cores) and CHUNKS (the private pages, bound by HBM) read the same inputs
 * and write disjoint parts of ws, so they may run concurrently on two
 * streams; MERGE reads ws and must be ordered after both.  Between the
 * stages nothing but ws may be written. */
typedef struct {
    int32_t first_req, num_reqs, prefix_pages;
} gp_prefix_group_t;
gp_status_t gp_decode_attention_shared(const gp_kv_layer_t *kv, const gp_page_state_t *ps,
                                       const void *q_post, int32_t num_q_heads, float scale, void *out,
                                       const gp_prefix_group_t *groups, int32_t num_groups, int32_t stages,
                                       void *ws, size_t ws_bytes, hipStream_t stream);

/* gp_decode_attention without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments and results as
 * gp_decode_attention; the split partials go to a static device array of
 * 8 MiB (one per device, held until the process ends), so the call allocates
 * nothing.  A batch whose decode workspace (gp_workspace_bytes(GP_OP_DECODE,
 * ...)) exceeds 8 MiB returns GP_ERR_SCRATCH without launching.  `stream`
 * must belong to the current device (else GP_ERR_INVALID).  Every call on a
 * device shares that device's array: calls that overlap on one device (on
 * different streams, or a later call before an earlier one has completed on
 * another stream) race and give undefined results; calls in one stream's
 * order are safe.  Nothing in the array needs to start at zero. */
gp_status_t gp_decode_attention_noalloc(const gp_kv_layer_t *kv, const gp_page_state_t *ps,
                                        const void *q_post, int32_t num_q_heads, float scale,
                                        void *out, hipStream_t stream);

/* gp_decode_attention in its two launches, for a caller that orders other
 * work after the first (Sec. 3.1, same outputs):
 *   GP_DECODE_CHUNKS  reads q_post and the cache through the page table: the
 *                     outputs of requests that fit in one chunk, partial
 *                     (max, sum, o) of the others into ws;
 *   GP_DECODE_MERGE   folds those partials into the remaining outputs: reads
 *                     ws (which also records each request's length), never
 *                     the cache.
 * `stages` is either bit or both; both stages in order, on one ws and the
 * same `ps` contents, give the bytes of gp_decode_attention.  Between them
 * the cache may be written (e.g. compacted), not ws, `out` or the lengths
 * and page counts.  Takes the decode workspace; GP_ERR_INVALID for any other
 * `stages`. */
enum { GP_DECODE_CHUNKS = 1, GP_DECODE_MERGE = 2, GP_DECODE_PREFIX = 4 };
gp_status_t gp_decode_attention_stages(const gp_kv_layer_t *kv, const gp_page_state_t *ps,
                                       const void *q_post, int32_t num_q_heads, float scale,
                                       void *out, int32_t stages, void *ws, size_t ws_bytes,
                                       hipStream_t stream);

/* The step's new token, the summary update and decode attention in a single
 * launch (Sec. 4.1 folds the per-step work into the attention kernel).
 *  - Without a token (k_new == v_new == NULL): on a batch with no held request
 *    the results are those of gp_update_summaries(q_pre, kv->dtype,
 *    ps->num_reqs, num_q_heads, kv->head_dim, slot_ids, init, qstate,
 *    num_slots, beta_s, beta_l) followed by gp_decode_attention(kv, ps,
 *    q_post, num_q_heads, scale, out, ws), bit for bit.
 *  - With a token (k_new, v_new [num_reqs][num_kv_heads][head_dim] in the KV
 *    dtype, post-RoPE): every request with room (0 <= m_r < P_r * page_size)
 *    takes it -- its K and V are written at slot m_r of the paged cache, the
 *    summaries of its slot take one EMA step with q_pre (or are set to it if
 *    init[r] != 0), and decode attention runs over its m_r + 1 tokens;
 *    requests with full pages (at a boundary, awaiting a decision) take no
 *    token, keep their summaries and attend over their m_r tokens.  With
 *    advance != 0, seq_lens[r] and positions[r] of the requests that took the
 *    token then grow by one; pass advance = 0 for every layer but the last
 *    when each layer of a model calls this (the lengths are shared by the
 *    layers).  One layer with advance != 0 equals gp_append_step(kv, 1, ps,
 *    positions, k_new, v_new, q_pre, ...) followed by gp_decode_attention, bit
 *    for bit.  positions may be NULL when advance == 0.
 *  - A held request (seq_lens[r] < 0) is out of the step: no token, no
 *    summary update, no output (gp_update_summaries, which does not see the
 *    lengths, would update it).
 * q_pre has the layout and dtype of q_post.  Takes the decode workspace.
 * GP_ERR_INVALID if only one of k_new, v_new is given, or advance != 0 with a
 * token and no positions. */
gp_status_t gp_decode_step(const gp_kv_layer_t *kv, const gp_page_state_t *ps, const void *q_post,
                           const void *q_pre, int32_t num_q_heads, float scale, void *out,
                           const int32_t *slot_ids, const uint8_t *init, float *qstate, int32_t num_slots,
                           float beta_s, float beta_l, const void *k_new, const void *v_new,
                           int32_t *positions, int32_t advance, void *ws, size_t ws_bytes,
                           hipStream_t stream);

/* Boundary scoring of one layer (Sec. 3.2 and 3.3; App. E.1).
 * For boundary request i (r = bnd[i], at a boundary, P = num_pages[r]):
 * candidates are slots [0, (P-1) * page_size) (the most recent page is left
 * out).  Each summary x of each query head is scaled to the RMS of q_pre[r]
 * (RMS calibration), rotated at positions[r], and its softmax over the
 * candidates' keys is taken; the G query heads of a KV head are averaged.
 * Outputs, per KV head h:
 *   k_counts[i][h][x]  working-set size K^x, x = 0 (S), 1 (L): with
 *                      GP_METRIC_TOP_P the min k whose k largest weights
 *                      reach p; with GP_METRIC_ENTROPY exp(H) of the weights
 *                      rounded to the nearest integer, clamped to [1, |C|];
 *   scores[i][h][c]    s_c = max(a^S_c, a^L_c) for c < (P-1) * page_size.
 * Weights are computed in fp64 and rounded to float32; K^x is decided on the
 * float32 weights.  Requests not at a boundary get k_counts 0.  Requires
 * max_cand >= (max_pages - 1) * page_size.  bnd [num_bnd] int32, positions
 * [num_reqs] int32 (logical index of the current token). */
gp_status_t gp_boundary_score(const gp_kv_layer_t *kv, const gp_page_state_t *ps,
                              const void *q_pre, const float *qstate, int32_t num_slots,
                              const int32_t *slot_ids, const int32_t *positions,
                              const int32_t *bnd, int32_t num_bnd, int32_t num_q_heads,
                              const gp_params_t *params, int32_t *k_counts, float *scores,
                              int32_t max_cand, void *ws, size_t ws_bytes, hipStream_t stream);

/* gp_boundary_score in two stream-ordered parts (stages, a bit mask), so that
 * the selection, which needs only the scores, can run beside the working-set
 * counts (the asynchronous overlap of App. E.3 applied inside one event):
 *  - GP_SCORE_WEIGHTS: calibration and rotation of the summaries, the
 *    per-view softmax weights in the workspace and scores[] (Sec. 3.2,
 *    Sec. 3.3 token score);
 *  - GP_SCORE_COUNTS:  k_counts[] from the weights in the workspace (Sec. 3.2
 *    working-set ratio; top-p or entropy by params->metric).
 * Same arguments and workspace in both calls; COUNTS after WEIGHTS on one
 * stream, or after an event that orders it so; both stages in one call is
 * gp_boundary_score.  The two write disjoint outputs, and COUNTS only reads
 * the workspace and the page state.  GP_ERR_INVALID for an empty or unknown
 * mask. */
enum { GP_SCORE_WEIGHTS = 1, GP_SCORE_COUNTS = 2 };
gp_status_t gp_boundary_score_stages(const gp_kv_layer_t *kv, const gp_page_state_t *ps,
                                     const void *q_pre, const float *qstate, int32_t num_slots,
                                     const int32_t *slot_ids, const int32_t *positions,
                                     const int32_t *bnd, int32_t num_bnd, int32_t num_q_heads,
                                     const gp_params_t *params, int32_t *k_counts, float *scores,
                                     int32_t max_cand, void *ws, size_t ws_bytes, hipStream_t stream,
                                     int32_t stages);

/* Decision, allocation, selection and compaction for the boundary requests,
 * over n_layers layers (layers[l], k_counts[l][num_bnd][Hkv][2] and
 * scores[l][num_bnd][Hkv][max_cand] from gp_boundary_score).
 *  - Delta = r^S - r^L, the mean over (layer, KV head) of K^x / |C|
 *    (Sec. 3.2, aggregation equation), evaluated from the integer counts;
 *    Grow iff Delta > tau.  delta[i] receives Delta as float32.  Threshold
 *    tests are exact: the integer sum D = sum (K^S - K^L) is compared with
 *    t * |C| * Hkv * n_layers in fp64.
 *  - params->policy replaces the grow test (App., alternative
 *    capacity-control policies): FIXED grows iff P < fixed_pages; RANDOM
 *    grows iff !(draws[i] < compress_prob); INVERSE grows iff Delta <= tau;
 *    SHRINK grows iff Delta > tau, shrinks iff Delta < shrink_threshold and
 *    P - 1 >= max(min_capacity_pages, 2), else compresses.  With P <= 1
 *    FIXED grows iff P < fixed_pages, the others always want to grow.
 *  - Requests are served in list order.  A grow pops the free-page stack
 *    (refcount 1, appended at index P); if no page can be granted (stack at or
 *    below reserve_pages, or the table row full) the request compresses
 *    (GP_FALLBACK).  P <= 1 cannot compress: grow or GP_PREEMPT.
 *  - Compress keeps P and sets m = (P-1) * page_size.  Per layer and KV head,
 *    exactly page_size candidates are evicted: each candidate page keeps its
 *    min(k_loc, K_t / (P-1)) best tokens, K_t = (P-2) * page_size, and the
 *    rest of K_t goes to the best remaining candidates (order: score
 *    descending, slot ascending).  Kept tokens stay in order, followed by the
 *    protected last page (Sec. 3.3, selection equation).
 *  - Shrink (GP_SHRINK) evicts two pages of candidates by the same rule with
 *    K_t = (P-3) * page_size, moves the last page right after the kept
 *    tokens, sets m = (P-2) * page_size and P = P - 1, and drops the table's
 *    reference to the old last page (released if its count reaches zero).
 *  - Shared pages (refcount > 1) are never written: a compressing request
 *    first pops one private page per shared page (GP_PREEMPT if too few), its
 *    compacted tokens go there, and the shared page loses one reference
 *    (App. E.2).  Sharing is judged on the counts as the call starts.  Pages
 *    whose count reaches zero are pushed on the stack at the end of the
 *    call, lowest page id first (the last pushed is popped first).
 *  - Entries of bnd must be distinct (one boundary step per request).
 *  - counters[4] (int64) += number of COMPRESS, GROW, FALLBACK, PREEMPT
 *    (a shrink counts as a compression). */
gp_status_t gp_boundary_apply(const gp_kv_layer_t *layers, int32_t n_layers,
                              const gp_page_state_t *ps, const int32_t *bnd, int32_t num_bnd,
                              const int32_t *k_counts, const float *scores, int32_t max_cand,
                              const gp_params_t *params, int32_t *decisions, float *delta,
                              int64_t *counters, void *ws, size_t ws_bytes, hipStream_t stream);

/* gp_boundary_apply in three stream-ordered parts, for overlap with decoding
 * (App. E.3, asynchronous decoding and compression).  Each takes exactly the
 * arguments of gp_boundary_apply, and the three calls of one event must get
 * the same arguments and the same workspace, in this order:
 *  - select:  the eviction lists of every boundary request (selection needs
 *             only the scores) and the rows compaction will read.  Reads the
 *             page state, K/V and scores; writes only the workspace, so it may
 *             run beside decode attention.  With params->select_skip_grows
 *             != 0 the caller guarantees that k_counts are final (e.g. select
 *             is stream-ordered after the scoring): select then also reads
 *             k_counts and *free_count and skips the lists and rows of every
 *             request whose decision can only be a grow -- it wants to grow
 *             (the decision rule on its counts, as decide applies it), P_r <
 *             max_pages, and *free_count - i * max_pages > reserve_pages for
 *             its list index i, so that no earlier request of the event can
 *             leave it short of a page.  No call may take pages from the free
 *             stack between an event's select and its decide.  Should decide
 *             nevertheless not grow such a request (counts changed after
 *             select, the stack shrank), it preempts it instead (state
 *             untouched, counted as PREEMPT).  gp_boundary_apply always skips
 *             (its k_counts are inputs).
 *  - decide:  decisions, delta, counters, page allocation and table updates.
 *             With hold != 0 a request that compresses or shrinks is left HELD
 *             (seq_lens[r] = -(new m) - 1) so that a decode step launched while
 *             its compaction runs leaves it out; otherwise as in apply.
 *  - compact: moves the rows of the requests that compress or shrink, and
 *             pushes the pages the event released onto the free stack
 *             (free_list and *free_count).  The cached rows it reads and
 *             writes are those of the moving requests only, so it may run
 *             beside the next step's append and decode of the other requests.
 * gp_boundary_apply == select, decide (hold 0), compact on one stream.
 * Ordering: decide pops the free stack and compact pushes onto it, so the
 * next event's decide -- and anything else that reads or changes free_list,
 * free_count or the refcounts -- must be stream-ordered after the previous
 * event's compact (otherwise a push and a pop race and a page can be handed
 * out twice).  The workspace holds the event until compact has completed: an
 * event whose select runs while the previous one's compact is still running
 * needs a second workspace. */
gp_status_t gp_boundary_select(const gp_kv_layer_t *layers, int32_t n_layers,
                               const gp_page_state_t *ps, const int32_t *bnd, int32_t num_bnd,
                               const int32_t *k_counts, const float *scores, int32_t max_cand,
                               const gp_params_t *params, int32_t *decisions, float *delta,
                               int64_t *counters, void *ws, size_t ws_bytes, hipStream_t stream);
gp_status_t gp_boundary_decide(const gp_kv_layer_t *layers, int32_t n_layers,
                               const gp_page_state_t *ps, const int32_t *bnd, int32_t num_bnd,
                               const int32_t *k_counts, const float *scores, int32_t max_cand,
                               const gp_params_t *params, int32_t *decisions, float *delta,
                               int64_t *counters, void *ws, size_t ws_bytes, hipStream_t stream,
                               int32_t hold);
gp_status_t gp_boundary_compact(const gp_kv_layer_t *layers, int32_t n_layers,
                                const gp_page_state_t *ps, const int32_t *bnd, int32_t num_bnd,
                                const int32_t *k_counts, const float *scores, int32_t max_cand,
                                const gp_params_t *params, int32_t *decisions, float *delta,
                                int64_t *counters, void *ws, size_t ws_bytes, hipStream_t stream);

/* Ends every hold: seq_lens[r] < 0 becomes -seq_lens[r] - 1 (App. E.3: a
 * compressed request rejoins the batch once its compaction has completed;
 * the caller orders this call after that compaction). */
gp_status_t gp_release_held(const gp_page_state_t *ps, hipStream_t stream);

/* Step prologue of the decode loop (Sec. 3.1 paged cache; Sec. 3.2 EMA;
 * App. E.1 query-state pool): for every request r that is not held and has
 * room (0 <= m_r < P_r * page_size), over all n_layers layers,
 *  - the token's keys and values k_new[l][r], v_new[l][r] ([Hkv][head_dim],
 *    post-RoPE, the KV dtype) are written at slot m_r of the paged cache;
 *  - the summaries of slot slot_ids[r] in layer l's pool take one EMA step
 *    with q_pre[l][r] (or are set to it if init[r] != 0), exactly as
 *    gp_update_summaries does;
 * then m_r and positions[r] advance by one.  Requests with full pages (at a
 * boundary, awaiting a decision) and held requests are left untouched.
 * k_new, v_new [n_layers][num_reqs][Hkv][head_dim]; q_pre
 * [n_layers][num_reqs][num_q_heads][head_dim]; qstate
 * [n_layers][num_slots][2][num_q_heads][head_dim] (the paper's per-layer
 * pool); init may be NULL (no new slots).  Slots must be distinct. */
gp_status_t gp_append_step(const gp_kv_layer_t *layers, int32_t n_layers, const gp_page_state_t *ps,
                           int32_t *positions, const void *k_new, const void *v_new, const void *q_pre,
                           int32_t num_q_heads, const int32_t *slot_ids, const uint8_t *init,
                           float *qstate, int32_t num_slots, float beta_s, float beta_l,
                           hipStream_t stream);

/* Bytes of workspace an operation needs (op = GP_OP_DECODE / SCORE / APPLY). */
size_t gp_workspace_bytes(int32_t op, int32_t num_reqs, int32_t num_bnd, int32_t num_q_heads,
                          int32_t num_kv_heads, int32_t head_dim, int32_t max_pages,
                          int32_t page_size, gp_dtype_t dtype, int32_t n_layers);

/* Measurement reference, not a step of the method: reads bytes (a multiple of
 * 16; device memory, 16-byte aligned) once with plain streaming loads and
 * XORs every word into *out (device, 4 bytes, caller-owned; not cleared
 * here).  Its bandwidth is the streaming-read ceiling the decode and scoring
 * kernels are set against.  The per-workgroup partial words go through one
 * device-wide array in the library, so calls that overlap on one device (on
 * different streams) race; calls in one stream do not.  GP_ERR_INVALID for a
 * null pointer or a size that is not a multiple of 16. */
gp_status_t gp_stream_read(const void *src, size_t bytes, uint32_t *out, hipStream_t stream);

/* Static description of a status code. */
const char *gp_status_string(gp_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* GROWPAGE_H */

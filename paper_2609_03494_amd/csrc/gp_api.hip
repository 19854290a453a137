// Host side of the C ABI: argument validation, workspace carving and launch.
// Every entry point checks what the host can see (pointers, shapes, sizes),
// then enqueues its kernels on the caller's stream and returns.
#include <math.h>

#include <mutex>

#include "gp_internal.h"

using namespace gp;

// Scratch of gp_decode_attention_noalloc, for callers that cannot allocate:
// the decode partials live in this array, one copy per device, held until the
// process ends.  In host code `scratch` only names the symbol; its device
// address comes from hipGetSymbolAddress (scratch_address below).
constexpr size_t kScratchBytes = size_t(8) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices];     // device address of `scratch`, per device

// The address of `scratch` on the device `stream` runs on, which must be the
// current device; looked up once per device, with that device current.
gp_status_t scratch_address(hipStream_t stream, void **out) {
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return GP_ERR_HIP;
    if (stream) {
        hipDevice_t sd = 0;
        if (hipStreamGetDevice(stream, &sd) != hipSuccess) return GP_ERR_HIP;
        if (sd != cur) return GP_ERR_INVALID;
    }
    if (cur < 0 || cur >= kMaxDevices) return GP_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[cur]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return GP_ERR_HIP;
        g_scratch_ptr[cur] = p;
    }
    *out = g_scratch_ptr[cur];
    return GP_OK;
}

bool dims_ok(int Hq, int Hkv, int D) {
    if (Hkv <= 0 || Hq <= 0 || Hq % Hkv) return false;
    const int G = Hq / Hkv;
    return (D == 64 || D == 128) && (G == 1 || G == 2 || G == 4 || G == 8);
}

gp_status_t check_layer(const gp_kv_layer_t *kv) {
    if (!kv || !kv->k || !kv->v) return GP_ERR_INVALID;
    if (kv->pool_pages <= 0 || kv->num_kv_heads <= 0) return GP_ERR_INVALID;
    if (kv->dtype != GP_F32 && kv->dtype != GP_BF16) return GP_ERR_INVALID;
    if (kv->page_size != kPage) return GP_ERR_UNSUPPORTED;
    if (kv->head_dim != 64 && kv->head_dim != 128) return GP_ERR_UNSUPPORTED;
    return GP_OK;
}

gp_status_t check_state(const gp_page_state_t *ps, const gp_kv_layer_t *kv) {
    if (!ps || !ps->page_table || !ps->num_pages || !ps->seq_lens) return GP_ERR_INVALID;
    if (ps->num_reqs < 0 || ps->max_pages <= 0) return GP_ERR_INVALID;
    if (kv && ps->pool_pages != kv->pool_pages) return GP_ERR_INVALID;
    return GP_OK;
}

gp_status_t from_hip(hipError_t e) { return e == hipSuccess ? GP_OK : GP_ERR_HIP; }

int elem_bytes(gp_dtype_t dt) { return dt == GP_F32 ? 4 : 2; }

}  // namespace

extern "C" {

const char *gp_status_string(gp_status_t s) {
    switch (s) {
        case GP_OK: return "ok";
        case GP_ERR_INVALID: return "invalid argument";
        case GP_ERR_UNSUPPORTED: return "unsupported shape (page size 16, head_dim 64/128, GQA ratio 1/2/4/8)";
        case GP_ERR_WORKSPACE: return "workspace too small";
        case GP_ERR_HIP: return "HIP launch failed";
        case GP_ERR_SCRATCH:
            return "problem needs more than the 8 MiB static scratch of gp_decode_attention_noalloc";
    }
    return "unknown status";
}

gp_status_t gp_stream_read(const void *src, size_t bytes, uint32_t *out, hipStream_t stream) {
    if (!src || !out || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(src) % 16 != 0) return GP_ERR_INVALID;
    if (bytes == 0) return GP_OK;
    return from_hip(launch_stream_read(src, bytes, out, stream));
}

size_t gp_workspace_bytes(int32_t op, int32_t num_reqs, int32_t num_bnd, int32_t num_q_heads,
                          int32_t num_kv_heads, int32_t head_dim, int32_t max_pages,
                          int32_t page_size, gp_dtype_t dtype, int32_t n_layers) {
    if (page_size != kPage || !dims_ok(num_q_heads, num_kv_heads, head_dim) || max_pages <= 0 ||
        num_reqs < 0 || num_bnd < 0 || n_layers <= 0)
        return 0;
    switch (op) {
        case GP_OP_DECODE:
            return decode_ws(num_reqs, num_q_heads, num_kv_heads, head_dim, max_pages).total;
        case GP_OP_SCORE: return score_ws(num_bnd, num_q_heads, num_kv_heads, max_pages).total;
        case GP_OP_APPLY:
            return apply_ws(num_bnd, num_kv_heads, head_dim, elem_bytes(dtype), max_pages, n_layers).total;
    }
    return 0;
}

gp_status_t gp_update_summaries(const void *q_pre, gp_dtype_t dtype, int32_t num_reqs,
                                int32_t num_q_heads, int32_t head_dim, const int32_t *slot_ids,
                                const uint8_t *init, float *qstate, int32_t num_slots, float beta_s,
                                float beta_l, hipStream_t stream) {
    if (num_reqs < 0 || num_q_heads <= 0 || head_dim <= 0 || num_slots <= 0) return GP_ERR_INVALID;
    if (dtype != GP_F32 && dtype != GP_BF16) return GP_ERR_INVALID;
    if (num_reqs == 0) return GP_OK;
    if (!q_pre || !slot_ids || !init || !qstate) return GP_ERR_INVALID;
    if (!(beta_s >= 0.0f && beta_s <= 1.0f && beta_l >= 0.0f && beta_l <= 1.0f)) return GP_ERR_INVALID;
    SummaryArgs a;
    a.q = q_pre;
    a.slot_ids = slot_ids;
    a.init = init;
    a.qstate = qstate;
    a.R = num_reqs;
    a.HqD = num_q_heads * head_dim;
    a.M = num_slots;
    a.beta_s = beta_s;
    a.beta_l = beta_l;
    return from_hip(launch_summaries(dtype, a, stream));
}

namespace {

// Shared by gp_decode_attention and gp_decode_step; `sum` is the folded
// summary update (q_pre == nullptr: none).
struct FoldedSummaries {
    const void *q_pre;
    const int32_t *slot_ids;
    const uint8_t *init;
    float *qstate;
    int32_t num_slots;
    float beta_s, beta_l;
    // the step's new token (k_new == nullptr: none)
    const void *k_new, *v_new;
    int32_t *positions;
    int32_t advance;
};

// noalloc: ws and ws_bytes are ignored; the partials go to the static scratch.
// groups (host, num_groups of them): the shared-prefix decode.
gp_status_t decode_call(const gp_kv_layer_t *kv, const gp_page_state_t *ps, const void *q_post,
                        int32_t num_q_heads, float scale, void *out, void *ws, size_t ws_bytes,
                        const FoldedSummaries *sum, int stages, hipStream_t stream, bool noalloc = false,
                        const gp_prefix_group_t *groups = nullptr, int32_t num_groups = 0) {
    gp_status_t st = check_layer(kv);
    if (st != GP_OK) return st;
    if ((st = check_state(ps, kv)) != GP_OK) return st;
    if (!dims_ok(num_q_heads, kv->num_kv_heads, kv->head_dim)) return GP_ERR_UNSUPPORTED;
    if (!(scale > 0.0f) || !isfinite(scale)) return GP_ERR_INVALID;
    if (sum) {
        if (sum->num_slots <= 0) return GP_ERR_INVALID;
        if (!(sum->beta_s >= 0.0f && sum->beta_s <= 1.0f && sum->beta_l >= 0.0f && sum->beta_l <= 1.0f))
            return GP_ERR_INVALID;
    }
    if (ps->num_reqs == 0) return GP_OK;
    if (!q_post || !out || (!ws && !noalloc)) return GP_ERR_INVALID;
    if (sum && (!sum->q_pre || !sum->slot_ids || !sum->init || !sum->qstate)) return GP_ERR_INVALID;
    if (sum && (!sum->k_new != !sum->v_new)) return GP_ERR_INVALID;
    if (sum && sum->k_new && sum->advance && !sum->positions) return GP_ERR_INVALID;
    const DecodeWs w = decode_ws(ps->num_reqs, num_q_heads, kv->num_kv_heads, kv->head_dim, ps->max_pages);
    if (ps->num_reqs > 65535 || w.max_chunks > kMaxDecodeChunks || w.chunk_pages > kMaxChunkPages)
        return GP_ERR_UNSUPPORTED;
    if (noalloc) {
        if (w.total > kScratchBytes) return GP_ERR_SCRATCH;
        if ((st = scratch_address(stream, &ws)) != GP_OK) return st;
        ws_bytes = kScratchBytes;
    }
    if (ws_bytes < w.total) return GP_ERR_WORKSPACE;
    DecodeArgs a = {};
    if (num_groups < 0 || num_groups > kMaxPrefixGroups || (num_groups > 0 && !groups)) return GP_ERR_INVALID;
    if (num_groups > 0 && kv->dtype != GP_BF16) return GP_ERR_UNSUPPORTED;
    {
        // groups: in order of first request, disjoint, inside the batch, a
        // prefix of at least one page and at most the table width
        int end = 0, blk = 0;
        const int rpb = kPrefixWaves * (16 / (num_q_heads / kv->num_kv_heads));
        for (int g = 0; g < num_groups; ++g) {
            const gp_prefix_group_t &gr = groups[g];
            if (gr.first_req < end || gr.num_reqs < 1 || gr.first_req + gr.num_reqs > ps->num_reqs ||
                gr.prefix_pages < 1 || gr.prefix_pages > ps->max_pages)
                return GP_ERR_INVALID;
            end = gr.first_req + gr.num_reqs;
            a.g_first[g] = gr.first_req;
            a.g_num[g] = gr.num_reqs;
            a.g_pages[g] = gr.prefix_pages;
            a.g_blk0[g] = blk;
            blk += cdiv(gr.num_reqs, rpb);
        }
        a.g_blk0[num_groups] = blk;
        a.ngroups = num_groups;
        if (blk > 65535) return GP_ERR_UNSUPPORTED;
    }
    a.k = kv->k;
    a.v = kv->v;
    a.page_table = ps->page_table;
    a.num_pages = ps->num_pages;
    a.seq_lens = ps->seq_lens;
    a.q = q_post;
    a.out = out;
    a.q_pre = sum ? sum->q_pre : nullptr;
    a.slot_ids = sum ? sum->slot_ids : nullptr;
    a.init = sum ? sum->init : nullptr;
    a.qstate = sum ? sum->qstate : nullptr;
    a.M = sum ? sum->num_slots : 0;
    a.beta_s = sum ? sum->beta_s : 0.0;
    a.beta_l = sum ? sum->beta_l : 0.0;
    a.k_w = kv->k;
    a.v_w = kv->v;
    a.k_new = sum ? sum->k_new : nullptr;
    a.v_new = sum ? sum->v_new : nullptr;
    a.seq_lens_w = ps->seq_lens;
    a.positions = sum ? sum->positions : nullptr;
    a.advance = sum && sum->k_new ? (sum->advance != 0) : 0;
    a.partial = reinterpret_cast<float *>(static_cast<unsigned char *>(ws) + w.partial);
    a.lens = reinterpret_cast<int32_t *>(static_cast<unsigned char *>(ws) + w.lens);
    a.R = ps->num_reqs;
    a.Hkv = kv->num_kv_heads;
    a.max_pages = ps->max_pages;
    a.pool_pages = kv->pool_pages;
    a.max_chunks = w.max_chunks;
    a.slots = w.slots;
    a.chunk_pages = w.chunk_pages;
    a.qscale = scale * 1.4426950408889634f;
    return from_hip(launch_decode(kv->dtype, kv->head_dim, num_q_heads / kv->num_kv_heads, a, stages, stream));
}

}  // namespace

gp_status_t gp_decode_attention(const gp_kv_layer_t *kv, const gp_page_state_t *ps, const void *q_post,
                                int32_t num_q_heads, float scale, void *out, void *ws, size_t ws_bytes,
                                hipStream_t stream) {
    return decode_call(kv, ps, q_post, num_q_heads, scale, out, ws, ws_bytes, nullptr,
                       GP_DECODE_CHUNKS | GP_DECODE_MERGE, stream);
}

gp_status_t gp_decode_attention_noalloc(const gp_kv_layer_t *kv, const gp_page_state_t *ps,
                                        const void *q_post, int32_t num_q_heads, float scale, void *out,
                                        hipStream_t stream) {
    return decode_call(kv, ps, q_post, num_q_heads, scale, out, nullptr, 0, nullptr,
                       GP_DECODE_CHUNKS | GP_DECODE_MERGE, stream, true);
}

gp_status_t gp_decode_attention_shared(const gp_kv_layer_t *kv, const gp_page_state_t *ps,
                                       const void *q_post, int32_t num_q_heads, float scale, void *out,
                                       const gp_prefix_group_t *groups, int32_t num_groups, int32_t stages,
                                       void *ws, size_t ws_bytes, hipStream_t stream) {
    if (num_groups < 0 || (num_groups > 0 && !groups)) return GP_ERR_INVALID;
    if (stages < 1 || stages > (GP_DECODE_PREFIX | GP_DECODE_CHUNKS | GP_DECODE_MERGE)) return GP_ERR_INVALID;
    // without groups it is plain decode attention (no prefix stage)
    return decode_call(kv, ps, q_post, num_q_heads, scale, out, ws, ws_bytes, nullptr, stages, stream, false,
                       groups, num_groups);
}

gp_status_t gp_decode_attention_stages(const gp_kv_layer_t *kv, const gp_page_state_t *ps, const void *q_post,
                                       int32_t num_q_heads, float scale, void *out, int32_t stages, void *ws,
                                       size_t ws_bytes, hipStream_t stream) {
    if (stages < 1 || stages > (GP_DECODE_CHUNKS | GP_DECODE_MERGE)) return GP_ERR_INVALID;
    return decode_call(kv, ps, q_post, num_q_heads, scale, out, ws, ws_bytes, nullptr, stages, stream);
}

gp_status_t gp_decode_step(const gp_kv_layer_t *kv, const gp_page_state_t *ps, const void *q_post,
                           const void *q_pre, int32_t num_q_heads, float scale, void *out,
                           const int32_t *slot_ids, const uint8_t *init, float *qstate, int32_t num_slots,
                           float beta_s, float beta_l, const void *k_new, const void *v_new,
                           int32_t *positions, int32_t advance, void *ws, size_t ws_bytes,
                           hipStream_t stream) {
    const FoldedSummaries sum{q_pre, slot_ids, init, qstate, num_slots, beta_s, beta_l,
                              k_new, v_new, positions, advance};
    return decode_call(kv, ps, q_post, num_q_heads, scale, out, ws, ws_bytes, &sum,
                       GP_DECODE_CHUNKS | GP_DECODE_MERGE, stream);
}

gp_status_t gp_boundary_score_stages(const gp_kv_layer_t *kv, const gp_page_state_t *ps, const void *q_pre,
                                     const float *qstate, int32_t num_slots, const int32_t *slot_ids,
                                     const int32_t *positions, const int32_t *bnd, int32_t num_bnd,
                                     int32_t num_q_heads, const gp_params_t *params, int32_t *k_counts,
                                     float *scores, int32_t max_cand, void *ws, size_t ws_bytes,
                                     hipStream_t stream, int32_t stages) {
    if (stages <= 0 || (stages & ~(GP_SCORE_WEIGHTS | GP_SCORE_COUNTS)) != 0) return GP_ERR_INVALID;
    gp_status_t st = check_layer(kv);
    if (st != GP_OK) return st;
    if ((st = check_state(ps, kv)) != GP_OK) return st;
    if (!dims_ok(num_q_heads, kv->num_kv_heads, kv->head_dim)) return GP_ERR_UNSUPPORTED;
    if (!params || num_bnd < 0 || num_slots <= 0) return GP_ERR_INVALID;
    if (num_bnd == 0) return GP_OK;
    if (!q_pre || !qstate || !slot_ids || !positions || !bnd || !k_counts || !scores || !ws)
        return GP_ERR_INVALID;
    if (max_cand < (ps->max_pages - 1) * kPage) return GP_ERR_INVALID;
    if (!(params->p > 0.0f && params->p <= 1.0f) || !(params->scale > 0.0f) ||
        !(params->rope_theta > 0.0f))
        return GP_ERR_INVALID;
    if (params->metric != GP_METRIC_TOP_P && params->metric != GP_METRIC_ENTROPY) return GP_ERR_INVALID;
    if (num_bnd > 65535 || ps->max_pages > kMaxBoundaryPages) return GP_ERR_UNSUPPORTED;
    const ScoreWs w = score_ws(num_bnd, num_q_heads, kv->num_kv_heads, ps->max_pages);
    if (ws_bytes < w.total) return GP_ERR_WORKSPACE;
    ScoreArgs a;
    unsigned char *base = static_cast<unsigned char *>(ws);
    a.k = kv->k;
    a.page_table = ps->page_table;
    a.num_pages = ps->num_pages;
    a.seq_lens = ps->seq_lens;
    a.q_pre = q_pre;
    a.qstate = qstate;
    a.slot_ids = slot_ids;
    a.positions = positions;
    a.bnd = bnd;
    a.k_counts = k_counts;
    a.scores = scores;
    a.cand = reinterpret_cast<int32_t *>(base + w.cand);
    a.expz = reinterpret_cast<float *>(base + w.expz);
    a.part = reinterpret_cast<double *>(base + w.part);
    a.weights = reinterpret_cast<float *>(base + w.weights);
    a.Rb = num_bnd;
    a.Hq = num_q_heads;
    a.Hkv = kv->num_kv_heads;
    a.M = num_slots;
    a.max_pages = ps->max_pages;
    a.pool_pages = kv->pool_pages;
    a.max_cand = max_cand;
    a.cmax = w.cmax;
    a.nch = w.nch;
    a.R = ps->num_reqs;
    a.scale = params->scale;
    a.theta = params->rope_theta;
    a.p = params->p;
    a.metric = params->metric;
    return from_hip(launch_score(kv->dtype, kv->head_dim, num_q_heads / kv->num_kv_heads, a, stages, stream));
}

gp_status_t gp_boundary_score(const gp_kv_layer_t *kv, const gp_page_state_t *ps, const void *q_pre,
                              const float *qstate, int32_t num_slots, const int32_t *slot_ids,
                              const int32_t *positions, const int32_t *bnd, int32_t num_bnd,
                              int32_t num_q_heads, const gp_params_t *params, int32_t *k_counts,
                              float *scores, int32_t max_cand, void *ws, size_t ws_bytes,
                              hipStream_t stream) {
    return gp_boundary_score_stages(kv, ps, q_pre, qstate, num_slots, slot_ids, positions, bnd, num_bnd,
                                    num_q_heads, params, k_counts, scores, max_cand, ws, ws_bytes, stream,
                                    GP_SCORE_WEIGHTS | GP_SCORE_COUNTS);
}

namespace {

gp_status_t apply_call(const gp_kv_layer_t *layers, int32_t n_layers, const gp_page_state_t *ps,
                       const int32_t *bnd, int32_t num_bnd, const int32_t *k_counts, const float *scores,
                       int32_t max_cand, const gp_params_t *params, int32_t *decisions, float *delta,
                       int64_t *counters, void *ws, size_t ws_bytes, hipStream_t stream, int stages,
                       int hold) {
    if (!layers || n_layers <= 0 || !params || num_bnd < 0) return GP_ERR_INVALID;
    if (n_layers > kMaxLayers) return GP_ERR_UNSUPPORTED;
    gp_status_t st;
    for (int l = 0; l < n_layers; ++l) {
        if ((st = check_layer(&layers[l])) != GP_OK) return st;
        if (layers[l].pool_pages != layers[0].pool_pages || layers[l].num_kv_heads != layers[0].num_kv_heads ||
            layers[l].head_dim != layers[0].head_dim || layers[l].dtype != layers[0].dtype)
            return GP_ERR_INVALID;
    }
    if ((st = check_state(ps, &layers[0])) != GP_OK) return st;
    if (num_bnd == 0) return GP_OK;
    if (!ps->refcount || !ps->free_list || !ps->free_count) return GP_ERR_INVALID;
    if (!bnd || !k_counts || !scores || !decisions || !delta || !counters || !ws) return GP_ERR_INVALID;
    if (max_cand < (ps->max_pages - 1) * kPage) return GP_ERR_INVALID;
    if (params->k_loc < 0 || params->reserve_pages < 0) return GP_ERR_INVALID;
    if (params->policy < GP_POLICY_GROWPAGE || params->policy > GP_POLICY_SHRINK) return GP_ERR_INVALID;
    if (params->policy == GP_POLICY_RANDOM &&
        (!params->draws || !(params->compress_prob >= 0.0f && params->compress_prob <= 1.0f)))
        return GP_ERR_INVALID;
    if (params->policy == GP_POLICY_SHRINK && !isfinite(params->shrink_threshold)) return GP_ERR_INVALID;
    if (params->layout != GP_LAYOUT_SHIFT && params->layout != GP_LAYOUT_FILL) return GP_ERR_INVALID;
    if (num_bnd > 2048 || ps->max_pages > kMaxBoundaryPages) return GP_ERR_UNSUPPORTED;
    const gp_kv_layer_t &L0 = layers[0];
    const int E = elem_bytes(L0.dtype);
    const ApplyWs w = apply_ws(num_bnd, L0.num_kv_heads, L0.head_dim, E, ps->max_pages, n_layers);
    if (ws_bytes < w.total) return GP_ERR_WORKSPACE;
    unsigned char *base = static_cast<unsigned char *>(ws);
    ApplyArgs a;
    a.page_table = ps->page_table;
    a.num_pages = ps->num_pages;
    a.seq_lens = ps->seq_lens;
    a.refcount = ps->refcount;
    a.free_list = ps->free_list;
    a.free_count = ps->free_count;
    a.bnd = bnd;
    a.k_counts = k_counts;
    a.scores = scores;
    a.decisions = decisions;
    a.delta = delta;
    a.counters = reinterpret_cast<long long *>(counters);
    a.req = reinterpret_cast<int32_t *>(base + w.req);
    a.hdr = reinterpret_cast<int32_t *>(base + w.hdr);
    a.nshc = reinterpret_cast<int32_t *>(base + w.nshc);
    a.shflag = base + w.shflag;
    a.old_table = reinterpret_cast<int32_t *>(base + w.old_table);
    a.released = reinterpret_cast<int32_t *>(base + w.released);
    a.evict = reinterpret_cast<int32_t *>(base + w.evict);
    a.border = base + w.border;
    a.R = ps->num_reqs;
    a.Rb = num_bnd;
    a.Hkv = L0.num_kv_heads;
    a.max_pages = ps->max_pages;
    a.pool_pages = ps->pool_pages;
    a.max_cand = max_cand;
    a.n_layers = n_layers;
    a.ncc = w.ncc;
    a.npc = w.npc;
    a.k_loc = params->k_loc;
    a.reserve = params->reserve_pages;
    a.tau = params->tau;
    a.policy = params->policy;
    a.fixed_pages = params->fixed_pages;
    a.min_cap = params->min_capacity_pages;
    a.compress_prob = params->compress_prob;
    a.shrink_threshold = params->shrink_threshold;
    a.draws = params->draws;
    a.layout = params->layout;
    a.hold = hold;
    // the whole apply takes its counts as inputs: they are final when it runs
    a.skip_grows = stages == (kStageSelect | kStageDecide | kStageCompact) ? 1 : params->select_skip_grows != 0;
    LayerPtrs lp[kMaxLayers];
    for (int l = 0; l < n_layers; ++l) {
        lp[l].k = layers[l].k;
        lp[l].v = layers[l].v;
    }
    return from_hip(launch_apply(L0.dtype, L0.head_dim, a, lp, stages, stream));
}

}  // namespace

#define GP_APPLY_ARGS                                                                              \
    const gp_kv_layer_t *layers, int32_t n_layers, const gp_page_state_t *ps, const int32_t *bnd, \
        int32_t num_bnd, const int32_t *k_counts, const float *scores, int32_t max_cand,          \
        const gp_params_t *params, int32_t *decisions, float *delta, int64_t *counters, void *ws,  \
        size_t ws_bytes, hipStream_t stream
#define GP_APPLY_PASS                                                                                \
    layers, n_layers, ps, bnd, num_bnd, k_counts, scores, max_cand, params, decisions, delta, counters, \
        ws, ws_bytes, stream

gp_status_t gp_boundary_apply(GP_APPLY_ARGS) {
    return apply_call(GP_APPLY_PASS, kStageSelect | kStageDecide | kStageCompact, 0);
}

gp_status_t gp_boundary_select(GP_APPLY_ARGS) { return apply_call(GP_APPLY_PASS, kStageSelect, 0); }

gp_status_t gp_boundary_decide(GP_APPLY_ARGS, int32_t hold) {
    return apply_call(GP_APPLY_PASS, kStageDecide, hold != 0);
}

gp_status_t gp_boundary_compact(GP_APPLY_ARGS) { return apply_call(GP_APPLY_PASS, kStageCompact, 0); }

gp_status_t gp_append_step(const gp_kv_layer_t *layers, int32_t n_layers, const gp_page_state_t *ps,
                           int32_t *positions, const void *k_new, const void *v_new, const void *q_pre,
                           int32_t num_q_heads, const int32_t *slot_ids, const uint8_t *init,
                           float *qstate, int32_t num_slots, float beta_s, float beta_l,
                           hipStream_t stream) {
    if (!layers || n_layers <= 0) return GP_ERR_INVALID;
    if (n_layers > kMaxLayers) return GP_ERR_UNSUPPORTED;
    gp_status_t st;
    for (int l = 0; l < n_layers; ++l) {
        if ((st = check_layer(&layers[l])) != GP_OK) return st;
        if (layers[l].pool_pages != layers[0].pool_pages || layers[l].num_kv_heads != layers[0].num_kv_heads ||
            layers[l].head_dim != layers[0].head_dim || layers[l].dtype != layers[0].dtype)
            return GP_ERR_INVALID;
    }
    if ((st = check_state(ps, &layers[0])) != GP_OK) return st;
    if (!dims_ok(num_q_heads, layers[0].num_kv_heads, layers[0].head_dim)) return GP_ERR_UNSUPPORTED;
    if (!(beta_s >= 0.0f && beta_s <= 1.0f) || !(beta_l >= 0.0f && beta_l <= 1.0f) || num_slots <= 0)
        return GP_ERR_INVALID;
    if (ps->num_reqs == 0) return GP_OK;
    if (!positions || !k_new || !v_new || !q_pre || !slot_ids || !qstate) return GP_ERR_INVALID;
    AppendArgs a;
    for (int l = 0; l < kMaxLayers; ++l) {
        a.k[l] = l < n_layers ? layers[l].k : nullptr;
        a.v[l] = l < n_layers ? layers[l].v : nullptr;
    }
    a.page_table = ps->page_table;
    a.num_pages = ps->num_pages;
    a.seq_lens = ps->seq_lens;
    a.positions = positions;
    a.k_new = k_new;
    a.v_new = v_new;
    a.q_pre = q_pre;
    a.slot_ids = slot_ids;
    a.init = init;
    a.qstate = qstate;
    a.R = ps->num_reqs;
    a.Hq = num_q_heads;
    a.Hkv = layers[0].num_kv_heads;
    a.M = num_slots;
    a.max_pages = ps->max_pages;
    a.pool_pages = ps->pool_pages;
    a.n_layers = n_layers;
    a.beta_s = beta_s;
    a.beta_l = beta_l;
    return from_hip(launch_append(layers[0].dtype, layers[0].head_dim, a, stream));
}

gp_status_t gp_release_held(const gp_page_state_t *ps, hipStream_t stream) {
    if (!ps || !ps->seq_lens || ps->num_reqs < 0) return GP_ERR_INVALID;
    if (ps->num_reqs == 0) return GP_OK;
    return from_hip(launch_release(ps->seq_lens, ps->num_reqs, stream));
}

}  // extern "C"

// Internal definitions shared by the library's translation units: workspace
// layouts, launch descriptors and small device helpers.  Nothing here is part
// of the public ABI (include/growpage.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "growpage.h"

namespace gp {

constexpr int kPage = 16;                 // tokens per page
#ifndef GP_DECODE_CHUNK_PAGES
#define GP_DECODE_CHUNK_PAGES 64
#endif
#ifndef GP_DECODE_PVM_MIN_G
#define GP_DECODE_PVM_MIN_G 4
#endif
constexpr int kDecodePvmMinG = GP_DECODE_PVM_MIN_G;   // GQA ratios whose decode P.V runs on the matrix cores
constexpr int kDecodeChunkPages = GP_DECODE_CHUNK_PAGES;   // pages per decode work item, about (split-K)
constexpr int kMaxChunkPages = 64;                         // pages per decode chunk at most (LDS id table)
#ifndef GP_DECODE_WAVES
#define GP_DECODE_WAVES 8
#endif
constexpr int kDecodeWaves = GP_DECODE_WAVES;              // waves per decode workgroup (bf16 path)
constexpr int kMaxDecodeChunks = 128;                      // chunks one request may span
constexpr int kMaxBoundaryPages = 4096;                    // table width the boundary calls accept
constexpr int kStatBlock = 64;            // candidate tokens per softmax-statistics block (one wave)
constexpr int kProbChunk = 1024;          // tokens per weight/score work item
constexpr int kCompactChunk = 256;        // slots per compaction work item
constexpr int kMaxLayers = 64;            // layers one gp_boundary_apply call can take
constexpr size_t kAlign = 256;

__host__ __device__ inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
__host__ __device__ inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------- layouts --

// One step of the dual-timescale EMA (Sec. 3.2) for one element: the fp64
// value beta * prev + (1 - beta) * x with products and the sum rounded one at
// a time (no fused multiply-add), then rounded once to float32.  Every kernel
// that updates summaries goes through this, so they agree bit for bit.
__device__ inline float ema_step(float prev, float x, double beta, double one_minus_beta) {
#pragma clang fp contract(off)
    const double a = beta * (double)prev;
    const double b = one_minus_beta * (double)x;
    return (float)(a + b);
}

struct DecodeWs {
    size_t partial, lens, total;
    int max_chunks, chunk_pages, slots;
};

// Work split of decode attention: every request is cut into chunks of about
// kDecodeChunkPages pages (sized so that max_pages splits evenly); when a
// request spans several chunks a second kernel merges their partial results.
__host__ __device__ inline int decode_chunk_pages(int max_pages) {
    int chunks = cdiv(max_pages, kDecodeChunkPages);
    if (chunks > kMaxDecodeChunks) chunks = kMaxDecodeChunks;
    return cdiv(max_pages, chunks);
}

__host__ __device__ inline DecodeWs decode_ws(int R, int Hq, int Hkv, int D, int max_pages) {
    DecodeWs w;
    const int G = Hq / Hkv;
    w.chunk_pages = decode_chunk_pages(max_pages);
    w.max_chunks = cdiv(max_pages, w.chunk_pages);
    size_t off = 0;
    // partial slots per (request, KV head): the chunks of the request, plus one
    // more for a shared prefix (its chunks have the decode chunk size, so a
    // request of a prefix group needs at most one slot more than its pages)
    w.slots = w.max_chunks + 1;
    w.partial = off;    // float: [R][Hkv][slots][G][D + 2] (o, max, sum)
    off = align_up(off + (size_t)R * Hkv * w.slots * G * (D + 2) * sizeof(float));
    w.lens = off;       // int32: [R] tokens attended (-1: held), [R] token appended (0/1),
                        //        [R] partial slots the merge folds (0: none)
    off = align_up(off + (size_t)R * 3 * sizeof(int32_t));
    w.total = off;
    return w;
}

struct ScoreWs {
    size_t cand, expz, part, weights, total;
    int cmax, nch;
};

// cmax = (max_pages - 1) * page: the most candidates any request can have.
__host__ __device__ inline ScoreWs score_ws(int Rb, int Hq, int Hkv, int max_pages) {
    ScoreWs w;
    const int G = Hq / Hkv;
    w.cmax = max_pages > 1 ? (max_pages - 1) * kPage : 0;
    w.nch = cdiv(w.cmax > 0 ? w.cmax : 1, kStatBlock);
    size_t off = 0;
    w.cand = off;     // [Rb] int32: candidates of the event (0: not a boundary), written by the logits
    off = align_up(off + (size_t)Rb * sizeof(int32_t));
    w.expz = off;     // [Rb][Hkv][2G][cmax] float: exp(z - block max), z the fp64 logit
    off = align_up(off + (size_t)Rb * Hkv * 2 * G * w.cmax * sizeof(float));
    w.part = off;     // [Rb][Hkv][nch][2G][2] double: block max, block sum of exp
    off = align_up(off + (size_t)Rb * Hkv * w.nch * 2 * G * 2 * sizeof(double));
    w.weights = off;  // [Rb][Hkv][2][cmax] float
    off = align_up(off + (size_t)Rb * Hkv * 2 * w.cmax * sizeof(float));
    w.total = off;
    return w;
}

struct ApplyWs {
    size_t req, hdr, nshc, shflag, old_table, released, evict, border, total;
    int ncc, npc;
};

// Per boundary request scratch (int32 fields).
// RQ_SKIP: written by the selection, 1 if it skipped the request as a
// certain grow (its lists and border rows were not made).
enum { RQ_R = 0, RQ_P, RQ_FLAGS, RQ_NSH, RQ_POP, RQ_DEC, RQ_SKIP, RQ_STRIDE = 8 };
// Call header (int32): free count before pops, after pops, released pages.
enum { HDR_FC0 = 0, HDR_FC1, HDR_NREL, HDR_SIZE = 4 };
constexpr int kPageBlock = 1024;  // pages per work item when walking a page-table row
// Eviction lists per (layer, boundary request, KV head): slots [0, 16) for a
// Compress & Hold, [16, 48) for a shrink.  Rows move down by at most 32 slots.
constexpr int kShrinkEvict = 2 * kPage;
constexpr int kEvictSlots = kPage + kShrinkEvict;
constexpr int kBorderRows = kShrinkEvict;
constexpr int kBordersPerGroup = 4;   // chunk boundaries whose border rows one workgroup saves

__host__ __device__ inline ApplyWs apply_ws(int Rb, int Hkv, int D, int elem, int max_pages,
                                            int n_layers) {
    ApplyWs w;
    w.ncc = cdiv(max_pages * kPage, kCompactChunk);
    w.npc = cdiv(max_pages, kPageBlock);
    size_t off = 0;
    w.req = off;        // [Rb][RQ_STRIDE]
    off = align_up(off + (size_t)Rb * RQ_STRIDE * sizeof(int32_t));
    w.hdr = off;        // [HDR_SIZE]
    off = align_up(off + HDR_SIZE * sizeof(int32_t));
    w.nshc = off;       // [Rb][npc] shared pages per block of the table row
    off = align_up(off + (size_t)Rb * w.npc * sizeof(int32_t));
    w.shflag = off;     // [Rb][max_pages] uint8: page shared when the call starts
    off = align_up(off + (size_t)Rb * max_pages);
    w.old_table = off;  // [Rb][max_pages]
    off = align_up(off + (size_t)Rb * max_pages * sizeof(int32_t));
    w.released = off;   // [Rb * max_pages]
    off = align_up(off + (size_t)Rb * max_pages * sizeof(int32_t));
    w.evict = off;      // [L][Rb][Hkv][kEvictSlots]
    off = align_up(off + (size_t)n_layers * Rb * Hkv * kEvictSlots * sizeof(int32_t));
    w.border = off;     // [L][Rb][Hkv][ncc][2][kBorderRows][D] elements
    off = align_up(off + (size_t)n_layers * Rb * Hkv * w.ncc * 2 * kBorderRows * D * elem);
    w.total = off;
    return w;
}

// ------------------------------------------------------------ launch args --

constexpr int kMaxPrefixGroups = 16;      // prefix groups one shared decode call takes
constexpr int kPrefixWaves = 4;           // waves per workgroup of the shared-prefix pass

struct DecodeArgs {
    const void *k, *v;
    const int32_t *page_table, *num_pages, *seq_lens;
    const void *q;
    void *out;
    // summary update folded into the launch (gp_decode_step); qstate == nullptr: none
    const void *q_pre;
    const int32_t *slot_ids;
    const uint8_t *init;
    float *qstate;
    int M;
    double beta_s, beta_l;
    // the step's new token folded into the launch (gp_decode_step with k_new):
    // written at slot m_r of every request with room and attended to; with
    // advance != 0 the merge pass then advances seq_lens and positions
    void *k_w, *v_w;              // the pools, written at the new token's slot
    const void *k_new, *v_new;    // [R][Hkv][D]; nullptr: no token
    int32_t *seq_lens_w, *positions;
    int advance;
    float *partial;
    int32_t *lens;                // [R] tokens attended (-1: held), [R] appended flags, [R] merge slots
    // shared-prefix decode (gp_decode_attention_shared): requests
    // [g_first, g_first + g_num) share the first g_pages pages of g_first's
    // table; workgroup blocks [g_blk0[g], g_blk0[g + 1]) of the prefix pass
    int ngroups;
    int g_first[kMaxPrefixGroups], g_num[kMaxPrefixGroups], g_pages[kMaxPrefixGroups];
    int g_blk0[kMaxPrefixGroups + 1];
    int R, Hkv, max_pages, pool_pages, max_chunks, chunk_pages, slots;
    float qscale;   // scale * log2(e)
};

struct SummaryArgs {
    const void *q;
    const int32_t *slot_ids;
    const uint8_t *init;
    float *qstate;
    int R, HqD, M;
    double beta_s, beta_l;
};

struct AppendArgs {
    void *k[kMaxLayers];
    void *v[kMaxLayers];
    int32_t *page_table, *num_pages, *seq_lens, *positions;
    const void *k_new, *v_new, *q_pre;
    const int32_t *slot_ids;
    const uint8_t *init;
    float *qstate;
    int R, Hq, Hkv, M, max_pages, pool_pages, n_layers;
    double beta_s, beta_l;
};

struct ScoreArgs {
    const void *k;
    const int32_t *page_table, *num_pages, *seq_lens;
    const void *q_pre;
    const float *qstate;
    const int32_t *slot_ids, *positions, *bnd;
    int32_t *k_counts;
    float *scores;
    double *part;
    int32_t *cand;    // [Rb] candidates per event, 0 if the entry is not a boundary (logits -> later kernels)
    float *expz;
    float *weights;
    int Rb, Hq, Hkv, M, max_pages, pool_pages, max_cand, cmax, nch, R;
    double scale, theta, p;
    int metric;       // GP_METRIC_*
    int lg_iters;     // statistics blocks per logits workgroup (set at launch)
};

struct ApplyArgs {
    int32_t *page_table, *num_pages, *seq_lens, *refcount, *free_list, *free_count;
    const int32_t *bnd, *k_counts;
    const float *scores;
    int32_t *decisions;
    float *delta;
    long long *counters;
    int32_t *req, *hdr, *nshc, *old_table, *released, *evict;
    uint8_t *shflag;
    unsigned char *border;
    int R, Rb, Hkv, max_pages, pool_pages, max_cand, n_layers, ncc, npc, k_loc, reserve;
    double tau;
    // policy variant (GP_POLICY_*) and its constants
    int policy, fixed_pages, min_cap;
    float compress_prob;
    double shrink_threshold;
    const float *draws;
    int layout;       // GP_LAYOUT_*
    int hold;         // mark compressing requests held (negative seq_len)
    int skip_grows;   // the selection may skip requests whose decision can only be a grow
};

struct LayerPtrs {
    void *k, *v;
};

// ---------------------------------------------------------------- launchers --

hipError_t launch_summaries(gp_dtype_t dt, const SummaryArgs &a, hipStream_t s);
hipError_t launch_append(gp_dtype_t dt, int D, const AppendArgs &a, hipStream_t s);
hipError_t launch_decode(gp_dtype_t dt, int D, int G, const DecodeArgs &a, int stages, hipStream_t s);
hipError_t launch_score(gp_dtype_t dt, int D, int G, const ScoreArgs &a, int stages, hipStream_t s);
// Stages of the boundary apply (selection, decision, compaction).
constexpr int kStageSelect = 1, kStageDecide = 2, kStageCompact = 4;

hipError_t launch_apply(gp_dtype_t dt, int D, const ApplyArgs &a, const LayerPtrs *layers, int stages,
                        hipStream_t s);
hipError_t launch_release(int32_t *seq_lens, int R, hipStream_t s);
hipError_t launch_stream_read(const void *src, size_t bytes, uint32_t *out, hipStream_t s);

// ---------------------------------------------------------- device helpers --

__device__ inline float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ inline float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }
__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bfloat16, round to nearest even; NaN stays NaN.
__device__ inline uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)0x7fc0;
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

}  // namespace gp

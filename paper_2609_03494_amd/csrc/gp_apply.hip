// Capacity decision, page allocation, selection and compaction at capacity
// boundaries (Sec. 3.2 aggregation and threshold, Sec. 3.3 Compress & Hold /
// Grow by One Page, Sec. 4.2 fallback, App. E.2 prefix-preserving compaction).
//
// Five kernels, in stream order:
//  count    per (boundary request, block of 256 table entries): how many of the
//           request's pages are shared (refcount > 1).
//  decide   one workgroup.  Per request, in parallel: Delta from the integer
//           working-set counts (exact sign for tau = 0), want-grow.  Then one
//           thread walks the requests in list order over LDS-resident data to
//           hand out pages from the free stack (grow: 1 page, compress with a
//           shared prefix: one page per shared page), writes the decision and
//           applies grows and the new resident length of compressing requests.
//  replace  per (request, block of 256 entries): a compressing request with
//           shared pages gets its private replacement pages (ranked by logical
//           page) and keeps a copy of its old table row for the copy step.
//  select   per (request, KV head, layer): every candidate page keeps its
//           local quota; the page_size lowest-ranked remaining tokens
//           (score ascending, slot descending) are found with per-thread
//           register lists merged pairwise in LDS.  The same workgroup saves the
//           first rows of every compaction chunk boundary ("border" rows) that a
//           neighbouring chunk will overwrite, and (head 0, layer 0) drops the
//           request's references to replaced shared pages.
//  compact  per (chunk of 256 slots, KV head x layer, request): reads every row
//           that moves (the border rows from the saved copy), then writes it to
//           its new slot; rows move down by at most page_size slots, so the only
//           cross-chunk hazard is covered by the border copy.  Workgroup 0 also
//           pushes the pages whose count reached zero, in page-id order.
//
// Bound: compaction is HBM-bound: 2 (K, V) x 2 (read + write) x d x elem bytes
// per moved row and KV head; everything else is latency-bound bookkeeping.
#include "gp_internal.h"

namespace gp {

namespace {

constexpr int kMaxBnd = 2048;

struct LayerTable {
    void *k[kMaxLayers];
    void *v[kMaxLayers];
};

__device__ inline bool compressing(int dec) { return dec == GP_COMPRESS || dec == GP_FALLBACK; }

// ---------------------------------------------------------------- prepare --
// Grid (compaction chunk cc, KV head x layer, boundary request), run before the
// page table changes.  Every workgroup saves the rows of the page just below
// compaction-chunk boundary cc (K and V of its head and layer); a neighbouring
// chunk's writes may land there before the chunk that owns them has read them.
// Workgroups of head 0, layer 0 and cc < npc also count the shared pages in
// block cc of the request's table row.
template <int D, int E>
__global__ __launch_bounds__(256) void prepare_kernel(ApplyArgs a, LayerTable lt) {
    __shared__ int s_n;
    const int cc = blockIdx.x, i = blockIdx.z;
    const int h = blockIdx.y % a.Hkv, l = blockIdx.y / a.Hkv;
    const int tid = threadIdx.x;
    const int r = a.bnd[i];
    int P = 0;
    bool at_boundary = false;
    if (r >= 0 && r < a.R) {
        P = a.num_pages[r];
        at_boundary = P >= 2 && P <= a.max_pages && a.seq_lens[r] == P * kPage;
    }
    const int32_t *row = a.page_table + (size_t)(at_boundary ? r : 0) * a.max_pages;
    if (blockIdx.y == 0 && cc < a.npc) {
        if (tid == 0) s_n = 0;
        __syncthreads();
        const int j = cc * kPageBlock + tid;
        if (at_boundary && j < P) {
            const int pid = row[j];
            if (pid >= 0 && pid < a.pool_pages && a.refcount[pid] > 1) atomicAdd(&s_n, 1);
        }
        __syncthreads();
        if (tid == 0) a.nshc[(size_t)i * a.npc + cc] = s_n;
    }
    if (!at_boundary || cc == 0 || cc >= cdiv(P * kPage, kCompactChunk)) return;
    constexpr int UPP = D * E / 16 * kPage;          // 16-byte units per page slice
    const int lp = cc * kCompactChunk / kPage - 1;
    const int phys = row[lp];
    if (phys < 0 || phys >= a.pool_pages) return;
    const size_t src_off = (size_t)phys * a.Hkv * kPage * D * E + (size_t)h * kPage * D * E;
    unsigned char *bd = a.border + ((((size_t)l * a.Rb + i) * a.Hkv + h) * a.ncc + cc) * 2 * kPage * D * E;
    const unsigned char *kp = reinterpret_cast<const unsigned char *>(lt.k[l]) + src_off;
    const unsigned char *vp = reinterpret_cast<const unsigned char *>(lt.v[l]) + src_off;
    for (int u = tid; u < UPP; u += 256) {
        const uint4 kx = *reinterpret_cast<const uint4 *>(kp + (size_t)u * 16);
        const uint4 vx = *reinterpret_cast<const uint4 *>(vp + (size_t)u * 16);
        *reinterpret_cast<uint4 *>(bd + (size_t)u * 16) = kx;
        *reinterpret_cast<uint4 *>(bd + (size_t)(UPP + u) * 16) = vx;
    }
}

// ----------------------------------------------------------------- decide --
__global__ __launch_bounds__(1024) void decide_kernel(ApplyArgs a) {
    __shared__ int s_P[kMaxBnd];
    __shared__ int s_flags[kMaxBnd];   // bit 0: at a boundary, bit 1: wants to grow
    __shared__ int s_nsh[kMaxBnd];
    __shared__ int s_dec[kMaxBnd];
    __shared__ int s_pop[kMaxBnd];
    __shared__ long long s_cnt[4];
    __shared__ int s_fc0, s_popped;
    const int tid = threadIdx.x;
    const int Rb = a.Rb;

    for (int i = tid; i < Rb; i += blockDim.x) {
        const int r = a.bnd[i];
        int P = 0, flags = 0, nsh = 0;
        float dl = 0.0f;
        if (r >= 0 && r < a.R) {
            P = a.num_pages[r];
            if (P >= 0 && P <= a.max_pages && a.seq_lens[r] == P * kPage) {
                flags = 1;
                bool want = true;
                if (P >= 2) {
                    long long D = 0;
                    for (int l = 0; l < a.n_layers; ++l)
                        for (int h = 0; h < a.Hkv; ++h) {
                            const int32_t *kc = a.k_counts + (((size_t)l * Rb + i) * a.Hkv + h) * 2;
                            D += (long long)kc[0] - (long long)kc[1];
                        }
                    // Delta = (sum K^S - sum K^L) / (|C| * Hkv * layers); the
                    // quotient is correctly rounded, so its sign is exact.
                    const double denom = (double)(P - 1) * kPage * a.Hkv * a.n_layers;
                    const double dd = (double)D / denom;
                    dl = (float)dd;
                    want = dd > a.tau;
                    for (int c = 0; c < a.npc; ++c) nsh += a.nshc[(size_t)i * a.npc + c];
                }
                if (want) flags |= 2;
            }
        }
        a.delta[i] = dl;
        s_P[i] = P;
        s_flags[i] = flags;
        s_nsh[i] = nsh;
    }
    if (tid == 0) {
        const int fc = *a.free_count;
        s_fc0 = fc < 0 ? 0 : (fc > a.pool_pages ? a.pool_pages : fc);
    }
    __syncthreads();

    if (tid == 0) {
        const int fc0 = s_fc0;
        int popped = 0;
        long long cnt[4] = {0, 0, 0, 0};
        for (int i = 0; i < Rb; ++i) {
            const int P = s_P[i], fl = s_flags[i];
            int dec = GP_NOT_BOUNDARY, pop = 0;
            if (fl & 1) {
                const bool want = (fl & 2) != 0;
                const int avail = fc0 - popped;
                const bool can_grow = avail > a.reserve && P < a.max_pages;
                if (want && can_grow) {
                    dec = GP_GROW;
                    pop = popped;
                    popped += 1;
                } else if (P <= 1) {
                    dec = GP_PREEMPT;
                } else if (s_nsh[i] > avail) {
                    dec = GP_PREEMPT;
                } else {
                    dec = want ? GP_FALLBACK : GP_COMPRESS;
                    pop = popped;
                    popped += s_nsh[i];
                }
                cnt[dec] += 1;
            }
            s_dec[i] = dec;
            s_pop[i] = pop;
        }
        s_popped = popped;
        for (int k = 0; k < 4; ++k) s_cnt[k] = cnt[k];
    }
    __syncthreads();

    const int fc0 = s_fc0;
    for (int i = tid; i < Rb; i += blockDim.x) {
        const int dec = s_dec[i], P = s_P[i];
        const int r = a.bnd[i];
        a.decisions[i] = dec;
        int32_t *rq = a.req + (size_t)i * RQ_STRIDE;
        rq[RQ_R] = r;
        rq[RQ_P] = P;
        rq[RQ_FLAGS] = s_flags[i];
        rq[RQ_NSH] = compressing(dec) ? s_nsh[i] : 0;
        rq[RQ_POP] = s_pop[i];
        rq[RQ_DEC] = dec;
        if (dec == GP_GROW) {
            const int pid = a.free_list[fc0 - 1 - s_pop[i]];
            a.page_table[(size_t)r * a.max_pages + P] = pid;
            if (pid >= 0 && pid < a.pool_pages) a.refcount[pid] = 1;
            a.num_pages[r] = P + 1;
        } else if (compressing(dec)) {
            a.seq_lens[r] = (P - 1) * kPage;
        }
    }
    if (tid == 0) {
        a.hdr[HDR_FC0] = fc0;
        a.hdr[HDR_FC1] = fc0 - s_popped;
        *a.free_count = fc0 - s_popped;
        for (int k = 0; k < 4; ++k) a.counters[k] += s_cnt[k];
    }
}

// ---------------------------------------------------------------- replace --
__global__ __launch_bounds__(256) void replace_kernel(ApplyArgs a) {
    __shared__ int s_scan[256];
    const int blk = blockIdx.x, i = blockIdx.y;
    const int32_t *rq = a.req + (size_t)i * RQ_STRIDE;
    if (!compressing(rq[RQ_DEC]) || rq[RQ_NSH] == 0) return;
    const int r = rq[RQ_R], P = rq[RQ_P];
    const int j = blk * kPageBlock + threadIdx.x;
    if (blk * kPageBlock >= P) return;
    int32_t *row = a.page_table + (size_t)r * a.max_pages;
    int shared = 0, old = -1;
    if (j < P) {
        old = row[j];
        shared = (old >= 0 && old < a.pool_pages && a.refcount[old] > 1) ? 1 : 0;
        a.old_table[(size_t)i * a.max_pages + j] = old;
    }
    // rank of this page among the request's shared pages
    int base = 0;
    for (int c = 0; c < blk; ++c) base += a.nshc[(size_t)i * a.npc + c];
    s_scan[threadIdx.x] = shared;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int y = threadIdx.x >= off ? s_scan[threadIdx.x - off] : 0;
        __syncthreads();
        s_scan[threadIdx.x] += y;
        __syncthreads();
    }
    if (shared) {
        const int k = base + s_scan[threadIdx.x] - 1;
        const int pid = a.free_list[a.hdr[HDR_FC0] - 1 - rq[RQ_POP] - k];
        row[j] = pid;
        if (pid >= 0 && pid < a.pool_pages) a.refcount[pid] = 1;
    }
}

// ----------------------------------------------------------------- select --
// Per (boundary request, KV head, layer) of a compressing request: every
// candidate page keeps its q best tokens (score descending, slot ascending);
// the 16 remaining candidates that come last in that order are evicted.
// Eviction order is the ascending order of the 47-bit key
// (score bits << 16) | (0xffff - slot): scores are non-negative floats, so
// their bit patterns sort like their values, and a later slot loses a tie.
// The 16th smallest key is found by a radix select over the key (fields of
// 11, 11, 9 score bits and 11, 5 slot bits), each pass a histogram of the
// keys that share the prefix found so far; wave 0 scans it for the bucket
// that holds the next needed key.  Each pass re-reads the scores (L2-resident).
constexpr int kSelPagesPerThread = 4;
constexpr int kSelThreads = 1024;
constexpr int kSelMaxPages = kSelPagesPerThread * kSelThreads;

__global__ __launch_bounds__(1024) void select_kernel(ApplyArgs a) {
    constexpr int NB = 2048;
    __shared__ unsigned int s_hist[NB];
    __shared__ int s_bucket, s_below, s_nev;
    __shared__ int s_ev[kPage];
    const int h = blockIdx.x, i = blockIdx.y, l = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63;
    const int32_t *rq = a.req + (size_t)i * RQ_STRIDE;
    const int dec = rq[RQ_DEC];
    if (!compressing(dec)) return;
    const int r = rq[RQ_R], P = rq[RQ_P], nsh = rq[RQ_NSH];
    const int32_t *row = a.page_table + (size_t)r * a.max_pages;
    const int32_t *src_row = nsh > 0 ? a.old_table + (size_t)i * a.max_pages : row;

    // the request drops its references to the shared pages it replaced
    if (h == 0 && l == 0 && nsh > 0) {
        for (int j = tid; j < P; j += blockDim.x) {
            const int old = src_row[j];
            if (old != row[j]) {
                const int prev = atomicSub(&a.refcount[old], 1);
                if (prev == 1) a.released[atomicAdd(&a.hdr[HDR_NREL], 1)] = old;
            }
        }
    }

    const int npages = min(P - 1, kSelMaxPages);
    const int Kt = (P - 2) * kPage;
    const int q = P >= 3 ? min(a.k_loc, Kt / (P - 1)) : 0;
    const float *s = a.scores + (((size_t)l * a.Rb + i) * a.Hkv + h) * a.max_cand;

    // local-quota masks of this thread's pages
    uint32_t keep[kSelPagesPerThread];
#pragma unroll
    for (int u = 0; u < kSelPagesPerThread; ++u) {
        const int j = tid + u * kSelThreads;
        uint32_t mask = 0;
        if (j < npages) {
            float v[kPage];
#pragma unroll
            for (int t = 0; t < kPage; ++t) v[t] = s[j * kPage + t];
#pragma unroll
            for (int t = 0; t < kPage; ++t) {
                int rank = 0;
#pragma unroll
                for (int w = 0; w < kPage; ++w) rank += (v[w] > v[t] || (v[w] == v[t] && w < t)) ? 1 : 0;
                mask |= (rank < q ? 1u : 0u) << t;
            }
        }
        keep[u] = mask;
    }

    const int fsh[5] = {36, 25, 16, 5, 0};      // field shifts in the 47-bit key
    const int fbits[5] = {11, 11, 9, 11, 5};
    unsigned long long prefix = 0;
    int need = kPage;                            // keys still to place at or below the prefix
    for (int pass = 0; pass < 5; ++pass) {
        const int sh = fsh[pass], nb = 1 << fbits[pass];
        for (int b = tid; b < nb; b += blockDim.x) s_hist[b] = 0;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kSelPagesPerThread; ++u) {
            const int j = tid + u * kSelThreads;
            if (j >= npages) continue;
            uint32_t sbits[kPage];
#pragma unroll
            for (int t = 0; t < kPage; ++t) sbits[t] = __float_as_uint(s[j * kPage + t]);
#pragma unroll
            for (int t = 0; t < kPage; ++t) {
                if (keep[u] & (1u << t)) continue;
                const unsigned long long key = ((unsigned long long)sbits[t] << 16) |
                                               (unsigned long long)(0xffffu - (uint32_t)(j * kPage + t));
                if ((key >> (sh + fbits[pass])) == prefix) atomicAdd(&s_hist[(key >> sh) & (nb - 1)], 1u);
            }
        }
        __syncthreads();
        if (tid < 64) {
            // lane owns nb/64 consecutive buckets, lane 0 the lowest
            const int per = nb >= 64 ? nb / 64 : 1;
            const int lo = lane * per;
            unsigned int cc = 0;
            for (int k = 0; k < per; ++k) cc += lo + k < nb ? s_hist[lo + k] : 0u;
            unsigned int ic = cc;
            for (int off = 1; off < 64; off <<= 1) {
                const unsigned int y = __shfl_up(ic, off, 64);
                if (lane >= off) ic += y;
            }
            const unsigned int ec = ic - cc;
            if (ec < (unsigned)need && ic >= (unsigned)need) {
                unsigned int cum = ec;
                for (int k = 0; k < per && lo + k < nb; ++k) {
                    if (cum + s_hist[lo + k] >= (unsigned)need) {
                        s_bucket = lo + k;
                        s_below = (int)cum;
                        break;
                    }
                    cum += s_hist[lo + k];
                }
            }
            if (lane == 63 && ic < (unsigned)need) {   // fewer candidates than page_size
                s_bucket = nb - 1;
                s_below = (int)ic;
            }
        }
        __syncthreads();
        need -= s_below;
        prefix = (prefix << fbits[pass]) | (unsigned long long)s_bucket;
        __syncthreads();
    }
    // evict every candidate whose key is at most the threshold key
    if (tid == 0) s_nev = 0;
    if (tid < kPage) s_ev[tid] = -1;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kSelPagesPerThread; ++u) {
        const int j = tid + u * kSelThreads;
        if (j >= npages) continue;
        uint32_t sbits[kPage];
#pragma unroll
        for (int t = 0; t < kPage; ++t) sbits[t] = __float_as_uint(s[j * kPage + t]);
#pragma unroll
        for (int t = 0; t < kPage; ++t) {
            if (keep[u] & (1u << t)) continue;
            const unsigned long long key = ((unsigned long long)sbits[t] << 16) |
                                           (unsigned long long)(0xffffu - (uint32_t)(j * kPage + t));
            if (key <= prefix) {
                const int at = atomicAdd(&s_nev, 1);
                if (at < kPage) s_ev[at] = j * kPage + t;
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        int ev[kPage];
#pragma unroll
        for (int k = 0; k < kPage; ++k) ev[k] = s_ev[k] < 0 ? 0x7fffffff : s_ev[k];
        // ascending slot order (bitonic sorting network, static indices)
#pragma unroll
        for (int k = 2; k <= kPage; k <<= 1)
#pragma unroll
            for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
                for (int x = 0; x < kPage; ++x) {
                    const int y = x ^ j;
                    if (y > x) {
                        const bool up = (x & k) == 0;
                        const int lo = ev[x] < ev[y] ? ev[x] : ev[y];
                        const int hi = ev[x] < ev[y] ? ev[y] : ev[x];
                        ev[x] = up ? lo : hi;
                        ev[y] = up ? hi : lo;
                    }
                }
        int32_t *out = a.evict + (((size_t)l * a.Rb + i) * a.Hkv + h) * kPage;
#pragma unroll
        for (int k = 0; k < kPage; ++k) out[k] = ev[k] == 0x7fffffff ? -1 : ev[k];
    }
}

// ---------------------------------------------------------------- compact --
template <int D, int E>
__global__ __launch_bounds__(256) void compact_kernel(ApplyArgs a, LayerTable lt) {
    constexpr int UPR = D * E / 16;
    constexpr int ROWS = kCompactChunk;
    constexpr int UNITS = ROWS * UPR / 256;         // 16-byte units per thread
    __shared__ int s_ev[kPage];
    __shared__ int s_dst[ROWS];
    __shared__ long long s_src_off[ROWS], s_dst_off[ROWS];
    __shared__ int s_rel[1024];
    const int cc = blockIdx.x, i = blockIdx.z;
    const int h = blockIdx.y % a.Hkv, l = blockIdx.y / a.Hkv;
    const int tid = threadIdx.x;

    if (cc == 0 && blockIdx.y == 0 && i == 0) {
        // pages released by this call go back on the stack, lowest id first
        const int n = a.hdr[HDR_NREL];
        const int fc1 = a.hdr[HDR_FC1];
        for (int base = 0; base < n; base += 1024) {
            for (int k = tid; k < 1024 && base + k < n; k += blockDim.x) s_rel[k] = a.released[base + k];
            __syncthreads();
            for (int k = tid; k < 1024 && base + k < n; k += blockDim.x) {
                const int id = s_rel[k];
                int rank = 0;
                for (int u = 0; u < n; ++u) rank += a.released[u] < id ? 1 : 0;
                if (fc1 + rank < a.pool_pages) a.free_list[fc1 + rank] = id;
            }
            __syncthreads();
        }
        if (tid == 0) {
            *a.free_count = fc1 + n;
            a.hdr[HDR_NREL] = 0;
        }
    }

    const int32_t *rq = a.req + (size_t)i * RQ_STRIDE;
    if (!compressing(rq[RQ_DEC])) return;
    const int r = rq[RQ_R], P = rq[RQ_P], nsh = rq[RQ_NSH];
    const int total = P * kPage;
    const int s0 = cc * ROWS;
    if (s0 >= total) return;
    const int32_t *row = a.page_table + (size_t)r * a.max_pages;
    const int32_t *src_row = nsh > 0 ? a.old_table + (size_t)i * a.max_pages : row;
    if (tid < kPage) s_ev[tid] = a.evict[(((size_t)l * a.Rb + i) * a.Hkv + h) * kPage + tid];
    __syncthreads();

    const size_t page_bytes = (size_t)a.Hkv * kPage * D * E;
    const size_t head_bytes = (size_t)h * kPage * D * E;
    const bool has_border = s0 + ROWS < total;
    {
        const int s = s0 + tid;
        int dst = -1;
        if (s < total) {
            int before = 0;
            bool gone = false;
#pragma unroll
            for (int k = 0; k < kPage; ++k) {
                before += (s_ev[k] >= 0 && s_ev[k] < s) ? 1 : 0;
                gone = gone || s_ev[k] == s;
            }
            if (!gone) {
                const int d = s - before;
                const int sp = src_row[s / kPage], dp = row[d / kPage];
                const bool ok = sp >= 0 && sp < a.pool_pages && dp >= 0 && dp < a.pool_pages;
                const long long so = (long long)sp * page_bytes + head_bytes + (long long)(s % kPage) * D * E;
                const long long dof = (long long)dp * page_bytes + head_bytes + (long long)(d % kPage) * D * E;
                if (ok && so != dof) {
                    dst = d;
                    s_src_off[tid] = so;
                    s_dst_off[tid] = dof;
                }
            }
        }
        s_dst[tid] = dst;
    }
    __syncthreads();

    const unsigned char *bd = a.border + ((((size_t)l * a.Rb + i) * a.Hkv + h) * a.ncc) * 2 * kPage * D * E;
    unsigned char *pools[2] = {reinterpret_cast<unsigned char *>(lt.k[l]),
                               reinterpret_cast<unsigned char *>(lt.v[l])};
#pragma unroll
    for (int kv = 0; kv < 2; ++kv) {
        unsigned char *pool = pools[kv];
        uint4 val[UNITS];
#pragma unroll
        for (int k = 0; k < UNITS; ++k) {
            const int u = k * 256 + tid;
            const int rr = u / UPR, w = u % UPR;
            val[k] = make_uint4(0u, 0u, 0u, 0u);
            if (s_dst[rr] >= 0) {
                if (has_border && rr >= ROWS - kPage) {
                    const unsigned char *src = bd + ((size_t)(cc + 1) * 2 + kv) * kPage * D * E +
                                               (size_t)(rr - (ROWS - kPage)) * D * E + (size_t)w * 16;
                    val[k] = *reinterpret_cast<const uint4 *>(src);
                } else {
                    val[k] = *reinterpret_cast<const uint4 *>(pool + s_src_off[rr] + (size_t)w * 16);
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < UNITS; ++k) {
            const int u = k * 256 + tid;
            const int rr = u / UPR, w = u % UPR;
            if (s_dst[rr] >= 0) *reinterpret_cast<uint4 *>(pool + s_dst_off[rr] + (size_t)w * 16) = val[k];
        }
        __syncthreads();
    }
}

template <int D, int E>
hipError_t launch_de(const ApplyArgs &a, const LayerTable &lt, hipStream_t s) {
    dim3 gprep(a.ncc, a.Hkv * a.n_layers, a.Rb), grep_(a.npc, a.Rb), gsel(a.Hkv, a.Rb, a.n_layers),
        gcomp(a.ncc, a.Hkv * a.n_layers, a.Rb);
    prepare_kernel<D, E><<<gprep, 256, 0, s>>>(a, lt);
    decide_kernel<<<1, 1024, 0, s>>>(a);
    replace_kernel<<<grep_, 256, 0, s>>>(a);
    select_kernel<<<gsel, kSelThreads, 0, s>>>(a);
    compact_kernel<D, E><<<gcomp, 256, 0, s>>>(a, lt);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_apply(gp_dtype_t dt, int D, const ApplyArgs &a, const LayerPtrs *layers,
                        hipStream_t s) {
    if (a.Rb == 0) return hipSuccess;
    LayerTable lt;
    for (int l = 0; l < kMaxLayers; ++l) {
        lt.k[l] = l < a.n_layers ? layers[l].k : nullptr;
        lt.v[l] = l < a.n_layers ? layers[l].v : nullptr;
    }
    if (dt == GP_BF16) return D == 128 ? launch_de<128, 2>(a, lt, s) : launch_de<64, 2>(a, lt, s);
    return D == 128 ? launch_de<128, 4>(a, lt, s) : launch_de<64, 4>(a, lt, s);
}

}  // namespace gp

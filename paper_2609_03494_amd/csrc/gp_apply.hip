// Capacity decision, page allocation, selection and compaction at capacity
// boundaries (Sec. 3.2 aggregation and threshold, Sec. 3.3 Compress & Hold /
// Grow by One Page, Sec. 4.2 fallback, App. E.2 prefix-preserving compaction).
//
// Three kernels, in stream order:
//  pre      grid (KV head x layer, 1 + column groups, boundary request).
//           Column 0 selects, for every request at a boundary, the tokens a
//           compression would evict (the selection needs only the scores, so it
//           does not wait for the decision).  The other columns save the rows
//           just below each compaction-chunk boundary ("border" rows, 16
//           boundaries per workgroup), which a neighbouring chunk may overwrite
//           before their owner reads them, and record which pages of the table
//           row are shared (refcount > 1).
//  decide   one workgroup.  Delta from the integer working-set counts per
//           request in parallel; then one thread walks the requests in list
//           order over LDS-resident data to hand out pages from the free stack
//           (grow: one page; compress with a shared prefix: one page per shared
//           page); then grows are applied, compressing requests get their new
//           resident length, and shared pages are replaced by private ones, the
//           old references dropped (pages reaching zero are listed).
//  compact  per (K or V x KV head x layer, chunk of 256 slots, request): reads every row
//           that moves (the border rows from the saved copy), then writes it to
//           its new slot; in the shift layout rows move down by at most two
//           pages (a shrink), so the only cross-chunk hazard is the one the
//           border copy covers (16 rows, 32 under the Shrink policy).  In the
//           fill layout only the survivors at or above the new resident length
//           move, into evicted slots below it,
//           so no row is written that another chunk reads and chunks with no
//           moving row leave at once.  Workgroup 0 also pushes the released
//           pages back on the stack, lowest id first.
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

// The action boundary request i (P >= 2 pages) wants (Sec. 3.2 aggregation
// and threshold; the policy variants): grow, and under the Shrink policy
// shrink.  D = sum over layers and KV heads of K^S - K^L; Delta = D / denom
// with denom = |C| * Hkv * layers, and thresholds compare exactly as D
// against t * denom (t is a float and denom < 2^29, so the product is exact
// in fp64).  The decision and the selection's grow prediction both use it.
__device__ inline void wanted_action(const ApplyArgs &a, int i, int P, long long D, bool &grow, bool &shrink,
                                     float &dl) {
    const long long denom = (long long)(P - 1) * kPage * a.Hkv * a.n_layers;
    dl = (float)((double)D / (double)denom);
    const bool above = (double)D > a.tau * (double)denom;      // Delta > tau
    shrink = false;
    switch (a.policy) {
        case GP_POLICY_INVERSE: grow = !above; break;
        case GP_POLICY_FIXED: grow = P < a.fixed_pages; break;
        case GP_POLICY_RANDOM: grow = !(a.draws[i] < a.compress_prob); break;
        case GP_POLICY_SHRINK:
            grow = above;
            shrink = (double)D < a.shrink_threshold * (double)denom && P - 1 >= max(a.min_cap, 2);
            break;
        default: grow = above; break;
    }
}

// ----------------------------------------------------------------- select --
// Per (boundary request, KV head, layer): every candidate page keeps its q
// best tokens (score descending, slot ascending); the NEV remaining candidates
// that come last in that order are evicted (NEV = 16 for Compress & Hold, 32
// for a shrink, which keeps K_t = (P - 1 - drop) * 16 tokens).
// Eviction order is the ascending order of the 48-bit key
// (score bits << 16) | (0xffff - slot): scores are non-negative floats, so
// their bit patterns sort like their values, and a later slot loses a tie;
// keys are distinct, so the NEV smallest are one set.  They are found by
// merging sorted lists, with no atomics and one read of every score: each
// thread sorts the candidates of each of its pages (a sorting network over
// the 16 keys, kept tokens as the largest key) and keeps the NEV smallest of
// its pages; the lanes of a wave then merge their lists pairwise over six
// exchange rounds (each merge keeps the NEV smallest of two sorted lists: the
// element-wise minimum of one list and the other reversed, then a bitonic
// clean-up), and wave 0 merges the waves' lists.  The workgroup is one wave
// per SIMD at no more than 128 registers, so that it starts where a decode
// attention workgroup has retired.
constexpr int kSelThreads = 256;
constexpr int kSelMaxPages = 16 * kSelThreads;
constexpr unsigned long long kNoKey = ~0ull;

__device__ inline void load_page_scores(const float *s, int j, uint32_t (&v)[kPage]) {
#pragma unroll
    for (int t = 0; t < kPage; ++t) v[t] = __float_as_uint(s[j * kPage + t]);
}

__device__ inline void cas_asc(unsigned long long &x, unsigned long long &y) {
    const unsigned long long lo = x < y ? x : y, hi = x < y ? y : x;
    x = lo;
    y = hi;
}

// c (a bitonic sequence of N keys) sorted ascending
template <int N>
__device__ inline void bitonic_clean(unsigned long long (&c)[N]) {
#pragma unroll
    for (int st = N / 2; st > 0; st >>= 1)
#pragma unroll
        for (int x = 0; x < N; ++x)
            if ((x & st) == 0) cas_asc(c[x], c[x + st]);
}

// a := the N smallest keys of a and b (both sorted ascending), sorted ascending
template <int N>
__device__ inline void merge_keep(unsigned long long (&a)[N], const unsigned long long (&b)[N]) {
#pragma unroll
    for (int k = 0; k < N; ++k) a[k] = a[k] < b[N - 1 - k] ? a[k] : b[N - 1 - k];
    bitonic_clean<N>(a);
}

template <int NEV>
__device__ void select_tokens(const ApplyArgs &a, int i, int h, int l, int P, int drop, int out_offset) {
    constexpr int NW = kSelThreads / 64;
    __shared__ unsigned long long s_wl[NW][NEV];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int npages = min(P - 1, kSelMaxPages);
    const int Kt = (P - 1 - drop) * kPage;
    const int q = Kt > 0 ? min(a.k_loc, Kt / (P - 1)) : 0;
    const float *s = a.scores + (((size_t)l * a.Rb + i) * a.Hkv + h) * a.max_cand;

    unsigned long long best[NEV];
#pragma unroll
    for (int k = 0; k < NEV; ++k) best[k] = kNoKey;
#pragma unroll 1
    for (int j = tid; j < npages; j += kSelThreads) {
        uint32_t v[kPage];
        load_page_scores(s, j, v);
        // the page's candidates: its q best tokens are kept (no key)
        unsigned long long pk[NEV];
#pragma unroll
        for (int t = 0; t < kPage; ++t) {
            int rank = 0;
#pragma unroll
            for (int w = 0; w < kPage; ++w) {
                const float x = __uint_as_float(v[w]), y = __uint_as_float(v[t]);
                rank += (x > y || (x == y && w < t)) ? 1 : 0;
            }
            pk[t] = rank < q ? kNoKey
                             : ((unsigned long long)v[t] << 16) | (unsigned long long)(0xffffu - (uint32_t)(j * kPage + t));
        }
#pragma unroll
        for (int t = kPage; t < NEV; ++t) pk[t] = kNoKey;
        // sort the page's 16 keys ascending (the padding is already largest)
#pragma unroll
        for (int k = 2; k <= kPage; k <<= 1)
#pragma unroll
            for (int jj = k >> 1; jj > 0; jj >>= 1)
#pragma unroll
                for (int x = 0; x < kPage; ++x) {
                    const int y = x ^ jj;
                    if (y > x) {
                        if ((x & k) == 0) cas_asc(pk[x], pk[y]);
                        else cas_asc(pk[y], pk[x]);
                    }
                }
        merge_keep<NEV>(best, pk);
    }
    // the lanes of the wave: six exchange rounds (both partners keep the merge)
#pragma unroll 1
    for (int off = 1; off < 64; off <<= 1) {
        unsigned long long other[NEV];
#pragma unroll
        for (int k = 0; k < NEV; ++k) other[k] = __shfl_xor(best[k], off, 64);
        merge_keep<NEV>(best, other);
    }
    if (lane == 0) {
#pragma unroll
        for (int k = 0; k < NEV; ++k) s_wl[wave][k] = best[k];
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < NW; ++w) {
            unsigned long long other[NEV];
#pragma unroll
            for (int k = 0; k < NEV; ++k) other[k] = s_wl[w][k];
            merge_keep<NEV>(best, other);
        }
        // the evicted slots, ascending (bitonic sorting network, static indices)
        int ev[NEV];
#pragma unroll
        for (int k = 0; k < NEV; ++k) ev[k] = best[k] == kNoKey ? 0x7fffffff : (int)(0xffffu - (uint32_t)(best[k] & 0xffffu));
#pragma unroll
        for (int k = 2; k <= NEV; k <<= 1)
#pragma unroll
            for (int jj = k >> 1; jj > 0; jj >>= 1)
#pragma unroll
                for (int x = 0; x < NEV; ++x) {
                    const int y = x ^ jj;
                    if (y > x) {
                        const bool up = (x & k) == 0;
                        const int lo = ev[x] < ev[y] ? ev[x] : ev[y];
                        const int hi2 = ev[x] < ev[y] ? ev[y] : ev[x];
                        ev[x] = up ? lo : hi2;
                        ev[y] = up ? hi2 : lo;
                    }
                }
        int32_t *out = a.evict + (((size_t)l * a.Rb + i) * a.Hkv + h) * kEvictSlots + out_offset;
        for (int k = 0; k < NEV; ++k) out[k] = ev[k] == 0x7fffffff ? -1 : ev[k];
    }
    __syncthreads();
}

// -------------------------------------------------------------------- pre --
// SHRINK: the Shrink policy's variant, which also selects the 32 tokens a
// shrink would evict
template <int D, int E, bool SHRINK>
__global__ __launch_bounds__(kSelThreads) __attribute__((amdgpu_waves_per_eu(4))) void pre_kernel(ApplyArgs a, LayerTable lt) {
    __builtin_amdgcn_s_setprio(3);   // issue ahead of co-resident decode waves
    __shared__ int s_n;
    const int x = blockIdx.y, i = blockIdx.z;
    const int h = blockIdx.x % a.Hkv, l = blockIdx.x / a.Hkv;
    const int tid = threadIdx.x;
    __shared__ unsigned long long s_D;
    __shared__ int s_fc;
    // the request's counts and the free count (skip_grows only) are requested
    // with the request index
    long long dpart = 0;
    if (a.skip_grows) {
        for (int e = tid; e < a.n_layers * a.Hkv; e += blockDim.x) {
            const int ll = e / a.Hkv, hh = e % a.Hkv;
            const int32_t *kc = a.k_counts + (((size_t)ll * a.Rb + i) * a.Hkv + hh) * 2;
            dpart += (long long)kc[0] - (long long)kc[1];
        }
        if (tid == 0) s_fc = *a.free_count;
    }
    const int r = a.bnd[i];
    int P = 0;
    bool at_boundary = false;
    if (a.R > 0) {
        // page count and length in one round trip (clamped index)
        const int rc = min(max(r, 0), a.R - 1);
        const int Pr = a.num_pages[rc], m = a.seq_lens[rc];
        at_boundary = (r >= 0) & (r < a.R) & (Pr >= 2) & (Pr <= a.max_pages) & (m == Pr * kPage);
        P = at_boundary ? Pr : 0;
    }
    // A request whose decision can only be a grow needs no eviction lists and
    // no border rows: it wants to grow, has room for one more page, and even
    // if every request before it in the list took max_pages pages the free
    // stack would keep more than reserve_pages (the decision pops only; the
    // stack can only have grown by the time it runs).
    bool skip = false;
    if (a.skip_grows) {
        if (tid == 0) s_D = 0ull;
        __syncthreads();
        if (dpart != 0) atomicAdd(&s_D, (unsigned long long)dpart);
        __syncthreads();
        if (at_boundary) {
            bool grow, shrink;
            float dl;
            wanted_action(a, i, P, (long long)s_D, grow, shrink, dl);
            const long long fc = min(max(s_fc, 0), a.pool_pages);
            skip = grow && P < a.max_pages && fc - (long long)i * a.max_pages > (long long)a.reserve;
        }
    }
    if (blockIdx.x == 0 && x == 0 && tid == 0) a.req[(size_t)i * RQ_STRIDE + RQ_SKIP] = skip ? 1 : 0;
    if (x == 0) {
        if (at_boundary && !skip) {
            select_tokens<kPage>(a, i, h, l, P, 1, 0);
            if constexpr (SHRINK) {
                if (P - 1 >= max(a.min_cap, 2)) select_tokens<kShrinkEvict>(a, i, h, l, P, 2, kPage);
            }
        }
        return;
    }
    const int col = x - 1;
    const int32_t *row = a.page_table + (size_t)(at_boundary ? r : 0) * a.max_pages;
    if (blockIdx.x == 0 && col < a.npc) {
        // shared pages of block col of the table row, as the call starts
        if (tid == 0) s_n = 0;
        __syncthreads();
        for (int j = col * kPageBlock + tid; j < min((col + 1) * kPageBlock, a.max_pages); j += blockDim.x) {
            int shared = 0;
            if (at_boundary && j < P) {
                const int pid = row[j];
                shared = pid >= 0 && pid < a.pool_pages && a.refcount[pid] > 1;
            }
            a.shflag[(size_t)i * a.max_pages + j] = (uint8_t)shared;
            if (shared) atomicAdd(&s_n, 1);
        }
        __syncthreads();
        if (tid == 0) a.nshc[(size_t)i * a.npc + col] = s_n;
    }
    // the fill layout never overwrites a row that another chunk still reads
    if (!at_boundary || skip || a.layout == GP_LAYOUT_FILL) return;
    // Border rows of the chunk boundaries cc in [col * kBordersPerGroup, +kBordersPerGroup)
    // (cc >= 1, below the resident length): the rows just below slot
    // cc * kCompactChunk that the chunk above may overwrite.  Rows move down
    // by at most one page in a Compress & Hold and two in a shrink, so one
    // page is saved, or two under the Shrink policy (in the last pages of the
    // kBorderRows-row buffer).
    constexpr int UPP = D * E / 16 * kPage;          // 16-byte units per page slice
    constexpr int NBP = kBorderRows / kPage;         // pages the buffer holds
    const int nbp = a.policy == GP_POLICY_SHRINK ? NBP : 1;
    const int cc0 = max(col * kBordersPerGroup, 1);
    const int cc1 = min((col + 1) * kBordersPerGroup, cdiv(P * kPage, kCompactChunk));
    if (cc0 >= cc1) return;
    const int per_cc = 2 * nbp * UPP;                 // units saved per boundary
    unsigned char *bd0 = a.border + (((size_t)l * a.Rb + i) * a.Hkv + h) * a.ncc * 2 * kBorderRows * D * E;
    const unsigned char *kpool = reinterpret_cast<const unsigned char *>(lt.k[l]);
    const unsigned char *vpool = reinterpret_cast<const unsigned char *>(lt.v[l]);
    // the page ids of the saved pages first (one round trip), then each
    // thread's units in batches whose loads are all in flight before their
    // stores (beside decode attention every round trip costs microseconds)
    __shared__ int s_bp[kBordersPerGroup * NBP];
    for (int k = tid; k < (cc1 - cc0) * nbp; k += blockDim.x) {
        const int cc = cc0 + k / nbp, pg = k % nbp;
        const int phys = row[cc * kCompactChunk / kPage - nbp + pg];
        s_bp[k] = phys >= 0 && phys < a.pool_pages ? phys : -1;
    }
    __syncthreads();
    // (four units per thread per batch, in named registers: as an array the
    // compiler moved them to LDS)
    const int total = (cc1 - cc0) * per_cc;
    auto unit = [&](int u, int &at) -> const uint4 * {
        const int uc = min(u, total - 1);
        const int c = uc / per_cc, uu = uc % per_cc;
        const int kv = uu / (nbp * UPP), rem = uu % (nbp * UPP), pg = rem / UPP, w = rem % UPP;
        const int phys = s_bp[c * nbp + pg];
        at = u < total && phys >= 0 ? (((cc0 + c) * 2 + kv) * NBP + (NBP - nbp + pg)) * UPP + w : -1;
        const size_t src_off = (size_t)max(phys, 0) * a.Hkv * kPage * D * E + (size_t)h * kPage * D * E;
        return reinterpret_cast<const uint4 *>((kv ? vpool : kpool) + src_off + (size_t)w * 16);
    };
    const int nt = blockDim.x;
    for (int base = tid; base < total; base += 4 * nt) {
        int a0, a1, a2, a3;
        const uint4 v0 = *unit(base, a0), v1 = *unit(base + nt, a1);
        const uint4 v2 = *unit(base + 2 * nt, a2), v3 = *unit(base + 3 * nt, a3);
        if (a0 >= 0) *reinterpret_cast<uint4 *>(bd0 + (size_t)a0 * 16) = v0;
        if (a1 >= 0) *reinterpret_cast<uint4 *>(bd0 + (size_t)a1 * 16) = v1;
        if (a2 >= 0) *reinterpret_cast<uint4 *>(bd0 + (size_t)a2 * 16) = v2;
        if (a3 >= 0) *reinterpret_cast<uint4 *>(bd0 + (size_t)a3 * 16) = v3;
    }
}

// ----------------------------------------------------------------- decide --
// Flags per boundary request: bit 0 at a boundary, bit 1 wants to grow, bit 2
// wants to shrink.
enum { F_BOUNDARY = 1, F_GROW = 2, F_SHRINK = 4, F_SKIPPED = 8 };

__global__ __launch_bounds__(1024) void decide_kernel(ApplyArgs a) {
    __builtin_amdgcn_s_setprio(3);   // issue ahead of co-resident decode waves
    __shared__ int s_P[kMaxBnd];
    __shared__ int s_flags[kMaxBnd];
    __shared__ int s_nsh[kMaxBnd];     // shared pages to replace (after the decision)
    __shared__ int s_nsh_last[kMaxBnd];  // whether the last page is one of them
    __shared__ int s_dec[kMaxBnd];
    __shared__ int s_pop[kMaxBnd];
    __shared__ long long s_cnt[4];
    __shared__ unsigned long long s_D[kMaxBnd];     // sum of K^S - K^L (two's complement)
    __shared__ int s_fc0, s_popped;
    const int tid = threadIdx.x;
    const int Rb = a.Rb;

    // The free count, this thread's first boundary request with its page
    // count and length (clamped index) and its first shared-page count are
    // requested before anything waits: they arrive while the counts below
    // are summed.
    const int fc = tid == 0 ? *a.free_count : 0;
    const int r_first = tid < Rb ? a.bnd[tid] : -1;
    const int rc_first = min(max(r_first, 0), a.R - 1);
    const int P_first = tid < Rb && a.R > 0 ? a.num_pages[rc_first] : 0;
    const int m_first = tid < Rb && a.R > 0 ? a.seq_lens[rc_first] : -1;
    const int nshc_first = tid < Rb * a.npc ? a.nshc[tid] : 0;
    for (int i = tid; i < Rb; i += blockDim.x) {
        s_D[i] = 0;
        s_nsh[i] = 0;
    }
    if (tid == 0) s_fc0 = fc < 0 ? 0 : (fc > a.pool_pages ? a.pool_pages : fc);
    __syncthreads();
    // The per-(layer, KV head) counts and the shared-page counts of every
    // request are summed by the whole workgroup, one entry per thread, so
    // that their loads are in flight together (integer sums: exact in any
    // order).
    const int LH = a.n_layers * a.Hkv;
    for (int e = tid; e < Rb * LH; e += blockDim.x) {
        const int i = e / LH, l = e % LH / a.Hkv, h = e % a.Hkv;
        const int32_t *kc = a.k_counts + (((size_t)l * Rb + i) * a.Hkv + h) * 2;
        atomicAdd(&s_D[i], (unsigned long long)((long long)kc[0] - (long long)kc[1]));
    }
    for (int e = tid; e < Rb * a.npc; e += blockDim.x) {
        const int v = e == tid ? nshc_first : a.nshc[e];
        if (v) atomicAdd(&s_nsh[e / a.npc], v);
    }
    __syncthreads();

    for (int i = tid; i < Rb; i += blockDim.x) {
        const bool first = i == tid;
        const int r = first ? r_first : a.bnd[i];
        int P = 0, flags = 0, nsh = 0, last_shared = 0;
        float dl = 0.0f;
        const int rc = min(max(r, 0), a.R - 1);     // page count and length in one round trip
        const int Pr = first ? P_first : (a.R > 0 ? a.num_pages[rc] : 0);
        const int mr = first ? m_first : (a.R > 0 ? a.seq_lens[rc] : -1);
        if (r >= 0 && r < a.R) {
            P = Pr;
            if (P >= 0 && P <= a.max_pages && mr == P * kPage) {
                flags = F_BOUNDARY;
                bool grow, shrink = false;
                if (P >= 2) {
                    wanted_action(a, i, P, (long long)s_D[i], grow, shrink, dl);
                    nsh = s_nsh[i];
                    last_shared = a.shflag[(size_t)i * a.max_pages + P - 1];
                } else {
                    grow = a.policy == GP_POLICY_FIXED ? P < a.fixed_pages : true;
                }
                if (grow) flags |= F_GROW;
                if (shrink) flags |= F_SHRINK;
                if (a.req[(size_t)i * RQ_STRIDE + RQ_SKIP] != 0) flags |= F_SKIPPED;
            }
        }
        a.delta[i] = dl;
        s_P[i] = P;
        s_flags[i] = flags;
        s_nsh[i] = nsh;
        s_nsh_last[i] = last_shared;
    }
    __syncthreads();

    if (tid == 0) {
        const int fc0 = s_fc0;
        int popped = 0;
        long long cnt[4] = {0, 0, 0, 0};
        for (int i = 0; i < Rb; ++i) {
            const int P = s_P[i], fl = s_flags[i];
            int dec = GP_NOT_BOUNDARY, pop = 0;
            if (fl & F_BOUNDARY) {
                const bool want = (fl & F_GROW) != 0, shrink = (fl & F_SHRINK) != 0;
                const int avail = fc0 - popped;
                const bool can_grow = avail > a.reserve && P < a.max_pages;
                // a shrink keeps pages [0, P - 1) only: the last page needs no copy
                const int nsh = shrink ? s_nsh[i] - s_nsh_last[i] : s_nsh[i];
                if (want && can_grow) {
                    dec = GP_GROW;
                    pop = popped;
                    popped += 1;
                } else if (P <= 1 || nsh > avail || (fl & F_SKIPPED)) {
                    // (a request the selection skipped as a certain grow has
                    // no eviction lists: it is left as it is)
                    dec = GP_PREEMPT;
                } else {
                    dec = shrink ? GP_SHRINK : (want ? GP_FALLBACK : GP_COMPRESS);
                    pop = popped;
                    popped += nsh;
                    s_nsh[i] = nsh;
                }
                cnt[dec == GP_SHRINK ? GP_COMPRESS : dec] += 1;   // a shrink counts as a compression
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
        const bool moves = compressing(dec) || dec == GP_SHRINK;
        a.decisions[i] = dec;
        int32_t *rq = a.req + (size_t)i * RQ_STRIDE;
        rq[RQ_R] = r;
        rq[RQ_P] = P;
        rq[RQ_FLAGS] = s_flags[i];
        rq[RQ_NSH] = moves ? s_nsh[i] : 0;
        rq[RQ_POP] = s_pop[i];
        rq[RQ_DEC] = dec;
        if (dec == GP_GROW) {
            const int pid = a.free_list[fc0 - 1 - s_pop[i]];
            a.page_table[(size_t)r * a.max_pages + P] = pid;
            if (pid >= 0 && pid < a.pool_pages) a.refcount[pid] = 1;
            a.num_pages[r] = P + 1;
        } else if (compressing(dec)) {
            // a held request is left out of decoding until released: -(m + 1)
            const int m = (P - 1) * kPage;
            a.seq_lens[r] = a.hold ? -m - 1 : m;
        } else if (dec == GP_SHRINK) {
            const int m = (P - 2) * kPage;
            a.seq_lens[r] = a.hold ? -m - 1 : m;
            a.num_pages[r] = P - 1;
        }
    }
    if (tid == 0) {
        a.hdr[HDR_FC0] = fc0;
        a.hdr[HDR_FC1] = fc0 - s_popped;
        *a.free_count = fc0 - s_popped;
        for (int k = 0; k < 4; ++k) a.counters[k] += s_cnt[k];
    }

    // Requests whose table row changes: the old row is kept for the copy; a
    // private page replaces each shared page that stays (ranked by logical
    // page) and the old reference is dropped; a shrink also drops the last
    // page.  Pages whose count reaches zero are listed.
    __shared__ int s_scan[1024];
    for (int i = 0; i < Rb; ++i) {
        const int dec = s_dec[i];
        const bool shrink = dec == GP_SHRINK;
        if (!(compressing(dec) && s_nsh[i] > 0) && !shrink) continue;      // uniform
        const int r = a.bnd[i], P = s_P[i];
        const int keep = shrink ? P - 1 : P;
        int32_t *row = a.page_table + (size_t)r * a.max_pages;
        int base = 0;
        for (int j0 = 0; j0 < P; j0 += 1024) {
            const int j = j0 + tid;
            const int sh = j < keep ? a.shflag[(size_t)i * a.max_pages + j] : 0;
            s_scan[tid] = sh;
            __syncthreads();
            for (int off = 1; off < 1024; off <<= 1) {
                const int y = tid >= off ? s_scan[tid - off] : 0;
                __syncthreads();
                s_scan[tid] += y;
                __syncthreads();
            }
            if (j < P) {
                const int old = row[j];
                a.old_table[(size_t)i * a.max_pages + j] = old;
                if (sh) {
                    const int k = base + s_scan[tid] - 1;
                    const int pid = a.free_list[fc0 - 1 - s_pop[i] - k];
                    row[j] = pid;
                    if (pid >= 0 && pid < a.pool_pages) a.refcount[pid] = 1;
                }
                if (sh || (shrink && j == P - 1)) {
                    if (shrink && j == P - 1) row[j] = -1;
                    if (old >= 0 && old < a.pool_pages) {
                        const int prev = atomicSub(&a.refcount[old], 1);
                        if (prev == 1) a.released[atomicAdd(&a.hdr[HDR_NREL], 1)] = old;
                    }
                }
            }
            base += s_scan[1023];
            __syncthreads();
        }
    }
}

// ---------------------------------------------------------------- compact --
// Grid (2 x KV head x layer, chunk of kCompactChunk slots, boundary request):
// the lowest bit of x picks K or V, so each workgroup moves one of them.  The
// kernel sits on the step's critical path and its work is small, so it is
// built around few memory round trips: (1) the decision, the request id and
// both eviction lists, (2) every page-table entry the chunk can need (its
// source pages in the old and the current table row, the destination range of
// the shift layout, the pages of the evicted slots for the fill layout),
// (3) the rows themselves, then the stores.
template <int D, int E>
__global__ __launch_bounds__(256) void compact_kernel(ApplyArgs a, LayerTable lt) {
    __builtin_amdgcn_s_setprio(3);   // issue ahead of co-resident decode waves
    constexpr int UPR = D * E / 16;                 // 16-byte units per row
    constexpr int ROWS = kCompactChunk;
    constexpr int UNITS = ROWS * UPR / 256;         // 16-byte units per thread
    constexpr int PPC = ROWS / kPage;               // pages per chunk
    constexpr int NBP = kShrinkEvict / kPage;       // pages a row can move down by
    __shared__ int s_ev[kShrinkEvict];
    __shared__ int s_dst[ROWS];
    __shared__ long long s_src_off[ROWS], s_dst_off[ROWS];
    __shared__ int s_rel[1024];
    __shared__ int s_src_pg[PPC];                   // source page of each chunk page
    __shared__ int s_lo_pg[NBP + PPC];              // current row, pages [s0/16 - NBP, s0/16 + PPC)
    __shared__ int s_ev_pg[kShrinkEvict];           // current row, page of each evicted slot
    const int cc = blockIdx.y, i = blockIdx.z;
    const int kv = blockIdx.x & 1;
    const int h = (blockIdx.x >> 1) % a.Hkv, l = (blockIdx.x >> 1) / a.Hkv;
    const int tid = threadIdx.x;

    if (cc == 0 && blockIdx.x == 0 && i == 0) {
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

    // (1) decision, request, both eviction lists (the shrink list starts at kPage)
    const int32_t *rq = a.req + (size_t)i * RQ_STRIDE;
    const int dec = rq[RQ_DEC], P = rq[RQ_P], nsh = rq[RQ_NSH];
    const int r = a.bnd[i];
    const int32_t *evl = a.evict + (((size_t)l * a.Rb + i) * a.Hkv + h) * kEvictSlots;
    int ev_c = -1, ev_s = -1;
    if (tid < kShrinkEvict) {
        ev_s = evl[kPage + tid];
        if (tid < kPage) ev_c = evl[tid];
    }
    const bool shrink = dec == GP_SHRINK;
    if (!compressing(dec) && !shrink) return;
    if (r < 0 || r >= a.R) return;
    const int nev = shrink ? kShrinkEvict : kPage;
    const int total = P * kPage;
    const int s0 = cc * ROWS;
    if (s0 >= total) return;
    const int ev_mine = shrink ? ev_s : ev_c;
    if (tid < kShrinkEvict) s_ev[tid] = tid < nev ? ev_mine : -1;

    // (2) page-table entries
    const int32_t *row = a.page_table + (size_t)r * a.max_pages;
    const int32_t *src_row = nsh > 0 || shrink ? a.old_table + (size_t)i * a.max_pages : row;
    const int pg0 = s0 / kPage;
    if (tid < kShrinkEvict) {
        // thread k holds evicted slot k
        const int ev = tid < nev ? ev_mine : -1;
        s_ev_pg[tid] = ev >= 0 && ev / kPage < P ? row[ev / kPage] : -1;
    } else if (tid < kShrinkEvict + PPC) {
        const int k = tid - kShrinkEvict, j = pg0 + k;
        s_src_pg[k] = j < P ? src_row[j] : -1;
    } else if (tid < kShrinkEvict + 2 * PPC + NBP) {
        const int k = tid - kShrinkEvict - PPC, j = pg0 - NBP + k;
        s_lo_pg[k] = j >= 0 && j < P ? row[j] : -1;
    }
    __syncthreads();

    const size_t page_bytes = (size_t)a.Hkv * kPage * D * E;
    const size_t head_bytes = (size_t)h * kPage * D * E;
    const bool fill = a.layout == GP_LAYOUT_FILL;
    const bool has_border = !fill && s0 + ROWS < total;
    const int brows = a.policy == GP_POLICY_SHRINK ? kBorderRows : kPage;   // rows the select pass saved
    const int T = total - nev;              // resident length after the event
    int dst = -1;
    {
        const int s = s0 + tid;
        if (s < total) {
            int before = 0, between = 0;    // evicted below s; evicted in [T, s)
            bool gone = false;
#pragma unroll
            for (int k = 0; k < kShrinkEvict; ++k) {
                before += (s_ev[k] >= 0 && s_ev[k] < s) ? 1 : 0;
                between += (s_ev[k] >= T && s_ev[k] < s) ? 1 : 0;
                gone = gone || s_ev[k] == s;
            }
            if (!gone) {
                // shift: down past the evicted slots below.  fill: rows below T
                // stay; the k-th survivor at or above T takes the k-th evicted
                // slot (the list is sorted, so the slots below T come first).
                const int rank = min(max(s - T - between, 0), kShrinkEvict - 1);
                const int d = !fill ? s - before : (s < T ? s : s_ev[rank]);
                const int sp = s_src_pg[tid / kPage];
                int dp = -1;
                if (d >= 0) {
                    if (!fill || s < T) dp = s_lo_pg[d / kPage - (pg0 - NBP)];   // d in [s0 - 32, s0 + ROWS)
                    else dp = s_ev_pg[rank];
                }
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
    if (!__syncthreads_or(dst >= 0)) return;   // nothing moves in this chunk

    // (3) the rows: all loads, then all stores (rows move down within the chunk)
    const unsigned char *bd = a.border + ((((size_t)l * a.Rb + i) * a.Hkv + h) * a.ncc) * 2 * kBorderRows * D * E;
    unsigned char *pool = reinterpret_cast<unsigned char *>(kv == 0 ? lt.k[l] : lt.v[l]);
    uint4 val[UNITS];
#pragma unroll
    for (int k = 0; k < UNITS; ++k) {
        const int u = k * 256 + tid;
        const int rr = u / UPR, w = u % UPR;
        val[k] = make_uint4(0u, 0u, 0u, 0u);
        if (s_dst[rr] >= 0) {
            if (has_border && rr >= ROWS - brows) {
                const unsigned char *src = bd + ((size_t)(cc + 1) * 2 + kv) * kBorderRows * D * E +
                                           (size_t)(rr - (ROWS - kBorderRows)) * D * E + (size_t)w * 16;
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
}

// ---------------------------------------------------------------- release --
// Held requests (seq_len = -(m + 1)) get their resident length back.
__global__ __launch_bounds__(256) void release_kernel(int32_t *seq_lens, int R) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r < R) {
        const int m = seq_lens[r];
        if (m < 0) seq_lens[r] = -m - 1;
    }
}

template <int D, int E>
hipError_t launch_de(const ApplyArgs &a, const LayerTable &lt, int stages, hipStream_t s) {
    // (KV head, layer) is the fastest grid index: each head stays on one XCD
    dim3 gpre(a.Hkv * a.n_layers, 1 + max(a.npc, cdiv(a.ncc, kBordersPerGroup)), a.Rb),
        gcomp(2 * a.Hkv * a.n_layers, a.ncc, a.Rb);
    if (stages & kStageSelect) {
        if (a.policy == GP_POLICY_SHRINK)
            pre_kernel<D, E, true><<<gpre, kSelThreads, 0, s>>>(a, lt);
        else
            pre_kernel<D, E, false><<<gpre, kSelThreads, 0, s>>>(a, lt);
    }
    if (stages & kStageDecide) decide_kernel<<<1, 1024, 0, s>>>(a);
    if (stages & kStageCompact) compact_kernel<D, E><<<gcomp, 256, 0, s>>>(a, lt);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_release(int32_t *seq_lens, int R, hipStream_t s) {
    release_kernel<<<cdiv(R, 256), 256, 0, s>>>(seq_lens, R);
    return hipGetLastError();
}

hipError_t launch_apply(gp_dtype_t dt, int D, const ApplyArgs &a, const LayerPtrs *layers, int stages,
                        hipStream_t s) {
    if (a.Rb == 0) return hipSuccess;
    LayerTable lt;
    for (int l = 0; l < kMaxLayers; ++l) {
        lt.k[l] = l < a.n_layers ? layers[l].k : nullptr;
        lt.v[l] = l < a.n_layers ? layers[l].v : nullptr;
    }
    if (dt == GP_BF16) return D == 128 ? launch_de<128, 2>(a, lt, stages, s) : launch_de<64, 2>(a, lt, stages, s);
    return D == 128 ? launch_de<128, 4>(a, lt, stages, s) : launch_de<64, 4>(a, lt, stages, s);
}

}  // namespace gp

// Paged GQA decode attention (Sec. 3.1, attention-output equation), split over
// the sequence.
//
// Work item = (KV head h, chunk of the request's pages, request r): one
// workgroup serves the whole GQA group of h (G query heads), so every K/V byte
// is read from HBM once per step.  A request of m tokens has cdiv(m, chunk
// tokens) chunks, chunk tokens being about kDecodeChunkPages pages sized so
// that a request of max_pages pages splits evenly; its pages are then divided
// into that many nearly equal chunks, which keeps workgroup durations even.
// A request that
// spans several chunks leaves one (o, max, sum) partial per chunk, which a
// second, small kernel merges; a request of a single chunk gets its output
// from the first kernel.  Consecutive workgroups are the KV heads of one
// chunk, so the head slices of the same pages are read at about the same
// time.
//
// fp32 (vector ALUs): lane l holds dims [c*EPL, c*EPL+EPL) of token
// j*TPL + l/LPT for each of the LPP loads of a page, c = l % LPT; dot products
// finish with cross-lane sums over the LPT lanes of a token.  Four waves take
// pages round-robin, two pages in flight per wave.
//
// bf16: see decode_split_kernel.
//
// Bound: HBM.  Algorithmic bytes per resident token and KV head:
// 2 * d * sizeof(elem) (K and V), plus the page-table entries, q and out.
#include "gp_internal.h"

namespace gp {

namespace {

template <typename T>
struct Traits;

template <>
struct Traits<uint16_t> {
    static constexpr int EPL = 8;  // bf16 elements per 16-byte load
    __device__ static inline void unpack(const uint4 &u, float *f) {
        f[0] = bf16_lo(u.x); f[1] = bf16_hi(u.x);
        f[2] = bf16_lo(u.y); f[3] = bf16_hi(u.y);
        f[4] = bf16_lo(u.z); f[5] = bf16_hi(u.z);
        f[6] = bf16_lo(u.w); f[7] = bf16_hi(u.w);
    }
    __device__ static inline void store(uint16_t *p, float x) { *p = f32_to_bf16(x); }
    __device__ static inline float load(const uint16_t *p) { return bf16_to_f32(*p); }
};

template <>
struct Traits<float> {
    static constexpr int EPL = 4;
    __device__ static inline void unpack(const uint4 &u, float *f) {
        f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
        f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
    }
    __device__ static inline void store(float *p, float x) { *p = x; }
    __device__ static inline float load(const float *p) { return *p; }
};

constexpr float kNegInf = -__builtin_huge_valf();

// K and V are read exactly once per step, so their loads carry the
// non-temporal hint: the caches do not keep them at the expense of data that
// is reused (page tables, partials, and the workspaces of the boundary
// kernels that run beside decode attention).  On MI355X this also raised the
// decode call's own bandwidth (0.123 -> 0.115 ms at the Qwen3-8B layer shape).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ inline uint4 stream16(const void *p) {
    const u32x4_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(x[0], x[1], x[2], x[3]);
}

// s_waitcnt immediates: vmcnt(0) (vmcnt in bits 3:0 and 15:14, the others at
// their maximum), lgkmcnt(0); and the cache-policy operand of a direct-to-LDS
// load that marks it non-temporal
constexpr int kWaitVm0 = 0x0F70;
constexpr int kWaitLgkm0 = 0xC07F;
constexpr int kCpolNT = 2;
typedef const __attribute__((address_space(1))) void global_cvoid_t;
typedef __attribute__((address_space(3))) void lds_void_t;

// The request's view of one step: resident tokens m, pages P (clamped to the
// table), whether the step's new token goes in (room: a token is given and the
// last page has a free slot, Sec. 3.1 paged cache) and the tokens attended.
struct StepView {
    int m, P, m_attn;
    bool room;
};
__device__ inline StepView step_view(const DecodeArgs &a, int r, int m) {
    StepView v;
    int P = a.num_pages[r];
    v.P = P < 0 ? 0 : (P > a.max_pages ? a.max_pages : P);
    v.m = m > v.P * kPage ? v.P * kPage : m;
    v.room = a.k_new != nullptr && v.m < v.P * kPage;
    v.m_attn = v.m + (v.room ? 1 : 0);
    return v;
}

// For the merge pass: the tokens attended (-1: held), whether a token went in
// and how many partial slots the merge folds (0: the output is written by the
// chunk pass), written once per request by the workgroup of (KV head 0,
// chunk 0).
__device__ inline void record_step(const DecodeArgs &a, int r, int h, int chunk, int m_attn, bool room,
                                   int merge_slots) {
    if (h == 0 && chunk == 0 && threadIdx.x == 0) {
        a.lens[r] = m_attn;
        a.lens[a.R + r] = room ? 1 : 0;
        a.lens[2 * a.R + r] = merge_slots;
    }
}

// gp_decode_attention_shared: whether request r (not held, at least pp pages
// and pp * page_size tokens, within its table) may read a prefix pass of pp
// pages; the prefix pass and the tail pass also require the leader's page ids
// on every prefix page.  Both passes evaluate this on their own.
__device__ inline bool prefix_reader(const DecodeArgs &a, int r, int pp) {
    const int m = a.seq_lens[r], P = a.num_pages[r];
    return m >= pp * kPage && P >= pp && P <= a.max_pages && m <= P * kPage;
}

// gp_decode_step: the summary update of query heads [h G, h G + G) of request
// r, done by the workgroup of the pair's first chunk (Sec. 4.1 folds the
// update into the attention kernel).  Same arithmetic as the update kernel.
template <typename T, int D, int G>
__device__ inline void fold_summaries(const DecodeArgs &a, int r, int h) {
    if (!a.qstate) return;
    const int slot = a.slot_ids[r];
    if (slot < 0 || slot >= a.M) return;
    const int Hq = a.Hkv * G;
    const bool ini = a.init[r] != 0;
    const T *q = reinterpret_cast<const T *>(a.q_pre) + ((size_t)r * Hq + (size_t)h * G) * D;
    float *S = a.qstate + (size_t)slot * 2 * Hq * D + (size_t)h * G * D;
    float *L = S + (size_t)Hq * D;
    const double cs = 1.0 - a.beta_s, cl = 1.0 - a.beta_l;
    for (int i = threadIdx.x; i < G * D; i += blockDim.x) {
        const float x = Traits<T>::load(q + i);
        if (ini) {
            S[i] = x;
            L[i] = x;
        } else {
            S[i] = ema_step(S[i], x, a.beta_s, cs);
            L[i] = ema_step(L[i], x, a.beta_l, cl);
        }
    }
}

template <typename T, int D, int G>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a) {
    using Tr = Traits<T>;
    constexpr int EPL = Tr::EPL;
    constexpr int LPT = D / EPL;          // lanes per token
    constexpr int TPL = 64 / LPT;         // tokens per wave load
    constexpr int LPP = kPage / TPL;      // loads per page
    constexpr int NW = 4;                 // waves per workgroup
    const int CHUNK = a.chunk_pages * kPage;
    static_assert(LPT >= 1 && LPT <= 64 && TPL * LPP == kPage, "layout");

    __shared__ float s_m[NW][G], s_l[NW][G];
    __shared__ float s_o[NW][G][D];

    __shared__ float s_new[2][D];             // the step's new token (K, V) of head h

    const int h = blockIdx.x, chunk = blockIdx.y, r = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int Hkv = a.Hkv;
    const int Hq = Hkv * G;
    const int m_in = a.seq_lens[r];
    if (m_in < 0) {                           // held: not in this step's batch
        record_step(a, r, h, chunk, -1, false, 0);
        return;
    }
    const StepView sv = step_view(a, r, m_in);
    // with a new token, only the requests that take it update their summaries
    if (chunk == 0 && (a.k_new == nullptr || sv.room)) fold_summaries<T, D, G>(a, r, h);
    const int m = sv.m_attn;
    const int nchunks = cdiv(m, CHUNK);
    record_step(a, r, h, chunk, sv.m_attn, sv.room, nchunks > 1 ? nchunks : 0);
    T *out = reinterpret_cast<T *>(a.out) + ((size_t)r * Hq + (size_t)h * G) * D;
    if (m == 0) {
        if (chunk == 0)
            for (int i = threadIdx.x; i < G * D; i += blockDim.x) Tr::store(out + i, 0.0f);
        return;
    }
    if (chunk >= nchunks) return;

    // the request's pages split into nchunks nearly equal chunks (the chunk
    // count is the merge's; equal lengths keep the workgroups' durations even)
    const int npg = cdiv(m, kPage), cs = cdiv(npg, nchunks);
    const int page_begin = min(npg, chunk * cs), page_end = min(npg, page_begin + cs);

    // the new token: the workgroup whose pages hold slot m_in writes it into
    // the cache and takes its K and V from LDS (the cache slot is not read back)
    const int p_new = sv.room ? sv.m / kPage : -1, slot_new = sv.m % kPage;
    const bool owns_new = p_new >= page_begin && p_new < page_end;
    if (owns_new) {
        const T *kn = reinterpret_cast<const T *>(a.k_new) + ((size_t)r * Hkv + h) * D;
        const T *vn = reinterpret_cast<const T *>(a.v_new) + ((size_t)r * Hkv + h) * D;
        const int pid = a.page_table[(size_t)r * a.max_pages + p_new];
        const bool okp = pid >= 0 && pid < a.pool_pages;
        const size_t dst = (((size_t)(okp ? pid : 0) * Hkv + h) * kPage + slot_new) * D;
        for (int i = threadIdx.x; i < 2 * D; i += blockDim.x) {
            const int kvsel = i / D, dd = i % D;
            const T x = kvsel ? vn[dd] : kn[dd];
            s_new[kvsel][dd] = Tr::load(&x);
            if (okp) (kvsel ? reinterpret_cast<T *>(a.v_w) : reinterpret_cast<T *>(a.k_w))[dst + dd] = x;
        }
    }
    __syncthreads();

    const int c = lane % LPT, row = lane / LPT;
    const T *qp = reinterpret_cast<const T *>(a.q) + ((size_t)r * Hq + (size_t)h * G) * D + c * EPL;
    float q[G][EPL];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < EPL; ++e) q[g][e] = Tr::load(qp + (size_t)g * D + e) * a.qscale;

    float mrun[G], l[G], o[G][EPL];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        mrun[g] = kNegInf;
        l[g] = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[g][e] = 0.0f;
    }

    const int32_t *table = a.page_table + (size_t)r * a.max_pages;
    const T *kpool = reinterpret_cast<const T *>(a.k);
    const T *vpool = reinterpret_cast<const T *>(a.v);
    const size_t head_off = (size_t)h * kPage * D;
    const size_t page_elems = (size_t)Hkv * kPage * D;
    const int lane_off = row * D + c * EPL;

    for (int p0 = page_begin + wave; p0 < page_end; p0 += 2 * NW) {
        uint4 kr[2][LPP], vr[2][LPP];
        int ntok[2];
        bool ok[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int p = p0 + u * NW;
            int phys = p < page_end ? table[p] : -1;
            ok[u] = phys >= 0 && phys < a.pool_pages;
            ntok[u] = ok[u] ? min(kPage, m - p * kPage) : 0;
            const size_t base = (size_t)(ok[u] ? phys : 0) * page_elems + head_off + lane_off;
            if (ok[u]) {
#pragma unroll
                for (int j = 0; j < LPP; ++j) {
                    kr[u][j] = stream16(kpool + base + (size_t)j * TPL * D);
                    vr[u][j] = stream16(vpool + base + (size_t)j * TPL * D);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (!ok[u]) continue;   // wave-uniform
            float s[LPP][G];
            const bool patch = p0 + u * NW == p_new;     // wave-uniform
#pragma unroll
            for (int j = 0; j < LPP; ++j) {
                float kf[EPL];
                Tr::unpack(kr[u][j], kf);
                if (patch && j * TPL + row == slot_new) {
#pragma unroll
                    for (int e = 0; e < EPL; ++e) kf[e] = s_new[0][c * EPL + e];
                }
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    float acc = 0.0f;
#pragma unroll
                    for (int e = 0; e < EPL; ++e) acc = fmaf(q[g][e], kf[e], acc);
                    s[j][g] = acc;
                }
            }
#pragma unroll
            for (int off = LPT / 2; off >= 1; off >>= 1)
#pragma unroll
                for (int j = 0; j < LPP; ++j)
#pragma unroll
                    for (int g = 0; g < G; ++g) s[j][g] += __shfl_xor(s[j][g], off, 64);
            const bool full = ntok[u] == kPage;
            float pmax[G];
#pragma unroll
            for (int g = 0; g < G; ++g) pmax[g] = kNegInf;
#pragma unroll
            for (int j = 0; j < LPP; ++j) {
                const bool valid = full || (j * TPL + row) < ntok[u];
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    s[j][g] = valid ? s[j][g] : kNegInf;
                    pmax[g] = fmaxf(pmax[g], s[j][g]);
                }
            }
#pragma unroll
            for (int off = LPT; off < 64; off <<= 1)
#pragma unroll
                for (int g = 0; g < G; ++g) pmax[g] = fmaxf(pmax[g], __shfl_xor(pmax[g], off, 64));
            float alpha[G];
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const float mn = fmaxf(mrun[g], pmax[g]);
                alpha[g] = exp2f(mrun[g] - mn);
                mrun[g] = mn;
                l[g] *= alpha[g];
#pragma unroll
                for (int e = 0; e < EPL; ++e) o[g][e] *= alpha[g];
            }
#pragma unroll
            for (int j = 0; j < LPP; ++j) {
                const bool valid = full || (j * TPL + row) < ntok[u];
                float vf[EPL];
                Tr::unpack(vr[u][j], vf);
                if (patch && j * TPL + row == slot_new) {
#pragma unroll
                    for (int e = 0; e < EPL; ++e) vf[e] = s_new[1][c * EPL + e];
                }
#pragma unroll
                for (int e = 0; e < EPL; ++e) vf[e] = valid ? vf[e] : 0.0f;
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const float pw = exp2f(s[j][g] - mrun[g]);
                    l[g] += pw;
#pragma unroll
                    for (int e = 0; e < EPL; ++e) o[g][e] = fmaf(pw, vf[e], o[g][e]);
                }
            }
        }
    }

    // sum over the token rows of the wave (all rows share the running max)
#pragma unroll
    for (int off = LPT; off < 64; off <<= 1)
#pragma unroll
        for (int g = 0; g < G; ++g) {
            l[g] += __shfl_xor(l[g], off, 64);
#pragma unroll
            for (int e = 0; e < EPL; ++e) o[g][e] += __shfl_xor(o[g][e], off, 64);
        }
    if (row == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
#pragma unroll
            for (int e = 0; e < EPL; ++e) s_o[wave][g][c * EPL + e] = o[g][e];
            if (c == 0) {
                s_m[wave][g] = mrun[g];
                s_l[wave][g] = l[g];
            }
        }
    }
    __syncthreads();

    // merge the waves: thread -> (g, dim) pairs
    const bool single = nchunks == 1;
    float *part = a.partial + (((size_t)r * Hkv + h) * a.slots + chunk) * G * (D + 2);
    for (int i = threadIdx.x; i < G * D; i += blockDim.x) {
        const int g = i / D, dd = i % D;
        float M = kNegInf;
#pragma unroll
        for (int w = 0; w < NW; ++w) M = fmaxf(M, s_m[w][g]);
        float Ls = 0.0f, Os = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const float f = s_m[w][g] == kNegInf ? 0.0f : exp2f(s_m[w][g] - M);
            Ls += s_l[w][g] * f;
            Os += s_o[w][g][dd] * f;
        }
        if (single) {
            Tr::store(out + (size_t)g * D + dd, Os / Ls);
        } else {
            part[(size_t)g * (D + 2) + dd] = Os;
            if (dd == 0) {
                part[(size_t)g * (D + 2) + D] = M;
                part[(size_t)g * (D + 2) + D + 1] = Ls;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// bf16 path: Q.K^T on the matrix cores.  For one page, v_mfma_f32_16x16x32_bf16
// computes S^T = Q (16 rows: the G query heads, rest zero) x K^T (16 tokens)
// in D/32 steps.  In step kk, lane l supplies token l%16 and head dimensions
// [32 kk + 8 (l/16), +8), so one load instruction reads 64 contiguous bytes of
// each of the page's 16 key rows; Q is laid out with the same assignment.  The
// result leaves head 4*(l/16)+i of token l%16 in register i of lane l, so the
// per-page max and the row sums are 16-lane DPP reductions and every score is
// exponentiated once.  P.V stays on the vector ALUs in fp32, with the weights
// exchanged through LDS.
// ---------------------------------------------------------------------------
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

template <int N>
__device__ inline float dpp_ror(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x120 + N, 0xf, 0xf, false));
}
// 16-byte load of streamed K data (non-temporal, see stream16).
__device__ inline uint4 ld16(const uint16_t *p) { return stream16(p); }

// LDS traffic between lanes of one wave: wait for the wave's LDS operations
// and keep the compiler from moving memory accesses across this point.
__device__ inline void wave_lds_sync() { __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ inline float row_max16(float x) {
    x = fmaxf(x, dpp_ror<8>(x));
    x = fmaxf(x, dpp_ror<4>(x));
    x = fmaxf(x, dpp_ror<2>(x));
    return fmaxf(x, dpp_ror<1>(x));
}
__device__ inline float row_sum16(float x) {
    x += dpp_ror<8>(x);
    x += dpp_ror<4>(x);
    x += dpp_ror<2>(x);
    return x + dpp_ror<1>(x);
}

// Split decode (bf16): one workgroup of kDecodeWaves waves per (KV head,
// chunk, request); the waves take the chunk's pages round-robin.  Each wave
// owns one LDS page of keys and one of values, filled by direct-to-LDS loads;
// as soon as a stage has been read out, the wave requests the same part of its
// next page, so a page is on its way while softmax and P.V run.  Q waits in
// LDS.  For G >= kDecodePvmMinG, P.V runs on the matrix cores (S^T = K.Q^T
// puts P in the B layout; V^T comes by transposed LDS reads); for smaller G on
// the vector ALUs, each lane owning D/64 head dimensions for all 16 tokens of
// the page (accumulators G * D / 64 registers).  The waves merge through LDS
// at the end.
// MODE 0: decode attention; 1: gp_decode_step with the step's new token (its
// summary update is in the merge pass); 2: the private tails of gp_decode_attention_shared (a request
// that reads its group's shared prefix pass covers the pages after the prefix
// only, and its partials follow the prefix's).
template <int D, int G, int MODE>
__global__ __launch_bounds__(64 * kDecodeWaves) __attribute__((amdgpu_waves_per_eu(4))) void decode_split_kernel(
    DecodeArgs a) {
    constexpr bool STEP = MODE == 1, PREFIX = MODE == 2;
    constexpr bool PVM = G >= kDecodePvmMinG;   // P.V on the matrix cores (see the page step)
    constexpr int KK = D / 32;            // MFMA steps per page
    constexpr int DPL = D / 64;           // head dims per lane in P.V (2 or 1)
    constexpr int HR = (G + 3) / 4;       // lane rows that carry real heads
    constexpr int GI = G < 4 ? G : 4;     // heads per lane row
    constexpr int NW = kDecodeWaves;
    constexpr int NT = 64 * NW;
    constexpr int UPP = kPage * D / 8;                // 16-byte units of one page of one head (keys or values)
    constexpr int STAGE_BYTES = NW * 2 * UPP * 16, MERGE_BYTES = NW * G * D * 4;
    __shared__ float s_m[NW][G], s_l[NW][G];
    __shared__ float s_p[NW][kPage][G];
    __shared__ float s_alpha[NW][G];
    __shared__ bf16x8_t s_q[KK][4][G];
    __shared__ int s_ids[kMaxChunkPages];
    __shared__ __attribute__((aligned(16))) uint16_t s_new[STEP ? 2 : 1][STEP ? D : 8];   // new token K, V
    // per wave one page of keys and one of values while the pages are read,
    // then the waves' o for the merge
    __shared__ __attribute__((aligned(16))) char s_big[STAGE_BYTES > MERGE_BYTES ? STAGE_BYTES : MERGE_BYTES];
    auto s_o = reinterpret_cast<float (*)[G][D]>(s_big);

    const int h = blockIdx.x, chunk = blockIdx.y, r = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int Hkv = a.Hkv, Hq = Hkv * G;
    const int m_in = a.seq_lens[r];
    // PREFIX: a request whose prefix pages the prefix pass read starts after
    // them, in the partial slots after the prefix chunks' (the pass wrote
    // matched[r] for every request of a group)
    int base_page = 0, slot0 = 0;
    bool pmatch = false;
    int spec_n = 0, spec_pid = -1;                    // PREFIX: page ids requested ahead
    bool spec_hit = false;
    if constexpr (PREFIX) {
        int gsel = -1;
        for (int g = 0; g < a.ngroups; ++g)
            if (r >= a.g_first[g] && r < a.g_first[g] + a.g_num[g]) gsel = g;
        if (gsel >= 0) {                                  // uniform
            // the prefix pass's test for this request, evaluated here as well
            const int pp = a.g_pages[gsel];
            const bool reader = prefix_reader(a, r, pp);
            const int32_t *row = a.page_table + (size_t)r * a.max_pages;
            const int32_t *lrow = a.page_table + (size_t)a.g_first[gsel] * a.max_pages;
            // while the table rows are compared, the page ids of this chunk's
            // range as it is when the rows match (the usual case) are already
            // requested: one memory round trip less before the pages
            if (reader) {
                const int mt_s = m_in - pp * kPage, nch_s = cdiv(mt_s, a.chunk_pages * kPage);
                if (mt_s > 0 && chunk < nch_s) {
                    const int npg_s = cdiv(mt_s, kPage), cs_s = cdiv(npg_s, nch_s);
                    const int pb = pp + min(npg_s, chunk * cs_s), pe = pp + min(npg_s, chunk * cs_s + cs_s);
                    spec_n = pe - pb;
                    if (spec_n <= (int)blockDim.x && tid < spec_n) spec_pid = row[pb + tid];
                }
            }
            bool ok = reader;
            for (int j = tid; j < pp; j += blockDim.x) ok = ok && row[j] == lrow[j];
            pmatch = __syncthreads_and(ok);
            if (pmatch) {
                base_page = pp;
                slot0 = cdiv(pp, a.chunk_pages);
            }
            spec_hit = pmatch && spec_n > 0 && spec_n <= (int)blockDim.x;
        }
    }
    if (m_in < 0) {                           // held: not in this step's batch
        record_step(a, r, h, chunk, -1, false, 0);
        return;
    }
    const StepView sv = step_view(a, r, m_in);
    const int CHUNK = a.chunk_pages * kPage;

    const int m = sv.m_attn;
    const int mt = m - base_page * kPage;         // tokens this pass covers
    const int nchunks = cdiv(mt, CHUNK);
    record_step(a, r, h, chunk, m, sv.room, (pmatch || nchunks > 1) ? slot0 + nchunks : 0);
    uint16_t *out = reinterpret_cast<uint16_t *>(a.out) + ((size_t)r * Hq + (size_t)h * G) * D;
    if (mt == 0) {
        if (chunk == 0 && !pmatch)
            for (int i = tid; i < G * D; i += blockDim.x) out[i] = 0;
        return;
    }
    if (chunk >= nchunks) return;
    // the request's pages split into nchunks nearly equal chunks (the chunk
    // count is the merge's; equal lengths keep the workgroups' durations even)
    const int npg = cdiv(mt, kPage), cs = cdiv(npg, nchunks);
    const int page_begin = base_page + min(npg, chunk * cs);
    const int page_end = base_page + min(npg, chunk * cs + cs);

    const int n = lane & 15, kg = lane >> 4;          // score layout: token n, key slice kg
    const int v_off = lane * DPL;                     // P.V: lane owns dims [lane * DPL, +DPL)

    // page ids and Q (MFMA A layout, rows < G) into LDS
    const int32_t *table = a.page_table + (size_t)r * a.max_pages;
    if (PREFIX && spec_hit) {
        // (the same range: the prefix pages matched, as the request assumed)
        if (tid < page_end - page_begin) s_ids[tid] = spec_pid >= 0 && spec_pid < a.pool_pages ? spec_pid : -1;
    } else {
        for (int k = tid; k < page_end - page_begin; k += blockDim.x) {
            const int pid = table[page_begin + k];
            s_ids[k] = pid >= 0 && pid < a.pool_pages ? pid : -1;
        }
    }
    const uint16_t *qg = reinterpret_cast<const uint16_t *>(a.q) + ((size_t)r * Hq + (size_t)h * G) * D;
    if (tid < KK * 4 * G) {
        const int kk = tid / (4 * G), rem = tid % (4 * G), q_kg = rem / G, q_n = rem % G;
        s_q[kk][q_kg][q_n] = *reinterpret_cast<const bf16x8_t *>(qg + (size_t)q_n * D + kk * 32 + q_kg * 8);
    }
    // gp_decode_step with a new token: the workgroup whose pages hold slot
    // m_in stages the token's K and V of head h in LDS (its waves take them
    // from there, not from the cache) and writes them into the cache
    const int p_new = STEP && sv.room ? sv.m / kPage : -1, slot_new = sv.m % kPage;
    const bool owns_new = STEP && p_new >= page_begin && p_new < page_end;
    constexpr int NU16 = D / 8;                       // 16-byte units of one row
    uint4 nv = make_uint4(0u, 0u, 0u, 0u);
    if constexpr (STEP) {
        if (owns_new && tid < 2 * NU16) {
            const int kvsel = tid / NU16, u = tid % NU16;
            const uint16_t *src = reinterpret_cast<const uint16_t *>(kvsel ? a.v_new : a.k_new) +
                                  ((size_t)r * Hkv + h) * D + u * 8;
            nv = *reinterpret_cast<const uint4 *>(src);
            *reinterpret_cast<uint4 *>(&s_new[kvsel][u * 8]) = nv;
        }
    }
    __syncthreads();
    if constexpr (STEP) {
        if (owns_new && tid < 2 * NU16) {
            const int kvsel = tid / NU16, u = tid % NU16;
            const int phys = s_ids[p_new - page_begin];
            if (phys >= 0) {
                uint16_t *dst = reinterpret_cast<uint16_t *>(kvsel ? a.v_w : a.k_w) +
                                (((size_t)phys * Hkv + h) * kPage + slot_new) * D + u * 8;
                *reinterpret_cast<uint4 *>(dst) = nv;
            }
        }
    }

    float mrun[GI], lrun[GI], o[G][DPL];
#pragma unroll
    for (int i = 0; i < GI; ++i) {
        mrun[i] = kNegInf;
        lrun[i] = 0.0f;
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[g][e] = 0.0f;

    const uint16_t *kpool = reinterpret_cast<const uint16_t *>(a.k);
    const uint16_t *vpool = reinterpret_cast<const uint16_t *>(a.v);
    const size_t head_off = (size_t)h * kPage * D;
    const size_t page_elems = (size_t)Hkv * kPage * D;
    uint4 kb[KK];
    // Keys and values go straight to the wave's two LDS pages (no registers
    // in flight, so the request for the next page can go out as soon as this
    // one has been read out), each load instruction one contiguous 64 x
    // 16-byte run of the page (RPI whole rows).  Keys are swizzled: lane l of
    // instruction q takes row R = q RPI + l / UPR, unit (l % UPR) ^ (R % UPR),
    // so that unit u of row R sits at R UPR + (u ^ (R % UPR)) and the 16 rows
    // a score-layout read touches fall on distinct banks; values keep the row
    // layout (a P.V read is one whole row).  (Loading the keys in the score
    // layout itself, sixteen rows of 64 bytes per instruction, reads paged
    // keys about 7 % slower.)
    constexpr int UPR = D / 8;                        // 16-byte units per row
    constexpr int RPI = 64 / UPR;                     // rows per load instruction
    constexpr int KLD = kPage / RPI;                  // load instructions per page (keys or values)
    uint4 *kstage = reinterpret_cast<uint4 *>(s_big) + (size_t)wave * 2 * UPP;
    uint4 *vstage = kstage + UPP;
    auto load_kv = [&](int phys) {
        const size_t off = (size_t)phys * page_elems + head_off;
#pragma unroll
        for (int q = 0; q < KLD; ++q) {
            const int R = q * RPI + lane / UPR, u = (lane % UPR) ^ (R % UPR);
            __builtin_amdgcn_global_load_lds((global_cvoid_t *)(kpool + off + R * D + u * 8),
                                             (lds_void_t *)(kstage + q * 64), 16, 0, kCpolNT);
        }
#pragma unroll
        for (int q = 0; q < KLD; ++q) {
            // PVM: values swizzled by fv(R) = 2 (R % (UPR / 2)) for the
            // transposed reads; otherwise the plain row layout
            const int R = q * RPI + lane / UPR, u = PVM ? (lane % UPR) ^ (2 * (R % (UPR / 2))) : lane % UPR;
            __builtin_amdgcn_global_load_lds((global_cvoid_t *)(vpool + off + R * D + u * 8),
                                             (lds_void_t *)(vstage + q * 64), 16, 0, kCpolNT);
        }
    };
    // once the page has landed: the score-layout key operand of step kk (unit
    // 4 kk + kg of row n) and this lane's dims of every value row; the stages
    // are free again when the reads are done
    auto read_kv = [&](uint32_t (&vw)[kPage]) {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) kb[kk] = kstage[n * UPR + ((4 * kk + kg) ^ (n % UPR))];
#pragma unroll
        for (int t = 0; t < kPage; ++t) {
            if constexpr (DPL == 2)
                vw[t] = reinterpret_cast<const uint32_t *>(vstage)[t * (D / 2) + lane];
            else
                vw[t] = reinterpret_cast<const uint16_t *>(vstage)[t * D + lane];
        }
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
        __builtin_amdgcn_sched_barrier(0);
    };
    // One page of the wave: Q.K^T on the matrix cores, then the keys and
    // values of the wave's next page are requested together (the values into
    // the other buffer), then softmax and P.V on this page's values.
    auto page = [&](int p, int &phys) {
        const int ntok = phys >= 0 ? min(kPage, m - p * kPage) : 0;
        uint32_t vw[kPage];                          // this lane's dims of the page's value rows
        if (phys >= 0) {                             // wave-uniform
            read_kv(vw);
        } else {
#pragma unroll
            for (int t = 0; t < kPage; ++t) vw[t] = 0u;
        }
        if constexpr (STEP) {
            if (p == p_new) {     // wave-uniform: the new token's slot comes from LDS
                if (n == slot_new) {
#pragma unroll
                    for (int kk = 0; kk < KK; ++kk) kb[kk] = *reinterpret_cast<const uint4 *>(&s_new[0][kk * 32 + kg * 8]);
                }
                const uint32_t nvv = DPL == 2 ? *reinterpret_cast<const uint32_t *>(&s_new[1][v_off])
                                              : (uint32_t)s_new[1][v_off];
#pragma unroll
                for (int t = 0; t < kPage; ++t) vw[t] = t == slot_new ? nvv : vw[t];
            }
        }
        f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
        if (ntok > 0) {
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                bf16x8_t qa = {};
                if (n < G) qa = s_q[kk][kg][n];
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa, __builtin_bit_cast(bf16x8_t, kb[kk]), acc, 0, 0, 0);
            }
        }
        const int pn = p + NW;
        const int phys_next = pn < page_end ? s_ids[pn - page_begin] : -1;
        if (phys_next >= 0) load_kv(phys_next);
        const bool valid = n < ntok;
        float sc[GI], alpha[GI];
#pragma unroll
        for (int i = 0; i < GI; ++i) {
            sc[i] = valid ? acc[i] * a.qscale : kNegInf;
            const float pm = row_max16(sc[i]);
            const float mn = fmaxf(mrun[i], pm);
            alpha[i] = mn == kNegInf ? 1.0f : exp2f(mrun[i] - mn);
            mrun[i] = mn;
            sc[i] = mn == kNegInf ? 0.0f : exp2f(sc[i] - mn);
            lrun[i] = lrun[i] * alpha[i] + sc[i];
        }
        // hand the weights and the rescale factors to the P.V layout
        if (kg < HR) {
#pragma unroll
            for (int i = 0; i < GI; ++i) {
                s_p[wave][n][kg * 4 + i] = sc[i];
                if (n == 0) s_alpha[wave][kg * 4 + i] = alpha[i];
            }
        }
        wave_lds_sync();
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const float al = s_alpha[wave][g];
#pragma unroll
            for (int e = 0; e < DPL; ++e) o[g][e] *= al;
        }
#pragma unroll
        for (int t = 0; t < kPage; ++t) {
            if (t < ntok) {      // wave-uniform; slots past the last token may hold anything
                const float v0 = bf16_lo(vw[t]);
                const float v1 = DPL == 2 ? bf16_hi(vw[t]) : 0.0f;
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const float pw = s_p[wave][t][g];
                    o[g][0] = fmaf(pw, v0, o[g][0]);
                    if constexpr (DPL == 2) o[g][DPL - 1] = fmaf(pw, v1, o[g][DPL - 1]);
                }
            }
        }
        wave_lds_sync();
        phys = phys_next;
    };
    // PVM (G >= kDecodePvmMinG): S^T = K.Q^T, so that lane (n, kg) holds
    // tokens 4 kg + e of head n -- the B layout of the P.V product -- and
    // O^T += V^T.P^T on v_mfma_f32_16x16x16bf16_1k, V^T by transposed LDS
    // reads, P in two bfloat16 terms (hi + lo carry 16 significant bits): the
    // per-page P.V costs the matrix cores what it costs at any G, where the
    // vector-ALU form grows with G.  Heads n >= G of the 16 columns carry zero
    // queries and are never written.
    constexpr int DT = D / 16;                        // O^T tiles of 16 dims
    f32x4_t ot[PVM ? DT : 1];
    float pm_run = kNegInf, pl_run = 0.0f;            // head n: running max, this lane's share of the sum
#pragma unroll
    for (int t = 0; t < (PVM ? DT : 1); ++t) ot[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    typedef short bf16x4v_t __attribute__((ext_vector_type(4)));
    // keys and values of a page go out as two requests here, so that the
    // keys' stage is refilled as soon as its operands are read and the
    // values' once P.V has read them
    auto load_k_only = [&](int phys) {
        const size_t off = (size_t)phys * page_elems + head_off;
#pragma unroll
        for (int q = 0; q < KLD; ++q) {
            const int R = q * RPI + lane / UPR, u = (lane % UPR) ^ (R % UPR);
            __builtin_amdgcn_global_load_lds((global_cvoid_t *)(kpool + off + R * D + u * 8),
                                             (lds_void_t *)(kstage + q * 64), 16, 0, kCpolNT);
        }
    };
    auto load_v_only = [&](int phys) {
        const size_t off = (size_t)phys * page_elems + head_off;
#pragma unroll
        for (int q = 0; q < KLD; ++q) {
            const int R = q * RPI + lane / UPR, u = (lane % UPR) ^ (2 * (R % (UPR / 2)));
            __builtin_amdgcn_global_load_lds((global_cvoid_t *)(vpool + off + R * D + u * 8),
                                             (lds_void_t *)(vstage + q * 64), 16, 0, kCpolNT);
        }
    };
    auto page_pvm = [&](int p, int &phys) {
        const int ntok = phys >= 0 ? min(kPage, m - p * kPage) : 0;
        const int pn = p + NW;
        const int phys_next = pn < page_end ? s_ids[pn - page_begin] : -1;
        if (phys >= 0) {                              // wave-uniform
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) kb[kk] = kstage[n * UPR + ((4 * kk + kg) ^ (n % UPR))];
            __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (phys_next >= 0) load_k_only(phys_next);
        if constexpr (STEP) {
            if (p == p_new && n == slot_new) {        // the new token's key comes from LDS
#pragma unroll
                for (int kk = 0; kk < KK; ++kk) kb[kk] = *reinterpret_cast<const uint4 *>(&s_new[0][kk * 32 + kg * 8]);
            }
        }
        f32x4_t st = {0.0f, 0.0f, 0.0f, 0.0f};
        if (ntok > 0) {
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                bf16x8_t qb = {};
                if (n < G) qb = s_q[kk][kg][n];
                st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kb[kk]), qb, st, 0, 0, 0);
            }
        }
        // online softmax of head n over tokens 4 kg + e
        float sc[4], ml = kNegInf;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sc[e] = 4 * kg + e < ntok ? st[e] * a.qscale : kNegInf;
            ml = fmaxf(ml, sc[e]);
        }
        ml = fmaxf(ml, __shfl_xor(ml, 16, 64));
        ml = fmaxf(ml, __shfl_xor(ml, 32, 64));
        const float mn = fmaxf(pm_run, ml);
        const float alpha = mn == kNegInf ? 1.0f : exp2f(pm_run - mn);
        float psum = 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sc[e] = mn == kNegInf ? 0.0f : exp2f(sc[e] - mn);
            psum += sc[e];
        }
        pl_run = pl_run * alpha + psum;
        pm_run = mn;
        if (__any(alpha != 1.0f)) {                   // skip while no head's max has moved
#pragma unroll
            for (int t = 0; t < DT; ++t)
#pragma unroll
                for (int e = 0; e < 4; ++e) ot[t][e] *= alpha;
        }
        bf16x4v_t phi, plo;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const __bf16 hb = (__bf16)sc[e];              // round to nearest even
            phi[e] = __builtin_bit_cast(short, hb);
            plo[e] = __builtin_bit_cast(short, (__bf16)(sc[e] - (float)hb));   // p - hi is exact in float32
        }
        if (ntok > 0) {
            // V^T tile t as the A operand by transposed reads: lane j of group
            // kg names row R = 4 kg + j / 4, dims 16 t + 4 (j % 4); lane n
            // receives tokens 4 kg .. + 3 at dim 16 t + n.  Slots past the last
            // token may hold anything (0 x inf would reach o), so they read as
            // zero; the step's new token comes from LDS.
            const int R = 4 * kg + n / 4, qd = n % 4, fv = 2 * (R % (UPR / 2));
            const char *vrow = reinterpret_cast<const char *>(vstage + R * UPR) + (qd & 1) * 8;
#pragma unroll
            for (int t = 0; t < DT; ++t) {
                bf16x4v_t vt = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) bf16x4v_t *)(vrow + ((2 * t + qd / 2) ^ fv) * 16));
                if (ntok < kPage) {                   // wave-uniform
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (4 * kg + e >= ntok) vt[e] = 0;
                }
                if constexpr (STEP) {
                    if (p == p_new && kg == slot_new / 4) vt[slot_new % 4] = (short)s_new[1][16 * t + n];
                }
                ot[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, phi, ot[t], 0, 0, 0);
                ot[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, plo, ot[t], 0, 0, 0);
            }
            __builtin_amdgcn_s_waitcnt(kWaitLgkm0);   // the values' stage is read
            __builtin_amdgcn_sched_barrier(0);
        }
        if (phys_next >= 0) load_v_only(phys_next);
        phys = phys_next;
    };
    int p = page_begin + wave;
    int phys = p < page_end ? s_ids[p - page_begin] : -1;
    if (phys >= 0) load_kv(phys);
    if constexpr (PVM) {
        for (; p < page_end; p += NW) page_pvm(p, phys);
    } else {
        for (; p < page_end; p += NW) page(p, phys);
    }

    // merge the waves: per-wave (max, sum) of each head, o of every dim (o
    // goes where the stages were, once every wave is done with them)
    if constexpr (PVM) {
        pl_run += __shfl_xor(pl_run, 16, 64);
        pl_run += __shfl_xor(pl_run, 32, 64);
    } else {
#pragma unroll
        for (int i = 0; i < GI; ++i) lrun[i] = row_sum16(lrun[i]);
    }
    __syncthreads();
    if constexpr (PVM) {
        if (n < G) {
            if (kg == 0) {
                s_m[wave][n] = pm_run;
                s_l[wave][n] = pl_run;
            }
#pragma unroll
            for (int t = 0; t < DT; ++t)
#pragma unroll
                for (int e = 0; e < 4; ++e) s_o[wave][n][16 * t + 4 * kg + e] = ot[t][e];
        }
    } else {
        if (kg < HR && n == 0) {
#pragma unroll
            for (int i = 0; i < GI; ++i) {
                s_m[wave][kg * 4 + i] = mrun[i];
                s_l[wave][kg * 4 + i] = lrun[i];
            }
        }
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < DPL; ++e) s_o[wave][g][v_off + e] = o[g][e];
    }
    __syncthreads();

    const bool single = nchunks == 1 && !pmatch;
    float *part = a.partial + (((size_t)r * Hkv + h) * a.slots + slot0 + chunk) * G * (D + 2);
    for (int i = tid; i < G * D; i += blockDim.x) {
        const int g = i / D, dd = i % D;
        float M = kNegInf;
#pragma unroll
        for (int w = 0; w < NW; ++w) M = fmaxf(M, s_m[w][g]);
        float Ls = 0.0f, Os = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const float f = s_m[w][g] == kNegInf ? 0.0f : exp2f(s_m[w][g] - M);
            Ls += s_l[w][g] * f;
            Os += s_o[w][g][dd] * f;
        }
        if (single) {
            out[(size_t)g * D + dd] = f32_to_bf16(Ls > 0.0f ? Os / Ls : 0.0f);
        } else {
            part[(size_t)g * (D + 2) + dd] = Os;
            if (dd == 0) {
                part[(size_t)g * (D + 2) + D] = M;
                part[(size_t)g * (D + 2) + D + 1] = Ls;
            }
        }
    }
}

// Second pass for requests that span several chunks: one workgroup per
// (KV head, request) merges the chunks' (max, sum, o) partials.  Running it
// as its own launch lets the kernel boundary publish the partials; a
// device-scope fence per workgroup would write back and invalidate the L2 of
// every XCD thousands of times per step.
constexpr int kFastMerge = 8;   // chunks a merge folds without staging
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void merge_kernel(DecodeArgs a) {
    using Tr = Traits<T>;
    constexpr int MAXC = kMaxDecodeChunks + 1;       // partial slots (a shared prefix takes one more)
    __shared__ float s_f[MAXC][G];                 // exp2(m_k - M) / L per chunk and head
    __shared__ float s_ml[MAXC][G][2];
    const int h = blockIdx.x, r = blockIdx.y;
    const int tid = threadIdx.x;
    const int kmax = a.max_chunks + (a.ngroups > 0 ? 1 : 0);   // slots any request can fill

    // gp_decode_step, bfloat16: the summaries of query heads [h G, h G + G)
    // are updated here (Sec. 4.1) rather than in the chunk pass, where the
    // memory round trip it adds lengthened the workgroups that end the grid.
    // The slot is requested first, the query and the old values after the
    // partials (one more round trip at most), and the update is stored after
    // the output.  A held request, or with a new token one without room, keeps
    // its summaries, as in the float32 kernel.
    constexpr bool FOLD = sizeof(T) == 2;
    constexpr int FE = (G * D + 255) / 256;          // summary elements per thread
    float f_q[FE], f_s[FE], f_l[FE];
    float *fS = nullptr;
    int f_slot = -1;
    bool f_init = false;
    if constexpr (FOLD) {
        if (a.qstate) {
            f_slot = a.slot_ids[r];
            f_init = a.init[r] != 0;
        }
    }
    auto load_fold = [&]() {
        if constexpr (FOLD) {
            if (a.qstate && f_slot >= 0 && f_slot < a.M) {
                const size_t Hq = (size_t)a.Hkv * G;
                const uint16_t *qp = reinterpret_cast<const uint16_t *>(a.q_pre) + ((size_t)r * Hq + (size_t)h * G) * D;
                fS = a.qstate + (size_t)f_slot * 2 * Hq * D + (size_t)h * G * D;
#pragma unroll
                for (int e = 0; e < FE; ++e) {
                    const int i = min(tid + 256 * e, G * D - 1);
                    f_q[e] = bf16_to_f32(qp[i]);
                    f_s[e] = fS[i];
                    f_l[e] = fS[Hq * D + i];
                }
            }
        }
    };
    auto fold = [&](int took) {
        if constexpr (FOLD) {
            if (fS && (a.k_new == nullptr || took)) {
                const size_t Hq = (size_t)a.Hkv * G;
                const double cs_ = 1.0 - a.beta_s, cl_ = 1.0 - a.beta_l;
#pragma unroll
                for (int e = 0; e < FE; ++e) {
                    const int i = tid + 256 * e;
                    if (i < G * D) {
                        fS[i] = f_init ? f_q[e] : ema_step(f_s[e], f_q[e], a.beta_s, cs_);
                        fS[Hq * D + i] = f_init ? f_q[e] : ema_step(f_l[e], f_q[e], a.beta_l, cl_);
                    }
                }
            }
        }
    };
    if (kmax <= kFastMerge) {
        // few slots: every thread requests its elements of every slot a
        // request can fill together with the lengths (one round trip; the
        // recorded count then decides which slots are folded)
        constexpr int EPT = (G * D + 255) / 256;     // elements per thread
        const float *base = a.partial + ((size_t)r * a.Hkv + h) * a.slots * G * (D + 2);
        float mk[EPT][kFastMerge], lk[EPT][kFastMerge], ok[EPT][kFastMerge];
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            const int i = min(tid + 256 * e, G * D - 1);
            const int g = i / D, dd = i % D;
#pragma unroll
            for (int k = 0; k < kFastMerge; ++k) {
                mk[e][k] = kNegInf;
                lk[e][k] = 0.0f;
                ok[e][k] = 0.0f;
                if (k < kmax) {
                    const float *pp = base + ((size_t)k * G + g) * (D + 2);
                    mk[e][k] = pp[D];
                    lk[e][k] = pp[D + 1];
                    ok[e][k] = pp[dd];
                }
            }
        }
        load_fold();
        const int m = a.lens[r], took = a.lens[a.R + r], nslots = a.lens[2 * a.R + r];
        if (m < 0) return;
        if (a.advance && h == 0 && tid == 0 && took) {
            a.seq_lens_w[r] = m;
            if (a.positions) a.positions[r] += 1;
        }
        if (nslots == 0) {
            fold(took);
            return;
        }
        T *out = reinterpret_cast<T *>(a.out) + ((size_t)r * a.Hkv * G + (size_t)h * G) * D;
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            const int i = tid + 256 * e;
            float M = kNegInf;
#pragma unroll
            for (int k = 0; k < kFastMerge; ++k)
                if (k < nslots) M = fmaxf(M, mk[e][k]);
            float L = 0.0f, Os = 0.0f;
#pragma unroll
            for (int k = 0; k < kFastMerge; ++k) {
                // slots past the count hold whatever an earlier call left
                if (k < nslots) {
                    const float f = mk[e][k] == kNegInf ? 0.0f : exp2f(mk[e][k] - M);
                    L += lk[e][k] * f;
                    Os += ok[e][k] * f;
                }
            }
            if (i < G * D) Tr::store(out + i, L > 0.0f ? Os / L : 0.0f);
        }
        fold(took);
        return;
    }
    // tokens attended and partial slots, as the chunk pass recorded them
    // (-1: held; 0 slots: the chunk pass wrote the output)
    load_fold();
    const int m = a.lens[r];
    if (m < 0) return;
    const int took = a.lens[a.R + r];
    if (a.advance && h == 0 && threadIdx.x == 0 && took) {
        // gp_decode_step: the request took the step's token
        a.seq_lens_w[r] = m;
        if (a.positions) a.positions[r] += 1;
    }
    const int nchunks = a.lens[2 * a.R + r];
    if (nchunks == 0) {
        fold(took);
        return;
    }
    const int Hq = a.Hkv * G;
    T *out = reinterpret_cast<T *>(a.out) + ((size_t)r * Hq + (size_t)h * G) * D;
    const float *base = a.partial + ((size_t)r * a.Hkv + h) * a.slots * G * (D + 2);
    if (nchunks <= kFastMerge) {
        // few chunks: every thread loads all it needs at once (one round trip,
        // the (max, sum) of a head are the same address for a whole wave) and
        // folds them itself
        for (int i = tid; i < G * D; i += blockDim.x) {
            const int g = i / D, dd = i % D;
            float mk[kFastMerge], lk[kFastMerge], ok[kFastMerge];
#pragma unroll
            for (int k = 0; k < kFastMerge; ++k) {
                mk[k] = kNegInf;
                lk[k] = 0.0f;
                ok[k] = 0.0f;
                if (k < nchunks) {
                    const float *pp = base + ((size_t)k * G + g) * (D + 2);
                    mk[k] = pp[D];
                    lk[k] = pp[D + 1];
                    ok[k] = pp[dd];
                }
            }
            float M = kNegInf;
#pragma unroll
            for (int k = 0; k < kFastMerge; ++k) M = fmaxf(M, mk[k]);
            float L = 0.0f, Os = 0.0f;
#pragma unroll
            for (int k = 0; k < kFastMerge; ++k) {
                const float f = mk[k] == kNegInf ? 0.0f : exp2f(mk[k] - M);
                L += lk[k] * f;
                Os += ok[k] * f;
            }
            Tr::store(out + (size_t)g * D + dd, L > 0.0f ? Os / L : 0.0f);
        }
        fold(took);
        return;
    }
    // all (max, sum) pairs at once, then one thread per head folds them
    for (int t = tid; t < nchunks * G && t < MAXC * G; t += blockDim.x) {
        const int k = t / G, g = t % G;
        s_ml[k][g][0] = base[((size_t)k * G + g) * (D + 2) + D];
        s_ml[k][g][1] = base[((size_t)k * G + g) * (D + 2) + D + 1];
    }
    __syncthreads();
    const int nc = nchunks < MAXC ? nchunks : MAXC;
    if (tid < G) {
        float M = kNegInf;
        for (int k = 0; k < nc; ++k) M = fmaxf(M, s_ml[k][tid][0]);
        float L = 0.0f;
        for (int k = 0; k < nc; ++k) {
            const float f = s_ml[k][tid][0] == kNegInf ? 0.0f : exp2f(s_ml[k][tid][0] - M);
            s_f[k][tid] = f;
            L += s_ml[k][tid][1] * f;
        }
        const float inv = 1.0f / L;
        for (int k = 0; k < nc; ++k) s_f[k][tid] *= inv;
    }
    __syncthreads();
    for (int i = tid; i < G * D; i += blockDim.x) {
        const int g = i / D, dd = i % D;
        float Os = 0.0f;
#pragma unroll 8
        for (int k = 0; k < nc; ++k) Os += base[((size_t)k * G + g) * (D + 2) + dd] * s_f[k][g];
        Tr::store(out + (size_t)g * D + dd, Os);
    }
    fold(took);
}

// ---------------------------------------------------------------------------
// Shared-prefix pass (gp_decode_attention_shared; App. E.2 keeps a common
// prefix in reference-counted blocks that many requests read).  Work item =
// (KV head h, prefix slot c, block of 4 * 16 / G requests of one group).  The
// prefix is split evenly over its slots; a slot's pages are read once per
// workgroup, kPrefixBatch at a time, straight into LDS by direct-to-LDS loads
// (the next batch in flight while this one is computed), and each of the four
// waves serves 16 query rows (16 / G requests x G heads) over all of them.
// Per page a wave computes S^T = K.Q^T on v_mfma_f32_16x16x32_bf16 (the keys
// as the A operand), so that every lane holds four tokens of one query row; an
// online softmax per row; and O^T += V^T.P^T on v_mfma_f32_16x16x16bf16_1k,
// with V^T read by ds_read_b64_tr_b16 and P, already in the B layout, split
// into two bfloat16 terms (hi + lo carry 16 significant bits, so P.V keeps
// float32-level accuracy while the values stay exact bfloat16).  Every lane
// holds output dims of one row, so the rescale needs no lane exchange.  The
// slot's (o, max, sum) per row go to partial slot c of each request; the
// private tails follow in the next slots and the merge folds them together.
// A request reads the pass only if it is not held, holds at least the
// prefix's tokens and its table matches the group leader's on every prefix
// page; otherwise the tail pass covers all of its pages (both passes make the
// same test).
// Bound: HBM on the tails; the prefix pages are read once per block of
// requests instead of once per request.
typedef short bf16x4s_t __attribute__((ext_vector_type(4)));

// The pass stages kPrefixBatch pages (keys and values) per round and keeps
// two rounds in LDS.
constexpr int kPrefixBatch = 4;

template <int D, int G>
__global__ __launch_bounds__(64 * kPrefixWaves) void prefix_kernel(DecodeArgs a) {
    constexpr int KK = D / 32;            // S^T MFMA steps per page
    constexpr int NW = kPrefixWaves;
    constexpr int NT = 64 * NW;
    constexpr int RPW = 16 / G;           // requests per wave (16 query rows)
    constexpr int RPB = NW * RPW;         // requests per workgroup
    constexpr int DT = D / 16;            // O^T tiles of 16 dims
    constexpr int UPR = D / 8;            // 16-byte units per row
    constexpr int UPP = kPage * UPR;      // units of one page of one head (keys or values)
    constexpr int NB = kPrefixBatch;      // pages per round
    constexpr int RPI = 64 / UPR;         // rows per load instruction
    constexpr int IPP = 2 * UPP / 64;     // load instructions per page (keys, then values)
    constexpr int IPW = NB * IPP / NW;    // load instructions per wave and round
    static_assert((NB * IPP) % NW == 0 && UPP % 64 == 0, "staging layout");
    __shared__ __attribute__((aligned(16))) uint4 s_stage[2][NB][2][UPP];   // [round % 2][page][keys, values]
    __shared__ int s_ids[kMaxChunkPages];
    __shared__ int s_match[RPB];

    const int h = blockIdx.x, c = blockIdx.y, blk = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 15, kg = lane >> 4;
    int gi = 0;
    while (gi + 1 < a.ngroups && blk >= a.g_blk0[gi + 1]) ++gi;
    const int first = a.g_first[gi], nreq = a.g_num[gi], ppages = a.g_pages[gi];
    const int r0 = first + (blk - a.g_blk0[gi]) * RPB;
    // the prefix split evenly over its cdiv(ppages, chunk_pages) slots (cs <=
    // chunk_pages; the last slot is never empty)
    const int nps = cdiv(ppages, a.chunk_pages), cs = cdiv(ppages, nps);
    const int p_begin = c * cs, p_end = min(ppages, p_begin + cs);
    const int Hkv = a.Hkv, Hq = Hkv * G;
    const int32_t *lead = a.page_table + (size_t)first * a.max_pages;

    // which requests of the block read the pass (the same test in every
    // workgroup of the block, so they agree without talking)
    for (int j = tid; j < RPB; j += NT) {
        const int r = r0 + j;
        s_match[j] = r < first + nreq && prefix_reader(a, r, ppages) ? 1 : 0;
    }
    for (int k = tid; k < p_end - p_begin; k += NT) {
        const int pid = lead[p_begin + k];
        s_ids[k] = pid >= 0 && pid < a.pool_pages ? pid : -1;
    }
    __syncthreads();
    for (int e = tid; e < RPB * ppages; e += NT) {
        const int j = e / ppages, pg = e % ppages;
        if (s_match[j] && a.page_table[(size_t)(r0 + j) * a.max_pages + pg] != lead[pg]) s_match[j] = 0;
    }
    __syncthreads();
    if (p_begin >= ppages) return;
    int any = 0;
    for (int j = 0; j < RPB; ++j) any |= s_match[j];
    if (!any) return;                                    // uniform

    // this wave's 16 query rows (row n = request wave * RPW + n / G, head
    // n % G) as the B operand of S^T = K Q^T: lane (n, kg) holds dims
    // 32 kk + 8 kg .. + 7
    const int jq = wave * RPW + n / G;
    const bool rowq = s_match[jq] != 0;
    bf16x8_t qb[KK];
    {
        const uint16_t *qp = reinterpret_cast<const uint16_t *>(a.q) +
                             ((size_t)(rowq ? r0 + jq : first) * Hq + (size_t)h * G + n % G) * D;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const bf16x8_t x = *reinterpret_cast<const bf16x8_t *>(qp + kk * 32 + kg * 8);
            qb[kk] = rowq ? x : bf16x8_t{};
        }
    }

    const uint16_t *kpool = reinterpret_cast<const uint16_t *>(a.k);
    const uint16_t *vpool = reinterpret_cast<const uint16_t *>(a.v);
    const size_t head_off = (size_t)h * kPage * D;
    const size_t page_elems = (size_t)Hkv * kPage * D;
    const int npage = p_end - p_begin;
    // Round rr's pages rr NB .. rr NB + NB - 1 go to stage rr % 2, each load
    // instruction one contiguous run of RPI rows; the waves split the
    // instructions.  Unit u of row R sits at R UPR + (u ^ fk(R)) for keys,
    // fk(R) = R % UPR (a score-layout read of 16 rows hits 16 bank groups),
    // and at R UPR + (u ^ fv(R)) for values, fv(R) = 2 (R % (UPR / 2)) (the
    // transposed reads of 4 rows x 2 units hit distinct bank groups).  An
    // invalid page id reads page 0 (its scores are masked).
    auto issue = [&](int rr) {
#pragma unroll
        for (int i = 0; i < IPW; ++i) {
            const int e = wave * IPW + i, j = e / IPP, w2 = e % IPP;
            const int k = rr * NB + j;
            if (k < npage) {                             // wave-uniform
                const bool isv = w2 >= IPP / 2;
                const int q = isv ? w2 - IPP / 2 : w2;
                const int R = q * RPI + lane / UPR, s = lane % UPR;
                const int u = s ^ (isv ? 2 * (R % (UPR / 2)) : R % UPR);
                const uint16_t *src = (isv ? vpool : kpool) + (size_t)max(s_ids[k], 0) * page_elems + head_off +
                                      (size_t)R * D + u * 8;
                __builtin_amdgcn_global_load_lds((global_cvoid_t *)src,
                                                 (lds_void_t *)(&s_stage[rr & 1][j][isv][q * 64]), 16, 0, kCpolNT);
            }
        }
    };

    float mrun = kNegInf, lrun = 0.0f;   // row n: running max (log2 units), this lane's share of the sum
    f32x4_t o[DT];                       // O^T tile t: lane (n, kg) holds dims 16 t + 4 kg + e of row n
#pragma unroll
    for (int t = 0; t < DT; ++t) o[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    auto page = [&](const uint4 *ks, const uint4 *vs, bool valid) {
        bf16x8_t kc[KK];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            kc[kk] = __builtin_bit_cast(bf16x8_t, ks[n * UPR + ((4 * kk + kg) ^ (n % UPR))]);
        f32x4_t st = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc[kk], qb[kk], st, 0, 0, 0);
        // online softmax of row n; this lane has tokens 4 kg + e
        float s[4], ml = kNegInf;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            s[e] = valid ? st[e] * a.qscale : kNegInf;
            ml = fmaxf(ml, s[e]);
        }
        ml = fmaxf(ml, __shfl_xor(ml, 16, 64));
        ml = fmaxf(ml, __shfl_xor(ml, 32, 64));
        const float mn = fmaxf(mrun, ml);
        // arguments are <= 0: the hardware exp2 needs no range fix-up
        const float alpha = mn == kNegInf ? 1.0f : __builtin_amdgcn_exp2f(mrun - mn);
        float p[4], psum = 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            p[e] = mn == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(s[e] - mn);
            psum += p[e];
        }
        lrun = lrun * alpha + psum;
        mrun = mn;
        if (__any(alpha != 1.0f)) {                      // skip while no row's max has moved
#pragma unroll
            for (int t = 0; t < DT; ++t)
#pragma unroll
                for (int e = 0; e < 4; ++e) o[t][e] *= alpha;
        }
        // P^T as the B operand (tokens 4 kg + e of row n) in two bf16 terms
        bf16x4s_t phi, plo;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const __bf16 hb = (__bf16)p[e];              // round to nearest even
            phi[e] = __builtin_bit_cast(short, hb);
            plo[e] = __builtin_bit_cast(short, (__bf16)(p[e] - (float)hb));   // p - hi is exact in float32
        }
        // V^T tile t as the A operand by transposed reads: lane j of group kg
        // names row R = 4 kg + j / 4, dims 16 t + 4 (j % 4) (unit 2 t + (j % 4)
        // / 2, half (j % 4) % 2); lane n receives the values of tokens
        // 4 kg .. 4 kg + 3 at dim 16 t + n
        const int R = 4 * kg + n / 4, qd = n % 4;
        const char *vrow = reinterpret_cast<const char *>(vs + R * UPR) + (qd & 1) * 8;
        const int fv = 2 * (R % (UPR / 2));
#pragma unroll
        for (int t = 0; t < DT; ++t) {
            const bf16x4s_t vt = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) bf16x4s_t *)(vrow + ((2 * t + qd / 2) ^ fv) * 16));
            o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, phi, o[t], 0, 0, 0);
            o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, plo, o[t], 0, 0, 0);
        }
    };

    issue(0);
    for (int rr = 0; rr * NB < npage; ++rr) {
        __builtin_amdgcn_s_waitcnt(kWaitVm0);            // this wave's part of round rr has landed
        __syncthreads();                                 // all of it; every wave is done with round rr - 1
        if ((rr + 1) * NB < npage) issue(rr + 1);        // into the stage round rr - 1 used
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int k = rr * NB + j;
            if (k < npage) page(s_stage[rr & 1][j][0], s_stage[rr & 1][j][1], s_ids[k] >= 0);
        }
    }

    // partials of row n: o of dims 16 t + 4 kg + e, (max, sum) by the kg 0 lanes
    lrun += __shfl_xor(lrun, 16, 64);
    lrun += __shfl_xor(lrun, 32, 64);
    if (rowq) {
        float *part = a.partial + (((size_t)(r0 + jq) * Hkv + h) * a.slots + c) * G * (D + 2) +
                      (size_t)(n % G) * (D + 2);
#pragma unroll
        for (int t = 0; t < DT; ++t) *reinterpret_cast<f32x4_t *>(part + 16 * t + 4 * kg) = o[t];
        if (kg == 0) {
            part[D] = mrun;
            part[D + 1] = lrun;
        }
    }
}

template <typename T, int D>
hipError_t launch_g(int G, const DecodeArgs &a, dim3 grid, int stages, hipStream_t s) {
    dim3 mgrid(a.Hkv, a.R);
    constexpr bool bf16 = sizeof(T) == 2;
    // the step variant with a new token and the tails of the shared-prefix
    // decode are their own instantiations, so plain decode attention carries
    // none of their code (a step call's summary update is in the merge pass:
    // without a new token its chunk pass is plain decode attention)
    const int mode = a.ngroups > 0 ? 2 : a.k_new != nullptr ? 1 : 0;
    // the merge pass also advances the lengths when a token went in, updates
    // the summaries of a bfloat16 step call, and folds the prefix partials of a
    // shared-prefix call
    const bool chunks = stages & GP_DECODE_CHUNKS, prefix = (stages & GP_DECODE_PREFIX) && mode == 2,
               merge = (stages & GP_DECODE_MERGE) &&
                       (a.max_chunks > 1 || (a.k_new && a.advance) || mode == 2 || (bf16 && a.qstate));
    // prefix pass grid: (KV head, prefix chunk, request block)
    int max_pc = 0;
    for (int g = 0; g < a.ngroups; ++g) max_pc = max(max_pc, cdiv(a.g_pages[g], a.chunk_pages));
    const dim3 pgrid(a.Hkv, max(max_pc, 1), max(a.g_blk0[a.ngroups], 1));
    switch (G) {
#define GP_CASE(GG)                                                  \
    case GG:                                                         \
        if (prefix && bf16)                                          \
            prefix_kernel<D, GG><<<pgrid, 64 * kPrefixWaves, 0, s>>>(a); \
        if (chunks && bf16 && mode == 2)                             \
            decode_split_kernel<D, GG, 2><<<grid, 64 * kDecodeWaves, 0, s>>>(a); \
        else if (chunks && bf16 && mode == 1)                        \
            decode_split_kernel<D, GG, 1><<<grid, 64 * kDecodeWaves, 0, s>>>(a); \
        else if (chunks && bf16)                                     \
            decode_split_kernel<D, GG, 0><<<grid, 64 * kDecodeWaves, 0, s>>>(a); \
        else if (chunks)                                             \
            decode_kernel<float, D, GG><<<grid, 256, 0, s>>>(a);     \
        if (merge) merge_kernel<T, D, GG><<<mgrid, 256, 0, s>>>(a);  \
        break;
        GP_CASE(1) GP_CASE(2) GP_CASE(4) GP_CASE(8)
#undef GP_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(gp_dtype_t dt, int D, int G, const DecodeArgs &a, int stages, hipStream_t s) {
    // the KV heads of one chunk are neighbours in dispatch order: they read the
    // head slices of the same pages at about the same time
    dim3 grid(a.Hkv, a.max_chunks, a.R);
    if (dt == GP_BF16)
        return D == 128 ? launch_g<uint16_t, 128>(G, a, grid, stages, s)
                        : launch_g<uint16_t, 64>(G, a, grid, stages, s);
    return D == 128 ? launch_g<float, 128>(G, a, grid, stages, s) : launch_g<float, 64>(G, a, grid, stages, s);
}

}  // namespace gp

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

// For the merge pass: the tokens attended (-1: held) and whether a token went
// in, written once per request by the workgroup of (KV head 0, chunk 0).
__device__ inline void record_step(const DecodeArgs &a, int r, int h, int chunk, int m_attn, bool room) {
    if (h == 0 && chunk == 0 && threadIdx.x == 0) {
        a.lens[r] = m_attn;
        a.lens[a.R + r] = room ? 1 : 0;
    }
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
        record_step(a, r, h, chunk, -1, false);
        return;
    }
    const StepView sv = step_view(a, r, m_in);
    record_step(a, r, h, chunk, sv.m_attn, sv.room);
    // with a new token, only the requests that take it update their summaries
    if (chunk == 0 && (a.k_new == nullptr || sv.room)) fold_summaries<T, D, G>(a, r, h);
    const int P = sv.P;
    const int m = sv.m_attn;
    const int nchunks = cdiv(m, CHUNK);
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
    float *part = a.partial + (((size_t)r * Hkv + h) * a.max_chunks + chunk) * G * (D + 2);
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
// chunk, request); the waves take the chunk's pages round-robin.  As soon as
// the matrix cores have consumed a page's keys, the wave requests the keys and
// the values of its next page (the values into the second of two buffers that
// alternate), so a whole page is on its way while softmax and P.V run.  In
// P.V each lane owns D/64 head dimensions for all 16 tokens of the page, so a
// value load reads one whole 2D-byte row per instruction and the accumulators
// take G * D / 64 registers; Q waits in LDS.  The waves merge through LDS at
// the end.
template <int D, int G, bool STEP>
__global__ __launch_bounds__(64 * kDecodeWaves) void decode_split_kernel(DecodeArgs a) {
    constexpr int KK = D / 32;            // MFMA steps per page
    constexpr int DPL = D / 64;           // head dims per lane in P.V (2 or 1)
    constexpr int HR = (G + 3) / 4;       // lane rows that carry real heads
    constexpr int GI = G < 4 ? G : 4;     // heads per lane row
    constexpr int NW = kDecodeWaves;
    constexpr int NT = 64 * NW;
    constexpr int FE = STEP ? (G * D + NT - 1) / NT : 1;   // summary elements per thread
    __shared__ float s_m[NW][G], s_l[NW][G];
    __shared__ float s_o[NW][G][D];
    __shared__ float s_p[NW][kPage][G];
    __shared__ float s_alpha[NW][G];
    __shared__ bf16x8_t s_q[KK][4][G];
    __shared__ int s_ids[kMaxChunkPages];
    __shared__ __attribute__((aligned(16))) uint16_t s_new[STEP ? 2 : 1][STEP ? D : 8];   // new token K, V

    const int h = blockIdx.x, chunk = blockIdx.y, r = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int Hkv = a.Hkv, Hq = Hkv * G;
    const int m_in = a.seq_lens[r];
    if (m_in < 0) {                           // held: not in this step's batch
        record_step(a, r, h, chunk, -1, false);
        return;
    }
    const StepView sv = step_view(a, r, m_in);
    record_step(a, r, h, chunk, sv.m_attn, sv.room);
    const int CHUNK = a.chunk_pages * kPage;

    // gp_decode_step: the summaries of query heads [h G, h G + G) are updated
    // by the first chunk's workgroup (with a new token: only if the request
    // takes it).  The old values and the query are requested here, with the
    // other loads of the prologue; the update is stored when the workgroup ends.
    float f_q[FE], f_s[FE], f_l[FE];
    float *fS = nullptr;
    bool f_init = false;
    if constexpr (STEP) {
        if (chunk == 0 && a.qstate && (a.k_new == nullptr || sv.room)) {
            const int slot = a.slot_ids[r];
            if (slot >= 0 && slot < a.M) {
                fS = a.qstate + (size_t)slot * 2 * Hq * D + (size_t)h * G * D;
                f_init = a.init[r] != 0;
                const uint16_t *qp = reinterpret_cast<const uint16_t *>(a.q_pre) + ((size_t)r * Hq + (size_t)h * G) * D;
#pragma unroll
                for (int e = 0; e < FE; ++e) {
                    const int i = min(tid + e * NT, G * D - 1);
                    f_q[e] = bf16_to_f32(qp[i]);
                    f_s[e] = fS[i];
                    f_l[e] = fS[(size_t)Hq * D + i];
                }
            }
        }
    }
    auto finish_fold = [&]() {
        if constexpr (STEP) {
            if (fS) {
                const double cs_ = 1.0 - a.beta_s, cl_ = 1.0 - a.beta_l;
#pragma unroll
                for (int e = 0; e < FE; ++e) {
                    const int i = tid + e * NT;
                    if (i < G * D) {
                        fS[i] = f_init ? f_q[e] : ema_step(f_s[e], f_q[e], a.beta_s, cs_);
                        fS[(size_t)Hq * D + i] = f_init ? f_q[e] : ema_step(f_l[e], f_q[e], a.beta_l, cl_);
                    }
                }
            }
        }
    };

    const int m = sv.m_attn;
    const int nchunks = cdiv(m, CHUNK);
    uint16_t *out = reinterpret_cast<uint16_t *>(a.out) + ((size_t)r * Hq + (size_t)h * G) * D;
    if (m == 0) {
        if (chunk == 0)
            for (int i = tid; i < G * D; i += blockDim.x) out[i] = 0;
        finish_fold();
        return;
    }
    if (chunk >= nchunks) return;
    // the request's pages split into nchunks nearly equal chunks (the chunk
    // count is the merge's; equal lengths keep the workgroups' durations even)
    const int npg = cdiv(m, kPage), cs = cdiv(npg, nchunks);
    const int page_begin = min(npg, chunk * cs), page_end = min(npg, page_begin + cs);

    const int n = lane & 15, kg = lane >> 4;          // score layout: token n, key slice kg
    const int v_off = lane * DPL;                     // P.V: lane owns dims [lane * DPL, +DPL)
    const int k_off = n * D + kg * 8;

    // page ids and Q (MFMA A layout, rows < G) into LDS
    const int32_t *table = a.page_table + (size_t)r * a.max_pages;
    for (int k = tid; k < page_end - page_begin; k += blockDim.x) {
        const int pid = table[page_begin + k];
        s_ids[k] = pid >= 0 && pid < a.pool_pages ? pid : -1;
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
    uint32_t vwa[kPage], vwb[kPage];                 // values of this page and of the next
    auto load_k = [&](int phys) {
        const uint16_t *kp = kpool + (size_t)phys * page_elems + head_off + k_off;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) kb[kk] = ld16(kp + kk * 32);
    };
    auto load_v = [&](int phys, uint32_t (&vw)[kPage]) {
        // one 2D-byte row per instruction: fully coalesced
        const uint16_t *vp = vpool + (size_t)phys * page_elems + head_off + v_off;
#pragma unroll
        for (int t = 0; t < kPage; ++t) {
            if constexpr (DPL == 2)
                vw[t] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(vp + t * D));
            else
                vw[t] = __builtin_nontemporal_load(vp + t * D);
        }
    };
    // One page of the wave: Q.K^T on the matrix cores, then the keys and
    // values of the wave's next page are requested together (the values into
    // the other buffer), then softmax and P.V on this page's values.
    auto page = [&](int p, int &phys, uint32_t (&vw)[kPage], uint32_t (&vn)[kPage]) {
        const int ntok = phys >= 0 ? min(kPage, m - p * kPage) : 0;
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
        if (phys_next >= 0) {
            load_k(phys_next);
            load_v(phys_next, vn);
        }
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
    int p = page_begin + wave;
    int phys = p < page_end ? s_ids[p - page_begin] : -1;
    if (phys >= 0) {
        load_k(phys);
        load_v(phys, vwa);
    }
    // pages alternate between the two value buffers
    for (; p < page_end; p += 2 * NW) {
        page(p, phys, vwa, vwb);
        if (p + NW >= page_end) break;
        page(p + NW, phys, vwb, vwa);
    }

    // merge the waves: per-wave (max, sum) of each head, o of every dim
#pragma unroll
    for (int i = 0; i < GI; ++i) lrun[i] = row_sum16(lrun[i]);
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
    __syncthreads();

    const bool single = nchunks == 1;
    float *part = a.partial + (((size_t)r * Hkv + h) * a.max_chunks + chunk) * G * (D + 2);
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
    finish_fold();
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
    const int CHUNK = a.chunk_pages * kPage;
    constexpr int MAXC = kMaxDecodeChunks;
    __shared__ float s_f[MAXC][G];                 // exp2(m_k - M) / L per chunk and head
    __shared__ float s_ml[MAXC][G][2];
    const int h = blockIdx.x, r = blockIdx.y;
    // tokens attended, as the chunk pass recorded them (-1: held, nothing to merge)
    const int m = a.lens[r];
    if (m < 0) return;
    if (a.advance && h == 0 && threadIdx.x == 0 && a.lens[a.R + r]) {
        // gp_decode_step: the request took the step's token
        a.seq_lens_w[r] = m;
        if (a.positions) a.positions[r] += 1;
    }
    const int nchunks = cdiv(m, CHUNK);
    if (nchunks <= 1) return;
    const int Hq = a.Hkv * G;
    T *out = reinterpret_cast<T *>(a.out) + ((size_t)r * Hq + (size_t)h * G) * D;
    const float *base = a.partial + ((size_t)r * a.Hkv + h) * a.max_chunks * G * (D + 2);
    const int tid = threadIdx.x;
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
}

template <typename T, int D>
hipError_t launch_g(int G, const DecodeArgs &a, dim3 grid, int stages, hipStream_t s) {
    dim3 mgrid(a.Hkv, a.R);
    constexpr bool bf16 = sizeof(T) == 2;
    // the step variant (summaries and/or the new token folded in) is its own
    // instantiation, so plain decode attention carries none of its code
    const bool step = a.qstate != nullptr || a.k_new != nullptr;
    // the merge pass also advances the lengths when a token went in
    const bool chunks = stages & GP_DECODE_CHUNKS,
               merge = (stages & GP_DECODE_MERGE) && (a.max_chunks > 1 || (a.k_new && a.advance));
    switch (G) {
#define GP_CASE(GG)                                                  \
    case GG:                                                         \
        if (chunks && bf16 && step)                                  \
            decode_split_kernel<D, GG, true><<<grid, 64 * kDecodeWaves, 0, s>>>(a); \
        else if (chunks && bf16)                                     \
            decode_split_kernel<D, GG, false><<<grid, 64 * kDecodeWaves, 0, s>>>(a); \
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

// Paged GQA decode attention (Sec. 3.1, attention-output equation), split over
// the sequence.
//
// Work item = (request r, KV head h, chunk of kDecodeChunkPages pages).  One
// workgroup of wave64s serves the whole GQA group of h (G query heads),
// so every K/V byte is read from HBM exactly once per step.  Inside a wave a
// page (16 tokens x d) is read with fully coalesced 16-byte loads: lane l
// holds dims [c*EPL, c*EPL+EPL) of token j*TPL + l/LPT for each of the LPP
// loads, c = l % LPT.  Dot products are finished with cross-lane sums over
// the LPT lanes of a token; the online-softmax running max is made
// wave-uniform per page so that each lane can keep partial sums over its own
// tokens.  Waves take pages round-robin and two pages are in flight per wave.
// The four waves merge through LDS; a request that spans several chunks
// writes (max, sum, o) partials that a second, small kernel merges.
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

    const int h = blockIdx.x, chunk = blockIdx.y, r = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int Hkv = a.Hkv;
    const int Hq = Hkv * G;

    int P = a.num_pages[r];
    P = P < 0 ? 0 : (P > a.max_pages ? a.max_pages : P);
    int m = a.seq_lens[r];
    m = m < 0 ? 0 : (m > P * kPage ? P * kPage : m);
    const int nchunks = cdiv(m, CHUNK);
    T *out = reinterpret_cast<T *>(a.out) + ((size_t)r * Hq + (size_t)h * G) * D;
    if (m == 0) {
        if (chunk == 0)
            for (int i = threadIdx.x; i < G * D; i += blockDim.x) Tr::store(out + i, 0.0f);
        return;
    }
    if (chunk >= nchunks) return;

    const int tok_begin = chunk * CHUNK;
    const int tok_end = min(m, tok_begin + CHUNK);
    const int page_begin = tok_begin / kPage, page_end = cdiv(tok_end, kPage);

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
                    kr[u][j] = *reinterpret_cast<const uint4 *>(kpool + base + (size_t)j * TPL * D);
                    vr[u][j] = *reinterpret_cast<const uint4 *>(vpool + base + (size_t)j * TPL * D);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (!ok[u]) continue;   // wave-uniform
            float s[LPP][G];
#pragma unroll
            for (int j = 0; j < LPP; ++j) {
                float kf[EPL];
                Tr::unpack(kr[u][j], kf);
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
// in D/32 steps.  Lane l supplies token l%16 and a 32-element slice of the
// head dimension, so a lane reads D/4 consecutive elements of its token's
// key row; the same permutation of the head dimension is applied to Q.  The
// result leaves head 4*(l/16)+i of token l%16 in register i of lane l, so the
// per-page max and the row sums are 16-lane DPP reductions and every score is
// exponentiated once.  P.V stays on the vector ALUs in fp32: V is read in the
// coalesced layout of the fp32 path and the weights it needs are exchanged
// through LDS.
// ---------------------------------------------------------------------------
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

template <int N>
__device__ inline float dpp_ror(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x120 + N, 0xf, 0xf, false));
}
#ifndef GP_DECODE_PREFETCH
#define GP_DECODE_PREFETCH 0
#endif
#ifndef GP_DECODE_NT
#define GP_DECODE_NT 0
#endif
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte load of streamed K/V data.
__device__ inline uint4 ld16(const uint16_t *p) {
#if GP_DECODE_NT
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
#else
    return *reinterpret_cast<const uint4 *>(p);
#endif
}

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

template <int D, int G>
__global__ __launch_bounds__(64 * kDecodeWaves) void decode_mfma_kernel(DecodeArgs a) {
    constexpr int KK = D / 32;            // MFMA steps per page
    constexpr int KSPAN = D / 4;          // key elements per lane per page
    constexpr int LPT = D / 8;            // lanes per token, value layout
    constexpr int TPL = 64 / LPT;         // tokens per value load
    constexpr int LPP = kPage / TPL;      // value loads per page
    constexpr int HR = (G + 3) / 4;       // lane rows that carry real heads
    constexpr int GI = G < 4 ? G : 4;     // heads per lane row
    constexpr int NW = kDecodeWaves;
    constexpr int NP = kDecodeInFlight;   // pages per iteration and wave
    const int CHUNK = a.chunk_pages * kPage;

    __shared__ float s_m[NW][G], s_l[NW][G];
    __shared__ float s_o[NW][G][D];
    __shared__ float s_p[NW][NP][kPage][G];
    __shared__ float s_alpha[NW][G];
    __shared__ int s_ids[kDecodeChunkPages];

    const int h = blockIdx.x, chunk = blockIdx.y, r = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int Hkv = a.Hkv;
    const int Hq = Hkv * G;

    int P = a.num_pages[r];
    P = P < 0 ? 0 : (P > a.max_pages ? a.max_pages : P);
    int m = a.seq_lens[r];
    m = m < 0 ? 0 : (m > P * kPage ? P * kPage : m);
    const int nchunks = cdiv(m, CHUNK);
    uint16_t *out = reinterpret_cast<uint16_t *>(a.out) + ((size_t)r * Hq + (size_t)h * G) * D;
    if (m == 0) {
        if (chunk == 0)
            for (int i = threadIdx.x; i < G * D; i += blockDim.x) out[i] = 0;
        return;
    }
    if (chunk >= nchunks) return;
    const int tok_begin = chunk * CHUNK;
    const int tok_end = min(m, tok_begin + CHUNK);
    const int page_begin = tok_begin / kPage, page_end = cdiv(tok_end, kPage);

    // score layout: token n, key slice kg; value layout: token row vr, dims vc*8
    const int n = lane & 15, kg = lane >> 4;
    const int vrow = lane / LPT, vc = lane % LPT;

    // Q as the MFMA A operand (rows >= G are zero)
    const uint16_t *qg = reinterpret_cast<const uint16_t *>(a.q) + ((size_t)r * Hq + (size_t)h * G) * D;
    bf16x8_t qa[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        uint4 u = make_uint4(0u, 0u, 0u, 0u);
        if (n < G) u = *reinterpret_cast<const uint4 *>(qg + (size_t)n * D + kg * KSPAN + kk * 8);
        qa[kk] = __builtin_bit_cast(bf16x8_t, u);
    }

    float mrun[GI], lrun[GI], o[G][8];
#pragma unroll
    for (int i = 0; i < GI; ++i) {
        mrun[i] = kNegInf;
        lrun[i] = 0.0f;
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] = 0.0f;

    const int32_t *table = a.page_table + (size_t)r * a.max_pages;
    const uint16_t *kpool = reinterpret_cast<const uint16_t *>(a.k);
    const uint16_t *vpool = reinterpret_cast<const uint16_t *>(a.v);
    const size_t head_off = (size_t)h * kPage * D;
    const size_t page_elems = (size_t)Hkv * kPage * D;
    const int k_off = n * D + kg * KSPAN;
    const int v_off = vrow * D + vc * 8;

    // page ids of the chunk, read once into LDS; a wave reads its page's id
    // with a uniform LDS load
    for (int k = threadIdx.x; k < page_end - page_begin; k += blockDim.x) s_ids[k] = table[page_begin + k];
    __syncthreads();
    auto load_pages = [&](int pstart, uint4 (&kb)[NP][KK], uint4 (&vb)[NP][LPP], int (&ntok)[NP]) {
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            const int p = pstart + u * NW;
            const int phys = p < page_end ? s_ids[p - page_begin] : -1;
            const bool ok = phys >= 0 && phys < a.pool_pages;
            ntok[u] = ok ? min(kPage, m - p * kPage) : 0;
            const size_t base = (size_t)(ok ? phys : 0) * page_elems + head_off;
            if (ok) {
#pragma unroll
                for (int kk = 0; kk < KK; ++kk) kb[u][kk] = ld16(kpool + base + k_off + kk * 8);
#pragma unroll
                for (int j = 0; j < LPP; ++j) vb[u][j] = ld16(vpool + base + v_off + (size_t)j * TPL * D);
            }
        }
    };

    uint4 kb[NP][KK], vb[NP][LPP];
    int ntok[NP];
    int p0 = page_begin + wave;
#pragma unroll
    for (int u = 0; u < NP; ++u) ntok[u] = 0;
    if (p0 < page_end) load_pages(p0, kb, vb, ntok);
    for (; p0 < page_end; p0 += NP * NW) {
#if GP_DECODE_PREFETCH
        uint4 kn[NP][KK], vn[NP][LPP];
        int ntn[NP];
#pragma unroll
        for (int u = 0; u < NP; ++u) ntn[u] = 0;
        if (p0 + NP * NW < page_end) load_pages(p0 + NP * NW, kn, vn, ntn);
#endif
        // scores of NP pages; token n of page u, head 4*kg + i in s[u][i]
        float s[NP][GI];
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
            if (ntok[u] > 0) {
#pragma unroll
                for (int kk = 0; kk < KK; ++kk)
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kk], __builtin_bit_cast(bf16x8_t, kb[u][kk]),
                                                                  acc, 0, 0, 0);
            }
            const bool valid = n < ntok[u];
#pragma unroll
            for (int i = 0; i < GI; ++i) s[u][i] = valid ? acc[i] * a.qscale : kNegInf;
        }
        float alpha[GI];
#pragma unroll
        for (int i = 0; i < GI; ++i) {
            float pm = s[0][i];
#pragma unroll
            for (int u = 1; u < NP; ++u) pm = fmaxf(pm, s[u][i]);
            pm = row_max16(pm);
            const float mn = fmaxf(mrun[i], pm);
            alpha[i] = mn == kNegInf ? 1.0f : exp2f(mrun[i] - mn);
            mrun[i] = mn;
            float ps = 0.0f;
#pragma unroll
            for (int u = 0; u < NP; ++u) {
                s[u][i] = mn == kNegInf ? 0.0f : exp2f(s[u][i] - mn);
                ps += s[u][i];
            }
            lrun[i] = lrun[i] * alpha[i] + ps;
        }
        // hand the weights and the rescale factors to the value layout
        if (kg < HR) {
#pragma unroll
            for (int i = 0; i < GI; ++i) {
#pragma unroll
                for (int u = 0; u < NP; ++u) s_p[wave][u][n][kg * 4 + i] = s[u][i];
                if (n == 0) s_alpha[wave][kg * 4 + i] = alpha[i];
            }
        }
        wave_lds_sync();
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const float al = s_alpha[wave][g];
#pragma unroll
            for (int e = 0; e < 8; ++e) o[g][e] *= al;
        }
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            if (ntok[u] == 0) continue;   // wave-uniform
            const bool full = ntok[u] == kPage;
#pragma unroll
            for (int j = 0; j < LPP; ++j) {
                const int t = j * TPL + vrow;
                const bool valid = full || t < ntok[u];
                float vf[8];
                vf[0] = bf16_lo(vb[u][j].x); vf[1] = bf16_hi(vb[u][j].x);
                vf[2] = bf16_lo(vb[u][j].y); vf[3] = bf16_hi(vb[u][j].y);
                vf[4] = bf16_lo(vb[u][j].z); vf[5] = bf16_hi(vb[u][j].z);
                vf[6] = bf16_lo(vb[u][j].w); vf[7] = bf16_hi(vb[u][j].w);
#pragma unroll
                for (int e = 0; e < 8; ++e) vf[e] = valid ? vf[e] : 0.0f;
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const float pw = s_p[wave][u][t][g];
#pragma unroll
                    for (int e = 0; e < 8; ++e) o[g][e] = fmaf(pw, vf[e], o[g][e]);
                }
            }
        }
        wave_lds_sync();
#if GP_DECODE_PREFETCH
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            ntok[u] = ntn[u];
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) kb[u][kk] = kn[u][kk];
#pragma unroll
            for (int j = 0; j < LPP; ++j) vb[u][j] = vn[u][j];
        }
#else
#pragma unroll
        for (int u = 0; u < NP; ++u) ntok[u] = 0;
        if (p0 + NP * NW < page_end) load_pages(p0 + NP * NW, kb, vb, ntok);
#endif
    }

    // finish the wave: sums over the token rows of both layouts
#pragma unroll
    for (int i = 0; i < GI; ++i) lrun[i] = row_sum16(lrun[i]);
#pragma unroll
    for (int off = LPT; off < 64; off <<= 1)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < 8; ++e) o[g][e] += __shfl_xor(o[g][e], off, 64);
    if (kg < HR && n == 0) {
#pragma unroll
        for (int i = 0; i < GI; ++i) {
            s_m[wave][kg * 4 + i] = mrun[i];
            s_l[wave][kg * 4 + i] = lrun[i];
        }
    }
    if (vrow == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int e = 0; e < 8; ++e) s_o[wave][g][vc * 8 + e] = o[g][e];
    }
    __syncthreads();

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
            out[(size_t)g * D + dd] = f32_to_bf16(Os / Ls);
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
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void merge_kernel(DecodeArgs a) {
    using Tr = Traits<T>;
    const int CHUNK = a.chunk_pages * kPage;
    constexpr int MAXC = kMaxDecodeChunks;
    __shared__ float s_f[MAXC][G];                 // exp2(m_k - M) / L per chunk and head
    __shared__ float s_ml[MAXC][G][2];
    const int h = blockIdx.x, r = blockIdx.y;
    int P = a.num_pages[r];
    P = P < 0 ? 0 : (P > a.max_pages ? a.max_pages : P);
    int m = a.seq_lens[r];
    m = m < 0 ? 0 : (m > P * kPage ? P * kPage : m);
    const int nchunks = cdiv(m, CHUNK);
    if (nchunks <= 1) return;
    const int Hq = a.Hkv * G;
    T *out = reinterpret_cast<T *>(a.out) + ((size_t)r * Hq + (size_t)h * G) * D;
    const float *base = a.partial + ((size_t)r * a.Hkv + h) * a.max_chunks * G * (D + 2);
    const int tid = threadIdx.x;
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
hipError_t launch_g(int G, const DecodeArgs &a, dim3 grid, hipStream_t s) {
    dim3 mgrid(a.Hkv, a.R);
    constexpr bool bf16 = sizeof(T) == 2;
    switch (G) {
#define GP_CASE(GG)                                                  \
    case GG:                                                         \
        if (bf16)                                                    \
            decode_mfma_kernel<D, GG><<<grid, 64 * kDecodeWaves, 0, s>>>(a); \
        else                                                         \
            decode_kernel<float, D, GG><<<grid, 256, 0, s>>>(a);     \
        if (a.max_chunks > 1) merge_kernel<T, D, GG><<<mgrid, 256, 0, s>>>(a); \
        break;
        GP_CASE(1) GP_CASE(2) GP_CASE(4) GP_CASE(8)
#undef GP_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(gp_dtype_t dt, int D, int G, const DecodeArgs &a, hipStream_t s) {
    // the KV heads of one chunk are neighbours in dispatch order: they read the
    // head slices of the same pages at about the same time
    dim3 grid(a.Hkv, a.max_chunks, a.R);
    if (dt == GP_BF16)
        return D == 128 ? launch_g<uint16_t, 128>(G, a, grid, s) : launch_g<uint16_t, 64>(G, a, grid, s);
    return D == 128 ? launch_g<float, 128>(G, a, grid, s) : launch_g<float, 64>(G, a, grid, s);
}

}  // namespace gp

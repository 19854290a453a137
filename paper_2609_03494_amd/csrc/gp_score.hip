// Boundary scoring (Sec. 3.2 "attention-demand trend", Sec. 3.3 token score,
// App. E.1 "demand estimation at capacity boundaries").
//
// Three kernels per layer:
//  0. prep: per (boundary request, KV head) the 2G aligned summaries of its
//     GQA group (RMS calibration to the current query, then rotation at the
//     current position; fp64, angles computed on the device in fp64).
//  1. logits: per (boundary request, KV head, block of kStatBlock candidate
//     tokens), one wave: the block's 2G logits per token in fp64; the block's
//     max and sum of exponentials per view go to the workspace (fp64), and
//     exp(z - block max) per token is stored in float32 (relative error below
//     2^-24, about one rounding of the float32 weight it feeds).
//  2. weights: merge the block statistics per view, scale each token's
//     exponentials into softmax weights, average the G query heads of each
//     view (fp64), round to float32 and write a^S, a^L (workspace) and
//     s = max(a^S, a^L) (output).
//  3. top-p: per (request, KV head, view) a three-pass radix select on the
//     float32 bit patterns finds the smallest k whose k largest weights reach
//     p.  Per-bucket masses are accumulated as 2^-60 fixed-point integers, so
//     sums are exact and independent of thread order.
//
// Bound: the key read (|C| * d * sizeof(elem) per KV head) plus 2G float32
// exponentials written and read back; kernel 1 does 2G fp64 FMAs per key
// element.
#include "gp_internal.h"

namespace gp {

namespace {

template <typename T>
__device__ inline double ld(const T *p);
template <>
__device__ inline double ld<float>(const float *p) { return (double)*p; }
template <>
__device__ inline double ld<uint16_t>(const uint16_t *p) { return (double)bf16_to_f32(*p); }

template <typename T>
struct KRow;   // one element of a 16-byte unit of a key row, widened to fp64
template <>
struct KRow<uint16_t> {
    static constexpr int EPV = 8;
    __device__ static inline double elem(const uint4 &u, int e) {
        const uint32_t w = e < 2 ? u.x : e < 4 ? u.y : e < 6 ? u.z : u.w;
        return (e & 1) ? bf16_hi(w) : bf16_lo(w);
    }
};
template <>
struct KRow<float> {
    static constexpr int EPV = 4;
    __device__ static inline double elem(const uint4 &u, int e) {
        return __uint_as_float(e == 0 ? u.x : e == 1 ? u.y : e == 2 ? u.z : u.w);
    }
};

__device__ inline bool boundary_of(const ScoreArgs &a, int i, int &r, int &P) {
    r = a.bnd[i];
    if (r < 0 || r >= a.R) return false;
    P = a.num_pages[r];
    if (P < 2 || P > a.max_pages) return false;
    return a.seq_lens[r] == P * kPage;
}

// Products and sums are rounded one at a time, as in a plain fp64 evaluation.
#pragma clang fp contract(off)

// --------------------------------------------------------------------- prep --
// One workgroup per (boundary request, KV head): the 2G summaries of its GQA
// group scaled to the RMS of the current query (RMS calibration) and rotated
// at the current position; angles pos * theta^(-2k/D) and their sine and
// cosine are computed in fp64 on the device.
template <typename T, int D, int G>
__global__ __launch_bounds__(256, 5) void prep_kernel(ScoreArgs a) {
    constexpr int V = 2 * G;
    constexpr int H = D / 2;
    __shared__ double s_q[V][D];
    __shared__ double s_qt[G][D];
    __shared__ double s_cos[H], s_sin[H];
    __shared__ double s_ss[3 * G];
    const int h = blockIdx.x, i = blockIdx.y;
    int r, P;
    if (!boundary_of(a, i, r, P)) return;
    const int slot = a.slot_ids[r];
    if (slot < 0 || slot >= a.M) return;
    const int tid = threadIdx.x;
    const int Hq = a.Hkv * G;
    const float *qs = a.qstate + (size_t)slot * 2 * Hq * D;
    const T *qp = reinterpret_cast<const T *>(a.q_pre) + (size_t)r * Hq * D;
    for (int e = tid; e < V * D; e += blockDim.x) {
        const int v = e / D, d = e % D, x = v / G, g = v % G;
        s_q[v][d] = (double)qs[((size_t)x * Hq + h * G + g) * D + d];
    }
    for (int e = tid; e < G * D; e += blockDim.x) {
        const int g = e / D, d = e % D;
        s_qt[g][d] = ld<T>(qp + (size_t)(h * G + g) * D + d);
    }
    const double pos = (double)a.positions[r];
    for (int k = tid; k < H; k += blockDim.x) {
        const double ang = pos * pow(a.theta, (-2.0 * k) / D);
        s_cos[k] = cos(ang);
        s_sin[k] = sin(ang);
    }
    __syncthreads();
    // 3G sums of squares, 8 lanes each
    if (tid < 3 * G * 8) {
        const int which = tid / 8, part = tid % 8;
        const double *src = which < V ? s_q[which] : s_qt[which - V];
        double acc = 0.0;
#pragma unroll
        for (int d = part * (D / 8); d < (part + 1) * (D / 8); ++d) acc += src[d] * src[d];
        acc += __shfl_xor(acc, 1, 8);
        acc += __shfl_xor(acc, 2, 8);
        acc += __shfl_xor(acc, 4, 8);
        if (part == 0) s_ss[which] = acc;
    }
    __syncthreads();
    double *out = a.qt + ((size_t)i * a.Hkv + h) * V * D;
    for (int e = tid; e < V * H; e += blockDim.x) {
        const int v = e / H, k = e % H, g = v % G;
        const double den = s_ss[v];
        const double gam = den == 0.0 ? 0.0 : sqrt(s_ss[V + g] / D) / sqrt(den / D);
        const double x1 = gam * s_q[v][k], x2 = gam * s_q[v][k + H];
        out[(size_t)v * D + k] = x1 * s_cos[k] - x2 * s_sin[k];
        out[(size_t)v * D + k + H] = x2 * s_cos[k] + x1 * s_sin[k];
    }
}

// ------------------------------------------------------------------- logits --
// Grid (KV head, blocks of kStatBlock candidates, boundary request), two
// waves per workgroup, 32 candidates each.  The 2G x D logits of the block are a small fp64 matrix
// product, done on the matrix cores with v_mfma_f64_16x16x4f64: the A operand
// is the aligned summaries (row = view, padded to 16 rows with zeros), B the
// keys of 16 candidates, so each wave runs two chains of D/4 MFMAs.  The
// contraction over head dimensions is split four ways across lane groups: in
// step s, lane group q (lanes 16q .. 16q+15) supplies dimension (D/4) q + s,
// so each lane reads one contiguous quarter row of summaries (once) and of
// each of its keys.  The result leaves view 4j + q of candidate l % 16 in
// register j of lane l.  Per view, the block's max m and sum of exp(z - m)
// (16-lane reductions, then across the two waves in LDS) go to the
// statistics array; exp(z - m) of each token
// is stored (float32), so that the weights need a product, not an
// exponential, per token.  A lane whose page id is invalid contributes zero logits.
typedef double f64x4_t __attribute__((ext_vector_type(4)));
constexpr int kLogitsWaves = 2;                 // waves per block of kStatBlock candidates

template <typename T, int D, int G>
__global__ __launch_bounds__(64 * kLogitsWaves) void logits_kernel(ScoreArgs a) {
    constexpr int V = 2 * G;
    constexpr int S = D / 4;                         // MFMA steps (head dimensions per lane group)
    constexpr int EPU = 16 / sizeof(T);              // key elements per 16-byte unit
    constexpr int NU = S / EPU;                      // 16-byte units of a quarter key row
    constexpr int NW = kLogitsWaves;
    constexpr int NGRP = kStatBlock / 16 / NW;       // candidate groups of 16 per wave
    static_assert(kStatBlock == 64 && V <= 16 && S % EPU == 0 && NGRP * 16 * NW == kStatBlock, "layout");
    __shared__ double s_wm[NW][16], s_ws[NW][16];

    const int h = blockIdx.x, blk = blockIdx.y, i = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, q = lane >> 4;
    int r, P;
    if (!boundary_of(a, i, r, P)) return;
    const int C = (P - 1) * kPage;
    const int t0 = blk * kStatBlock;
    if (t0 >= C) return;
    const int slot = a.slot_ids[r];
    if (slot < 0 || slot >= a.M) return;

    // A: this lane's quarter row of summary `col` (zero rows pad the views to 16)
    // (every load below reads a valid address, clamped where the lane has no
    // data, and the value is zeroed afterwards: the loads are all in flight at
    // once instead of one masked load and wait at a time)
    const double *qt = a.qt + (((size_t)i * a.Hkv + h) * V + min(col, V - 1)) * D + q * S;
    double qa[S];
#pragma unroll
    for (int s2 = 0; s2 < S; s2 += 2) {
        const double2 u = *reinterpret_cast<const double2 *>(qt + s2);
        qa[s2] = col < V ? u.x : 0.0;
        qa[s2 + 1] = col < V ? u.y : 0.0;
    }
    // B: this lane's quarter row of candidate t0 + 16 g + col, for the 4 groups
    uint4 kb[NGRP][NU];
    const int tw = t0 + 16 * NGRP * wave;            // this wave's first candidate
#pragma unroll
    for (int g = 0; g < NGRP; ++g) {
        const int t = tw + 16 * g + col;
        const int pe = a.page_table[(size_t)r * a.max_pages + min(t, C - 1) / kPage];
        const int phys = t < C ? pe : -1;
        const bool ok = phys >= 0 && phys < a.pool_pages;
        const uint4 *kp = reinterpret_cast<const uint4 *>(reinterpret_cast<const T *>(a.k) +
                          (((size_t)(ok ? phys : 0) * a.Hkv + h) * kPage + (t % kPage)) * D + q * S);
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const uint4 x = kp[u];
            kb[g][u] = ok ? x : make_uint4(0u, 0u, 0u, 0u);
        }
    }
    f64x4_t acc[NGRP];
#pragma unroll
    for (int g = 0; g < NGRP; ++g) acc[g] = f64x4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int s2 = 0; s2 < S; ++s2) {
#pragma unroll
        for (int g = 0; g < NGRP; ++g) {
            const double b = KRow<T>::elem(kb[g][s2 / EPU], s2 % EPU);
            acc[g] = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[s2], b, acc[g], 0, 0, 0);
        }
    }

    // statistics and exponentials per view (register j holds view 4j + q):
    // per wave over its candidates, then the block's max and sum across the
    // waves through LDS
    float *lgv = a.expz + ((size_t)i * a.Hkv + h) * V * a.cmax;
    double *pt = a.part + (((size_t)i * a.Hkv + h) * a.nch + blk) * V * 2;
    double z[4][NGRP], mv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        mv[j] = -__builtin_huge_val();
        if (4 * j >= V) continue;                    // uniform: no real view in this register
#pragma unroll
        for (int g = 0; g < NGRP; ++g) {
            z[j][g] = acc[g][j] * a.scale;
            if (tw + 16 * g + col < C) mv[j] = fmax(mv[j], z[j][g]);
        }
        for (int off = 8; off >= 1; off >>= 1) mv[j] = fmax(mv[j], __shfl_xor(mv[j], off, 16));
        if (NW > 1 && col == 0) s_wm[wave][4 * j + q] = mv[j];
    }
    if (NW > 1) {
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (4 * j >= V) continue;
            double m = s_wm[0][4 * j + q];
#pragma unroll
            for (int w = 1; w < NW; ++w) m = fmax(m, s_wm[w][4 * j + q]);
            mv[j] = m;
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int v = 4 * j + q;
        if (4 * j >= V) continue;
        double sv = 0.0;
#pragma unroll
        for (int g = 0; g < NGRP; ++g) {
            const int t = tw + 16 * g + col;
            if (t < C && v < V) {
                const double ev = exp(z[j][g] - mv[j]);
                sv += ev;
                lgv[(size_t)v * a.cmax + t] = (float)ev;
            }
        }
        for (int off = 8; off >= 1; off >>= 1) sv += __shfl_xor(sv, off, 16);
        if (NW > 1) {
            if (col == 0) s_ws[wave][v] = sv;
        } else if (col == 0 && v < V) {
            pt[v * 2] = mv[j];
            pt[v * 2 + 1] = sv;
        }
    }
    if (NW > 1) {
        __syncthreads();
        if (wave == 0 && col == 0) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int v = 4 * j + q;
                if (4 * j >= V || v >= V) continue;
                double tot = 0.0;
#pragma unroll
                for (int w = 0; w < NW; ++w) tot += s_ws[w][v];
                pt[v * 2] = mv[j];
                pt[v * 2 + 1] = tot;
            }
        }
    }
}

// ------------------------------------------------------------------ weights --
// Grid (KV head, chunks of kProbChunk candidates, boundary request).  The
// statistics blocks are merged per view: M = max m_b, L = sum s_b exp(m_b - M);
// then each block b of the chunk gets the factor f_b = exp(m_b - M) / L, and a
// token's softmax weight in view (g, x) is its stored exp(z - m_b) times f_b.
// The G query heads of a view are averaged in fp64 and rounded to float32.
template <int G>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(G >= 8 ? 4 : 5))) void weights_kernel(ScoreArgs a) {
    constexpr int V = 2 * G;
    constexpr int BPC = kProbChunk / kStatBlock;     // statistics blocks per chunk
    constexpr int TPT = kProbChunk / 256;            // tokens per thread
    constexpr int NPL = 4;                           // statistics blocks per lane kept in registers
    __shared__ double s_M[V], s_L[V];
    __shared__ double s_f[BPC][V];
    const int h = blockIdx.x, chunk = blockIdx.y, i = blockIdx.z;
    int r, P;
    if (!boundary_of(a, i, r, P)) return;
    const int C = (P - 1) * kPage;
    const int t0 = chunk * kProbChunk;
    if (t0 >= C) return;
    const int tid = threadIdx.x;
    const int used = cdiv(C, kStatBlock);
    const int b0 = t0 / kStatBlock;
    const double *pt = a.part + (((size_t)i * a.Hkv + h) * a.nch) * V * 2;
    const float *lg = a.expz + ((size_t)i * a.Hkv + h) * V * a.cmax;

    // The kernel runs beside decode attention, where every memory round trip
    // is slow: the exponentials of this thread's tokens and the statistics
    // are all requested before any of them is used.
    float e[TPT][V];
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int t = t0 + k * 256 + tid;
#pragma unroll
        for (int v = 0; v < V; ++v) e[k][v] = lg[(size_t)v * a.cmax + min(t, C - 1)];
    }
    // merge the block statistics: 32 lanes per view, views 8 at a time; lane
    // c0 holds blocks c0, c0 + 32, ... (the first NPL of them in registers)
    for (int vb = 0; vb < V; vb += 8) {
        const int v = vb + tid / 32, c0 = tid % 32;
        if (v < V) {
            double mk[NPL], sk[NPL];
#pragma unroll
            for (int k = 0; k < NPL; ++k) {
                const int c = c0 + 32 * k;
                const double *pc = pt + ((size_t)min(c, used - 1) * V + v) * 2;
                mk[k] = pc[0];
                sk[k] = pc[1];
            }
            double M = -__builtin_huge_val();
#pragma unroll
            for (int k = 0; k < NPL; ++k) M = fmax(M, mk[k]);
            for (int c = c0 + 32 * NPL; c < used; c += 32) M = fmax(M, pt[((size_t)c * V + v) * 2]);
            for (int off = 16; off >= 1; off >>= 1) M = fmax(M, __shfl_xor(M, off, 32));
            double L = 0.0;
#pragma unroll
            for (int k = 0; k < NPL; ++k)
                if (c0 + 32 * k < used) L += sk[k] * exp(mk[k] - M);
            for (int c = c0 + 32 * NPL; c < used; c += 32)
                L += pt[((size_t)c * V + v) * 2 + 1] * exp(pt[((size_t)c * V + v) * 2] - M);
            for (int off = 16; off >= 1; off >>= 1) L += __shfl_xor(L, off, 32);
            // factors of the chunk's blocks: f_b = exp(m_b - M) / L
#pragma unroll
            for (int k = 0; k < NPL; ++k) {
                const int c = c0 + 32 * k;
                if (c < used && c >= b0 && c < b0 + BPC) s_f[c - b0][v] = exp(mk[k] - M) / L;
            }
            for (int c = c0 + 32 * NPL; c < used; c += 32)
                if (c >= b0 && c < b0 + BPC) s_f[c - b0][v] = exp(pt[((size_t)c * V + v) * 2] - M) / L;
        }
    }
    __syncthreads();
    float *w = a.weights + ((size_t)i * a.Hkv + h) * 2 * a.cmax;
    float *sc = a.scores + ((size_t)i * a.Hkv + h) * a.max_cand;
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int t = t0 + k * 256 + tid;
        if (t >= C) continue;
        const int bb = (t - t0) / kStatBlock;
        float ax[2];
#pragma unroll
        for (int x = 0; x < 2; ++x) {
            double acc = 0.0;
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const int v = x * G + g;
                acc += (double)e[k][v] * s_f[bb][v];
            }
            ax[x] = (float)(acc / G);
            w[(size_t)x * a.cmax + t] = ax[x];
        }
        sc[t] = fmaxf(ax[0], ax[1]);
    }
}

__device__ inline unsigned long long fixed60(uint32_t bits) {
    return (unsigned long long)ldexp((double)__uint_as_float(bits), 60);
}

// -------------------------------------------------------------------- top-p --
// One workgroup of kTopPThreads threads per (boundary request, KV head, view).
// Each of the three radix passes histograms the weights that share the prefix
// found so far (count and 2^-60 fixed-point mass per bucket), then the
// workgroup scans the buckets from the top to find the one where the running
// mass reaches p.  The workgroup is small (one wave per SIMD) so that it can
// start beside decode attention, which leaves a quarter of each SIMD's
// registers free.
constexpr int kTopPThreads = 256;
__global__ __launch_bounds__(kTopPThreads, 5) void top_p_kernel(ScoreArgs a) {
    constexpr int NT = kTopPThreads;
    constexpr int NB = 2048;
    constexpr int CW = 4096 / NT;                   // weights per thread kept in registers
    constexpr int NWV = NT / 64;
    __shared__ unsigned int s_cnt[NB];
    __shared__ unsigned long long s_mass[NB];
    __shared__ int s_bucket;
    __shared__ unsigned long long s_above_mass;
    __shared__ unsigned int s_above_cnt;
    __shared__ unsigned long long s_wmass[NWV];
    __shared__ unsigned int s_wcnt[NWV];

    const int h = blockIdx.x, x = blockIdx.y, i = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63;
    int32_t *out = a.k_counts + ((size_t)i * a.Hkv + h) * 2 + x;
    int r, P;
    if (!boundary_of(a, i, r, P)) {
        if (tid == 0) *out = 0;
        return;
    }
    const int C = (P - 1) * kPage;
    const float *wv = a.weights + (((size_t)i * a.Hkv + h) * 2 + x) * a.cmax;
    const unsigned long long target = (unsigned long long)ldexp(a.p, 60);

    // the first CW * NT weights stay in registers across the passes (every
    // candidate set up to 4096 tokens); longer ones re-read the rest
    // (loads at clamped indices, so that all of them are in flight at once)
    uint32_t cached[CW];
#pragma unroll
    for (int k = 0; k < CW; ++k) cached[k] = 0xffffffffu;
    if (C > 0) {
#pragma unroll
        for (int k = 0; k < CW; ++k) {
            const int t = k * NT + tid;
            const uint32_t u = __float_as_uint(wv[min(t, C - 1)]);
            cached[k] = t < C ? u : 0xffffffffu;
        }
    }
    uint32_t prefix = 0;
    unsigned long long above_mass = 0;
    unsigned int above_cnt = 0;
    const int shifts[3] = {20, 9, 0};
    const int nbits[3] = {11, 11, 9};
    for (int pass = 0; pass < 3; ++pass) {
        const int sh = shifts[pass], nb = 1 << nbits[pass];
        for (int b = tid; b < nb; b += NT) {
            s_cnt[b] = 0;
            s_mass[b] = 0;
        }
        __syncthreads();
        auto count = [&](uint32_t u) {
            if (u != 0xffffffffu && (u >> (sh + nbits[pass])) == prefix) {
                const int b = (u >> sh) & (nb - 1);
                atomicAdd(&s_cnt[b], 1u);
                atomicAdd(&s_mass[b], fixed60(u));
            }
        };
#pragma unroll
        for (int k = 0; k < CW; ++k) count(cached[k]);
        for (int base = CW * NT; base < C; base += 4 * NT) {
            uint32_t u[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int t = base + k * NT + tid;
                const uint32_t y = __float_as_uint(wv[min(t, C - 1)]);
                u[k] = t < C ? y : 0xffffffffu;
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) count(u[k]);
        }
        __syncthreads();
        // Scan of the buckets from the highest down, over the whole workgroup:
        // thread t owns descending positions [t * per, (t + 1) * per).  The
        // thread whose range holds the position where the running mass first
        // reaches the mass still needed names that bucket, with the count and
        // mass strictly above it.
        {
            const int per = nb >= NT ? nb / NT : 1;
            const bool owns = tid * per < nb;
            unsigned long long mm = 0;
            unsigned int cc = 0;
            if (owns)
                for (int k = 0; k < per; ++k) {
                    const int b = nb - 1 - (tid * per + k);
                    mm += s_mass[b];
                    cc += s_cnt[b];
                }
            unsigned long long im = mm;
            unsigned int ic = cc;
            for (int off = 1; off < 64; off <<= 1) {
                const unsigned long long ym = __shfl_up(im, off, 64);
                const unsigned int yc = __shfl_up(ic, off, 64);
                if (lane >= off) {
                    im += ym;
                    ic += yc;
                }
            }
            if (lane == 63) {
                s_wmass[tid >> 6] = im;
                s_wcnt[tid >> 6] = ic;
            }
            __syncthreads();
            for (int w = 0; w < (tid >> 6); ++w) {
                im += s_wmass[w];
                ic += s_wcnt[w];
            }
            const unsigned long long need = target > above_mass ? target - above_mass : 0ull;
            const unsigned long long em = im - mm;
            const unsigned int ec = ic - cc;
            if (tid == NT - 1 && im < need) s_bucket = -1;    // the candidates fall short of p
            if (owns && em < need && im >= need) {
                unsigned long long cum = em;
                unsigned int cnt = ec;
                for (int k = 0; k < per; ++k) {
                    const int b = nb - 1 - (tid * per + k);
                    if (cum + s_mass[b] >= need) {
                        s_bucket = b;
                        s_above_mass = cum;
                        s_above_cnt = cnt;
                        break;
                    }
                    cum += s_mass[b];
                    cnt += s_cnt[b];
                }
            }
        }
        __syncthreads();
        const int B = s_bucket;
        if (B < 0) {
            // the weights sum to less than p: every candidate is needed
            if (tid == 0) *out = C;
            return;
        }
        above_mass += s_above_mass;
        above_cnt += s_above_cnt;
        prefix = (prefix << nbits[pass]) | (uint32_t)B;
        __syncthreads();
    }
    if (tid == 0) {
        // prefix is now the float32 bit pattern of the K-th largest weight T
        const unsigned long long tf = fixed60(prefix);
        const unsigned long long need = target - above_mass;   // > 0
        const unsigned long long j = tf == 0 ? 0ull : (need + tf - 1) / tf;
        long long K = (long long)above_cnt + (long long)j;
        if (tf == 0 || K > C) K = C;
        *out = (int32_t)K;
    }
}

// ------------------------------------------------------------------ entropy --
// The signal ablation's alternative demand metric: per (request, KV head,
// view) the entropy H = -sum a ln a of the float32 weights (fp64, zero weights
// contribute nothing) and K = exp(H) rounded to the nearest integer, clamped
// to [1, |C|].
__global__ __launch_bounds__(256) void entropy_kernel(ScoreArgs a) {
    __shared__ double s_red[4];
    const int h = blockIdx.x, x = blockIdx.y, i = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int32_t *out = a.k_counts + ((size_t)i * a.Hkv + h) * 2 + x;
    int r, P;
    if (!boundary_of(a, i, r, P)) {
        if (tid == 0) *out = 0;
        return;
    }
    const int C = (P - 1) * kPage;
    const float *wv = a.weights + (((size_t)i * a.Hkv + h) * 2 + x) * a.cmax;
    double acc = 0.0;
    // four weights per round, loaded at clamped indices so that they are in
    // flight together; the sum runs in the same order as one at a time
    for (int t = tid; t < C; t += 4 * blockDim.x) {
        float y[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) y[k] = wv[min(t + k * (int)blockDim.x, C - 1)];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const double w = (double)y[k];
            if (t + k * (int)blockDim.x < C && w > 0.0) acc += w * log(w);
        }
    }
    for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (lane == 0) s_red[wave] = acc;
    __syncthreads();
    if (tid == 0) {
        const double H = -(s_red[0] + s_red[1] + s_red[2] + s_red[3]);
        const double e = floor(exp(H) + 0.5);
        *out = e < 1.0 ? 1 : (e > (double)C ? C : (int)e);
    }
}

template <typename T, int D>
hipError_t launch_gd(int G, const ScoreArgs &a, hipStream_t s) {
    // the KV head is the fastest grid index everywhere: workgroups are handed to
    // the XCDs round-robin, so head h's workgroups all run on one XCD and read
    // back what the previous kernel left in that XCD's L2
    dim3 g0(a.Hkv, a.Rb), g1(a.Hkv, cdiv(a.cmax, kStatBlock), a.Rb), g2(a.Hkv, cdiv(a.cmax, kProbChunk), a.Rb), g3(a.Hkv, 2, a.Rb);
    if (a.cmax == 0) {
        // no request can have candidates: the counts are written as zero
        top_p_kernel<<<g3, kTopPThreads, 0, s>>>(a);
        return hipGetLastError();
    }
    switch (G) {
#define GP_CASE(GG)                                                   \
    case GG:                                                          \
        prep_kernel<T, D, GG><<<g0, 256, 0, s>>>(a);                  \
        logits_kernel<T, D, GG><<<g1, 64 * kLogitsWaves, 0, s>>>(a);                \
        weights_kernel<GG><<<g2, 256, 0, s>>>(a);                     \
        break;
        GP_CASE(1) GP_CASE(2) GP_CASE(4) GP_CASE(8)
#undef GP_CASE
        default: return hipErrorInvalidValue;
    }
    if (a.metric == GP_METRIC_ENTROPY)
        entropy_kernel<<<g3, 256, 0, s>>>(a);
    else
        top_p_kernel<<<g3, kTopPThreads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_score(gp_dtype_t dt, int D, int G, const ScoreArgs &a, hipStream_t s) {
    if (a.Rb == 0) return hipSuccess;
    if (dt == GP_BF16) return D == 128 ? launch_gd<uint16_t, 128>(G, a, s) : launch_gd<uint16_t, 64>(G, a, s);
    return D == 128 ? launch_gd<float, 128>(G, a, s) : launch_gd<float, 64>(G, a, s);
}

}  // namespace gp

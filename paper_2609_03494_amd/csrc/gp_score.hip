// Boundary scoring (Sec. 3.2 "attention-demand trend", Sec. 3.3 token score,
// App. E.1 "demand estimation at capacity boundaries").
//
// Three kernels per layer:
//  0. logits: per (boundary request, KV head, set of blocks of kStatBlock
//     candidate tokens), one wave: first the 2G aligned summaries of the GQA
//     group (RMS calibration to the current query, then rotation at the
//     current position; fp64, angles computed on the device in fp64), then
//     each block's 2G logits per token in fp64
//     on the fp64 matrix cores; the block's max and sum of exponentials per
//     view go to the workspace (fp64), and exp(z - block max) per token is
//     stored in float32 (relative error about 2^-24: one rounding of the
//     float32 weight it feeds).
//  1. weights: merge the block statistics per view, scale each token's
//     exponentials into softmax weights, average the G query heads of each
//     view (fp64), round to float32 and write a^S, a^L (workspace) and
//     s = max(a^S, a^L) (output).
//  2. top-p: per (request, KV head, view) a three-pass radix select on the
//     float32 bit patterns finds the smallest k whose k largest weights reach
//     p.  Per-bucket masses are accumulated as 2^-60 fixed-point integers, so
//     sums are exact and independent of thread order.
//
// Bound: the key read (|C| * d * sizeof(elem) per KV head) plus 2G float32
// exponentials written and read back; kernel 0 does 2G fp64 FMAs per key
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

// exp(x) for x <= 0 in fp64, to a relative error below 2^-36: x = n ln 2 + r
// with |r| <= ln 2 / 2 (n = rint(x / ln 2), ln 2 in two parts so that r is
// exact to fp64 rounding), exp(r) by its Taylor polynomial of degree 9
// (truncation below 0.35^10 / 10! < 2^-37), then scaled by 2^n; results
// below the smallest fp64 denormal flush to zero in the scaling.  The
// exponentials feed float32 values and an fp64 sum, so this is far below
// the rounding they then take.
// (The coefficients are pinned to scalar registers, so that each Horner step
// is one three-operand FMA rather than a copy of the constant and an FMA.)
__device__ inline double sreg(double c) {
    double r;
    asm("" : "=s"(r) : "0"(c));
    return r;
}
__device__ inline double exp_nonpos(double x) {
    const double n = __builtin_rint(x * sreg(1.4426950408889634));
    double r = __builtin_fma(-n, sreg(6.93147180369123816490e-01), x);
    r = __builtin_fma(-n, sreg(1.90821492927058770002e-10), r);
    double p = sreg(1.0 / 362880.0);
    p = __builtin_fma(p, r, sreg(1.0 / 40320.0));
    p = __builtin_fma(p, r, sreg(1.0 / 5040.0));
    p = __builtin_fma(p, r, sreg(1.0 / 720.0));
    p = __builtin_fma(p, r, sreg(1.0 / 120.0));
    p = __builtin_fma(p, r, sreg(1.0 / 24.0));
    p = __builtin_fma(p, r, sreg(1.0 / 6.0));
    p = __builtin_fma(p, r, 0.5);
    p = __builtin_fma(p, r, 1.0);
    p = __builtin_fma(p, r, 1.0);
    return __builtin_ldexp(p, (int)fmax(n, -2100.0));
}

// LDS traffic between lanes of one wave: wait for the wave's LDS operations
// and keep the compiler from moving memory accesses across this point.
__device__ inline void wave_lds_sync() { __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// max without the NaN canonicalisation of fmax (the operands are finite or -inf)
__device__ inline double max_f64(double a, double b) { return a > b ? a : b; }

// x from the lane N places down in its row of 16 (rotating), for an fp64 value
template <int N>
__device__ inline double dpp_ror_f64(double x) {
    const long long b = __builtin_bit_cast(long long, x);
    const int lo = __builtin_amdgcn_mov_dpp((int)b, 0x120 + N, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), 0x120 + N, 0xf, 0xf, false);
    return __builtin_bit_cast(double, ((long long)hi << 32) | (unsigned)lo);
}

// slot (optional): the request's summary slot, which must lie in [0, M).
__device__ inline bool boundary_of(const ScoreArgs &a, int i, int &r, int &P, int *slot = nullptr) {
    r = a.bnd[i];
    if (a.R <= 0) return false;
    // the page count, the length (and the slot) are requested together, at a
    // clamped index: beside decode attention every round trip costs
    // microseconds
    const int rc = min(max(r, 0), a.R - 1);
    P = a.num_pages[rc];
    const int m = a.seq_lens[rc];
    bool ok = true;
    if (slot) {
        *slot = a.slot_ids[rc];
        ok = (*slot >= 0) & (*slot < a.M);
    }
    // one test of all the values (no branch between the loads)
    return ok & (r >= 0) & (r < a.R) & (P >= 2) & (P <= a.max_pages) & (m == P * kPage);
}

// Products and sums are rounded one at a time, as in a plain fp64 evaluation.
#pragma clang fp contract(off)

// ------------------------------------------------------------------- logits --
// Grid (KV head, split / kLogitsWaves, boundary request); each wave of a
// workgroup is one split, and the waves share the summaries in LDS (with one
// wave per workgroup the LDS copy of the summaries, not registers, would cap
// the waves per CU).  Split y of a request handles statistics blocks y,
// y + splits, y + 2 splits, ... (at most kLogitsMaxIters) of kStatBlock = 64
// candidates each.  The 2G x D
// logits of a block are a small fp64 matrix product on the matrix cores,
// v_mfma_f64_4x4x4f64: four independent 4 x 4 x 4 products per instruction
// (16 cycles for 512 flops, the same rate per flop as 16x16x4, but with no
// padding rows at 2G <= 8 views).  Lane l = 16 k + 4 b + j holds row j of
// block b's A and column j of its B for contraction index k, and element
// (k, j) of its result.  The four blocks are four groups of 4 candidates
// (B = their keys), A is one quarter of the views (4 vh .. 4 vh + 3, the same
// in all blocks), so one key operand feeds ceil(2G / 4) instructions and each
// key element is loaded and widened once.  The four lanes of a candidate (k =
// 0..3) read adjacent 16-byte units of its key row, so that one load
// instruction touches one 64-byte segment per candidate: unit u of lane k is
// unit 4 u + k of the row, and contraction step s of lane group k takes head
// dimension dim(k, s) = 4 E (s / E) + E k + s % E (E elements per unit).  The
// summaries come from LDS, laid out [k][view][s] in that order, with paddings
// that put the 16 doubles of one read on distinct banks.
//
// A block is taken in two halves of 32 candidates (two groups of 16, one key
// register set each); while one half is multiplied the keys of the next half
// are in flight, and the page ids of all the workgroup's blocks are read
// once at the start, so the wave waits for memory once, not once per block.
// Per view, the block's max m and sum of exp(z - m) (fp64, 16-lane DPP
// reductions) go to the statistics array, and exp(z - m) of each token is
// stored (float32), so that the weights need a product, not an exponential,
// per token.  A candidate whose page id is invalid contributes zero logits.
constexpr int kLogitsMaxIters = 32;
#ifndef GP_LOGITS_WAVES
#define GP_LOGITS_WAVES 2
#endif
constexpr int kLogitsWaves = GP_LOGITS_WAVES;   // waves per workgroup, sharing the summaries in LDS
#ifndef GP_LOGITS_TARGET_WAVES
#define GP_LOGITS_TARGET_WAVES 16384
#endif

template <typename T, int D, int G>
__global__ __launch_bounds__(64 * kLogitsWaves) void logits_kernel(ScoreArgs a) {
    __builtin_amdgcn_s_setprio(3);   // issue ahead of co-resident decode waves
    constexpr int V = 2 * G;
    constexpr int VH = (V + 3) / 4;                  // view quarters (MFMAs per key operand)
    constexpr int VR = 4 * VH;                       // view rows in LDS (rows >= V are zero)
    constexpr int S = D / 4;                         // MFMA steps (head dimensions per lane group)
    constexpr int EPU = 16 / sizeof(T);              // key elements per 16-byte unit
    constexpr int NU = S / EPU;                      // 16-byte units of a quarter key row
    constexpr int SP = S + 1;                        // view row stride (doubles)
    constexpr int KS = VR * SP + (8 - (VR * SP) % 32 + 32) % 32;   // k stride, = 8 mod 32 doubles
    static_assert(kStatBlock == 64 && kPage == 16 && S % EPU == 0, "layout");
    __shared__ double s_a[4 * KS];
    __shared__ int s_pgs[kLogitsWaves][4 * kLogitsMaxIters];

    // wave w of the workgroup takes block set y = blockIdx.y * waves + w
    const int h = blockIdx.x, i = blockIdx.z;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int y = blockIdx.y * kLogitsWaves + wave, ny = gridDim.y * kLogitsWaves;
    int *s_pg = s_pgs[wave];
    const int k = lane >> 4, cand = lane & 15;      // contraction / output row; candidate 4 b + j
    // Round trips are slow beside decode attention, so the prologue takes
    // three: the request index; then, together, everything that needs only
    // the request (its page count, length and summary slot, the page ids of
    // this wave's blocks, the query and the position; clamped indices, values
    // dropped afterwards where unused); then the summaries, which need the
    // slot, beside the first keys.  The candidate count of the event goes to
    // the workspace for the kernels that follow.
    constexpr int PPL = 4 * kLogitsMaxIters / 64;               // page ids per lane
    static_assert(4 * kLogitsMaxIters % 64 == 0, "page ids per lane");
    constexpr int NT = 64 * kLogitsWaves;
    const bool writer = h == 0 && blockIdx.y == 0 && threadIdx.x == 0;
    if (a.R <= 0) {
        if (writer) a.cand[i] = 0;
        return;
    }
    const int r = a.bnd[i];
    const int rc = min(max(r, 0), a.R - 1);
    const int P = a.num_pages[rc], m_r = a.seq_lens[rc], slot = a.slot_ids[rc];
    int pev[PPL];
#pragma unroll
    for (int j = 0; j < PPL; ++j) {
        const int e = lane + 64 * j, pg = 4 * (y + ny * (e / 4)) + e % 4;
        pev[j] = a.page_table[(size_t)rc * a.max_pages + min(pg, a.max_pages - 1)];
    }
    // The 2G summaries of the workgroup's GQA group (Sec. 3.2, App. E.1):
    // thread (view row vr, lane lr of TPR) holds the rotation pairs (k, k +
    // D/2), k = lr, lr + TPR, ...; each row is scaled to the RMS of its query
    // head (RMS calibration) and rotated at the current position (angles pos *
    // theta^(-2k/D), sine and cosine in fp64 on the device).
    constexpr int H = D / 2;
    constexpr int TPR = NT / V;                                 // threads per view row
    constexpr int PP = (H + TPR - 1) / TPR;                     // rotation pairs per thread
    static_assert(NT % V == 0 && TPR <= 64 && H <= NT, "summary prologue layout");
    __shared__ double s_cs[2][H];
    const int Hq = a.Hkv * G;
    const int vrow = threadIdx.x / TPR, lr = threadIdx.x % TPR;
    const T *qrow = reinterpret_cast<const T *>(a.q_pre) + ((size_t)rc * Hq + h * G + vrow % G) * D;
    double q1[PP], q2[PP];
#pragma unroll
    for (int j = 0; j < PP; ++j) {
        const int kk = min(lr + TPR * j, H - 1);
        q1[j] = ld<T>(qrow + kk);
        q2[j] = ld<T>(qrow + kk + H);
    }
    const double pos = (double)a.positions[rc];
    const bool ok = (r >= 0) & (r < a.R) & (slot >= 0) & (slot < a.M) & (P >= 2) & (P <= a.max_pages) &
                    (m_r == P * kPage);
    const int C = ok ? (P - 1) * kPage : 0;
    const int nblk = cdiv(C, kStatBlock);
    const bool active = y < nblk;
    const int nit = active ? min(cdiv(nblk - y, ny), min(a.lg_iters, kLogitsMaxIters)) : 0;
    // (everything the second round trip brought is used before the first branch)
#pragma unroll
    for (int j = 0; j < PPL; ++j) {
        const int e = lane + 64 * j, pg = 4 * (y + ny * (e / 4)) + e % 4;
        if (e < 4 * nit) s_pg[e] = pg < P - 1 && pev[j] >= 0 && pev[j] < a.pool_pages ? pev[j] : -1;
    }
    if ((int)threadIdx.x < H) {
        const double ang = pos * pow(a.theta, (-2.0 * (int)threadIdx.x) / D);
        s_cs[0][threadIdx.x] = cos(ang);
        s_cs[1][threadIdx.x] = sin(ang);
    }
    double qq = 0.0;
#pragma unroll
    for (int j = 0; j < PP; ++j) {
        if (lr + TPR * j < H) {
            qq += q1[j] * q1[j];
            qq += q2[j] * q2[j];
        }
    }
    if (writer) a.cand[i] = C;
    if (blockIdx.y * kLogitsWaves >= nblk) return;  // no wave of the workgroup has a block (or no event)

    // keys of half `hf` of block `it`: lane (k, cand) reads units k, 4 + k,
    // ... of token cand of the block's pages 2 hf and 2 hf + 1.  The loads are
    // unconditional (an invalid page reads page 0, and its logits are zeroed
    // after the product), and the last half prefetches itself again, so that
    // every wait for the current keys leaves the next half's loads in flight.
    const T *kbase = reinterpret_cast<const T *>(a.k) + (size_t)h * kPage * D + (size_t)cand * D + k * EPU;
    auto load_keys = [&](int it, int hf, uint4 (&kb)[2][NU]) {
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            const int pe = s_pg[4 * it + 2 * hf + g];
            const uint4 *kp = reinterpret_cast<const uint4 *>(kbase + (size_t)max(pe, 0) * a.Hkv * kPage * D);
#pragma unroll
            for (int u = 0; u < NU; ++u) kb[g][u] = kp[4 * u];
        }
    };
    const double *arow = s_a + k * KS + (lane & 3) * SP;    // A: view 4 vh + (lane & 3), dims dim(k, s)
    auto multiply = [&](const uint4 (&kb)[2][NU], double (&acc)[VH][2]) {
#pragma unroll
        for (int vh = 0; vh < VH; ++vh) acc[vh][0] = acc[vh][1] = 0.0;
#pragma unroll
        for (int s2 = 0; s2 < S; ++s2) {
            double av[VH];
#pragma unroll
            for (int vh = 0; vh < VH; ++vh) av[vh] = arow[4 * vh * SP + s2];
#pragma unroll
            for (int g = 0; g < 2; ++g) {
                const double bv = KRow<T>::elem(kb[g][s2 / EPU], s2 % EPU);
#pragma unroll
                for (int vh = 0; vh < VH; ++vh)
                    acc[vh][g] = __builtin_amdgcn_mfma_f64_4x4x4f64(av[vh], bv, acc[vh][g], 0, 0, 0);
            }
        }
    };
    float *lgv = a.expz + ((size_t)i * a.Hkv + h) * V * a.cmax;
    uint4 k0[2][NU], k1[2][NU];
    // the first keys of an active wave (its page ids are in its own LDS row),
    // then the summaries
    wave_lds_sync();
    if (active) load_keys(0, 0, k0);
    const float *srow = a.qstate + ((size_t)slot * 2 * Hq + (size_t)(vrow / G) * Hq + h * G + vrow % G) * D;
    double s1[PP], s2[PP];
#pragma unroll
    for (int j = 0; j < PP; ++j) {
        const int kk = min(lr + TPR * j, H - 1);
        s1[j] = (double)srow[kk];
        s2[j] = (double)srow[kk + H];
    }
    double ss = 0.0;
#pragma unroll
    for (int j = 0; j < PP; ++j) {
        if (lr + TPR * j < H) {
            ss += s1[j] * s1[j];
            ss += s2[j] * s2[j];
        }
    }
#pragma unroll
    for (int off = TPR / 2; off >= 1; off >>= 1) {
        ss += __shfl_xor(ss, off, TPR);
        qq += __shfl_xor(qq, off, TPR);
    }
    const double gam = ss == 0.0 ? 0.0 : sqrt(qq / D) / sqrt(ss / D);
    // rows V .. VR - 1 of the MFMA operand are zero
    for (int e = threadIdx.x; e < 4 * (VR - V) * S; e += NT) {
        const int q = e / ((VR - V) * S), rem = e % ((VR - V) * S);
        s_a[q * KS + (V + rem / S) * SP + rem % S] = 0.0;
    }
    __syncthreads();
    // head dimension d of view row vr goes to s_a[q][vr][s] with d = 4 E (s / E)
    // + E q + s % E (the lane-group layout of the product below)
    auto put = [&](int d, double val) {
        const int q = (d / EPU) % 4, s2i = (d / (4 * EPU)) * EPU + d % EPU;
        s_a[q * KS + vrow * SP + s2i] = val;
    };
#pragma unroll
    for (int j = 0; j < PP; ++j) {
        const int kk = lr + TPR * j;
        if (kk < H) {
            const double x1 = gam * s1[j], x2 = gam * s2[j];
            const double c = s_cs[0][kk], sn = s_cs[1][kk];
            put(kk, x1 * c - x2 * sn);
            put(kk + H, x2 * c + x1 * sn);
        }
    }
    __syncthreads();
    if (!active) return;
    for (int it = 0; it < nit; ++it) {
        const int blk = y + ny * it;
        double acc[VH][4];
        {
            double a2[VH][2];
            load_keys(it, 1, k1);
            __builtin_amdgcn_sched_barrier(0);      // the next half's loads go out first
            multiply(k0, a2);
#pragma unroll
            for (int vh = 0; vh < VH; ++vh) acc[vh][0] = a2[vh][0], acc[vh][1] = a2[vh][1];
            load_keys(min(it + 1, nit - 1), 0, k0);
            __builtin_amdgcn_sched_barrier(0);
            multiply(k1, a2);
#pragma unroll
            for (int vh = 0; vh < VH; ++vh) acc[vh][2] = a2[vh][0], acc[vh][3] = a2[vh][1];
        }

        // this lane's logits: view 4 vh + k of candidate 16 g + cand of the block
        const int t0 = blk * kStatBlock + cand;
#pragma unroll
        for (int vh = 0; vh < VH; ++vh) {
            const int v = 4 * vh + k;
            double z[4], m = -__builtin_huge_val();
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const bool ok = s_pg[4 * it + g] >= 0;
                z[g] = ok ? acc[vh][g] * a.scale : 0.0;
                if (t0 + 16 * g < C) m = max_f64(m, z[g]);
            }
            m = max_f64(m, dpp_ror_f64<8>(m));
            m = max_f64(m, dpp_ror_f64<4>(m));
            m = max_f64(m, dpp_ror_f64<2>(m));
            m = max_f64(m, dpp_ror_f64<1>(m));
            double sv = 0.0;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int t = t0 + 16 * g;
                if (t < C) {
                    const double ev = exp_nonpos(z[g] - m);
                    sv += ev;
                    if (v < V) lgv[(size_t)v * a.cmax + t] = (float)ev;
                }
            }
            sv += dpp_ror_f64<8>(sv);
            sv += dpp_ror_f64<4>(sv);
            sv += dpp_ror_f64<2>(sv);
            sv += dpp_ror_f64<1>(sv);
            if (cand == 0 && v < V) {
                double *pt = a.part + (((size_t)i * a.Hkv + h) * a.nch + blk) * V * 2;
                pt[v * 2] = m;
                pt[v * 2 + 1] = sv;
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
    __builtin_amdgcn_s_setprio(3);   // issue ahead of co-resident decode waves
    constexpr int V = 2 * G;
    constexpr int BPC = kProbChunk / kStatBlock;     // statistics blocks per chunk
    constexpr int TPT = kProbChunk / 256;            // tokens per thread
    constexpr int NPL = 4;                           // statistics blocks per lane kept in registers
    __shared__ double s_M[V], s_L[V];
    __shared__ double s_f[BPC][V];
    const int h = blockIdx.x, chunk = blockIdx.y, i = blockIdx.z;
    const int t0 = chunk * kProbChunk;
    if (t0 >= a.cmax) return;
    const int tid = threadIdx.x;
    const int b0 = t0 / kStatBlock;
    const double *pt = a.part + (((size_t)i * a.Hkv + h) * a.nch) * V * 2;
    const float *lg = a.expz + ((size_t)i * a.Hkv + h) * V * a.cmax;

    // The kernel runs beside decode attention, where every memory round trip
    // is slow: the event's candidate count (which the logits left in the
    // workspace), the exponentials of this thread's tokens and the first
    // statistics are all requested at once (clamped indices: values beyond
    // the candidates are dropped), in one round trip.
    const int C = a.cand[i];
    float e[TPT][V];
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
        const int t = t0 + k * 256 + tid;
#pragma unroll
        for (int v = 0; v < V; ++v) e[k][v] = lg[(size_t)v * a.cmax + min(t, a.cmax - 1)];
    }
    double mk0[(V + 7) / 8][NPL], sk0[(V + 7) / 8][NPL];
#pragma unroll
    for (int vb = 0; vb < V; vb += 8) {
        const int v = min(vb + tid / 32, V - 1), c0 = tid % 32;
#pragma unroll
        for (int k = 0; k < NPL; ++k) {
            const double *pc = pt + ((size_t)min(c0 + 32 * k, a.nch - 1) * V + v) * 2;
            mk0[vb / 8][k] = pc[0];
            sk0[vb / 8][k] = pc[1];
        }
    }
    if (t0 >= C) return;        // (C = 0: not a boundary)
    const int used = cdiv(C, kStatBlock);
    // merge the block statistics: 32 lanes per view, views 8 at a time; lane
    // c0 holds blocks c0, c0 + 32, ... (the first NPL of them in registers)
#pragma unroll
    for (int vb = 0; vb < V; vb += 8) {
        const int v = vb + tid / 32, c0 = tid % 32;
        if (v < V) {
            double mk[NPL], sk[NPL];
#pragma unroll
            for (int k = 0; k < NPL; ++k) {
                const bool in = c0 + 32 * k < used;       // (blocks past the candidates: stale values)
                mk[k] = in ? mk0[vb / 8][k] : -__builtin_huge_val();
                sk[k] = in ? sk0[vb / 8][k] : 0.0;
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
// Each of the three radix passes (10-bit digits of the weights' float32 bit
// patterns below bit 30) histograms the weights that share the prefix
// found so far (count and 2^-60 fixed-point mass per bucket), then the
// workgroup scans the buckets from the top to find the one where the running
// mass reaches p.  The workgroup is small (one wave per SIMD, 12 KB of LDS)
// so that it starts on any CU with room beside decode attention.
constexpr int kTopPThreads = 256;
__global__ __launch_bounds__(kTopPThreads, 5) void top_p_kernel(ScoreArgs a) {
    __builtin_amdgcn_s_setprio(3);   // issue ahead of co-resident decode waves
    constexpr int NT = kTopPThreads;
    constexpr int NB = 1024;
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
    if (a.cmax == 0) {                     // no request can have candidates
        if (tid == 0) *out = 0;
        return;
    }
    const float *wv = a.weights + (((size_t)i * a.Hkv + h) * 2 + x) * a.cmax;
    const unsigned long long target = (unsigned long long)ldexp(a.p, 60);

    // the first CW * NT weights stay in registers across the passes (every
    // candidate set up to 4096 tokens); longer ones re-read the rest.  They
    // are requested with the event's candidate count (which the logits left
    // in the workspace), at clamped indices, in one round trip.
    const int C = a.cand[i];
    uint32_t cached[CW];
#pragma unroll
    for (int k = 0; k < CW; ++k) cached[k] = __float_as_uint(wv[min(k * NT + tid, a.cmax - 1)]);
    if (C == 0) {                          // not a boundary
        if (tid == 0) *out = 0;
        return;
    }
#pragma unroll
    for (int k = 0; k < CW; ++k) cached[k] = k * NT + tid < C ? cached[k] : 0xffffffffu;
    uint32_t prefix = 0;
    unsigned long long above_mass = 0;
    unsigned int above_cnt = 0;
    // the weights are at most 1, so bits 31 and 30 of their float32 patterns
    // are clear (0x3f800000 and below) and three 10-bit digits cover the rest
    const int shifts[3] = {20, 10, 0};
    const int nbits[3] = {10, 10, 10};
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
hipError_t launch_gd(int G, const ScoreArgs &a, int stages, hipStream_t s) {
    // the KV head is the fastest grid index everywhere: workgroups are handed to
    // the XCDs round-robin, so head h's workgroups all run on one XCD and read
    // back what the previous kernel left in that XCD's L2
    // logits: each wave takes lg_iters statistics blocks, enough that there
    // are about 16384 waves (64 per CU) when the candidate sets are long, one
    // block each when they are short
    ScoreArgs b = a;
    const int nblocks = a.Hkv * a.nch * a.Rb;
    b.lg_iters = std::min(kLogitsMaxIters, std::max(1, cdiv(nblocks, GP_LOGITS_TARGET_WAVES)));
    dim3 g1(a.Hkv, cdiv(cdiv(a.nch, b.lg_iters), kLogitsWaves), a.Rb), g2(a.Hkv, cdiv(a.cmax, kProbChunk), a.Rb), g3(a.Hkv, 2, a.Rb);
    const bool weights = stages & GP_SCORE_WEIGHTS, counts = stages & GP_SCORE_COUNTS;
    if (a.cmax == 0) {
        // no request can have candidates: the counts are written as zero
        if (counts) top_p_kernel<<<g3, kTopPThreads, 0, s>>>(a);
        return hipGetLastError();
    }
    if (weights) {
    switch (G) {
#define GP_CASE(GG)                                                   \
    case GG:                                                          \
        logits_kernel<T, D, GG><<<g1, 64 * kLogitsWaves, 0, s>>>(b);  \
        weights_kernel<GG><<<g2, 256, 0, s>>>(a);                     \
        break;
        GP_CASE(1) GP_CASE(2) GP_CASE(4) GP_CASE(8)
#undef GP_CASE
        default: return hipErrorInvalidValue;
    }
    }
    if (counts) {
        if (a.metric == GP_METRIC_ENTROPY)
            entropy_kernel<<<g3, 256, 0, s>>>(a);
        else
            top_p_kernel<<<g3, kTopPThreads, 0, s>>>(a);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_score(gp_dtype_t dt, int D, int G, const ScoreArgs &a, int stages, hipStream_t s) {
    if (a.Rb == 0) return hipSuccess;
    if (dt == GP_BF16)
        return D == 128 ? launch_gd<uint16_t, 128>(G, a, stages, s) : launch_gd<uint16_t, 64>(G, a, stages, s);
    return D == 128 ? launch_gd<float, 128>(G, a, stages, s) : launch_gd<float, 64>(G, a, stages, s);
}

}  // namespace gp

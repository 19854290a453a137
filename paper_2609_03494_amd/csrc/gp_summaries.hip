// Dual-timescale query summaries (Sec. 3.2, EMA equation; App. E.1).
//
// One thread per four consecutive elements of a request's [Hq][d] query; the
// pool row of the request's slot is updated in place.  Arithmetic is fp64 and
// rounded once to float32 (ema_step), the plain fp64 evaluation of
// beta * qbar + (1 - beta) * q.  The kernel moves
// 2 x 4 B (read + write) x 2 views per element plus the query: it is a few
// microseconds of HBM traffic per step and is bound by launch latency.
#include "gp_internal.h"

namespace gp {

template <typename T>
__device__ inline float load_q(const T *p, size_t i);

template <>
__device__ inline float load_q<float>(const float *p, size_t i) { return p[i]; }

template <>
__device__ inline float load_q<uint16_t>(const uint16_t *p, size_t i) { return bf16_to_f32(p[i]); }

template <typename T>
__global__ __launch_bounds__(256) void summaries_kernel(SummaryArgs a) {
    const int r = blockIdx.y;
    const int i0 = blockIdx.x * blockDim.x + threadIdx.x;
    // the slot, the init flag and the thread's first query element are
    // requested together (the first at a clamped index), so the kernel makes
    // two memory round trips, not four: it heads the boundary chain of a step
    const T *q = reinterpret_cast<const T *>(a.q) + (size_t)r * a.HqD;
    const float x0 = load_q<T>(q, min(i0, a.HqD - 1));
    const int slot = a.slot_ids[r];
    const int init_flag = a.init[r];
    __asm__ volatile("" ::"v"(x0), "v"(slot), "v"(init_flag));   // all three issued before any wait
    const bool init = init_flag != 0;
    if (slot < 0 || slot >= a.M) return;
    float *S = a.qstate + (size_t)slot * 2 * a.HqD;
    float *L = S + a.HqD;
    const double cs = 1.0 - a.beta_s, cl = 1.0 - a.beta_l;
    for (int i = i0; i < a.HqD; i += gridDim.x * blockDim.x) {
        const float x = i == i0 ? x0 : load_q<T>(q, i);
        if (init) {
            S[i] = x;
            L[i] = x;
        } else {
            S[i] = ema_step(S[i], x, a.beta_s, cs);
            L[i] = ema_step(L[i], x, a.beta_l, cl);
        }
    }
}

hipError_t launch_summaries(gp_dtype_t dt, const SummaryArgs &a, hipStream_t s) {
    const int threads = 256;
    dim3 grid(cdiv(a.HqD, threads), a.R);
    if (dt == GP_F32)
        summaries_kernel<float><<<grid, threads, 0, s>>>(a);
    else
        summaries_kernel<uint16_t><<<grid, threads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace gp

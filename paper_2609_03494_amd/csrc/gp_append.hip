// Step prologue of the decode loop: the current token's K and V go into the
// paged cache of every layer and the dual-timescale summaries take their EMA
// step (Sec. 3.1 paged KV cache, Sec. 3.2 EMA equation, App. E.1 query-state
// pool), for every request that is in the step's batch and has room.
//
// One workgroup per request covers all layers, so the resident length is read
// once and advanced once, after every write of the request.  Held requests
// (seq_len < 0) and requests whose pages are full (at a capacity boundary,
// waiting for a decision) take no token and keep their summaries.  The
// summary arithmetic is ema_step, the same as the summaries kernel's, so the
// two agree bit for bit.  Bound: launch latency (a few KiB per request).
#include "gp_internal.h"

namespace gp {

namespace {

template <typename T>
__device__ inline float load_elem(const T *p, size_t i);
template <>
__device__ inline float load_elem<float>(const float *p, size_t i) { return p[i]; }
template <>
__device__ inline float load_elem<uint16_t>(const uint16_t *p, size_t i) { return bf16_to_f32(p[i]); }

template <typename T, int D>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
    const int r = blockIdx.x, tid = threadIdx.x;
    const int P = a.num_pages[r], m = a.seq_lens[r];
    if (m < 0 || P <= 0 || P > a.max_pages || m >= P * kPage) return;
    const int pid = a.page_table[(size_t)r * a.max_pages + m / kPage];
    if (pid < 0 || pid >= a.pool_pages) return;
    const int slot = a.slot_ids[r];
    const bool has_slot = slot >= 0 && slot < a.M;
    const bool init = a.init != nullptr && a.init[r] != 0;
    const int HkvD = a.Hkv * D, HqD = a.Hq * D;
    const double cs = 1.0 - a.beta_s, cl = 1.0 - a.beta_l;
    for (int l = 0; l < a.n_layers; ++l) {
        // K, V: token slot m % 16 of page pid, every KV head
        const T *kn = reinterpret_cast<const T *>(a.k_new) + ((size_t)l * a.R + r) * HkvD;
        const T *vn = reinterpret_cast<const T *>(a.v_new) + ((size_t)l * a.R + r) * HkvD;
        T *kp = reinterpret_cast<T *>(a.k[l]);
        T *vp = reinterpret_cast<T *>(a.v[l]);
        for (int i = tid; i < HkvD; i += blockDim.x) {
            const int h = i / D, dd = i % D;
            const size_t dst = (((size_t)pid * a.Hkv + h) * kPage + m % kPage) * D + dd;
            kp[dst] = kn[i];
            vp[dst] = vn[i];
        }
        // summaries of layer l: [M][2][Hq][D] slice of the [L][M][2][Hq][D] pool
        if (has_slot) {
            const T *q = reinterpret_cast<const T *>(a.q_pre) + ((size_t)l * a.R + r) * HqD;
            float *S = a.qstate + ((size_t)l * a.M + slot) * 2 * HqD;
            float *Lv = S + HqD;
            for (int i = tid; i < HqD; i += blockDim.x) {
                const float x = load_elem<T>(q, i);
                if (init) {
                    S[i] = x;
                    Lv[i] = x;
                } else {
                    S[i] = ema_step(S[i], x, a.beta_s, cs);
                    Lv[i] = ema_step(Lv[i], x, a.beta_l, cl);
                }
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        a.seq_lens[r] = m + 1;
        a.positions[r] += 1;
    }
}

}  // namespace

hipError_t launch_append(gp_dtype_t dt, int D, const AppendArgs &a, hipStream_t s) {
    if (a.R == 0) return hipSuccess;
    if (dt == GP_BF16) {
        if (D == 128) append_kernel<uint16_t, 128><<<a.R, 256, 0, s>>>(a);
        else append_kernel<uint16_t, 64><<<a.R, 256, 0, s>>>(a);
    } else {
        if (D == 128) append_kernel<float, 128><<<a.R, 256, 0, s>>>(a);
        else append_kernel<float, 64><<<a.R, 256, 0, s>>>(a);
    }
    return hipGetLastError();
}

}  // namespace gp

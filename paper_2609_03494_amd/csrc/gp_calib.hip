// Streaming-read reference kernel: reads a buffer once, as fast as the memory
// system allows, so that the bandwidth the GrowPage kernels reach can be set
// against what a plain read of the same size reaches on the same device.
//
// Each workgroup reads 16-byte units with non-temporal loads in a grid-stride
// loop (8 units in flight per thread), XORs them together and adds one word
// to the output; the XOR keeps every load live.
#include "gp_internal.h"

namespace gp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kStreamThreads = 256;
constexpr int kStreamUnroll = 8;

__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(const u32x4 *src, size_t n_units,
                                                                     uint32_t *out) {
    const size_t stride = (size_t)gridDim.x * kStreamThreads;
    size_t u = (size_t)blockIdx.x * kStreamThreads + threadIdx.x;
    uint32_t acc = 0;
    for (; u + (kStreamUnroll - 1) * stride < n_units; u += kStreamUnroll * stride) {
        u32x4 x[kStreamUnroll];
#pragma unroll
        for (int k = 0; k < kStreamUnroll; ++k) x[k] = __builtin_nontemporal_load(src + u + k * stride);
#pragma unroll
        for (int k = 0; k < kStreamUnroll; ++k) acc ^= x[k].x ^ x[k].y ^ x[k].z ^ x[k].w;
    }
    for (; u < n_units; u += stride) {
        const u32x4 x = __builtin_nontemporal_load(src + u);
        acc ^= x.x ^ x.y ^ x.z ^ x.w;
    }
    __shared__ uint32_t s_acc[kStreamThreads / 64];
    for (int off = 32; off >= 1; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
    if ((threadIdx.x & 63) == 0) s_acc[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int w = 0; w < kStreamThreads / 64; ++w) t ^= s_acc[w];
        atomicXor(out, t);
    }
}

}  // namespace

hipError_t launch_stream_read(const void *src, size_t bytes, uint32_t *out, hipStream_t s) {
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const size_t n_units = bytes / 16;
    const int blocks = (int)std::max<size_t>(1, std::min<size_t>((size_t)cus * 16, cdiv(n_units, kStreamThreads)));
    stream_read_kernel<<<blocks, kStreamThreads, 0, s>>>(reinterpret_cast<const u32x4 *>(src), n_units, out);
    return hipGetLastError();
}

}  // namespace gp

// Streaming-read reference kernel: reads a buffer once, as fast as the memory
// system allows, so that the bandwidth the GrowPage kernels reach can be set
// against what a plain read of the same size reaches on the same device.
//
// Each workgroup reads one contiguous chunk of the buffer (a whole number of
// 4 KiB runs) with non-temporal 16-byte loads, 16 in flight per thread, XORs
// the units together and stores one partial word; the XOR keeps every load
// live. A one-workgroup kernel then XORs the partials into the output.
// Contiguous chunks beat a grid-stride loop on MI355X (about 7.0 against
// 6.5-6.7 TB/s in a sweep). The partials go through a device array rather than
// a device-scope atomic on the output word: 2048 workgroups ending together
// serialise on one address, which cost about 80 us per 4 GiB pass (13 %).
#include "gp_internal.h"

namespace gp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kStreamThreads = 256;
constexpr int kStreamUnroll = 16;
constexpr int kStreamBlocksPerCu = 8;

constexpr int kStreamMaxBlocks = 4096;

inline size_t cdiv_size(size_t a, size_t b) { return (a + b - 1) / b; }

// one partial checksum per workgroup of the last pass on this device; only
// device code names it, so no host-side address is needed
__device__ uint32_t g_stream_partials[kStreamMaxBlocks];

__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(const u32x4 *src, size_t n_units,
                                                                     size_t chunk) {
    const size_t b0 = (size_t)blockIdx.x * chunk;
    const size_t b1 = std::min(b0 + chunk, n_units);
    size_t u = b0 + threadIdx.x;
    uint32_t acc = 0;
    for (; u + (kStreamUnroll - 1) * kStreamThreads < b1; u += kStreamUnroll * kStreamThreads) {
        u32x4 x[kStreamUnroll];
#pragma unroll
        for (int k = 0; k < kStreamUnroll; ++k) x[k] = __builtin_nontemporal_load(src + u + k * kStreamThreads);
#pragma unroll
        for (int k = 0; k < kStreamUnroll; ++k) acc ^= x[k].x ^ x[k].y ^ x[k].z ^ x[k].w;
    }
    for (; u < b1; u += kStreamThreads) {
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
        g_stream_partials[blockIdx.x] = t;
    }
}

__global__ __launch_bounds__(kStreamThreads) void stream_fold_kernel(int nblocks, uint32_t *out) {
    uint32_t acc = 0;
    for (int i = threadIdx.x; i < nblocks; i += kStreamThreads) acc ^= g_stream_partials[i];
    __shared__ uint32_t s_acc[kStreamThreads / 64];
    for (int off = 32; off >= 1; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
    if ((threadIdx.x & 63) == 0) s_acc[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = *out;
        for (int w = 0; w < kStreamThreads / 64; ++w) t ^= s_acc[w];
        *out = t;
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
    // chunk: units per workgroup, rounded up to whole 4 KiB runs (256 units)
    const size_t runs = std::max<size_t>(1, cdiv_size(n_units, kStreamThreads));
    const size_t blocks_max = std::min<size_t>(kStreamMaxBlocks, (size_t)std::max(1, cus) * kStreamBlocksPerCu);
    const size_t chunk = cdiv_size(runs, std::min(runs, blocks_max)) * kStreamThreads;
    const int blocks = (int)std::max<size_t>(1, cdiv_size(n_units, chunk));
    stream_read_kernel<<<blocks, kStreamThreads, 0, s>>>(reinterpret_cast<const u32x4 *>(src), n_units, chunk);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    stream_fold_kernel<<<1, kStreamThreads, 0, s>>>(blocks, out);
    return hipGetLastError();
}

}  // namespace gp

// HBM rate probes: the measured ceilings that the streaming kernels are set
// against, beside the vendor figure.
//
// read_probe_kernel   the workgroups walk the buffer together (workgroup b
//                     reads 32 KB blocks b, b + grid, ...) with 16-byte
//                     nontemporal loads (the load form of the vocabulary
//                     pass), eight in flight per thread: of the read forms
//                     measured (contiguous shares or a common walk, 256 to
//                     1024 threads, 2 to 8 loads in flight, 256 to 8192
//                     workgroups) the fastest on large buffers.  It writes
//                     the XOR of the 32-bit words each workgroup read, so the
//                     loads cannot be dropped and the result is checkable.
// copy_probe_kernel   the same share copied with 16-byte loads and stores.
#include "internal.h"

namespace fb {
namespace {

constexpr int kProbeThreads = 512;      // copy probe
constexpr int kReadThreads = 256;       // read probe
constexpr int kReadBatch = 8;           // loads in flight per thread

__global__ void __launch_bounds__(kReadThreads)
read_probe_kernel(const uint4* __restrict__ src, size_t n16, uint32_t* __restrict__ out) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    constexpr size_t kBlock = (size_t)kReadThreads * kReadBatch;   // 16-byte words
    uint32_t x = 0;
    for (size_t b0 = (size_t)blockIdx.x * kBlock; b0 < n16; b0 += (size_t)gridDim.x * kBlock) {
        u32x4 v[kReadBatch];
#pragma unroll
        for (int j = 0; j < kReadBatch; ++j) {
            const size_t k = b0 + (size_t)j * kReadThreads + threadIdx.x;
            v[j] = k < n16 ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + k))
                           : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int j = 0; j < kReadBatch; ++j) x ^= v[j][0] ^ v[j][1] ^ v[j][2] ^ v[j][3];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x ^= __shfl_xor(x, off, 64);
    __shared__ uint32_t s[kReadThreads / 64];
    if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = 0;
        for (int w = 0; w < kReadThreads / 64; ++w) r ^= s[w];
        out[blockIdx.x] = r;
    }
}

__global__ void __launch_bounds__(kProbeThreads)
copy_probe_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, size_t n16) {
    const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const size_t lo = (size_t)blockIdx.x * per;
    const size_t hi = lo + per < n16 ? lo + per : n16;
    constexpr int kBatch = 4;
    for (size_t i = lo + threadIdx.x; i < hi; i += (size_t)kBatch * kProbeThreads) {
        uint4 v[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const size_t k = i + (size_t)j * kProbeThreads;
            if (k < hi) v[j] = src[k];
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const size_t k = i + (size_t)j * kProbeThreads;
            if (k < hi) dst[k] = v[j];
        }
    }
}

}  // namespace

hipError_t launch_read_probe(const void* src, size_t bytes, uint32_t* out,
                             hipStream_t stream) {
    hipLaunchKernelGGL(read_probe_kernel, dim3(FB_PROBE_BLOCKS), dim3(kReadThreads), 0,
                       stream, static_cast<const uint4*>(src), bytes / 16, out);
    return hipGetLastError();
}

hipError_t launch_copy_probe(const void* src, void* dst, size_t bytes, hipStream_t stream) {
    hipLaunchKernelGGL(copy_probe_kernel, dim3(FB_PROBE_BLOCKS), dim3(kProbeThreads), 0,
                       stream, static_cast<const uint4*>(src), static_cast<uint4*>(dst),
                       bytes / 16);
    return hipGetLastError();
}

}  // namespace fb

// Plain streaming read of a device buffer (measurement helper): the reference for the read bandwidth the
// tree-verification kernels reach.  Not part of the method.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dreams.h"
#include "kernels.h"

namespace dreams {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kStreamThreads = 256;
constexpr int kStreamUnroll = 8;   // independent 16-byte loads in flight per thread

__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(const u32x4* __restrict__ p, size_t n16,
                                                                     uint32_t* __restrict__ sink) {
  const size_t stride = (size_t)gridDim.x * kStreamThreads;
  size_t i = (size_t)blockIdx.x * kStreamThreads + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (; i + (kStreamUnroll - 1) * stride < n16; i += kStreamUnroll * stride) {
    u32x4 v[kStreamUnroll];
#pragma unroll
    for (int u = 0; u < kStreamUnroll; ++u) v[u] = p[i + u * stride];
#pragma unroll
    for (int u = 0; u < kStreamUnroll; ++u) acc ^= v[u];
  }
  for (; i < n16; i += stride) acc ^= p[i];
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x ^= __shfl_xor(x, off);
  if ((threadIdx.x & 63) == 0) sink[blockIdx.x * (kStreamThreads / 64) + (threadIdx.x >> 6)] = x;   // one word per wave
}

}  // namespace

hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream) {
  static_assert(DREAMS_STREAM_READ_SINK_WORDS % (kStreamThreads / 64) == 0, "one sink word per wave");
  hipLaunchKernelGGL(stream_read_kernel, dim3(DREAMS_STREAM_READ_SINK_WORDS / (kStreamThreads / 64)),
                     dim3(kStreamThreads), 0, stream,
                     (const u32x4*)src, bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace dreams

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
constexpr int kStreamWaves = kStreamThreads / 64;
constexpr int kStreamUnroll = 8;   // independent 16-byte loads in flight per thread
constexpr int kStreamGroups = DREAMS_STREAM_READ_SINK_WORDS / kStreamWaves;

// Workgroup g reads the g-th of kStreamGroups contiguous chunks of the buffer with non-temporal 16-byte
// loads (the fastest plain read measured on gfx950: 512 workgroups, 8 loads in flight per thread).
__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(const u32x4* __restrict__ p, size_t n16,
                                                                     uint32_t* __restrict__ sink) {
  const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const size_t b0 = (size_t)blockIdx.x * per, b1 = b0 + per < n16 ? b0 + per : n16;
  size_t i = b0 + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (; i + (kStreamUnroll - 1) * kStreamThreads < b1; i += kStreamUnroll * kStreamThreads) {
    u32x4 v[kStreamUnroll];
#pragma unroll
    for (int u = 0; u < kStreamUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * kStreamThreads);
#pragma unroll
    for (int u = 0; u < kStreamUnroll; ++u) acc ^= v[u];
  }
  for (; i < b1; i += kStreamThreads) acc ^= p[i];
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x ^= __shfl_xor(x, off);
  if ((threadIdx.x & 63) == 0) sink[blockIdx.x * kStreamWaves + (threadIdx.x >> 6)] = x;   // one word per wave
}

}  // namespace

hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream) {
  static_assert(DREAMS_STREAM_READ_SINK_WORDS % kStreamWaves == 0, "one sink word per wave");
  hipLaunchKernelGGL(stream_read_kernel, dim3(kStreamGroups), dim3(kStreamThreads), 0, stream,
                     (const u32x4*)src, bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace dreams

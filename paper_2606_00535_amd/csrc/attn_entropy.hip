// Layer-level attention entropy (the paper's Section 3.2, "Adaptive Intermediate Feature Distillation"): the
// average attention entropy AE of a layer is the mean of its rows' entropies (rows of every query head and
// sequence), and the layer chosen for distillation minimises AE(l) + |AE(l) - AE(l-1)|.  Both reductions
// are tiny (one value per row, one per layer) and run in one workgroup each, in a fixed order.
#include "kernels.h"

namespace dreams {
namespace {

constexpr int kMeanThreads = 256;

// Each thread sums a strided subset in fp64, then a fixed-shape tree over the threads.
__global__ __launch_bounds__(kMeanThreads) void attn_entropy_mean_kernel(long long count, const float* e, float* ae) {
  __shared__ double part[kMeanThreads];
  double acc = 0.0;
  for (long long i = threadIdx.x; i < count; i += kMeanThreads) acc += (double)e[i];
  part[threadIdx.x] = acc;
  __syncthreads();
  for (int w = kMeanThreads / 2; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *ae = (float)(part[0] / (double)count);
}

// Candidates are the layers with a predecessor (1 .. num_layers-1); scores in fp32; ties to the smaller layer.
__global__ __launch_bounds__(64) void attn_entropy_select_kernel(int num_layers, const float* ae, int32_t* best) {
  if (threadIdx.x != 0) return;
  int arg = 1;
  float lo = ae[1] + fabsf(ae[1] - ae[0]);
  for (int l = 2; l < num_layers; ++l) {
    const float sc = ae[l] + fabsf(ae[l] - ae[l - 1]);
    if (sc < lo) {
      lo = sc;
      arg = l;
    }
  }
  *best = arg;
}

}  // namespace

hipError_t launch_attn_entropy_mean(long long count, const float* entropy, float* ae, hipStream_t stream) {
  hipLaunchKernelGGL(attn_entropy_mean_kernel, dim3(1), dim3(kMeanThreads), 0, stream, count, entropy, ae);
  return hipGetLastError();
}

hipError_t launch_attn_entropy_select(int num_layers, const float* ae, int32_t* best, hipStream_t stream) {
  hipLaunchKernelGGL(attn_entropy_select_kernel, dim3(1), dim3(64), 0, stream, num_layers, ae, best);
  return hipGetLastError();
}

}  // namespace dreams

// Tree-masked verification attention, fp32 inputs (the small fp32 workload; latency-bound, so plain VALU).
//
// One wave per output row (sequence b, query head h, node i).  Lane t visits keys t, t+64, ... of the
// visible set, keeping its own online softmax (running max, running sum, D-wide accumulator) in fp32; the 64
// per-lane states are then merged pairwise with the log-sum-exp identity (butterfly over lanes), so the
// merge order is fixed and results are reproducible.  With an entropy output, each state also carries
// e = sum 2^(x-m) (x-m) (scores x in log2 units), from which the row's attention entropy follows as
// ln2 * (log2 l - e/l); re-referencing a state to M with weight w = 2^(m-M) turns e into w (e + (m-M) l).
#include "kernels.h"

#include <math.h>

namespace dreams {
namespace {

constexpr float kLn2 = 0.69314718055994530942f;

__device__ __forceinline__ float ent_term(float w, float e, float m, float M, float l) {
  return w == 0.f ? 0.f : w * fmaf(m - M, l, e);
}

template <int D>
__global__ __launch_bounds__(64) void tree_attn_f32_kernel(AttnArgs a) {
  __shared__ float q_lds[D];
  const int lane = threadIdx.x;
  const int T = a.T;
  const int r = blockIdx.x;                       // ((b * Hq) + h) * T + i
  const int i = r % T, bh = r / T;
  const int h = bh % a.Hq, b = bh / a.Hq;
  const int g = h / a.G;
  int L = a.kv_len[b];
  L = L < 0 ? 0 : (L > a.S_cap - T ? a.S_cap - T : L);
  const int N = L + T;

  // ancestors-or-self of node i (every lane walks the same chain)
  uint64_t anc0 = 0, anc1 = 0;
  if (a.mask) {
    const int W = (T + 63) / 64;
    const uint64_t* mr = a.mask + ((size_t)b * T + i) * W;
    anc0 = mr[0];
    anc1 = W > 1 ? mr[1] : 0;
  } else {
    const int32_t* par = a.parent + (size_t)b * T;
    int j = i;
    for (int step = 0; step <= T && j >= 0; ++step) {
      if (j < 64) anc0 |= 1ull << j; else anc1 |= 1ull << (j - 64);
      const int p = par[j];
      if (p >= j) break;
      j = p;
    }
  }

  const float* qrow = (const float*)a.q + (size_t)r * D;
  for (int d = lane; d < D; d += 64) q_lds[d] = qrow[d];
  __syncthreads();

  const float* kb = (const float*)a.k + ((size_t)b * a.Hkv + g) * a.S_cap * D;
  const float* vb = (const float*)a.v + ((size_t)b * a.Hkv + g) * a.S_cap * D;
  const bool ent = a.entropy != nullptr;
  float m = -INFINITY, l = 0.f, e = 0.f;
  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.f;

  for (int s = lane; s < N; s += 64) {
    if (s >= L) {
      const int j = s - L;
      if ((((j < 64) ? anc0 >> j : anc1 >> (j - 64)) & 1ull) == 0) continue;
    }
    const float* kr = kb + (size_t)s * D;
    float dot = 0.f;
#pragma unroll
    for (int d = 0; d < D; ++d) dot = fmaf(q_lds[d], kr[d], dot);
    const float x = dot * a.scale_log2;
    const float m_new = fmaxf(m, x);
    const float alpha = exp2f(m - m_new);
    const float p = exp2f(x - m_new);
    if (ent) e = ent_term(l == 0.f ? 0.f : alpha, e, m, m_new, l) + p * (x - m_new);
    l = l * alpha + p;
    const float* vr = vb + (size_t)s * D;
#pragma unroll
    for (int d = 0; d < D; ++d) acc[d] = fmaf(p, vr[d], acc[d] * alpha);
    m = m_new;
  }

  for (int off = 32; off >= 1; off >>= 1) {
    const float mo = __shfl_xor(m, off);
    const float lo = __shfl_xor(l, off);
    const float eo = __shfl_xor(e, off);
    const float M = fmaxf(m, mo);
    const float w = M == -INFINITY ? 0.f : exp2f(m - M);
    const float wo = M == -INFINITY ? 0.f : exp2f(mo - M);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const float ao = __shfl_xor(acc[d], off);
      acc[d] = acc[d] * w + ao * wo;
    }
    if (ent) e = ent_term(w, e, m, M, l) + ent_term(wo, eo, mo, M, lo);
    l = l * w + lo * wo;
    m = M;
  }

  const float inv = l > 0.f ? 1.0f / l : 0.f;
  float* orow = (float*)a.out + (size_t)r * D;
#pragma unroll
  for (int d = 0; d < D; ++d)
    if ((d & 63) == lane) orow[d] = acc[d] * inv;
  if (a.lse && lane == 0) a.lse[r] = l > 0.f ? (m + log2f(l)) * kLn2 : -INFINITY;
  if (ent && lane == 0) a.entropy[r] = l > 0.f ? kLn2 * (log2f(l) - e / l) : 0.f;
}

}  // namespace

hipError_t launch_tree_attn_f32(const AttnArgs& a, hipStream_t stream) {
  const int rows = a.B * a.Hq * a.T;
  if (a.D == 64) {
    hipLaunchKernelGGL(tree_attn_f32_kernel<64>, dim3(rows), dim3(64), 0, stream, a);
  } else if (a.D == 128) {
    hipLaunchKernelGGL(tree_attn_f32_kernel<128>, dim3(rows), dim3(64), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dreams

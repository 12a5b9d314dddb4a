// Greedy tree acceptance (the paper's Section 2, "Speculative decoding": drafts are kept while they equal the
// target's own token at their position; at the first mismatch the target's token replaces the draft).
//
// One kernel, two phases:
//   1. Row argmax of the target logits.  Each (sequence, node) row of V logits is cut into `chunks` pieces,
//      one 256-thread workgroup per piece, streamed with 16-byte loads (the logits are the only large input:
//      B*T*V*4 bytes).  Ties go to the smallest index: every thread visits its elements in increasing order
//      and replaces its candidate only on a strictly larger value, and every merge prefers the smaller index
//      on equal values (fp32 comparison, so -0.0 and +0.0 are equal).
//   2. Path scan, by the last workgroup of the sequence to finish (arrival counter; pieces travel through
//      device-scope stores and loads): per node, merge the
//      pieces in index order, then every node walks its own ancestor chain (at most depth steps, no
//      barriers) to decide whether each draft on it equals the target token at its parent.  The deepest
//      consistent node (smallest index among equals) is found with one block-wide max over the key
//      depth*256 + (255 - node).
#include "kernels.h"

#include <limits.h>
#include <math.h>

namespace dreams {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct Cand {
  float v;
  int i;
};

// true iff (v2, i2) beats (v1, i1): larger value, or equal value and smaller index
__device__ __forceinline__ bool better(float v2, int i2, float v1, int i1) {
  return v2 > v1 || (v2 == v1 && i2 < i1);
}

__device__ __forceinline__ Cand wave_best(Cand c) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float v2 = __shfl_xor(c.v, off);
    const int i2 = __shfl_xor(c.i, off);
    if (better(v2, i2, c.v, c.i)) { c.v = v2; c.i = i2; }
  }
  return c;
}

__device__ __forceinline__ int wave_max(int x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = max(x, __shfl_xor(x, off));
  return x;
}

template <bool VEC>
__global__ __launch_bounds__(kAcceptThreads) void tree_accept_kernel(AcceptArgs a) {
  constexpr int NT = kAcceptThreads, NW = NT / 64;
  __shared__ float red_v[NW];
  __shared__ int red_i[NW];
  __shared__ int last_flag;
  __shared__ int am_s[kMaxNodes], tok_s[kMaxNodes], par_s[kMaxNodes];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = blockIdx.x;                 // ((b * T) + i) * chunks + c
  const int bi = n / a.chunks, c = n - bi * a.chunks;
  const int b = bi / a.T;
  const float* row = a.logits + (size_t)bi * a.V;
  const int x0 = c * a.chunk, x1 = min(a.V, x0 + a.chunk);

  // ---- phase 1: best (value, index) of this piece
  Cand best{-INFINITY, INT_MAX};
  if (VEC) {
    constexpr int STEP = NT * 4;
    int x = x0 + tid * 4;
    for (; x + 3 * STEP < x1; x += 4 * STEP) {  // four independent 16-byte loads in flight
      f32x4 r[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) r[u] = *(const f32x4*)(row + x + u * STEP);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (r[u][e] > best.v || best.i == INT_MAX) { best.v = r[u][e]; best.i = x + u * STEP + e; }
    }
    for (; x < x1; x += STEP) {
      const f32x4 r = *(const f32x4*)(row + x);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (r[e] > best.v || best.i == INT_MAX) { best.v = r[e]; best.i = x + e; }
    }
  } else {
    for (int x = x0 + tid; x < x1; x += NT) {
      const float r = row[x];
      if (r > best.v || best.i == INT_MAX) { best.v = r; best.i = x; }
    }
  }
  best = wave_best(best);
  if (lane == 0) { red_v[wave] = best.v; red_i[wave] = best.i; }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < NW; ++w)
      if (better(red_v[w], red_i[w], best.v, best.i)) { best.v = red_v[w]; best.i = red_i[w]; }
    store_coherent(a.part_val + n, best.v);
    store_coherent(a.part_idx + n, best.i);
    wait_vector_memory();
    last_flag = arrive_last(&a.counters[b], (uint32_t)(a.T * a.chunks));
  }
  __syncthreads();
  if (!last_flag) return;

  // ---- phase 2: the sequence's path scan.  One parallel round trip stages all of the sequence's pieces.
  const int T = a.T;
  __shared__ float pv_s[kAcceptMaxParts];
  __shared__ int pi_s[kAcceptMaxParts];
  const int parts = T * a.chunks;
  const size_t p0 = (size_t)b * parts;
  for (int e = tid; e < parts; e += NT) {
    pv_s[e] = load_coherent(a.part_val + p0 + e);
    pi_s[e] = load_coherent(a.part_idx + p0 + e);
  }
  if (tid < T) {
    tok_s[tid] = a.tokens[(size_t)b * T + tid];
    par_s[tid] = a.parent[(size_t)b * T + tid];
  }
  __syncthreads();
  if (tid < T) {
    const int q0 = tid * a.chunks;
    float bv = pv_s[q0];
    int bx = pi_s[q0];
    for (int cc = 1; cc < a.chunks; ++cc)
      if (better(pv_s[q0 + cc], pi_s[q0 + cc], bv, bx)) { bv = pv_s[q0 + cc]; bx = pi_s[q0 + cc]; }
    am_s[tid] = bx;
  }
  __syncthreads();

  int key = -1;
  if (tid < T) {
    int j = tid, depth = 0;
    bool ok = true;
    while (j != 0) {
      const int p = par_s[j];
      if (p < 0 || p >= j || tok_s[j] != am_s[p]) { ok = false; break; }
      j = p;
      ++depth;
    }
    if (ok) key = depth * 256 + (255 - tid);
  }
  key = wave_max(key);
  __shared__ int red_k[NW];
  if (lane == 0) red_k[wave] = key;
  __syncthreads();
  key = red_k[0];
  for (int w = 1; w < NW; ++w) key = max(key, red_k[w]);

  const int last = 255 - (key & 255), alen = key >> 8;   // the root is always consistent: key >= 255
  int32_t* path = a.accept_path + (size_t)b * T;
  if (tid == 0) {
    a.accept_len[b] = alen;
    a.next_token[b] = am_s[last];
    int j = last;
    for (int k = alen; k >= 0; --k) { path[k] = j; j = par_s[j]; }
    reset_counter(&a.counters[b]);  // ready for the next call
  }
  if (tid > alen && tid < T) path[tid] = -1;
  if (a.target_argmax && tid < T) a.target_argmax[(size_t)b * T + tid] = am_s[tid];
}

}  // namespace

hipError_t launch_tree_accept(const AcceptArgs& a, hipStream_t stream) {
  const int grid = a.B * a.T * a.chunks;
  if (a.vec4)
    hipLaunchKernelGGL(tree_accept_kernel<true>, dim3(grid), dim3(kAcceptThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(tree_accept_kernel<false>, dim3(grid), dim3(kAcceptThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dreams

// Greedy tree acceptance (the paper's Section 2, "Speculative decoding": drafts are kept while they equal the
// target's own token at their position; at the first mismatch the target's token replaces the draft).
//
// One kernel, three levels, each finished by the last workgroup to arrive at an arrival counter (pieces
// travel through device-scope stores and loads, see kernels.h):
//   1. Row argmax of the target logits.  Each (sequence, node) row of V logits is cut into `chunks` pieces,
//      one 256-thread workgroup per piece, every thread issuing its piece's 16-byte loads UNROLL at a time
//      (8, 16 or 32, from the piece size; the logits are the only large input: B*T*V*4 bytes).  Ties go to the smallest index: every thread visits its
//      elements in increasing order and replaces its candidate only on a strictly larger value, and every
//      merge prefers the smaller index on equal values (fp32 comparison, so -0.0 and +0.0 are equal).
//   2. The last piece of a row to finish merges the row's pieces (one counter per row, so at most `chunks`
//      workgroups ever touch the same counter) and publishes the row's argmax.
//   3. The last row of a sequence to finish runs the path scan: every node walks its own ancestor chain (at
//      most depth steps, no barriers) to decide whether each draft on it equals the target token at its
//      parent; the deepest consistent node (smallest index among equals) comes out of one block-wide max
//      over the key depth*256 + (255 - node).
#include "kernels.h"

#include <limits.h>
#include <math.h>

namespace dreams {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// true iff (v2, i2) beats (v1, i1): larger value, or equal value and smaller index
__device__ __forceinline__ bool better(float v2, int i2, float v1, int i1) {
  return v2 > v1 || (v2 == v1 && i2 < i1);
}

// Block-wide best (value, index); the result is valid in every thread.
__device__ __forceinline__ void block_best(float& v, int& i, float* red_v, int* red_i) {
  constexpr int NW = kAcceptThreads / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float v2 = __shfl_xor(v, off);
    const int i2 = __shfl_xor(i, off);
    if (better(v2, i2, v, i)) { v = v2; i = i2; }
  }
  __syncthreads();   // earlier readers of red_v / red_i are done
  if (lane == 0) { red_v[wave] = v; red_i[wave] = i; }
  __syncthreads();
  v = red_v[0];
  i = red_i[0];
#pragma unroll
  for (int w = 1; w < NW; ++w)
    if (better(red_v[w], red_i[w], v, i)) { v = red_v[w]; i = red_i[w]; }
}

__device__ __forceinline__ int wave_max(int x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = max(x, __shfl_xor(x, off));
  return x;
}

template <bool VEC, int UNROLL>
__global__ __launch_bounds__(kAcceptThreads) void tree_accept_kernel(AcceptArgs a) {
  constexpr int NT = kAcceptThreads, NW = NT / 64;
  __shared__ float red_v[NW];
  __shared__ int red_i[NW];
  __shared__ int flag;
  __shared__ int am_s[kMaxNodes], tok_s[kMaxNodes], par_s[kMaxNodes];
  __shared__ int red_k[NW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = blockIdx.x;                 // ((b * T) + i) * chunks + c
  const int bi = n / a.chunks, c = n - bi * a.chunks;
  const int b = bi / a.T;
  const float* row = a.logits + (size_t)bi * a.V;
  const int x0 = c * a.chunk, x1 = min(a.V, x0 + a.chunk);

  // ---- level 1: best (value, index) of this piece
  float bv = -INFINITY;
  int bx = INT_MAX;
  if (VEC) {
    constexpr int STEP = NT * 4;
    for (int xb = x0 + tid * 4; xb < x1; xb += UNROLL * STEP) {
      f32x4 r[UNROLL];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {   // unconditional loads (clamped) so that all are in flight together
        const int x = min(xb + u * STEP, x1 - 4);
        r[u] = *(const f32x4*)(row + x);
      }
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {
        const int x = xb + u * STEP;
        if (x < x1) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (r[u][e] > bv || bx == INT_MAX) { bv = r[u][e]; bx = x + e; }
        }
      }
    }
  } else {
    for (int xb = x0 + tid; xb < x1; xb += UNROLL * NT) {
      float r[UNROLL];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) r[u] = row[min(xb + u * NT, x1 - 1)];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {
        const int x = xb + u * NT;
        if (x < x1 && (r[u] > bv || bx == INT_MAX)) { bv = r[u]; bx = x; }
      }
    }
  }
  block_best(bv, bx, red_v, red_i);

  // ---- level 2: the row's pieces (skipped when a row is one piece)
  uint32_t* seq_counter = a.counters + b;
  if (a.chunks > 1) {
    uint32_t* row_counter = a.counters + a.B + bi;
    if (tid == 0) {
      store_coherent(a.part_val + n, bv);
      store_coherent(a.part_idx + n, bx);
      wait_vector_memory();
      flag = arrive_last(row_counter, (uint32_t)a.chunks);
    }
    __syncthreads();
    if (!flag) return;
    float v = -INFINITY;
    int x = INT_MAX;
    if (tid < a.chunks) {
      v = load_coherent(a.part_val + (size_t)bi * a.chunks + tid);
      x = load_coherent(a.part_idx + (size_t)bi * a.chunks + tid);
    }
    block_best(v, x, red_v, red_i);
    bx = x;
    if (tid == 0) reset_counter(row_counter);
  }
  if (tid == 0) {
    store_coherent(a.row_am + bi, bx);
    wait_vector_memory();
    flag = arrive_last(seq_counter, (uint32_t)a.T);
  }
  __syncthreads();
  if (!flag) return;

  // ---- level 3: the sequence's path scan
  const int T = a.T;
  if (tid < T) {
    am_s[tid] = load_coherent(a.row_am + (size_t)b * T + tid);
    tok_s[tid] = a.tokens[(size_t)b * T + tid];
    par_s[tid] = a.parent[(size_t)b * T + tid];
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
  if (lane == 0) red_k[wave] = key;
  __syncthreads();
  key = red_k[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) key = max(key, red_k[w]);

  const int last = 255 - (key & 255), alen = key >> 8;   // the root is always consistent: key >= 255
  int32_t* path = a.accept_path + (size_t)b * T;
  if (tid == 0) {
    a.accept_len[b] = alen;
    a.next_token[b] = am_s[last];
    int j = last;
    for (int k = alen; k >= 0; --k) { path[k] = j; j = par_s[j]; }
    reset_counter(seq_counter);  // ready for the next call
  }
  if (tid > alen && tid < T) path[tid] = -1;
  if (a.target_argmax && tid < T) a.target_argmax[(size_t)b * T + tid] = am_s[tid];
}

}  // namespace

hipError_t launch_tree_accept(const AcceptArgs& a, hipStream_t stream) {
  const int grid = a.B * a.T * a.chunks;
  // the piece's loads in one batch per thread where they fit 8, 16 or 32 per thread
  const int per_batch = kAcceptThreads * (a.vec4 ? 4 : 1);
  const int u = a.chunk <= 8 * per_batch ? 8 : a.chunk <= 16 * per_batch ? 16 : 32;
  auto go = [&](auto kern) { hipLaunchKernelGGL(kern, dim3(grid), dim3(kAcceptThreads), 0, stream, a); };
  if (a.vec4) {
    if (u == 8) go(tree_accept_kernel<true, 8>);
    else if (u == 16) go(tree_accept_kernel<true, 16>);
    else go(tree_accept_kernel<true, 32>);
  } else {
    if (u == 8) go(tree_accept_kernel<false, 8>);
    else if (u == 16) go(tree_accept_kernel<false, 16>);
    else go(tree_accept_kernel<false, 32>);
  }
  return hipGetLastError();
}

}  // namespace dreams

// Greedy tree acceptance (the paper's Section 2, "Speculative decoding": drafts are kept while they equal the
// target's own token at their position; at the first mismatch the target's token replaces the draft).
//
// One kernel.  Each (sequence, node) row of V logits is cut into `chunks` pieces, one 256-thread workgroup per
// piece, every thread issuing its piece's 16-byte loads UNROLL at a time (8, 16 or 32, from the piece size;
// the logits are the only large input: B*T*V*4 bytes).  A workgroup publishes its piece's best (value, index)
// and arrives at its sequence's counters; the last workgroup of the sequence to arrive merges all of the
// sequence's pieces and runs the path scan:
//   * piece best: ties go to the smallest index -- every thread visits its elements in increasing order and
//     replaces its candidate only on a strictly larger value, and every merge prefers the smaller index on
//     equal values (fp32 comparison, so -0.0 and +0.0 are equal);
//   * arrival: a sequence's workgroups are dealt round-robin to up to 8 group counters (each on a cache line
//     of its own where the counter region allows), and the last arrival of each group arrives at the
//     sequence counter, so that no counter takes more than a few dozen atomics (atomics on one line
//     serialise);
//   * path scan: one wave sweeps the tree from the root, one depth per round, growing the set of consistent
//     nodes (every draft on the way equal to the target's token at its parent) by ballots; the last round's
//     smallest new member is the deepest consistent node (smallest index among equals).
// The pieces travel through device-scope stores and loads (see kernels.h); the tree (tokens, parents) is
// fetched by every workgroup at entry, ahead of its logits, for whichever one ends up finishing the sequence.
#include "accept_scan.h"
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

template <bool VEC, int UNROLL>
__global__ __launch_bounds__(kAcceptThreads) void tree_accept_kernel(AcceptArgs a) {
  constexpr int NT = kAcceptThreads, NW = NT / 64;
  __shared__ float red_v[NW];
  __shared__ int red_i[NW];
  __shared__ int flag;
  __shared__ int am_s[kMaxNodes], tok_s[kMaxNodes], par_s[kMaxNodes];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T;
  const int n = blockIdx.x;                 // ((b * T) + i) * chunks + c
  const int per_seq = T * a.chunks;         // workgroups of one sequence
  const int b = n / per_seq, local = n - b * per_seq;
  const int bi = n / a.chunks, c = n - bi * a.chunks;
  int tok_r = 0, par_r = 0;
  if (tid < T) {
    tok_r = a.tokens[(size_t)b * T + tid];
    par_r = a.parent[(size_t)b * T + tid];
  }
  const float* row = a.logits + (size_t)bi * a.V;
  const int x0 = c * a.chunk, x1 = min(a.V, x0 + a.chunk);

  // ---- best (value, index) of this piece
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

  // ---- publish it and arrive: group counter, then (last of the group) the sequence counter
  if (tid == 0) {
    store_coherent(a.part_val + n, bv);
    store_coherent(a.part_idx + n, bx);
    wait_vector_memory();
    const int NG = a.groups;
    const int g = local % NG;
    uint32_t* gc = a.counters + a.group_base + ((size_t)b * NG + g) * a.group_stride;
    bool last = arrive_last(gc, (uint32_t)((per_seq - g + NG - 1) / NG));
    if (last) {
      reset_counter(gc);   // every workgroup of the group has arrived: ready for the next call
      last = arrive_last(a.counters + b, (uint32_t)NG);
    }
    flag = last;
  }
  __syncthreads();
  if (!flag) return;

  // ---- the sequence's last workgroup: every row's argmax from its pieces (all loads of a batch of 8 pieces
  // in flight together, merged in piece order), then the path scan
  if (tid < T) {
    float v = -INFINITY;
    int x = INT_MAX;
    const size_t p0 = ((size_t)b * T + tid) * a.chunks;
    for (int c0 = 0; c0 < a.chunks; c0 += 8) {
      float pv[8];
      int px[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const size_t pp = p0 + min(c0 + k, a.chunks - 1);
        pv[k] = load_coherent(a.part_val + pp);
        px[k] = load_coherent(a.part_idx + pp);
      }
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (c0 + k < a.chunks && better(pv[k], px[k], v, x)) { v = pv[k]; x = px[k]; }
    }
    am_s[tid] = x;
    tok_s[tid] = tok_r;
    par_s[tid] = par_r;
  }
  if (tid == 0) reset_counter(a.counters + b);   // ready for the next call
  __syncthreads();
  if (a.target_argmax && tid < T) a.target_argmax[(size_t)b * T + tid] = am_s[tid];
  if (wave != 0) return;

  path_scan_wave(am_s, tok_s, par_s, T, a.accept_len + b, a.accept_path + (size_t)b * T, a.next_token + b);
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

// Sampled tree acceptance at temperature tau: speculative sampling's accept-or-resample rule (the paper's
// Section 1 and Section 2, "Speculative decoding"; its Table 2 runs at temperature 1) applied down the tree.
//
// The rule.  p and q are the target's and the draft's softmax(logits / tau) at a node.  Its children are tested
// in index order: child c, carrying token x, is kept with probability min(1, r(x) / q(x)), and the walk descends
// into the first kept child; after a rejection r becomes max(r - q, 0) renormalised (unchanged if that is zero).
// r starts as p.  Where no child is kept (or at a leaf) the emitted token is drawn from r.  Child c is decided
// by the caller's uniform u[c]; the emitted token by u[0], through the inverse CDF of r.
//
// The residual after k rejections at a node has the closed form r_k = max(p - C_k q, 0) / D_k, with C_0 = 0,
// D_0 = 1, and after rejecting one more child C_{k+1} = C_k + D_k, D_{k+1} = sum_x max(p - C_{k+1} q, 0) (both
// unchanged when that sum is zero).  It does not depend on which tokens were rejected, only on how many, so
// every child's test can be prepared before the walk: the state before child c is the state after its previous
// sibling.  That turns the sequential walk into
//   (1) per row and per piece of the vocabulary: maximum and sum of exp((l - max) / tau), target and draft,
//       merged per row by the row's last piece ("stats" pieces);
//   (2) per child c and per piece: the residual mass sum max(p - (C + D) q, 0) over the piece, where (C, D) is
//       the state after c's previous sibling; the row's last piece sums the pieces and publishes the state
//       after c ("pass" pieces).  Pass pieces wait for the stats of c's parent and for the previous sibling's
//       state, a chain of waits as long as the widest sibling group;
//   (3) the last workgroup of the sequence to finish a row: every child's test in parallel (one thread per
//       node: u q(x) D < max(p(x) - C q(x), 0)), the walk by ballots (the first kept child of each node), and
//       the emitted token from the final state's piece masses (prefix in piece order, then a block scan inside
//       the chosen piece).
// Every probability is fp64, so that the integer outcome is decided in the precision of the definition.
//
// Forward progress.  Workgroups do their work in the order of a ticket taken on entry, not in blockIdx order:
// stats pieces first, then pass pieces by child index.  A workgroup only ever waits for results of workgroups
// with smaller tickets, which are already running or finished, so every wait ends; waits are nevertheless
// bounded (0.2 s), after which the results are unspecified.
//
// Results cross workgroups through device-scope stores and loads, published before a relaxed device-scope
// increment of an arrival word (see kernels.h).  Every arrival word is back at zero when the launch ends: the
// walker of each sequence clears that sequence's words, the workgroup with the last ticket the ticket.
#include "kernels.h"

#include <limits.h>
#include <math.h>

namespace dreams {
namespace {

constexpr int NT = kSampledThreads, NW = NT / 64, EPT = kSampledPerThread, CHUNK = kSampledChunk;
constexpr uint64_t kWaitTicks = 20000000;   // 100 MHz real-time ticks: 0.2 s
constexpr uint32_t kStatsOne = 1u, kPassOne = 1u << 16;

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void store_d(double* p, double v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double load_d(const double* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t add_word(uint32_t* w, uint32_t v) {
  return __hip_atomic_fetch_add(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// exp(d / tau) as exp(d * (1 / tau)); d = 0 (the row maximum itself) gives exactly 1, also where 1 / tau is
// infinite
__device__ __forceinline__ double scaled_exp(double d, double inv_tau) { return d == 0.0 ? 1.0 : exp(d * inv_tau); }

struct Shared {
  double pm[kSampledMaxChunks];
  double red_d[NW];
  float red_f[NW];
  int red_i[NW];
  double scan[NW];
  int flag;
  int par[kMaxNodes];
  int acc[kMaxNodes];
  int path[kMaxNodes];
  int fin_node, fin_depth, fin_slot, fin_piece;
  double fin_c, fin_before, fin_thr;
};

// Block reductions: every lane reduces its wave by a butterfly, lane 0's value is kept, waves are combined in
// wave order -- the same order on every call.
__device__ __forceinline__ double block_sum(double v, Shared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  __syncthreads();
  if (lane == 0) sh.red_d[wave] = v;
  __syncthreads();
  double s = sh.red_d[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) s += sh.red_d[w];
  return s;
}
__device__ __forceinline__ float block_max(float v, Shared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  __syncthreads();
  if (lane == 0) sh.red_f[wave] = v;
  __syncthreads();
  float m = sh.red_f[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) m = fmaxf(m, sh.red_f[w]);
  return m;
}
template <bool MAX>
__device__ __forceinline__ int block_int(int v, Shared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const int o = __shfl_xor(v, off);
    v = MAX ? max(v, o) : min(v, o);
  }
  __syncthreads();
  if (lane == 0) sh.red_i[wave] = v;
  __syncthreads();
  int r = sh.red_i[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) r = MAX ? max(r, sh.red_i[w]) : min(r, sh.red_i[w]);
  return r;
}
// Exclusive prefix of v over the threads in thread order.
__device__ __forceinline__ double block_exclusive_scan(double v, Shared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  double inc = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double o = __shfl_up(inc, off);
    if (lane >= off) inc += o;
  }
  __syncthreads();
  if (lane == 63) sh.scan[wave] = inc;
  __syncthreads();
  double base = 0.0;
  for (int w = 0; w < wave; ++w) base += sh.scan[w];
  return base + inc - v;
}

// Thread t holds entries x0 + t * EPT + e (e < EPT) of the piece [x0, x1); entries past x1 read as -inf.
template <bool VEC>
__device__ __forceinline__ void load_piece(const float* row, int x0, int x1, float (&v)[EPT]) {
  const int base = x0 + (int)threadIdx.x * EPT;
  if (VEC) {
#pragma unroll
    for (int k = 0; k < EPT / 4; ++k) {
      const int x = base + 4 * k;   // x0, x1 and x are multiples of 4: a vector is wholly in or out
      f32x4 r = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      if (x < x1) r = *(const f32x4*)(row + x);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[4 * k + e] = r[e];
    }
  } else {
#pragma unroll
    for (int e = 0; e < EPT; ++e) v[e] = base + e < x1 ? row[base + e] : -INFINITY;
  }
}

// Wait (one thread) until a half of an arrival word reads `target`.
__device__ __forceinline__ void wait_half(const uint32_t* w, int shift, uint32_t target) {
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  while (((__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >> shift) & 0xffffu) != target) {
    if (__builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) break;
    __builtin_amdgcn_s_sleep(2);
  }
}

__device__ __forceinline__ uint32_t* row_word(const SampledArgs& a, int b, int i) {
  return a.row_ctr + ((size_t)b * a.T + i) * a.row_stride;
}

// ---------------------------------------------------------------------------------------------------- walk
template <bool VEC>
__device__ void walk(const SampledArgs& a, int b, Shared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T, V = a.V;
  const size_t rb = (size_t)b * T;
  if (tid < T) sh.par[tid] = a.parent[rb + tid];
  __syncthreads();

  // every child's test, in parallel: the state before c is the state after c's previous sibling
  int kept = 0;
  if (tid >= 1 && tid < T) {
    const int n = sh.par[tid];
    const int x = a.tokens[rb + tid];
    if (n >= 0 && n < tid && x >= 0 && x < V) {
      int prev = -1;
      for (int k = tid - 1; k > n; --k)
        if (sh.par[k] == n) { prev = k; break; }
      double C = 0.0, D = 1.0;
      if (prev >= 0) {
        C = load_d(a.post + (rb + prev) * 4 + 0);
        D = load_d(a.post + (rb + prev) * 4 + 1);
      }
      const double* rs = a.row_stat + (rb + n) * 4;
      const double Mt = load_d(rs + 0), St = load_d(rs + 1), Md = load_d(rs + 2), Sd = load_d(rs + 3);
      const double lt = a.target_logits[(rb + n) * V + x], ld = a.draft_logits[(rb + n) * V + x];
      const double p = scaled_exp(lt - Mt, a.inv_tau) / St;
      const double q = scaled_exp(ld - Md, a.inv_tau) / Sd;
      const double u = a.uniforms[rb + tid];
      kept = (u * q) * D < fmax(p - C * q, 0.0);
    }
  }
  if (tid < T) sh.acc[tid] = kept;
  __syncthreads();

  // the walk (wave 0; lane l holds nodes l and l + 64): the first kept child of each node, then the state
  // after the last node's last child
  if (wave == 0) {
    int par_h[2], acc_h[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int i = lane + 64 * h;
      par_h[h] = i < T ? sh.par[i] : -1;
      acc_h[h] = i < T ? sh.acc[i] : 0;
    }
    int node = 0, depth = 0;
    if (lane == 0) sh.path[0] = 0;
    while (true) {
      const uint64_t k0 = __ballot(acc_h[0] && par_h[0] == node && lane > node);
      const uint64_t k1 = __ballot(acc_h[1] && par_h[1] == node && lane + 64 > node);
      if ((k0 | k1) == 0) break;
      node = k0 ? __builtin_ctzll(k0) : 64 + __builtin_ctzll(k1);
      ++depth;
      if (lane == 0) sh.path[depth] = node;
    }
    const uint64_t c0 = __ballot(par_h[0] == node && lane > node);
    const uint64_t c1 = __ballot(par_h[1] == node && lane + 64 > node);
    if (lane == 0) {
      double C = 0.0;
      int slot = node;
      if (c0 | c1) {
        const int lc = c1 ? 127 - __builtin_clzll(c1) : 63 - __builtin_clzll(c0);
        C = load_d(a.post + (rb + lc) * 4 + 0);
        slot = (int)load_d(a.post + (rb + lc) * 4 + 2);
      }
      sh.fin_node = node;
      sh.fin_depth = depth;
      sh.fin_c = C;
      sh.fin_slot = slot;
    }
  }
  __syncthreads();
  // the piece in which the cumulative mass (piece order) first exceeds u0 * total
  {
    const double* m = a.mass + ((size_t)b * 2 * T + sh.fin_slot) * a.chunks;
    for (int k = tid; k < a.chunks; k += NT) sh.pm[k] = load_d(m + k);
    __syncthreads();
    if (tid == 0) {
      double total = 0.0;
      for (int k = 0; k < a.chunks; ++k) total += sh.pm[k];
      const double thr = (double)a.uniforms[rb] * total;
      double cum = 0.0, before = 0.0, pos_before = 0.0;
      int piece = -1, pos_piece = 0;
      for (int k = 0; k < a.chunks; ++k) {
        const double mk = sh.pm[k];
        if (mk > 0.0) {
          pos_piece = k;
          pos_before = cum;
        }
        if (cum + mk > thr) {
          piece = k;
          before = cum;
          break;
        }
        cum += mk;
      }
      if (piece < 0) {   // no crossing (an all-zero residual): the last piece of positive mass
        piece = pos_piece;
        before = pos_before;
      }
      sh.fin_piece = piece;
      sh.fin_before = before;
      sh.fin_thr = thr;
    }
  }
  __syncthreads();
  const int node = sh.fin_node, depth = sh.fin_depth, piece = sh.fin_piece;
  const double C = sh.fin_c, before = sh.fin_before, thr = sh.fin_thr;

  // the emitted token: prefix of max(p - C q, 0) inside the chosen piece
  const size_t row = rb + node;
  const double* rs = a.row_stat + row * 4;
  const double Mt = load_d(rs + 0), St = load_d(rs + 1), Md = load_d(rs + 2), Sd = load_d(rs + 3);
  const int x0 = piece * CHUNK, x1 = min(V, x0 + CHUNK);
  float lt[EPT], ld[EPT];
  load_piece<VEC>(a.target_logits + row * V, x0, x1, lt);
  load_piece<VEC>(a.draft_logits + row * V, x0, x1, ld);
  const int base = x0 + tid * EPT;
  double r[EPT], mine = 0.0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    r[e] = 0.0;
    if (base + e < x1) {
      const double p = scaled_exp((double)lt[e] - Mt, a.inv_tau) / St;
      const double q = C == 0.0 ? 0.0 : scaled_exp((double)ld[e] - Md, a.inv_tau) / Sd;
      r[e] = fmax(p - C * q, 0.0);
    }
    mine += r[e];
  }
  double cum = before + block_exclusive_scan(mine, sh);
  int pick = INT_MAX, last_pos = -1;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    cum += r[e];
    if (pick == INT_MAX && cum > thr) pick = base + e;
    if (r[e] > 0.0) last_pos = base + e;
  }
  pick = block_int<false>(pick, sh);
  last_pos = block_int<true>(last_pos, sh);
  // (rounding between the piece masses and this prefix can leave the crossing just outside the piece: then
  // the piece's last entry of positive mass)
  if (pick == INT_MAX) pick = last_pos >= 0 ? last_pos : x0;

  int32_t* path = a.accept_path + rb;
  if (tid < T) path[tid] = tid <= depth ? sh.path[tid] : -1;
  if (tid == 0) {
    a.accept_len[b] = depth;
    a.next_token[b] = pick;
    reset_counter(a.seq_ctr + b);
  }
  if (tid < T) reset_counter(row_word(a, b, tid));
}

// Arrival of a finished row at its sequence; the sequence's last row runs the walk.
template <bool VEC>
__device__ __forceinline__ void row_done(const SampledArgs& a, int b, Shared& sh) {
  if (threadIdx.x == 0) sh.flag = add_word(a.seq_ctr + b, 1u) == (uint32_t)(2 * a.T - 2);
  __syncthreads();
  if (sh.flag) walk<VEC>(a, b, sh);
}

// ------------------------------------------------------------------------------------------ stats pieces
template <bool VEC>
__device__ void stats_piece(const SampledArgs& a, int b, int i, int j, Shared& sh) {
  const int tid = threadIdx.x;
  const size_t row = (size_t)b * a.T + i;
  const int x0 = j * CHUNK, x1 = min(a.V, x0 + CHUNK);
  float lt[EPT], ld[EPT];
  load_piece<VEC>(a.target_logits + row * a.V, x0, x1, lt);
  load_piece<VEC>(a.draft_logits + row * a.V, x0, x1, ld);
  float mt = -INFINITY, md = -INFINITY;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    mt = fmaxf(mt, lt[e]);
    md = fmaxf(md, ld[e]);
  }
  mt = block_max(mt, sh);
  md = block_max(md, sh);
  double st = 0.0, sd = 0.0;
  const int base = x0 + tid * EPT;
#pragma unroll
  for (int e = 0; e < EPT; ++e)
    if (base + e < x1) {
      st += scaled_exp((double)lt[e] - (double)mt, a.inv_tau);
      sd += scaled_exp((double)ld[e] - (double)md, a.inv_tau);
    }
  st = block_sum(st, sh);
  sd = block_sum(sd, sh);
  uint32_t* w = row_word(a, b, i);
  if (tid == 0) {
    double* ps = a.piece_stat + (row * a.chunks + j) * 4;
    store_d(ps + 0, mt);
    store_d(ps + 1, st);
    store_d(ps + 2, md);
    store_d(ps + 3, sd);
    wait_vector_memory();
    sh.flag = (add_word(w, kStatsOne) & 0xffffu) == (uint32_t)(a.chunks - 1);
  }
  __syncthreads();
  if (!sh.flag) return;

  // the row's last piece: maxima, normalisers and the target mass of every piece
  const double* ps = a.piece_stat + row * a.chunks * 4;
  float Mt = -INFINITY, Md = -INFINITY;
  for (int k = tid; k < a.chunks; k += NT) {
    Mt = fmaxf(Mt, (float)load_d(ps + 4 * k + 0));
    Md = fmaxf(Md, (float)load_d(ps + 4 * k + 2));
  }
  Mt = block_max(Mt, sh);
  Md = block_max(Md, sh);
  double St = 0.0, Sd = 0.0;
  for (int k = tid; k < a.chunks; k += NT) {
    St += load_d(ps + 4 * k + 1) * scaled_exp(load_d(ps + 4 * k + 0) - (double)Mt, a.inv_tau);
    Sd += load_d(ps + 4 * k + 3) * scaled_exp(load_d(ps + 4 * k + 2) - (double)Md, a.inv_tau);
  }
  St = block_sum(St, sh);
  Sd = block_sum(Sd, sh);
  double* m = a.mass + ((size_t)b * 2 * a.T + i) * a.chunks;
  for (int k = tid; k < a.chunks; k += NT)
    store_d(m + k, load_d(ps + 4 * k + 1) * scaled_exp(load_d(ps + 4 * k + 0) - (double)Mt, a.inv_tau) / St);
  if (tid == 0) {
    double* rs = a.row_stat + row * 4;
    store_d(rs + 0, Mt);
    store_d(rs + 1, St);
    store_d(rs + 2, Md);
    store_d(rs + 3, Sd);
  }
  wait_vector_memory();
  __syncthreads();
  if (tid == 0) add_word(w, kStatsOne);   // the half now reads chunks + 1: published
  row_done<VEC>(a, b, sh);
}

// ------------------------------------------------------------------------------------------- pass pieces
template <bool VEC>
__device__ void pass_piece(const SampledArgs& a, int b, int c, int j, Shared& sh) {
  const int tid = threadIdx.x;
  const int T = a.T;
  const size_t rb = (size_t)b * T;
  if (tid < c) sh.par[tid] = a.parent[rb + tid];
  const int n = a.parent[rb + c];
  __syncthreads();
  const bool valid = n >= 0 && n < c;
  double z = 0.0, C = 0.0, D = 1.0, CC = 1.0;
  int slot = n;
  if (valid) {
    int prev = -1;
    for (int k = tid; k < c; k += NT)
      if (k > n && sh.par[k] == n) prev = max(prev, k);
    prev = block_int<true>(prev, sh);
    const size_t row = rb + n;
    const int x0 = j * CHUNK, x1 = min(a.V, x0 + CHUNK);
    float lt[EPT], ld[EPT];
    load_piece<VEC>(a.target_logits + row * a.V, x0, x1, lt);
    load_piece<VEC>(a.draft_logits + row * a.V, x0, x1, ld);
    if (tid == 0) wait_half(row_word(a, b, n), 0, (uint32_t)a.chunks + 1);
    __syncthreads();
    const double* rs = a.row_stat + row * 4;
    const double Mt = load_d(rs + 0), St = load_d(rs + 1), Md = load_d(rs + 2), Sd = load_d(rs + 3);
    const int base = x0 + tid * EPT;
    double p[EPT], q[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool in = base + e < x1;
      p[e] = in ? scaled_exp((double)lt[e] - Mt, a.inv_tau) / St : 0.0;
      q[e] = in ? scaled_exp((double)ld[e] - Md, a.inv_tau) / Sd : 0.0;
    }
    if (prev >= 0) {
      if (tid == 0) wait_half(row_word(a, b, prev), 16, (uint32_t)a.chunks + 1);
      __syncthreads();
      C = load_d(a.post + (rb + prev) * 4 + 0);
      D = load_d(a.post + (rb + prev) * 4 + 1);
      slot = (int)load_d(a.post + (rb + prev) * 4 + 2);
    }
    CC = C + D;
#pragma unroll
    for (int e = 0; e < EPT; ++e) z += fmax(p[e] - CC * q[e], 0.0);
  }
  z = block_sum(z, sh);
  uint32_t* w = row_word(a, b, c);
  double* m = a.mass + ((size_t)b * 2 * T + T + c) * a.chunks;
  if (tid == 0) {
    store_d(m + j, z);
    wait_vector_memory();
    sh.flag = ((add_word(w, kPassOne) >> 16) & 0xffffu) == (uint32_t)(a.chunks - 1);
  }
  __syncthreads();
  if (!sh.flag) return;

  // the row's last piece: the state after rejecting c
  double Z = 0.0;
  for (int k = tid; k < a.chunks; k += NT) Z += load_d(m + k);
  Z = block_sum(Z, sh);
  if (tid == 0) {
    double* ps = a.post + (rb + c) * 4;
    const bool moved = valid && Z > 0.0;
    store_d(ps + 0, moved ? CC : C);
    store_d(ps + 1, moved ? Z : D);
    store_d(ps + 2, (double)(moved ? T + c : slot));
    wait_vector_memory();
    add_word(w, kPassOne);   // the half now reads chunks + 1: published
  }
  row_done<VEC>(a, b, sh);
}

template <bool VEC>
__global__ __launch_bounds__(NT) void tree_accept_sampled_kernel(SampledArgs a) {
  __shared__ Shared sh;
  __shared__ uint32_t ticket_s;
  if (threadIdx.x == 0) {
    const uint32_t t = add_word(a.ticket, 1u);
    if (t == gridDim.x - 1) reset_counter(a.ticket);   // every workgroup has drawn: clear for the next call
    ticket_s = t;
  }
  __syncthreads();
  const long long t = ticket_s;
  const long long stats = (long long)a.B * a.T * a.chunks;
  if (t < stats) {
    const int j = (int)(t % a.chunks);
    const long long r = t / a.chunks;
    stats_piece<VEC>(a, (int)(r / a.T), (int)(r % a.T), j, sh);
  } else {
    const long long u = t - stats;
    const long long per_child = (long long)a.B * a.chunks;
    const int c = 1 + (int)(u / per_child);
    const long long v = u % per_child;
    pass_piece<VEC>(a, (int)(v / a.chunks), c, (int)(v % a.chunks), sh);
  }
}

}  // namespace

hipError_t launch_tree_accept_sampled(const SampledArgs& a, hipStream_t stream) {
  const long long grid = (long long)a.B * (2 * a.T - 1) * a.chunks;
  if (a.vec4)
    hipLaunchKernelGGL(tree_accept_sampled_kernel<true>, dim3((unsigned)grid), dim3(NT), 0, stream, a);
  else
    hipLaunchKernelGGL(tree_accept_sampled_kernel<false>, dim3((unsigned)grid), dim3(NT), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dreams

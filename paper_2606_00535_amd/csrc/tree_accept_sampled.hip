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
// unchanged when that sum is zero).  So the children of a node need only the node's own p and q: one workgroup
// per piece of each row (2048 entries, each thread holding 8, or 8192 in four parts for problems of many
// pieces) keeps that piece's logits in registers for the whole call and
//   (1) computes the piece's maxima and sums of exp((l - max) / tau), target and draft, and waits for the row's
//       other pieces; every piece then merges the row's statistics itself, in piece order (the same bits
//       everywhere), and forms p and q of its entries;
//   (2) takes the node's children in index order: child c, token x, is decided by the piece holding x
//       (u q(x) D < max(p(x) - C q(x), 0)) against the state its earlier siblings left; each piece adds its part
//       of c's residual mass sum max(p - (C + D) q, 0) and its arrival to c's 64-bit accumulator in one atomic
//       (fixed point, units of 2^-51, so the sum does not depend on the order of arrival) and waits for the
//       whole sum before the next child -- a chain of waits as long as the node's sibling group, among the
//       row's own pieces;
//   (3) draws the token emitted if the walk ends at the node: the prefix of the piece masses (of the last
//       child that moved the state, or of p) finds the piece where the cumulative mass first exceeds
//       u0 * total, and that piece alone finds the token by a block scan; the row's last piece to finish
//       counts the row as done;
//   (4) the sequence's last row to finish walks the tree by ballots (the first kept child of each node) and
//       emits the token prepared for the node it stops at.
// Problems of many pieces (pieces of four 2048-entry parts) use a split form instead, with twice the workgroups:
// first a "stats" workgroup per piece of every row (its last piece draws a leaf's token), then a "pass"
// workgroup per piece of every child c, by c, which merges the parent's statistics, computes p and q of the
// parent's piece and adds c's part of the residual mass once the earlier siblings' sums are complete; the last
// piece of a node's last child draws the node's token.  (At gqa_long's 16 x 128 x 152064 it takes 1.8 ms
// against 2.7 ms for the row-piece form, whose pieces re-stream their parts for every child.)
// Probabilities are fp64, so that the integer outcome is decided in the precision of the definition; exp is
// Tang's table-driven method.
//
// Forward progress.  A row piece only waits for the other pieces of its own row, which are consecutive
// workgroups and wait for nothing outside the row; in the split form a workgroup only waits for rows whose
// pieces all have smaller blockIdx.  Workgroups are dispatched in blockIdx order, so every wait ends.  Waits are nevertheless bounded (0.2 s by default), after which the results are unspecified and the
// workspace's failure flag is set.  Nothing a wait that gave up leaves behind is used as a memory index (piece
// and token positions are clamped, node indices come from the tree), and every arrival word still returns to
// zero.
//
// Results cross workgroups through device-scope stores and loads, published before a relaxed device-scope
// atomic on an arrival word (see kernels.h).  The walker of each sequence clears that sequence's arrival words,
// so every one is back at zero when the launch ends.
#include "kernels.h"

#include <limits.h>
#include <math.h>

namespace dreams {
namespace {

constexpr int NT = kSampledThreads, NW = NT / 64;
constexpr uint64_t kMassMask = (1ull << 53) - 1;   // accumulator: fixed-point mass in the low 53 bits,
constexpr int kArrivalShift = 53;                  // arrivals above
constexpr double kFixScale = 2251799813685248.0;   // 2^51 units per unit of mass
constexpr double kFixUnit = 1.0 / kFixScale;

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void store_d(double* p, double v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double load_d(const double* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_u64(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// exp(x) for x <= 0, by Tang's table-driven method: x = k ln2/256 + r with k = round(x 256/ln2) and
// |r| <= ln2/512 (ln2/256 split in two so that k times the high part is exact), e^x = 2^(k/256) e^r, with
// 2^(j/256) from a 256-entry table and e^r - 1 by its Taylor series to r^5/120 (the next term is below
// 2^-66).  Arguments below -745.5 (past the smallest subnormal) give 0.
__device__ __forceinline__ double exp_nonpos(double x, const double* tab) {
  if (!(x >= -745.5)) return 0.0;
  const double kd = rint(x * 369.3299304675746);
  const int k = (int)kd;
  double r = fma(-kd, 0x1.62e42fefp-9, x);
  r = fma(-kd, 0x1.473de6af278edp-42, r);
  const double em1 = r * fma(r, fma(r, fma(r, fma(r, 1.0 / 120.0, 1.0 / 24.0), 1.0 / 6.0), 0.5), 1.0);
  const double t = tab[k & 255];
  return ldexp(fma(t, em1, t), k >> 8);
}
// exp(d / tau) for d <= 0 as exp(d * (1 / tau)); d = 0 (the maximum itself) gives exactly 1, also where 1 / tau
// is infinite
__device__ __forceinline__ double scaled_exp(double d, double inv_tau, const double* tab) {
  return d == 0.0 ? 1.0 : exp_nonpos(d * inv_tau, tab);
}

struct Shared {
  double tab[256];                 // 2^(j/256)
  double pm[kSampledMaxChunks];    // piece masses of the emitted token's distribution
  double red_d[NW];
  float red_f[NW];
  int red_i[NW];
  double scan[NW];
  int flag, nsib, last_child, depth;
  int par[kMaxNodes];
  int sib[kMaxNodes];
  int path[kMaxNodes];
  double zs[kMaxNodes];            // residual masses of earlier siblings (split form)
  double st_c, st_d;               // a child's whole residual mass; the state (split form)
  int st_slot;
  int fin_piece;
  double fin_before, fin_thr;
  int gave_up;                     // a wait of this workgroup reached its bound
  double rs_mt, rs_ist, rs_md, rs_isd;   // the row's merged statistics
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
// Exclusive prefix of v over the threads in thread order; `total` receives the sum over the block.
__device__ __forceinline__ double block_exclusive_scan(double v, double& total, Shared& sh) {
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
  total = 0.0;
#pragma unroll
  for (int w = 0; w < NW; ++w) total += sh.scan[w];
  return base + inc - v;
}

// A piece is SUB sub-pieces of NT * EPT entries.  In a sub-piece starting at x0, thread t holds entries
// x0 + t * EPT + e (e < EPT); entries at or past x1 read as -inf.  (The split form's EPT; the row-piece form
// holds kSampledPerThreadRow entries a thread.)
constexpr int EPT = kSampledPerThread, SUBW = NT * EPT;
template <bool VEC, int E>
__device__ __forceinline__ void load_sub(const float* row, int x0, int x1, float (&v)[E]) {
  const int base = x0 + (int)threadIdx.x * E;
  if (VEC) {
#pragma unroll
    for (int k = 0; k < E / 4; ++k) {
      const int x = base + 4 * k;   // x0, x1 and x are multiples of 4: a vector is wholly in or out
      f32x4 r = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      if (x < x1) r = *(const f32x4*)(row + x);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[4 * k + e] = r[e];
    }
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = base + e < x1 ? row[base + e] : -INFINITY;
  }
}

__device__ __forceinline__ uint64_t* acc_word(const SampledArgs& a, int b, int i) {
  return (uint64_t*)(a.row_words + ((size_t)b * a.T + i) * a.row_stride);
}
__device__ __forceinline__ uint32_t* stats_word(const SampledArgs& a, int b, int i) {
  return a.row_words + ((size_t)b * a.T + i) * a.row_stride + 2;
}

// A row's maxima and normalisers from its pieces' statistics, merged in piece order by whichever workgroup
// needs them (every one gets the same bits).
struct RowStat {
  double mt, inv_st, md, inv_sd;
};
__device__ RowStat merge_stats(const SampledArgs& a, size_t row, Shared& sh) {
  const int tid = threadIdx.x;
  const double* ps = a.piece_stat + row * a.chunks * 4;
  if (a.chunks <= 64) {
    // one wave, lane k holding piece k: all loads in one round trip, butterfly reductions (the same order in
    // every workgroup)
    if (tid < 64) {
      const bool in = tid < a.chunks;
      const double v0 = in ? load_d(ps + 4 * tid + 0) : -INFINITY, v1 = in ? load_d(ps + 4 * tid + 1) : 0.0;
      const double v2 = in ? load_d(ps + 4 * tid + 2) : -INFINITY, v3 = in ? load_d(ps + 4 * tid + 3) : 0.0;
      float mt = (float)v0, md = (float)v2;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        mt = fmaxf(mt, __shfl_xor(mt, off));
        md = fmaxf(md, __shfl_xor(md, off));
      }
      double st = in ? v1 * scaled_exp(v0 - (double)mt, a.inv_tau, sh.tab) : 0.0;
      double sd = in ? v3 * scaled_exp(v2 - (double)md, a.inv_tau, sh.tab) : 0.0;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        st += __shfl_xor(st, off);
        sd += __shfl_xor(sd, off);
      }
      if (tid == 0) {
        sh.rs_mt = mt;
        sh.rs_ist = 1.0 / st;
        sh.rs_md = md;
        sh.rs_isd = 1.0 / sd;
      }
    }
    __syncthreads();
    return RowStat{sh.rs_mt, sh.rs_ist, sh.rs_md, sh.rs_isd};
  }
  float mt = -INFINITY, md = -INFINITY;
  for (int k = tid; k < a.chunks; k += NT) {
    mt = fmaxf(mt, (float)load_d(ps + 4 * k + 0));
    md = fmaxf(md, (float)load_d(ps + 4 * k + 2));
  }
  mt = block_max(mt, sh);
  md = block_max(md, sh);
  double st = 0.0, sd = 0.0;
  for (int k = tid; k < a.chunks; k += NT) {
    st += load_d(ps + 4 * k + 1) * scaled_exp(load_d(ps + 4 * k + 0) - (double)mt, a.inv_tau, sh.tab);
    sd += load_d(ps + 4 * k + 3) * scaled_exp(load_d(ps + 4 * k + 2) - (double)md, a.inv_tau, sh.tab);
  }
  st = block_sum(st, sh);
  sd = block_sum(sd, sh);
  return RowStat{mt, 1.0 / st, md, 1.0 / sd};
}

// The token emitted if the walk ends at node n with residual max(p - C q, 0): its piece masses are those of
// child `src`'s residual, or, for src < 0, the target's own (from n's piece statistics).  Stored to
// final_token by thread 0 (every thread then waits for its stores).
template <bool VEC, int SUB>
__device__ void final_draw(const SampledArgs& a, int b, int n, const RowStat& rs, double C, int src, Shared& sh) {
  const int tid = threadIdx.x, T = a.T, V = a.V;
  const size_t row = (size_t)b * T + n;
  if (src >= 0) {
    const double* m = a.mass + ((size_t)b * T + src) * a.chunks;
    for (int k = tid; k < a.chunks; k += NT) sh.pm[k] = load_d(m + k);
  } else {
    const double* ps = a.piece_stat + row * a.chunks * 4;
    for (int k = tid; k < a.chunks; k += NT)
      sh.pm[k] = load_d(ps + 4 * k + 1) * scaled_exp(load_d(ps + 4 * k + 0) - rs.mt, a.inv_tau, sh.tab) * rs.inv_st;
  }
  __syncthreads();
  if (tid == 0) {
    double total = 0.0;
    for (int k = 0; k < a.chunks; ++k) total += sh.pm[k];
    const double thr = (double)a.uniforms[(size_t)b * T] * total;
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
  __syncthreads();
  const int piece = sh.fin_piece;
  const double thr = sh.fin_thr;
  double before = sh.fin_before;
  const float* trow = a.target_logits + row * V;
  const float* drow = a.draft_logits + row * V;
  int pick = INT_MAX, last_pos = -1;
#pragma unroll 1
  for (int sp = 0; sp < SUB && pick == INT_MAX; ++sp) {
    const int x0 = (piece * SUB + sp) * SUBW, x1 = min(V, x0 + SUBW);
    if (x0 >= V) break;
    float lt[EPT], ld[EPT];
    load_sub<VEC>(trow, x0, x1, lt);
    load_sub<VEC>(drow, x0, x1, ld);
    const int base = x0 + tid * EPT;
    double r[EPT], mine = 0.0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      r[e] = 0.0;
      if (base + e < x1) {
        const double p = scaled_exp((double)lt[e] - rs.mt, a.inv_tau, sh.tab) * rs.inv_st;
        const double q = C == 0.0 ? 0.0 : scaled_exp((double)ld[e] - rs.md, a.inv_tau, sh.tab) * rs.inv_sd;
        r[e] = fmax(p - C * q, 0.0);
      }
      mine += r[e];
    }
    double total;
    double cum = before + block_exclusive_scan(mine, total, sh);
    int pk = INT_MAX, lp = -1;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      cum += r[e];
      if (pk == INT_MAX && cum > thr) pk = base + e;
      if (r[e] > 0.0) lp = base + e;
    }
    pick = block_int<false>(pk, sh);
    last_pos = max(last_pos, block_int<true>(lp, sh));
    before += total;
  }
  // (rounding between the piece masses and this prefix can leave the crossing just outside the piece: then
  // the piece's last entry of positive mass)
  if (pick == INT_MAX) pick = last_pos >= 0 ? last_pos : min(V - 1, piece * SUB * SUBW);
  if (tid == 0) store_coherent(a.final_token + row, pick);
  wait_vector_memory();
}

// ---------------------------------------------------------------------------------------------------- walk
__device__ void walk(const SampledArgs& a, int b, Shared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T;
  const size_t rb = (size_t)b * T;
  if (wave == 0) {
    // lane l holds nodes l and l + 64; the first kept child of each node, from the root
    int par_h[2], kept_h[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int i = lane + 64 * h;
      par_h[h] = i < T ? a.parent[rb + i] : -1;
      kept_h[h] = i > 0 && i < T ? load_coherent(a.kept + rb + i) : 0;
    }
    int node = 0, depth = 0;
    if (lane == 0) sh.path[0] = 0;
    while (true) {
      const uint64_t k0 = __ballot(kept_h[0] && par_h[0] == node && lane > node);
      const uint64_t k1 = __ballot(kept_h[1] && par_h[1] == node && lane + 64 > node);
      if ((k0 | k1) == 0) break;
      node = k0 ? __builtin_ctzll(k0) : 64 + __builtin_ctzll(k1);
      ++depth;
      if (lane == 0) sh.path[depth] = node;
    }
    if (lane == 0) {
      a.accept_len[b] = depth;
      a.next_token[b] = load_coherent(a.final_token + rb + node);
      reset_counter(a.seq_ctr + b);
      sh.depth = depth;
    }
  }
  __syncthreads();
  const int depth = sh.depth;
  if (tid < T) {
    a.accept_path[rb + tid] = tid <= depth ? sh.path[tid] : -1;
    __hip_atomic_store(acc_word(a, b, tid), (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    reset_counter(stats_word(a, b, tid));
  }
}

// ------------------------------------------------------------- split form (pieces of many sub-pieces)
// Arrival of a finished row at its sequence; the sequence's last row runs the walk.
__device__ __forceinline__ void row_done(const SampledArgs& a, int b, Shared& sh) {
  __syncthreads();   // every thread has read the previous flag
  if (threadIdx.x == 0)
    sh.flag = __hip_atomic_fetch_add(a.seq_ctr + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              (uint32_t)(2 * a.T - 2);
  __syncthreads();
  if (sh.flag) walk(a, b, sh);
}

// ------------------------------------------------------------------------------------------ stats pieces
template <bool VEC, int SUB>
__device__ void stats_piece(const SampledArgs& a, int b, int i, int j, Shared& sh) {
  const int tid = threadIdx.x;
  const size_t row = (size_t)b * a.T + i;
  const float* trow = a.target_logits + row * a.V;
  const float* drow = a.draft_logits + row * a.V;
  // per thread: running maxima and sums relative to them (rescaled when a maximum grows)
  float mt = -INFINITY, md = -INFINITY;
  double st = 0.0, sd = 0.0;
  float lt[EPT], ld[EPT], nt[EPT], nd[EPT];
  int x0 = j * SUB * SUBW;
  load_sub<VEC>(trow, x0, min(a.V, x0 + SUBW), lt);
  load_sub<VEC>(drow, x0, min(a.V, x0 + SUBW), ld);
#pragma unroll 1
  for (int sp = 0; sp < SUB; ++sp, x0 += SUBW) {
    if (sp + 1 < SUB) {   // the next sub-piece's loads in flight during this one's arithmetic
      const int y0 = x0 + SUBW;
      load_sub<VEC>(trow, y0, min(a.V, y0 + SUBW), nt);
      load_sub<VEC>(drow, y0, min(a.V, y0 + SUBW), nd);
    }
    float ct = -INFINITY, cd = -INFINITY;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      ct = fmaxf(ct, lt[e]);
      cd = fmaxf(cd, ld[e]);
    }
    if (ct > mt) {
      if (st != 0.0) st *= scaled_exp((double)mt - (double)ct, a.inv_tau, sh.tab);
      mt = ct;
    }
    if (cd > md) {
      if (sd != 0.0) sd *= scaled_exp((double)md - (double)cd, a.inv_tau, sh.tab);
      md = cd;
    }
    const int base = x0 + tid * EPT, x1 = min(a.V, x0 + SUBW);
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (base + e < x1) {
        st += scaled_exp((double)lt[e] - (double)mt, a.inv_tau, sh.tab);
        sd += scaled_exp((double)ld[e] - (double)md, a.inv_tau, sh.tab);
      }
    if (sp + 1 < SUB) {
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        lt[e] = nt[e];
        ld[e] = nd[e];
      }
    }
  }
  const float bt = block_max(mt, sh), bd = block_max(md, sh);
  if (st != 0.0) st *= scaled_exp((double)mt - (double)bt, a.inv_tau, sh.tab);
  if (sd != 0.0) sd *= scaled_exp((double)md - (double)bd, a.inv_tau, sh.tab);
  mt = bt;
  md = bd;
  st = block_sum(st, sh);
  sd = block_sum(sd, sh);
  uint32_t* w = stats_word(a, b, i);
  if (tid == 0) {
    double* ps = a.piece_stat + (row * a.chunks + j) * 4;
    store_d(ps + 0, mt);
    store_d(ps + 1, st);
    store_d(ps + 2, md);
    store_d(ps + 3, sd);
    wait_vector_memory();
    sh.flag = arrive_last(w, (uint32_t)a.chunks);
  }
  __syncthreads();
  if (!sh.flag) return;

  // the row's last piece: at a leaf, the token emitted if the walk ends here (the target's own distribution)
  const int T = a.T;
  const bool child = tid > i && tid < T && a.parent[(size_t)b * T + tid] == i;
  if (!__syncthreads_or(child)) {
    const RowStat rs = merge_stats(a, row, sh);
    final_draw<VEC, SUB>(a, b, i, rs, 0.0, -1, sh);
  }
  row_done(a, b, sh);
}

// ------------------------------------------------------------------------------------------- pass pieces
template <bool VEC, int SUB>
__device__ void pass_piece(const SampledArgs& a, int b, int c, int j, Shared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T;
  const size_t rb = (size_t)b * T;
  if (tid < T) sh.par[tid] = a.parent[rb + tid];
  if (tid == 0) sh.gave_up = 0;
  __syncthreads();
  const int n = sh.par[c];
  const bool valid = n >= 0 && n < c;
  const int x = a.tokens[rb + c];
  double z = 0.0, C = 0.0, D = 1.0, CC = 1.0;
  int src = -1;
  RowStat rs{};
  if (valid) {
    const size_t row = rb + n;
    const float* trow = a.target_logits + row * a.V;
    const float* drow = a.draft_logits + row * a.V;
    // one-sub-piece pieces: loaded now, p and q computed while the earlier siblings may still be running;
    // larger pieces (where throughput matters more than the wait chain) are streamed after the waits
    constexpr bool HOLD = SUB == 1;
    const int x0 = j * SUB * SUBW, x1 = min(a.V, x0 + SUBW);
    float lt[EPT], ld[EPT];
    if (HOLD) {
      load_sub<VEC>(trow, x0, x1, lt);
      load_sub<VEC>(drow, x0, x1, ld);
    }
    // c's earlier siblings (in index order) and whether c is n's last child
    if (wave == 0) {
      const int k0 = lane, k1 = lane + 64;
      const bool s0 = k0 > n && k0 < c && sh.par[k0] == n;
      const bool s1 = k1 > n && k1 < c && k1 < T && sh.par[k1] == n;
      const bool l0 = k0 > c && k0 < T && sh.par[k0] == n;
      const bool l1 = k1 > c && k1 < T && sh.par[k1] == n;
      const uint64_t b0 = __ballot(s0), b1 = __ballot(s1);
      const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
      if (s0) sh.sib[__builtin_popcountll(b0 & below)] = k0;
      if (s1) sh.sib[__builtin_popcountll(b0) + __builtin_popcountll(b1 & below)] = k1;
      const bool later = (__ballot(l0) | __ballot(l1)) != 0;
      if (lane == 0) {
        sh.nsib = __builtin_popcountll(b0) + __builtin_popcountll(b1);
        sh.last_child = !later;
      }
      // every piece of n's statistics
      if (lane == 0) {
        const uint32_t* w = stats_word(a, b, n);
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        while (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < (uint32_t)a.chunks) {
          if (__builtin_amdgcn_s_memrealtime() - t0 > a.wait_ticks) {
            raise_device_error(a.err, kErrWaitTimeout);
            sh.gave_up = 1;
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
      }
    }
    __syncthreads();
    rs = merge_stats(a, row, sh);
    double p[EPT], q[EPT];
    if (HOLD) {
      const int base = x0 + tid * EPT;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const bool in = base + e < x1;
        p[e] = in ? scaled_exp((double)lt[e] - rs.mt, a.inv_tau, sh.tab) * rs.inv_st : 0.0;
        q[e] = in ? scaled_exp((double)ld[e] - rs.md, a.inv_tau, sh.tab) * rs.inv_sd : 0.0;
      }
    }
    // the earlier siblings' residual masses: complete once their accumulators count every piece
    const int nsib = sh.nsib;
    if (wave == 0 && nsib > 0) {
      const uint64_t* w0 = lane < nsib ? acc_word(a, b, sh.sib[lane]) : nullptr;
      const uint64_t* w1 = lane + 64 < nsib ? acc_word(a, b, sh.sib[lane + 64]) : nullptr;
      uint64_t v0 = 0, v1 = 0;
      const uint64_t full = (uint64_t)a.chunks << kArrivalShift;
      const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
      while (true) {
        if (w0) v0 = load_u64(w0);
        if (w1) v1 = load_u64(w1);
        const bool done = (!w0 || (v0 & ~kMassMask) == full) && (!w1 || (v1 & ~kMassMask) == full);
        if (__ballot(!done) == 0) break;
        if (__builtin_amdgcn_s_memrealtime() - t0 > a.wait_ticks) {
          if (lane == 0) {
            raise_device_error(a.err, kErrWaitTimeout);
            sh.gave_up = 1;
          }
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
      if (w0) sh.zs[lane] = (double)(v0 & kMassMask) * kFixUnit;
      if (w1) sh.zs[lane + 64] = (double)(v1 & kMassMask) * kFixUnit;
    }
    __syncthreads();
    if (tid == 0) {
      double c_run = 0.0, d_run = 1.0;
      int s_run = -1;
      for (int k = 0; k < nsib; ++k) {
        const double zk = sh.zs[k];
        if (zk > 0.0) {
          c_run += d_run;
          d_run = zk;
          s_run = sh.sib[k];
        }
      }
      sh.st_c = c_run;
      sh.st_d = d_run;
      sh.st_slot = s_run;
    }
    __syncthreads();
    C = sh.st_c;
    D = sh.st_d;
    src = sh.st_slot;
    CC = C + D;
    double px = 0.0, qx = 0.0;
    bool mine = false;
    if (HOLD) {
      const int base = x0 + tid * EPT;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        z += fmax(p[e] - CC * q[e], 0.0);
        if (base + e == x && base + e < x1) {
          px = p[e];
          qx = q[e];
          mine = true;
        }
      }
    } else {
      float nt[EPT], nd[EPT];
      int y0 = x0;
      load_sub<VEC>(trow, y0, min(a.V, y0 + SUBW), lt);
      load_sub<VEC>(drow, y0, min(a.V, y0 + SUBW), ld);
#pragma unroll 1
      for (int sp = 0; sp < SUB; ++sp, y0 += SUBW) {
        if (sp + 1 < SUB) {   // the next sub-piece's loads in flight during this one's arithmetic
          load_sub<VEC>(trow, y0 + SUBW, min(a.V, y0 + 2 * SUBW), nt);
          load_sub<VEC>(drow, y0 + SUBW, min(a.V, y0 + 2 * SUBW), nd);
        }
        const int base = y0 + tid * EPT, y1 = min(a.V, y0 + SUBW);
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
          if (base + e < y1) {
            const double pe = scaled_exp((double)lt[e] - rs.mt, a.inv_tau, sh.tab) * rs.inv_st;
            const double qe = scaled_exp((double)ld[e] - rs.md, a.inv_tau, sh.tab) * rs.inv_sd;
            z += fmax(pe - CC * qe, 0.0);
            if (base + e == x) {
              px = pe;
              qx = qe;
              mine = true;
            }
          }
        }
        if (sp + 1 < SUB) {
#pragma unroll
          for (int e = 0; e < EPT; ++e) {
            lt[e] = nt[e];
            ld[e] = nd[e];
          }
        }
      }
    }
    // c's decision, by the thread holding its token
    if (mine) store_coherent(a.kept + rb + c, (int32_t)(((double)a.uniforms[rb + c] * qx) * D < fmax(px - C * qx, 0.0)));
  }
  if ((!valid || x < 0 || x >= a.V) && j == 0 && tid == 0) store_coherent(a.kept + rb + c, 0);
  z = block_sum(z, sh);
  if (tid == 0) store_d(a.mass + (rb + c) * a.chunks + j, z);
  wait_vector_memory();
  __syncthreads();
  if (tid == 0) {
    // A piece's mass is at most 1 (up to rounding); after a wait gave up it is meaningless and counts as 0, so
    // that it can never carry into the arrival bits: the count, and with it the walk, still completes.
    const double zc = sh.gave_up ? 0.0 : fmin(fmax(z, 0.0), 2.0);
    const uint64_t mine = (uint64_t)rint(zc * kFixScale);
    const uint64_t old = __hip_atomic_fetch_add(acc_word(a, b, c), (1ull << kArrivalShift) + mine, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    sh.flag = (int)(old >> kArrivalShift) == a.chunks - 1;
    sh.zs[0] = (double)((old & kMassMask) + mine) * kFixUnit;   // the row's whole residual mass
  }
  __syncthreads();
  if (!sh.flag) return;
  // c's last piece: if c is n's last child, the token emitted if the walk ends at n (every child rejected)
  if (valid && sh.last_child) {
    const bool moved = sh.zs[0] > 0.0;
    final_draw<VEC, SUB>(a, b, n, rs, moved ? CC : C, moved ? c : src, sh);
    __syncthreads();
  }
  row_done(a, b, sh);
}

// ------------------------------------------------------------------------------------------- row pieces
// Workgroup (b, n, j): piece j of row n.  Its logits stay in registers for the whole call.
template <bool VEC, int SUB, int E>
__device__ void row_piece(const SampledArgs& a, int b, int n, int j, Shared& sh) {
  constexpr int EPT = E, SUBW = NT * E;   // (this form's entries per thread and per sub-piece)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T, V = a.V;
  const size_t rb = (size_t)b * T, row = rb + n;
  const float* trow = a.target_logits + row * V;
  const float* drow = a.draft_logits + row * V;
  // One-part pieces keep their logits (and later p and q) in registers; four-part pieces stream their parts
  // from memory in every pass (the registers would not hold them).
  constexpr bool HOLD = SUB == 1;
  float lt0[EPT], ld0[EPT];
  if (HOLD) {
    load_sub<VEC>(trow, j * SUBW, min(V, j * SUBW + SUBW), lt0);
    load_sub<VEC>(drow, j * SUBW, min(V, j * SUBW + SUBW), ld0);
  }
  // f(sp, e, x, target logit, draft logit) for every entry x < V of the piece, in order
  auto entries = [&](auto&& f) {
    if (HOLD) {
      const int base = j * SUBW + tid * EPT;
#pragma unroll
      for (int e = 0; e < EPT; ++e)
        if (base + e < V) f(0, e, base + e, lt0[e], ld0[e]);
    } else {
#pragma unroll 1
      for (int sp = 0; sp < SUB; ++sp) {
        const int x0 = (j * SUB + sp) * SUBW;
        if (x0 >= V) break;
        float ta[EPT], da[EPT];
        load_sub<VEC>(trow, x0, min(V, x0 + SUBW), ta);
        load_sub<VEC>(drow, x0, min(V, x0 + SUBW), da);
        const int base = x0 + tid * EPT;
#pragma unroll
        for (int e = 0; e < EPT; ++e)
          if (base + e < V) f(sp, e, base + e, ta[e], da[e]);
      }
    }
  };
  // n's children in index order (every piece of the row lists them the same way)
  if (wave == 0) {
    const int k0 = lane, k1 = lane + 64;
    const bool c0 = k0 > n && k0 < T && a.parent[rb + k0] == n;
    const bool c1 = k1 > n && k1 < T && a.parent[rb + k1] == n;
    const uint64_t b0 = __ballot(c0), b1 = __ballot(c1);
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
    if (c0) sh.sib[__builtin_popcountll(b0 & below)] = k0;
    if (c1) sh.sib[__builtin_popcountll(b0) + __builtin_popcountll(b1 & below)] = k1;
    if (lane == 0) {
      sh.nsib = __builtin_popcountll(b0) + __builtin_popcountll(b1);
      sh.gave_up = 0;
    }
  }

  // ---- the piece's statistics: maxima and sums of exp((l - max) / tau), target and draft.  A one-part piece
  // takes its thread's maxima first and keeps the exponentials relative to them, from which p and q follow by
  // one factor each; a streamed piece re-references its sums when a maximum grows.
  float mt = -INFINITY, md = -INFINITY;
  double st = 0.0, sd = 0.0;
  double et[EPT], ed[EPT];   // (one-part pieces)
  if (HOLD) {
    const int base = j * SUBW + tid * EPT;
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (base + e < V) {
        mt = fmaxf(mt, lt0[e]);
        md = fmaxf(md, ld0[e]);
      }
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool in = base + e < V;
      et[e] = in ? scaled_exp((double)lt0[e] - (double)mt, a.inv_tau, sh.tab) : 0.0;
      ed[e] = in ? scaled_exp((double)ld0[e] - (double)md, a.inv_tau, sh.tab) : 0.0;
      st += et[e];
      sd += ed[e];
    }
  } else {
    entries([&](int, int, int, float t, float d) {
      if (t > mt) {
        if (st != 0.0) st *= scaled_exp((double)mt - (double)t, a.inv_tau, sh.tab);
        mt = t;
      }
      if (d > md) {
        if (sd != 0.0) sd *= scaled_exp((double)md - (double)d, a.inv_tau, sh.tab);
        md = d;
      }
      st += scaled_exp((double)t - (double)mt, a.inv_tau, sh.tab);
      sd += scaled_exp((double)d - (double)md, a.inv_tau, sh.tab);
    });
  }
  const float mt_own = mt, md_own = md;
  const float bt = block_max(mt, sh), bd = block_max(md, sh);
  if (st != 0.0) st *= scaled_exp((double)mt - (double)bt, a.inv_tau, sh.tab);
  if (sd != 0.0) sd *= scaled_exp((double)md - (double)bd, a.inv_tau, sh.tab);
  st = block_sum(st, sh);
  sd = block_sum(sd, sh);
  if (tid == 0) {
    double* ps = a.piece_stat + (row * a.chunks + j) * 4;
    store_d(ps + 0, bt);
    store_d(ps + 1, st);
    store_d(ps + 2, bd);
    store_d(ps + 3, sd);
    wait_vector_memory();
    uint32_t* w = stats_word(a, b, n);
    __hip_atomic_fetch_add(w, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // every piece of the row
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < (uint32_t)a.chunks) {
      if (__builtin_amdgcn_s_memrealtime() - t0 > a.wait_ticks) {
        raise_device_error(a.err, kErrWaitTimeout);
        sh.gave_up = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
  const RowStat rs = merge_stats(a, row, sh);
  auto prob_p = [&](float t) { return scaled_exp((double)t - rs.mt, a.inv_tau, sh.tab) * rs.inv_st; };
  auto prob_q = [&](float d) { return scaled_exp((double)d - rs.md, a.inv_tau, sh.tab) * rs.inv_sd; };
  double pc[EPT], qc[EPT];   // (one-part pieces: the kept exponentials times one factor each)
  if (HOLD) {
    const double ft = mt_own == -INFINITY ? 0.0 : scaled_exp((double)mt_own - rs.mt, a.inv_tau, sh.tab) * rs.inv_st;
    const double fd = md_own == -INFINITY ? 0.0 : scaled_exp((double)md_own - rs.md, a.inv_tau, sh.tab) * rs.inv_sd;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      pc[e] = et[e] * ft;
      qc[e] = ed[e] * fd;
    }
  }

  // ---- n's children in index order.  Child c (token x) is tested against the state (C, D) its earlier
  // siblings left; its residual mass sum max(p - (C + D) q, 0) is summed over the row's pieces in its 64-bit
  // accumulator (fixed point, so the sum does not depend on the order of arrival), and every piece waits for
  // the whole sum before the next child.
  const int nsib = sh.nsib;
  double C = 0.0, D = 1.0;
  int src = -1;
  for (int k = 0; k < nsib; ++k) {
    const int c = sh.sib[k];
    const int x = a.tokens[rb + c];
    const double CC = C + D;
    double z = 0.0, px = 0.0, qx = 0.0;
    bool mine = false;
    entries([&](int, int e, int xi, float t, float d) {
      const double pe = HOLD ? pc[e] : prob_p(t), qe = HOLD ? qc[e] : prob_q(d);
      z += fmax(pe - CC * qe, 0.0);
      if (xi == x) {
        px = pe;
        qx = qe;
        mine = true;
      }
    });
    // c's decision, by the thread holding its token (a token outside the vocabulary is never kept)
    if (mine) store_coherent(a.kept + rb + c, (int32_t)(((double)a.uniforms[rb + c] * qx) * D < fmax(px - C * qx, 0.0)));
    if ((x < 0 || x >= V) && j == 0 && tid == 0) store_coherent(a.kept + rb + c, 0);
    z = block_sum(z, sh);
    if (tid == 0) {
      // this piece's part of c's residual mass (read by the row's draw if c is the last child to move the
      // state); the last child's arrival waits for every such store of the piece first
      store_d(a.mass + (rb + c) * a.chunks + j, z);
      if (k == nsib - 1) wait_vector_memory();
      // A piece's mass is at most 1 (up to rounding); after a wait gave up it is meaningless and counts as 0,
      // so that it can never carry into the arrival bits: the count, and with it the walk, still completes.
      const double zc = sh.gave_up ? 0.0 : fmin(fmax(z, 0.0), 2.0);
      const uint64_t fix = (uint64_t)rint(zc * kFixScale);
      uint64_t* w = acc_word(a, b, c);
      __hip_atomic_fetch_add(w, (1ull << kArrivalShift) + fix, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const uint64_t full = (uint64_t)a.chunks << kArrivalShift;
      const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
      uint64_t v;
      while (((v = load_u64(w)) & ~kMassMask) != full) {
        if (__builtin_amdgcn_s_memrealtime() - t0 > a.wait_ticks) {
          raise_device_error(a.err, kErrWaitTimeout);
          sh.gave_up = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      sh.st_c = (double)(v & kMassMask) * kFixUnit;   // c's whole residual mass
    }
    __syncthreads();
    const double Zc = sh.st_c;
    if (Zc > 0.0) {
      C = CC;
      D = Zc;
      src = c;
    }
  }

  // ---- the token emitted if the walk ends at n (every child rejected, or a leaf): drawn from max(p - C q, 0)
  // through the inverse CDF with u0; the piece masses are those of child src's residual (every piece stored
  // its part before its last arrival, which this piece has seen), or the target's own
  if (src >= 0) {
    const double* m = a.mass + (rb + src) * a.chunks;
    for (int k = tid; k < a.chunks; k += NT) sh.pm[k] = load_d(m + k);
  } else {
    const double* ps = a.piece_stat + row * a.chunks * 4;
    for (int k = tid; k < a.chunks; k += NT)
      sh.pm[k] = load_d(ps + 4 * k + 1) * scaled_exp(load_d(ps + 4 * k + 0) - rs.mt, a.inv_tau, sh.tab) * rs.inv_st;
  }
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
  __syncthreads();
  if (sh.fin_piece == j) {   // (one piece of the row draws)
    const double thr = sh.fin_thr;
    double before = sh.fin_before;
    int pick = INT_MAX, last_pos = -1;
    // part by part (a one-part piece has one): the block's prefix of r = max(p - C q, 0) in entry order
#pragma unroll 1
    for (int sp = 0; sp < SUB && pick == INT_MAX; ++sp) {
      const int x0 = (j * SUB + sp) * SUBW;
      if (x0 >= V) break;
      const int base = x0 + tid * EPT;
      float ta[EPT], da[EPT];
      if (HOLD) {
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
          ta[e] = lt0[e];
          da[e] = ld0[e];
        }
      } else {
        load_sub<VEC>(trow, x0, min(V, x0 + SUBW), ta);
        load_sub<VEC>(drow, x0, min(V, x0 + SUBW), da);
      }
      double r[EPT], mine_sum = 0.0;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        r[e] = 0.0;
        if (base + e < V) {
          const double pe = HOLD ? pc[e] : prob_p(ta[e]);
          const double qe = C == 0.0 ? 0.0 : (HOLD ? qc[e] : prob_q(da[e]));
          r[e] = fmax(pe - C * qe, 0.0);
        }
        mine_sum += r[e];
      }
      double total;
      double cum = before + block_exclusive_scan(mine_sum, total, sh);
      int pk = INT_MAX, lp = -1;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        cum += r[e];
        if (pk == INT_MAX && cum > thr) pk = base + e;
        if (r[e] > 0.0) lp = base + e;
      }
      pick = block_int<false>(pk, sh);
      last_pos = max(last_pos, block_int<true>(lp, sh));
      before += total;
    }
    // (rounding between the piece masses and this prefix can leave the crossing just outside the piece: then
    // the piece's last entry of positive mass)
    if (pick == INT_MAX) pick = last_pos >= 0 ? last_pos : min(V - 1, j * SUB * SUBW);
    if (tid == 0) store_coherent(a.final_token + row, pick);
    wait_vector_memory();
  }
  // Every piece counts itself out on the row's statistics word (which already holds one arrival per piece),
  // once its decisions and token are stored; the row's last piece counts the row as done, and the sequence's
  // last row runs the walk.  (So each row is counted once even where a wait gave up and the pieces disagree on
  // which one draws.)
  wait_vector_memory();
  __syncthreads();
  if (tid == 0) {
    int walker = 0;
    if (__hip_atomic_fetch_add(stats_word(a, b, n), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
        (uint32_t)(2 * a.chunks - 1))
      walker = __hip_atomic_fetch_add(a.seq_ctr + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (uint32_t)(T - 1);
    sh.flag = walker;
  }
  __syncthreads();
  if (sh.flag) walk(a, b, sh);
}

template <bool VEC, int SUB>
__global__ __launch_bounds__(NT) void tree_accept_sampled_kernel(SampledArgs a) {
  __shared__ Shared sh;
  sh.tab[threadIdx.x] = exp2((double)threadIdx.x * (1.0 / 256.0));
  __syncthreads();
  const long long t = blockIdx.x;
  const int j = (int)(t % a.chunks);
  const long long r = t / a.chunks;
  row_piece<VEC, SUB, kSampledPerThreadRow>(a, (int)(r / a.T), (int)(r % a.T), j, sh);
}

template <bool VEC, int SUB>
__global__ __launch_bounds__(NT) void tree_accept_sampled_split_kernel(SampledArgs a) {
  __shared__ Shared sh;
  sh.tab[threadIdx.x] = exp2((double)threadIdx.x * (1.0 / 256.0));
  __syncthreads();
  const long long t = blockIdx.x;
  const long long stats = (long long)a.B * a.T * a.chunks;
  if (t < stats) {
    const int j = (int)(t % a.chunks);
    const long long r = t / a.chunks;
    stats_piece<VEC, SUB>(a, (int)(r / a.T), (int)(r % a.T), j, sh);
  } else {
    const long long u = t - stats;
    const long long per_child = (long long)a.B * a.chunks;
    const int c = 1 + (int)(u / per_child);
    const long long v = u % per_child;
    pass_piece<VEC, SUB>(a, (int)(v / a.chunks), c, (int)(v % a.chunks), sh);
  }
}

}  // namespace

hipError_t launch_tree_accept_sampled(const SampledArgs& a, hipStream_t stream) {
  static_assert(NT == 256, "the exp table is filled one entry per thread");
  // one-part pieces: a workgroup per row piece; four-part pieces (problems of many pieces): the split form
  const bool large = a.sub_pieces == kSampledSubLarge;
  const long long grid = large ? (long long)a.B * (2 * a.T - 1) * a.chunks : (long long)a.B * a.T * a.chunks;
  auto go = [&](auto kern) { hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(NT), 0, stream, a); };
  if (a.vec4) {
    if (large) go(tree_accept_sampled_split_kernel<true, kSampledSubLarge>);
    else go(tree_accept_sampled_kernel<true, 1>);
  } else {
    if (large) go(tree_accept_sampled_split_kernel<false, kSampledSubLarge>);
    else go(tree_accept_sampled_kernel<false, 1>);
  }
  return hipGetLastError();
}

}  // namespace dreams

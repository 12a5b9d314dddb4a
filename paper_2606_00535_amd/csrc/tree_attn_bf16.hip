// Tree-masked verification attention on the gfx950 matrix cores (bf16 inputs, fp32 accumulation).
//
// What is computed (the paper's Section 3.2 attention matrix, applied to the target's verification pass of
// Section 2): for every tree node i of every query head, softmax(scale * q_i . k_j) v_j over the committed
// prefix slots and the slots of node i's ancestors-or-self.  A row's visible set is "all prefix slots" plus
// at most depth+1 tree slots, so the mask is only evaluated on key tiles that reach the tree part.
//
// Work decomposition
//   * A workgroup (4 waves) owns kAttnRows = 64 query rows of one KV head.  With grouped-query attention
//     the rows of all G query heads that share the KV head are packed together (row r -> head r / T, node
//     r % T), so every K/V tile read from HBM is used by all of them.
//   * The key axis of a (sequence, KV head) is cut into `splits` contiguous pieces, one per workgroup, so a
//     single-sequence shape still fills all compute units.  Each piece keeps an online softmax (running max
//     m, running sum l, unnormalised accumulator); the last workgroup of a piece set to finish (arrival
//     counter) merges them with the log-sum-exp identity in fixed split order, so results are reproducible
//     bit for bit whichever workgroup arrives last.
//   * Workgroup ids are remapped so that every workgroup of one (sequence, KV head) runs on the same XCD
//     (the dispatcher deals consecutive ids round-robin over the 8 XCDs): row groups that read the same K/V
//     tile share it in that XCD's L2.  Partial results travel through device-scope stores and loads.
//   * This kernel serves shapes with many query rows per KV head (grouped-query heads x tree nodes); shapes
//     with few rows go to the streaming kernel, whose waves split the keys instead of the rows.
//
// Per key tile (KT keys): the whole workgroup streams K and V rows with 16-byte coalesced loads into LDS
// (register double-buffered: the next tile's loads are in flight while this one is computed).  Each wave
// then computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (K rows as the A operand, read straight from LDS
// in operand layout; the wave's 16 query rows stay in registers as the B operand).  Producing S^T rather
// than S leaves each lane holding one query row's scores, which is exactly the B-operand layout of the next
// product, O^T += V^T P^T, so the probabilities never leave registers; only V needs a transposed read from
// LDS.  All row statistics are lane-local up to a 4-way cross-lane reduction.
#include "kernels.h"

#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Ancestor-or-self bit sets of every tree node of sequence b, into LDS (2 x 64 bits per node).
__device__ __forceinline__ void build_ancestors(const AttnArgs& a, int b, uint64_t* anc, int tid) {
  const int T = a.T;
  if (tid < T) {
    uint64_t m0 = 0, m1 = 0;
    if (a.mask) {
      const int W = (T + 63) / 64;
      const uint64_t* mr = a.mask + ((size_t)b * T + tid) * W;
      m0 = mr[0];
      m1 = W > 1 ? mr[1] : 0;
    } else {
      const int32_t* par = a.parent + (size_t)b * T;
      int j = tid;
      for (int step = 0; step <= T && j >= 0; ++step) {
        if (j < 64) m0 |= 1ull << j; else m1 |= 1ull << (j - 64);
        const int p = par[j];
        if (p >= j) break;  // not a valid parent: the walk ends here
        j = p;              // -1 at the root ends the walk
      }
    }
    anc[2 * tid] = m0;
    anc[2 * tid + 1] = m1;
  }
}

template <int D, int KT>
__global__ __launch_bounds__(kAttnThreads) void tree_attn_bf16_kernel(AttnArgs a) {
  constexpr int NT = kAttnThreads;
  constexpr int DS = D / 32;          // k-steps of S^T = K Q^T
  constexpr int DB = D / 16;          // 16-column blocks of O^T
  constexpr int KB = KT / 16;         // 16-key blocks per tile
  constexpr int KC = KT / 32;         // 32-key chunks per tile (one O^T MFMA each)
  constexpr int KS = D + 8;           // LDS row stride of K (elements): conflict-free 16-byte operand reads
  constexpr int VS = D + 16;          // LDS row stride of V: conflict-free transposed 2-byte reads
  constexpr int CPR = D / 8;          // 16-byte chunks per key row
  constexpr int LPT = KT * CPR / NT;  // chunks of K (and of V) each thread moves per tile
  static_assert(LPT * NT == KT * CPR, "tile must split evenly over the workgroup");

  // K tile, then V tile; after the main loop the same bytes hold the merge's staging (see below)
  __shared__ __attribute__((aligned(16))) __bf16 tiles[KT * KS + KT * VS];
  __bf16* const k_lds = tiles;
  __bf16* const v_lds = tiles + KT * KS;
  static_assert(kAttnMaxSplits * kAttnRows * 8 + 2 * kAttnRows * 4 <= (KT * KS + KT * VS) * 2,
                "merge staging must fit in the tile buffers");
  __shared__ uint64_t anc_lds[2 * kMaxNodes];
  __shared__ int last_flag;

  // ---- which (unit = sequence x KV head, split, row group) this workgroup owns
  const int n = blockIdx.x;
  const int xcd = n & 7, slot = n >> 3;
  const int per_unit = a.splits * a.row_groups;
  const int u = xcd + 8 * (slot / per_unit);
  if (u >= a.units) return;
  const int within = slot - (slot / per_unit) * per_unit;
  const int split = within / a.row_groups;
  const int rg = within - split * a.row_groups;
  const int b = u / a.Hkv, g = u - b * a.Hkv;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, quad = lane >> 4, col = lane & 15;
  const int T = a.T;
  int L = a.kv_len[b];
  L = L < 0 ? 0 : (L > a.S_cap - T ? a.S_cap - T : L);
  const int N = L + T;
  int piece = (N + a.splits - 1) / a.splits;
  piece = (piece + KT - 1) / KT * KT;
  const int k_begin = split * piece;
  const int k_end = min(N, k_begin + piece);

  build_ancestors(a, b, anc_lds, tid);
  __syncthreads();

  // ---- this lane's query row (B operand of S^T and of O^T): row = col within the wave's 16 rows
  const int rows_total = a.G * T;
  const int row_local = wave * 16 + col;
  const int row = rg * kAttnRows + row_local;
  const bool row_ok = row < rows_total;
  const int head_in_group = row_ok ? row / T : 0;
  const int node = row_ok ? row - head_in_group * T : 0;
  const int h = g * a.G + head_in_group;
  const uint64_t anc0 = anc_lds[2 * node], anc1 = anc_lds[2 * node + 1];

  bf16x8 qf[DS];
  {
    const __bf16* qrow = (const __bf16*)a.q + (((size_t)b * a.Hq + h) * T + node) * D;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      if (row_ok) {
        qf[s] = *(const bf16x8*)(qrow + s * 32 + quad * 8);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[s][e] = (__bf16)0.0f;
      }
    }
  }

  f32x4 o[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const __bf16* kbase = (const __bf16*)a.k + (size_t)u * a.S_cap * D;
  const __bf16* vbase = (const __bf16*)a.v + (size_t)u * a.S_cap * D;

  u32x4 kreg[LPT], vreg[LPT];
  auto load_tile = [&](int t0) {
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      const int c = tid + j * NT;
      const int key = c / CPR, cc = c - key * CPR;
      const int s = t0 + key;
      if (s < k_end) {
        kreg[j] = *(const u32x4*)(kbase + (size_t)s * D + cc * 8);
        vreg[j] = *(const u32x4*)(vbase + (size_t)s * D + cc * 8);
      } else {  // past this piece: zeros, so masked keys can never inject NaN/Inf through V
        kreg[j] = u32x4{0u, 0u, 0u, 0u};
        vreg[j] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
      const int c = tid + j * NT;
      const int key = c / CPR, cc = c - key * CPR;
      *(u32x4*)(k_lds + key * KS + cc * 8) = kreg[j];
      *(u32x4*)(v_lds + key * VS + cc * 8) = vreg[j];
    }
  };

  if (k_begin < k_end) {
    load_tile(k_begin);
    for (int t0 = k_begin; t0 < k_end; t0 += KT) {
      __syncthreads();  // every wave is done reading the previous tile
      store_tile();
      __syncthreads();
      if (t0 + KT < k_end) load_tile(t0 + KT);

      // S^T block kb: A-operand row m holds key kb*16 + (m%4)*4 + m/4, so that accumulator element e of a
      // lane in quad q is key kb*16 + e*4 + q (see the V read below for why).
      f32x4 s[KB];
      {
        const int keyA = (col & 3) * 4 + (col >> 2);
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
          const __bf16* kr = k_lds + (kb * 16 + keyA) * KS + quad * 8;
#pragma unroll
          for (int ds = 0; ds < DS; ++ds)
            s[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8*)(kr + ds * 32), qf[ds], s[kb], 0, 0, 0);
        }
      }

      // scale into log2 units, mask, tile row-max
      float tmax = -INFINITY;
      const bool tree_tile = t0 + KT > L;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = t0 + kb * 16 + e * 4 + quad;
          float x = s[kb][e] * a.scale_log2;
          bool vis = key < k_end;
          if (tree_tile && key >= L) {
            const int j = key - L;
            vis = vis && (((j < 64 ? anc0 >> j : anc1 >> (j - 64)) & 1ull) != 0);
          }
          x = vis ? x : -INFINITY;
          s[kb][e] = x;
          tmax = fmaxf(tmax, x);
        }
      }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      const float m_new = fmaxf(m_run, tmax);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(m_run - m_use);
      m_run = m_new;
      float psum = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = fast_exp2(s[kb][e] - m_use);
          s[kb][e] = p;
          psum += p;
        }
      }
      l_run = l_run * alpha + psum;
#pragma unroll
      for (int d = 0; d < DB; ++d) o[d] *= alpha;

      // O^T[d][row] += sum over 32 keys V[key][d] * P[row][key].  k-slot 0..3 of quad q = keys e*4+q of the
      // even 16-key block, k-slots 4..7 = the same of the odd block: exactly what this lane holds in s[].
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        bf16x8 pb;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pb[e] = (__bf16)s[2 * c][e];
          pb[4 + e] = (__bf16)s[2 * c + 1][e];
        }
        const __bf16* vr0 = v_lds + (c * 32 + quad) * VS + col;
        const __bf16* vr1 = vr0 + 16 * VS;
#pragma unroll
        for (int d = 0; d < DB; ++d) {
          bf16x8 va;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            va[e] = vr0[e * 4 * VS + d * 16];
            va[4 + e] = vr1[e * 4 * VS + d * 16];
          }
          o[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb, o[d], 0, 0, 0);
        }
      }
    }
  }

  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  // lane holds O[row][d*16 + quad*4 + e] for e = 0..3
  if (a.splits == 1) {
    if (row_ok) {
      const size_t orow = (((size_t)b * a.Hq + h) * T + node);
      const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
      __bf16* op = (__bf16*)a.out + orow * D + quad * 4;
#pragma unroll
      for (int d = 0; d < DB; ++d) {
        bf16x4 r;
#pragma unroll
        for (int e = 0; e < 4; ++e) r[e] = (__bf16)(o[d][e] * inv);
        *(bf16x4*)(op + d * 16) = r;
      }
      if (a.lse && quad == 0) a.lse[orow] = l_run > 0.f ? (m_run + __log2f(l_run)) * kLn2 : -INFINITY;
    }
    return;
  }

  // ---- several pieces: publish this piece's partial result, the last arrival merges
  const size_t pset = (size_t)u * a.row_groups + rg;
  const size_t pbase = (pset * a.splits + split) * kAttnRows + row_local;
  {
    float* pa = a.part_acc + pbase * D + quad * 4;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int e = 0; e < 4; ++e) store_coherent(pa + d * 16 + e, o[d][e]);
    if (quad == 0) {
      store_coherent(a.part_ml + 2 * pbase, m_run);
      store_coherent(a.part_ml + 2 * pbase + 1, l_run);
    }
  }
  wait_vector_memory();
  __syncthreads();
  if (tid == 0) last_flag = arrive_last(&a.counters[pset], (uint32_t)a.splits);
  __syncthreads();
  if (!last_flag) return;
  if (tid == 0) reset_counter(&a.counters[pset]);

  // Merge.  (1) one round trip stages every piece's (m, l) for the 64 rows in LDS (the K/V tile buffers are
  // free now); (2) one thread per row turns them into weights 2^(m_s - M) and 1/sum; (3) every thread owns
  // one 4-column slice of several rows and streams the pieces' accumulators with many loads in flight.
  float2* ml = (float2*)tiles;                       // [splits][kAttnRows]
  float* inv_l = (float*)(ml + kAttnMaxSplits * kAttnRows);  // [kAttnRows]
  float* row_m = inv_l + kAttnRows;                  // [kAttnRows]
  const int S = a.splits;
  const size_t pset_rows = pset * S * kAttnRows;
  for (int e = tid; e < S * kAttnRows; e += NT)
    ml[e] = make_float2(load_coherent(a.part_ml + 2 * (pset_rows + e)), load_coherent(a.part_ml + 2 * (pset_rows + e) + 1));
  __syncthreads();
  if (tid < kAttnRows) {
    float M = -INFINITY;
    for (int sp = 0; sp < S; ++sp) M = fmaxf(M, ml[sp * kAttnRows + tid].x);
    float lsum = 0.f;
    for (int sp = 0; sp < S; ++sp) {
      const float2 v = ml[sp * kAttnRows + tid];
      const float w = v.x == -INFINITY ? 0.f : fast_exp2(v.x - M);
      lsum += w * v.y;
      ml[sp * kAttnRows + tid].x = w;
    }
    inv_l[tid] = lsum > 0.f ? 1.0f / lsum : 0.f;
    row_m[tid] = lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
  }
  __syncthreads();

  constexpr int D4 = D / 4;                          // 4-column slices per row
  constexpr int RSTEP = NT / D4;                     // rows covered by one pass of the workgroup
  constexpr int RPT = kAttnRows / RSTEP;             // rows per thread
  const int d4 = tid % D4, r0 = tid / D4;
  f32x4 acc[RPT];
#pragma unroll
  for (int j = 0; j < RPT; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float* pacc = a.part_acc + pset_rows * D + d4 * 4;
  auto load4 = [&](size_t idx) {
    const float* p = pacc + idx * D;
    return f32x4{load_coherent(p), load_coherent(p + 1), load_coherent(p + 2), load_coherent(p + 3)};
  };
  int sp = 0;
  for (; sp + 1 < S; sp += 2) {                      // two pieces x RPT rows of loads in flight
    f32x4 x0[RPT], x1[RPT];
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      x0[j] = load4((size_t)sp * kAttnRows + r0 + j * RSTEP);
      x1[j] = load4((size_t)(sp + 1) * kAttnRows + r0 + j * RSTEP);
    }
#pragma unroll
    for (int j = 0; j < RPT; ++j)
      acc[j] += ml[sp * kAttnRows + r0 + j * RSTEP].x * x0[j] + ml[(sp + 1) * kAttnRows + r0 + j * RSTEP].x * x1[j];
  }
  if (sp < S) {
#pragma unroll
    for (int j = 0; j < RPT; ++j)
      acc[j] += ml[sp * kAttnRows + r0 + j * RSTEP].x * load4((size_t)sp * kAttnRows + r0 + j * RSTEP);
  }
  const int rows_here = min(kAttnRows, rows_total - rg * kAttnRows);
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const int rl = r0 + j * RSTEP;
    if (rl >= rows_here) continue;
    const int r = rg * kAttnRows + rl;
    const int hg = r / T, nd = r - hg * T;
    const size_t orow = ((size_t)b * a.Hq + g * a.G + hg) * T + nd;
    const float inv = inv_l[rl];
    bf16x4 res;
#pragma unroll
    for (int e = 0; e < 4; ++e) res[e] = (__bf16)(acc[j][e] * inv);
    *(bf16x4*)((__bf16*)a.out + orow * D + d4 * 4) = res;
    if (a.lse && d4 == 0) a.lse[orow] = row_m[rl];
  }
}

template <int D, int KT>
hipError_t launch(const AttnArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((tree_attn_bf16_kernel<D, KT>), dim3(tree_attn_bf16_grid(a)), dim3(kAttnThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

int tree_attn_bf16_grid(const AttnArgs& a) {
  const int unit_rounds = (a.units + 7) / 8;
  return 8 * unit_rounds * a.splits * a.row_groups;
}

hipError_t launch_tree_attn_bf16(const AttnArgs& a, hipStream_t stream) {
  if (a.D == 128) return a.key_tile == 128 ? launch<128, 128>(a, stream) : launch<128, 64>(a, stream);
  if (a.D == 64) return a.key_tile == 128 ? launch<64, 128>(a, stream) : launch<64, 64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace dreams

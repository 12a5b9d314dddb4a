// Tree-masked verification attention for the bandwidth-bound regime (a few query rows per KV head, as in
// tree verification of a batch of sequences): bf16 inputs, fp32 accumulation on the matrix cores.
//
// What is computed (the paper's Section 3.2 attention matrix applied to the target's verification pass of
// Section 2): for every tree node i of every query head, softmax(scale * q_i . k_j) v_j over the committed
// prefix slots and the slots of node i's ancestors-or-self.
//
// Work decomposition
//   * A workgroup owns RB*16 query rows of one KV head (rows of the G query heads sharing it are packed:
//     row r -> head r / T, node r % T) and one contiguous piece of that head's key axis.  Pieces come from
//     the host's bound on the key count, so the first loads need nothing from the device.
//   * Its W waves split the piece's keys: wave w handles 32-key steps w, w + W, ... for all of the
//     workgroup's rows, so each K/V byte is read once and used by every row, and waves never wait on each
//     other inside the loop.
//   * Per step a wave copies the 32 K rows and 32 V rows straight from global memory into its own LDS
//     buffer (global_load_lds_dwordx4: no registers in between, two buffers so the next step is in flight
//     while this one is computed).  Each lane fetches the source chunk that lands where the XOR-swizzled
//     layout wants it, which makes both operand reads below bank-conflict free:
//       S^T = K Q^T        v_mfma_f32_16x16x32_bf16, K rows as the A operand (16-byte LDS reads)
//       online softmax     per query row; each lane holds one row's scores, 4-way cross-lane reductions
//       O^T += V^T P^T     A operand read with ds_read_b64_tr_b16 (a 4 x 16 transposing LDS read); the
//                          probabilities are already in B-operand layout, so they never leave registers.
//     The copies are issued with inline assembly so that their completion is waited for explicitly and
//     exactly (the compiler would otherwise drain every outstanding copy before any LDS read).
//   * At the end the waves' (max, sum, accumulator) states are merged through LDS.  With several pieces per
//     (KV head, row group), each workgroup publishes its state with device-scope stores and bumps an
//     arrival counter; the last arrival merges the pieces in piece order (reproducible bit for bit).
//   * Workgroup ids are remapped so that all workgroups of one (sequence, KV head) run on the same XCD
//     (consecutive ids are dealt round-robin over the 8 XCDs); row groups reading the same keys then share
//     them in that XCD's L2.
#include "kernels.h"

#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kStep = 32;  // keys per step
constexpr int kBufs = 2;   // LDS step buffers per wave
constexpr float kLazyLog2 = 8.0f;  // slack of the running maximum, log2 units

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(lds_void*)p; }

// One wave-wide copy of 64 x 16 bytes from global memory into LDS: lane l's 16 bytes land at LDS byte
// address m0 + 16*l.  m0 must be wave-uniform.
__device__ __forceinline__ void copy_to_lds(uint32_t m0, const void* src) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(m0), "v"(src) : "memory", "m0");
}
// Same, addressed as SGPR base + per-lane 32-bit offset + immediate.
template <int IMM>
__device__ __forceinline__ void copy_to_lds_s(uint32_t m0, const void* sbase, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 offset:%3" ::"s"(m0), "v"(voff), "s"(sbase),
               "n"(IMM) : "memory", "m0");
}
// Waits for these copies, expressed as "at most N of this wave's vector-memory operations outstanding".
template <int N>
__device__ __forceinline__ void wait_copies() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }
// All of this wave's LDS reads have returned (the buffer they read may now be overwritten by a copy).
__device__ __forceinline__ void wait_lds_reads() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// LDS step buffer of one wave: 32 K rows then 32 V rows of D bf16, unpadded; the 16-byte chunk c of row r sits
// at position c ^ swz(r), which spreads the 16 rows one operand read touches over distinct banks.
template <int D>
struct Tile {
  static constexpr int ROW = D * 2;             // bytes per row
  static constexpr int CPR = D / 8;             // 16-byte chunks per row
  static constexpr int RPL = 256 / ROW;         // rows per 256-byte bank line
  static constexpr int HALF = kStep * ROW;      // bytes of the K (or V) part
  static constexpr int BYTES = 2 * HALF;
  static constexpr int COPIES = HALF / 1024;    // wave-wide 1 KB copies per part
  __device__ static __forceinline__ int swz(int r) { return (r / RPL) % CPR; }
  __device__ static __forceinline__ int off(int r, int c) { return r * ROW + ((c ^ swz(r)) << 4); }
};

template <int D, int RB, int W>
__global__ __launch_bounds__(64 * W) void tree_attn_stream_kernel(AttnArgs a) {
  constexpr int NT = 64 * W;
  constexpr int R = RB * 16;            // query rows per workgroup
  constexpr int DS = D / 32;            // k-steps of S^T = K Q^T
  constexpr int DB = D / 16;            // 16-column blocks of O^T
  using TL = Tile<D>;
  constexpr int CPS = 2 * TL::COPIES;   // wave-wide copies per step

  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  __shared__ uint64_t anc_lds[2 * kMaxNodes];
  __shared__ int par_lds[kMaxNodes];
  __shared__ int last_flag;

  // ---- work item
  const int n = blockIdx.x;
  const int xcd = n & 7, slot = n >> 3;
  const int per_unit = a.splits * a.row_groups;
  const int u = xcd + 8 * (slot / per_unit);
  if (u >= a.units) return;
  const int within = slot - (slot / per_unit) * per_unit;
  const int split = within / a.row_groups;
  const int rg = within - split * a.row_groups;
  const int b = u / a.Hkv, g = u - b * a.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, quad = lane >> 4, col = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T;

  // ---- this workgroup's piece of the key axis (from the host's bound) and this wave's steps in it
  int piece = (a.max_keys + a.splits - 1) / a.splits;
  piece = (piece + kStep - 1) / kStep * kStep;
  const int k_begin = split * piece;
  const __bf16* kbase = (const __bf16*)a.k + (size_t)u * a.S_cap * D;
  const __bf16* vbase = (const __bf16*)a.v + (size_t)u * a.S_cap * D;
  unsigned char* wtile = smem + wave * kBufs * TL::BYTES;
  const uint32_t wtile_lds = __builtin_amdgcn_readfirstlane(lds_addr(wtile));

  // Copy step `idx` of this wave into buffer `buf`: LDS byte j*1024 + 16*lane of a part holds row
  // r = (j*1024 + 16*lane) / ROW at position p = lane % CPR, i.e. global chunk p ^ swz(r) of that row.
  // The swizzle repeats every 16 rows, so OFFS per-lane offsets address all of a step's copies from two
  // per-step scalar bases (row 0 and row 16 of the step).
  static_assert(TL::COPIES == 8 || TL::COPIES == 4, "copy layout");
  constexpr int OFFS = TL::COPIES / 2;                 // distinct per-lane offsets
  uint32_t coff[OFFS];
#pragma unroll
  for (int j = 0; j < OFFS; ++j) {
    const int e = j * 64 + lane;
    const int r = e / TL::CPR, p = e - r * TL::CPR;
    coff[j] = (uint32_t)(r * TL::ROW + ((p ^ TL::swz(r)) << 4));
  }
  static_assert(16 * TL::ROW == OFFS * 1024 && (16 / TL::RPL) % TL::CPR == 0, "swizzle repeats every 16 rows");
  auto issue_step = [&](int idx, int buf) {
    const int key0 = k_begin + (wave + idx * W) * kStep;
    const uint32_t dst = wtile_lds + buf * TL::BYTES;
    if (key0 + kStep <= a.S_cap) {
      const unsigned char* ks = (const unsigned char*)kbase + (size_t)key0 * TL::ROW;
      const unsigned char* vs = (const unsigned char*)vbase + (size_t)key0 * TL::ROW;
#pragma unroll
      for (int j = 0; j < OFFS; ++j) {
        copy_to_lds_s<0>(dst + j * 1024, ks, coff[j]);
        copy_to_lds_s<0>(dst + TL::HALF + j * 1024, vs, coff[j]);
        copy_to_lds_s<0>(dst + (j + OFFS) * 1024, ks + OFFS * 1024, coff[j]);
        copy_to_lds_s<0>(dst + TL::HALF + (j + OFFS) * 1024, vs + OFFS * 1024, coff[j]);
      }
    } else {  // a step reaching past the cache capacity: clamp row by row
#pragma unroll
      for (int j = 0; j < TL::COPIES; ++j) {
        const int e = j * 64 + lane;
        const int r = e / TL::CPR, p = e - r * TL::CPR;
        const int key = min(key0 + r, a.S_cap - 1);
        const size_t src = (size_t)key * D + ((p ^ TL::swz(r)) << 3);
        copy_to_lds(dst + j * 1024, kbase + src);
        copy_to_lds(dst + TL::HALF + j * 1024, vbase + src);
      }
    }
  };
  issue_step(0, 0);   // in flight while the prologue runs

  // ---- prologue: prefix length, parents (one parallel round trip), ancestor sets in LDS, queries
  int L = a.kv_len[b];
  L = L < 0 ? 0 : (L > a.S_cap - T ? a.S_cap - T : L);
  const int N = L + T;
  if (a.mask) {
    if (tid < T) {
      const int Wm = (T + 63) / 64;
      const uint64_t* mr = a.mask + ((size_t)b * T + tid) * Wm;
      anc_lds[2 * tid] = mr[0];
      anc_lds[2 * tid + 1] = Wm > 1 ? mr[1] : 0;
    }
  } else {
    if (tid < T) par_lds[tid] = a.parent[(size_t)b * T + tid];
    __syncthreads();
    if (tid < T) {
      uint64_t m0 = 0, m1 = 0;
      int j = tid;
      for (int step = 0; step <= T && j >= 0; ++step) {
        if (j < 64) m0 |= 1ull << j; else m1 |= 1ull << (j - 64);
        const int p = par_lds[j];
        if (p >= j) break;  // not a valid parent: the walk ends here
        j = p;
      }
      anc_lds[2 * tid] = m0;
      anc_lds[2 * tid + 1] = m1;
    }
  }
  __syncthreads();

  const int rows_total = a.G * T;
  bf16x8 qf[RB][DS];
  uint64_t anc0[RB], anc1[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = rg * R + rb * 16 + col;
    const bool ok = row < rows_total;
    const int hg = ok ? row / T : 0;
    const int node = ok ? row - hg * T : 0;
    const __bf16* qrow = (const __bf16*)a.q + (((size_t)b * a.Hq + g * a.G + hg) * T + node) * D;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      if (ok) {
        qf[rb][s] = *(const bf16x8*)(qrow + s * 32 + quad * 8);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[rb][s][e] = (__bf16)0.0f;
      }
    }
    anc0[rb] = anc_lds[2 * node];
    anc1[rb] = anc_lds[2 * node + 1];
  }

  f32x4 o[RB][DB];
  float m_run[RB], l_run[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int d = 0; d < DB; ++d) o[rb][d] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[rb] = -INFINITY;
    l_run[rb] = 0.f;
  }

  // the last piece runs to this sequence's true end, whatever the host's bound said
  const int k_end = split == a.splits - 1 ? N : min(N, k_begin + piece);
  const int nsteps_piece = k_end > k_begin ? (k_end - k_begin + kStep - 1) / kStep : 0;
  const int nsteps = nsteps_piece > wave ? (nsteps_piece - wave + W - 1) / W : 0;

  // The prologue's own loads (queries, lengths, parents) are complete here; saying so with a wait the
  // compiler can see keeps it from draining the in-flight step copies at the first use inside the loop.
  wait_vector_memory();

  const int ka_row = (col & 3) * 4 + (col >> 2);       // A row m holds key kb*16 + (m%4)*4 + m/4
  const int tr_row = (col >> 2) * 4 + quad;            // transposed read: 4 keys j*4+quad, 16 columns
  const int tr_c = (col & 3) >> 1, tr_half = (col & 1) * 8;

  for (int it = 0; it < nsteps; ++it) {
    const int buf = it & 1;
    const int key0 = k_begin + (wave + it * W) * kStep;
    // the other buffer was last read by the previous step: finish those reads, refill it one step ahead,
    // then wait for this step's copies (everything but the CPS just issued)
    wait_lds_reads();
    if (it + 1 < nsteps) {
      issue_step(it + 1, buf ^ 1);
      wait_copies<CPS>();
    } else {
      wait_copies<0>();
    }
    unsigned char* tile = wtile + buf * TL::BYTES;
    const unsigned char* vt = tile + TL::HALF;
    if (key0 + kStep > N) {
      // rows at or past the sequence end hold whatever the cache had there: zero their values so that no
      // bit pattern can reach the value product (their keys are masked below)
      const int r = lane >> 1, c0 = (lane & 1) * (TL::CPR / 2);
      if (key0 + r >= N) {
#pragma unroll
        for (int c = 0; c < TL::CPR / 2; ++c) *(u32x4*)(tile + TL::HALF + TL::off(r, c0 + c)) = u32x4{0u, 0u, 0u, 0u};
      }
      __builtin_amdgcn_wave_barrier();
    }

    // S^T blocks kb = 0, 1: element e of a lane in quad q is key kb*16 + e*4 + q, row col
    f32x4 s[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) s[rb][0] = s[rb][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    bf16x8 kf[2][DS];   // all K fragments of the step first, so their LDS latencies overlap
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[kb][ds] = *(const bf16x8*)(tile + TL::off(kb * 16 + ka_row, ds * 4 + quad));
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          s[rb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kb][ds], qf[rb][ds], s[rb][kb], 0, 0, 0);

    // scale to log2 units; only steps that reach the tree slots or the piece end need the mask
    const bool masked = key0 + kStep > L || key0 + kStep > k_end;
    bf16x8 pb[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float lmax = -INFINITY;   // this lane's maximum over its 8 keys of the row
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float x = s[rb][kb][e] * a.scale_log2;
          if (masked) {
            const int key = key0 + kb * 16 + e * 4 + quad;
            const int j = key - L;                       // tree node of a key past the prefix
            const uint64_t word = j < 64 ? anc0[rb] : anc1[rb];
            const bool anc = ((word >> (j & 63)) & 1ull) != 0;
            const bool vis = (key < k_end) & ((key < L) | anc);
            x = vis ? x : -INFINITY;
          }
          s[rb][kb][e] = x;
          lmax = fmaxf(lmax, x);
        }
      }
      // The reference maximum m only moves when some score exceeds it by more than 2^8 (the exponentials
      // then stay <= 256, and softmax does not depend on the reference), which after the first steps is
      // rare: in the common case no cross-lane reduction and no rescale happen at all.
      if (__any(lmax > m_run[rb] + kLazyLog2)) {
        float tmax = fmaxf(lmax, __shfl_xor(lmax, 16));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        if (tmax > m_run[rb] + kLazyLog2) {
          const float alpha = m_run[rb] == -INFINITY ? 0.f : fast_exp2(m_run[rb] - tmax);
          m_run[rb] = tmax;
          l_run[rb] *= alpha;
#pragma unroll
          for (int d = 0; d < DB; ++d) o[rb][d] *= alpha;
        }
      }
      const float m_use = m_run[rb] == -INFINITY ? 0.f : m_run[rb];
      float psum = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = fast_exp2(s[rb][kb][e] - m_use);
          psum += p;
          pb[rb][kb * 4 + e] = (__bf16)p;
        }
      }
      l_run[rb] += psum;
    }

    // O^T[d][row] += sum over the 32 keys of V[key][d] P[row][key]; k-slots 0..3 = keys j*4+quad,
    // 4..7 = keys 16+j*4+quad, exactly the keys whose probabilities this lane holds in pb.
#pragma unroll
    for (int d = 0; d < DB; ++d) {
      const int c = d * 2 + tr_c;
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(vt + TL::off(tr_row, c) + tr_half));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(vt + TL::off(16 + tr_row, c) + tr_half));
      bf16x8 va;
      const bf16x4 lo_b = __builtin_bit_cast(bf16x4, lo), hi_b = __builtin_bit_cast(bf16x4, hi);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        va[e] = lo_b[e];
        va[4 + e] = hi_b[e];
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        o[rb][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[rb], o[rb][d], 0, 0, 0);
    }
  }
  wait_copies<0>();   // the entry copy of a wave without steps lands before LDS is reused

  // ---- merge the W waves' states through LDS
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    l_run[rb] += __shfl_xor(l_run[rb], 16);
    l_run[rb] += __shfl_xor(l_run[rb], 32);
  }
  __syncthreads();
  float* o_lds = (float*)smem;                       // [W][R][D]
  float2* ml_lds = (float2*)(o_lds + W * R * D);     // [W][R]
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = rb * 16 + col;
#pragma unroll
    for (int d = 0; d < DB; ++d) *(f32x4*)(o_lds + ((size_t)wave * R + row) * D + d * 16 + quad * 4) = o[rb][d];
    if (quad == 0) ml_lds[wave * R + row] = make_float2(m_run[rb], l_run[rb]);
  }
  __syncthreads();

  constexpr int D4 = D / 4;
  constexpr int ITEMS = R * D4;
  const int rows_here = min(R, rows_total - rg * R);
  const bool single = a.splits == 1;
  const size_t pset = (size_t)u * a.row_groups + rg;
  for (int item = tid; item < ITEMS; item += NT) {
    const int row = item / D4, d4 = item - row * D4;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < W; ++w) M = fmaxf(M, ml_lds[w * R + row].x);
    float lsum = 0.f;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const float2 ml = ml_lds[w * R + row];
      const float wt = ml.x == -INFINITY ? 0.f : fast_exp2(ml.x - M);
      lsum += wt * ml.y;
      acc += wt * *(const f32x4*)(o_lds + ((size_t)w * R + row) * D + d4 * 4);
    }
    if (single) {
      if (row < rows_here) {
        const int r = rg * R + row;
        const int hg = r / T, nd = r - hg * T;
        const size_t orow = ((size_t)b * a.Hq + g * a.G + hg) * T + nd;
        const float inv = lsum > 0.f ? 1.0f / lsum : 0.f;
        bf16x4 res;
#pragma unroll
        for (int e = 0; e < 4; ++e) res[e] = (__bf16)(acc[e] * inv);
        *(bf16x4*)((__bf16*)a.out + orow * D + d4 * 4) = res;
        if (a.lse && d4 == 0) a.lse[orow] = lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
      }
    } else {
      const size_t pr = (pset * a.splits + split) * R + row;
#pragma unroll
      for (int e = 0; e < 4; ++e) store_coherent(a.part_acc + pr * D + d4 * 4 + e, acc[e]);
      if (d4 == 0) {
        store_coherent(a.part_ml + 2 * pr, M);
        store_coherent(a.part_ml + 2 * pr + 1, lsum);
      }
    }
  }
  if (single) return;

  // ---- publish, count arrivals, the last arrival merges the pieces
  wait_vector_memory();   // this thread's device-scope stores have completed
  __syncthreads();
  if (tid == 0) last_flag = arrive_last(&a.counters[pset], (uint32_t)a.splits);
  __syncthreads();
  if (!last_flag) return;
  if (tid == 0) reset_counter(&a.counters[pset]);

  const int S = a.splits;
  float2* w_lds = ml_lds;                             // [S][R] weights and sums (S <= kAttnMaxSplits)
  float* fin = (float*)(w_lds + kAttnMaxSplits * R);  // [R] 1/l, [R] lse
  {
    // all pieces' (m, l) in one round trip, loads issued before any is used
    constexpr int PER = (kAttnMaxSplits * R + NT - 1) / NT;
    float mv[PER], lv[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + k * NT;
      const int ec = e < S * R ? e : 0;
      const size_t pr = (pset * S + ec / R) * R + ec % R;
      mv[k] = load_coherent(a.part_ml + 2 * pr);
      lv[k] = load_coherent(a.part_ml + 2 * pr + 1);
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + k * NT;
      if (e < S * R) w_lds[e] = make_float2(mv[k], lv[k]);
    }
  }
  __syncthreads();
  if (tid < R) {
    float M = -INFINITY;
    for (int sp = 0; sp < S; ++sp) M = fmaxf(M, w_lds[sp * R + tid].x);
    float lsum = 0.f;
    for (int sp = 0; sp < S; ++sp) {
      const float2 v = w_lds[sp * R + tid];
      const float wt = v.x == -INFINITY ? 0.f : fast_exp2(v.x - M);
      lsum += wt * v.y;
      w_lds[sp * R + tid].x = wt;
    }
    fin[tid] = lsum > 0.f ? 1.0f / lsum : 0.f;
    fin[R + tid] = lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
  }
  __syncthreads();

  // every thread owns IPT (row, 4-column) items; pieces are read four at a time, all loads of a group
  // issued before any is used
  constexpr int IPT = ITEMS / NT;
  static_assert(IPT * NT == ITEMS, "items must split evenly");
  f32x4 acc[IPT];
#pragma unroll
  for (int k = 0; k < IPT; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int sp0 = 0; sp0 < S; sp0 += 4) {
    float x[4][IPT][4];
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int sp = min(sp0 + q4, S - 1);
#pragma unroll
      for (int k = 0; k < IPT; ++k) {
        const int item = tid + k * NT;
        const int row = item / D4, d4 = item - row * D4;
        const float* src = a.part_acc + ((pset * S + sp) * R + row) * D + d4 * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[q4][k][e] = load_coherent(src + e);
      }
    }
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      if (sp0 + q4 < S) {
#pragma unroll
        for (int k = 0; k < IPT; ++k) {
          const int row = (tid + k * NT) / D4;
          const float wt = w_lds[(sp0 + q4) * R + row].x;
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[k][e] += wt * x[q4][k][e];
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < IPT; ++k) {
    const int item = tid + k * NT;
    const int row = item / D4, d4 = item - row * D4;
    if (row >= rows_here) continue;
    const int r = rg * R + row;
    const int hg = r / T, nd = r - hg * T;
    const size_t orow = ((size_t)b * a.Hq + g * a.G + hg) * T + nd;
    bf16x4 res;
#pragma unroll
    for (int e = 0; e < 4; ++e) res[e] = (__bf16)(acc[k][e] * fin[row]);
    *(bf16x4*)((__bf16*)a.out + orow * D + d4 * 4) = res;
    if (a.lse && d4 == 0) a.lse[orow] = fin[R + row];
  }
}

// Dynamic LDS: the waves' step buffers during the loop; afterwards the waves' states, then the pieces'
// weights.
template <int D, int RB, int W>
constexpr size_t stream_lds_bytes() {
  constexpr size_t tiles = (size_t)W * kBufs * Tile<D>::BYTES;
  constexpr size_t states = (size_t)W * RB * 16 * D * 4 + (size_t)W * RB * 16 * 8;
  constexpr size_t pieces = (size_t)W * RB * 16 * D * 4 + (size_t)kAttnMaxSplits * RB * 16 * 8 + 2 * RB * 16 * 4;
  constexpr size_t m = tiles > states ? tiles : states;
  return m > pieces ? m : pieces;
}

template <int D, int RB, int W>
hipError_t launch(const AttnArgs& a, hipStream_t stream) {
  constexpr size_t lds = stream_lds_bytes<D, RB, W>();
  static_assert(lds + 2 * kMaxNodes * 8 + kMaxNodes * 4 + 64 <= 160 * 1024, "LDS budget");
  auto kern = tree_attn_stream_kernel<D, RB, W>;
  static bool configured = false;
  if (!configured) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    configured = true;
  }
  const unsigned units_rounded = (a.units + 7) / 8 * 8;
  const unsigned grid = units_rounded * (unsigned)(a.splits * a.row_groups);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * W), lds, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tree_attn_stream(const AttnArgs& a, hipStream_t stream) {
  if (a.D == 128) return launch<128, kStreamRows / 16, kStreamWaves>(a, stream);
  if (a.D == 64) return launch<64, kStreamRows / 16, kStreamWaves>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace dreams

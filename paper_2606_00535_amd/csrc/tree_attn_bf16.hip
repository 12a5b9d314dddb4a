// Tree-masked verification attention, bf16 inputs, fp32 accumulation on the matrix cores.
//
// What is computed (the paper's Section 3.2 attention mask applied to the target's verification pass of
// Section 2): for every tree node i of every query head, softmax(scale * q_i . k_j) v_j over the committed
// prefix slots and the slots of node i's ancestors-or-self.
//
// Work decomposition
//   * A workgroup of W waves (4 or 8) owns R query rows of one KV head (the rows of the G query heads sharing it
//     are packed: row r -> head r / T, node r % T, which is also their order in memory) and one piece of that
//     head's key axis.  Each wave owns 16*RB rows of its key group (below) for every key the group takes, and
//     every K/V byte the workgroup reads serves all of its rows.  The 64- and 128-row configurations take at
//     most half of a compute unit's LDS and registers (WPC = 2), so two workgroups share a compute unit.
//   * The pieces are cut from the host's bound on the key count (the first copies need nothing from the
//     device), or, with several sequences, from each sequence's own count.
//   * K/V stream through a ring of NST step slots in LDS (a step = 32 keys: 32 K rows then 32 V rows).  The
//     waves copy their share of every step straight from global memory into LDS (global_load_lds_dwordx4: no
//     registers in between), a whole ring ahead.  One barrier per super-step hands a landed step to all waves;
//     in the pipelined loop a second one frees the slots every wave has read, which are refilled at once.  The
//     copies are issued with inline assembly and waited for by exact count; nothing else in the kernel loads
//     through the vector memory path before the epilogue, so the compiler never inserts a wait that would
//     drain the ring.
//   * Each lane fetches the source chunk that lands where an XOR-swizzled row layout wants it, which makes
//     both operand reads below bank-conflict free:
//       S^T = K Q^T        v_mfma_f32_16x16x32_bf16, K rows as the A operand (16-byte LDS reads)
//       online softmax     per query row; each lane holds one row's scores, 4-way cross-lane reductions
//       O^T += V^T P^T     A operand read with ds_read_b64_tr_b16 (a 4 x 16 transposing LDS read); the
//                          probabilities are already in B-operand layout, so they never leave registers.
//   * Waves are arranged as KW key groups of W/KW waves: the groups take alternate steps (group k the steps
//     k, k+KW, ...), so a wave's operand reads serve as many rows as possible; the groups' (max, sum,
//     accumulator) states are merged through LDS at the end.
//   * With several pieces per (sequence, KV head, row group) -- a set -- each piece stores its rows' output
//     normalised by their softmax sum (bf16) and their (max, sum) to the workspace and arrives on the set's
//     counter.  A piece whose set has fully started waits for every arrival and merges its own slice of the
//     rows; a piece that finds its set not yet fully started leaves its slice to the piece that started last,
//     which learnt at its start which pieces had already arrived.  So a wait is only ever for a running piece.
//     The merge goes in piece order, so the result does not depend on which piece came last.  All pieces of
//     a set run on one XCD (below), so their rows are exchanged through that XCD's L2: plain stores, no
//     device-scope write-through, no second launch.  Each piece adds its XCD id (and its square) to the set's
//     counter when it starts, and a merging piece checks that they all match its own.
//   * Workgroup ids are remapped so that all workgroups of one (sequence, KV head) share blockIdx % 8:
//     consecutive ids of a dispatch are dealt round-robin over the 8 XCDs, so these run on one XCD (which one
//     takes id 0 varies between dispatches), and row groups reading the same keys share them in its L2.
#include "kernels.h"

#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kStep = 32;          // keys per step
constexpr float kLazyLog2 = 8.0f;  // slack of the running maximum, log2 units

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Attention entropy from a row's softmax state.  With scores z in log2 units, a reference m, l = sum 2^(z-m)
// and e = sum 2^(z-m) (z-m), the row's probabilities are 2^(z-m)/l and its entropy (nats) is
// ln2 * (log2 l - e/l).  Re-referencing a state to M (weight w = 2^(m-M)) turns e into w (e + (m-M) l).
__device__ __forceinline__ float ent_term(float w, float e, float m, float M, float l) {
  return w == 0.f ? 0.f : w * fmaf(m - M, l, e);
}
__device__ __forceinline__ float row_entropy(float l, float e) {
  return l > 0.f ? 0.69314718055994530942f * (__log2f(l) - e / l) : 0.f;
}

typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(lds_void*)p; }

// Wave-wide copies from global memory into LDS.  m0 (wave-uniform) is the LDS byte address of lane 0's
// data; lane l's data lands at m0 + 16*l (dwordx4) or m0 + 4*l (dword).  The 16-byte copies move data that
// is read exactly once (queries, keys, values) and carry the non-temporal hint.
__device__ __forceinline__ void copy16_to_lds(uint32_t m0, const void* src) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off nt" ::"s"(m0), "v"(src) : "memory");
}
// Same, addressed as a wave-uniform base plus a per-lane 32-bit byte offset.
__device__ __forceinline__ void copy16_to_lds(uint32_t m0, const void* sbase, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 nt" ::"s"(m0), "v"(voff), "s"(sbase)
               : "memory");
}
__device__ __forceinline__ void copy4_to_lds(uint32_t m0, const void* src) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off" ::"s"(m0), "v"(src) : "memory");
}
// At most N of this wave's vector-memory operations still outstanding (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// wait_vm<PER * k> for a run-time k in [0, K]
template <int PER, int K>
__device__ __forceinline__ void wait_vm_steps(int k) {
  if constexpr (K > 0) {
    if (k >= K) {
      wait_vm<PER * K>();
      return;
    }
    wait_vm_steps<PER, K - 1>(k);
  } else {
    wait_vm<0>();
  }
}
// Workgroup barrier after this wave's LDS reads and writes have completed; outstanding copies stay in
// flight (a __syncthreads() would also wait for them).  The wait is the compiler's own instruction
// (vmcnt and expcnt at their maxima, lgkmcnt 0), so its wait-count bookkeeping knows that every LDS read
// issued before the barrier has returned.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Row layout in LDS: rows of D bf16, unpadded; the 16-byte chunk c of row r sits at position c ^ swz(r),
// which spreads the 16 rows one operand read touches over distinct banks.  The swizzle repeats every 16
// rows.  A step slot holds 32 K rows then 32 V rows; the query rows use the same layout.
template <int D>
struct Rows {
  static constexpr int ROW = D * 2;           // bytes per row
  static constexpr int CPR = D / 8;           // 16-byte chunks per row
  static constexpr int RPL = 256 / ROW;       // rows per 256-byte bank line
  static constexpr int HALF = kStep * ROW;    // bytes of the K (or V) part of a step
  static constexpr int SLOT = 2 * HALF;       // bytes of a step
  static constexpr int C16 = 16 * ROW / 1024; // wave-wide 1 KB copies per 16 rows
  // D = 128 (one row per 256-byte bank line): gfx950 serves a 16-byte read (ds_read_b128) in groups of lanes
  // and a transposing 8-byte read (ds_read_b64_tr_b16) in two halves of 32 lanes over 64 banks.  The key
  // reads touch rows (m%4)*4 + m/4 at one chunk, the value reads rows 4j+q, q in {0,1} (or {2,3}), at an
  // aligned pair of chunks; swz(r) = 4*((r/4)%4) + 2*(r%2) + 1 puts both on distinct banks (measured: 213 and
  // 165 B/clk per compute unit, against 126 and 122 with r % 16).  D = 64: two rows per bank line.
  __device__ static __forceinline__ int swz(int r) {
    if constexpr (D == 128) return ((r >> 2) & 3) * 4 + (r & 1) * 2 + 1;
    return (r / RPL) % CPR;
  }
  __device__ static __forceinline__ int off(int r, int c) { return r * ROW + ((c ^ swz(r)) << 4); }
};

// Merge of a set's pieces for rows [r0, r0 + nrows) of the set, in piece order (so the result does not
// depend on which piece finished last): out = sum_s w_s l_s o_s / sum_s w_s l_s, w_s = 2^(m_s - max_s m_s).
// Every piece's rows come from this XCD's L2 (not from this compute unit's L1, which has never held them):
// non-temporal 16-byte loads, a row's pieces side by side, whole 128-byte lines.  The loads are issued
// unconditionally (addresses clamped into the set), so that all of them are in flight together (loads under a
// branch are each waited for before the branch joins); waves with no row of the slice skip it.  Rows at or
// past rows_valid are not written.  good = false writes NaN rows (a failed wait).
template <int D, int W, bool ENT>
__device__ __forceinline__ void merge_pieces(const AttnArgs& a, size_t prow0, int R, __bf16* out_rows, float* lse_rows,
                                             float* ent_rows, int rows_valid, int r0, int nrows, bool good) {
  constexpr int CPR = D / 8;
  constexpr int PCH = 8;    // pieces per batch of loads
  typedef __bf16 bf16x8m __attribute__((ext_vector_type(8)));
  const int S = a.splits;
  const int items = nrows * CPR;
  const int wave = (int)threadIdx.x >> 6;
  for (int base = 0; base < items; base += 64 * W) {
    if (base + 64 * wave >= items) break;   // (wave-uniform) nothing left for this wave
    const int item = base + (int)threadIdx.x;
    const int ch = item % CPR;
    const bool live = item < items && r0 + item / CPR < rows_valid;
    const int rl = min(r0 + item / CPR, R - 1);   // (a dead item's loads stay inside the set)
    float M = -INFINITY, lsum = 0.f, esum = 0.f;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int s0 = 0; s0 < S; s0 += PCH) {
      f32x2 ml[PCH];
      float ev[PCH];
      bf16x8m x[PCH];
#pragma unroll
      for (int k = 0; k < PCH; ++k) {
        const size_t pr = prow0 + (size_t)min(s0 + k, S - 1) * R + rl;
        ml[k] = __builtin_nontemporal_load((const f32x2*)(a.part_ml + 2 * pr));
        ev[k] = ENT ? __builtin_nontemporal_load(a.part_e + pr) : 0.f;
        x[k] = __builtin_nontemporal_load((const bf16x8m*)(a.part_o + pr * D + ch * 8));
      }
      float Mn = M;
#pragma unroll
      for (int k = 0; k < PCH; ++k)
        if (s0 + k < S) Mn = fmaxf(Mn, ml[k].x);
      const float scale_old = M == -INFINITY ? 0.f : fast_exp2(M - Mn);
      if (ENT) esum = ent_term(scale_old, esum, M, Mn, lsum);
      lsum *= scale_old;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] *= scale_old;
#pragma unroll
      for (int k = 0; k < PCH; ++k) {
        const float w = (s0 + k >= S || ml[k].x == -INFINITY) ? 0.f : fast_exp2(ml[k].x - Mn);
        if (ENT) esum += ent_term(w, ev[k], ml[k].x, Mn, ml[k].y);
        const float wl = w * ml[k].y;
        lsum += wl;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(wl, (float)x[k][e], acc[e]);
      }
      M = Mn;
    }
    if (!live) continue;
    const float inv = !good ? NAN : lsum > 0.f ? 1.0f / lsum : 0.f;
    bf16x8m res;
#pragma unroll
    for (int e = 0; e < 8; ++e) res[e] = (__bf16)(acc[e] * inv);
    *(bf16x8m*)(out_rows + (size_t)rl * D + ch * 8) = res;
    if (ch == 0) {
      if (lse_rows) lse_rows[rl] = !good ? NAN : lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
      if (ENT) ent_rows[rl] = !good ? NAN : row_entropy(lsum, esum);
    }
  }
}

// LDS of a workgroup: the ring, the query rows when they sit beside it, the ancestor sets and the tree as
// copied (static), and a few words; WPC workgroups share a compute unit's 160 KB.
template <int D, int NST, int WPC>
constexpr bool q_beside_ring(int R) {
  return (size_t)NST * Rows<D>::SLOT + (size_t)R * D * 2 + 4 * kMaxNodes * 8 + 64 <= 160 * 1024 / WPC;
}
template <int D, int NST, int WPC>
constexpr size_t dynamic_lds(int R) {
  return (size_t)NST * Rows<D>::SLOT + (q_beside_ring<D, NST, WPC>(R) ? (size_t)R * D * 2 : 0);
}

// WPC: workgroups meant to share a compute unit (their waves share each SIMD, so the register budget is that
// of WPC * W / 4 waves per SIMD).
template <int D, int RB, int KW, int W, int NST, bool PIPE, bool ENT, int WPC>
__global__ __launch_bounds__(64 * W, WPC * W / 4) void tree_attn_bf16_kernel(AttnArgs a) {
  constexpr int WR = W / KW;          // waves per key group; each owns a different slice of the rows
  constexpr int RW = 16 * RB;         // query rows per wave
  constexpr int R = WR * RW;          // query rows per workgroup
  constexpr int DS = D / 32;          // k-steps of S^T = K Q^T
  constexpr int DB = D / 16;          // 16-column blocks of O^T
  using L = Rows<D>;
  constexpr int C16 = L::C16;         // wave-wide copies per 16 rows
  constexpr int NSS = NST / KW;       // ring slots in super-steps (KW consecutive steps, one per key group)
  // The query rows get an LDS region of their own beside the ring where it fits (so the first copies fill the
  // whole ring); otherwise they occupy the ring's last step slots until the prologue has read them.
  constexpr bool QSEP = q_beside_ring<D, NST, WPC>(R);
  constexpr int QSLOTS = QSEP ? 0 : (R * L::ROW + L::SLOT - 1) / L::SLOT;   // step slots the query rows occupy
  constexpr int QSS = (QSLOTS + KW - 1) / KW;                                // ... in super-steps
  constexpr int CPS = 4 * KW * C16 / W;   // copies per wave per super-step (4*KW blocks of 16 rows)
  constexpr int QB = R / 16;          // 16-row blocks of query rows, dealt to the waves round-robin
  static_assert(W % KW == 0 && (NST & (NST - 1)) == 0 && NSS > QSS && NSS >= 2, "ring layout");
  static_assert(CPS * W == 4 * KW * C16 && CPS >= 1 && (C16 % CPS == 0 || CPS % C16 == 0), "copy split");
  static_assert(16 * L::ROW == C16 * 1024 && (16 / L::RPL) % L::CPR == 0, "swizzle repeats every 16 rows");
  static_assert(NSS * CPS + ((QB + W - 1) / W) * C16 + 8 <= 63, "outstanding copies fit the counter");
  static_assert((size_t)(KW - 1) * R * D * 4 + (size_t)KW * R * 12 <= (size_t)NST * L::SLOT, "group states fit the ring");

  extern __shared__ __attribute__((aligned(1024))) unsigned char ring[];   // NST step slots (+ the query rows)
  __shared__ uint64_t anc_lds[2 * kMaxNodes];
  __shared__ uint64_t meta_lds[2 * kMaxNodes];   // the sequence's parents or tree mask rows, as copied
  __shared__ uint32_t merge_lds;                  // slices of the set's rows this workgroup merges
  __shared__ uint32_t good_lds;                   // 0: a wait gave up (the merged rows are written as NaN)

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
  const int kw = wave / WR, rh = wave - kw * WR;   // key group; row slice [rh*RW, rh*RW + RW)
  const int T = a.T;
  const int rows_total = a.G * T;
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(lds_addr(ring));
  const int kv_len_b = a.kv_len[b];   // issued before the copies below, ahead of their traffic

  // ---- this workgroup's piece of the key axis, planned from the host's bound on the key count, or (several
  // sequences of different lengths) from this sequence's own count, so that a short sequence's pieces are
  // shorter rather than its last piece nearly empty; the first copies then wait for its length
  int keys = a.max_keys;
  if (a.piece_by_len) keys = min(max(kv_len_b, 0), a.S_cap - T) + T;
  int piece = (keys + a.splits - 1) / a.splits;
  piece = (piece + kStep - 1) / kStep * kStep;
  const int k_begin = split * piece;
  const int k_end_plan = split == a.splits - 1 ? keys : min(keys, k_begin + piece);
  const int nplan = k_end_plan > k_begin ? (k_end_plan - k_begin + kStep - 1) / kStep : 0;
  const int nsp = (nplan + KW - 1) / KW;
  const unsigned char* kbase = (const unsigned char*)a.k + (size_t)u * a.S_cap * L::ROW;
  const unsigned char* vbase = (const unsigned char*)a.v + (size_t)u * a.S_cap * L::ROW;

  // Per-lane byte offsets of the copies of 16 consecutive rows: copy j, lane l brings row r = (j*1024 +
  // 16*l) / ROW, position p = l % CPR, i.e. the global chunk p ^ swz(r) of that row.
  uint32_t coff[C16];
#pragma unroll
  for (int j = 0; j < C16; ++j) {
    const int e = j * 64 + lane;
    const int r = e / L::CPR, p = e - r * L::CPR;
    coff[j] = (uint32_t)(r * L::ROW + ((p ^ L::swz(r)) << 4));
  }
  // A super-step is KW steps x (32 K rows + 32 V rows) = 4*KW blocks of 16 rows = 4*KW*C16 wave-wide 1 KB
  // copies; wave w issues copies w*CPS .. w*CPS + CPS - 1 (copy ci: block bi = ci / C16 -- step bi/4 of the
  // super-step, K or V part (bi/2)%2, rows 16*(bi%2).. -- and copy ci % C16 of that block), in groups of
  // GRP = min(CPS, C16) copies that share a block.
  constexpr int GRP = CPS < C16 ? CPS : C16;
  constexpr int NGRP = CPS / GRP;
  auto issue_group = [&](int jj, int t) {
    const uint32_t sbase = ring_lds + (jj & (NSS - 1)) * KW * L::SLOT;
    const int ci0 = wave * CPS + t * GRP;
    const int bi = ci0 / C16, j0 = ci0 - bi * C16;
    const int sis = bi >> 2, part = (bi >> 1) & 1, half = bi & 1;
    const int key0 = k_begin + (jj * KW + sis) * kStep + 16 * half;
    const unsigned char* pbase = part ? vbase : kbase;
    const uint32_t dst = sbase + sis * L::SLOT + part * L::HALF + half * C16 * 1024;
    if (key0 + 16 <= a.S_cap) {
      const unsigned char* src = pbase + (size_t)key0 * L::ROW;
#pragma unroll
      for (int j = 0; j < GRP; ++j) copy16_to_lds(dst + (j0 + j) * 1024, src, coff[j0 + j]);
    } else {  // rows past the cache capacity repeat its last row
#pragma unroll
      for (int j = 0; j < GRP; ++j) {
        const int r = ((j0 + j) * 64 + lane) / L::CPR;
        const int key = min(key0 + r, a.S_cap - 1);
        copy16_to_lds(dst + (j0 + j) * 1024, pbase + (size_t)key * L::ROW + (coff[j0 + j] - r * L::ROW));
      }
    }
  };
  auto issue_super = [&](int jj) {
#pragma unroll
    for (int t = 0; t < NGRP; ++t) issue_group(jj, t);
  };

  // ---- first copies: the query rows (into the last step slots), the tree (wave 0), then the ring
  const size_t qrow0 = ((size_t)b * a.Hq + (size_t)g * a.G) * T;   // row 0 of this KV head's query rows
  const unsigned char* qslab = QSEP ? ring + NST * L::SLOT : ring + (NST - QSLOTS) * L::SLOT;
#pragma unroll
  for (int qb = wave; qb < QB; qb += W) {
#pragma unroll
    for (int j = 0; j < C16; ++j) {
      const int r = (j * 64 + lane) / L::CPR;
      const int row = min(rg * R + qb * 16 + r, rows_total - 1);
      copy16_to_lds(lds_addr(qslab) + (qb * C16 + j) * 1024,
                    (const unsigned char*)a.q + (qrow0 + row) * L::ROW + (coff[j] - r * L::ROW));
    }
  }
  const int Wm = (T + 63) / 64;
  if (wave == 0) {
    const uint32_t mdst = lds_addr(meta_lds);
    if (a.mask) {
      const int nd = 2 * T * Wm;   // dwords of this sequence's mask rows
      const uint32_t* src = (const uint32_t*)(a.mask + (size_t)b * T * Wm);
      for (int c = 0; c * 64 < nd; ++c) copy4_to_lds(mdst + c * 256, src + min(c * 64 + lane, nd - 1));
    } else {
      const int32_t* src = a.parent + (size_t)b * T;
      for (int c = 0; c * 64 < T; ++c) copy4_to_lds(mdst + c * 256, src + min(c * 64 + lane, T - 1));
    }
  }
  const int fa = min(NSS - QSS, nsp);
  for (int j = 0; j < fa; ++j) issue_super(j);
  // This piece has started (the merge at the end relies on knowing that every piece of the set runs), on the
  // XCD it adds to the set's sums.  The counter's value before this start is kept (thread 0) until the
  // epilogue: the piece that starts last finds there the pieces that arrived before the whole set was running,
  // whose rows it then merges.
  unsigned long long start_old = 0;
  if (a.splits > 1 && tid == 0) {
    const unsigned long long x = xcd_id();
    start_old = __hip_atomic_fetch_add(a.set_ctr + ((size_t)u * a.row_groups + rg) * a.ctr_stride,
                                       1ull | (x << kCtrXcdSum) | ((x * x) << kCtrXcdSq), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  }

  // ---- prologue: prefix length, ancestor sets, queries (all overlapping the copies above)
  int Lp = kv_len_b;
  Lp = Lp < 0 ? 0 : (Lp > a.S_cap - T ? a.S_cap - T : Lp);
  const int N = Lp + T;
  // the last piece runs to this sequence's true end, whatever the host's bound said
  const int k_end = split == a.splits - 1 ? N : min(N, k_begin + piece);
  const int nact = k_end > k_begin ? (k_end - k_begin + kStep - 1) / kStep : 0;
  const int nsa = (nact + KW - 1) / KW;

  wait_vm_steps<CPS, NSS - QSS>(fa);   // this wave's query rows and the tree have landed
  barrier_lds();
  // Only a piece that reaches the tree slots consults ancestor sets (a step before them has key < L_b
  // everywhere, and a masked step past k_end hides its keys whatever the sets say).
  const bool need_anc = k_end > Lp;
  if (need_anc && tid < T) {
    uint64_t m0 = 0, m1 = 0;
    if (a.mask) {
      const uint64_t* mr = meta_lds + tid * Wm;
      m0 = mr[0];
      m1 = Wm > 1 ? mr[1] : 0;
    } else {
      const int* par = (const int*)meta_lds;
      int j = tid;
      for (int st = 0; st <= T && j >= 0; ++st) {
        if (j < 64) m0 |= 1ull << j; else m1 |= 1ull << (j - 64);
        const int p = par[j];
        if (p >= j) break;  // not a valid parent: the walk ends here
        j = p;
      }
    }
    anc_lds[2 * tid] = m0;
    anc_lds[2 * tid + 1] = m1;
  }
  bf16x8 qf[RB][DS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = *(const bf16x8*)(qslab + L::off(rh * RW + rb * 16 + col, ds * 4 + quad));
  // Scores are scaled by c = |scale| log2(e) > 0 inside the exponent (one fma per score); a negative scale
  // flips the sign of the queries instead (exact in bf16), a zero scale becomes the smallest normal float.
  const float c_scale = fmaxf(fabsf(a.scale_log2), 1.17549435e-38f);
  if (a.scale_log2 < 0.f) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, qf[rb][ds]) ^ 0x80008000u);
  }
  barrier_lds();   // ancestor sets written; every wave's query reads returned (their slots are reused next)
  uint64_t anc0[RB], anc1[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = min(rg * R + rh * RW + rb * 16 + col, rows_total - 1);
    const int node = row % T;
    anc0[rb] = need_anc ? anc_lds[2 * node] : 0;
    anc1[rb] = need_anc ? anc_lds[2 * node + 1] : 0;
  }
  // Ring depth: the pipelined loop frees a super-step's slots at the barrier that follows its operand reads,
  // so every slot can hold a copy in flight; the plain loop keeps one slot for the super-step being read.
  constexpr int AHEAD = PIPE ? NSS : NSS - 1;
  const int fb = max(fa, min(AHEAD, nsa));
  for (int j = fa; j < fb; ++j) issue_super(j);
  // super-steps issued by this wave once the refill of iteration js - 1 is out
  auto issued_by = [&](int js) { return max(fa, min(js + AHEAD, nsa)); };

  f32x4 o[RB][DB];
  float m_run[RB], l_run[RB];
  float e_run[RB];   // entropy term: sum of p * (z - m) over the keys so far (ENT only)
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int d = 0; d < DB; ++d) o[rb][d] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[rb] = -INFINITY;
    l_run[rb] = 0.f;
    e_run[rb] = 0.f;
  }

  const int ka_row = (col & 3) * 4 + (col >> 2);       // A row m holds key kb*16 + (m%4)*4 + m/4
  const int tr_row = (col >> 2) * 4 + quad;            // transposed read: 4 keys j*4+quad, 16 columns
  const int tr_c = (col & 3) >> 1, tr_half = (col & 1) * 8;

  // Key and value rows at or past the sequence end hold whatever the cache had there: the waves that copied
  // them zero them once their own copies have landed, so that no bit pattern (an infinity, a NaN) can reach
  // the products; their scores are then exactly the mask's -inf.
  auto zero_tail = [&](int jj) {
    unsigned char* sslot = ring + (jj & (NSS - 1)) * KW * L::SLOT;
#pragma unroll
    for (int t = 0; t < NGRP; ++t) {
      const int ci0 = wave * CPS + t * GRP;
      const int bi = ci0 / C16, j0 = ci0 - bi * C16;
      const int sis = bi >> 2, part = (bi >> 1) & 1, half = bi & 1;
      const int key0 = k_begin + (jj * KW + sis) * kStep;
      if (key0 + kStep > N) {
        // the rows this wave's copies brought: 64*GRP lanes' worth of 16-byte chunks, rows j0*1024/ROW ..
        constexpr int RPG = GRP * 1024 / L::ROW;   // rows per group of copies
        constexpr int LPR = 64 / RPG;              // lanes per row
        constexpr int PER = L::CPR / LPR;          // chunks per lane
        const int r = 16 * half + j0 * 1024 / L::ROW + lane / LPR;
        if (key0 + r >= N) {
          unsigned char* vrow = sslot + sis * L::SLOT + part * L::HALF + r * L::ROW;
#pragma unroll
          for (int c = 0; c < PER; ++c) *(u32x4*)(vrow + ((lane % LPR) * PER + c) * 16) = u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
  };

  // A step's operands: K fragments (A operand of S^T: A row m holds key kb*16 + (m%4)*4 + m/4) and V^T
  // fragments (A operand of O^T, transposing reads: lo = keys j*4+quad, hi = keys 16+j*4+quad, matching the
  // probabilities' slots).  All are issued together, so their LDS latencies overlap.
  struct Ops {
    bf16x8 kf[2][DS];
    s16x4 vlo[DB], vhi[DB];
  };
  auto read_ops = [&](Ops& op, int jj) {
    const unsigned char* tile = ring + (jj & (NSS - 1)) * KW * L::SLOT + kw * L::SLOT;
    const unsigned char* vt = tile + L::HALF;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) op.kf[kb][ds] = *(const bf16x8*)(tile + L::off(kb * 16 + ka_row, ds * 4 + quad));
#pragma unroll
    for (int d = 0; d < DB; ++d) {
      const int c = d * 2 + tr_c;
      op.vlo[d] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(vt + L::off(tr_row, c) + tr_half));
      op.vhi[d] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(vt + L::off(16 + tr_row, c) + tr_half));
    }
  };

  // One step (32 keys) of this wave's rows: scores, mask, online softmax, value product.
  auto compute = [&](const Ops& op, int step) {
    const int key0 = k_begin + step * kStep;
    // S^T blocks kb = 0, 1: element e of a lane in quad q is key kb*16 + e*4 + q, row col.  The mask enters
    // as the products' starting value (0 or -inf), so nothing rewrites the scores after the matrix cores
    // have written them; only steps that reach the tree slots or the piece end need it.
    f32x4 s[RB][2];
    auto products = [&](bool from_zero) {
      // (the products are issued at a raised wave priority, so that the SIMD's other wave -- in its softmax --
      // does not hold them back: gqa_long 355 -> 339 us)
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int ds = 0; ds < DS; ++ds)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            s[rb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                op.kf[kb][ds], qf[rb][ds], (from_zero && ds == 0) ? f32x4{0.f, 0.f, 0.f, 0.f} : s[rb][kb], 0, 0, 0);
      __builtin_amdgcn_s_setprio(0);
    };
    if (key0 + kStep > Lp || key0 + kStep > k_end) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int key = key0 + kb * 16 + e * 4 + quad;
            const int j = key - Lp;                      // tree node of a key past the prefix
            const uint64_t word = j < 64 ? anc0[rb] : anc1[rb];
            const bool anc = ((word >> (j & 63)) & 1ull) != 0;
            const bool vis = (key < k_end) & ((key < Lp) | anc);
            s[rb][kb][e] = vis ? 0.f : -INFINITY;
          }
        }
      }
      products(false);
    } else {
      products(true);   // the first products start from an inline zero (no accumulator to clear)
    }

    // this lane's maximum over its 8 keys of each row, in scaled log2 units (c > 0 keeps the order)
    float lmax[RB];
    bool grow = false;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      // (NaN-propagating maximum: three-input instructions, no canonicalising of the products' results; a
      // score is never NaN, the rows past a sequence's end being zeroed)
      lmax[rb] = c_scale * vmax(vmax(vmax(s[rb][0][0], s[rb][0][1]), vmax(s[rb][0][2], s[rb][0][3])),
                                vmax(vmax(s[rb][1][0], s[rb][1][1]), vmax(s[rb][1][2], s[rb][1][3])));
      grow |= lmax[rb] > m_run[rb] + kLazyLog2;
    }
    // The reference maximum m only moves when some score exceeds it by more than 2^8 (the exponentials then
    // stay <= 256, and softmax does not depend on the reference), which after the first steps is rare: in
    // the common case no cross-lane reduction and no rescale happen at all, and one branch covers every
    // row block, so the exponentials and value products of all of them form one scheduling region.
    if (__any(grow)) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float tmax = fmaxf(lmax[rb], __shfl_xor(lmax[rb], 16));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        if (tmax > m_run[rb] + kLazyLog2) {
          const float alpha = m_run[rb] == -INFINITY ? 0.f : fast_exp2(m_run[rb] - tmax);
          // p * (z - m) with the new reference: each old term gains (m_old - m_new) before the rescale
          if (ENT) e_run[rb] = alpha == 0.f ? 0.f : alpha * fmaf(m_run[rb] - tmax, l_run[rb], e_run[rb]);
          m_run[rb] = tmax;
          l_run[rb] *= alpha;
#pragma unroll
          for (int d = 0; d < DB; ++d) o[rb][d] *= alpha;
        }
      }
    }
    bf16x8 pb[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const float m_use = m_run[rb] == -INFINITY ? 0.f : m_run[rb];
      float psum = 0.f, esum = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float t = fmaf(s[rb][kb][e], c_scale, -m_use);
          const float p = fast_exp2(t);
          psum += p;
          // (a masked key has t = -inf and p = 0; the clamp keeps its term 0 rather than NaN)
          if (ENT) esum = fmaf(p, fmaxf(t, -1.0e4f), esum);
          pb[rb][kb * 4 + e] = (__bf16)p;
        }
      }
      l_run[rb] += psum;
      if (ENT) e_run[rb] += esum;
    }

    // O^T[d][row] += sum over the 32 keys of V[key][d] P[row][key]
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int d = 0; d < DB; ++d) {
      bf16x8 va;
      const bf16x4 lo_b = __builtin_bit_cast(bf16x4, op.vlo[d]), hi_b = __builtin_bit_cast(bf16x4, op.vhi[d]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        va[e] = lo_b[e];
        va[4 + e] = hi_b[e];
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) o[rb][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[rb], o[rb][d], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
  };

  if constexpr (PIPE) {
    // Software-pipelined: after the barrier that hands over super-step js+1, a wave issues that super-step's
    // operand reads and then computes super-step js from registers, so the LDS reads of one step overlap the
    // products and softmax of the previous one on every wave.
    Ops op[2];
    if (nsa > 0) {
      wait_vm_steps<CPS, NSS - 1>(issued_by(0) - 1);   // this wave's copies of super-step 0 have landed
      zero_tail(0);
      barrier_lds();
      if (kw < nact) read_ops(op[0], 0);
    }
    auto half_step = [&](int js, const Ops& cur, Ops& nxt) {
      const bool more = js + 1 < nsa;
      // Every wave has computed super-step js-1, and its reads of super-step js (issued before that) have
      // returned: the slots of super-step js take the copies of super-step js+NSS at once, without waiting for
      // super-step js+1 to land.
      barrier_lds();
      if (js + NSS < nsa) issue_super(js + NSS);
      if (more) {
        wait_vm_steps<CPS, NSS - 1>(issued_by(js + 1) - 2 - js);   // this wave's copies of super-step js+1
        zero_tail(js + 1);
      }
      // super-step js+1 complete in LDS for every wave.  (Also taken after the last super-step, so that on
      // every path the operands of super-step js are known to have landed in registers.)
      barrier_lds();
      if (more && (js + 1) * KW + kw < nact) read_ops(nxt, js + 1);
      __builtin_amdgcn_sched_barrier(0);
      if (js * KW + kw < nact) compute(cur, js * KW + kw);
    };
    for (int js = 0; js < nsa; js += 2) {
      half_step(js, op[0], op[1]);
      if (js + 1 < nsa) half_step(js + 1, op[1], op[0]);
    }
  } else {
    // One pass of the inner loop per turn of the ring: the slot is a constant in each unrolled copy, so the
    // operand reads take it as an immediate offset (no per-step address arithmetic).
    for (int js0 = 0; js0 < nsa; js0 += NSS) {
#pragma unroll
      for (int sl = 0; sl < NSS; ++sl) {
        const int js = js0 + sl;
        if (js >= nsa) break;
        wait_vm_steps<CPS, NSS - 2>(issued_by(js) - 1 - js);   // this wave's copies of super-step js have landed
        zero_tail(js);
        barrier_lds();   // super-step js complete in LDS for every wave; the slots of super-step js-1 are free
        if (js + NSS - 1 < nsa) issue_super(js + NSS - 1);
        const int step = js * KW + kw;   // this wave's step
        if (step >= nact) continue;
        Ops op;
        read_ops(op, sl);
        __builtin_amdgcn_sched_barrier(0);
        compute(op, step);
      }
    }
  }
  wait_vm<0>();   // copies planned past a sequence's own end land before LDS is reused

#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    l_run[rb] += __shfl_xor(l_run[rb], 16);
    l_run[rb] += __shfl_xor(l_run[rb], 32);
    if (ENT) {
      e_run[rb] += __shfl_xor(e_run[rb], 16);
      e_run[rb] += __shfl_xor(e_run[rb], 32);
    }
  }

  // ---- key groups: group k finalises output columns [16*DBK*k, 16*DBK*(k+1)) of its rows, from every group's
  // state for those columns (exchanged through LDS, merged in group order)
  constexpr int DBK = DB / KW;     // 16-column blocks of the output this wave finalises
  static_assert(DB % KW == 0, "column share");
  f32x4 fin[RB][DBK];
  if constexpr (KW == 1) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int dd = 0; dd < DBK; ++dd) fin[rb][dd] = o[rb][dd];
  } else {
    barrier_lds();   // every wave is done with the ring
    // [owner group][source group, own one left out][DBK*4 16-byte chunks][R rows]: the 16 lanes of a quad touch
    // 256 consecutive bytes, so neither the writes nor the reads conflict on banks
    f32x4* st_o = (f32x4*)ring;
    float2* st_ml = (float2*)(st_o + (size_t)KW * (KW - 1) * DBK * 4 * R);   // [KW][R]
    float* st_e = (float*)(st_ml + KW * R);                                   // [KW][R]
    auto chunk = [&](int owner, int source, int dd, int row) {
      return ((owner * (KW - 1) + (source < owner ? source : source - 1)) * DBK * 4 + dd * 4 + quad) * R + row;
    };
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = rh * RW + rb * 16 + col;
#pragma unroll
      for (int d = 0; d < DB; ++d)
        if (d / DBK != kw) st_o[chunk(d / DBK, kw, d % DBK, row)] = o[rb][d];
      if (quad == 0) {
        st_ml[kw * R + row] = make_float2(m_run[rb], l_run[rb]);
        if (ENT) st_e[kw * R + row] = e_run[rb];
      }
    }
    barrier_lds();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = rh * RW + rb * 16 + col;
      float mk[KW], lk[KW], ek[KW];
#pragma unroll
      for (int k = 0; k < KW; ++k) {
        const float2 ml = st_ml[k * R + row];
        mk[k] = k == kw ? m_run[rb] : ml.x;
        lk[k] = k == kw ? l_run[rb] : ml.y;
        ek[k] = ENT ? (k == kw ? e_run[rb] : st_e[k * R + row]) : 0.f;
      }
      float M = mk[0];
#pragma unroll
      for (int k = 1; k < KW; ++k) M = fmaxf(M, mk[k]);
      float L = 0.f, E = 0.f;
#pragma unroll
      for (int dd = 0; dd < DBK; ++dd) fin[rb][dd] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < KW; ++k) {
        const float w = mk[k] == -INFINITY ? 0.f : fast_exp2(mk[k] - M);
        if (ENT) E += ent_term(w, ek[k], mk[k], M, lk[k]);
        L += w * lk[k];
#pragma unroll
        for (int dd = 0; dd < DBK; ++dd) {
          f32x4 x;
          if (k == kw) {   // this wave's own state: block kw*DBK + dd of o (kw is wave-uniform)
            x = o[rb][dd];
#pragma unroll
            for (int j = 1; j < KW; ++j)
              if (j == kw) x = o[rb][j * DBK + dd];
          } else {
            x = st_o[chunk(kw, k, dd, row)];
          }
          fin[rb][dd] += w * x;
        }
      }
      m_run[rb] = M;
      l_run[rb] = L;
      e_run[rb] = E;
    }
  }
  const int c0 = kw * DBK * 16 + quad * 4;   // first output column of this lane's block dd = 0

  // ---- the workgroup's rows, normalised and rounded to bf16, go row-major into LDS (after the key groups'
  // exchange area; 16-byte pieces of a row XOR-swizzled by the row, so neither the matrix-core-layout writes
  // nor the row reads conflict on banks), with each row's (max, sum) and entropy term; they are then written
  // out as whole 16-byte pieces of rows.
  constexpr int CPR = D / 8;                  // 16-byte pieces per row
  constexpr size_t XBYTES = KW > 1 ? ((size_t)(KW - 1) * R * D * 4 + (size_t)KW * R * 12 + 1023) / 1024 * 1024 : 0;
  static_assert(XBYTES + (size_t)R * D * 2 + (size_t)R * 12 <= (size_t)NST * L::SLOT, "row staging fits the ring");
  unsigned char* row_lds = ring + XBYTES;                               // [R][CPR] 16-byte pieces
  float2* ml_lds = (float2*)(row_lds + (size_t)R * D * 2);              // [R]
  float* e_lds = (float*)(ml_lds + R);                                  // [R]
  auto row_piece = [&](int r, int ch) { return row_lds + ((size_t)r * CPR + (ch ^ (r & (CPR - 1)))) * 16; };
  if constexpr (KW == 1) barrier_lds();   // every wave's last operand reads of the ring have returned
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int rl = rh * RW + rb * 16 + col;
    const float inv = l_run[rb] > 0.f ? 1.0f / l_run[rb] : 0.f;
#pragma unroll
    for (int dd = 0; dd < DBK; ++dd) {
      bf16x4 res;
#pragma unroll
      for (int e = 0; e < 4; ++e) res[e] = (__bf16)(fin[rb][dd][e] * inv);
      const int c = c0 + dd * 16;
      *(bf16x4*)(row_piece(rl, c / 8) + (c % 8) * 2) = res;
    }
    if (kw == 0 && quad == 0) {
      ml_lds[rl] = make_float2(m_run[rb], l_run[rb]);
      if (ENT) e_lds[rl] = e_run[rb];
    }
  }
  barrier_lds();

  // (row, 16-byte piece) items of the workgroup's rows, dealt to the threads
  constexpr int ITEMS = (R * CPR + 64 * W - 1) / (64 * W);   // items per thread
  const int S = a.splits;
  const size_t pset = (size_t)u * a.row_groups + rg;
  const size_t prow0 = pset * S * R;   // the set's piece 0, row 0
  const int rows_valid = min(R, rows_total - rg * R);
  // One piece writes the output; with several, every piece stores its rows (normalised, bf16), their (max,
  // sum) and entropy terms as piece `split` of its set.  Rows of one KV head are consecutive in memory.
  {
    __bf16* dst = S == 1 ? (__bf16*)a.out + (qrow0 + (size_t)rg * R) * D : a.part_o + (prow0 + (size_t)split * R) * D;
#pragma unroll
    for (int t = 0; t < ITEMS; ++t) {
      const int item = t * 64 * W + tid;
      const int r = item / CPR, ch = item % CPR;
      if (item < R * CPR && r < rows_valid) *(u32x4*)(dst + (size_t)r * D + ch * 8) = *(const u32x4*)row_piece(r, ch);
    }
    if (tid < rows_valid) {
      const float2 ml = ml_lds[tid];
      if (S == 1) {
        const size_t orow = qrow0 + rg * R + tid;
        if (a.lse) a.lse[orow] = ml.y > 0.f ? (ml.x + __log2f(ml.y)) * kLn2 : -INFINITY;
        if (ENT) a.entropy[orow] = row_entropy(ml.y, e_lds[tid]);
      } else {
        const size_t pr = prow0 + (size_t)split * R + tid;
        *(float2*)(a.part_ml + 2 * pr) = ml;
        if (ENT) a.part_e[pr] = e_lds[tid];
      }
    }
  }
  if (S == 1) return;

  // ---- the set's merge, spread over its pieces.  One 64-bit counter word per set (fields at the kCtr*
  // shifts): pieces started, pieces arrived, a bit per arrived piece, and the sum and the sum of squares of the
  // started pieces' XCD ids.  A piece that arrives when its whole set has started waits for every arrival and
  // merges its own slice of the rows: every piece it waits for is running and arrives without waiting for
  // anything.  A piece that arrives earlier leaves; the piece whose start completed the set saw it among the
  // arrived bits then, and merges its slice too (that piece arrives after the set is complete, so it never
  // leaves).  So every wait ends, and each slice is merged once.  The last arrival puts the word back to zero
  // for the next call; a waiting piece takes either the full count or that zero as the end of its wait.  The
  // pieces' rows are read from this XCD's L2: all pieces of a set share blockIdx % 8, and consecutive
  // workgroups of a dispatch go to consecutive XCDs (which XCD takes workgroup 0 differs, e.g. between direct
  // and graph launches).  A merging piece checks that: S ids whose sum is S x and sum of squares S x^2 all
  // equal x, this piece's own.
  unsigned long long* ctr = a.set_ctr + pset * a.ctr_stride;
  wait_vector_memory();   // this piece's rows have reached the L2
  __syncthreads();
  if (tid == 0) {
    const unsigned long long old = __hip_atomic_fetch_add(
        ctr, (1ull << kCtrArrived) | (1ull << (kCtrMask + split)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned long long cnt = (1ull << kCtrCountBits) - 1;
    const bool coop = (old & cnt) == (unsigned long long)S;
    const bool last = ((old >> kCtrArrived) & cnt) == (unsigned long long)(S - 1);
    bool good = true;
    if (coop) {
      const unsigned long long x = xcd_id();
      const unsigned long long sum = (old >> kCtrXcdSum) & ((1ull << (kCtrXcdSq - kCtrXcdSum)) - 1);
      const unsigned long long sq = old >> kCtrXcdSq;
      if (sum != S * x || sq != S * x * x) {
        raise_device_error(a.err, kErrXcdSplit);
        good = false;
      }
    }
    if (last) {
      __hip_atomic_store(ctr, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else if (coop) {
      const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
      for (;;) {
        const unsigned long long now = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (((now >> kCtrArrived) & cnt) == (unsigned long long)S || (now & cnt) == 0ull) break;
        if (__builtin_amdgcn_s_memrealtime() - t0 > a.wait_ticks) {
          raise_device_error(a.err, kErrWaitTimeout);
          good = false;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    // slices this workgroup merges: its own (when it waited), and those of the pieces that left before this
    // piece's start completed the set
    uint32_t slices = coop ? 1u << split : 0u;
    if ((start_old & cnt) == (unsigned long long)(S - 1))
      slices |= (uint32_t)(start_old >> kCtrMask) & (uint32_t)((1ull << S) - 1);
    merge_lds = slices;
    good_lds = good ? 1u : 0u;
  }
  __syncthreads();
  const uint32_t slices = merge_lds;
  const size_t orow0 = qrow0 + (size_t)rg * R;
  for (int k = 0; k < S; ++k) {
    if (!((slices >> k) & 1u)) continue;
    const int r0 = k * R / S, r1 = (k + 1) * R / S;
    merge_pieces<D, W, ENT>(a, prow0, R, (__bf16*)a.out + orow0 * D, a.lse ? a.lse + orow0 : nullptr,
                            ENT ? a.entropy + orow0 : nullptr, rows_valid, r0, r1 - r0, good_lds == 1u);
  }
}

template <int D, int RB, int KW, int W, int NST, int WPC, bool ENT>
hipError_t launch_streaming(const AttnArgs& a, hipStream_t stream) {
  constexpr size_t lds = dynamic_lds<D, NST, WPC>(16 * RB * (W / KW));
  static_assert(lds + 2 * kMaxNodes * 8 + 2 * kMaxNodes * 8 + 64 <= 160 * 1024 / WPC, "LDS budget");
  // two sets of operand registers fit beside one 16-row block's state, not beside two
  auto kern = tree_attn_bf16_kernel<D, RB, KW, W, NST, RB == 1, ENT, WPC>;
  static bool configured = false;
  if (!configured) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    configured = true;
  }
  if (a.rows_per_wg != 16 * RB * (W / KW)) return hipErrorInvalidValue;
  if (a.splits > 1 && (!a.part_o || !a.part_ml || !a.set_ctr || (ENT && !a.part_e))) return hipErrorInvalidValue;
  if (a.splits > 1 && a.ctr_stride < 2) return hipErrorInvalidValue;
  const unsigned units_rounded = (a.units + 7) / 8 * 8;
  const unsigned grid = units_rounded * (unsigned)(a.splits * a.row_groups);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * W), lds, stream, a);
  return hipGetLastError();
}

// Every configuration in two builds: with the entropy term (a.entropy given) and without (no extra work).
template <int D, int RB, int KW, int W, int NST, int WPC = 1>
hipError_t launch(const AttnArgs& a, hipStream_t stream) {
  return a.entropy ? launch_streaming<D, RB, KW, W, NST, WPC, true>(a, stream)
                   : launch_streaming<D, RB, KW, W, NST, WPC, false>(a, stream);
}

template <int D, int NST>
hipError_t launch_for_rows(const AttnArgs& a, hipStream_t stream) {
  switch (a.rows_per_wg) {
    case 16: return launch<D, 1, 4, 4, NST>(a, stream);
    case 32: return launch<D, 1, 4, 8, NST>(a, stream);
    case 64: return launch<D, 2, 2, 4, NST / 2, 2>(a, stream);
    case 128: return launch<D, 2, 1, 4, NST / 2, 2>(a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

// Rows per workgroup: the narrowest of 16 and 32 rows (4 waves in 4 key groups, 8 waves in 4 key groups; every
// wave owns 16 rows, and 8 waves put two on each SIMD, so one's softmax overlaps the other's products) and 64
// rows (4 waves of 32 rows in 2 key groups) that holds every row of a KV head, else 128: 4 waves of 32 rows on
// the same keys, several row groups.  The 64- and 128-row workgroups take half a compute unit's LDS, so two
// share a compute unit (a wave's partner on its SIMD belongs to the other workgroup, so their phases are not
// tied by a barrier).
int tree_attn_bf16_rows_per_wg(int rows_total) {
  return rows_total <= 16 ? 16 : rows_total <= 32 ? 32 : rows_total <= 64 ? 64 : 128;
}

int tree_attn_bf16_wgs_per_cu(int rows_per_wg) { return rows_per_wg >= 64 ? 2 : 1; }

hipError_t launch_tree_attn_bf16(const AttnArgs& a, hipStream_t stream) {
  if (a.D == 128) return launch_for_rows<128, 8>(a, stream);
  if (a.D == 64) return launch_for_rows<64, 16>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace dreams

// Tree-masked verification attention, bf16 inputs, fp32 accumulation on the matrix cores.
//
// What is computed (the paper's Section 3.2 attention mask applied to the target's verification pass of
// Section 2): for every tree node i of every query head, softmax(scale * q_i . k_j) v_j over the committed
// prefix slots and the slots of node i's ancestors-or-self.
//
// Work decomposition
//   * A workgroup of 4 waves owns R = 64*RB query rows of one KV head (the rows of the G query heads sharing
//     it are packed: row r -> head r / T, node r % T, which is also their order in memory) and one piece of
//     that head's key axis.  Wave w owns rows [16*RB*w, 16*RB*(w+1)) for every key of the piece, so there
//     is no merge between waves, and every K/V byte the workgroup reads serves all of its rows.
//   * K/V stream through a ring of NST step slots in LDS (a step = 32 keys: 32 K rows then 32 V rows).  The
//     four waves each copy a quarter of every step straight from global memory into LDS
//     (global_load_lds_dwordx4: no registers in between), NST-1 steps ahead, so up to NST-1 steps per
//     compute unit are in flight.  One barrier per step hands a landed step to all waves and frees the slot
//     of the previous step for the next copy.  The copies are issued with inline assembly and waited for by
//     exact count; nothing else in the kernel loads through the vector memory path before the epilogue, so
//     the compiler never inserts a wait that would drain the ring.
//   * Each lane fetches the source chunk that lands where an XOR-swizzled row layout wants it, which makes
//     both operand reads below bank-conflict free:
//       S^T = K Q^T        v_mfma_f32_16x16x32_bf16, K rows as the A operand (16-byte LDS reads)
//       online softmax     per query row; each lane holds one row's scores, 4-way cross-lane reductions
//       O^T += V^T P^T     A operand read with ds_read_b64_tr_b16 (a 4 x 16 transposing LDS read); the
//                          probabilities are already in B-operand layout, so they never leave registers.
//   * Waves are arranged as KW key groups of 4/KW waves: the groups take alternate steps (group k the steps
//     k, k+KW, ...) and each wave owns 16*RB rows, so a wave's operand reads serve as many rows as possible;
//     the groups' (max, sum, accumulator) states are merged through LDS at the end.
//   * With several pieces per (sequence, KV head, row group), each workgroup writes its rows' (max, sum,
//     accumulator) to the workspace and the pieces are merged in piece order (so the result does not depend
//     on scheduling), in one of two ways:
//       - one round of workgroups: a second, small kernel; the kernel boundary makes the partial results
//         visible across XCDs, with no device-scope stores, fences or counters on the streaming path;
//       - several rounds: extra workgroups at the end of the same launch, which wait for their set's pieces
//         (device-scope stores, then one arrival per piece) and merge them while the last round streams.
//   * Workgroup ids are remapped so that all workgroups of one (sequence, KV head) run on the same XCD
//     (consecutive ids are dealt round-robin over the 8 XCDs): row groups reading the same keys share them
//     in that XCD's L2.
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

// Device-scope (sc1) accesses through a buffer resource over [base, base + bytes): coherent across the
// XCDs' L2s, which the pieces' partial results need when the merge runs in the same launch.
// (the buffer builtins take and return plain `vector_size` vectors: values cross to and from them by bit_cast
// only, never by assignment)
typedef uint32_t buf_b128 __attribute__((vector_size(16)));
typedef uint32_t buf_b64 __attribute__((vector_size(8)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
constexpr int kDeviceScope = 16;   // sc1 bit of the buffer instructions' cache-policy operand
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// Bound on a merging workgroup's wait for the pieces (100 MHz real-time ticks): 0.2 s, far beyond any call.
constexpr uint64_t kMergeWaitTicks = 20000000;

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
  __device__ static __forceinline__ int swz(int r) { return (r / RPL) % CPR; }
  __device__ static __forceinline__ int off(int r, int c) { return r * ROW + ((c ^ swz(r)) << 4); }
};

// Merge of a set's pieces by workgroups of the streaming launch (the ones past a.stream_wgs), laid out like
// the merge kernel below: each wave covers 64 / (D/4) rows at 4 columns per lane; a set takes
// ceil(R / (W * those rows)) workgroups.  They are dispatched after every streaming workgroup, so the pieces
// they wait for are already running or done and never wait themselves: the wait ends.  The pieces' rows are
// read with device-scope loads after their arrival count is complete; the last merging workgroup of the set
// clears both counters for the next call.
template <int D, int W, bool ENT>
__device__ __forceinline__ void merge_in_launch(const AttnArgs& a, int m) {
  constexpr int CPT = 4;                // columns per lane
  constexpr int TPR = D / CPT;          // lanes per row
  constexpr int MR = 64 / TPR;          // rows per wave
  constexpr int CH = 8;                 // pieces per batch of loads
  const int R = a.rows_per_wg, S = a.splits;
  const int MB = (R + W * MR - 1) / (W * MR);
  const int sets = a.units * a.row_groups;
  const int pset = m / MB, mb = m - pset * MB;
  const int wave = threadIdx.x >> 6, t = threadIdx.x & 63;
  const int r = (mb * W + wave) * MR + t / TPR, c0 = (t % TPR) * CPT;
  uint32_t* arrive = a.merge_ctr + (size_t)pset * a.merge_stride;
  uint32_t* done = a.merge_ctr + (size_t)(sets + pset) * a.merge_stride;

  // wave 0 waits for the set's pieces; the others wait for wave 0
  __shared__ int in_time_lds;
  if (wave == 0) {
    bool in_time = true;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (__hip_atomic_load(arrive, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < (uint32_t)S) {
      if (__builtin_amdgcn_s_memrealtime() - t0 > kMergeWaitTicks) {
        in_time = false;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    if (t == 0) in_time_lds = in_time;
  }
  __syncthreads();
  const bool in_time = in_time_lds != 0;
  // This workgroup is done with the arrival counter: count it as done now, so that the atomic's round trip
  // overlaps the loads below; the last workgroup of the set clears both counters at its end.
  uint32_t done_before = 0;
  if (threadIdx.x == 0) done_before = __hip_atomic_fetch_add(done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  if (r < R) {
    const size_t row0 = (size_t)pset * S * R;   // the set's piece 0, row 0
    const auto racc = buffer_rsrc(a.part_acc + row0 * D, (uint32_t)S * R * D * 4);
    const auto rml = buffer_rsrc(a.part_ml + row0 * 2, (uint32_t)S * R * 8);
    const auto re = buffer_rsrc(a.part_e + row0, (uint32_t)S * R * 4);
    constexpr bool ent = ENT;
    float M = -INFINITY, lsum = 0.f, esum = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < S; s0 += CH) {
      float2 ml[CH];
      f32x4 x[CH];
      float ev[CH];
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const int pr = min(s0 + k, S - 1) * R + r;
        const f32x2 mlv = __builtin_bit_cast(f32x2, __builtin_amdgcn_raw_buffer_load_b64(rml, pr * 8, 0, kDeviceScope));
        ml[k] = make_float2(mlv.x, mlv.y);
        x[k] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(racc, (pr * D + c0) * 4, 0, kDeviceScope));
        ev[k] = ent ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(re, pr * 4, 0, kDeviceScope)) : 0.f;
      }
      float Mn = M;
#pragma unroll
      for (int k = 0; k < CH; ++k)
        if (s0 + k < S) Mn = fmaxf(Mn, ml[k].x);
      const float scale_old = M == -INFINITY ? 0.f : fast_exp2(M - Mn);
      esum = ent_term(scale_old, esum, M, Mn, lsum);
      lsum *= scale_old;
      acc *= scale_old;
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const float w = (s0 + k >= S || ml[k].x == -INFINITY) ? 0.f : fast_exp2(ml[k].x - Mn);
        esum += ent_term(w, ev[k], ml[k].x, Mn, ml[k].y);
        lsum += w * ml[k].y;
        acc += w * x[k];
      }
      M = Mn;
    }
    const int rg = pset % a.row_groups, u = pset / a.row_groups;
    const int b = u / a.Hkv, g = u - b * a.Hkv;
    const int row = rg * R + r;   // row within the KV head's G*T rows
    if (row < a.G * a.T) {
      const size_t orow = ((size_t)b * a.Hq + (size_t)g * a.G) * a.T + row;
      const float inv = !in_time ? NAN : lsum > 0.f ? 1.0f / lsum : 0.f;
      bf16x4 res;
#pragma unroll
      for (int e = 0; e < CPT; ++e) res[e] = (__bf16)(acc[e] * inv);
      *(bf16x4*)((__bf16*)a.out + orow * D + c0) = res;
      if (a.lse && c0 == 0) a.lse[orow] = !in_time ? NAN : lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
      if (ent && c0 == 0) a.entropy[orow] = !in_time ? NAN : row_entropy(lsum, esum);
    }
  }
  if (threadIdx.x == 0 && done_before == (uint32_t)MB - 1) {
    reset_counter(done);
    reset_counter(arrive);
  }
}

template <int D, int RB, int KW, int W, int NST, bool PIPE, bool ENT>
__global__ __launch_bounds__(64 * W) void tree_attn_bf16_kernel(AttnArgs a) {
  constexpr int WR = W / KW;          // waves per key group; each owns a different slice of the rows
  constexpr int RW = 16 * RB;         // query rows per wave
  constexpr int R = WR * RW;          // query rows per workgroup
  constexpr int DS = D / 32;          // k-steps of S^T = K Q^T
  constexpr int DB = D / 16;          // 16-column blocks of O^T
  using L = Rows<D>;
  constexpr int C16 = L::C16;         // wave-wide copies per 16 rows
  constexpr int NSS = NST / KW;       // ring slots in super-steps (KW consecutive steps, one per key group)
  constexpr int QSLOTS = (R * L::ROW + L::SLOT - 1) / L::SLOT;   // step slots the query rows occupy
  constexpr int QSS = (QSLOTS + KW - 1) / KW;                      // ... in super-steps
  constexpr int CPS = 4 * KW * C16 / W;   // copies per wave per super-step (4*KW blocks of 16 rows)
  constexpr int QB = R / 16;          // 16-row blocks of query rows, dealt to the waves round-robin
  static_assert(W % KW == 0 && (NST & (NST - 1)) == 0 && NSS > QSS && NSS >= 2, "ring layout");
  static_assert(CPS * W == 4 * KW * C16 && CPS >= 1 && (C16 % CPS == 0 || CPS % C16 == 0), "copy split");
  static_assert(16 * L::ROW == C16 * 1024 && (16 / L::RPL) % L::CPR == 0, "swizzle repeats every 16 rows");
  static_assert(NSS * CPS + ((QB + W - 1) / W) * C16 + 8 <= 63, "outstanding copies fit the counter");
  static_assert((size_t)(KW - 1) * R * (D + 3) * 4 <= (size_t)NST * L::SLOT, "group states fit the ring");

  extern __shared__ __attribute__((aligned(1024))) unsigned char ring[];   // NST step slots
  __shared__ uint64_t anc_lds[2 * kMaxNodes];
  __shared__ uint32_t meta_lds[4 * kMaxNodes];   // the sequence's parents or tree mask rows, as copied
  __shared__ uint32_t stored_lds;                 // owner waves whose partial rows are stored (merge in launch)

  if (a.merge_ctr && (int)blockIdx.x >= a.stream_wgs) {
    merge_in_launch<D, W, ENT>(a, (int)blockIdx.x - a.stream_wgs);
    return;
  }

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
  if (tid == 0) stored_lds = 0;       // (published by the prologue's barriers)

  // ---- this workgroup's piece of the key axis, planned from the host's bound on the key count
  int piece = (a.max_keys + a.splits - 1) / a.splits;
  piece = (piece + kStep - 1) / kStep * kStep;
  const int k_begin = split * piece;
  const int k_end_plan = split == a.splits - 1 ? a.max_keys : min(a.max_keys, k_begin + piece);
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
  const unsigned char* qslab = ring + (NST - QSLOTS) * L::SLOT;
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
      const uint64_t* mr = (const uint64_t*)meta_lds + tid * Wm;
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
    } else {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) s[rb][0] = s[rb][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // (the products are issued at a raised wave priority, so that the SIMD's other wave -- in its softmax --
    // does not hold them back: gqa_long 355 -> 339 us)
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) s[rb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(op.kf[kb][ds], qf[rb][ds], s[rb][kb], 0, 0, 0);
    __builtin_amdgcn_s_setprio(0);

    // this lane's maximum over its 8 keys of each row, in scaled log2 units (c > 0 keeps the order)
    float lmax[RB];
    bool grow = false;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      lmax[rb] = c_scale * fmaxf(fmaxf(fmaxf(s[rb][0][0], s[rb][0][1]), fmaxf(s[rb][0][2], s[rb][0][3])),
                                 fmaxf(fmaxf(s[rb][1][0], s[rb][1][1]), fmaxf(s[rb][1][2], s[rb][1][3])));
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
      if (more) {
        wait_vm_steps<CPS, NSS - 2>(issued_by(js) - 2 - js);   // ... and of super-step js+1
        zero_tail(js + 1);
      }
      // super-step js+1 complete in LDS for every wave; every wave's reads of super-step js have returned,
      // so its slots take the copies of super-step js+NSS.  (Also taken after the last super-step, so that
      // on every path the operands of super-step js are known to have landed in registers.)
      barrier_lds();
      if (more) {
        if (js + NSS < nsa) issue_super(js + NSS);
        if ((js + 1) * KW + kw < nact) read_ops(nxt, js + 1);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (js * KW + kw < nact) compute(cur, js * KW + kw);
    };
    for (int js = 0; js < nsa; js += 2) {
      half_step(js, op[0], op[1]);
      if (js + 1 < nsa) half_step(js + 1, op[1], op[0]);
    }
  } else {
    for (int js = 0; js < nsa; ++js) {
      wait_vm_steps<CPS, NSS - 2>(issued_by(js) - 1 - js);   // this wave's copies of super-step js have landed
      zero_tail(js);
      barrier_lds();   // super-step js complete in LDS for every wave; the slots of super-step js-1 are free
      if (js + NSS - 1 < nsa) issue_super(js + NSS - 1);
      const int step = js * KW + kw;   // this wave's step
      if (step >= nact) continue;
      Ops op;
      read_ops(op, js);
      __builtin_amdgcn_sched_barrier(0);
      compute(op, step);
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

  // ---- key groups 1.. hand their states to group 0 through LDS (merged in group order)
  if constexpr (KW > 1) {
    barrier_lds();   // every wave is done with the ring
    // accumulators as [KW-1][D/4][R] 16-byte chunks: the 16 lanes of a quad touch 256 consecutive bytes,
    // so neither the writes nor the reads below conflict on banks
    f32x4* st_o = (f32x4*)ring;
    float2* st_ml = (float2*)(st_o + (KW - 1) * R * (D / 4));  // [KW-1][R]
    float* st_e = (float*)(st_ml + (KW - 1) * R);                // [KW-1][R]
    if (kw > 0) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int row = (kw - 1) * R + rh * RW + rb * 16 + col;
#pragma unroll
        for (int d = 0; d < DB; ++d) st_o[((kw - 1) * (D / 4) + d * 4 + quad) * R + rh * RW + rb * 16 + col] = o[rb][d];
        if (quad == 0) {
          st_ml[row] = make_float2(m_run[rb], l_run[rb]);
          if (ENT) st_e[row] = e_run[rb];
        }
      }
    }
    barrier_lds();
    if (kw == 0) {
#pragma unroll
      for (int k = 1; k < KW; ++k) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int row = (k - 1) * R + rh * RW + rb * 16 + col;
          const float2 ml = st_ml[row];
          const float M = fmaxf(m_run[rb], ml.x);
          const float w0 = m_run[rb] == -INFINITY ? 0.f : fast_exp2(m_run[rb] - M);
          const float w1 = ml.x == -INFINITY ? 0.f : fast_exp2(ml.x - M);
          if (ENT) e_run[rb] = ent_term(w0, e_run[rb], m_run[rb], M, l_run[rb]) + ent_term(w1, st_e[row], ml.x, M, ml.y);
          m_run[rb] = M;
          l_run[rb] = l_run[rb] * w0 + ml.y * w1;
#pragma unroll
          for (int d = 0; d < DB; ++d) o[rb][d] = o[rb][d] * w0 + st_o[((k - 1) * (D / 4) + d * 4 + quad) * R + rh * RW + rb * 16 + col] * w1;
        }
      }
    }
  }
  const bool owner = kw == 0;   // the waves that now hold the workgroup's final states

  // ---- a single piece: normalise and write.  Rows of one KV head are consecutive in memory.
  if (a.splits == 1) {
    if (!owner) return;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = rg * R + rh * RW + rb * 16 + col;
      if (row >= rows_total) continue;
      const size_t orow = qrow0 + row;
      const float inv = l_run[rb] > 0.f ? 1.0f / l_run[rb] : 0.f;
#pragma unroll
      for (int d = 0; d < DB; ++d) {
        bf16x4 res;
#pragma unroll
        for (int e = 0; e < 4; ++e) res[e] = (__bf16)(o[rb][d][e] * inv);
        *(bf16x4*)((__bf16*)a.out + orow * D + d * 16 + quad * 4) = res;
      }
      if (a.lse && quad == 0)
        a.lse[orow] = l_run[rb] > 0.f ? (m_run[rb] + __log2f(l_run[rb])) * kLn2 : -INFINITY;
      if (ENT && quad == 0) a.entropy[orow] = row_entropy(l_run[rb], e_run[rb]);
    }
    return;
  }

  // ---- several pieces: write this piece's unnormalised rows and (max, sum) for the merge
  if (!owner) return;
  const size_t pset = (size_t)u * a.row_groups + rg;
  if (a.merge_ctr) {
    // merged in this launch: device-scope stores, then one arrival per workgroup once every owner wave's
    // stores have completed
    const size_t row0 = pset * a.splits * R;
    const auto racc = buffer_rsrc(a.part_acc + row0 * D, (uint32_t)a.splits * R * D * 4);
    const auto rml = buffer_rsrc(a.part_ml + row0 * 2, (uint32_t)a.splits * R * 8);
    const auto re = buffer_rsrc(a.part_e + row0, (uint32_t)a.splits * R * 4);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int pr = split * R + rh * RW + rb * 16 + col;   // row within the set's pieces
#pragma unroll
      for (int d = 0; d < DB; ++d)
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(buf_b128, o[rb][d]), racc, (pr * D + d * 16 + quad * 4) * 4, 0,
                                               kDeviceScope);
      if (quad == 0) {
        const f32x2 mlv = {m_run[rb], l_run[rb]};
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(buf_b64, mlv), rml, pr * 8, 0, kDeviceScope);
        if (ENT) __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, e_run[rb]), re, pr * 4, 0, kDeviceScope);
      }
    }
    wait_vector_memory();
    if (lane == 0 &&
        __hip_atomic_fetch_add(&stored_lds, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == (uint32_t)WR - 1)
      __hip_atomic_fetch_add(a.merge_ctr + pset * a.merge_stride, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  // separate merge kernel: plain stores, which the kernel boundary makes visible to it
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const size_t pr = (pset * a.splits + split) * R + rh * RW + rb * 16 + col;
#pragma unroll
    for (int d = 0; d < DB; ++d) *(f32x4*)(a.part_acc + pr * D + d * 16 + quad * 4) = o[rb][d];
    if (quad == 0) {
      *(float2*)(a.part_ml + 2 * pr) = make_float2(m_run[rb], l_run[rb]);
      if (ENT) a.part_e[pr] = e_run[rb];
    }
  }
}

// Merge of the key-axis pieces: out = sum_s w_s acc_s / sum_s w_s l_s with w_s = 2^(m_s - max_s m_s), in
// piece order.  A one-wave workgroup merges the 64 / (D/4) rows (2 for D = 128, 4 for D = 64) of one
// (sequence, KV head, row group) that its lanes cover at 4 columns (one 16-byte load per piece) each, so the
// merge spreads over many compute units with many requests in flight.  All loads of a chunk of 8 pieces are
// issued before any is used.
template <int D>
constexpr int merge_rows() { return 64 / (D / 4); }
template <int D, bool ENT>
__global__ __launch_bounds__(64) void tree_attn_merge_kernel(AttnArgs a) {
  constexpr int CPT = 4;                // columns per thread
  constexpr int TPR = D / CPT;          // threads per row
  constexpr int MR = merge_rows<D>();   // rows per workgroup
  static_assert(TPR * MR == 64, "one wave per workgroup");
  constexpr int CH = 8;                 // pieces per batch of loads
  typedef float fv __attribute__((ext_vector_type(CPT)));
  const int R = a.rows_per_wg;
  const int blocks = R / MR;
  // same XCD as the streaming kernel's workgroups of this (sequence, KV head): ids dealt round-robin over
  // the 8 XCDs, unit u on XCD u % 8
  const int n = blockIdx.x;
  const int xcd = n & 7, slot = n >> 3;
  const int per_unit = a.row_groups * blocks;
  const int u = xcd + 8 * (slot / per_unit);
  if (u >= a.units) return;
  const int within = slot - (slot / per_unit) * per_unit;
  const int rg = within / blocks, rblk = within - rg * blocks;
  const int pset = u * a.row_groups + rg;
  const int b = u / a.Hkv, g = u - b * a.Hkv;
  const int t = threadIdx.x, r = rblk * MR + t / TPR, c0 = (t % TPR) * CPT;
  const int row = rg * R + r;                     // row within the KV head's G*T rows
  const int S = a.splits;
  const size_t prow0 = (size_t)pset * S * R + r;  // this row in piece 0; piece s adds s * R

  constexpr bool ent = ENT;
  float M = -INFINITY, lsum = 0.f, esum = 0.f;
  fv acc = {};
  for (int s0 = 0; s0 < S; s0 += CH) {
    float2 ml[CH];
    fv x[CH];
    float ev[CH];
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      const size_t pr = prow0 + (size_t)min(s0 + k, S - 1) * R;
      ml[k] = *(const float2*)(a.part_ml + 2 * pr);
      x[k] = *(const fv*)(a.part_acc + pr * D + c0);
      ev[k] = ent ? a.part_e[pr] : 0.f;
    }
    float Mn = M;
#pragma unroll
    for (int k = 0; k < CH; ++k)
      if (s0 + k < S) Mn = fmaxf(Mn, ml[k].x);
    const float scale_old = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
    esum = ent_term(scale_old, esum, M, Mn, lsum);
    lsum *= scale_old;
    acc *= scale_old;
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      const float w = (s0 + k >= S || ml[k].x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ml[k].x - Mn);
      esum += ent_term(w, ev[k], ml[k].x, Mn, ml[k].y);
      lsum += w * ml[k].y;
      acc += w * x[k];
    }
    M = Mn;
  }
  if (row >= a.G * a.T) return;
  const size_t orow = ((size_t)b * a.Hq + (size_t)g * a.G) * a.T + row;
  const float inv = lsum > 0.f ? 1.0f / lsum : 0.f;
  __bf16 res[CPT];
#pragma unroll
  for (int e = 0; e < CPT; ++e) res[e] = (__bf16)(acc[e] * inv);
  __builtin_memcpy((__bf16*)a.out + orow * D + c0, res, sizeof(res));
  if (a.lse && c0 == 0) a.lse[orow] = lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
  if (ent && c0 == 0) a.entropy[orow] = row_entropy(lsum, esum);
}

template <int D, int RB, int KW, int W, int NST, bool ENT>
hipError_t launch_streaming(const AttnArgs& a, hipStream_t stream) {
  constexpr size_t lds = (size_t)NST * Rows<D>::SLOT;
  static_assert(lds + 2 * kMaxNodes * 8 + 4 * kMaxNodes * 4 + 64 <= 160 * 1024, "LDS budget");
  // two sets of operand registers fit beside one 16-row block's state, not beside two
  auto kern = tree_attn_bf16_kernel<D, RB, KW, W, NST, RB == 1, ENT>;
  static bool configured = false;
  if (!configured) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    configured = true;
  }
  if (a.rows_per_wg != 16 * RB * (W / KW)) return hipErrorInvalidValue;
  const unsigned units_rounded = (a.units + 7) / 8 * 8;
  const unsigned grid = units_rounded * (unsigned)(a.splits * a.row_groups);
  if (a.splits > 1 && a.merge_ctr) {
    // the merging workgroups follow the streaming ones in the same launch
    constexpr int MRW = W * merge_rows<D>();
    const unsigned merge_wgs = (unsigned)(a.units * a.row_groups) * ((a.rows_per_wg + MRW - 1) / MRW);
    AttnArgs b = a;
    b.stream_wgs = (int)grid;
    hipLaunchKernelGGL(kern, dim3(grid + merge_wgs), dim3(64 * W), lds, stream, b);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * W), lds, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  const unsigned mgrid = units_rounded * a.row_groups * (a.rows_per_wg / merge_rows<D>());
  auto merge = tree_attn_merge_kernel<D, ENT>;
  hipLaunchKernelGGL(merge, dim3(mgrid), dim3(64), 0, stream, a);
  return hipGetLastError();
}

// Every configuration in two builds: with the entropy term (a.entropy given) and without (no extra work).
template <int D, int RB, int KW, int W, int NST>
hipError_t launch(const AttnArgs& a, hipStream_t stream) {
  return a.entropy ? launch_streaming<D, RB, KW, W, NST, true>(a, stream)
                   : launch_streaming<D, RB, KW, W, NST, false>(a, stream);
}

template <int D, int NST>
hipError_t launch_for_rows(const AttnArgs& a, hipStream_t stream) {
  switch (a.rows_per_wg) {
    case 16: return launch<D, 1, 4, 4, NST>(a, stream);
    case 32: return launch<D, 1, 4, 8, NST>(a, stream);
    case 64: return launch<D, 1, 2, 8, NST>(a, stream);
    case 128: return launch<D, 1, 1, 8, NST>(a, stream);
    case 256: return launch<D, 2, 1, 8, NST>(a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

// Rows per workgroup: the narrowest of 16, 32, 64 rows (4 waves in 4 key groups; 8 waves in 4 or 2 key
// groups) that holds every row of a KV head, else 128 (all 8 waves on the same keys, several row groups).
// Every wave owns 16 rows; 8 waves put two on each SIMD, so one's softmax overlaps the other's products.
int tree_attn_bf16_rows_per_wg(int rows_total) {
  return rows_total <= 16 ? 16 : rows_total <= 32 ? 32 : rows_total <= 64 ? 64 : rows_total <= 128 ? 128 : 256;
}

hipError_t launch_tree_attn_bf16(const AttnArgs& a, hipStream_t stream) {
  if (a.D == 128) return launch_for_rows<128, 8>(a, stream);
  if (a.D == 64) return launch_for_rows<64, 16>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace dreams

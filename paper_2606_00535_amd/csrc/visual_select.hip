// Target-aware visual-token selection (the paper's Section 3.1, "Visual Token Compression", Eq. 2): the
// importance of visual token j is its attention weight averaged over every query head and every query row,
// I_j = (1/(Hq*T)) sum_h sum_i A[h,i,j]; the r most important tokens are kept and their K/V rows gathered.
//
//   * visual_importance_kernel: one workgroup per (sequence, KV head, 256 visual tokens), 4 waves of 64 tokens.
//     Each wave holds its 64 key rows as matrix-core A operands (four 16-token blocks, so every query row it
//     loads serves 64 tokens) and runs over the KV head's G*T query rows 64 at a time (all of their loads in
//     flight together), in 16-row matrix-core chunks: S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (operands straight from global memory, 16-byte
//     loads), A = 2^(s*c - lse2(row)) with the row's log-sum-exp from the attention call, summed over the rows
//     in registers, then across the 16 row lanes.  One fp32 partial per (sequence, KV head, token): the keys
//     are read once and each workgroup reads one head's queries.
//     The last KV head to finish a block of tokens (an arrival counter per (sequence, block)) forms
//     I_j = (sum over KV heads, in order) / (Hq*T).
//     With a prompt's own rows (the prefilling pass, which is where Eq. 2 reads the target's attention), row i of
//     every query head sees slots 0..i, only rows i < n_b count, and I_j is the same sum over (Hq*n_b).
//   * visual_topk_kernel: one workgroup per sequence: radix selection of the r-th largest importance over
//     order-preserving integer keys in LDS, then the kept tokens in token order by prefix sums (ties between
//     equal importances go to the smaller token).
//   * visual_gather_kernel: the kept tokens' K/V rows into [B, Hkv, r, D], 16 bytes per lane.
#include "kernels.h"

#include <limits.h>
#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kImpKeys = 256;       // visual tokens per workgroup (64 per wave, in 16-token blocks)
static_assert(kImpKeys == 256, "one thread per token in the final sum");
constexpr int kTopkThreads = 1024;

template <int D>
__global__ __launch_bounds__(256) void visual_importance_kernel(VisualArgs a) {
  constexpr int DS = D / 32;
  constexpr int KB = kImpKeys / 64;   // 16-token blocks per wave
  const int blocks = (a.vis_count + kImpKeys - 1) / kImpKeys;
  const int n = blockIdx.x;
  const int blk = n % blocks, bg = n / blocks;
  const int g = bg % a.Hkv, b = bg / a.Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, quad = lane >> 4;
  const int T = a.T, rows = a.G * T;
  int L = a.kv_len[b];
  if (a.prefill) L = L < 0 ? 0 : (L > T ? T : L);   // the prompt's length
  else L = L < 0 ? 0 : (L > a.S_cap - T ? a.S_cap - T : L);

  // the wave's tokens j0 .. j0 + 16*KB - 1: key rows as A operands (row col of each 16-token block); the
  // outputs of block kb are tokens j0 + 16*kb + 4*quad + e
  const int j0 = blk * kImpKeys + wave * 16 * KB;
  const unsigned char* kbase = (const unsigned char*)a.k + (((size_t)b * a.Hkv + g) * a.S_cap + a.vis_begin) * (D * 2);
  bf16x8 kf[KB][DS];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    const int jk = min(j0 + kb * 16 + col, a.vis_count - 1);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) kf[kb][ds] = *(const bf16x8*)(kbase + (size_t)jk * (D * 2) + (ds * 32 + quad * 8) * 2);
  }

  const size_t row0 = ((size_t)b * a.Hq + (size_t)g * a.G) * T;   // the KV head's first query row
  const unsigned char* qbase = (const unsigned char*)a.q + row0 * (D * 2);
  auto load_q = [&](bf16x8 (&qf)[DS], float& lse, int r0) {
    const int rr = min(r0 + col, rows - 1);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[ds] = *(const bf16x8*)(qbase + (size_t)rr * (D * 2) + (ds * 32 + quad * 8) * 2);
    lse = a.lse[row0 + rr];
  };
  f32x4 acc[KB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) acc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // 64 query rows at a time: all of their loads are issued together (one memory round trip per 64 rows)
  constexpr int QC = 4;
  if (a.prefill) {
    // A prompt's own rows: row i of each of the G heads sees slots 0..i, and only rows i < L count.  Rows below
    // the wave's first token see none of its tokens, so each head's walk starts there.
    const int istart = max(0, a.vis_begin + j0) & ~15;
    for (int hh = 0; hh < a.G; ++hh)
      for (int i0 = istart; i0 < L; i0 += 16 * QC) {
        bf16x8 qf[QC][DS];
        float lse[QC];
#pragma unroll
        for (int c = 0; c < QC; ++c) load_q(qf[c], lse[c], hh * T + i0 + 16 * c);   // (a lane past its head's rows is dead: i >= L)
#pragma unroll
        for (int c = 0; c < QC; ++c) {
          const int i = i0 + 16 * c + col;
          const bool live = i < L && lse[c] != -INFINITY;
          const float lse2 = live ? lse[c] * 1.4426950408889634f : 0.f;
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) {
            f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ds = 0; ds < DS; ++ds) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kb][ds], qf[c][ds], s, 0, 0, 0);
            if (live) {
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int slot = a.vis_begin + j0 + kb * 16 + quad * 4 + e;
                if (slot <= i) acc[kb][e] += __builtin_amdgcn_exp2f(fmaf(s[e], a.scale_log2, -lse2));
              }
            }
          }
        }
      }
  }
  for (int r0 = 0; r0 < (a.prefill ? 0 : rows); r0 += 16 * QC) {
    bf16x8 qf[QC][DS];
    float lse[QC];
#pragma unroll
    for (int c = 0; c < QC; ++c) load_q(qf[c], lse[c], min(r0 + 16 * c, rows - 1));
#pragma unroll
    for (int c = 0; c < QC; ++c) {
      // a row that saw nothing (lse = -inf) attends to no visual token
      const bool live = r0 + 16 * c + col < rows && lse[c] != -INFINITY;
      const float lse2 = live ? lse[c] * 1.4426950408889634f : 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kb][ds], qf[c][ds], s, 0, 0, 0);
        if (live) {
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[kb][e] += __builtin_amdgcn_exp2f(fmaf(s[e], a.scale_log2, -lse2));
        }
      }
    }
  }
  // sum over the 16 row lanes of each quad (fixed order)
#pragma unroll
  for (int off = 1; off < 16; off <<= 1)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[kb][e] += __shfl_xor(acc[kb][e], off);
  if (col == 0) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = j0 + kb * 16 + quad * 4 + e;
        if (j < a.vis_count)
          store_coherent(a.partial + ((size_t)b * a.Hkv + g) * a.vis_count + j, a.vis_begin + j < L ? acc[kb][e] : 0.f);
      }
  }

  // The last of the sequence's KV heads to finish this block of tokens sums the heads' partials, in head
  // order (device-scope stores and loads; the counter is left at zero for the next call).
  __shared__ int last;
  wait_vector_memory();
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t* ctr = a.counters + ((size_t)b * blocks + blk) * a.counter_stride;
    last = arrive_last(ctr, (uint32_t)a.Hkv);
    if (last) reset_counter(ctr);
  }
  __syncthreads();
  if (!last) return;
  const int j = blk * kImpKeys + threadIdx.x;
  if (j >= a.vis_count) return;
  const float* pp = a.partial + (size_t)b * a.Hkv * a.vis_count + j;
  float sum = 0.f;
  for (int g0 = 0; g0 < a.Hkv; g0 += 8) {
    float x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = g0 + k < a.Hkv ? load_coherent(pp + (size_t)(g0 + k) * a.vis_count) : 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) sum += x[k];
  }
  const float rows_counted = a.prefill ? (float)L : (float)T;   // rows per head that count
  a.importance[(size_t)b * a.vis_count + j] = rows_counted > 0.f ? sum / ((float)a.Hq * rows_counted) : 0.f;
}

// ---- Eq. 2 over a prompt's own rows (the prefilling pass): visual_importance_prefill_kernel.  A workgroup of 8
// waves owns 256 visual tokens of one (sequence, KV head), 32 per wave held as matrix-core A operands; the query
// rows that can see them (rows i >= the block's first token slot, of each of the G heads) stream through an LDS
// ring of 64-row stages with their log-sum-exps (LDS-DMA copies, several stages ahead), which all eight waves
// read.  The key rows and query rows use the attention kernel's swizzled layout and operand order (A row m
// holds block row (m%4)*4 + m/4), so every 16-byte operand read is bank-conflict free.  Workgroups are ordered
// so that the blocks with the most rows (the first tokens) start first and share a compute unit with those
// with the fewest.
namespace pf {
constexpr int kWaves = 8, kTokPerWave = kImpKeys / kWaves, KB = kTokPerWave / 16;
constexpr int kRows = 64, kStages = 4;
static_assert(KB == 2 && kWaves * kTokPerWave == kImpKeys, "8 waves of 32 tokens");
template <int D>
struct Rows {
  static constexpr int ROW = D * 2, CPR = D / 8, RPL = 256 / ROW;
  static __device__ __forceinline__ int swz(int r) {
    if constexpr (D == 128) return ((r >> 2) & 3) * 4 + (r & 1) * 2 + 1;
    return (r / RPL) % CPR;
  }
  static __device__ __forceinline__ int off(int r, int c) { return r * ROW + ((c ^ swz(r)) << 4); }
};
typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(lds_void*)p; }
__device__ __forceinline__ void copy16(uint32_t m0, const void* src) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(m0), "v"(src) : "memory");
}
__device__ __forceinline__ void copy4(uint32_t m0, const void* src) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off" ::"s"(m0), "v"(src) : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
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
__device__ __forceinline__ void barrier_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
}  // namespace pf

template <int D>
__global__ __launch_bounds__(64 * pf::kWaves, 2) void visual_importance_prefill_kernel(VisualArgs a) {
  using L_ = pf::Rows<D>;
  constexpr int DS = D / 32;
  constexpr int QBYTES = pf::kRows * L_::ROW;             // a stage's query rows
  constexpr int STAGE = QBYTES + pf::kRows * 4;          // ... and their log-sum-exps
  constexpr int CPW = QBYTES / 1024 / pf::kWaves;         // wave-wide 1 KB query copies per wave per stage
  constexpr int OPS = CPW + 1;                            // vector-memory operations per wave per stage
  static_assert(CPW >= 1 && CPW * 1024 * pf::kWaves == QBYTES, "copy split");
  extern __shared__ __attribute__((aligned(1024))) unsigned char ring[];   // kStages x STAGE
  const int blocks = (a.vis_count + kImpKeys - 1) / kImpKeys, BG = a.B * a.Hkv;
  const int n = blockIdx.x, W = gridDim.x;
  const int rank = (n >= a.cus && W <= 2 * a.cus) ? W - 1 - (n - a.cus) : n;
  const int blk = rank / BG, bg = rank - blk * BG;        // blocks of the first tokens (the most rows) first
  const int g = bg % a.Hkv, b = bg / a.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, quad = lane >> 4;
  const int T = a.T;
  int L = __builtin_amdgcn_readfirstlane(a.kv_len[b]);
  L = L < 0 ? 0 : (L > T ? T : L);                        // the prompt's length

  // the wave's tokens j0 .. j0 + 31 as A operands (A row m of block kb holds token j0 + 16 kb + (m%4)*4 + m/4,
  // so the outputs of block kb at lane (col, quad) are tokens j0 + 16 kb + 4 e + quad)
  const int j0 = blk * kImpKeys + wave * pf::kTokPerWave;
  const int ka_row = (col & 3) * 4 + (col >> 2);
  const unsigned char* kbase = (const unsigned char*)a.k + (((size_t)b * a.Hkv + g) * a.S_cap + a.vis_begin) * L_::ROW;
  bf16x8 kf[pf::KB][DS];
#pragma unroll
  for (int kb = 0; kb < pf::KB; ++kb) {
    const int jk = min(j0 + kb * 16 + ka_row, a.vis_count - 1);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) kf[kb][ds] = *(const bf16x8*)(kbase + (size_t)jk * L_::ROW + (ds * 32 + quad * 8) * 2);
  }
  // (the key loads complete before the first copies are issued, so that the copies' waits count only copies)
#pragma unroll
  for (int kb = 0; kb < pf::KB; ++kb)
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) asm volatile("" : "+v"(kf[kb][ds]));
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // rows that can see the block's tokens: i >= its first token's slot, in 64-row stages, head after head
  const int istart = min(L, max(0, a.vis_begin + blk * kImpKeys) & ~15);
  const int nsh = (L - istart + pf::kRows - 1) / pf::kRows;   // stages per head
  const int nst = a.G * nsh;
  const size_t row0 = ((size_t)b * a.Hq + (size_t)g * a.G) * T;   // the KV head's first query row
  const unsigned char* qbase = (const unsigned char*)a.q + row0 * L_::ROW;
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(pf::lds_addr(ring));
  auto issue = [&](int t) {
    const int hh = t / max(nsh, 1), s0 = istart + (t - hh * nsh) * pf::kRows;
    const uint32_t dst = __builtin_amdgcn_readfirstlane(ring_lds + (t % pf::kStages) * STAGE);
#pragma unroll
    for (int jc = 0; jc < CPW; ++jc) {
      const int ci = wave * CPW + jc;
      const int e = ci * 64 + lane;
      const int r = e / L_::CPR, pos = e - r * L_::CPR;
      const int i = min(s0 + r, T - 1);
      pf::copy16(dst + ci * 1024, qbase + ((size_t)hh * T + i) * L_::ROW + ((pos ^ L_::swz(r)) << 4));
    }
    // the stage's log-sum-exps: 8 rows a wave (lanes 0..7)
    if (lane < 8) {
      const int i = min(s0 + wave * 8 + lane, T - 1);
      pf::copy4(dst + QBYTES + wave * 32, a.lse + row0 + (size_t)hh * T + i);
    }
  };
  f32x4 acc[pf::KB];
#pragma unroll
  for (int kb = 0; kb < pf::KB; ++kb) acc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int first_slot = a.vis_begin + j0;   // the wave's first token's slot
  const int pre = min(pf::kStages - 1, nst);
  for (int t = 0; t < pre; ++t) issue(t);
  for (int t = 0; t < nst; ++t) {
    // this wave's copies of stage t have landed (the later stages it issued may still be in flight)
    pf::wait_vm_steps<OPS, pf::kStages - 2>(min(nst, t + pf::kStages - 1) - t - 1);
    pf::barrier_lds();   // stage t complete for every wave; every wave is past stage t - 1, whose slot is free
    if (t + pf::kStages - 1 < nst) issue(t + pf::kStages - 1);
    const int hh = t / nsh, s0 = istart + (t - hh * nsh) * pf::kRows;
    if (s0 + pf::kRows - 1 < first_slot) continue;   // (wave-uniform) no row of the stage sees the wave's tokens
    const unsigned char* st = ring + (t % pf::kStages) * STAGE;
    const float* lse_s = (const float*)(st + QBYTES);
    // (wave-uniform) every row of the stage is a prompt row past every token of the wave: no per-score test
    const bool inner = s0 >= first_slot + pf::kTokPerWave - 1 && s0 + pf::kRows <= L;
#pragma unroll
    for (int c = 0; c < pf::kRows / 16; ++c) {
      // B operand: lane (col, quad) holds row 16 c + ka_row of the stage (the same order as the keys)
      bf16x8 qf[DS];
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[ds] = *(const bf16x8*)(st + L_::off(16 * c + ka_row, ds * 4 + quad));
      const int i = s0 + 16 * c + ka_row;
      const float lse = lse_s[16 * c + ka_row];
      const bool live = i < L && lse != -INFINITY;
      const float lse2 = live ? lse * 1.4426950408889634f : 0.f;
#pragma unroll
      for (int kb = 0; kb < pf::KB; ++kb) {
        f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kb][ds], qf[ds], sc, 0, 0, 0);
        if (inner) {
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[kb][e] += __builtin_amdgcn_exp2f(fmaf(sc[e], a.scale_log2, -lse2));
        } else if (live) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int slot = first_slot + kb * 16 + e * 4 + quad;
            if (slot <= i) acc[kb][e] += __builtin_amdgcn_exp2f(fmaf(sc[e], a.scale_log2, -lse2));
          }
        }
      }
    }
  }
  pf::wait_vm<0>();   // (copies issued past the last stage land before the workgroup's LDS is released)

  // sum over the 16 row lanes of each quad (fixed order); the outputs of lane (col, quad) are tokens
  // j0 + 16 kb + 4 e + quad
#pragma unroll
  for (int off = 1; off < 16; off <<= 1)
#pragma unroll
    for (int kb = 0; kb < pf::KB; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[kb][e] += __shfl_xor(acc[kb][e], off);
  if (col == 0) {
#pragma unroll
    for (int kb = 0; kb < pf::KB; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = j0 + kb * 16 + e * 4 + quad;
        if (j < a.vis_count)
          store_coherent(a.partial + ((size_t)b * a.Hkv + g) * a.vis_count + j, a.vis_begin + j < L ? acc[kb][e] : 0.f);
      }
  }
  // The last of the sequence's KV heads to finish this block of tokens sums the heads' partials, in head
  // order (device-scope stores and loads; the counter is left at zero for the next call).
  __shared__ int last;
  wait_vector_memory();
  __syncthreads();
  if (tid == 0) {
    uint32_t* ctr = a.counters + ((size_t)b * blocks + blk) * a.counter_stride;
    last = arrive_last(ctr, (uint32_t)a.Hkv);
    if (last) reset_counter(ctr);
  }
  __syncthreads();
  if (!last || tid >= kImpKeys) return;
  const int j = blk * kImpKeys + tid;
  if (j >= a.vis_count) return;
  const float* pp = a.partial + (size_t)b * a.Hkv * a.vis_count + j;
  float sum = 0.f;
  for (int g0 = 0; g0 < a.Hkv; g0 += 8) {
    float x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = g0 + k < a.Hkv ? load_coherent(pp + (size_t)(g0 + k) * a.vis_count) : 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) sum += x[k];
  }
  a.importance[(size_t)b * a.vis_count + j] = L > 0 ? sum / ((float)a.Hq * (float)L) : 0.f;
}

// Order-preserving key of an fp32 value: larger value <=> larger key; -0.0 is taken as +0.0 (they compare
// equal), so equal values always have equal keys.
__device__ __forceinline__ uint32_t order_key(float v) {
  uint32_t u = __builtin_bit_cast(uint32_t, v);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the workgroup's threads (kTopkThreads values, one per thread); *total gets the sum.
__device__ __forceinline__ int block_exclusive_scan(int x, int* scratch, int* total) {
  constexpr int NW = kTopkThreads / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) scratch[wave] = incl;
  __syncthreads();
  int base = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int c = scratch[w];
    base += w < wave ? c : 0;
    sum += c;
  }
  __syncthreads();   // scratch may be reused by the caller
  *total = sum;
  return base + incl - x;
}

// Top-r by radix selection: the r-th largest key K is found digit by digit (8 bits at a time, most
// significant first, histograms in LDS); then every token with a key above K is kept, and of the tokens equal
// to K the first r - #above in token order.  The output is produced in token order by two prefix sums.
__global__ __launch_bounds__(kTopkThreads) void visual_topk_kernel(int n, int r, const float* importance,
                                                                   int32_t* keep) {
  constexpr int PER = kVisualMaxTokens / kTopkThreads;   // tokens per thread, a contiguous run
  __shared__ uint32_t keys[kVisualMaxTokens];
  __shared__ int hist[256];
  __shared__ int scratch[kTopkThreads / 64];
  __shared__ uint32_t sel_prefix;
  __shared__ int sel_rank;
  const int b = blockIdx.x, tid = threadIdx.x;
  const float* v = importance + (size_t)b * n;
  for (int t = tid; t < n; t += kTopkThreads) keys[t] = order_key(v[t]);
  if (tid == 0) {
    sel_prefix = 0u;
    sel_rank = r;   // rank, counted from the top, of the wanted key among the keys matching the prefix
  }
  __syncthreads();
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    const uint32_t prefix = sel_prefix;
    const uint32_t mask = shift == 24 ? 0u : ~0u << (shift + 8);
    for (int t = tid; t < n; t += kTopkThreads) {
      const uint32_t k = keys[t];
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1);
    }
    __syncthreads();
    if (tid < 64) {
      // wave 0 finds the bin holding the wanted rank: lane l owns bins 4l..4l+3; counts above a lane's bins come
      // from a suffix sum over the lanes, and the one lane whose bins hold the rank walks them from the top
      const int rank = sel_rank;
      const int c = hist[4 * tid] + hist[4 * tid + 1] + hist[4 * tid + 2] + hist[4 * tid + 3];
      int suffix = c;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_down(suffix, off);
        if (tid + off < 64) suffix += y;
      }
      const int above_lane = suffix - c;
      if (above_lane < rank && rank <= suffix) {
        int rr = rank - above_lane, d = 4 * tid + 3;
        for (; d > 4 * tid; --d) {
          if (rr <= hist[d]) break;
          rr -= hist[d];
        }
        sel_prefix = prefix | ((uint32_t)d << shift);
        sel_rank = rr;
      }
    }
    __syncthreads();
  }
  const uint32_t K = sel_prefix;
  // tokens equal to K that are kept: the first `need` of them in token order
  const int t0 = tid * PER;
  int above = 0, equal = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int t = t0 + e;
    if (t < n) {
      above += keys[t] > K;
      equal += keys[t] == K;
    }
  }
  int total_above, total_equal;
  block_exclusive_scan(above, scratch, &total_above);
  int eq_rank = block_exclusive_scan(equal, scratch, &total_equal);
  const int need = r - total_above;
  int take = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int t = t0 + e;
    if (t < n) {
      const uint32_t k = keys[t];
      if (k > K) ++take;
      else if (k == K) take += eq_rank++ < need;
    }
  }
  int total;
  int pos = block_exclusive_scan(take, scratch, &total);
  eq_rank -= equal;   // back to this thread's first equal token
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int t = t0 + e;
    if (t < n) {
      const uint32_t k = keys[t];
      const bool kept = k > K || (k == K && eq_rank++ < need);
      if (kept) keep[(size_t)b * r + pos++] = t;
    }
  }
}

// grid (B * Hkv, ceil(r * chunks_per_row / 256)); a kept token outside the cache leaves its rows unwritten
__global__ __launch_bounds__(256) void visual_gather_kernel(VisualGatherArgs a) {
  const int bg = blockIdx.x, b = bg / a.Hkv;
  const int cpr = a.row_bytes / 16;
  const long long e = (long long)blockIdx.y * 256 + threadIdx.x;
  if (e >= (long long)a.r * cpr) return;
  const int m = (int)(e / cpr), c = (int)(e - (long long)m * cpr);
  const int slot = a.vis_begin + a.keep[(size_t)b * a.r + m];
  if (slot < 0 || slot >= a.S_cap) return;
  const size_t src = ((size_t)bg * a.S_cap + slot) * a.row_bytes + (size_t)c * 16;
  const size_t dst = ((size_t)bg * a.r + m) * a.row_bytes + (size_t)c * 16;
  *(u32x4*)((unsigned char*)a.k_out + dst) = *(const u32x4*)((const unsigned char*)a.k + src);
  *(u32x4*)((unsigned char*)a.v_out + dst) = *(const u32x4*)((const unsigned char*)a.v + src);
}

}  // namespace

template <int D>
hipError_t launch_importance_prefill(const VisualArgs& a, dim3 grid, hipStream_t stream) {
  constexpr size_t lds = (size_t)pf::kStages * (pf::kRows * D * 2 + pf::kRows * 4);
  static bool configured = false;
  if (!configured) {
    hipError_t e = hipFuncSetAttribute((const void*)visual_importance_prefill_kernel<D>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    configured = true;
  }
  hipLaunchKernelGGL(visual_importance_prefill_kernel<D>, grid, dim3(64 * pf::kWaves), lds, stream, a);
  return hipGetLastError();
}

hipError_t launch_visual_importance(const VisualArgs& a, hipStream_t stream) {
  const int blocks = (a.vis_count + kImpKeys - 1) / kImpKeys;
  const dim3 grid((unsigned)(a.B * a.Hkv * blocks));
  if (a.prefill) {
    if (a.D == 128) return launch_importance_prefill<128>(a, grid, stream);
    if (a.D == 64) return launch_importance_prefill<64>(a, grid, stream);
    return hipErrorInvalidValue;
  }
  if (a.D == 128) hipLaunchKernelGGL(visual_importance_kernel<128>, grid, dim3(256), 0, stream, a);
  else if (a.D == 64) hipLaunchKernelGGL(visual_importance_kernel<64>, grid, dim3(256), 0, stream, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_visual_topk(int B, int n, int r, const float* importance, int32_t* keep, hipStream_t stream) {
  if (n > kVisualMaxTokens || r > n || r < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(visual_topk_kernel, dim3(B), dim3(kTopkThreads), 0, stream, n, r, importance, keep);
  return hipGetLastError();
}

hipError_t launch_visual_gather(const VisualGatherArgs& a, hipStream_t stream) {
  const long long per = (long long)a.r * (a.row_bytes / 16);
  hipLaunchKernelGGL(visual_gather_kernel, dim3(a.B * a.Hkv, (unsigned)((per + 255) / 256)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dreams

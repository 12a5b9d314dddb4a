// Greedy acceptance straight from the target's final hidden states: the LM head fused with the argmax, so the
// logits never reach HBM (the paper's Section 2, "Speculative decoding": the target's token at a position is
// the argmax of its logits there; the logits are the final hidden state times the LM head's weight).
//
// lm_head_argmax_kernel: a workgroup of 8 waves per (64-row tile, 128-entry vocabulary tile) of the logits,
// row tiles fastest; wave w owns the tile's vocabulary entries 16 w .. 16 w + 15 over the whole hidden axis.
// Each wave streams its 16 weight rows through a private LDS ring (LDS-DMA copies of whole 128-byte row pieces,
// several 64-deep stages ahead), and the tile's 64 hidden rows go through LDS once for all eight waves.  The
// products run on v_mfma_f32_16x16x32_bf16 with the weights as the A operand, so that a lane's four outputs are
// four vocabulary entries of one row.  Each row's best (value, index) over the tile's entries is written:
// ties go to the smallest index (fp32 comparison, -0.0 equal to +0.0), as for logits held in memory.
// lm_head_argmax_big_kernel (more than 64 rows): 256 vocabulary entries by 128 or 256 rows per workgroup, both
// operands through a shared LDS ring (see below).
// lm_head_finish_kernel: a workgroup of 16 waves per sequence merges every row's candidates over the tiles
// (the row's argmax; 4 rows a wave with all their loads in flight) and one wave runs the greedy path scan on
// them.
#include "accept_scan.h"
#include "kernels.h"

#include <limits.h>
#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = kLmThreads, NW = NT / 64;

// true iff (v2, i2) beats (v1, i1): larger value, or equal value and smaller index
__device__ __forceinline__ bool better(float v2, int i2, float v1, int i1) {
  return v2 > v1 || (v2 == v1 && i2 < i1);
}

typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(lds_void*)p; }
// Wave-wide 16-byte copy from global memory into LDS: lane l's 16 bytes land at LDS byte address m0 + 16 l
// (m0 wave-uniform).  STREAM adds the non-temporal hint, for data read once (the 64-row kernel's weights);
// operands that other workgroups read again (the large tiles') are copied without it (gqa_long's shape:
// 2.34 ms with the hint, 1.82 ms without).
template <bool STREAM>
__device__ __forceinline__ void copy16_to_lds(uint32_t m0, const void* src) {
  if (STREAM)
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off nt" ::"s"(m0), "v"(src) : "memory");
  else
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(m0), "v"(src) : "memory");
}
// At most N of this wave's vector-memory operations still outstanding (they complete in issue order).
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
// Workgroup barrier after this wave's LDS reads have returned; outstanding copies stay in flight (a
// __syncthreads() would also wait for them).  The wait is the compiler's own instruction (vmcnt and expcnt at
// their maxima, lgkmcnt 0), so its bookkeeping knows every LDS read issued before the barrier has returned.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Large row counts: a workgroup per (64 WR rows, 64 WN vocabulary entries), WR x WN waves as blocks of
// 64 x 64 products, both operands staged in a shared LDS ring (a stage: 64 WN weight rows and 64 WR hidden
// rows x 64 hidden entries, copied by all waves together), STAGES - 1 stages ahead; one barrier per stage
// hands a landed stage to every wave and frees the oldest.  Each operand tile is read from the caches once
// per 64 WR rows or 64 WN entries instead of once per 64.

constexpr int FIN_THREADS = 1024, FIN_WAVES = FIN_THREADS / 64, FIN_PER = 4, FIN_ROWS = 4;

__device__ __forceinline__ void best_of_batch(const float* pv, const int* px, int p0, int n, int lane, float& v,
                                              int& x) {
  float cv[FIN_PER];
  int cx[FIN_PER];
#pragma unroll
  for (int k = 0; k < FIN_PER; ++k) {
    const int p = min(p0 + k * 64 + lane, n - 1);
    cv[k] = pv[p];
    cx[k] = px[p];
  }
#pragma unroll
  for (int k = 0; k < FIN_PER; ++k)
    if (p0 + k * 64 + lane < n && better(cv[k], cx[k], v, x)) {
      v = cv[k];
      x = cx[k];
    }
}
__device__ __forceinline__ void wave_best(float& v, int& x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float v2 = __shfl_xor(v, off);
    const int x2 = __shfl_xor(x, off);
    if (better(v2, x2, v, x)) {
      v = v2;
      x = x2;
    }
  }
}

__global__ __launch_bounds__(FIN_THREADS) void lm_head_finish_kernel(LmHeadArgs a) {
  __shared__ int am_s[kMaxNodes], tok_s[kMaxNodes], par_s[kMaxNodes];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int b = blockIdx.x, T = a.T, n = a.ntiles;
  if ((int)threadIdx.x < T) {
    tok_s[threadIdx.x] = a.tokens[(size_t)b * T + threadIdx.x];
    par_s[threadIdx.x] = a.parent[(size_t)b * T + threadIdx.x];
  }
  // FIN_ROWS rows a wave at a time (rows past T read row T - 1 and are dropped), every load of a batch in
  // flight together: up to 64 rows in one round of memory latency
  for (int i0 = wave; i0 < T; i0 += FIN_ROWS * FIN_WAVES) {
    float v[FIN_ROWS];
    int x[FIN_ROWS];
#pragma unroll
    for (int r = 0; r < FIN_ROWS; ++r) {
      v[r] = -INFINITY;
      x[r] = INT_MAX;
    }
    for (int p0 = 0; p0 < n; p0 += FIN_PER * 64) {
#pragma unroll
      for (int r = 0; r < FIN_ROWS; ++r) {
        const size_t ri = (size_t)b * T + min(i0 + r * FIN_WAVES, T - 1);
        best_of_batch(a.part_val + ri * n, a.part_idx + ri * n, p0, n, lane, v[r], x[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < FIN_ROWS; ++r) {
      const int i = i0 + r * FIN_WAVES;
      wave_best(v[r], x[r]);
      if (lane == 0 && i < T) {
        am_s[i] = x[r];
        if (a.target_argmax) a.target_argmax[(size_t)b * T + i] = x[r];
      }
    }
  }
  __syncthreads();
  if (wave == 0)
    path_scan_wave(am_s, tok_s, par_s, T, a.accept_len + b, a.accept_path + (size_t)b * T, a.next_token + b);
}

// The 64-row kernel.  A stage is 64 hidden entries (128 bytes of a row).  Per stage, each wave copies its 16
// weight rows into its ring slot (two wave-wide LDS-DMA copies of 8 rows x 128 bytes) and loads 16 bytes of the
// tile's hidden rows per thread into registers (thread t: row t / 8, chunk t % 8); a stage's hidden rows are
// written to one of three shared LDS buffers one stage before they are used, and a barrier publishes them.
// Every vector-memory operation of the loop is issued by inline assembly and waited for by exact count: a
// stage is issued DW - 1 stages ahead, and at stage s the wave waits for stage s + 1, leaving DW - 2 stages of
// copies in flight.  The 16-byte chunk c of a row r sits at position c ^ (r % 8) of its 128-byte LDS row, so
// that the 16 rows one operand read touches fall on distinct banks.
constexpr int LM_WAVES = kLmTileSmall / 16, LM_SK = 64, LM_DW = 8, LM_XBUF = 3;
constexpr int LM_WSLOT = 16 * LM_SK * 2, LM_XSTAGE = kLmTile * LM_SK * 2;
constexpr size_t LM_LDS = (size_t)LM_WAVES * LM_DW * LM_WSLOT + (size_t)LM_XBUF * LM_XSTAGE;

__device__ __forceinline__ void load16_async(bf16x8& dst, const void* src) {
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(dst) : "v"(src) : "memory");
}
// wait until at most N of this wave's vector-memory operations are outstanding; x (the data of a load issued
// before them) is tied to the wait, so that no use of it is scheduled ahead of it
template <int N>
__device__ __forceinline__ void wait_vm_tied(bf16x8& x) {
  asm volatile("s_waitcnt vmcnt(%1)" : "+v"(x) : "n"(N) : "memory");
}

__global__ __launch_bounds__(64 * LM_WAVES) void lm_head_argmax_kernel(LmHeadArgs a) {
  static_assert(kLmTile == 64 && LM_WAVES == 8, "64 rows; eight waves, each owning 16 vocabulary entries");
  static_assert(LM_LDS + 2 * LM_WAVES * kLmTile * 4 <= 160 * 1024, "LDS budget");
  extern __shared__ __attribute__((aligned(1024))) char lm_lds[];
  char* wring = lm_lds;                                         // [wave][DW][16 rows x 128 B]
  char* xs = lm_lds + (size_t)LM_WAVES * LM_DW * LM_WSLOT;      // [3][64 rows x 128 B]
  __shared__ float best_v[LM_WAVES][kLmTile];
  __shared__ int best_i[LM_WAVES][kLmTile];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, quad = lane >> 4;
  // the row tiles of one vocabulary tile are consecutive workgroups, so its weights are fetched from HBM once
  // and found in the caches by the others
  const int mt = blockIdx.x % a.mtiles, nt = blockIdx.x / a.mtiles;
  const int n0 = nt * kLmTileSmall + 16 * wave, m0 = mt * kLmTile;
  const int H = a.H, nstages = H / LM_SK;
  // weight copies: copy j brings rows 8 j + lane / 8 of the wave's 16 (clamped past the vocabulary: their
  // results are discarded), chunk position lane % 8, i.e. the row's chunk (lane % 8) ^ (row % 8)
  const int crow = lane >> 3, cchunk = (lane & 7) ^ (crow & 7);
  const __bf16* wsrc0 = a.weight + (size_t)min(n0 + crow, a.V - 1) * H + 8 * cchunk;
  const __bf16* wsrc1 = a.weight + (size_t)min(n0 + 8 + crow, a.V - 1) * H + 8 * cchunk;
  const uint32_t wring_lds = __builtin_amdgcn_readfirstlane(lds_addr(wring + (size_t)wave * LM_DW * LM_WSLOT));
  // hidden piece of this thread: row t / 8 (clamped past the rows), chunk t % 8, written at c ^ (r % 8)
  const int xr = threadIdx.x >> 3, xc = threadIdx.x & 7;
  const __bf16* xsrc = a.hidden + (size_t)min(m0 + xr, a.M - 1) * H + 8 * xc;
  const int xw = xr * 128 + ((xc ^ (xr & 7)) << 4);

  bf16x8 hv[LM_DW];
  auto issue = [&](int slot, int s) {
    const int k = min(s, nstages - 1) * LM_SK;   // (stages past the end repeat the last one, unused)
    const uint32_t dst = wring_lds + slot * LM_WSLOT;
    copy16_to_lds<true>(dst, wsrc0 + k);
    copy16_to_lds<true>(dst + 1024, wsrc1 + k);
    load16_async(hv[slot], xsrc + k);
  };
  f32x4 acc[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) acc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int slot, int s) {
    const char* wst = wring + ((size_t)wave * LM_DW + slot) * LM_WSLOT;
    const char* xst = xs + (size_t)(s % LM_XBUF) * LM_XSTAGE;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = 4 * ks + quad;
      const bf16x8 wa = *(const bf16x8*)(wst + col * 128 + ((c ^ (col & 7)) << 4));
      bf16x8 xb[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) xb[r] = *(const bf16x8*)(xst + (16 * r + col) * 128 + ((c ^ (col & 7)) << 4));
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, xb[r], acc[r], 0, 0, 0);
    }
  };
#pragma unroll
  for (int j = 0; j < LM_DW - 1; ++j) issue(j, j);
  wait_vm_tied<3 * (LM_DW - 2)>(hv[0]);   // stage 0 has landed
  *(bf16x8*)(xs + xw) = hv[0];
  // Stage s: its slot's registers and ring slot take stage s + DW - 1 (the slot held stage s - 1, whose
  // weights were read by this wave's products and whose hidden rows went to LDS before); stage s + 1 lands and
  // its hidden rows go to their LDS buffer; the barrier publishes them and retires every wave's reads of the
  // buffer stage s + 2 will take; then stage s is computed.
  for (int s0 = 0; s0 < nstages; s0 += LM_DW) {
#pragma unroll
    for (int j = 0; j < LM_DW; ++j) {
      const int s = s0 + j;
      if (s >= nstages) break;
      issue((j + LM_DW - 1) % LM_DW, s + LM_DW - 1);
      wait_vm_tied<3 * (LM_DW - 2)>(hv[(j + 1) % LM_DW]);
      *(bf16x8*)(xs + (size_t)((s + 1) % LM_XBUF) * LM_XSTAGE + xw) = hv[(j + 1) % LM_DW];
      barrier_lds();
      compute(j, s);
    }
  }
  wait_vm<0>();   // copies issued past the last stage land before the workgroup's LDS is released

  // lane (col, quad) of wave w: rows 16 r + col, vocabulary entries n0 + 4 quad + e
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float v = -INFINITY;
    int x = INT_MAX;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int n = n0 + 4 * quad + e;
      if (n < a.V && (acc[r][e] > v || x == INT_MAX)) {
        v = acc[r][e];
        x = n;
      }
    }
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float v2 = __shfl_xor(v, off);
      const int x2 = __shfl_xor(x, off);
      if (better(v2, x2, v, x)) {
        v = v2;
        x = x2;
      }
    }
    if (quad == 0) {
      best_v[wave][16 * r + col] = v;
      best_i[wave][16 * r + col] = x;
    }
  }
  __syncthreads();
  // each row's best over the tile's sub-tiles, in vocabulary order
  if (threadIdx.x < kLmTile && m0 + (int)threadIdx.x < a.M) {
    const int row = threadIdx.x;
    float v = best_v[0][row];
    int x = best_i[0][row];
#pragma unroll
    for (int w = 1; w < LM_WAVES; ++w)
      if (better(best_v[w][row], best_i[w][row], v, x)) {
        v = best_v[w][row];
        x = best_i[w][row];
      }
    const size_t p = (size_t)(m0 + row) * a.ntiles + nt;
    a.part_val[p] = v;
    a.part_idx[p] = x;
  }
}

template <int WR, int WN, int TW, int SK, int STAGES>
__global__ __launch_bounds__(64 * WR * WN) void lm_head_argmax_big_kernel(LmHeadArgs a) {
  // a stage holds SK hidden entries of each of the tile's rows: RB bytes per row, CPR 16-byte chunks, chunk c
  // of row r at position c ^ swz(r) (the 16 rows of one operand read on distinct banks)
  constexpr int BIG_M = 64 * WR, WB = 16 * TW, BN = WB * WN, WAVES = WR * WN;
  constexpr int RB = SK * 2, CPR = SK / 8, RPC = 1024 / RB, KS = SK / 32, STAGE = (BN + BIG_M) * RB;
  constexpr int CPW = (BN + BIG_M) / RPC / WAVES;   // wave-wide copies (RPC rows each) per wave per stage
  static_assert(CPW * RPC * WAVES == BN + BIG_M, "the copies cover the stage");
  static_assert(SK == 64 || SK == 32, "64 or 32 hidden entries per stage");
  auto swz = [](int r) { return SK == 64 ? (r & 7) : ((r >> 2) & 3); };
  __shared__ __attribute__((aligned(16))) char ring[STAGES][STAGE];   // [stage][W rows | X rows]
  __shared__ float best_v[WN][BIG_M];
  __shared__ int best_i[WN][BIG_M];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, quad = lane >> 4;
  const int wr = wave / WN, wn = wave % WN;   // this wave's 64 rows and WB vocabulary entries of the tile
  const int mt = blockIdx.x % a.mtiles, nt = blockIdx.x / a.mtiles;
  const int n0 = nt * BN, m0 = mt * BIG_M;
  const int H = a.H, nstages = H / SK;

  // copies: copy q = CPW wave + j of a stage moves rows RPC q .. (weight rows first, then hidden rows); lane
  // l takes row RPC q + l / CPR, position l % CPR, i.e. the logical chunk that position holds
  const int crow = lane / CPR, cchunk = (lane % CPR) ^ swz(crow);
  const __bf16* csrc[CPW];
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    const int q = CPW * wave + j;
    csrc[j] = q < BN / RPC ? a.weight + (size_t)min(n0 + RPC * q + crow, a.V - 1) * H + 8 * cchunk
                           : a.hidden + (size_t)min(m0 + RPC * (q - BN / RPC) + crow, a.M - 1) * H + 8 * cchunk;
  }
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(lds_addr(&ring[0][0]));
  auto issue = [&](int s) {
    const uint32_t dst = ring_lds + (s % STAGES) * STAGE + wave * CPW * 1024;
#pragma unroll
    for (int j = 0; j < CPW; ++j) copy16_to_lds<false>(dst + j * 1024, csrc[j] + s * SK);
  };
  f32x4 acc[TW][4];
#pragma unroll
  for (int t = 0; t < TW; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[t][r] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < STAGES - 1 && s < nstages; ++s) issue(s);
  for (int s = 0; s < nstages; ++s) {
    // this wave's copies of stage s have landed (later stages may stay in flight), then every wave's have
    wait_vm_steps<CPW, STAGES - 2>(min(STAGES - 2, nstages - 1 - s));
    barrier_lds();
    // every wave is past stage s - 1: its slot takes stage s + STAGES - 1
    if (s + STAGES - 1 < nstages) issue(s + STAGES - 1);
    const char* wst = &ring[s % STAGES][0];
    const char* xst = wst + BN * RB;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 wa[TW], xb[4];
      const int c = 4 * ks + quad;
#pragma unroll
      for (int t = 0; t < TW; ++t) {
        const int rw = WB * wn + 16 * t + col;
        wa[t] = *(const bf16x8*)(wst + rw * RB + ((c ^ swz(rw)) << 4));
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int rx = 64 * wr + 16 * t + col;
        xb[t] = *(const bf16x8*)(xst + rx * RB + ((c ^ swz(rx)) << 4));
      }
#pragma unroll
      for (int t = 0; t < TW; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[t][r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[t], xb[r], acc[t][r], 0, 0, 0);
    }
  }

  // each row's best over this wave's WB entries (lane: rows 64 wr + 16 r + col, entries
  // n0 + WB wn + 16 t + 4 quad + e, visited in increasing order), then over the WN vocabulary blocks
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float v = -INFINITY;
    int x = INT_MAX;
#pragma unroll
    for (int t = 0; t < TW; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int n = n0 + WB * wn + 16 * t + 4 * quad + e;
        if (n < a.V && (acc[t][r][e] > v || x == INT_MAX)) {
          v = acc[t][r][e];
          x = n;
        }
      }
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float v2 = __shfl_xor(v, off);
      const int x2 = __shfl_xor(x, off);
      if (better(v2, x2, v, x)) {
        v = v2;
        x = x2;
      }
    }
    if (quad == 0) {
      best_v[wn][64 * wr + 16 * r + col] = v;
      best_i[wn][64 * wr + 16 * r + col] = x;
    }
  }
  __syncthreads();
  if (threadIdx.x < BIG_M && m0 + (int)threadIdx.x < a.M) {
    const int row = threadIdx.x;
    float v = best_v[0][row];
    int x = best_i[0][row];
#pragma unroll
    for (int w = 1; w < WN; ++w)
      if (better(best_v[w][row], best_i[w][row], v, x)) {
        v = best_v[w][row];
        x = best_i[w][row];
      }
    const size_t p = (size_t)(m0 + row) * a.ntiles + nt;
    a.part_val[p] = v;
    a.part_idx[p] = x;
  }
}

// Each row's best over every tile, then the greedy path scan: a workgroup of 16 waves per sequence; wave w
// merges rows w, w + 16, ..., two rows at a time with all of both rows' candidates in flight (up to 8 per lane
// per row, then the next batch).
}  // namespace

hipError_t launch_lm_head_accept(const LmHeadArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)((long long)a.ntiles * a.mtiles));
  static_assert(kLmTileBig == 256, "four vocabulary waves");
  if (a.rows == kLmBigRows)
    hipLaunchKernelGGL((lm_head_argmax_big_kernel<4, 4, 4, 64, 2>), grid, dim3(1024), 0, stream, a);
  else if (a.rows == kLmMidRows)
    hipLaunchKernelGGL((lm_head_argmax_big_kernel<2, 4, 4, 64, 3>), grid, dim3(512), 0, stream, a);
  else {
    static bool configured = false;
    if (!configured) {
      hipError_t e = hipFuncSetAttribute((const void*)lm_head_argmax_kernel,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)LM_LDS);
      if (e != hipSuccess) return e;
      configured = true;
    }
    hipLaunchKernelGGL(lm_head_argmax_kernel, grid, dim3(64 * LM_WAVES), LM_LDS, stream, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lm_head_finish_kernel, dim3((unsigned)a.B), dim3(FIN_THREADS), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dreams

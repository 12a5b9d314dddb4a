// Greedy acceptance straight from the target's final hidden states: the LM head fused with the argmax, so the
// logits never reach HBM (the paper's Section 2, "Speculative decoding": the target's token at a position is
// the argmax of its logits there; the logits are the final hidden state times the LM head's weight).
//
// lm_head_argmax_kernel: a workgroup per (64-row tile, 64-entry vocabulary tile) of the logits, row tiles
// fastest, four waves splitting the hidden axis in quarters.  A wave streams its quarter of the tile's 64
// weight rows through a private two-stage LDS ring (LDS-DMA copies of whole 128-byte row pieces, non-temporal)
// and reads the 64 hidden rows' operands straight from global memory (they stay in the caches); the products
// run on v_mfma_f32_16x16x32_bf16 with the weights as the A operand, so that a lane's four outputs are four
// vocabulary entries of one row.  The four partial sums are added through LDS in wave order (each wave then owns 16
// vocabulary entries of the tile), and each row's best (value, index) over the tile's 64 entries is written:
// ties go to the smallest index (fp32 comparison, -0.0 equal to +0.0), as for logits held in memory.
// lm_head_argmax_big_kernel (more than 64 rows): 256 vocabulary entries by 128 or 256 rows per workgroup, both
// operands through a shared LDS ring (see below).
// lm_head_finish_kernel: a workgroup of 16 waves per sequence merges every row's candidates over the tiles
// (the row's argmax) and one wave runs the greedy path scan on them.
#include "accept_scan.h"
#include "kernels.h"

#include <limits.h>
#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = kLmThreads, NW = NT / 64, TILE = kLmTile;

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

// A stage is 64 weight rows x 64 hidden entries (128 bytes per row, 8 KB), copied by 8 wave-wide copies of
// 8 rows each; 16-byte chunk c of row r sits at position c ^ (r % 8) of the row, so that the 16 rows one
// operand read touches fall on distinct banks (each copy lane fetches the chunk its position wants).
constexpr int STAGE_K = 64, STAGE_BYTES = TILE * STAGE_K * 2, STAGES = 2;

__global__ __launch_bounds__(NT) void lm_head_argmax_kernel(LmHeadArgs a) {
  static_assert(NW == 4 && TILE == 64, "four waves, each owning 16 of the tile's 64 vocabulary entries");
  static_assert(NW * STAGES * STAGE_BYTES >= NW * 16 * 64 * 16, "the partial sums reuse the copy rings");
  __shared__ __attribute__((aligned(16))) char ring[NW][STAGES][STAGE_BYTES];   // one ring per wave
  __shared__ float best_v[NW][TILE];
  __shared__ int best_i[NW][TILE];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, quad = lane >> 4;
  // the row tiles of one vocabulary tile are consecutive workgroups, so its weights are fetched from HBM
  // once and found in the caches by the others
  const int mt = blockIdx.x % a.mtiles, nt = blockIdx.x / a.mtiles;
  const int n0 = nt * TILE, m0 = mt * TILE;
  const int H = a.H, KQ = H / NW, k0 = wave * KQ, nstages = KQ / STAGE_K;

  // copy lanes: copy j moves rows 8 j + lane / 8, chunk position lane % 8 (logical chunk cpos ^ row % 8)
  const int crow = lane >> 3, cchunk = (lane & 7) ^ (crow & 7);
  const __bf16* csrc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
    csrc[j] = a.weight + (size_t)min(n0 + 8 * j + crow, a.V - 1) * H + k0 + 8 * cchunk;
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(lds_addr(&ring[wave][0][0]));
  auto issue = [&](int s) {   // the copies of stage s into ring slot s % STAGES
    const uint32_t dst = ring_lds + (s % STAGES) * STAGE_BYTES;
#pragma unroll
    for (int j = 0; j < 8; ++j) copy16_to_lds<true>(dst + j * 1024, csrc[j] + s * STAGE_K);
  };
  // hidden operand rows (clamped; their results are discarded below), read straight from global memory
  const __bf16* xrow[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) xrow[r] = a.hidden + (size_t)min(m0 + 16 * r + col, a.M - 1) * H + k0 + quad * 8;

  f32x4 acc[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[t][r] = f32x4{0.f, 0.f, 0.f, 0.f};
  // The hidden operands are loaded one stage ahead, before that stage's copies: the wait for stage s (at most
  // 8 operations outstanding) then leaves exactly stage s + 1's copies in flight, which is also the wait the
  // compiler derives for the hidden registers from the loads it can see.  The loop is unrolled by two so that
  // the two register sets swap roles without copies (a copy would make the compiler wait for everything).
  bf16x8 xa[2][4], xb[2][4];
  auto load_hidden = [&](int s, bf16x8 (&dst)[2][4]) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int r = 0; r < 4; ++r) dst[ks][r] = *(const bf16x8*)(xrow[r] + s * STAGE_K + 32 * ks);
  };
  auto compute = [&](int s, const bf16x8 (&x)[2][4]) {
    const char* st = &ring[wave][s % STAGES][0];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 wa[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int r = 16 * t + col, c = 4 * ks + quad;
        wa[t] = *(const bf16x8*)(st + r * 128 + ((c ^ (r & 7)) << 4));
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[t][r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[t], x[ks][r], acc[t][r], 0, 0, 0);
    }
  };
  issue(0);
  load_hidden(0, xa);
  int s = 0;
  for (; s + 2 < nstages; s += 2) {
    load_hidden(s + 1, xb);
    issue(s + 1);
    wait_vm<8>();
    compute(s, xa);
    load_hidden(s + 2, xa);
    issue(s + 2);
    wait_vm<8>();
    compute(s + 1, xb);
  }
  if (s + 1 < nstages) {   // two stages left
    load_hidden(s + 1, xb);
    issue(s + 1);
    wait_vm<8>();
    compute(s, xa);
    wait_vm<0>();
    compute(s + 1, xb);
  } else {                 // one stage left
    wait_vm<0>();
    compute(s, xa);
  }
  __syncthreads();   // every wave is done with its ring: the partial sums reuse it
  f32x4 (*red)[16][64] = (f32x4(*)[16][64])&ring[0][0][0];

  // sum the four quarters: wave w owns vocabulary sub-tile w; the others' partials of it come through LDS
  f32x4 own[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (t == wave) own[r] = acc[t][r];
      else red[wave][t * 4 + r][lane] = acc[t][r];
    }
  __syncthreads();
  // lane (col, quad) of wave w: rows 16 r + col, vocabulary entries n0 + 16 w + 4 quad + e
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int src = 0; src < NW; ++src) s += src == wave ? own[r] : red[src][wave * 4 + r][lane];
    float v = -INFINITY;
    int x = INT_MAX;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int n = n0 + 16 * wave + 4 * quad + e;
      if (n < a.V && (s[e] > v || x == INT_MAX)) {
        v = s[e];
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
  // each row's best over the tile's four sub-tiles, in vocabulary order
  if (threadIdx.x < TILE && m0 + (int)threadIdx.x < a.M) {
    const int row = threadIdx.x;
    float v = best_v[0][row];
    int x = best_i[0][row];
#pragma unroll
    for (int w = 1; w < NW; ++w)
      if (better(best_v[w][row], best_i[w][row], v, x)) {
        v = best_v[w][row];
        x = best_i[w][row];
      }
    const size_t p = (size_t)(m0 + row) * a.ntiles + nt;
    a.part_val[p] = v;
    a.part_idx[p] = x;
  }
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
constexpr int FIN_THREADS = 1024, FIN_WAVES = FIN_THREADS / 64, FIN_PER = 8;

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
  for (int i = wave; i < T; i += 2 * FIN_WAVES) {
    const int j = i + FIN_WAVES;   // the second row of the pair (may be past T)
    const size_t ri = (size_t)b * T + i, rj = (size_t)b * T + min(j, T - 1);
    float vi = -INFINITY, vj = -INFINITY;
    int xi = INT_MAX, xj = INT_MAX;
    for (int p0 = 0; p0 < n; p0 += FIN_PER * 64) {
      best_of_batch(a.part_val + ri * n, a.part_idx + ri * n, p0, n, lane, vi, xi);
      best_of_batch(a.part_val + rj * n, a.part_idx + rj * n, p0, n, lane, vj, xj);
    }
    wave_best(vi, xi);
    wave_best(vj, xj);
    if (lane == 0) {
      am_s[i] = xi;
      if (a.target_argmax) a.target_argmax[ri] = xi;
      if (j < T) {
        am_s[j] = xj;
        if (a.target_argmax) a.target_argmax[rj] = xj;
      }
    }
  }
  __syncthreads();
  if (wave == 0)
    path_scan_wave(am_s, tok_s, par_s, T, a.accept_len + b, a.accept_path + (size_t)b * T, a.next_token + b);
}

}  // namespace

hipError_t launch_lm_head_accept(const LmHeadArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)((long long)a.ntiles * a.mtiles));
  static_assert(kLmTileBig == 256, "four vocabulary waves");
  if (a.rows == kLmBigRows)
    hipLaunchKernelGGL((lm_head_argmax_big_kernel<4, 4, 4, 64, 2>), grid, dim3(1024), 0, stream, a);
  else if (a.rows == kLmMidRows)
    hipLaunchKernelGGL((lm_head_argmax_big_kernel<2, 4, 4, 64, 3>), grid, dim3(512), 0, stream, a);
  else
    hipLaunchKernelGGL(lm_head_argmax_kernel, grid, dim3(NT), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lm_head_finish_kernel, dim3((unsigned)a.B), dim3(FIN_THREADS), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dreams

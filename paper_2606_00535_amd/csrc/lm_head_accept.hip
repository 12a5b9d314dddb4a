// Greedy acceptance straight from the target's final hidden states: the LM head fused with the argmax, so the
// logits never reach HBM (the paper's Section 2, "Speculative decoding": the target's token at a position is
// the argmax of its logits there; the logits are the final hidden state times the LM head's weight).
//
// lm_head_argmax_kernel: a workgroup per (64-entry vocabulary tile, 64-row tile) of the logits, four waves
// splitting the hidden axis in quarters.  A wave streams its quarter of the tile's 64 weight rows and 64 hidden
// rows with 16-byte loads straight into matrix-core operands (v_mfma_f32_16x16x32_bf16, weights as the A
// operand, so that a lane's four outputs are four vocabulary entries of one row; the weights, read once, with
// the non-temporal hint).  The four partial sums are added through LDS in wave order (each wave then owns 16
// vocabulary entries of the tile), and each row's best (value, index) over the tile's 64 entries is written:
// ties go to the smallest index (fp32 comparison, -0.0 equal to +0.0), as for logits held in memory.
// lm_head_finish_kernel: a workgroup per sequence; wave w merges rows w, w + 4, ... over every tile, then one
// wave runs the greedy path scan.
#include "accept_scan.h"
#include "kernels.h"

#include <limits.h>
#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = kLmThreads, NW = NT / 64, TILE = kLmTile;
constexpr int U = 2;   // 32-deep steps per batch of loads

// true iff (v2, i2) beats (v1, i1): larger value, or equal value and smaller index
__device__ __forceinline__ bool better(float v2, int i2, float v1, int i1) {
  return v2 > v1 || (v2 == v1 && i2 < i1);
}

__global__ __launch_bounds__(NT) void lm_head_argmax_kernel(LmHeadArgs a) {
  static_assert(NW == 4 && TILE == 64, "four waves, each owning 16 of the tile's 64 vocabulary entries");
  __shared__ f32x4 red[NW][16][64];   // [source wave][vocab sub-tile * 4 + row sub-tile][lane]
  __shared__ float best_v[NW][TILE];
  __shared__ int best_i[NW][TILE];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, quad = lane >> 4;
  const int n0 = blockIdx.x * TILE, m0 = blockIdx.y * TILE;
  const int H = a.H, KQ = H / NW, k0 = wave * KQ;

  // operand rows, clamped into the tensors (results of clamped rows are discarded below)
  const __bf16* wrow[4];
  const __bf16* xrow[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    wrow[t] = a.weight + (size_t)min(n0 + 16 * t + col, a.V - 1) * H + k0 + quad * 8;
    xrow[t] = a.hidden + (size_t)min(m0 + 16 * t + col, a.M - 1) * H + k0 + quad * 8;
  }
  f32x4 acc[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[t][r] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < KQ; k += 32 * U) {
    bf16x8 wa[U][4], xb[U][4];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        wa[u][t] = __builtin_nontemporal_load((const bf16x8*)(wrow[t] + k + 32 * u));
        xb[u][t] = *(const bf16x8*)(xrow[t] + k + 32 * u);
      }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[t][r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[u][t], xb[u][r], acc[t][r], 0, 0, 0);
  }

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
    const size_t p = (size_t)(m0 + row) * a.ntiles + blockIdx.x;
    a.part_val[p] = v;
    a.part_idx[p] = x;
  }
}

__global__ __launch_bounds__(NT) void lm_head_finish_kernel(LmHeadArgs a) {
  __shared__ int am_s[kMaxNodes], tok_s[kMaxNodes], par_s[kMaxNodes];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int b = blockIdx.x, T = a.T;
  if ((int)threadIdx.x < T) {
    tok_s[threadIdx.x] = a.tokens[(size_t)b * T + threadIdx.x];
    par_s[threadIdx.x] = a.parent[(size_t)b * T + threadIdx.x];
  }
  for (int i = wave; i < T; i += NW) {
    const size_t row = (size_t)b * T + i;
    const float* pv = a.part_val + row * a.ntiles;
    const int* px = a.part_idx + row * a.ntiles;
    float v = -INFINITY;
    int x = INT_MAX;
    for (int p0 = 0; p0 < a.ntiles; p0 += 4 * 64) {   // four candidates per lane in flight
      float cv[4];
      int cx[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int p = min(p0 + k * 64 + lane, a.ntiles - 1);
        cv[k] = pv[p];
        cx[k] = px[p];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (p0 + k * 64 + lane < a.ntiles && better(cv[k], cx[k], v, x)) {
          v = cv[k];
          x = cx[k];
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float v2 = __shfl_xor(v, off);
      const int x2 = __shfl_xor(x, off);
      if (better(v2, x2, v, x)) {
        v = v2;
        x = x2;
      }
    }
    if (lane == 0) {
      am_s[i] = x;
      if (a.target_argmax) a.target_argmax[row] = x;
    }
  }
  __syncthreads();
  if (wave == 0)
    path_scan_wave(am_s, tok_s, par_s, T, a.accept_len + b, a.accept_path + (size_t)b * T, a.next_token + b);
}

}  // namespace

hipError_t launch_lm_head_accept(const LmHeadArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)a.ntiles, (unsigned)((a.M + TILE - 1) / TILE));
  hipLaunchKernelGGL(lm_head_argmax_kernel, grid, dim3(NT), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lm_head_finish_kernel, dim3((unsigned)a.B), dim3(NT), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dreams

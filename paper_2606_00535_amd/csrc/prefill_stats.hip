// Attention statistics of a prompt's own causal attention (the prefilling pass), where the paper reads them:
// AE(l) of Section 3.2 averages the entropy of a layer's attention rows over the n prompt tokens, and Eq. 2 of
// Section 3.1 scores the visual tokens with the final layer's attention of the prefill.  Row i of query head h
// attends the prompt's slots 0..i (the decoder's causal mask):
//     lse[h,i]     = log sum_{j <= i} exp(scale * q_i . k_j)
//     entropy[h,i] = -sum_{j <= i} A[h,i,j] log A[h,i,j],   A[h,i,j] = exp(scale * q_i . k_j - lse[h,i]).
// No value product is needed, so this is half of a causal attention forward.
//
//   * prefill_stats_kernel: a workgroup of 4 waves owns 256 query rows of one query head; a wave owns 64 rows
//     as four 16-row matrix-core B operands (its queries stay in registers) and walks the keys 0 .. its last
//     row in 16-key blocks, S^T = K Q^T on v_mfma_f32_16x16x32_bf16 with the key rows as the A operand (16-byte
//     loads straight from global memory; the four row blocks share them).  Each lane keeps, for each of its 4
//     rows, the online (max, sum, entropy term) over the keys its quad sees, in log2 units; the four quads are
//     merged at the end.  Only the blocks that cross the diagonal are masked.  Workgroups are ordered from the
//     last rows (the most keys) to the first.
//   * prefill_entropy_mean_kernel: one workgroup, the fp64 mean of the prompt rows' entropies over every head
//     and sequence (rows i >= n_b hold 0 and do not count).
#include "kernels.h"

#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kRowsPerWave = 64;
constexpr int kWaves = 4;
constexpr int kRowsPerWg = kRowsPerWave * kWaves;
constexpr int kKeyUnroll = 2;   // 16-key blocks whose loads are in flight together

// A state (m, l, e) in log2 units: l = sum 2^(z-m), e = sum 2^(z-m) (z-m).  Re-referenced to M >= m with weight
// w = 2^(m-M): l -> w l, e -> w (e + (m-M) l).
__device__ __forceinline__ void rescale(float& m, float& l, float& e, float M) {
  if (m == M) return;
  const float w = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
  e = w == 0.f ? 0.f : w * fmaf(m - M, l, e);
  l *= w;
  m = M;
}

template <int D>
__global__ __launch_bounds__(64 * kWaves) void prefill_stats_kernel(PrefillArgs a) {
  constexpr int DS = D / 32;
  constexpr int RB = kRowsPerWave / 16;
  const int nblk = (a.N + kRowsPerWg - 1) / kRowsPerWg;
  const int n = blockIdx.x;
  const int blk = nblk - 1 - n % nblk;   // the row blocks with the most keys first
  const int bh = n / nblk;
  const int h = bh % a.Hq, b = bh / a.Hq;
  const int g = h / a.G;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, quad = lane >> 4;
  int nb = a.prompt_len[b];
  nb = nb < 0 ? 0 : (nb > a.N ? a.N : nb);

  const int r0 = blk * kRowsPerWg + wave * kRowsPerWave;   // the wave's first row
  const size_t qrow0 = ((size_t)b * a.Hq + h) * a.N;
  const unsigned char* qbase = (const unsigned char*)a.q + qrow0 * (D * 2);
  const unsigned char* kbase = (const unsigned char*)a.k + ((size_t)b * a.Hkv + g) * a.S_cap * (D * 2);

  bf16x8 qf[RB][DS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = min(r0 + rb * 16 + col, a.N - 1);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = *(const bf16x8*)(qbase + (size_t)row * (D * 2) + (ds * 32 + quad * 8) * 2);
  }
  float m[RB], l[RB], e[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m[rb] = -INFINITY;
    l[rb] = 0.f;
    e[rb] = 0.f;
  }
  // a lane's scores of row rb are keys kk0 + 4*quad + {0..3} of row r0 + 16*rb + col
  const float c = a.scale_log2;
  const int kend = min(r0 + kRowsPerWave, nb);   // keys any of the wave's live rows can see
  const int nkb = (kend + 15) / 16;
  auto block = [&](const bf16x8 (&kf)[DS], int kk0) {
    f32x4 s[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) s[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) s[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ds], qf[rb][ds], s[rb], 0, 0, 0);
    const bool edge = kk0 + 16 > r0 || kk0 + 16 > nb;   // (wave-uniform) the block crosses a row or the prompt end
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = r0 + rb * 16 + col;
      float z[4];
      float zmax = -INFINITY;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = kk0 + quad * 4 + t;
        z[t] = s[rb][t] * c;
        if (edge && (key > row || key >= nb)) z[t] = -INFINITY;
        zmax = fmaxf(zmax, z[t]);
      }
      if (zmax > m[rb]) rescale(m[rb], l[rb], e[rb], zmax);
      if (m[rb] != -INFINITY) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const float d = z[t] - m[rb];
          const float p = __builtin_amdgcn_exp2f(d);
          l[rb] += p;
          e[rb] = fmaf(p, fmaxf(d, -1.0e4f), e[rb]);   // (a masked key: p = 0, and its term stays 0)
        }
      }
    }
  };
  // keys in 16-key blocks, kKeyUnroll blocks' loads in flight together
  for (int kb0 = 0; kb0 < nkb; kb0 += kKeyUnroll) {
    bf16x8 kf[kKeyUnroll][DS];
#pragma unroll
    for (int u = 0; u < kKeyUnroll; ++u) {
      const int key = min((kb0 + u) * 16 + col, a.S_cap - 1);
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[u][ds] = *(const bf16x8*)(kbase + (size_t)key * (D * 2) + (ds * 32 + quad * 8) * 2);
    }
#pragma unroll
    for (int u = 0; u < kKeyUnroll; ++u)
      if (kb0 + u < nkb) block(kf[u], (kb0 + u) * 16);
  }
  // merge the four quads' states of every row (fixed order: xor 16, then xor 32)
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float mo = __shfl_xor(m[rb], off), lo = __shfl_xor(l[rb], off), eo = __shfl_xor(e[rb], off);
      const float M = fmaxf(m[rb], mo);
      float m1 = m[rb], l1 = l[rb], e1 = e[rb], m2 = mo, l2 = lo, e2 = eo;
      if (M != -INFINITY) {
        rescale(m1, l1, e1, M);
        rescale(m2, l2, e2, M);
      }
      m[rb] = M;
      l[rb] = l1 + l2;
      e[rb] = e1 + e2;
    }
    const int row = r0 + rb * 16 + col;
    if (quad == 0 && row < a.N) {
      const bool live = row < nb && l[rb] > 0.f;
      if (a.lse) a.lse[qrow0 + row] = live ? (m[rb] + __log2f(l[rb])) * 0.69314718055994530942f : -INFINITY;
      if (a.entropy) a.entropy[qrow0 + row] = live ? 0.69314718055994530942f * (__log2f(l[rb]) - e[rb] / l[rb]) : 0.f;
    }
  }
}

// Mean of the prompt rows' entropies: sum over [B, Hq, N] (rows past n_b hold 0) / (Hq * sum_b n_b), fp64, in a
// fixed order (each thread a fixed stride of rows, then a tree over the threads).
__global__ __launch_bounds__(1024) void prefill_entropy_mean_kernel(int B, int Hq, int N, const float* entropy,
                                                                    const int32_t* prompt_len, float* ae) {
  __shared__ double part[1024];
  const long long total = (long long)B * Hq * N;
  double s = 0.0;
  for (long long i = threadIdx.x; i < total; i += blockDim.x) s += (double)entropy[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    long long rows = 0;
    for (int b = 0; b < B; ++b) {
      const int nb = prompt_len[b];
      rows += nb < 0 ? 0 : (nb > N ? N : nb);
    }
    *ae = rows > 0 ? (float)(part[0] / ((double)Hq * (double)rows)) : 0.f;
  }
}

}  // namespace

hipError_t launch_prefill_stats(const PrefillArgs& a, hipStream_t stream) {
  const long long grid = (long long)a.B * a.Hq * ((a.N + kRowsPerWg - 1) / kRowsPerWg);
  if (grid <= 0) return hipSuccess;
  if (a.D == 128) hipLaunchKernelGGL(prefill_stats_kernel<128>, dim3((unsigned)grid), dim3(64 * kWaves), 0, stream, a);
  else if (a.D == 64) hipLaunchKernelGGL(prefill_stats_kernel<64>, dim3((unsigned)grid), dim3(64 * kWaves), 0, stream, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_prefill_entropy_mean(int B, int Hq, int N, const float* entropy, const int32_t* prompt_len, float* ae,
                                       hipStream_t stream) {
  hipLaunchKernelGGL(prefill_entropy_mean_kernel, dim3(1), dim3(1024), 0, stream, B, Hq, N, entropy, prompt_len, ae);
  return hipGetLastError();
}

}  // namespace dreams

// Attention statistics of a prompt's own causal attention (the prefilling pass), where the paper reads them:
// AE(l) of Section 3.2 averages the entropy of a layer's attention rows over the n prompt tokens, and Eq. 2 of
// Section 3.1 scores the visual tokens with the final layer's attention of the prefill.  Row i of query head h
// attends the prompt's slots 0..i (the decoder's causal mask):
//     lse[h,i]     = log sum_{j <= i} exp(scale * q_i . k_j)
//     entropy[h,i] = -sum_{j <= i} A[h,i,j] log A[h,i,j],   A[h,i,j] = exp(scale * q_i . k_j - lse[h,i]).
// No value product is needed, so this is half of a causal attention forward.
//
//   * prefill_stats_kernel: a workgroup of 8 waves owns 256 query rows of one query head; a wave owns 32 rows
//     as two 16-row matrix-core B operands (its queries stay in registers).  The prompt's keys 0 .. the
//     workgroup's last row stream through an LDS ring of 64-key stages (LDS-DMA copies, several stages ahead)
//     that all eight waves read: S^T = K Q^T on v_mfma_f32_16x16x32_bf16 with the key rows as the A operand.
//     Each lane keeps, for each of its 2 rows, an online (reference, sum, entropy term) over the keys its
//     quad sees, in log2 units; the reference only moves when a score passes it by more than 2^8 (the sums
//     stay finite and the statistics do not depend on it), and the four quads are merged at the end.  Only
//     16-key blocks that cross the diagonal or the prompt's end are masked.  Workgroups are ordered so that
//     the row blocks with the most keys start first and share a compute unit with those with the fewest.
//   * prefill_entropy_mean_kernel: one workgroup, the fp64 mean of the prompt rows' entropies over every head
//     and sequence (rows i >= n_b hold 0 and do not count).
#include "kernels.h"

#include <math.h>

namespace dreams {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kRB = 2;                        // 16-row blocks per wave
constexpr int kRowsPerWave = 16 * kRB;
constexpr int kRowsPerWg = kRowsPerWave * kWaves;
constexpr int kKeys = 64;                     // keys per ring stage
constexpr int kStages = 4;                    // ring stages
constexpr float kLazyLog2 = 8.0f;             // slack of the reference before it moves

// Key rows in LDS: rows of D bf16, the 16-byte chunk c of row r at position c ^ swz(r), which puts the 16 rows
// of one operand read (rows (m%4)*4 + m/4 of a 16-row block, one chunk) on distinct banks.
template <int D>
struct KRows {
  static constexpr int ROW = D * 2, CPR = D / 8, RPL = 256 / ROW;
  static __device__ __forceinline__ int swz(int r) {
    if constexpr (D == 128) return ((r >> 2) & 3) * 4 + (r & 1) * 2 + 1;
    return (r / RPL) % CPR;
  }
  static __device__ __forceinline__ int off(int r, int c) { return r * ROW + ((c ^ swz(r)) << 4); }
};

typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(lds_void*)p; }
// wave-wide 16-byte copy into LDS: lane l's 16 bytes land at m0 + 16 l (m0 wave-uniform)
__device__ __forceinline__ void copy16_to_lds(uint32_t m0, const void* src) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(m0), "v"(src) : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// 16-byte load into registers, issued like the copies (so that a wait for it can leave later copies in flight)
__device__ __forceinline__ void load16(bf16x8& dst, const void* src) {
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(dst) : "v"(src) : "memory");
}
// at most N vector-memory operations of this wave outstanding; the registers loaded before them are tied to the
// wait (one statement for all of them, so that no use or copy of any is scheduled ahead of it)
template <int N>
__device__ __forceinline__ void wait_vm_tied(bf16x8 (&x)[4]) {
  asm volatile("s_waitcnt vmcnt(%4)" : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]) : "n"(N) : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm_tied(bf16x8 (&x)[2][4]) {
  asm volatile("s_waitcnt vmcnt(%8)"
               : "+v"(x[0][0]), "+v"(x[0][1]), "+v"(x[0][2]), "+v"(x[0][3]), "+v"(x[1][0]), "+v"(x[1][1]),
                 "+v"(x[1][2]), "+v"(x[1][3])
               : "n"(N)
               : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm_tied(bf16x8 (&x)[2][2]) {
  asm volatile("s_waitcnt vmcnt(%4)" : "+v"(x[0][0]), "+v"(x[0][1]), "+v"(x[1][0]), "+v"(x[1][1]) : "n"(N) : "memory");
}
// at most k * PER of this wave's copies outstanding (k <= K)
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
// workgroup barrier once this wave's LDS accesses are done; copies stay in flight
__device__ __forceinline__ void barrier_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// A state (m, l, e) in log2 units: l = sum 2^(z-m), e = sum 2^(z-m) (z-m).  Re-referenced to M with weight
// w = 2^(m-M): l -> w l, e -> w (e + (m-M) l).
__device__ __forceinline__ void rescale(float& m, float& l, float& e, float M) {
  if (m == M) return;
  const float w = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
  e = w == 0.f ? 0.f : w * fmaf(m - M, l, e);
  l *= w;
  m = M;
}

template <int D>
__global__ __launch_bounds__(64 * kWaves, 2) void prefill_stats_kernel(PrefillArgs a) {
  using L = KRows<D>;
  constexpr int DS = D / 32;
  constexpr int STAGE = kKeys * L::ROW;          // bytes of a stage
  constexpr int CPW = STAGE / 1024 / kWaves;     // wave-wide 1 KB copies per wave per stage
  static_assert(CPW >= 1 && CPW * 1024 * kWaves == STAGE, "copy split");
  extern __shared__ __attribute__((aligned(1024))) unsigned char ring[];   // kStages x STAGE
  // Workgroup order: row blocks with the most keys first, one per compute unit; the workgroups beyond the
  // first round (which share a compute unit with one of the first) take the blocks in the opposite order, so
  // that the longest block is paired with the shortest.
  const int nblk = (a.N + kRowsPerWg - 1) / kRowsPerWg, BH = a.B * a.Hq;
  const int n = blockIdx.x, W = gridDim.x;
  const int rank = (n >= a.cus && W <= 2 * a.cus) ? W - 1 - (n - a.cus) : n;
  const int blk = nblk - 1 - rank / BH;
  const int bh = rank - (rank / BH) * BH;
  const int h = bh % a.Hq, b = bh / a.Hq;
  const int g = h / a.G;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, quad = lane >> 4;
  int nb = __builtin_amdgcn_readfirstlane(a.prompt_len[b]);
  nb = nb < 0 ? 0 : (nb > a.N ? a.N : nb);

  const int r0 = blk * kRowsPerWg;                  // the workgroup's first row
  const int rw0 = r0 + wave * kRowsPerWave;         // the wave's first row
  const size_t qrow0 = ((size_t)b * a.Hq + h) * a.N;
  const unsigned char* kbase = (const unsigned char*)a.k + ((size_t)b * a.Hkv + g) * a.S_cap * L::ROW;
  const int kend = min(r0 + kRowsPerWg, nb);        // keys any live row of the workgroup can see
  const int nst = kend > 0 ? (kend + kKeys - 1) / kKeys : 0;
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane(lds_addr(ring));

  // copies of stage st: 1 KB block ci = wave * CPW + j; lane l brings row r = (ci * 1024 + 16 l) / ROW of the
  // stage, position l % CPR, i.e. the key row's chunk (l % CPR) ^ swz(r); rows past the cache repeat its last
  auto issue = [&](int st) {
    const uint32_t dst = __builtin_amdgcn_readfirstlane(ring_lds + (st % kStages) * STAGE);
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const int ci = wave * CPW + j;
      const int e = ci * 64 + lane;
      const int r = e / L::CPR, p = e - r * L::CPR;
      const int key = min(st * kKeys + r, a.S_cap - 1);
      copy16_to_lds(dst + ci * 1024, kbase + (size_t)key * L::ROW + ((p ^ L::swz(r)) << 4));
    }
  };
  // queries first (registers), then the first stages' copies; the wait for the queries leaves those in flight
  bf16x8 qf[kRB][DS];
  const unsigned char* qbase = (const unsigned char*)a.q + qrow0 * L::ROW;
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    const int row = min(rw0 + rb * 16 + col, a.N - 1);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) load16(qf[rb][ds], qbase + (size_t)row * L::ROW + (ds * 32 + quad * 8) * 2);
  }
  // always kStages - 1 stages (past the last one they repeat it, unread), so that the wait count is fixed
  for (int st = 0; st < kStages - 1; ++st) issue(min(st, max(nst - 1, 0)));
  wait_vm_tied<(kStages - 1) * CPW>(qf);
  // scores are scaled by c = |scale| log2(e) inside the exponent; a negative scale flips the queries' signs
  // (exact in bf16)
  const float c = fabsf(a.scale_log2);
  if (a.scale_log2 < 0.f) {
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, qf[rb][ds]) ^ 0x80008000u);
  }

  float m[kRB], l[kRB], e[kRB];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    m[rb] = -INFINITY;
    l[rb] = 0.f;
    e[rb] = 0.f;
  }
  const int ka_row = (col & 3) * 4 + (col >> 2);   // A row m holds key kb*16 + (m%4)*4 + m/4
  const int wlast = min(rw0 + kRowsPerWave, nb) - 1;   // the wave's last live row (< rw0: none)

  // a 16-key block: lane (col, quad) gets keys kk0 + 4 t + quad (t = 0..3) of rows rw0 + 16 rb + col
  auto block = [&](const unsigned char* tile, int kb, int kk0) {
    bf16x8 kf[DS];
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) kf[ds] = *(const bf16x8*)(tile + L::off(kb * 16 + ka_row, ds * 4 + quad));
    f32x4 s[kRB];
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) s[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) s[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ds], qf[rb][ds], s[rb], 0, 0, 0);
    const bool edge = kk0 + 15 > rw0 || kk0 + 16 > nb;   // (wave-uniform) a key past some row or the prompt
    if (!edge) {
      // every key visible: the reference moves (rarely) when a score passes it by more than 2^8, then each
      // score costs one fma, one exp2, one add and one fma
      float zmax[kRB];
      bool grow = false;
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) {
        zmax[rb] = c * vmax(vmax(s[rb][0], s[rb][1]), vmax(s[rb][2], s[rb][3]));
        grow |= zmax[rb] > m[rb] + kLazyLog2;
      }
      if (__any(grow)) {
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb)
          if (zmax[rb] > m[rb] + kLazyLog2) rescale(m[rb], l[rb], e[rb], zmax[rb]);
      }
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const float d = fmaf(s[rb][t], c, -m[rb]);
          const float p = __builtin_amdgcn_exp2f(d);
          l[rb] += p;
          e[rb] = fmaf(p, d, e[rb]);
        }
      }
      return;
    }
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
      float z[4];
      const int row = rw0 + rb * 16 + col;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = kk0 + 4 * t + quad;
        z[t] = (key > row || key >= nb) ? -INFINITY : s[rb][t] * c;
      }
      const float zmax = vmax(vmax(z[0], z[1]), vmax(z[2], z[3]));
      if (zmax > m[rb] + kLazyLog2) rescale(m[rb], l[rb], e[rb], zmax);
      if (m[rb] != -INFINITY) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const float d = fmaxf(z[t] - m[rb], -1.0e4f);   // (a masked key: p = 0 and a zero term)
          const float p = __builtin_amdgcn_exp2f(d);
          l[rb] += p;
          e[rb] = fmaf(p, d, e[rb]);
        }
      }
    }
  };

  for (int st = 0; st < nst; ++st) {
    // this wave's copies of stage st have landed (the later stages it issued may still be in flight)
    wait_vm_steps<CPW, kStages - 2>(min(nst, max(st + kStages - 1, kStages - 1)) - st - 1);
    barrier_lds();   // stage st complete for every wave; every wave is past stage st - 1, whose slot is free
    if (st + kStages - 1 < nst) issue(st + kStages - 1);
    const unsigned char* tile = ring + (st % kStages) * STAGE;
#pragma unroll
    for (int kb = 0; kb < kKeys / 16; ++kb) {
      const int kk0 = st * kKeys + kb * 16;
      if (kk0 > wlast) break;   // (wave-uniform) no live row of this wave sees these keys
      block(tile, kb, kk0);
    }
  }

  wait_vm<0>();   // (a workgroup with no live row has not waited for its first copies)

  // merge the four quads' states of every row (fixed order: xor 16, then xor 32)
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
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
    const int row = rw0 + rb * 16 + col;
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

template <int D>
hipError_t launch_stats(const PrefillArgs& a, unsigned grid, hipStream_t stream) {
  constexpr size_t lds = (size_t)kStages * kKeys * D * 2;
  static bool configured = false;
  if (!configured) {
    hipError_t e = hipFuncSetAttribute((const void*)prefill_stats_kernel<D>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
    configured = true;
  }
  hipLaunchKernelGGL(prefill_stats_kernel<D>, dim3(grid), dim3(64 * kWaves), lds, stream, a);
  return hipGetLastError();
}

hipError_t launch_prefill_stats(const PrefillArgs& a, hipStream_t stream) {
  const long long grid = (long long)a.B * a.Hq * ((a.N + kRowsPerWg - 1) / kRowsPerWg);
  if (grid <= 0) return hipSuccess;
  if (a.D == 128) return launch_stats<128>(a, (unsigned)grid, stream);
  if (a.D == 64) return launch_stats<64>(a, (unsigned)grid, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_prefill_entropy_mean(int B, int Hq, int N, const float* entropy, const int32_t* prompt_len, float* ae,
                                       hipStream_t stream) {
  hipLaunchKernelGGL(prefill_entropy_mean_kernel, dim3(1), dim3(1024), 0, stream, B, Hq, N, entropy, prompt_len, ae);
  return hipGetLastError();
}

}  // namespace dreams

// Tree-masked verification attention, fp32 inputs (the small fp32 workload; latency-bound, so plain VALU).
//
// One workgroup per output row (sequence b, query head h, node i): NTH threads, thread t visiting keys t,
// t + NTH, ... of the visible set, each key's K and V rows loaded whole (16-byte loads, all in flight together),
// so that a row's keys take only ceil(N / NTH) dependent rounds of memory latency.  Each thread keeps its own
// online softmax (running max, running sum, D-wide accumulator) in fp32; the states are merged pairwise with
// the log-sum-exp identity, first within each wave (butterfly over lanes), then across the waves in wave order
// through LDS, so the merge order is fixed and results are reproducible.  The sequence's parents are copied to
// LDS and walked there for node i's ancestors.  With an entropy output, each state also carries
// e = sum 2^(x-m) (x-m) (scores x in log2 units), from which the row's attention entropy follows as
// ln2 * (log2 l - e/l); re-referencing a state to M with weight w = 2^(m-M) turns e into w (e + (m-M) l).
#include "kernels.h"

#include <math.h>

namespace dreams {
namespace {

constexpr float kLn2 = 0.69314718055994530942f;

__device__ __forceinline__ float ent_term(float w, float e, float m, float M, float l) {
  return w == 0.f ? 0.f : w * fmaf(m - M, l, e);
}

// threads per row: D = 64 holds a key's K and V rows and the accumulator in about 200 registers (two waves a
// SIMD), D = 128 in about 400 (one)
template <int D>
constexpr int f32_threads() { return D == 64 ? 512 : 256; }

template <int D>
__global__ __launch_bounds__(f32_threads<D>()) void tree_attn_f32_kernel(AttnArgs a) {
  constexpr int NTH = f32_threads<D>(), NW = NTH / 64, V4 = D / 4;
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  __shared__ f32x4 q_lds[V4];
  __shared__ int par_lds[kMaxNodes];
  __shared__ uint64_t anc_lds[2];
  __shared__ float st_mle[NW][3];
  __shared__ float st_acc[NW][D];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T;
  const int r = blockIdx.x;                       // ((b * Hq) + h) * T + i
  const int i = r % T, bh = r / T;
  const int h = bh % a.Hq, b = bh / a.Hq;
  const int g = h / a.G;
  int L = a.kv_len[b];
  L = L < 0 ? 0 : (L > a.S_cap - T ? a.S_cap - T : L);
  const int N = L + T;

  // the query row and the sequence's parents into LDS; node i's ancestors-or-self (a walk in LDS, or the mask)
  const f32x4* qrow = (const f32x4*)((const float*)a.q + (size_t)r * D);
  for (int t = tid; t < V4; t += NTH) q_lds[t] = qrow[t];
  if (!a.mask)
    for (int t = tid; t < T; t += NTH) par_lds[t] = a.parent[(size_t)b * T + t];
  __syncthreads();
  if (tid == 0) {
    uint64_t anc0 = 0, anc1 = 0;
    if (a.mask) {
      const int W = (T + 63) / 64;
      const uint64_t* mr = a.mask + ((size_t)b * T + i) * W;
      anc0 = mr[0];
      anc1 = W > 1 ? mr[1] : 0;
    } else {
      int j = i;
      for (int step = 0; step <= T && j >= 0; ++step) {
        if (j < 64) anc0 |= 1ull << j; else anc1 |= 1ull << (j - 64);
        const int p = par_lds[j];
        if (p >= j) break;
        j = p;
      }
    }
    anc_lds[0] = anc0;
    anc_lds[1] = anc1;
  }
  __syncthreads();
  const uint64_t anc0 = anc_lds[0], anc1 = anc_lds[1];

  const float* kb = (const float*)a.k + ((size_t)b * a.Hkv + g) * a.S_cap * D;
  const float* vb = (const float*)a.v + ((size_t)b * a.Hkv + g) * a.S_cap * D;
  const bool ent = a.entropy != nullptr;
  float m = -INFINITY, l = 0.f, e = 0.f;
  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.f;

  for (int s = tid; s < N; s += NTH) {
    if (s >= L) {
      const int j = s - L;
      if ((((j < 64) ? anc0 >> j : anc1 >> (j - 64)) & 1ull) == 0) continue;
    }
    const f32x4* kr = (const f32x4*)(kb + (size_t)s * D);
    const f32x4* vr = (const f32x4*)(vb + (size_t)s * D);
    f32x4 kk[V4], vv[V4];
#pragma unroll
    for (int c = 0; c < V4; ++c) kk[c] = kr[c];
#pragma unroll
    for (int c = 0; c < V4; ++c) vv[c] = vr[c];
    float dot = 0.f;
#pragma unroll
    for (int c = 0; c < V4; ++c) {
      const f32x4 q = q_lds[c];
      dot = fmaf(q[0], kk[c][0], dot);
      dot = fmaf(q[1], kk[c][1], dot);
      dot = fmaf(q[2], kk[c][2], dot);
      dot = fmaf(q[3], kk[c][3], dot);
    }
    const float x = dot * a.scale_log2;
    const float m_new = fmaxf(m, x);
    const float alpha = exp2f(m - m_new);
    const float p = exp2f(x - m_new);
    if (ent) e = ent_term(l == 0.f ? 0.f : alpha, e, m, m_new, l) + p * (x - m_new);
    l = l * alpha + p;
#pragma unroll
    for (int c = 0; c < V4; ++c)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[4 * c + t] = fmaf(p, vv[c][t], acc[4 * c + t] * alpha);
    m = m_new;
  }

  // within the wave: butterfly over the lanes (every lane ends with the wave's state)
  for (int off = 32; off >= 1; off >>= 1) {
    const float mo = __shfl_xor(m, off);
    const float lo = __shfl_xor(l, off);
    const float eo = __shfl_xor(e, off);
    const float M = fmaxf(m, mo);
    const float w = M == -INFINITY ? 0.f : exp2f(m - M);
    const float wo = M == -INFINITY ? 0.f : exp2f(mo - M);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const float ao = __shfl_xor(acc[d], off);
      acc[d] = acc[d] * w + ao * wo;
    }
    if (ent) e = ent_term(w, e, m, M, l) + ent_term(wo, eo, mo, M, lo);
    l = l * w + lo * wo;
    m = M;
  }
  // across the waves, in wave order: every wave's state through LDS, merged by wave 0 (lane d % 64 owns
  // output column d)
  if (lane == 0) {
    st_mle[wave][0] = m;
    st_mle[wave][1] = l;
    st_mle[wave][2] = e;
  }
  // (every lane holds the same state: lane l stores columns l, 64 + l, ... -- selected without branches)
#pragma unroll
  for (int k = 0; k < D / 64; ++k) {
    float own = 0.f;
#pragma unroll
    for (int d = 0; d < 64; ++d) own = lane == d ? acc[64 * k + d] : own;
    st_acc[wave][64 * k + lane] = own;
  }
  __syncthreads();
  if (wave != 0) return;
  float M = st_mle[0][0];
#pragma unroll
  for (int w = 1; w < NW; ++w) M = fmaxf(M, st_mle[w][0]);
  float lt = 0.f, et = 0.f, o[D / 64];
#pragma unroll
  for (int k = 0; k < D / 64; ++k) o[k] = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const float mw = st_mle[w][0], lw = st_mle[w][1], ew = st_mle[w][2];
    const float wt = M == -INFINITY ? 0.f : exp2f(mw - M);
    if (ent) et += ent_term(wt, ew, mw, M, lw);
    lt = fmaf(lw, wt, lt);
#pragma unroll
    for (int k = 0; k < D / 64; ++k) o[k] = fmaf(st_acc[w][64 * k + lane], wt, o[k]);
  }

  const float inv = lt > 0.f ? 1.0f / lt : 0.f;
  float* orow = (float*)a.out + (size_t)r * D;
#pragma unroll
  for (int k = 0; k < D / 64; ++k) orow[64 * k + lane] = o[k] * inv;
  if (a.lse && lane == 0) a.lse[r] = lt > 0.f ? (M + log2f(lt)) * kLn2 : -INFINITY;
  if (ent && lane == 0) a.entropy[r] = lt > 0.f ? kLn2 * (log2f(lt) - et / lt) : 0.f;
}

}  // namespace

hipError_t launch_tree_attn_f32(const AttnArgs& a, hipStream_t stream) {
  const int rows = a.B * a.Hq * a.T;
  if (a.D == 64) {
    hipLaunchKernelGGL(tree_attn_f32_kernel<64>, dim3(rows), dim3(f32_threads<64>()), 0, stream, a);
  } else if (a.D == 128) {
    hipLaunchKernelGGL(tree_attn_f32_kernel<128>, dim3(rows), dim3(f32_threads<128>()), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dreams

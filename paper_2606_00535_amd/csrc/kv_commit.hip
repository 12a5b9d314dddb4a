// KV commit: move the accepted path's K/V rows into the next contiguous cache slots.
//
// Slot L+k receives slot L+path[k] for k = 0..a.  A node at depth k has k ancestors with smaller indices,
// so path[k] >= k: every source lies at or after its destination.  A destination can still be another
// row's source (path = [0, 2, 5]: slot L+2 is read for k = 1 and written for k = 2), so each pass first
// gathers all of its rows into LDS and only then scatters them.  Passes over k run in increasing order;
// a later pass only reads slots >= its own k, which no earlier pass wrote.  Rows with path[k] == k need no
// move and are skipped.  One workgroup per (layer, sequence, KV head); copies are bitwise (16-byte words).
#include "kernels.h"

namespace dreams {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kCommitThreads) void kv_commit_kernel(CommitArgs a) {
  constexpr int RW = kCommitRowsPerPass;
  constexpr int MAXW = kCommitMaxRowBytes / 16;
  __shared__ u32x4 kbuf[RW * MAXW];
  __shared__ u32x4 vbuf[RW * MAXW];

  const int n = blockIdx.x;                  // (layer * B + b) * Hkv + g
  const int g = n % a.Hkv;
  const int lb = n / a.Hkv;
  const int b = lb % a.B, layer = lb / a.B;
  const int L = a.kv_len_in[b];
  int A = a.accept_len[b];
  A = A < 0 ? 0 : (A > a.path_stride - 1 ? a.path_stride - 1 : A);
  if (layer == 0 && g == 0 && threadIdx.x == 0) a.kv_len_out[b] = L + A + 1;
  if (L < 0) return;

  const int words = a.row_bytes / 16;
  const size_t head = (size_t)layer * a.layer_stride_bytes + ((size_t)b * a.Hkv + g) * a.S_cap * (size_t)a.row_bytes;
  char* kc = a.k + head;
  char* vc = a.v + head;
  const int32_t* path = a.path + (size_t)b * a.path_stride;

  for (int k0 = 0; k0 <= A; k0 += RW) {
    const int rows = min(RW, A + 1 - k0);
    for (int e = threadIdx.x; e < rows * words; e += kCommitThreads) {
      const int r = e / words, w = e - r * words;
      const int k = k0 + r;
      const int src = path[k];
      if (src > k && (long long)L + src < a.S_cap) {
        kbuf[r * MAXW + w] = *(const u32x4*)(kc + (size_t)(L + src) * a.row_bytes + w * 16);
        vbuf[r * MAXW + w] = *(const u32x4*)(vc + (size_t)(L + src) * a.row_bytes + w * 16);
      }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < rows * words; e += kCommitThreads) {
      const int r = e / words, w = e - r * words;
      const int k = k0 + r;
      const int src = path[k];
      if (src > k && (long long)L + src < a.S_cap) {
        *(u32x4*)(kc + (size_t)(L + k) * a.row_bytes + w * 16) = kbuf[r * MAXW + w];
        *(u32x4*)(vc + (size_t)(L + k) * a.row_bytes + w * 16) = vbuf[r * MAXW + w];
      }
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_kv_commit(const CommitArgs& a, hipStream_t stream) {
  const long long grid = (long long)a.NL * a.B * a.Hkv;
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(kv_commit_kernel, dim3((unsigned)grid), dim3(kCommitThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dreams

// Path scan of greedy acceptance, shared by the kernels that end in it (logits in HBM, or the LM head's).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dreams {

// Run by one whole wave.  am_s, tok_s, par_s: LDS arrays of the T nodes' target token, draft token and parent
// (T <= 128).  Writes accept_len, next_token (lane 0) and the T entries of accept_path.
__device__ inline void path_scan_wave(const int* am_s, const int* tok_s, const int* par_s, int T,
                                      int32_t* accept_len, int32_t* path, int32_t* next_token) {
  const int lane = threadIdx.x & 63;
  // A sweep from the root, one depth per round (lane l holds nodes l and l + 64).
  // A node joins the consistent set when its draft equals the target's token at its parent and the parent
  // joined the round before; the set lives in two 64-bit wave-uniform masks grown by ballots.  The last
  // non-empty round holds the deepest consistent nodes: the smallest index among them is `last`, the number
  // of rounds its depth.
  int par_h[2];
  bool ok_h[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = lane + 64 * h;
    const int p = i < T ? par_s[i] : -1;
    par_h[h] = p;
    ok_h[h] = i > 0 && i < T && p >= 0 && p < i && tok_s[i] == am_s[p];
  }
  auto in_set = [](uint64_t s0, uint64_t s1, int x) {
    return (((x < 64 ? s0 : s1) >> (x & 63)) & 1ull) != 0;
  };
  uint64_t c0 = 1, c1 = 0;      // the root is always consistent
  uint64_t l0 = 1, l1 = 0;      // the last round's new members
  int depth = 0;
  while (true) {
    const bool j0 = ok_h[0] && !in_set(c0, c1, lane) && in_set(c0, c1, par_h[0]);
    const bool j1 = ok_h[1] && !in_set(c0, c1, lane + 64) && in_set(c0, c1, par_h[1]);
    const uint64_t n0 = __ballot(j0), n1 = __ballot(j1);
    if ((n0 | n1) == 0) break;
    c0 |= n0;
    c1 |= n1;
    l0 = n0;
    l1 = n1;
    ++depth;
  }
  const int last = l0 ? __builtin_ctzll(l0) : 64 + __builtin_ctzll(l1);
  const int alen = depth;
  if (lane == 0) {
    *accept_len = alen;
    *next_token = am_s[last];
  }
  // the path from the root to `last`, read off the parents held in the lanes (uniform steps, no LDS)
  int j = last;
  for (int k = alen; k >= 0; --k) {
    if (lane == 0) path[k] = j;
    j = j < 64 ? __builtin_amdgcn_readlane(par_h[0], j) : __builtin_amdgcn_readlane(par_h[1], j - 64);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = lane + 64 * h;
    if (i > alen && i < T) path[i] = -1;
  }
}

}  // namespace dreams

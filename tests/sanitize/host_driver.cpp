// Drives the host layer of libdreams.so (csrc/dreams_api.hip: argument checks, work planning, workspace sizes,
// status text) for a build with the host address and undefined-behaviour sanitizers.  Nothing here touches a
// device: every call either answers from the arguments alone or fails its checks before anything is enqueued.
// Exit status 0 on success.
#include <stdio.h>
#include <string.h>

#include "dreams.h"

#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond);     \
      return 1;                                                              \
    }                                                                        \
  } while (0)

static dreams_attn_desc_t desc(int B, int Hq, int Hkv, int D, int T, int S, int max_len, int splits, dreams_dtype_t dt) {
  dreams_attn_desc_t d;
  d.batch = B; d.num_q_heads = Hq; d.num_kv_heads = Hkv; d.head_dim = D; d.num_nodes = T;
  d.cache_capacity = S; d.max_kv_len = max_len; d.num_splits = splits; d.dtype = dt; d.scale = 0.088f;
  return d;
}

int main() {
  for (int s = 0; s >= -6; --s) CHECK(dreams_status_string((dreams_status_t)s) != nullptr);
  CHECK(strcmp(dreams_last_error_message(), "") == 0);
  const int32_t good[5] = {-1, 0, 0, 1, 2}, bad[3] = {-1, 0, 3};
  CHECK(dreams_check_tree_host(good, 5) == DREAMS_OK);
  CHECK(dreams_check_tree_host(bad, 3) == DREAMS_ERR_INVALID_ARG && strlen(dreams_last_error_message()) > 0);
  CHECK(dreams_check_tree_host(nullptr, 3) == DREAMS_ERR_INVALID_ARG);

  // workspace sizes and split counts for explicit split counts (no device query)
  size_t n = 0;
  int32_t sp = 0;
  const int shapes[][7] = {{1, 32, 32, 128, 60, 3200, 8}, {4, 32, 32, 128, 60, 4160, 2}, {16, 28, 4, 128, 128, 8320, 3},
                           {3, 7, 1, 64, 100, 900, 32}, {2, 4, 4, 64, 1, 64, 5000}};
  for (const auto& s : shapes) {
    dreams_attn_desc_t d = desc(s[0], s[1], s[2], s[3], s[4], s[5], 0, s[6], DREAMS_BF16);
    const dreams_status_t st = dreams_tree_verify_attn_workspace_size(&d, &n);
    CHECK(st == (s[6] > 4096 ? DREAMS_ERR_INVALID_ARG : DREAMS_OK));
    if (st == DREAMS_OK) {
      CHECK(dreams_tree_verify_attn_splits(&d, &sp) == DREAMS_OK && sp >= 1 && sp <= 32);
      CHECK((sp == 1) == (n == 0));
    }
  }
  dreams_attn_desc_t bad_desc = desc(1, 30, 4, 128, 60, 3200, 0, 8, DREAMS_BF16);
  CHECK(dreams_tree_verify_attn_workspace_size(&bad_desc, &n) == DREAMS_ERR_INVALID_ARG);
  bad_desc = desc(1, 32, 32, 96, 60, 3200, 0, 8, DREAMS_BF16);
  CHECK(dreams_tree_verify_attn_workspace_size(&bad_desc, &n) == DREAMS_ERR_UNSUPPORTED);
  CHECK(dreams_tree_verify_attn_workspace_size(nullptr, &n) == DREAMS_ERR_INVALID_ARG);

  // calls that fail their checks before anything is enqueued; batch 0 is a no-op
  dreams_attn_desc_t d = desc(1, 32, 32, 128, 60, 3200, 0, 8, DREAMS_BF16);
  CHECK(dreams_tree_verify_attn(&d, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0,
                                nullptr) == DREAMS_ERR_INVALID_ARG);
  CHECK(dreams_tree_verify_attn_noalloc(&d, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                        nullptr) == DREAMS_ERR_INVALID_ARG);
  dreams_attn_desc_t d0 = desc(0, 32, 32, 128, 60, 3200, 0, 8, DREAMS_BF16);
  CHECK(dreams_tree_verify_attn(&d0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0,
                                nullptr) == DREAMS_OK);
  CHECK(dreams_tree_verify_attn_entropy(&d, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                        nullptr, nullptr, 0, nullptr) == DREAMS_ERR_INVALID_ARG);

  CHECK(dreams_tree_accept_workspace_size(4, 60, 32000, &n) == DREAMS_OK && n > DREAMS_WORKSPACE_COUNTER_BYTES);
  CHECK(dreams_tree_accept_workspace_size(1, 0, 32000, &n) == DREAMS_ERR_INVALID_ARG);
  CHECK(dreams_tree_accept(2, 60, 32000, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0,
                           nullptr) == DREAMS_ERR_INVALID_ARG);
  CHECK(dreams_tree_accept_sampled_workspace_size(4, 60, 32000, &n) == DREAMS_OK && n > DREAMS_WORKSPACE_COUNTER_BYTES);
  CHECK(dreams_tree_accept_sampled_workspace_size(4, 60, 1 << 24, &n) == DREAMS_ERR_UNSUPPORTED);
  CHECK(dreams_tree_accept_sampled(1, 8, 100, 0.0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                   nullptr, nullptr, 0, nullptr) == DREAMS_ERR_INVALID_ARG);
  CHECK(dreams_tree_accept_lm_head_workspace_size(1, 60, 4096, 32000, &n) == DREAMS_OK);
  CHECK(dreams_tree_accept_lm_head_workspace_size(1, 60, 4000, 32000, &n) == DREAMS_ERR_UNSUPPORTED);
  CHECK(dreams_kv_commit(0, 0, 1, 1, 128, 64, DREAMS_BF16, nullptr, nullptr, nullptr, nullptr, nullptr, 8, nullptr,
                         nullptr) == DREAMS_ERR_INVALID_ARG);
  CHECK(dreams_visual_importance_workspace_size(2, 4, 2880, &n) == DREAMS_OK);
  CHECK(dreams_visual_topk(1, 10000, 5, nullptr, nullptr, nullptr) == DREAMS_ERR_UNSUPPORTED);
  CHECK(dreams_visual_gather(1, 1, 100, 64, DREAMS_BF16, nullptr, nullptr, 0, nullptr, 1, nullptr, nullptr, nullptr) ==
        DREAMS_ERR_UNSUPPORTED);
  CHECK(dreams_attn_entropy_mean(0, nullptr, nullptr, nullptr) == DREAMS_ERR_INVALID_ARG);
  CHECK(dreams_attn_entropy_select(1, nullptr, nullptr, nullptr) == DREAMS_ERR_INVALID_ARG);
  CHECK(dreams_stream_read(nullptr, 64, nullptr, nullptr) == DREAMS_ERR_INVALID_ARG);
  CHECK(dreams_set_wait_limit(-1.0) == DREAMS_ERR_INVALID_ARG && dreams_set_wait_limit(0.2) == DREAMS_OK);
  CHECK(dreams_workspace_status(nullptr, 65536, nullptr) == DREAMS_ERR_INVALID_ARG);
  printf("host driver: ok\n");
  return 0;
}

/* Drives every entry point of the oracle (oracle/oracle.c) on small seeded inputs, for a build with the host
 * address and undefined-behaviour sanitizers: any out-of-bounds access, leak or undefined operation aborts the
 * run.  Also checks a few results that do not need a reference: probabilities in range, paths within the tree,
 * a commit that leaves the prefix untouched.  Exit status 0 on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_tree_attn(int, int, int, int, int, int, double, const float*, const float*, const float*, const int32_t*,
                     const int32_t*, const uint64_t*, double*, double*);
int oracle_tree_attn_rows(int, int, int, int, int, int, double, const float*, const float*, const float*,
                          const int32_t*, const int32_t*, const uint64_t*, int, const int32_t*, double*, double*);
int oracle_tree_attn_entropy(int, int, int, int, int, int, double, const float*, const float*, const int32_t*,
                             const int32_t*, const uint64_t*, double*);
int oracle_tree_accept_sampled(int, int, int, double, const float*, const float*, const int32_t*, const int32_t*,
                               const float*, int32_t*, int32_t*, int32_t*);
int oracle_visual_importance(int, int, int, int, int, int, double, const float*, const float*, const int32_t*,
                             const int32_t*, const uint64_t*, int, int, double*);
int oracle_visual_topk(int, int, int, const float*, int32_t*);
int oracle_visual_gather(int, int, int, int, int, const void*, const void*, int, const int32_t*, int, void*, void*);
int oracle_tree_accept(int, int, int, const float*, const int32_t*, const int32_t*, int32_t*, int32_t*, int32_t*,
                       int32_t*);
int oracle_kv_commit(int, int64_t, int, int, int, int, int, void*, void*, const int32_t*, const int32_t*,
                     const int32_t*, int, int32_t*);

static uint64_t state = 0x9E3779B97F4A7C15ull;
static double uni(void) { /* xorshift64*: inputs only */
  state ^= state >> 12; state ^= state << 25; state ^= state >> 27;
  return (double)((state * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
}
static float gauss(void) { return (float)(sqrt(-2.0 * log(uni() + 1e-300)) * cos(6.283185307179586 * uni())); }

#define CHECK(cond) do { if (!(cond)) { fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); return 1; } } while (0)

int main(void) {
  enum { B = 2, Hq = 4, Hkv = 2, T = 70, D = 16, V = 37, NL = 2 };
  const int L[B] = {41, 0};
  const int S = 128;
  int32_t parent[B * T], kv_len[B], tokens[B * T];
  for (int b = 0; b < B; ++b) {
    kv_len[b] = L[b];
    parent[b * T] = -1;
    for (int i = 1; i < T; ++i) parent[b * T + i] = (int)(uni() * i);
  }
  float* q = malloc(sizeof(float) * B * Hq * T * D);
  float* k = malloc(sizeof(float) * B * Hkv * S * D);
  float* v = malloc(sizeof(float) * B * Hkv * S * D);
  for (int i = 0; i < B * Hq * T * D; ++i) q[i] = gauss() * 0.3f;
  for (int i = 0; i < B * Hkv * S * D; ++i) { k[i] = gauss(); v[i] = gauss(); }
  double* out = malloc(sizeof(double) * B * Hq * T * D);
  double* lse = malloc(sizeof(double) * B * Hq * T);
  CHECK(oracle_tree_attn(B, Hq, Hkv, T, D, S, 0.25, q, k, v, kv_len, parent, NULL, out, lse) == 0);
  for (int i = 0; i < B * Hq * T; ++i) CHECK(isfinite(lse[i]));
  /* the same rows through the mask input: bit n of row i = ancestor-or-self */
  const int Wm = (T + 63) / 64;
  uint64_t* mask = calloc((size_t)B * T * Wm, sizeof(uint64_t));
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < T; ++i)
      for (int j = i; j >= 0; j = parent[b * T + j]) mask[((size_t)b * T + i) * Wm + j / 64] |= 1ull << (j % 64);
  double* out2 = malloc(sizeof(double) * B * Hq * T * D);
  CHECK(oracle_tree_attn(B, Hq, Hkv, T, D, S, 0.25, q, k, v, kv_len, NULL, mask, out2, NULL) == 0);
  for (int i = 0; i < B * Hq * T * D; ++i) CHECK(out[i] == out2[i]);
  int32_t rows[3 * 3] = {0, 0, 0, 1, 3, T - 1, 0, 2, 5};
  double orow[3 * D], lrow[3];
  CHECK(oracle_tree_attn_rows(B, Hq, Hkv, T, D, S, 0.25, q, k, v, kv_len, parent, NULL, 3, rows, orow, lrow) == 0);
  CHECK(orow[D] == out[((size_t)(1 * Hq + 3) * T + T - 1) * D]);
  double* ent = malloc(sizeof(double) * B * Hq * T);
  CHECK(oracle_tree_attn_entropy(B, Hq, Hkv, T, D, S, 0.25, q, k, kv_len, parent, NULL, ent) == 0);
  for (int i = 0; i < B * Hq * T; ++i) CHECK(ent[i] >= -1e-12);
  double* imp = malloc(sizeof(double) * B * 40);
  CHECK(oracle_visual_importance(B, Hq, Hkv, T, D, S, 0.25, q, k, kv_len, parent, NULL, 3, 40, imp) == 0);
  float impf[B * 40];
  for (int i = 0; i < B * 40; ++i) { CHECK(imp[i] >= 0.0 && imp[i] <= 1.0); impf[i] = (float)imp[i]; }
  int32_t keep[B * 9];
  CHECK(oracle_visual_topk(B, 40, 9, impf, keep) == 0);
  for (int i = 0; i < B * 9; ++i) CHECK(keep[i] >= 0 && keep[i] < 40);
  uint16_t* kg = malloc(2 * (size_t)B * Hkv * 9 * D);
  uint16_t* vg = malloc(2 * (size_t)B * Hkv * 9 * D);
  uint16_t* kb = malloc(2 * (size_t)B * Hkv * S * D);
  for (int i = 0; i < B * Hkv * S * D; ++i) kb[i] = (uint16_t)(uni() * 65535);
  CHECK(oracle_visual_gather(B, Hkv, D, S, 2, kb, kb, 3, keep, 9, kg, vg) == 0);

  float* logits = malloc(sizeof(float) * B * T * V);
  float* draft = malloc(sizeof(float) * B * T * V);
  for (int i = 0; i < B * T * V; ++i) { logits[i] = gauss() * 3.0f; draft[i] = logits[i] + gauss(); }
  for (int i = 0; i < B * T; ++i) tokens[i] = (int)(uni() * V);
  float uniforms[B * T];
  for (int i = 0; i < B * T; ++i) uniforms[i] = (float)uni();
  int32_t alen[B], path[B * T], next[B], am[B * T];
  CHECK(oracle_tree_accept(B, T, V, logits, tokens, parent, alen, path, next, am) == 0);
  for (int b = 0; b < B; ++b) CHECK(alen[b] >= 0 && alen[b] < T && path[b * T] == 0 && next[b] >= 0 && next[b] < V);
  CHECK(oracle_tree_accept_sampled(B, T, V, 0.7, logits, draft, tokens, parent, uniforms, alen, path, next) == 0);
  for (int b = 0; b < B; ++b) CHECK(alen[b] >= 0 && alen[b] < T && next[b] >= 0 && next[b] < V);

  /* commit into NL layers of bf16 caches; the prefix slots stay untouched */
  const int64_t stride = (int64_t)B * Hkv * S * D;
  uint16_t* kc = malloc(2 * (size_t)NL * stride);
  uint16_t* vc = malloc(2 * (size_t)NL * stride);
  for (int64_t i = 0; i < NL * stride; ++i) { kc[i] = (uint16_t)i; vc[i] = (uint16_t)(i * 7); }
  uint16_t* k0 = malloc(2 * (size_t)NL * stride);
  memcpy(k0, kc, 2 * (size_t)NL * stride);
  int32_t kv_out[B];
  CHECK(oracle_kv_commit(NL, stride, B, Hkv, D, S, 2, kc, vc, kv_len, path, alen, T, kv_out) == 0);
  for (int b = 0; b < B; ++b) {
    CHECK(kv_out[b] == kv_len[b] + alen[b] + 1);
    for (int l = 0; l < NL; ++l)
      for (int g = 0; g < Hkv; ++g)
        for (int s = 0; s < kv_len[b]; ++s)
          for (int d = 0; d < D; ++d) {
            const int64_t e = l * stride + (((int64_t)b * Hkv + g) * S + s) * D + d;
            CHECK(kc[e] == k0[e]);
          }
  }
  /* argument errors return non-zero without touching anything */
  CHECK(oracle_tree_accept(B, 0, V, logits, tokens, parent, alen, path, next, am) != 0);
  CHECK(oracle_tree_attn(B, 3, 2, T, D, S, 0.25, q, k, v, kv_len, parent, NULL, out, lse) != 0);

  free(q); free(k); free(v); free(out); free(out2); free(lse); free(mask); free(ent); free(imp);
  free(kg); free(vg); free(kb); free(logits); free(draft); free(kc); free(vc); free(k0);
  printf("oracle driver: ok\n");
  return 0;
}

/*
 * oracle.c -- plain, slow CPU oracle for the DREAM-S tree-verification step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or load this file: only the test
 * suite, the package smoke check and the benchmark's CPU-baseline leg use it.  It shares no code, header or
 * constant with the HIP library; both are fed from the same seeded input generator.
 *
 * Everything here is the plain definition of what the verification step computes, written out with
 * scalar loops and fp64 accumulation (inputs are fp32 values; bf16 inputs arrive already widened, which is
 * exact).  No blocking, no online softmax, no split of the key axis, no fast-math.
 *
 *  oracle_tree_attn / oracle_tree_attn_row
 *      Masked softmax attention  A = softmax(Q K^T * scale), out = A V  (the attention matrix as the paper
 *      defines it in Section 3.2, "Adaptive Intermediate Feature Distillation"; scale = 1/sqrt(head_dim)
 *      is passed explicitly).  Each tree node attends to every committed prefix slot -- image and text
 *      tokens alike, since the paper's Section 2 ("Vision-Language Models") notes that all visual tokens sit
 *      in the KV cache and are attended at every decoding step -- plus the tree slots of its own ancestors
 *      and itself, so that each root-to-node path is verified exactly as the sequential draft it stands for
 *      (Section 2, "Speculative decoding": drafts are verified in one parallel pass).
 *      Softmax is taken in two passes (max, then exp/sum), the textbook way.
 *
 *  oracle_tree_accept
 *      Greedy verification (Section 2, "Speculative decoding"): a draft token is kept while it equals the
 *      target's own choice at its position; at the first mismatch the target's token replaces it.  On a tree
 *      this is applied along every root-to-node path; the longest consistent path wins (deepest node,
 *      smallest index on ties) and the target's token at its end is emitted as the bonus token, so one
 *      step emits depth+1 tokens (the paper's Table 6 prints acceptance lengths above the draft window,
 *      which counts that bonus token).
 *
 *  oracle_kv_commit
 *      Keeps the root and the accepted nodes' K/V as the next contiguous cache slots, in path order.
 *
 *  oracle_tree_accept_sampled
 *      Sampled verification at temperature tau (the paper reports speedups at temperature 1, Table 2): the
 *      acceptance-rejection mechanism of speculative sampling (Section 1; Section 2, "Speculative decoding")
 *      run down the tree.  At a node, the target's distribution p and the draft's q (softmax of the logits
 *      over tau) are compared for each child in index order: the child's token x is accepted with
 *      probability min(1, r(x)/q(x)), r starting as p; after a rejection r becomes max(r - q, 0),
 *      renormalised.  The walk descends into the first accepted child; where none is accepted (or at a leaf)
 *      the emitted token is drawn from r.  The uniforms are inputs: u[b][c] decides child c, u[b][0] draws
 *      the final token (inverse CDF).
 *
 *  oracle_visual_importance / oracle_visual_topk / oracle_visual_gather
 *      Target-aware visual-token selection (Section 3.1, "Visual Token Compression", Eq. 2): the importance of
 *      visual token j is its attention weight averaged over every head and every query row of the call,
 *      I_j = (1/(H*Q)) sum_h sum_i A[h,i,j]; the r most important tokens are kept (ties to the smaller
 *      index), listed in increasing token order, and their K/V rows gathered into a compact cache.
 *
 *  oracle_prefill_attn_stats / oracle_prefill_visual_importance
 *      The same two statistics over a prompt's own causal attention (row i sees slots 0..i), which is where the
 *      paper reads them: Eq. 2 with the final layer's weights of the prefilling pass, AE(l) over the layer's
 *      n x n attention of the prompt (Sections 3.1 and 3.2).
 *
 *  oracle_tree_attn_entropy
 *      Attention entropy of every verification row: -sum_j A_ij log A_ij over the row's attention
 *      probabilities, the per-row quantity whose mean over rows and heads is the average attention entropy
 *      AE of a layer (Section 3.2, "Adaptive Intermediate Feature Distillation").  Same masking and scores as
 *      oracle_tree_attn; natural logarithm; a row with nothing visible has entropy 0.
 *
 * Return value of every entry point: 0 on success, negative on invalid input (nothing written then).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_BAD_ARG (-1)
#define ORACLE_BAD_TREE (-2)
#define ORACLE_NONFINITE (-3)

/* parent[0] = -1 and 0 <= parent[i] < i for i >= 1. */
static int tree_ok(const int32_t* parent, int T) {
  if (T < 1 || parent[0] != -1) return 0;
  for (int i = 1; i < T; ++i)
    if (parent[i] < 0 || parent[i] >= i) return 0;
  return 1;
}

/* visible[j] = 1 iff tree node j may be attended by tree node i. */
static void visible_nodes(const int32_t* parent, const uint64_t* mask_row, int T, int i, unsigned char* visible) {
  memset(visible, 0, (size_t)T);
  if (mask_row) {
    for (int j = 0; j < T; ++j) visible[j] = (unsigned char)((mask_row[j / 64] >> (j % 64)) & 1u);
  } else {
    for (int j = i; j >= 0; j = parent[j]) visible[j] = 1;   /* i, its parent, ..., the root */
  }
}

/* One output row: sequence b, query head h, tree node i. */
static void attn_row(int Hq, int Hkv, int T, int D, int S_cap, double scale, const float* q, const float* k,
                     const float* v, const int32_t* kv_len, const int32_t* parent, const uint64_t* tree_mask,
                     int b, int h, int i, double* out_row, double* lse_out, unsigned char* visible,
                     double* score) {
  const int G = Hq / Hkv;
  const int g = h / G;                      /* KV head shared by query head h */
  const int L = kv_len[b];
  const int W = (T + 63) / 64;
  const float* qi = q + (((size_t)b * Hq + h) * T + i) * D;
  const float* kb = k + ((size_t)b * Hkv + g) * (size_t)S_cap * D;
  const float* vb = v + ((size_t)b * Hkv + g) * (size_t)S_cap * D;
  visible_nodes(parent ? parent + (size_t)b * T : NULL,
                tree_mask ? tree_mask + ((size_t)b * T + i) * W : NULL, T, i, visible);

  /* slots 0..L-1 are the committed prefix; slot L+j holds tree node j */
  const int n = L + T;
  double m = -INFINITY;
  for (int s = 0; s < n; ++s) {
    if (s >= L && !visible[s - L]) continue;
    double dot = 0.0;
    for (int d = 0; d < D; ++d) dot += (double)qi[d] * (double)kb[(size_t)s * D + d];
    score[s] = scale * dot;
    if (score[s] > m) m = score[s];
  }
  for (int d = 0; d < D; ++d) out_row[d] = 0.0;
  if (m == -INFINITY) { /* nothing visible: defined as a zero row with lse = -inf */
    *lse_out = -INFINITY;
    return;
  }
  double l = 0.0;
  for (int s = 0; s < n; ++s) {
    if (s >= L && !visible[s - L]) continue;
    double p = exp(score[s] - m);
    l += p;
    for (int d = 0; d < D; ++d) out_row[d] += p * (double)vb[(size_t)s * D + d];
  }
  for (int d = 0; d < D; ++d) out_row[d] /= l;
  *lse_out = m + log(l);
}

static int attn_args_ok(int B, int Hq, int Hkv, int T, int D, int S_cap, const int32_t* kv_len,
                        const int32_t* parent, const uint64_t* tree_mask) {
  if (B < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || T < 1 || D < 1 || S_cap < T) return ORACLE_BAD_ARG;
  if (!parent && !tree_mask) return ORACLE_BAD_ARG;
  for (int b = 0; b < B; ++b) {
    if (kv_len[b] < 0 || kv_len[b] + T > S_cap) return ORACLE_BAD_ARG;
    if (!tree_mask && !tree_ok(parent + (size_t)b * T, T)) return ORACLE_BAD_TREE;
  }
  return 0;
}

/* Layouts: q, out [B,Hq,T,D]; k, v [B,Hkv,S_cap,D]; lse [B,Hq,T]; tree_mask [B,T,ceil(T/64)] or NULL. */
int oracle_tree_attn(int B, int Hq, int Hkv, int T, int D, int S_cap, double scale, const float* q,
                     const float* k, const float* v, const int32_t* kv_len, const int32_t* parent,
                     const uint64_t* tree_mask, double* out, double* lse) {
  int rc = attn_args_ok(B, Hq, Hkv, T, D, S_cap, kv_len, parent, tree_mask);
  if (rc) return rc;
#pragma omp parallel
  {
    unsigned char* visible = (unsigned char*)malloc((size_t)T);
    double* score = (double*)malloc(sizeof(double) * (size_t)(S_cap + 1));
#pragma omp for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < Hq; ++h)
        for (int i = 0; i < T; ++i) {
          size_t r = ((size_t)b * Hq + h) * T + i;
          double lse_r;
          attn_row(Hq, Hkv, T, D, S_cap, scale, q, k, v, kv_len, parent, tree_mask, b, h, i,
                   out + r * D, &lse_r, visible, score);
          if (lse) lse[r] = lse_r;
        }
    free(visible);
    free(score);
  }
  return 0;
}

/* Selected rows only: rows[3*n + {0,1,2}] = (b, h, i); out_rows [n, D], lse_rows [n]. */
int oracle_tree_attn_rows(int B, int Hq, int Hkv, int T, int D, int S_cap, double scale, const float* q,
                          const float* k, const float* v, const int32_t* kv_len, const int32_t* parent,
                          const uint64_t* tree_mask, int n_rows, const int32_t* rows, double* out_rows,
                          double* lse_rows) {
  int rc = attn_args_ok(B, Hq, Hkv, T, D, S_cap, kv_len, parent, tree_mask);
  if (rc) return rc;
  for (int r = 0; r < n_rows; ++r) {
    int b = rows[3 * r], h = rows[3 * r + 1], i = rows[3 * r + 2];
    if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= T) return ORACLE_BAD_ARG;
  }
#pragma omp parallel
  {
    unsigned char* visible = (unsigned char*)malloc((size_t)T);
    double* score = (double*)malloc(sizeof(double) * (size_t)(S_cap + 1));
#pragma omp for schedule(dynamic)
    for (int r = 0; r < n_rows; ++r) {
      double lse_r;
      attn_row(Hq, Hkv, T, D, S_cap, scale, q, k, v, kv_len, parent, tree_mask, rows[3 * r], rows[3 * r + 1],
               rows[3 * r + 2], out_rows + (size_t)r * D, &lse_r, visible, score);
      if (lse_rows) lse_rows[r] = lse_r;
    }
    free(visible);
    free(score);
  }
  return 0;
}

/* Entropy of one row (b, h, i): softmax of the visible scores (two passes), then -sum p log p. */
static double entropy_row(int Hq, int Hkv, int T, int D, int S_cap, double scale, const float* q, const float* k,
                          const int32_t* kv_len, const int32_t* parent, const uint64_t* tree_mask, int b, int h,
                          int i, unsigned char* visible, double* score) {
  const int G = Hq / Hkv;
  const int g = h / G;
  const int L = kv_len[b];
  const int W = (T + 63) / 64;
  const float* qi = q + (((size_t)b * Hq + h) * T + i) * D;
  const float* kb = k + ((size_t)b * Hkv + g) * (size_t)S_cap * D;
  visible_nodes(parent ? parent + (size_t)b * T : NULL,
                tree_mask ? tree_mask + ((size_t)b * T + i) * W : NULL, T, i, visible);
  const int n = L + T;
  double m = -INFINITY;
  for (int s = 0; s < n; ++s) {
    if (s >= L && !visible[s - L]) continue;
    double dot = 0.0;
    for (int d = 0; d < D; ++d) dot += (double)qi[d] * (double)kb[(size_t)s * D + d];
    score[s] = scale * dot;
    if (score[s] > m) m = score[s];
  }
  if (m == -INFINITY) return 0.0;
  double l = 0.0;
  for (int s = 0; s < n; ++s) {
    if (s >= L && !visible[s - L]) continue;
    l += exp(score[s] - m);
  }
  double H = 0.0;
  for (int s = 0; s < n; ++s) {
    if (s >= L && !visible[s - L]) continue;
    const double p = exp(score[s] - m) / l;   /* the row's attention probability of slot s */
    if (p > 0.0) H -= p * log(p);
  }
  return H;
}

/* Layouts as for oracle_tree_attn (v is not needed); entropy [B,Hq,T]. */
int oracle_tree_attn_entropy(int B, int Hq, int Hkv, int T, int D, int S_cap, double scale, const float* q,
                             const float* k, const int32_t* kv_len, const int32_t* parent,
                             const uint64_t* tree_mask, double* entropy) {
  int rc = attn_args_ok(B, Hq, Hkv, T, D, S_cap, kv_len, parent, tree_mask);
  if (rc) return rc;
#pragma omp parallel
  {
    unsigned char* visible = (unsigned char*)malloc((size_t)T);
    double* score = (double*)malloc(sizeof(double) * (size_t)(S_cap + 1));
#pragma omp for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < Hq; ++h)
        for (int i = 0; i < T; ++i)
          entropy[((size_t)b * Hq + h) * T + i] =
              entropy_row(Hq, Hkv, T, D, S_cap, scale, q, k, kv_len, parent, tree_mask, b, h, i, visible, score);
    free(visible);
    free(score);
  }
  return 0;
}

/* softmax(logits / tau) in fp64, two passes */
static void softmax_tau(const float* logits, int V, double tau, double* out) {
  double m = logits[0];
  for (int x = 1; x < V; ++x)
    if (logits[x] > m) m = logits[x];
  double s = 0.0;
  for (int x = 0; x < V; ++x) {
    out[x] = exp(((double)logits[x] - m) / tau);
    s += out[x];
  }
  for (int x = 0; x < V; ++x) out[x] /= s;
}

/*
 * Sampled tree acceptance.  target_logits, draft_logits [B,T,V]: row i holds the logits of the token that
 * follows node i, under the target and under the draft (the draft sampled node i's children from it);
 * tokens [B,T] (node 0 is the root, already emitted); parent [B,T]; uniforms [B,T] in [0,1).
 * Outputs as oracle_tree_accept: accept_len, accept_path (root .. last accepted node, then -1), next_token.
 */
int oracle_tree_accept_sampled(int B, int T, int V, double tau, const float* target_logits,
                               const float* draft_logits, const int32_t* tokens, const int32_t* parent,
                               const float* uniforms, int32_t* accept_len, int32_t* accept_path,
                               int32_t* next_token) {
  if (B < 0 || T < 1 || V < 1 || !(tau > 0.0) || !isfinite(tau)) return ORACLE_BAD_ARG;
  for (int b = 0; b < B; ++b) {
    if (!tree_ok(parent + (size_t)b * T, T)) return ORACLE_BAD_TREE;
    for (int i = 1; i < T; ++i) {
      const int x = tokens[(size_t)b * T + i];
      if (x < 0 || x >= V) return ORACLE_BAD_ARG;
    }
    for (int i = 0; i < T; ++i) {
      const float u = uniforms[(size_t)b * T + i];
      if (!(u >= 0.0f && u < 1.0f)) return ORACLE_BAD_ARG;
    }
  }
  for (size_t e = 0; e < (size_t)B * T * V; ++e)
    if (!isfinite(target_logits[e]) || !isfinite(draft_logits[e])) return ORACLE_NONFINITE;

  double* p = (double*)malloc(sizeof(double) * (size_t)V);
  double* q = (double*)malloc(sizeof(double) * (size_t)V);
  double* r = (double*)malloc(sizeof(double) * (size_t)V);
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    const int32_t* tok = tokens + (size_t)b * T;
    const float* u = uniforms + (size_t)b * T;
    int32_t* path = accept_path + (size_t)b * T;
    for (int k = 0; k < T; ++k) path[k] = -1;
    int node = 0, depth = 0;
    path[0] = 0;
    for (;;) {
      softmax_tau(target_logits + ((size_t)b * T + node) * V, V, tau, p);
      softmax_tau(draft_logits + ((size_t)b * T + node) * V, V, tau, q);
      for (int x = 0; x < V; ++x) r[x] = p[x];
      int accepted = -1;
      for (int c = node + 1; c < T && accepted < 0; ++c) {
        if (par[c] != node) continue;
        const int x = tok[c];
        if ((double)u[c] * q[x] < r[x]) {   /* accepted with probability min(1, r(x)/q(x)) */
          accepted = c;
          break;
        }
        double z = 0.0;   /* rejected: the residual max(r - q, 0), renormalised (kept if it vanishes) */
        for (int y = 0; y < V; ++y) z += r[y] > q[y] ? r[y] - q[y] : 0.0;
        if (z > 0.0)
          for (int y = 0; y < V; ++y) r[y] = (r[y] > q[y] ? r[y] - q[y] : 0.0) / z;
      }
      if (accepted < 0) break;
      node = accepted;
      path[++depth] = node;
    }
    /* the emitted token: inverse CDF of r at u[0] */
    double total = 0.0;
    for (int x = 0; x < V; ++x) total += r[x];
    const double thr = (double)u[0] * total;
    double cum = 0.0;
    int pick = -1, last_pos = 0;
    for (int x = 0; x < V; ++x) {
      if (r[x] > 0.0) last_pos = x;
      cum += r[x];
      if (pick < 0 && cum > thr) pick = x;
    }
    accept_len[b] = depth;
    next_token[b] = pick >= 0 ? pick : last_pos;
  }
  free(p);
  free(q);
  free(r);
  return 0;
}

/*
 * Visual-token importance.  The visual tokens are prefix slots vis_begin .. vis_begin+vis_count-1.  For every
 * sequence b, query head h and row i, A[h,i,.] is that row's attention (the same visible slots and scores as
 * oracle_tree_attn, softmax in two passes); importance[b][j] = sum over h, i of A[h,i,vis_begin+j], divided
 * by Hq*T.  A visual slot outside sequence b's committed prefix (>= kv_len[b]) has importance 0.
 */
int oracle_visual_importance(int B, int Hq, int Hkv, int T, int D, int S_cap, double scale, const float* q,
                             const float* k, const int32_t* kv_len, const int32_t* parent,
                             const uint64_t* tree_mask, int vis_begin, int vis_count, double* importance) {
  int rc = attn_args_ok(B, Hq, Hkv, T, D, S_cap, kv_len, parent, tree_mask);
  if (rc) return rc;
  if (vis_begin < 0 || vis_count < 1 || vis_begin + vis_count > S_cap) return ORACLE_BAD_ARG;
  const int G = Hq / Hkv;
  const int W = (T + 63) / 64;
#pragma omp parallel for schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    unsigned char* visible = (unsigned char*)malloc((size_t)T);
    double* score = (double*)malloc(sizeof(double) * (size_t)(S_cap + 1));
    double* imp = importance + (size_t)b * vis_count;
    for (int j = 0; j < vis_count; ++j) imp[j] = 0.0;
    const int L = kv_len[b];
    const int n = L + T;
    for (int h = 0; h < Hq; ++h) {
      const int g = h / G;
      const float* kb = k + ((size_t)b * Hkv + g) * (size_t)S_cap * D;
      for (int i = 0; i < T; ++i) {
        const float* qi = q + (((size_t)b * Hq + h) * T + i) * D;
        visible_nodes(parent ? parent + (size_t)b * T : NULL,
                      tree_mask ? tree_mask + ((size_t)b * T + i) * W : NULL, T, i, visible);
        double m = -INFINITY;
        for (int s = 0; s < n; ++s) {
          if (s >= L && !visible[s - L]) continue;
          double dot = 0.0;
          for (int d = 0; d < D; ++d) dot += (double)qi[d] * (double)kb[(size_t)s * D + d];
          score[s] = scale * dot;
          if (score[s] > m) m = score[s];
        }
        if (m == -INFINITY) continue;   /* a row that sees nothing attends to no visual token */
        double l = 0.0;
        for (int s = 0; s < n; ++s) {
          if (s >= L && !visible[s - L]) continue;
          l += exp(score[s] - m);
        }
        for (int j = 0; j < vis_count; ++j) {
          const int s = vis_begin + j;
          if (s < L) imp[j] += exp(score[s] - m) / l;   /* A[h,i,s]; prefix slots are visible to every row */
        }
      }
    }
    for (int j = 0; j < vis_count; ++j) imp[j] /= (double)Hq * T;
    free(visible);
    free(score);
  }
  return 0;
}

/* The r largest of each sequence's vis_count importances (ties: the smaller index first), as token indices in
 * increasing order: keep [B, r].  A plain selection by repeated maximum. */
int oracle_visual_topk(int B, int vis_count, int r, const float* importance, int32_t* keep) {
  if (B < 0 || vis_count < 1 || r < 1 || r > vis_count) return ORACLE_BAD_ARG;
  unsigned char* taken = (unsigned char*)malloc((size_t)vis_count);
  for (int b = 0; b < B; ++b) {
    const float* v = importance + (size_t)b * vis_count;
    memset(taken, 0, (size_t)vis_count);
    for (int t = 0; t < r; ++t) {
      int best = -1;
      for (int j = 0; j < vis_count; ++j)
        if (!taken[j] && (best < 0 || v[j] > v[best])) best = j;   /* first index among equal maxima */
      taken[best] = 1;
    }
    int m = 0;
    for (int j = 0; j < vis_count; ++j)
      if (taken[j]) keep[(size_t)b * r + m++] = j;
  }
  free(taken);
  return 0;
}

/* k_out/v_out [B, Hkv, r, D] (elem_bytes per element) receive the K/V rows of slots vis_begin + keep[b][m]. */
int oracle_visual_gather(int B, int Hkv, int D, int S_cap, int elem_bytes, const void* k_cache, const void* v_cache,
                         int vis_begin, const int32_t* keep, int r, void* k_out, void* v_out) {
  if (B < 0 || Hkv < 1 || D < 1 || r < 1 || elem_bytes < 1) return ORACLE_BAD_ARG;
  const size_t row = (size_t)D * elem_bytes;
  for (int b = 0; b < B; ++b)
    for (int m = 0; m < r; ++m) {
      const int s = vis_begin + keep[(size_t)b * r + m];
      if (s < 0 || s >= S_cap) return ORACLE_BAD_ARG;
    }
  for (int b = 0; b < B; ++b)
    for (int g = 0; g < Hkv; ++g)
      for (int m = 0; m < r; ++m) {
        const size_t src = (((size_t)b * Hkv + g) * S_cap + vis_begin + keep[(size_t)b * r + m]) * row;
        const size_t dst = (((size_t)b * Hkv + g) * r + m) * row;
        memcpy((char*)k_out + dst, (const char*)k_cache + src, row);
        memcpy((char*)v_out + dst, (const char*)v_cache + src, row);
      }
  return 0;
}

/*
 * Greedy tree acceptance.  logits [B,T,V] (target logits at every node), tokens [B,T] (draft token of every
 * node; tokens[b][0] is the root, already emitted), parent [B,T].
 * Outputs: accept_len [B] = number of accepted draft tokens a (the depth of the last accepted node);
 * accept_path [B,T] = node ids root..last then -1; next_token [B] = target token after the last accepted
 * node; target_argmax [B,T] (may be NULL) = the target's token at every node.
 */
int oracle_tree_accept(int B, int T, int V, const float* logits, const int32_t* tokens, const int32_t* parent,
                       int32_t* accept_len, int32_t* accept_path, int32_t* next_token, int32_t* target_argmax) {
  if (B < 0 || T < 1 || V < 1) return ORACLE_BAD_ARG;
  for (int b = 0; b < B; ++b)
    if (!tree_ok(parent + (size_t)b * T, T)) return ORACLE_BAD_TREE;
  for (size_t e = 0; e < (size_t)B * T * V; ++e)
    if (!isfinite(logits[e])) return ORACLE_NONFINITE;

  int* am = (int*)malloc(sizeof(int) * (size_t)T);
  int* ok = (int*)malloc(sizeof(int) * (size_t)T);
  int* depth = (int*)malloc(sizeof(int) * (size_t)T);
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    const int32_t* tok = tokens + (size_t)b * T;
    /* the target's token at node i: the smallest index attaining the row maximum */
    for (int i = 0; i < T; ++i) {
      const float* row = logits + ((size_t)b * T + i) * V;
      int best = 0;
      for (int x = 1; x < V; ++x)
        if (row[x] > row[best]) best = x;
      am[i] = best;
    }
    /* a node is consistent iff its parent is and its token is the target's token at the parent */
    ok[0] = 1;
    depth[0] = 0;
    for (int i = 1; i < T; ++i) {
      ok[i] = ok[par[i]] && tok[i] == am[par[i]];
      depth[i] = depth[par[i]] + 1;
    }
    int last = 0;
    for (int i = 1; i < T; ++i)
      if (ok[i] && depth[i] > depth[last]) last = i;
    const int a = depth[last];
    int32_t* path = accept_path + (size_t)b * T;
    for (int k = 0; k < T; ++k) path[k] = -1;
    for (int j = last; j >= 0; j = par[j]) path[depth[j]] = j;
    accept_len[b] = a;
    next_token[b] = am[last];
    if (target_argmax)
      for (int i = 0; i < T; ++i) target_argmax[(size_t)b * T + i] = am[i];
  }
  free(am);
  free(ok);
  free(depth);
  return 0;
}

/*
 * KV commit.  Cache layers are layer_stride_elems elements apart; inside a layer the layout is
 * [B, Hkv, S_cap, D] with elements of elem_bytes bytes.  For k = 0..a (increasing), slot L+path[k] is copied
 * to slot L+k for every layer and KV head; kv_len_out[b] = L + a + 1.  Copies are bytewise.
 */
int oracle_kv_commit(int NL, int64_t layer_stride_elems, int B, int Hkv, int D, int S_cap, int elem_bytes,
                     void* k_cache, void* v_cache, const int32_t* kv_len_in, const int32_t* accept_path,
                     const int32_t* accept_len, int path_stride, int32_t* kv_len_out) {
  if (NL < 1 || B < 0 || Hkv < 1 || D < 1 || S_cap < 1 || (elem_bytes != 2 && elem_bytes != 4)) return ORACLE_BAD_ARG;
  for (int b = 0; b < B; ++b) {
    const int a = accept_len[b];
    const int32_t* path = accept_path + (size_t)b * path_stride;
    if (a < 0 || a >= path_stride || path[0] != 0) return ORACLE_BAD_ARG;
    for (int k = 1; k <= a; ++k)
      if (path[k] < k || path[k] <= path[k - 1]) return ORACLE_BAD_ARG;
    if (kv_len_in[b] + path[a] >= S_cap) return ORACLE_BAD_ARG;
  }
  const size_t row = (size_t)D * elem_bytes;
  for (int layer = 0; layer < NL; ++layer)
    for (int b = 0; b < B; ++b)
      for (int g = 0; g < Hkv; ++g) {
        const size_t base = ((size_t)layer * layer_stride_elems + ((size_t)b * Hkv + g) * (size_t)S_cap * D) * elem_bytes;
        const int L = kv_len_in[b];
        const int32_t* path = accept_path + (size_t)b * path_stride;
        for (int k = 0; k <= accept_len[b]; ++k) {
          char* kc = (char*)k_cache + base;
          char* vc = (char*)v_cache + base;
          memmove(kc + (size_t)(L + k) * row, kc + (size_t)(L + path[k]) * row, row);
          memmove(vc + (size_t)(L + k) * row, vc + (size_t)(L + path[k]) * row, row);
        }
      }
  for (int b = 0; b < B; ++b) kv_len_out[b] = kv_len_in[b] + accept_len[b] + 1;
  return 0;
}

/*
 * Prefill attention statistics.  Eq. 2 (Section 3.1) scores the visual tokens with the final layer's attention
 * weights of the prefilling pass, and AE(l) (Section 3.2) averages the entropy of a layer's attention rows over
 * the n prompt tokens: both are read off the attention of the prompt's own positions among themselves.  Prompt
 * b holds n_b = prompt_len[b] tokens: keys at cache slots 0..n_b-1, queries at rows 0..n_b-1 of q.  Row i of
 * query head h attends slots 0..i (the decoder's causal mask):
 *     A[h,i,j] = exp(scale * q_i.k_j) / sum_{j' <= i} exp(scale * q_i.k_j'),   j <= i.
 * Rows i >= n_b are not queries of the prompt.  Layouts: q [B,Hq,N,D]; k [B,Hkv,S_cap,D]; query head h reads
 * KV head h / (Hq/Hkv).
 */
static int prefill_args_ok(int B, int Hq, int Hkv, int N, int D, int S_cap, const int32_t* prompt_len) {
  if (B < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || N < 1 || D < 1 || S_cap < N) return ORACLE_BAD_ARG;
  for (int b = 0; b < B; ++b)
    if (prompt_len[b] < 0 || prompt_len[b] > N) return ORACLE_BAD_ARG;
  return 0;
}

/* Scores of row (b, h, i) over slots 0..i into score[]; returns their maximum. */
static double prefill_scores(int Hq, int Hkv, int N, int D, int S_cap, double scale, const float* q, const float* k,
                             int b, int h, int i, double* score) {
  const int g = h / (Hq / Hkv);
  const float* qi = q + (((size_t)b * Hq + h) * N + i) * D;
  const float* kb = k + ((size_t)b * Hkv + g) * (size_t)S_cap * D;
  double m = -INFINITY;
  for (int s = 0; s <= i; ++s) {
    double dot = 0.0;
    for (int d = 0; d < D; ++d) dot += (double)qi[d] * (double)kb[(size_t)s * D + d];
    score[s] = scale * dot;
    if (score[s] > m) m = score[s];
  }
  return m;
}

/* lse [B,Hq,N] = log sum_{j<=i} exp(scale q_i.k_j) (natural log) and entropy [B,Hq,N] = -sum_j A_ij log A_ij
 * of every prompt row; rows i >= n_b get lse = -inf and entropy 0.  Either output may be NULL. */
int oracle_prefill_attn_stats(int B, int Hq, int Hkv, int N, int D, int S_cap, double scale, const float* q,
                              const float* k, const int32_t* prompt_len, double* lse, double* entropy) {
  int rc = prefill_args_ok(B, Hq, Hkv, N, D, S_cap, prompt_len);
  if (rc) return rc;
#pragma omp parallel
  {
    double* score = (double*)malloc(sizeof(double) * (size_t)N);
#pragma omp for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < Hq; ++h)
        for (int i = 0; i < N; ++i) {
          const size_t row = ((size_t)b * Hq + h) * N + i;
          if (i >= prompt_len[b]) {
            if (lse) lse[row] = -INFINITY;
            if (entropy) entropy[row] = 0.0;
            continue;
          }
          const double m = prefill_scores(Hq, Hkv, N, D, S_cap, scale, q, k, b, h, i, score);
          double l = 0.0;
          for (int s = 0; s <= i; ++s) l += exp(score[s] - m);
          if (lse) lse[row] = m + log(l);
          if (entropy) {
            double H = 0.0;
            for (int s = 0; s <= i; ++s) {
              const double p = exp(score[s] - m) / l;   /* A[h,i,s] */
              if (p > 0.0) H -= p * log(p);
            }
            entropy[row] = H;
          }
        }
    free(score);
  }
  return 0;
}

/* Eq. 2 over the prompt: importance [B, vis_count], importance[b][j] = (1/(Hq*n_b)) sum_h sum_{i<n_b}
 * A[h,i,vis_begin+j] (a slot past row i gets nothing from it, so a slot at or past n_b has importance 0); a
 * sequence with n_b = 0 has all zeros. */
int oracle_prefill_visual_importance(int B, int Hq, int Hkv, int N, int D, int S_cap, double scale, const float* q,
                                     const float* k, const int32_t* prompt_len, int vis_begin, int vis_count,
                                     double* importance) {
  int rc = prefill_args_ok(B, Hq, Hkv, N, D, S_cap, prompt_len);
  if (rc) return rc;
  if (vis_begin < 0 || vis_count < 1 || vis_begin + vis_count > S_cap) return ORACLE_BAD_ARG;
#pragma omp parallel for schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    double* score = (double*)malloc(sizeof(double) * (size_t)N);
    double* imp = importance + (size_t)b * vis_count;
    for (int j = 0; j < vis_count; ++j) imp[j] = 0.0;
    const int n = prompt_len[b];
    for (int h = 0; h < Hq; ++h)
      for (int i = 0; i < n; ++i) {
        const double m = prefill_scores(Hq, Hkv, N, D, S_cap, scale, q, k, b, h, i, score);
        double l = 0.0;
        for (int s = 0; s <= i; ++s) l += exp(score[s] - m);
        for (int j = 0; j < vis_count; ++j) {
          const int slot = vis_begin + j;
          if (slot <= i) imp[j] += exp(score[slot] - m) / l;   /* A[h,i,slot]; later slots are masked */
        }
      }
    if (n > 0)
      for (int j = 0; j < vis_count; ++j) imp[j] /= (double)Hq * n;
    free(score);
  }
  return 0;
}

/* Number of threads the parallel loops above use (reported beside CPU timings). */
int oracle_num_threads(void) { return omp_get_max_threads(); }

/* Threads of the parallel loops above (n >= 1); used to time the oracle on one core beside all of them. */
void oracle_set_num_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }

/*
 * dreams.h -- C ABI of libdreams.so, the MI355X (gfx950) tree-verification step of DREAM-S speculative
 * decoding for vision-language models.
 *
 * The step has three verbs (acceptance in three forms), run back to back on one HIP stream:
 *   dreams_tree_verify_attn  tree-masked attention of the draft-token tree against the KV cache
 *   dreams_tree_accept       greedy acceptance of the longest target-consistent root-to-node path
 *   dreams_tree_accept_sampled  acceptance at temperature tau > 0 (accept-or-resample down the tree)
 *   dreams_tree_accept_lm_head  greedy acceptance from final hidden states (LM head fused with the argmax)
 *   dreams_kv_commit         compaction of the accepted path's K/V into the cache
 *
 * Conventions shared by every entry point
 *   - Pointers named as "device" point to device memory the caller owns (allocated on the current HIP
 *     device).  The library never allocates or frees inside a call; scratch memory comes in through a
 *     caller-owned workspace sized by the matching *_workspace_size query.
 *   - Calls are asynchronous and stream-ordered: they enqueue kernels on `stream` and return.  Outputs are
 *     valid once the stream has reached that point.  Calls that share a workspace must be ordered (same
 *     stream, or synchronised streams).
 *   - Host-visible arguments (sizes, flags, null pointers) are checked before anything is enqueued; on a
 *     failed check the call returns a negative status, sets the thread's last error message and enqueues
 *     nothing.  Values that live in device memory (kv_len, parent, accept_path, ...) cannot be checked on the
 *     host; the kernels clamp or skip out-of-range entries so that no access leaves the caller's buffers,
 *     and the results for such entries are unspecified.
 *   - A HIP launch error returns DREAMS_ERR_HIP.
 *   - Element types: DREAMS_BF16 tensors hold bfloat16 bit patterns (round-to-nearest-even); DREAMS_F32
 *     tensors hold IEEE binary32.
 */
#ifndef DREAMS_H
#define DREAMS_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DREAMS_OK = 0,
  DREAMS_ERR_INVALID_ARG = -1,  /* a host-visible argument is out of range or a required pointer is NULL */
  DREAMS_ERR_UNSUPPORTED = -2,  /* valid in principle but not built (e.g. a head_dim other than 64/128)   */
  DREAMS_ERR_WORKSPACE = -3,    /* workspace NULL or smaller than the matching *_workspace_size           */
  DREAMS_ERR_HIP = -4,          /* the HIP runtime reported an error (device query or kernel launch)     */
  DREAMS_ERR_DEVICE = -5        /* a kernel of an earlier call flagged a failure (dreams_workspace_status) */
} dreams_status_t;

typedef enum { DREAMS_F32 = 0, DREAMS_BF16 = 1 } dreams_dtype_t;

/*
 * Workspaces.  Every workspace (of either verb that takes one) begins with DREAMS_WORKSPACE_COUNTER_BYTES
 * bytes of arrival counters.  Zero-fill that region once, before the workspace is first used (zeroing the
 * whole buffer after allocating it does this).  Every call, of any shape, leaves the region zero again when it
 * completes, so one workspace of sufficient size can serve calls of different shapes and of every verb one
 * after another.  The region's last 128 bytes hold failure flags instead of counters: a kernel that meets a
 * condition it cannot complete under (listed at dreams_workspace_status) sets one and leaves it set until
 * dreams_workspace_status reads and clears it.  Calls that overlap in time on one workspace (different
 * streams without synchronisation) race and give unspecified results.  Workspaces must be 256-byte aligned.
 */
#define DREAMS_WORKSPACE_COUNTER_BYTES 65536

/*
 * dreams_workspace_status -- the failures kernels flagged in `workspace` (device, 256-byte aligned, a workspace
 * of any verb, workspace_bytes >= DREAMS_WORKSPACE_COUNTER_BYTES, else DREAMS_ERR_WORKSPACE) since the last
 * check.  Synchronises `stream`, reads the flags, clears them, and returns DREAMS_OK if none was set, else
 * DREAMS_ERR_DEVICE with a message naming each flag.  The flags:
 *   attention (more than one piece per row set): the pieces of one set did not all run on one XCD, so the
 *       merge could not read their partial results from its XCD's L2 -- the rows of that set are NaN.  Not
 *       expected on an MI355X (consecutive workgroups of a dispatch run on consecutive XCDs, so workgroups
 *       whose ids agree mod 8 share one).
 *   a wait for another workgroup's results gave up (dreams_set_wait_limit; attention merges, sampled
 *       acceptance): that call's results are unspecified (attention rows NaN).
 * After a flagged failure, zero the workspace's counter region before it serves another call: arrivals that
 * came after a wait gave up can remain there.  Not for use under stream capture (it copies to the host and
 * synchronises).
 */
dreams_status_t dreams_workspace_status(void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * dreams_set_wait_limit -- the bound, in seconds (0 .. 60, default 0.2), on every wait of one workgroup for
 * another's results inside the library's kernels: the merging workgroups of dreams_tree_verify_attn (several
 * pieces per row set) and the pieces of dreams_tree_accept_sampled.  Those waits always end in normal operation
 * (a workgroup only waits for ones dispatched before it); a wait that reaches the bound gives up, its call's
 * results are unspecified, and the workspace's failure flag is set (dreams_workspace_status).  A limit of 0
 * makes every such wait give up at once, which exercises that path.  Applies to calls enqueued after it;
 * process-wide.
 */
dreams_status_t dreams_set_wait_limit(double seconds);

/*
 * Shape of one tree-verification attention call.
 *   batch            B >= 0 sequences
 *   num_q_heads      Hq >= 1 query heads
 *   num_kv_heads     Hkv >= 1 KV heads, Hq % Hkv == 0 (query head h reads KV head h / (Hq/Hkv))
 *   head_dim         D, 64 or 128
 *   num_nodes        T, 1..128 tree nodes per sequence, root included (node 0 = the last emitted token)
 *   cache_capacity   S_cap >= T slots per (sequence, KV head)
 *   max_kv_len       host-side upper bound on every kv_len[b], used only to plan the work split;
 *                    0 means S_cap - T.  Must satisfy 0 <= max_kv_len <= S_cap - T.
 *   num_splits       number of pieces the key axis of each (sequence, KV head) is cut into; 0 lets the
 *                    library choose from the shape and the device's compute-unit count.  Any value gives
 *                    the same result up to floating-point rounding order.
 *   dtype            type of q, the caches and out: DREAMS_BF16 (matrix-core path) or DREAMS_F32
 *   scale            softmax scale applied to q.k (normally 1/sqrt(D))
 */
typedef struct {
  int32_t batch;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t num_nodes;
  int32_t cache_capacity;
  int32_t max_kv_len;
  int32_t num_splits;
  dreams_dtype_t dtype;
  float scale;
} dreams_attn_desc_t;

/* Bytes of workspace dreams_tree_verify_attn needs for `desc` on the current device (0 if none: then the
 * call accepts a NULL workspace).  Non-zero when the key axis is cut into pieces: the pieces' partial
 * results live there, after the counter region every workspace starts with. */
dreams_status_t dreams_tree_verify_attn_workspace_size(const dreams_attn_desc_t* desc, size_t* bytes);

/* Number of pieces dreams_tree_verify_attn cuts the key axis of every (sequence, KV head) into for `desc` on
 * the current device (desc->num_splits, clamped, or the library's choice when it is 0). */
dreams_status_t dreams_tree_verify_attn_splits(const dreams_attn_desc_t* desc, int32_t* splits);

/*
 * dreams_tree_verify_attn -- the target model's parallel verification pass, attention part (the paper,
 * Section 2, "Speculative decoding": the target checks all draft tokens in one pass; Section 3.2 defines the
 * attention matrix softmax(Q K^T / sqrt(z))).  For every sequence b, query head h and tree node i:
 *
 *     out[b,h,i,:] = softmax_j( scale * q[b,h,i,:] . k[b,g,j,:] ) v[b,g,j,:],   g = h / (Hq/Hkv)
 *
 * over the visible slots j: every committed prefix slot 0..L_b-1 (image and text tokens alike -- the
 * paper's Section 2, "Vision-Language Models", notes every visual token stays in the KV cache and is
 * attended at each decoding step), plus slot L_b + n for every tree node n that is node i itself or one of
 * its ancestors.  lse[b,h,i] = log(sum_j exp(scale * q.k_j)) (natural log).  A row with no visible slot
 * (possible only with a tree_mask and L_b = 0) gives out = 0 and lse = -inf.
 *
 *   q          device [B, Hq, T, D]      queries of the tree nodes (after any positional rotation)
 *   k_cache    device [B, Hkv, S_cap, D] keys: slots [0, L_b) committed prefix, [L_b, L_b+T) the tree
 *                                         nodes' own keys in node order (written by the caller beforehand)
 *   v_cache    device [B, Hkv, S_cap, D] values, same layout
 *   kv_len     device [B] int32          L_b; the kernel clamps it into [0, S_cap - T]
 *   parent     device [B, T] int32       parent[b,0] = -1, 0 <= parent[b,i] < i; ignored when tree_mask is
 *                                         given.  An entry breaking these rules ends that node's ancestor walk.
 *   tree_mask  device [B, T, ceil(T/64)] uint64, or NULL: bit n of row i set <=> slot L_b+n is visible to
 *                                         node i.  Takes precedence over parent.
 *   out        device [B, Hq, T, D]      same dtype as q
 *   lse        device [B, Hq, T] float, or NULL
 *   workspace  device, >= dreams_tree_verify_attn_workspace_size bytes (see "Workspaces" above), or NULL
 *              when that size is 0.
 * Arithmetic: bf16 products accumulated in fp32 on the matrix cores, softmax statistics in fp32, one
 * rounding of the probabilities to bf16 before the value product; output rounded to the nearest bf16.  With
 * more than one piece of the key axis (dreams_tree_verify_attn_splits), each piece's output is rounded to
 * bf16 once more before the pieces are merged in fp32.
 */
dreams_status_t dreams_tree_verify_attn(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                        const void* v_cache, const int32_t* kv_len, const int32_t* parent,
                                        const uint64_t* tree_mask, void* out, float* lse, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/*
 * dreams_tree_verify_attn_noalloc -- dreams_tree_verify_attn for callers that cannot allocate device memory
 * (code under stream capture, tight serving loops, harnesses that forbid hipMalloc): the same arguments without
 * a workspace, the same kernels and the same results.  The scratch memory lives in a fixed array of
 * DREAMS_NOALLOC_SCRATCH_BYTES bytes inside the library, one per device, held until the process ends; the
 * call allocates and frees nothing.  Shapes whose workspace (dreams_tree_verify_attn_workspace_size) exceeds
 * that size return DREAMS_ERR_UNSUPPORTED before anything is enqueued.  The first call on a device also
 * enqueues one small kernel that clears the array's counters.  Every call on a device shares that device's
 * array, so calls that overlap in time on one device (different streams without synchronisation) race and
 * give unspecified results.  A failure a kernel flags (see dreams_workspace_status) stays in the array and
 * is not reported; the rows concerned are NaN.
 */
#define DREAMS_NOALLOC_SCRATCH_BYTES (16u << 20)
dreams_status_t dreams_tree_verify_attn_noalloc(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                                const void* v_cache, const int32_t* kv_len, const int32_t* parent,
                                                const uint64_t* tree_mask, void* out, float* lse, hipStream_t stream);

/*
 * dreams_tree_verify_attn_entropy -- dreams_tree_verify_attn, plus the attention entropy of every row: the
 * per-row term of the average attention entropy AE(l) by which the paper's Section 3.2 ("Adaptive
 * Intermediate Feature Distillation") ranks target layers.
 *
 *   entropy[b,h,i] = - sum_j A[j] ln A[j]   over the slots row (b,h,i) sees, A = its attention probabilities
 *                    (natural log; 0 for a row with no visible slot)
 *
 * Arguments, layouts, workspace and errors as dreams_tree_verify_attn; entropy is device [B, Hq, T] float
 * (required, 4-byte aligned).  The entropy is computed in the same pass over the keys as out and lse (one
 * more fp32 sum per row next to the softmax denominator), from the fp32 probabilities before their bf16
 * rounding.
 */
dreams_status_t dreams_tree_verify_attn_entropy(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                                const void* v_cache, const int32_t* kv_len, const int32_t* parent,
                                                const uint64_t* tree_mask, void* out, float* lse, float* entropy,
                                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * dreams_attn_entropy_mean -- AE of one layer (Section 3.2): the mean of `count` >= 1 row entropies, e.g. the
 * B*Hq*T values one dreams_tree_verify_attn_entropy call wrote (every head and sequence counts alike).
 * entropy: device [count] float; ae: device, one float (out).  Summed in fp64 in a fixed order.
 */
dreams_status_t dreams_attn_entropy_mean(int64_t count, const float* entropy, float* ae, hipStream_t stream);

/*
 * dreams_attn_entropy_select -- the distillation layer of Section 3.2: the layer l minimising
 * AE(l) + |AE(l) - AE(l-1)| (entropy plus its change from the layer below).  The change needs a
 * predecessor, so the candidates are l = 1 .. num_layers-1 (num_layers >= 2); scores are fp32 and ties go to
 * the smaller l.  ae: device [num_layers] float; best: device, one int32 (out).
 */
dreams_status_t dreams_attn_entropy_select(int32_t num_layers, const float* ae, int32_t* best, hipStream_t stream);

/*
 * Target-aware visual-token selection (the paper's Section 3.1, "Visual Token Compression", Eq. 2).
 *
 * dreams_visual_importance -- the importance of visual token j (cache slot vis_begin + j of every sequence):
 *   importance[b,j] = (1 / (Hq*T)) * sum over query heads h and rows i of A[b,h,i,vis_begin+j]
 * where A[b,h,i,.] is row (b,h,i)'s attention as dreams_tree_verify_attn defines it (same desc, q, k_cache and
 * kv_len; lse = that call's log-sum-exp output, [B, Hq, T]).  A visual slot at or past a sequence's prefix
 * length has importance 0; a row whose lse is -inf contributes nothing.  bf16 only (DREAMS_ERR_UNSUPPORTED
 * otherwise).  importance: device [B, vis_count] float (out).  Requires vis_begin >= 0, vis_count >= 1,
 * vis_begin + vis_count <= cache_capacity and B * ceil(vis_count / 256) <= (DREAMS_WORKSPACE_COUNTER_BYTES - 128) / 4
 * (DREAMS_ERR_UNSUPPORTED otherwise).  workspace: device, 256-byte aligned, >=
 * dreams_visual_importance_workspace_size bytes: the arrival-counter region every workspace starts with (see
 * "Workspaces" above), then B*Hkv*vis_count floats of per-KV-head partial sums.  Arithmetic: bf16 products, fp32
 * sums; the heads are summed in head order, so results are reproducible.
 */
dreams_status_t dreams_visual_importance_workspace_size(int32_t batch, int32_t num_kv_heads, int32_t vis_count,
                                                        size_t* bytes);
dreams_status_t dreams_visual_importance(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                         const int32_t* kv_len, const float* lse, int32_t vis_begin,
                                         int32_t vis_count, float* importance, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream);

/*
 * dreams_visual_topk -- the keep_count most important visual tokens of every sequence: keep[b] lists them in
 * increasing token order.  Ranking: larger importance first, the smaller token index among equal values
 * (exact fp32 comparisons; importance must not hold NaN).  importance device [B, vis_count] float, with
 * 1 <= vis_count <= DREAMS_VISUAL_MAX_TOKENS and 1 <= keep_count <= vis_count; keep device [B, keep_count] int32.
 */
#define DREAMS_VISUAL_MAX_TOKENS 8192
dreams_status_t dreams_visual_topk(int32_t batch, int32_t vis_count, int32_t keep_count, const float* importance,
                                   int32_t* keep, hipStream_t stream);

/*
 * dreams_visual_gather -- the kept tokens' K/V rows, for a cache that holds only them:
 *   k_out[b,g,m,:] = k_cache[b,g,vis_begin + keep[b,m],:]   (same for v), bit for bit
 * k_cache, v_cache device [B, Hkv, S_cap, D] of dtype; keep device [B, keep_count] int32 (as dreams_visual_topk
 * writes it); k_out, v_out device [B, Hkv, keep_count, D].  head_dim * element size must be a multiple of 16.
 * A kept token whose slot falls outside the cache leaves its output rows unwritten.
 */
dreams_status_t dreams_visual_gather(int32_t batch, int32_t num_kv_heads, int32_t head_dim, int32_t cache_capacity,
                                     dreams_dtype_t dtype, const void* k_cache, const void* v_cache,
                                     int32_t vis_begin, const int32_t* keep, int32_t keep_count, void* k_out,
                                     void* v_out, hipStream_t stream);

/*
 * Prefill statistics: the same quantities over a prompt's own causal attention, which is where the paper reads
 * them -- Eq. 2 (Section 3.1, "Visual Token Compression") scores visual tokens with the final layer's attention
 * weights of the prefilling pass, and AE(l) (Section 3.2) averages the attention entropy of a layer's rows over
 * the n prompt tokens.  Prompt b holds n_b = prompt_len[b] tokens (clamped to [0, num_rows]): queries in rows
 * 0..n_b-1 of q [B, Hq, num_rows, D], keys in slots 0..n_b-1 of k_cache [B, Hkv, cache_capacity, D], both bf16,
 * caller-owned device buffers; query head h reads KV head h / (Hq/Hkv).  Row i attends slots 0..i:
 *   A[b,h,i,j] = exp(scale * q_i . k_j - lse[b,h,i]),  lse[b,h,i] = log sum_{j <= i} exp(scale * q_i . k_j).
 * Arithmetic: bf16 products, fp32 sums.  head_dim 64 or 128 (DREAMS_ERR_UNSUPPORTED otherwise).
 */
typedef struct {
  int32_t batch;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t num_rows;        /* N: rows per head of q, the longest prompt */
  int32_t cache_capacity;  /* slots per (sequence, KV head) of k_cache, >= num_rows */
  float scale;
} dreams_prefill_desc_t;

/*
 * dreams_prefill_attn_stats -- lse[b,h,i] (natural log) and entropy[b,h,i] = -sum_{j<=i} A log A (nats) of every
 * prompt row; rows i >= n_b get lse = -inf and entropy 0.  lse and entropy: device [B, Hq, num_rows] float,
 * either may be NULL.  Nothing is allocated; no workspace.
 */
dreams_status_t dreams_prefill_attn_stats(const dreams_prefill_desc_t* desc, const void* q, const void* k_cache,
                                          const int32_t* prompt_len, float* lse, float* entropy,
                                          hipStream_t stream);

/*
 * dreams_prefill_attn_entropy_mean -- AE of one layer over prompts (Section 3.2): the sum of entropy
 * [B, Hq, num_rows] (as dreams_prefill_attn_stats wrote it: 0 past each prompt) over Hq * sum_b n_b rows, summed
 * in fp64 in a fixed order; 0 when no prompt has a row.  ae: device, one float (out).
 */
dreams_status_t dreams_prefill_attn_entropy_mean(int32_t batch, int32_t num_q_heads, int32_t num_rows,
                                                 const float* entropy, const int32_t* prompt_len, float* ae,
                                                 hipStream_t stream);

/*
 * dreams_prefill_visual_importance -- Eq. 2 over the prompt: for visual token j (slot vis_begin + j),
 *   importance[b,j] = (1 / (Hq * n_b)) * sum_h sum_{i < n_b} A[b,h,i,vis_begin+j]
 * (a slot past row i gets nothing from it; a slot at or past n_b has importance 0; n_b = 0 gives 0).  lse: the
 * [B, Hq, num_rows] output of dreams_prefill_attn_stats on the same inputs.  Requires vis_begin >= 0,
 * vis_count >= 1, vis_begin + vis_count <= num_rows.  workspace: as for dreams_visual_importance (size from
 * dreams_visual_importance_workspace_size(batch, num_kv_heads, vis_count); its counter region zero, and left
 * zero).  importance: device [B, vis_count] float (out).  The heads are summed in head order (reproducible).
 */
dreams_status_t dreams_prefill_visual_importance(const dreams_prefill_desc_t* desc, const void* q, const void* k_cache,
                                                 const int32_t* prompt_len, const float* lse, int32_t vis_begin,
                                                 int32_t vis_count, float* importance, void* workspace,
                                                 size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace dreams_tree_accept needs (0 only when batch is 0).  DREAMS_ERR_UNSUPPORTED if batch
 * exceeds (DREAMS_WORKSPACE_COUNTER_BYTES - 128) / 4 (one arrival counter per sequence, plus up to 8 group counters
 * per sequence while batch * 9 counters fit).  After the counters: one (value, index) pair per piece of each
 * row (rows of long vocabularies are cut into pieces). */
dreams_status_t dreams_tree_accept_workspace_size(int32_t batch, int32_t num_nodes, int32_t vocab,
                                                  size_t* bytes);

/*
 * dreams_tree_accept -- greedy acceptance (the paper, Section 2, "Speculative decoding": a draft token is
 * kept while it equals the target's own token at its position; at the first mismatch the target's token is
 * used instead), applied to every root-to-node path of the tree.
 *
 *   tgt[i]  = the smallest vocabulary index attaining max_v target_logits[b,i,v]   (-0.0 equals +0.0)
 *   node i is consistent iff i = 0, or its parent is consistent and draft_tokens[b,i] == tgt[parent[i]]
 *   last    = the consistent node of greatest depth, smallest index among equals
 *   accept_len[b]  = depth(last) = number of accepted draft tokens a  (the step emits a + 1 tokens)
 *   accept_path[b] = node ids root .. last (a + 1 entries), then -1 up to T entries
 *   next_token[b]  = tgt[last], the target's token emitted after the accepted drafts
 *
 *   target_logits  device [B, T, V] float, finite (NaN gives unspecified results)
 *   draft_tokens   device [B, T] int32 (entry 0 = root token, not checked)
 *   parent         device [B, T] int32, as for dreams_tree_verify_attn; a node whose ancestor walk
 *                  breaks the parent rules is never consistent
 *   accept_len     device [B] int32 (out)
 *   accept_path    device [B, T] int32 (out)
 *   next_token     device [B] int32 (out)
 *   target_argmax  device [B, T] int32 (out) or NULL: tgt[i] for every node
 *   workspace      device, >= dreams_tree_accept_workspace_size bytes (see "Workspaces" above).
 * Bit-exact: integer results only; every comparison is an fp32 comparison of the caller's logits.
 */
dreams_status_t dreams_tree_accept(int32_t batch, int32_t num_nodes, int32_t vocab, const float* target_logits,
                                   const int32_t* draft_tokens, const int32_t* parent, int32_t* accept_len,
                                   int32_t* accept_path, int32_t* next_token, int32_t* target_argmax,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace dreams_tree_accept_sampled needs (0 only when batch is 0).  DREAMS_ERR_UNSUPPORTED if
 * vocab exceeds 2^23 or if the arrival counters (one word per sequence, then 16 bytes per row: batch *
 * num_nodes rows) do not fit in DREAMS_WORKSPACE_COUNTER_BYTES - 128 (about 4000 rows).  After the counters: per row
 * 8 bytes of flags plus 40 bytes per piece of the vocabulary (pieces of 4096 entries, or of 8192 once
 * batch * num_nodes * ceil(vocab / 4096) exceeds 4096). */
dreams_status_t dreams_tree_accept_sampled_workspace_size(int32_t batch, int32_t num_nodes, int32_t vocab,
                                                          size_t* bytes);

/*
 * dreams_tree_accept_sampled -- acceptance at temperature tau > 0 (the paper reports its speedups at
 * temperature 1, Table 2): speculative sampling's accept-or-resample rule (Section 1; Section 2,
 * "Speculative decoding"), walked down the tree.  For every sequence b:
 *
 *   p_i = softmax(target_logits[b,i,:] / tau), q_i = softmax(draft_logits[b,i,:] / tau): the target's and the
 *         draft's distribution of the token that follows node i (node i's children are the draft's samples
 *         from q_i)
 *   walk: node = 0 (the root), r = p_node; the children c of node are tested in increasing index order:
 *         with x = draft_tokens[b,c], c is kept iff uniforms[b,c] * q_node(x) < r(x) (probability
 *         min(1, r(x)/q_node(x))); the walk moves to the first kept child and starts again there; after a
 *         rejection r becomes max(r - q_node, 0) / sum(max(r - q_node, 0)) (r is kept if that sum is 0)
 *   stop: at a node none of whose children is kept (a leaf included), with that node's residual r
 *   accept_len[b]  = number of kept children on the walk (the step emits accept_len + 1 tokens)
 *   accept_path[b] = node ids root .. last (accept_len + 1 entries), then -1 up to T entries
 *   next_token[b]  = the smallest x with sum_{y <= x} r(y) > uniforms[b,0] * sum_y r(y)
 *
 *   temperature    tau > 0, finite
 *   target_logits  device [B, T, V] float, finite
 *   draft_logits   device [B, T, V] float, finite
 *   draft_tokens   device [B, T] int32 (entry 0 = root token, not read); a token outside [0, V) is rejected
 *   parent         device [B, T] int32, as for dreams_tree_verify_attn; a node whose parent breaks the rules
 *                  (parent[i] outside [0, i)) is never kept
 *   uniforms       device [B, T] float in [0, 1): entry 0 draws the emitted token, entry c decides child c
 *   accept_len     device [B] int32 (out)
 *   accept_path    device [B, T] int32 (out)
 *   next_token     device [B] int32 (out)
 *   workspace      device, >= dreams_tree_accept_sampled_workspace_size bytes (see "Workspaces" above)
 * Probabilities are computed in fp64; the integer results equal those of the rule evaluated in fp64 except
 * where a uniform falls within rounding (about 1e-15 relative) of a decision threshold.
 */
dreams_status_t dreams_tree_accept_sampled(int32_t batch, int32_t num_nodes, int32_t vocab, double temperature,
                                           const float* target_logits, const float* draft_logits,
                                           const int32_t* draft_tokens, const int32_t* parent,
                                           const float* uniforms, int32_t* accept_len, int32_t* accept_path,
                                           int32_t* next_token, void* workspace, size_t workspace_bytes,
                                           hipStream_t stream);

/* Bytes of workspace dreams_tree_accept_lm_head needs (0 only when batch is 0): the 64 KiB counter region
 * (unused by this verb, kept so that one workspace serves every verb) and 8 bytes per row per tile of the
 * vocabulary (tiles of 128 entries while batch * num_nodes <= 64, else of 256).  DREAMS_ERR_UNSUPPORTED if
 * hidden is not a multiple of 256. */
dreams_status_t dreams_tree_accept_lm_head_workspace_size(int32_t batch, int32_t num_nodes, int32_t hidden,
                                                          int32_t vocab, size_t* bytes);

/*
 * dreams_tree_accept_lm_head -- dreams_tree_accept with the LM head fused in: the target logits of every tree
 * node are formed from its final hidden state and the LM head's weight (the paper, Section 2, "Speculative
 * decoding": the target's token at each position is the argmax of its logits),
 *
 *   logit[b,i,v] = sum_k hidden_states[b,i,k] * lm_weight[v,k]      (bf16 operands, fp32 accumulation)
 *
 * and the greedy rule of dreams_tree_accept is applied to them, without the logits ever being written to
 * memory.  tgt[i] is the smallest index attaining the row maximum of the logits as computed here (fp32, a
 * fixed order of accumulation); results are otherwise exactly those of dreams_tree_accept on these logits.
 *
 *   hidden         H, a multiple of 256
 *   hidden_states  device [B, T, H] bfloat16, 16-byte aligned
 *   lm_weight      device [V, H] bfloat16 (one row per vocabulary entry), 16-byte aligned
 *   draft_tokens, parent, accept_len, accept_path, next_token, target_argmax: as for dreams_tree_accept
 *   workspace      device, >= dreams_tree_accept_lm_head_workspace_size bytes (see "Workspaces" above).
 */
dreams_status_t dreams_tree_accept_lm_head(int32_t batch, int32_t num_nodes, int32_t hidden, int32_t vocab,
                                           const void* hidden_states, const void* lm_weight,
                                           const int32_t* draft_tokens, const int32_t* parent,
                                           int32_t* accept_len, int32_t* accept_path, int32_t* next_token,
                                           int32_t* target_argmax, void* workspace, size_t workspace_bytes,
                                           hipStream_t stream);

/*
 * dreams_kv_commit -- keeps the accepted path in the cache: for every layer, sequence b and KV head, and
 * k = 0 .. accept_len[b], slot kv_len_in[b] + k receives (bit for bit) the K and V rows of slot
 * kv_len_in[b] + accept_path[b,k]; then kv_len_out[b] = kv_len_in[b] + accept_len[b] + 1 (the root and the
 * accepted drafts are now committed; the bonus token's K/V is produced by the next step, where it is the
 * root).  Slots outside [kv_len_in[b], kv_len_in[b] + accept_len[b]] are not written.
 *
 *   num_layers          NL >= 1 caches; layer l starts layer_stride_elems elements after layer l-1
 *   k_cache, v_cache    device, per layer [B, Hkv, S_cap, D] of `dtype` (in place)
 *   kv_len_in           device [B] int32
 *   accept_path         device [B, path_stride] int32, as written by dreams_tree_accept
 *   accept_len          device [B] int32, clamped into [0, path_stride - 1]
 *   kv_len_out          device [B] int32 (out); must not alias kv_len_in
 * A path entry that is not a valid source (accept_path[b,k] < k, or kv_len_in[b] + accept_path[b,k] outside
 * the cache) is skipped.
 */
dreams_status_t dreams_kv_commit(int32_t num_layers, int64_t layer_stride_elems, int32_t batch,
                                 int32_t num_kv_heads, int32_t head_dim, int32_t cache_capacity,
                                 dreams_dtype_t dtype, void* k_cache, void* v_cache, const int32_t* kv_len_in,
                                 const int32_t* accept_path, const int32_t* accept_len, int32_t path_stride,
                                 int32_t* kv_len_out, hipStream_t stream);

/* Static description of a status code. */
const char* dreams_status_string(dreams_status_t status);

/* Message describing the calling thread's most recent failure ("" if none). Valid until its next call. */
const char* dreams_last_error_message(void);

/* Host-side check of a parent array (host memory): DREAMS_OK iff parent[0] == -1 and 0 <= parent[i] < i. */
dreams_status_t dreams_check_tree_host(const int32_t* parent, int32_t num_nodes);

/*
 * Measurement helper, not part of the method: reads `bytes` bytes at `src` once, with non-temporal 16-byte loads,
 * one contiguous chunk per workgroup over every compute unit, and writes one word per wave to `sink`
 * (DREAMS_STREAM_READ_SINK_WORDS words) so
 * that the loads cannot be elided.  Timed around, it gives the device's plain read bandwidth, the reference for
 * the share of the measured peak that the kernels above reach.
 *   src    device, 16-byte aligned; bytes a multiple of 16 (DREAMS_ERR_INVALID_ARG otherwise)
 *   sink   device, DREAMS_STREAM_READ_SINK_WORDS uint32 words (contents unspecified afterwards)
 */
#define DREAMS_STREAM_READ_SINK_WORDS 2048
dreams_status_t dreams_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DREAMS_H */

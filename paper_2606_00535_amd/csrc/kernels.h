// Internal interface between the host layer (dreams_api.hip) and the gfx950 kernels.  Not installed.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dreams {

// ------------------------------------------------------------------ cross-workgroup publication
// Workgroups hand partial results to the last of them to finish through device-scope ("sc1") stores and
// loads, which write through / read past the per-XCD L2 for exactly those words, plus a relaxed device-scope
// atomic counter issued after an explicit wait for the stores.  Release/acquire fences would instead write
// back and invalidate the whole L2 of the issuing XCD on every call.  (On gfx950 an atomic is the same
// instruction at every scope: it is always performed where every XCD sees it.)
__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_coherent(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t load_coherent(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Wait until every vector-memory operation this thread issued has completed (gfx9 s_waitcnt encoding:
// vmcnt = 0, expcnt and lgkmcnt left at their maxima).
__device__ __forceinline__ void wait_vector_memory() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }
// Arrival counter: returns true in exactly one workgroup, the one whose increment completes the count.
__device__ __forceinline__ bool arrive_last(uint32_t* counter, uint32_t expected) {
  return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == expected - 1;
}
__device__ __forceinline__ void reset_counter(uint32_t* counter) {
  __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Index of the accelerator complex die (XCD) the calling wave runs on.  Workgroup n of a launch runs on XCD
// n % 8 (the dispatcher deals workgroup ids round-robin over the dies); kernels that exchange data through a
// die's own L2 check this at run time.
__device__ __forceinline__ uint32_t xcd_id() {
  uint32_t x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return x & 7u;
}

// NaN-propagating maximum (IEEE maximum): lowers to v_maximum3_f32 chains with no canonicalising of the
// operands, where fmaxf needs both quietened first.  For maxima of scores, which are never NaN.
__device__ __forceinline__ float vmax(float x, float y) { return __builtin_elementwise_maximum(x, y); }

// ------------------------------------------------------------------------------ device-side failures
// The last 128 bytes of every workspace's counter region hold sticky failure flags: a kernel that detects a
// condition it cannot complete under sets a bit (device-scope atomic OR); dreams_workspace_status reports and
// clears them.  The counters of every verb live below kCounterWords.
constexpr int kCounterWords = (65536 - 128) / 4;    // words of the counter region that verbs may use
constexpr int kErrorWord = (65536 - 128) / 4;       // word index of the failure flags
constexpr uint32_t kErrXcdSplit = 1u;       // attention: pieces of one row set ran on different XCDs
constexpr uint32_t kErrWaitTimeout = 2u;    // a bounded wait for other workgroups gave up
// Default bound on every wait of one workgroup for another's results: 0.2 s of the 100 MHz real-time clock,
// far beyond any call (dreams_set_wait_limit changes it).
constexpr uint64_t kDefaultWaitTicks = 20000000;
__device__ __forceinline__ void raise_device_error(uint32_t* err, uint32_t bit) {
  if (err) __hip_atomic_fetch_or(err, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------------------------ tree attention
// Matrix-core (bf16) path: one workgroup = 4 waves, each wave owning 16 (narrow) or 32 (wide) query rows of
// one KV head for a whole piece of that head's key axis; the key axis of every (sequence, KV head, row
// group) is cut into `splits` pieces.
constexpr int kMaxNodes = 128;
constexpr int kAttnMaxSplits = 32;
// Fields of a row set's 64-bit merge counter: pieces started and pieces arrived (6-bit counts), a bit per
// arrived piece, then the sum (8 bits) and sum of squares (11 bits) of the started pieces' XCD ids (0..7).
constexpr int kCtrCountBits = 6, kCtrArrived = 6, kCtrMask = 12, kCtrXcdSum = 44, kCtrXcdSq = 52;
static_assert(kAttnMaxSplits < (1 << kCtrCountBits) && kCtrMask + kAttnMaxSplits <= kCtrXcdSum, "count fields");
static_assert(kAttnMaxSplits * 7 < (1 << (kCtrXcdSq - kCtrXcdSum)) && kAttnMaxSplits * 49 < (1 << (64 - kCtrXcdSq)),
              "XCD sum fields");

struct AttnArgs {
  const void* q;          // [B, Hq, T, D]
  const void* k;          // [B, Hkv, S_cap, D]
  const void* v;
  const int32_t* kv_len;  // [B]
  const int32_t* parent;  // [B, T] (unused when mask != nullptr)
  const uint64_t* mask;   // [B, T, ceil(T/64)] or nullptr
  void* out;              // [B, Hq, T, D]
  float* lse;             // [B, Hq, T] or nullptr
  float* entropy;         // [B, Hq, T] attention entropy of every row (nats), or nullptr
  // Several pieces per (sequence, KV head, row group) -- a "set": each piece stores its rows' normalised output
  // (bf16) and softmax state, and the set's pieces merge them, each a slice of the rows.
  __bf16* part_o;         // [sets, splits, rows_per_wg, D]   accumulator / sum, rounded to bf16
  float* part_ml;         // [sets, splits, rows_per_wg, 2]   (max in log2 units, sum)
  float* part_e;          // [sets, splits, rows_per_wg]      entropy terms (with entropy only)
  // The 64-bit counter word of set s at set_ctr[s * ctr_stride]: pieces started, pieces arrived, a bit per
  // arrived piece and an off-XCD mark (the next word is kept free).  Zero between calls.
  unsigned long long* set_ctr;
  int ctr_stride;         // 64-bit words between consecutive sets' counters (>= 2)
  uint32_t* err;          // the workspace's failure flags (splits > 1)
  uint64_t wait_ticks;    // bound on a piece's wait for the rest of its set (100 MHz real-time ticks)
  int B, Hq, Hkv, G, T, D, S_cap;
  int units;              // B * Hkv
  int rows_per_wg;        // query rows of one workgroup (64 or 128)
  int row_groups;         // ceil(G*T / rows_per_wg)
  int splits;
  int max_keys;           // host-side bound on L_b + T over the batch (plans the pieces of the key axis)
  int piece_by_len;       // 1: each sequence's pieces are cut from its own L_b + T (read before the first copies)
  float scale_log2;       // scale * log2(e)
};

// Query rows per workgroup the bf16 kernel uses for G*T rows per KV head.
int tree_attn_bf16_rows_per_wg(int rows_total);
int tree_attn_bf16_wgs_per_cu(int rows_per_wg);   // workgroups of that configuration per compute unit
hipError_t launch_tree_attn_bf16(const AttnArgs& a, hipStream_t stream);
hipError_t launch_tree_attn_f32(const AttnArgs& a, hipStream_t stream);

// ------------------------------------------------------------------------------- visual-token selection
constexpr int kCounterStride = 32;   // words between arrival counters that many workgroups hit (own cache line)
constexpr int kVisualMaxTokens = 8192;   // visual tokens per sequence the top-r sort holds (LDS)

struct VisualArgs {
  const void* q;          // [B, Hq, T, D] bf16
  const void* k;          // [B, Hkv, S_cap, D] bf16
  const int32_t* kv_len;  // [B] (verification rows: the prefix; prefill rows: the prompt length)
  const float* lse;       // [B, Hq, T] natural log-sum-exp of every row (from the attention call)
  // 0: the rows are a verification call's tree rows (every row sees the whole prefix); 1: the rows are a
  // prompt's own positions (T = the rows per head, row i sees slots 0..i, rows i >= kv_len[b] do not count)
  int prefill;
  float* partial;         // [B, Hkv, vis_count] workspace
  uint32_t* counters;     // [B, ceil(vis_count / 256)] arrival counters, counter_stride words apart (zero)
  int counter_stride;
  float* importance;      // [B, vis_count]
  int B, Hq, Hkv, G, T, D, S_cap;
  int vis_begin, vis_count;
  float scale_log2;       // scale * log2(e)
  int cus;                // compute units of the device (prefill rows: the workgroup order pairs long and short)
};
struct VisualGatherArgs {
  const void* k;
  const void* v;          // [B, Hkv, S_cap, D]
  const int32_t* keep;    // [B, r]
  void* k_out;
  void* v_out;            // [B, Hkv, r, D]
  int B, Hkv, S_cap, r, vis_begin;
  int row_bytes;          // D * element size, a multiple of 16
};
hipError_t launch_visual_importance(const VisualArgs& a, hipStream_t stream);

// ---------------------------------------------------------------------------- prefill attention statistics
struct PrefillArgs {
  const void* q;               // [B, Hq, N, D] bf16: the prompt's queries
  const void* k;               // [B, Hkv, S_cap, D] bf16: the prompt's keys in slots 0..N-1
  const int32_t* prompt_len;   // [B] n_b (clamped to [0, N])
  float* lse;                  // [B, Hq, N] or nullptr
  float* entropy;              // [B, Hq, N] or nullptr
  int B, Hq, Hkv, G, N, D, S_cap;
  float scale_log2;            // scale * log2(e)
  int cus;                     // compute units of the device (the workgroup order pairs long and short rows)
};
hipError_t launch_prefill_stats(const PrefillArgs& a, hipStream_t stream);
hipError_t launch_prefill_entropy_mean(int B, int Hq, int N, const float* entropy, const int32_t* prompt_len, float* ae,
                                       hipStream_t stream);
hipError_t launch_visual_topk(int B, int n, int r, const float* importance, int32_t* keep, hipStream_t stream);
hipError_t launch_visual_gather(const VisualGatherArgs& a, hipStream_t stream);

// Layer AE: the mean of `count` row entropies; the distillation layer from per-layer AE values.
hipError_t launch_attn_entropy_mean(long long count, const float* entropy, float* ae, hipStream_t stream);
hipError_t launch_attn_entropy_select(int num_layers, const float* ae, int32_t* best, hipStream_t stream);

// ---------------------------------------------------------------------------------------- acceptance
constexpr int kAcceptThreads = 256;
constexpr int kAcceptMaxChunks = kAcceptThreads;   // pieces per row, at most

struct AcceptArgs {
  const float* logits;    // [B, T, V]
  const int32_t* tokens;  // [B, T]
  const int32_t* parent;  // [B, T]
  int32_t* accept_len;    // [B]
  int32_t* accept_path;   // [B, T]
  int32_t* next_token;    // [B]
  int32_t* target_argmax; // [B, T] or nullptr
  float* part_val;        // [B, T, chunks] best value of each piece
  int32_t* part_idx;      // [B, T, chunks] its index
  uint32_t* counters;     // [B] per sequence, then group counters; zero between calls
  int B, T, V;
  int groups;             // group counters per sequence (1..8)
  int group_base;         // word index of the first group counter
  int group_stride;       // words between consecutive group counters (32: a 128-byte line each)
  int chunks;             // vocabulary pieces per row
  int chunk;              // elements per piece (multiple of 4 when vectorised)
  int vec4;               // logits rows are 16-byte aligned and V % 4 == 0
};

hipError_t launch_tree_accept(const AcceptArgs& a, hipStream_t stream);

// ------------------------------------------------------------------------------- sampled acceptance
// Every row of B * T vocabulary rows is cut into pieces.  With one-part pieces (4096 entries, a thread holding
// kSampledPerThreadRow consecutive entries) the launch has one workgroup per piece of every row, in row order:
// the piece's statistics, then the residual masses and accept decisions of the row's children, then (one
// piece per row) the token emitted if the walk ends there.  With four-part pieces (many pieces: 4 sub-pieces
// of 2048 entries, a thread holding kSampledPerThread consecutive entries of each) it has, in blockIdx order,
// first one per piece of every row ("stats" pieces: maxima and normalisers), then one per piece of every
// child node c, by c ("pass" pieces: the residual mass after c's rejection, and c's own accept decision).
constexpr int kSampledThreads = 256;
constexpr int kSampledPerThread = 8;
constexpr int kSampledPerThreadRow = 16;
constexpr int kSampledSubLarge = 4;         // sub-pieces per piece for problems of many pieces (else 1)
constexpr int kSampledMaxChunks = 1024;     // pieces per row, at most

struct SampledArgs {
  const float* target_logits;  // [B, T, V]
  const float* draft_logits;   // [B, T, V]
  const int32_t* tokens;       // [B, T]
  const int32_t* parent;       // [B, T]
  const float* uniforms;       // [B, T]
  int32_t* accept_len;         // [B]
  int32_t* accept_path;        // [B, T]
  int32_t* next_token;         // [B]
  uint32_t* seq_ctr;           // [B] rows finished per sequence
  uint32_t* row_words;         // [B * T] blocks of row_stride words: a 64-bit residual accumulator (arrivals in
                               // the top 11 bits, the fixed-point mass in the low 53), then the stats arrivals
  int row_stride;              // words per block: 4, 8 or 16
  double* piece_stat;          // [B, T, chunks, 4] per piece: target maximum and sum of exp((l - max) / tau)
                               // relative to it, then the same for the draft
  double* mass;                // [B, T, chunks] residual mass of each piece after rejecting child c
  int32_t* kept;               // [B, T] child c's decision
  int32_t* final_token;        // [B, T] the token emitted if the walk ends at node i
  double inv_tau;              // 1 / temperature (may be +inf)
  int B, T, V, chunks;
  int sub_pieces;              // 1 or kSampledSubLarge
  int vec4;                    // both logits tensors 16-byte aligned and V % 4 == 0
  uint32_t* err;               // the workspace's failure flags
  uint64_t wait_ticks;         // bound on every wait for another workgroup (100 MHz real-time ticks)
};

hipError_t launch_tree_accept_sampled(const SampledArgs& a, hipStream_t stream);

// ------------------------------------------------------------------------------ LM head + argmax
// A workgroup per (vocabulary tile, row tile) of the logits hidden * weight^T; each row's best (value, index)
// per vocabulary tile goes to part_val / part_idx, and a second kernel (a workgroup per sequence) merges them
// and runs the greedy path scan.
constexpr int kLmThreads = 256;
constexpr int kLmTile = 64;        // rows per workgroup while the rows fit one tile (by kLmTileSmall entries) ...
constexpr int kLmTileSmall = 128;  //     (vocabulary entries: 8 waves of 16)
constexpr int kLmTileBig = 256;    // ... and beyond: vocabulary entries per workgroup, by 128 rows (at most
constexpr int kLmMidRows = 128;    //     128 rows, three LDS ring stages) or by 256 rows (two stages)
constexpr int kLmBigRows = 256;
constexpr int kLmHiddenMultiple = 256;   // the hidden size must be a multiple (four quarters of 64-deep steps)

struct LmHeadArgs {
  const __bf16* hidden;    // [M, H], M = B * T
  const __bf16* weight;    // [V, H]
  const int32_t* tokens;   // [B, T]
  const int32_t* parent;   // [B, T]
  int32_t* accept_len;     // [B]
  int32_t* accept_path;    // [B, T]
  int32_t* next_token;     // [B]
  int32_t* target_argmax;  // [B, T] or nullptr
  float* part_val;         // [M, ntiles]
  int32_t* part_idx;       // [M, ntiles]
  int B, T, H, V, M, ntiles, mtiles;
  int rows;                // rows per workgroup: kLmTile (kLmTileSmall vocabulary entries each), else kLmMidRows or
                           // kLmBigRows (kLmTileBig entries each)
};

hipError_t launch_lm_head_accept(const LmHeadArgs& a, hipStream_t stream);

// ------------------------------------------------------------------------------------------ commit
constexpr int kCommitThreads = 256;
constexpr int kCommitRowsPerPass = 32;
constexpr int kCommitMaxRowBytes = 512;

struct CommitArgs {
  char* k;
  char* v;
  const int32_t* kv_len_in;
  const int32_t* path;
  const int32_t* accept_len;
  int32_t* kv_len_out;
  int64_t layer_stride_bytes;
  int NL, B, Hkv, S_cap, path_stride;
  int row_bytes;          // D * element size, multiple of 16, <= kCommitMaxRowBytes
};

hipError_t launch_kv_commit(const CommitArgs& a, hipStream_t stream);

// ------------------------------------------------------------------------------- stream read (measurement)
hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream);

}  // namespace dreams

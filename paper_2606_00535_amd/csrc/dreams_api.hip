// Host side of libdreams.so: argument checks, work planning, workspace layout, launches, error reporting.
// Every check that can be made on the host is made before anything is enqueued.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <atomic>
#include <mutex>
#include <string>

#include "dreams.h"
#include "kernels.h"

using namespace dreams;

namespace {

thread_local std::string g_error;

// Bound on every in-kernel wait for another workgroup (100 MHz real-time ticks); see dreams_set_wait_limit.
std::atomic<uint64_t> g_wait_ticks{kDefaultWaitTicks};

dreams_status_t fail(dreams_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return st;
}

dreams_status_t ok() {
  g_error.clear();
  return DREAMS_OK;
}

dreams_status_t hip_fail(hipError_t e, const char* what) {
  return fail(DREAMS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t n) { return ((uintptr_t)p % n) == 0; }

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Compute-unit count of the current device, cached per device.
dreams_status_t device_cus(int* cus) {
  static std::mutex mu;
  static int cache[64] = {0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(DREAMS_ERR_HIP, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (cache[dev] == 0) {
    int n = 0;
    e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(multiprocessor count)");
    cache[dev] = n > 0 ? n : 1;
  }
  *cus = cache[dev];
  return DREAMS_OK;
}

// ------------------------------------------------------------------------------------------ attention
// Every workspace starts with a fixed region of arrival counters, whatever the verb and shape, so a
// workspace left zero by one call is valid for any other call.
constexpr size_t kCounterBytes = DREAMS_WORKSPACE_COUNTER_BYTES;
static_assert(kCounterBytes == 65536, "counter region layout (kernels.h)");
// Counter words any verb may use; the region's last 128 bytes hold the device-side failure flags.
constexpr size_t kMaxCounters = kCounterWords;

struct AttnPlan {
  int G, rows_total, row_groups, units, splits;
  int rows_per_wg;   // query rows one workgroup owns
  int ctr_stride;    // 64-bit words between the sets' counters in the counter region
  size_t o_off, ml_off, e_off, bytes;
};

// 64-bit set counters the counter region holds (at the closest spacing).
constexpr long long kMaxSetCounters = (long long)kMaxCounters / 2;

constexpr int kPieceMinKeys = 128;   // keys per piece of the key axis, at least
constexpr int kPlanPieceKeys = 384;  // keys per piece, at least, where the library chooses the pieces

constexpr int kMaxSplitsRequest = 4096;

dreams_status_t check_attn_desc(const dreams_attn_desc_t* d) {
  if (!d) return fail(DREAMS_ERR_INVALID_ARG, "desc is NULL");
  if (d->batch < 0) return fail(DREAMS_ERR_INVALID_ARG, "batch = %d < 0", d->batch);
  if (d->num_q_heads < 1 || d->num_kv_heads < 1)
    return fail(DREAMS_ERR_INVALID_ARG, "num_q_heads = %d and num_kv_heads = %d must be >= 1", d->num_q_heads,
                d->num_kv_heads);
  if (d->num_q_heads % d->num_kv_heads != 0)
    return fail(DREAMS_ERR_INVALID_ARG, "num_q_heads = %d is not a multiple of num_kv_heads = %d", d->num_q_heads,
                d->num_kv_heads);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(DREAMS_ERR_UNSUPPORTED, "head_dim = %d (supported: 64, 128)", d->head_dim);
  if (d->num_nodes < 1 || d->num_nodes > kMaxNodes)
    return fail(DREAMS_ERR_INVALID_ARG, "num_nodes = %d outside [1, %d]", d->num_nodes, kMaxNodes);
  if (d->cache_capacity < d->num_nodes)
    return fail(DREAMS_ERR_INVALID_ARG, "cache_capacity = %d < num_nodes = %d", d->cache_capacity, d->num_nodes);
  if (d->max_kv_len < 0 || d->max_kv_len > d->cache_capacity - d->num_nodes)
    return fail(DREAMS_ERR_INVALID_ARG, "max_kv_len = %d outside [0, cache_capacity - num_nodes = %d]",
                d->max_kv_len, d->cache_capacity - d->num_nodes);
  if (d->num_splits < 0 || d->num_splits > kMaxSplitsRequest)
    return fail(DREAMS_ERR_INVALID_ARG, "num_splits = %d outside [0, %d]", d->num_splits, kMaxSplitsRequest);
  if (d->dtype != DREAMS_BF16 && d->dtype != DREAMS_F32)
    return fail(DREAMS_ERR_INVALID_ARG, "dtype = %d is not DREAMS_BF16 or DREAMS_F32", (int)d->dtype);
  if (!isfinite(d->scale)) return fail(DREAMS_ERR_INVALID_ARG, "scale is not finite");
  return DREAMS_OK;
}

dreams_status_t plan_attn(const dreams_attn_desc_t* d, AttnPlan* p) {
  dreams_status_t st = check_attn_desc(d);
  if (st != DREAMS_OK) return st;
  *p = AttnPlan{};
  p->G = d->num_q_heads / d->num_kv_heads;
  p->rows_total = p->G * d->num_nodes;
  p->rows_per_wg = tree_attn_bf16_rows_per_wg(p->rows_total);
  p->row_groups = (p->rows_total + p->rows_per_wg - 1) / p->rows_per_wg;
  p->units = d->batch * d->num_kv_heads;
  p->splits = 1;
  if (d->dtype == DREAMS_F32 || p->units == 0) return DREAMS_OK;

  const int max_len = d->max_kv_len > 0 ? d->max_kv_len : d->cache_capacity - d->num_nodes;
  const int n_keys = max_len + d->num_nodes;
  const int max_splits = (n_keys + kPieceMinKeys - 1) / kPieceMinKeys;
  int splits = d->num_splits;
  if (splits == 0) {
    int cus = 0;
    st = device_cus(&cus);
    if (st != DREAMS_OK) return st;
    // At most one workgroup per resident slot (one or two per compute unit, as the configuration's LDS allows),
    // in pieces of at least kPlanPieceKeys keys: shorter pieces cost more in their fixed start and merge than
    // they gain in parallel streams (llava7b_layer: 8 pieces of 400 keys 18.5 us, 16 of 200 keys 20.4 us).
    const long long slots = (long long)cus * tree_attn_bf16_wgs_per_cu(p->rows_per_wg);
    const long long wgs = (long long)p->units * p->row_groups;
    if (wgs < slots) {
      splits = (int)(slots / wgs);
      const int by_len = n_keys / kPlanPieceKeys;
      if (splits > by_len) splits = by_len;
    } else {
      // More workgroups than slots: a last round of workgroups that fills less than half of the chip cannot
      // keep the memory busy, so cut the key axis until it does (or the rounds come out whole).
      splits = 1;
      while (splits < 4 && (wgs * splits) % slots != 0 && (wgs * splits) % slots < slots / 2) ++splits;
    }
  }
  if (splits > max_splits) splits = max_splits;
  if (splits > kAttnMaxSplits) splits = kAttnMaxSplits;
  const long long sets = (long long)p->units * p->row_groups;
  if (2 * sets > kMaxSetCounters) splits = 1;   // no room for the sets' arrival counters: one piece each
  if (splits < 1) splits = 1;
  p->splits = splits;
  const long long grid = 8LL * ((p->units + 7) / 8) * splits * p->row_groups;
  if (grid > 0x7fffffffLL) return fail(DREAMS_ERR_UNSUPPORTED, "problem too large: %lld workgroups", grid);
  if (splits > 1) {
    // a 64-bit counter word per set (started, arrived, which arrived) and a free one, on a 128-byte line of their own
    // where there is room (atomics on one line serialise), then the pieces' partial results after the counter
    // region every workspace starts with
    int stride = 16;
    while (stride > 2 && sets * stride > kMaxSetCounters) stride >>= 1;
    p->ctr_stride = stride;
    const size_t rows = (size_t)sets * splits * p->rows_per_wg;
    p->o_off = kCounterBytes;
    p->ml_off = p->o_off + align_up(rows * d->head_dim * 2, 256);
    p->e_off = p->ml_off + align_up(rows * 2 * sizeof(float), 256);
    p->bytes = p->e_off + align_up(rows * sizeof(float), 256);
  }
  return DREAMS_OK;
}

// ----------------------------------------------------------------------------------------- acceptance
struct AcceptPlan {
  int chunks, chunk, groups, group_base, group_stride;
  size_t val_off, idx_off, bytes;
};

// Pieces of a row: 8192 logits (8 16-byte loads per thread) while the batch has fewer rows than about two
// workgroups per compute unit, so that the logits spread over the whole chip; otherwise up to 32768 logits
// (32 loads per thread) per piece, so that most rows are one piece and need no second merge level.
constexpr int kAcceptSmallPiece = 8192, kAcceptLargePiece = 32768, kAcceptTargetWgs = 512;
constexpr int kAcceptGroups = 8;   // group counters per sequence (see tree_accept.hip)

dreams_status_t plan_accept(int32_t B, int32_t T, int32_t V, AcceptPlan* p) {
  if (B < 0) return fail(DREAMS_ERR_INVALID_ARG, "batch = %d < 0", B);
  if (T < 1 || T > kMaxNodes) return fail(DREAMS_ERR_INVALID_ARG, "num_nodes = %d outside [1, %d]", T, kMaxNodes);
  if (V < 1) return fail(DREAMS_ERR_INVALID_ARG, "vocab = %d < 1", V);
  *p = AcceptPlan{};
  const long long rows = (long long)B * T;
  if (rows == 0) return DREAMS_OK;   // nothing to do, no workspace needed
  long long chunks = (V + kAcceptLargePiece - 1) / kAcceptLargePiece;
  if (rows < kAcceptTargetWgs) {
    const long long want = (kAcceptTargetWgs + rows - 1) / rows;
    const long long small = (V + kAcceptSmallPiece - 1) / kAcceptSmallPiece;
    chunks = want < small ? want : small;
    if (chunks < 1) chunks = 1;
  }
  if (chunks > kAcceptMaxChunks) chunks = kAcceptMaxChunks;
  long long chunk = (V + chunks - 1) / chunks;
  chunk = (chunk + 3) / 4 * 4;
  chunks = (V + chunk - 1) / chunk;
  if (rows * chunks > 0x7fffffffLL) return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");
  // counters: one per sequence, then up to 8 group counters per sequence while they fit
  if ((size_t)B > kMaxCounters)
    return fail(DREAMS_ERR_UNSUPPORTED, "batch = %d exceeds the %zu arrival counters", B, kMaxCounters);
  const long long per_seq = (long long)T * chunks;
  // group counters after the sequence counters, a 128-byte line apart where they fit (else closer); with
  // no room for them the sequence counter serves as the one group counter (its last arrival resets it and
  // arrives again, alone)
  const long long groups = per_seq < kAcceptGroups ? per_seq : kAcceptGroups;
  const size_t base = ((size_t)B + 31) / 32 * 32;
  size_t stride = 32;
  while (stride > 1 && base + (size_t)B * groups * stride > kMaxCounters) stride /= 2;
  p->chunks = (int)chunks;
  p->chunk = (int)chunk;
  if (base + (size_t)B * groups * stride <= kMaxCounters) {
    p->groups = (int)groups;
    p->group_base = (int)base;
    p->group_stride = (int)stride;
  } else {
    p->groups = 1;
    p->group_base = 0;
    p->group_stride = 1;
  }
  const size_t parts = (size_t)rows * chunks;
  p->val_off = kCounterBytes;
  p->idx_off = p->val_off + align_up(parts * sizeof(float), 256);
  p->bytes = p->idx_off + align_up(parts * sizeof(int32_t), 256);
  return DREAMS_OK;
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const char* pa = (const char*)a;
  const char* pb = (const char*)b;
  return pa < pb + nb && pb < pa + na;
}

}  // namespace

extern "C" {

dreams_status_t dreams_tree_verify_attn_workspace_size(const dreams_attn_desc_t* desc, size_t* bytes) {
  if (!bytes) return fail(DREAMS_ERR_INVALID_ARG, "bytes is NULL");
  AttnPlan p;
  dreams_status_t st = plan_attn(desc, &p);
  if (st != DREAMS_OK) return st;
  *bytes = p.bytes;
  return ok();
}

}  // extern "C"

namespace {

// The checks of an attention call's tensor arguments (batch 0 needs none).
dreams_status_t check_attn_tensors(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                   const void* v_cache, const int32_t* kv_len, const int32_t* parent,
                                   const uint64_t* tree_mask, const void* out, const float* lse) {
  dreams_status_t st = check_attn_desc(desc);
  if (st != DREAMS_OK) return st;
  if (desc->batch == 0) return DREAMS_OK;
  if (!q || !k_cache || !v_cache || !kv_len || !out)
    return fail(DREAMS_ERR_INVALID_ARG, "q, k_cache, v_cache, kv_len and out must not be NULL");
  if (!parent && !tree_mask) return fail(DREAMS_ERR_INVALID_ARG, "either parent or tree_mask must be given");
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16))
    return fail(DREAMS_ERR_INVALID_ARG, "q, k_cache, v_cache and out must be 16-byte aligned");
  if (!aligned(kv_len, 4) || (parent && !aligned(parent, 4)) || (lse && !aligned(lse, 4)) ||
      (tree_mask && !aligned(tree_mask, 8)))
    return fail(DREAMS_ERR_INVALID_ARG, "kv_len, parent, lse or tree_mask is misaligned");
  if (desc->dtype == DREAMS_F32 && (long long)desc->batch * desc->num_q_heads * desc->num_nodes > 0x7fffffffLL)
    return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");
  return DREAMS_OK;
}

dreams_status_t verify_attn(const dreams_attn_desc_t* desc, const void* q, const void* k_cache, const void* v_cache,
                            const int32_t* kv_len, const int32_t* parent, const uint64_t* tree_mask, void* out,
                            float* lse, float* entropy, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  dreams_status_t st = check_attn_tensors(desc, q, k_cache, v_cache, kv_len, parent, tree_mask, out, lse);
  if (st != DREAMS_OK) return st;
  if (desc->batch == 0) return ok();
  AttnPlan p;
  st = plan_attn(desc, &p);
  if (st != DREAMS_OK) return st;
  if (p.bytes > 0) {
    if (!workspace) return fail(DREAMS_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", p.bytes);
    if (workspace_bytes < p.bytes)
      return fail(DREAMS_ERR_WORKSPACE, "workspace has %zu bytes, %zu are needed", workspace_bytes, p.bytes);
    if (!aligned(workspace, 256)) return fail(DREAMS_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  }

  AttnArgs a{};
  a.q = q;
  a.k = k_cache;
  a.v = v_cache;
  a.kv_len = kv_len;
  a.parent = parent;
  a.mask = tree_mask;
  a.out = out;
  a.lse = lse;
  a.entropy = entropy;
  char* ws = (char*)workspace;
  a.part_o = p.bytes ? (__bf16*)(ws + p.o_off) : nullptr;
  a.part_ml = p.bytes ? (float*)(ws + p.ml_off) : nullptr;
  a.part_e = p.bytes ? (float*)(ws + p.e_off) : nullptr;
  a.set_ctr = p.bytes ? (unsigned long long*)ws : nullptr;
  a.ctr_stride = p.ctr_stride;
  a.wait_ticks = g_wait_ticks.load(std::memory_order_relaxed);
  a.err = p.bytes ? (uint32_t*)ws + kErrorWord : nullptr;
  a.B = desc->batch;
  a.Hq = desc->num_q_heads;
  a.Hkv = desc->num_kv_heads;
  a.G = p.G;
  a.T = desc->num_nodes;
  a.D = desc->head_dim;
  a.S_cap = desc->cache_capacity;
  a.units = p.units;
  a.rows_per_wg = p.rows_per_wg;
  a.row_groups = p.row_groups;
  a.splits = p.splits;
  a.max_keys = (desc->max_kv_len > 0 ? desc->max_kv_len : desc->cache_capacity - desc->num_nodes) + desc->num_nodes;
  a.piece_by_len = desc->batch > 1 && p.splits > 1 ? 1 : 0;
  a.scale_log2 = desc->scale * 1.4426950408889634f;
  hipError_t e = desc->dtype == DREAMS_F32 ? launch_tree_attn_f32(a, stream) : launch_tree_attn_bf16(a, stream);
  if (e != hipSuccess) return hip_fail(e, "tree attention launch");
  return ok();
}

// ------------------------------------------------------------------ scratch for the allocation-free call
// A file-scope device array replaces the caller's workspace in dreams_tree_verify_attn_noalloc.  In host code
// `scratch` names a host-side stand-in, not device memory: its device address is taken once per device with
// hipGetSymbolAddress (every device holds its own copy, at its own address) and only that address is used.
constexpr size_t kScratchBytes = DREAMS_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;

// zero-fills n words (used instead of hipMemsetAsync, which a graph capture must not record)
__global__ void fill_zero_words(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = 0u;
}

// The device address of this device's scratch array; on the first call on a device, also clears its counter
// region (stream-ordered before the caller's kernels).
dreams_status_t scratch_for_current_device(hipStream_t stream, void** ptr) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {nullptr};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(DREAMS_ERR_HIP, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || !aligned(p, 256)) return fail(DREAMS_ERR_HIP, "scratch array at %p is not 256-byte aligned", p);
    hipLaunchKernelGGL(fill_zero_words, dim3(64), dim3(256), 0, stream, (uint32_t*)p, kCounterBytes / 4);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "clearing the scratch counters");
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return DREAMS_OK;
}

}  // namespace

extern "C" {

dreams_status_t dreams_tree_verify_attn_noalloc(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                                const void* v_cache, const int32_t* kv_len, const int32_t* parent,
                                                const uint64_t* tree_mask, void* out, float* lse, hipStream_t stream) {
  dreams_status_t st = check_attn_tensors(desc, q, k_cache, v_cache, kv_len, parent, tree_mask, out, lse);
  if (st != DREAMS_OK) return st;
  if (desc->batch == 0) return ok();
  AttnPlan p;
  st = plan_attn(desc, &p);
  if (st != DREAMS_OK) return st;
  if (p.bytes > kScratchBytes)
    return fail(DREAMS_ERR_UNSUPPORTED,
                "this shape needs %zu bytes of scratch, more than the %zu bytes of the allocation-free call "
                "(use dreams_tree_verify_attn with a workspace)", p.bytes, kScratchBytes);
  void* ws = nullptr;
  if (p.bytes > 0) {
    st = scratch_for_current_device(stream, &ws);
    if (st != DREAMS_OK) return st;
  }
  return verify_attn(desc, q, k_cache, v_cache, kv_len, parent, tree_mask, out, lse, nullptr, ws, p.bytes, stream);
}

dreams_status_t dreams_tree_verify_attn(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                        const void* v_cache, const int32_t* kv_len, const int32_t* parent,
                                        const uint64_t* tree_mask, void* out, float* lse, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  return verify_attn(desc, q, k_cache, v_cache, kv_len, parent, tree_mask, out, lse, nullptr, workspace,
                     workspace_bytes, stream);
}

dreams_status_t dreams_tree_verify_attn_entropy(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                                const void* v_cache, const int32_t* kv_len, const int32_t* parent,
                                                const uint64_t* tree_mask, void* out, float* lse, float* entropy,
                                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!entropy) return fail(DREAMS_ERR_INVALID_ARG, "entropy must not be NULL");
  if (!aligned(entropy, 4)) return fail(DREAMS_ERR_INVALID_ARG, "entropy is misaligned");
  return verify_attn(desc, q, k_cache, v_cache, kv_len, parent, tree_mask, out, lse, entropy, workspace,
                     workspace_bytes, stream);
}

dreams_status_t dreams_attn_entropy_mean(int64_t count, const float* entropy, float* ae, hipStream_t stream) {
  if (count < 1) return fail(DREAMS_ERR_INVALID_ARG, "count = %lld, at least 1 row is needed", (long long)count);
  if (!entropy || !ae) return fail(DREAMS_ERR_INVALID_ARG, "entropy and ae must not be NULL");
  if (!aligned(entropy, 4) || !aligned(ae, 4)) return fail(DREAMS_ERR_INVALID_ARG, "entropy or ae is misaligned");
  hipError_t e = launch_attn_entropy_mean((long long)count, entropy, ae, stream);
  if (e != hipSuccess) return hip_fail(e, "attention entropy mean launch");
  return ok();
}

dreams_status_t dreams_attn_entropy_select(int32_t num_layers, const float* ae, int32_t* best, hipStream_t stream) {
  if (num_layers < 2) return fail(DREAMS_ERR_INVALID_ARG, "num_layers = %d, at least 2 are needed", num_layers);
  if (!ae || !best) return fail(DREAMS_ERR_INVALID_ARG, "ae and best must not be NULL");
  if (!aligned(ae, 4) || !aligned(best, 4)) return fail(DREAMS_ERR_INVALID_ARG, "ae or best is misaligned");
  hipError_t e = launch_attn_entropy_select(num_layers, ae, best, stream);
  if (e != hipSuccess) return hip_fail(e, "attention entropy layer selection launch");
  return ok();
}

dreams_status_t dreams_tree_accept_workspace_size(int32_t batch, int32_t num_nodes, int32_t vocab, size_t* bytes) {
  if (!bytes) return fail(DREAMS_ERR_INVALID_ARG, "bytes is NULL");
  AcceptPlan p;
  dreams_status_t st = plan_accept(batch, num_nodes, vocab, &p);
  if (st != DREAMS_OK) return st;
  *bytes = p.bytes;
  return ok();
}

dreams_status_t dreams_tree_accept(int32_t batch, int32_t num_nodes, int32_t vocab, const float* target_logits,
                                   const int32_t* draft_tokens, const int32_t* parent, int32_t* accept_len,
                                   int32_t* accept_path, int32_t* next_token, int32_t* target_argmax,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
  AcceptPlan p;
  dreams_status_t st = plan_accept(batch, num_nodes, vocab, &p);
  if (st != DREAMS_OK) return st;
  if (batch == 0) return ok();
  if (!target_logits || !draft_tokens || !parent || !accept_len || !accept_path || !next_token)
    return fail(DREAMS_ERR_INVALID_ARG,
                "target_logits, draft_tokens, parent, accept_len, accept_path and next_token must not be NULL");
  if (!aligned(target_logits, 4) || !aligned(draft_tokens, 4) || !aligned(parent, 4) || !aligned(accept_len, 4) ||
      !aligned(accept_path, 4) || !aligned(next_token, 4) || (target_argmax && !aligned(target_argmax, 4)))
    return fail(DREAMS_ERR_INVALID_ARG, "an int32/float argument is not 4-byte aligned");
  if (!workspace) return fail(DREAMS_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", p.bytes);
  if (workspace_bytes < p.bytes)
    return fail(DREAMS_ERR_WORKSPACE, "workspace has %zu bytes, %zu are needed", workspace_bytes, p.bytes);
  if (!aligned(workspace, 256)) return fail(DREAMS_ERR_WORKSPACE, "workspace must be 256-byte aligned");

  AcceptArgs a{};
  a.logits = target_logits;
  a.tokens = draft_tokens;
  a.parent = parent;
  a.accept_len = accept_len;
  a.accept_path = accept_path;
  a.next_token = next_token;
  a.target_argmax = target_argmax;
  char* ws = (char*)workspace;
  a.part_val = (float*)(ws + p.val_off);
  a.part_idx = (int32_t*)(ws + p.idx_off);
  a.counters = (uint32_t*)ws;
  a.B = batch;
  a.T = num_nodes;
  a.V = vocab;
  a.groups = p.groups;
  a.group_base = p.group_base;
  a.group_stride = p.group_stride;
  a.chunks = p.chunks;
  a.chunk = p.chunk;
  a.vec4 = (vocab % 4 == 0) && aligned(target_logits, 16);
  hipError_t e = launch_tree_accept(a, stream);
  if (e != hipSuccess) return hip_fail(e, "tree accept launch");
  return ok();
}

// ------------------------------------------------------------------------------------- sampled acceptance
constexpr long long kSampledLargeFrom = 4096;   // stats workgroups beyond which pieces are large

struct SampledPlan {
  int sub_pieces, chunks, row_stride;
  size_t row_base, piece_off, mass_off, flag_off, bytes;
};

dreams_status_t plan_sampled(int32_t B, int32_t T, int32_t V, SampledPlan* p) {
  if (B < 0) return fail(DREAMS_ERR_INVALID_ARG, "batch = %d < 0", B);
  if (T < 1 || T > kMaxNodes) return fail(DREAMS_ERR_INVALID_ARG, "num_nodes = %d outside [1, %d]", T, kMaxNodes);
  if (V < 1) return fail(DREAMS_ERR_INVALID_ARG, "vocab = %d < 1", V);
  *p = SampledPlan{};
  if (B == 0) return DREAMS_OK;
  // pieces of 4096 entries while there are at most 16 statistics workgroups per compute unit (the wait chain
  // dominates: each piece computes p and q before it waits, and fewer pieces a row wait for fewer arrivals:
  // llava7b_layer 29.5 -> 28.6 us, llava13b_layer 140 (split form) -> 114 us, against 2048-entry pieces);
  // beyond that, pieces of 8192 entries in four parts (the split form, each part streamed after the waits)
  const long long small = (long long)kSampledThreads * kSampledPerThreadRow;
  const long long large = (long long)kSampledThreads * kSampledPerThread * kSampledSubLarge;
  long long sub = 1, chunks = ((long long)V + small - 1) / small;
  if ((long long)B * T * chunks > kSampledLargeFrom || chunks > kSampledMaxChunks) {
    sub = kSampledSubLarge;
    chunks = ((long long)V + large - 1) / large;
  }
  if (chunks > kSampledMaxChunks)
    return fail(DREAMS_ERR_UNSUPPORTED, "vocab = %d exceeds %lld", V, (long long)kSampledMaxChunks * large);
  if ((long long)B * (2 * T - 1) * chunks > 0x7fffffffLL) return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");
  // counter region: one word per sequence, then a block of 4, 8 or 16 words per row (as many as fit)
  const size_t rows = (size_t)B * T, base = ((size_t)B + 63) / 64 * 64;
  if (base + rows * 4 > kMaxCounters)
    return fail(DREAMS_ERR_UNSUPPORTED, "batch * num_nodes = %zu rows exceed the arrival counters (%zu)", rows,
                (kMaxCounters - base) / 4);
  size_t stride = 16;
  while (stride > 4 && base + rows * stride > kMaxCounters) stride >>= 1;
  p->sub_pieces = (int)sub;
  p->chunks = (int)chunks;
  p->row_stride = (int)stride;
  p->row_base = base;
  size_t off = kCounterBytes;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) / 256 * 256;
    return at;
  };
  p->piece_off = take(rows * chunks * 4 * sizeof(double));
  p->mass_off = take(rows * chunks * sizeof(double));
  p->flag_off = take(rows * 2 * sizeof(int32_t));
  p->bytes = off;
  return DREAMS_OK;
}

dreams_status_t dreams_tree_accept_sampled_workspace_size(int32_t batch, int32_t num_nodes, int32_t vocab,
                                                          size_t* bytes) {
  if (!bytes) return fail(DREAMS_ERR_INVALID_ARG, "bytes is NULL");
  SampledPlan p;
  dreams_status_t st = plan_sampled(batch, num_nodes, vocab, &p);
  if (st != DREAMS_OK) return st;
  *bytes = p.bytes;
  return ok();
}

dreams_status_t dreams_tree_accept_sampled(int32_t batch, int32_t num_nodes, int32_t vocab, double temperature,
                                           const float* target_logits, const float* draft_logits,
                                           const int32_t* draft_tokens, const int32_t* parent,
                                           const float* uniforms, int32_t* accept_len, int32_t* accept_path,
                                           int32_t* next_token, void* workspace, size_t workspace_bytes,
                                           hipStream_t stream) {
  SampledPlan p;
  dreams_status_t st = plan_sampled(batch, num_nodes, vocab, &p);
  if (st != DREAMS_OK) return st;
  if (!(temperature > 0.0) || !isfinite(temperature))
    return fail(DREAMS_ERR_INVALID_ARG, "temperature = %g is not a positive finite number", temperature);
  if (batch == 0) return ok();
  if (!target_logits || !draft_logits || !draft_tokens || !parent || !uniforms || !accept_len || !accept_path ||
      !next_token)
    return fail(DREAMS_ERR_INVALID_ARG,
                "target_logits, draft_logits, draft_tokens, parent, uniforms, accept_len, accept_path and "
                "next_token must not be NULL");
  if (!aligned(target_logits, 4) || !aligned(draft_logits, 4) || !aligned(draft_tokens, 4) || !aligned(parent, 4) ||
      !aligned(uniforms, 4) || !aligned(accept_len, 4) || !aligned(accept_path, 4) || !aligned(next_token, 4))
    return fail(DREAMS_ERR_INVALID_ARG, "an int32/float argument is not 4-byte aligned");
  if (!workspace) return fail(DREAMS_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", p.bytes);
  if (workspace_bytes < p.bytes)
    return fail(DREAMS_ERR_WORKSPACE, "workspace has %zu bytes, %zu are needed", workspace_bytes, p.bytes);
  if (!aligned(workspace, 256)) return fail(DREAMS_ERR_WORKSPACE, "workspace must be 256-byte aligned");

  SampledArgs a{};
  a.target_logits = target_logits;
  a.draft_logits = draft_logits;
  a.tokens = draft_tokens;
  a.parent = parent;
  a.uniforms = uniforms;
  a.accept_len = accept_len;
  a.accept_path = accept_path;
  a.next_token = next_token;
  char* ws = (char*)workspace;
  uint32_t* ctr = (uint32_t*)ws;
  a.seq_ctr = ctr;
  a.row_words = ctr + p.row_base;
  a.row_stride = p.row_stride;
  a.piece_stat = (double*)(ws + p.piece_off);
  a.mass = (double*)(ws + p.mass_off);
  a.kept = (int32_t*)(ws + p.flag_off);
  a.final_token = a.kept + (size_t)batch * num_nodes;
  a.inv_tau = 1.0 / temperature;
  a.B = batch;
  a.T = num_nodes;
  a.V = vocab;
  a.chunks = p.chunks;
  a.sub_pieces = p.sub_pieces;
  a.vec4 = (vocab % 4 == 0) && aligned(target_logits, 16) && aligned(draft_logits, 16);
  a.err = ctr + kErrorWord;
  a.wait_ticks = g_wait_ticks.load(std::memory_order_relaxed);
  hipError_t e = launch_tree_accept_sampled(a, stream);
  if (e != hipSuccess) return hip_fail(e, "sampled tree accept launch");
  return ok();
}

// ----------------------------------------------------------------------------------- LM head + argmax
struct LmPlan {
  int tile, rows, ntiles;
  size_t val_off, idx_off, bytes;
};

dreams_status_t plan_lm_head(int32_t B, int32_t T, int32_t H, int32_t V, LmPlan* p) {
  if (B < 0) return fail(DREAMS_ERR_INVALID_ARG, "batch = %d < 0", B);
  if (T < 1 || T > kMaxNodes) return fail(DREAMS_ERR_INVALID_ARG, "num_nodes = %d outside [1, %d]", T, kMaxNodes);
  if (V < 1) return fail(DREAMS_ERR_INVALID_ARG, "vocab = %d < 1", V);
  if (H < 1) return fail(DREAMS_ERR_INVALID_ARG, "hidden = %d < 1", H);
  if (H % kLmHiddenMultiple)
    return fail(DREAMS_ERR_UNSUPPORTED, "hidden = %d is not a multiple of %d", H, kLmHiddenMultiple);
  *p = LmPlan{};
  if (B == 0) return DREAMS_OK;
  // one 64-row tile while the rows fit it (the weights stream once, 128 vocabulary entries per workgroup); beyond,
  // 256 vocabulary entries by 128
  // rows (up to 128 rows) or by 256 rows, so that every operand tile is re-read four to eight times less often
  const long long M = (long long)B * T;
  const int tile = M <= kLmTile ? kLmTileSmall : kLmTileBig;
  const int rows = M <= kLmTile ? kLmTile : M <= kLmMidRows ? kLmMidRows : kLmBigRows;
  const long long ntiles = ((long long)V + tile - 1) / tile;
  if ((M + rows - 1) / rows * ntiles > 0x7fffffffLL) return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");
  p->tile = tile;
  p->rows = rows;
  p->ntiles = (int)ntiles;
  size_t off = kCounterBytes;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) / 256 * 256;
    return at;
  };
  p->val_off = take((size_t)M * ntiles * sizeof(float));
  p->idx_off = take((size_t)M * ntiles * sizeof(int32_t));
  p->bytes = off;
  return DREAMS_OK;
}

dreams_status_t dreams_tree_accept_lm_head_workspace_size(int32_t batch, int32_t num_nodes, int32_t hidden,
                                                          int32_t vocab, size_t* bytes) {
  if (!bytes) return fail(DREAMS_ERR_INVALID_ARG, "bytes is NULL");
  LmPlan p;
  dreams_status_t st = plan_lm_head(batch, num_nodes, hidden, vocab, &p);
  if (st != DREAMS_OK) return st;
  *bytes = p.bytes;
  return ok();
}

dreams_status_t dreams_tree_accept_lm_head(int32_t batch, int32_t num_nodes, int32_t hidden, int32_t vocab,
                                           const void* hidden_states, const void* lm_weight,
                                           const int32_t* draft_tokens, const int32_t* parent,
                                           int32_t* accept_len, int32_t* accept_path, int32_t* next_token,
                                           int32_t* target_argmax, void* workspace, size_t workspace_bytes,
                                           hipStream_t stream) {
  LmPlan p;
  dreams_status_t st = plan_lm_head(batch, num_nodes, hidden, vocab, &p);
  if (st != DREAMS_OK) return st;
  if (batch == 0) return ok();
  if (!hidden_states || !lm_weight || !draft_tokens || !parent || !accept_len || !accept_path || !next_token)
    return fail(DREAMS_ERR_INVALID_ARG,
                "hidden_states, lm_weight, draft_tokens, parent, accept_len, accept_path and next_token must not be "
                "NULL");
  if (!aligned(hidden_states, 16) || !aligned(lm_weight, 16))
    return fail(DREAMS_ERR_INVALID_ARG, "hidden_states and lm_weight must be 16-byte aligned");
  if (!aligned(draft_tokens, 4) || !aligned(parent, 4) || !aligned(accept_len, 4) || !aligned(accept_path, 4) ||
      !aligned(next_token, 4) || (target_argmax && !aligned(target_argmax, 4)))
    return fail(DREAMS_ERR_INVALID_ARG, "an int32 argument is not 4-byte aligned");
  if (!workspace) return fail(DREAMS_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", p.bytes);
  if (workspace_bytes < p.bytes)
    return fail(DREAMS_ERR_WORKSPACE, "workspace has %zu bytes, %zu are needed", workspace_bytes, p.bytes);
  if (!aligned(workspace, 256)) return fail(DREAMS_ERR_WORKSPACE, "workspace must be 256-byte aligned");

  LmHeadArgs a{};
  a.hidden = (const __bf16*)hidden_states;
  a.weight = (const __bf16*)lm_weight;
  a.tokens = draft_tokens;
  a.parent = parent;
  a.accept_len = accept_len;
  a.accept_path = accept_path;
  a.next_token = next_token;
  a.target_argmax = target_argmax;
  char* ws = (char*)workspace;
  a.part_val = (float*)(ws + p.val_off);
  a.part_idx = (int32_t*)(ws + p.idx_off);
  a.B = batch;
  a.T = num_nodes;
  a.H = hidden;
  a.V = vocab;
  a.M = batch * num_nodes;
  a.ntiles = p.ntiles;
  a.rows = p.rows;
  a.mtiles = (a.M + p.rows - 1) / p.rows;
  hipError_t e = launch_lm_head_accept(a, stream);
  if (e != hipSuccess) return hip_fail(e, "LM head accept launch");
  return ok();
}

dreams_status_t dreams_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream) {
  if (!src || !sink) return fail(DREAMS_ERR_INVALID_ARG, "src and sink must not be NULL");
  if (!aligned(src, 16) || bytes % 16 != 0)
    return fail(DREAMS_ERR_INVALID_ARG, "src must be 16-byte aligned and bytes a multiple of 16 (bytes = %zu)", bytes);
  if (!aligned(sink, 4)) return fail(DREAMS_ERR_INVALID_ARG, "sink must be 4-byte aligned");
  if (bytes == 0) return ok();
  hipError_t e = launch_stream_read(src, bytes, sink, stream);
  if (e != hipSuccess) return hip_fail(e, "stream read launch");
  return ok();
}

static_assert(kVisualMaxTokens == DREAMS_VISUAL_MAX_TOKENS, "top-r capacity");

// visual importance workspace: the fixed counter region every workspace starts with (one arrival counter per
// (sequence, 256 tokens), on a cache line of its own where the region allows), then the per-KV-head partial
// sums.  The region's size does not depend on the shape, so a workspace left zero by any call serves any other.
size_t visual_workspace_bytes(int batch, int num_kv_heads, int vis_count) {
  return kCounterBytes + (size_t)batch * num_kv_heads * vis_count * sizeof(float);
}
int visual_counter_stride(int batch, int vis_count) {   // 0: the counters do not fit
  const long long n = (long long)batch * ((vis_count + 255) / 256);
  int stride = kCounterStride;
  while (stride > 1 && n * stride > (long long)kMaxCounters) stride >>= 1;
  return n * stride <= (long long)kMaxCounters ? stride : 0;
}

dreams_status_t dreams_visual_importance_workspace_size(int32_t batch, int32_t num_kv_heads, int32_t vis_count,
                                                        size_t* bytes) {
  if (!bytes) return fail(DREAMS_ERR_INVALID_ARG, "bytes is NULL");
  if (batch < 0 || num_kv_heads < 1 || vis_count < 1)
    return fail(DREAMS_ERR_INVALID_ARG, "batch = %d, num_kv_heads = %d, vis_count = %d", batch, num_kv_heads,
                vis_count);
  *bytes = visual_workspace_bytes(batch, num_kv_heads, vis_count);
  return ok();
}

dreams_status_t dreams_visual_importance(const dreams_attn_desc_t* desc, const void* q, const void* k_cache,
                                         const int32_t* kv_len, const float* lse, int32_t vis_begin,
                                         int32_t vis_count, float* importance, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream) {
  dreams_status_t st = check_attn_desc(desc);
  if (st != DREAMS_OK) return st;
  if (desc->dtype != DREAMS_BF16) return fail(DREAMS_ERR_UNSUPPORTED, "visual importance takes bf16 q and k_cache");
  if (vis_begin < 0 || vis_count < 1 || (long long)vis_begin + vis_count > desc->cache_capacity)
    return fail(DREAMS_ERR_INVALID_ARG, "visual tokens [%d, %d + %d) are not inside the cache (capacity %d)",
                vis_begin, vis_begin, vis_count, desc->cache_capacity);
  const size_t need = visual_workspace_bytes(desc->batch, desc->num_kv_heads, vis_count);
  if (desc->batch == 0) return ok();
  if (!q || !k_cache || !kv_len || !lse || !importance)
    return fail(DREAMS_ERR_INVALID_ARG, "q, k_cache, kv_len, lse and importance must not be NULL");
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(kv_len, 4) || !aligned(lse, 4) || !aligned(importance, 4))
    return fail(DREAMS_ERR_INVALID_ARG, "q and k_cache must be 16-byte aligned, kv_len, lse and importance 4-byte");
  if (!workspace) return fail(DREAMS_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
  if (workspace_bytes < need)
    return fail(DREAMS_ERR_WORKSPACE, "workspace has %zu bytes, %zu are needed", workspace_bytes, need);
  if (!aligned(workspace, 256)) return fail(DREAMS_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if ((long long)desc->batch * desc->num_kv_heads * ((vis_count + 63) / 64) > 0x7fffffffLL)
    return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");
  const int stride = visual_counter_stride(desc->batch, vis_count);
  if (stride == 0)
    return fail(DREAMS_ERR_UNSUPPORTED, "batch * ceil(vis_count / 256) = %lld exceeds %zu arrival counters",
                (long long)desc->batch * ((vis_count + 255) / 256), kMaxCounters);
  VisualArgs a{};
  a.q = q;
  a.k = k_cache;
  a.kv_len = kv_len;
  a.lse = lse;
  a.counters = (uint32_t*)workspace;
  a.counter_stride = stride;
  a.partial = (float*)((char*)workspace + kCounterBytes);
  a.importance = importance;
  a.B = desc->batch;
  a.Hq = desc->num_q_heads;
  a.Hkv = desc->num_kv_heads;
  a.G = desc->num_q_heads / desc->num_kv_heads;
  a.T = desc->num_nodes;
  a.D = desc->head_dim;
  a.S_cap = desc->cache_capacity;
  a.vis_begin = vis_begin;
  a.vis_count = vis_count;
  a.scale_log2 = desc->scale * 1.4426950408889634f;
  hipError_t e = launch_visual_importance(a, stream);
  if (e != hipSuccess) return hip_fail(e, "visual importance launch");
  return ok();
}

// ------------------------------------------------------------------------------ prefill attention statistics
namespace {
dreams_status_t check_prefill_desc(const dreams_prefill_desc_t* d) {
  if (!d) return fail(DREAMS_ERR_INVALID_ARG, "desc is NULL");
  if (d->batch < 0) return fail(DREAMS_ERR_INVALID_ARG, "batch = %d < 0", d->batch);
  if (d->num_q_heads < 1 || d->num_kv_heads < 1 || d->num_q_heads % d->num_kv_heads != 0)
    return fail(DREAMS_ERR_INVALID_ARG, "num_q_heads = %d must be a positive multiple of num_kv_heads = %d",
                d->num_q_heads, d->num_kv_heads);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(DREAMS_ERR_UNSUPPORTED, "head_dim = %d (supported: 64, 128)", d->head_dim);
  if (d->num_rows < 1 || d->cache_capacity < d->num_rows)
    return fail(DREAMS_ERR_INVALID_ARG, "num_rows = %d must be in [1, cache_capacity = %d]", d->num_rows,
                d->cache_capacity);
  if (!isfinite(d->scale)) return fail(DREAMS_ERR_INVALID_ARG, "scale is not finite");
  if ((long long)d->batch * d->num_q_heads * ((d->num_rows + 255) / 256) > 0x7fffffffLL)
    return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");
  return DREAMS_OK;
}
}  // namespace

dreams_status_t dreams_prefill_attn_stats(const dreams_prefill_desc_t* desc, const void* q, const void* k_cache,
                                          const int32_t* prompt_len, float* lse, float* entropy, hipStream_t stream) {
  dreams_status_t st = check_prefill_desc(desc);
  if (st != DREAMS_OK) return st;
  if (desc->batch == 0 || (!lse && !entropy)) return ok();
  if (!q || !k_cache || !prompt_len) return fail(DREAMS_ERR_INVALID_ARG, "q, k_cache and prompt_len must not be NULL");
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(prompt_len, 4) || !aligned(lse, 4) || !aligned(entropy, 4))
    return fail(DREAMS_ERR_INVALID_ARG, "q and k_cache must be 16-byte aligned, prompt_len, lse and entropy 4-byte");
  PrefillArgs a{};
  a.q = q;
  a.k = k_cache;
  a.prompt_len = prompt_len;
  a.lse = lse;
  a.entropy = entropy;
  a.B = desc->batch;
  a.Hq = desc->num_q_heads;
  a.Hkv = desc->num_kv_heads;
  a.G = desc->num_q_heads / desc->num_kv_heads;
  a.N = desc->num_rows;
  a.D = desc->head_dim;
  a.S_cap = desc->cache_capacity;
  a.scale_log2 = desc->scale * 1.4426950408889634f;
  st = device_cus(&a.cus);
  if (st != DREAMS_OK) return st;
  hipError_t e = launch_prefill_stats(a, stream);
  if (e != hipSuccess) return hip_fail(e, "prefill statistics launch");
  return ok();
}

dreams_status_t dreams_prefill_attn_entropy_mean(int32_t batch, int32_t num_q_heads, int32_t num_rows,
                                                 const float* entropy, const int32_t* prompt_len, float* ae,
                                                 hipStream_t stream) {
  if (batch < 1 || num_q_heads < 1 || num_rows < 1)
    return fail(DREAMS_ERR_INVALID_ARG, "batch = %d, num_q_heads = %d and num_rows = %d must be >= 1", batch,
                num_q_heads, num_rows);
  if (!entropy || !prompt_len || !ae) return fail(DREAMS_ERR_INVALID_ARG, "entropy, prompt_len and ae must not be NULL");
  if (!aligned(entropy, 4) || !aligned(prompt_len, 4) || !aligned(ae, 4))
    return fail(DREAMS_ERR_INVALID_ARG, "entropy, prompt_len or ae is misaligned");
  hipError_t e = launch_prefill_entropy_mean(batch, num_q_heads, num_rows, entropy, prompt_len, ae, stream);
  if (e != hipSuccess) return hip_fail(e, "prefill entropy mean launch");
  return ok();
}

dreams_status_t dreams_prefill_visual_importance(const dreams_prefill_desc_t* desc, const void* q, const void* k_cache,
                                                 const int32_t* prompt_len, const float* lse, int32_t vis_begin,
                                                 int32_t vis_count, float* importance, void* workspace,
                                                 size_t workspace_bytes, hipStream_t stream) {
  dreams_status_t st = check_prefill_desc(desc);
  if (st != DREAMS_OK) return st;
  if (vis_begin < 0 || vis_count < 1 || (long long)vis_begin + vis_count > desc->num_rows)
    return fail(DREAMS_ERR_INVALID_ARG, "visual tokens [%d, %d + %d) are not inside the prompt (%d rows)", vis_begin,
                vis_begin, vis_count, desc->num_rows);
  const size_t need = visual_workspace_bytes(desc->batch, desc->num_kv_heads, vis_count);
  if (desc->batch == 0) return ok();
  if (!q || !k_cache || !prompt_len || !lse || !importance)
    return fail(DREAMS_ERR_INVALID_ARG, "q, k_cache, prompt_len, lse and importance must not be NULL");
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(prompt_len, 4) || !aligned(lse, 4) || !aligned(importance, 4))
    return fail(DREAMS_ERR_INVALID_ARG, "q and k_cache must be 16-byte aligned, prompt_len, lse and importance 4-byte");
  if (!workspace) return fail(DREAMS_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
  if (workspace_bytes < need)
    return fail(DREAMS_ERR_WORKSPACE, "workspace has %zu bytes, %zu are needed", workspace_bytes, need);
  if (!aligned(workspace, 256)) return fail(DREAMS_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if ((long long)desc->batch * desc->num_kv_heads * ((vis_count + 63) / 64) > 0x7fffffffLL)
    return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");
  const int stride = visual_counter_stride(desc->batch, vis_count);
  if (stride == 0)
    return fail(DREAMS_ERR_UNSUPPORTED, "batch * ceil(vis_count / 256) = %lld exceeds %zu arrival counters",
                (long long)desc->batch * ((vis_count + 255) / 256), kMaxCounters);
  VisualArgs a{};
  a.q = q;
  a.k = k_cache;
  a.kv_len = prompt_len;
  a.lse = lse;
  a.prefill = 1;
  st = device_cus(&a.cus);
  if (st != DREAMS_OK) return st;
  a.counters = (uint32_t*)workspace;
  a.counter_stride = stride;
  a.partial = (float*)((char*)workspace + kCounterBytes);
  a.importance = importance;
  a.B = desc->batch;
  a.Hq = desc->num_q_heads;
  a.Hkv = desc->num_kv_heads;
  a.G = desc->num_q_heads / desc->num_kv_heads;
  a.T = desc->num_rows;
  a.D = desc->head_dim;
  a.S_cap = desc->cache_capacity;
  a.vis_begin = vis_begin;
  a.vis_count = vis_count;
  a.scale_log2 = desc->scale * 1.4426950408889634f;
  hipError_t e = launch_visual_importance(a, stream);
  if (e != hipSuccess) return hip_fail(e, "prefill visual importance launch");
  return ok();
}

dreams_status_t dreams_visual_topk(int32_t batch, int32_t vis_count, int32_t keep_count, const float* importance,
                                   int32_t* keep, hipStream_t stream) {
  if (batch < 0) return fail(DREAMS_ERR_INVALID_ARG, "batch = %d < 0", batch);
  if (vis_count < 1 || vis_count > kVisualMaxTokens)
    return fail(DREAMS_ERR_UNSUPPORTED, "vis_count = %d outside [1, %d]", vis_count, kVisualMaxTokens);
  if (keep_count < 1 || keep_count > vis_count)
    return fail(DREAMS_ERR_INVALID_ARG, "keep_count = %d outside [1, vis_count = %d]", keep_count, vis_count);
  if (batch == 0) return ok();
  if (!importance || !keep) return fail(DREAMS_ERR_INVALID_ARG, "importance and keep must not be NULL");
  if (!aligned(importance, 4) || !aligned(keep, 4))
    return fail(DREAMS_ERR_INVALID_ARG, "importance and keep must be 4-byte aligned");
  hipError_t e = launch_visual_topk(batch, vis_count, keep_count, importance, keep, stream);
  if (e != hipSuccess) return hip_fail(e, "visual top-r launch");
  return ok();
}

dreams_status_t dreams_visual_gather(int32_t batch, int32_t num_kv_heads, int32_t head_dim, int32_t cache_capacity,
                                     dreams_dtype_t dtype, const void* k_cache, const void* v_cache,
                                     int32_t vis_begin, const int32_t* keep, int32_t keep_count, void* k_out,
                                     void* v_out, hipStream_t stream) {
  if (batch < 0 || num_kv_heads < 1 || head_dim < 1 || cache_capacity < 1 || keep_count < 1 || vis_begin < 0)
    return fail(DREAMS_ERR_INVALID_ARG, "batch >= 0, num_kv_heads, head_dim, cache_capacity, keep_count >= 1 and "
                                        "vis_begin >= 0 are required");
  if (dtype != DREAMS_BF16 && dtype != DREAMS_F32)
    return fail(DREAMS_ERR_INVALID_ARG, "dtype = %d is not DREAMS_BF16 or DREAMS_F32", (int)dtype);
  const long long row_bytes = (long long)head_dim * (dtype == DREAMS_BF16 ? 2 : 4);
  if (row_bytes % 16 != 0 || row_bytes > (1 << 20))
    return fail(DREAMS_ERR_UNSUPPORTED, "head_dim * element size = %lld bytes (must be a multiple of 16)", row_bytes);
  if (batch == 0) return ok();
  if (!k_cache || !v_cache || !keep || !k_out || !v_out)
    return fail(DREAMS_ERR_INVALID_ARG, "cache, keep and output pointers must not be NULL");
  if (!aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(k_out, 16) || !aligned(v_out, 16) ||
      !aligned(keep, 4))
    return fail(DREAMS_ERR_INVALID_ARG, "caches and outputs must be 16-byte aligned, keep 4-byte");
  if ((long long)batch * num_kv_heads > 0x7fffffffLL || (long long)keep_count * (row_bytes / 16) / 256 > 65535)
    return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");
  VisualGatherArgs a{};
  a.k = k_cache;
  a.v = v_cache;
  a.keep = keep;
  a.k_out = k_out;
  a.v_out = v_out;
  a.B = batch;
  a.Hkv = num_kv_heads;
  a.S_cap = cache_capacity;
  a.r = keep_count;
  a.vis_begin = vis_begin;
  a.row_bytes = (int)row_bytes;
  hipError_t e = launch_visual_gather(a, stream);
  if (e != hipSuccess) return hip_fail(e, "visual gather launch");
  return ok();
}

dreams_status_t dreams_kv_commit(int32_t num_layers, int64_t layer_stride_elems, int32_t batch,
                                 int32_t num_kv_heads, int32_t head_dim, int32_t cache_capacity,
                                 dreams_dtype_t dtype, void* k_cache, void* v_cache, const int32_t* kv_len_in,
                                 const int32_t* accept_path, const int32_t* accept_len, int32_t path_stride,
                                 int32_t* kv_len_out, hipStream_t stream) {
  if (num_layers < 1) return fail(DREAMS_ERR_INVALID_ARG, "num_layers = %d < 1", num_layers);
  if (batch < 0) return fail(DREAMS_ERR_INVALID_ARG, "batch = %d < 0", batch);
  if (num_kv_heads < 1 || head_dim < 1 || cache_capacity < 1 || path_stride < 1)
    return fail(DREAMS_ERR_INVALID_ARG, "num_kv_heads, head_dim, cache_capacity and path_stride must be >= 1");
  if (dtype != DREAMS_BF16 && dtype != DREAMS_F32)
    return fail(DREAMS_ERR_INVALID_ARG, "dtype = %d is not DREAMS_BF16 or DREAMS_F32", (int)dtype);
  const int elem = dtype == DREAMS_BF16 ? 2 : 4;
  const long long row_bytes = (long long)head_dim * elem;
  if (row_bytes % 16 != 0 || row_bytes > kCommitMaxRowBytes)
    return fail(DREAMS_ERR_UNSUPPORTED, "head_dim * element size = %lld bytes (must be a multiple of 16, <= %d)",
                row_bytes, kCommitMaxRowBytes);
  const long long layer_elems = (long long)batch * num_kv_heads * cache_capacity * head_dim;
  if (num_layers > 1 && layer_stride_elems < layer_elems)
    return fail(DREAMS_ERR_INVALID_ARG, "layer_stride_elems = %lld is smaller than one layer (%lld elements)",
                (long long)layer_stride_elems, layer_elems);
  if (layer_stride_elems < 0) return fail(DREAMS_ERR_INVALID_ARG, "layer_stride_elems < 0");
  if (batch == 0) return ok();
  if (!k_cache || !v_cache || !kv_len_in || !accept_path || !accept_len || !kv_len_out)
    return fail(DREAMS_ERR_INVALID_ARG, "cache, length and path pointers must not be NULL");
  if (!aligned(k_cache, 16) || !aligned(v_cache, 16) || ((layer_stride_elems * elem) % 16) != 0)
    return fail(DREAMS_ERR_INVALID_ARG, "k_cache, v_cache and the layer stride must be 16-byte aligned");
  if (!aligned(kv_len_in, 4) || !aligned(accept_path, 4) || !aligned(accept_len, 4) || !aligned(kv_len_out, 4))
    return fail(DREAMS_ERR_INVALID_ARG, "an int32 argument is not 4-byte aligned");
  if (overlap(kv_len_out, (size_t)batch * 4, kv_len_in, (size_t)batch * 4))
    return fail(DREAMS_ERR_INVALID_ARG, "kv_len_out must not overlap kv_len_in");
  if ((long long)num_layers * batch * num_kv_heads > 0x7fffffffLL)
    return fail(DREAMS_ERR_UNSUPPORTED, "problem too large");

  CommitArgs a{};
  a.k = (char*)k_cache;
  a.v = (char*)v_cache;
  a.kv_len_in = kv_len_in;
  a.path = accept_path;
  a.accept_len = accept_len;
  a.kv_len_out = kv_len_out;
  a.layer_stride_bytes = layer_stride_elems * elem;
  a.NL = num_layers;
  a.B = batch;
  a.Hkv = num_kv_heads;
  a.S_cap = cache_capacity;
  a.path_stride = path_stride;
  a.row_bytes = (int)row_bytes;
  hipError_t e = launch_kv_commit(a, stream);
  if (e != hipSuccess) return hip_fail(e, "kv commit launch");
  return ok();
}

const char* dreams_status_string(dreams_status_t status) {
  switch (status) {
    case DREAMS_OK: return "DREAMS_OK";
    case DREAMS_ERR_INVALID_ARG: return "DREAMS_ERR_INVALID_ARG: an argument is out of range or NULL";
    case DREAMS_ERR_UNSUPPORTED: return "DREAMS_ERR_UNSUPPORTED: shape or type not supported by this build";
    case DREAMS_ERR_WORKSPACE: return "DREAMS_ERR_WORKSPACE: workspace missing or too small";
    case DREAMS_ERR_HIP: return "DREAMS_ERR_HIP: the HIP runtime reported an error";
    case DREAMS_ERR_DEVICE: return "DREAMS_ERR_DEVICE: a kernel flagged a failure in the workspace";
  }
  return "unknown dreams status";
}

const char* dreams_last_error_message(void) { return g_error.c_str(); }

dreams_status_t dreams_workspace_status(void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!workspace) return fail(DREAMS_ERR_INVALID_ARG, "workspace is NULL");
  if (!aligned(workspace, 256)) return fail(DREAMS_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < kCounterBytes)
    return fail(DREAMS_ERR_WORKSPACE, "workspace has %zu bytes, less than its %zu-byte counter region", workspace_bytes,
                kCounterBytes);
  uint32_t* word = (uint32_t*)workspace + kErrorWord;
  uint32_t flags = 0;
  hipError_t e = hipMemcpyAsync(&flags, word, sizeof(flags), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "reading the workspace's failure flags");
  if (flags == 0) return ok();
  e = hipMemsetAsync(word, 0, sizeof(flags), stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "clearing the workspace's failure flags");
  std::string what;
  if (flags & kErrXcdSplit) what += " [attention: pieces of one row set ran on different XCDs; outputs NaN]";
  if (flags & kErrWaitTimeout)
    what += " [a bounded wait for another workgroup gave up (attention merge or sampled acceptance); results "
            "unspecified]";
  if (flags & ~(kErrXcdSplit | kErrWaitTimeout)) what += " [unknown flag]";
  return fail(DREAMS_ERR_DEVICE, "failure flags 0x%x:%s", flags, what.c_str());
}

dreams_status_t dreams_set_wait_limit(double seconds) {
  if (!(seconds >= 0.0) || seconds > 60.0)
    return fail(DREAMS_ERR_INVALID_ARG, "wait limit %g s is outside [0, 60]", seconds);
  g_wait_ticks.store((uint64_t)(seconds * 1e8), std::memory_order_relaxed);
  return ok();
}

dreams_status_t dreams_tree_verify_attn_splits(const dreams_attn_desc_t* desc, int32_t* splits) {
  if (!splits) return fail(DREAMS_ERR_INVALID_ARG, "splits is NULL");
  AttnPlan p;
  dreams_status_t st = plan_attn(desc, &p);
  if (st != DREAMS_OK) return st;
  *splits = p.splits;
  return ok();
}

dreams_status_t dreams_check_tree_host(const int32_t* parent, int32_t num_nodes) {
  if (!parent) return fail(DREAMS_ERR_INVALID_ARG, "parent is NULL");
  if (num_nodes < 1) return fail(DREAMS_ERR_INVALID_ARG, "num_nodes = %d < 1", num_nodes);
  if (parent[0] != -1) return fail(DREAMS_ERR_INVALID_ARG, "parent[0] = %d, the root must have parent -1", parent[0]);
  for (int i = 1; i < num_nodes; ++i)
    if (parent[i] < 0 || parent[i] >= i)
      return fail(DREAMS_ERR_INVALID_ARG, "parent[%d] = %d is not in [0, %d)", i, parent[i], i);
  return ok();
}

}  // extern "C"

// C ABI of the library: argument validation on the host, then kernel launches
// on the caller's stream.  Nothing here allocates device memory or synchronizes.
#include <cstring>
#include <mutex>

#include "hack_internal.hpp"

// Split-K workspace of hack_attend_decode_noalloc: one copy per GPU, held until the
// process ends.  Layout as a caller's workspace (hack::DecodePlan): chunk counters
// from offset 0 (at most kScratchCounters of them), chunk records from
// kScratchCounterBytes (at most kScratchRecordBytes).  Static storage is zero-filled
// when the code object is loaded, so the counters start at zero; every call leaves
// them zero.  In host code `scratch` is only a handle for hipGetSymbolAddress: its
// device address is looked up per device and kept in g_scratch_ptr.
namespace {
constexpr int64_t kScratchCounters = 65536;
constexpr int64_t kScratchCounterBytes = kScratchCounters * 4;
constexpr int64_t kScratchRecordBytes = 16ll << 20;
constexpr int64_t kScratchBytes = kScratchCounterBytes + kScratchRecordBytes;
}  // namespace
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

using hack::CacheView;

namespace {

constexpr int kMaxGridYZ = 65535;  // largest y or z extent of a launch grid

// Bytes of one cached code sum: b + ceil(log2 pi) bits rounded up to 1 or 2 bytes.
int sum_width(int bits, int pi) {
  int need = bits;
  for (int v = 1; v < pi && v > 0; v <<= 1) ++need;
  return need <= 8 ? 1 : 2;
}

bool layout_ok(const hack_kv_layout* l) {
  if (!l) return false;
  const int pi = l->partition;
  if (!(pi == 16 || pi == 32 || pi == 64 || pi == 128)) return false;
  if (l->head_dim <= 0 || l->head_dim > 256 || l->head_dim % pi != 0) return false;
  if (l->num_kv_heads < 1) return false;
  if (!(l->kv_bits == 2 || l->kv_bits == 4)) return false;
  if (l->page_tokens <= 0 || l->page_tokens % pi != 0) return false;
  if (!(l->qp_bits == 8 || l->qp_bits == 4)) return false;
  if (!(l->rounding == HACK_ROUND_NEAREST_EVEN || l->rounding == HACK_ROUND_STOCHASTIC)) return false;
  return l->sum_bytes == 0 || l->sum_bytes == sum_width(l->kv_bits, pi);
}

// Validates the cache pointers for `batch` sequences; returns the per-sequence capacity or -1.
int64_t cache_capacity(const hack_kv_layout* l, const hack_kv_cache* c, int batch) {
  if (!c) return -1;
  if (!c->k_codes || !c->k_meta || !c->v_codes || !c->v_meta || !c->v_tail) return -1;
  if (l->sum_bytes != 0 && (!c->k_sums || !c->v_sums)) return -1;
  if (c->num_pages <= 0) return -1;
  if (c->block_table_dev) {
    if (c->max_blocks_per_seq <= 0) return -1;
    return (int64_t)c->max_blocks_per_seq * l->page_tokens;
  }
  if (c->num_pages < batch) return -1;
  return l->page_tokens;
}

CacheView make_view(const hack_kv_layout* l, const hack_kv_cache* c) {
  CacheView v;
  v.k_codes = static_cast<uint8_t*>(c->k_codes);
  v.k_meta = static_cast<__half2*>(c->k_meta);
  v.k_sums = static_cast<uint8_t*>(c->k_sums);
  v.v_codes = static_cast<uint8_t*>(c->v_codes);
  v.v_meta = static_cast<__half2*>(c->v_meta);
  v.v_sums = static_cast<uint8_t*>(c->v_sums);
  v.v_tail = static_cast<__half*>(c->v_tail);
  v.block_table = c->block_table_dev;
  v.mbps = c->max_blocks_per_seq;
  v.num_pages = c->num_pages;
  v.page_tokens = l->page_tokens;
  v.kv_heads = l->num_kv_heads;
  v.head_dim = l->head_dim;
  v.sum_bytes = l->sum_bytes;
  return v;
}

hack_status from_hip(hipError_t e) { return e == hipSuccess ? HACK_OK : HACK_ERR_HIP; }

// Shapes the attention kernels implement.
hack_status attention_shape(const hack_kv_layout* l, int num_q_heads) {
  if (num_q_heads < 1 || num_q_heads % l->num_kv_heads != 0) return HACK_ERR_INVALID_ARGUMENT;
  if (l->head_dim != 128) return HACK_ERR_UNSUPPORTED;
  if (!(l->partition == 32 || l->partition == 64 || l->partition == 128)) return HACK_ERR_UNSUPPORTED;
  if (num_q_heads / l->num_kv_heads > 8) return HACK_ERR_UNSUPPORTED;
  return HACK_OK;
}

// Decode attention: partitions of 32 and 64 run the matrix-core kernel, 128 its own
// (with its own chunking of the sequences).
hack::DecodePlan plan_attend(const hack_kv_layout& l, int batch, int num_q_heads, int max_len) {
  return l.partition == 128 ? hack::plan_decode128(l, batch, num_q_heads, max_len)
                            : hack::plan_decode(l, batch, num_q_heads, max_len);
}

// Points the split-K fields of `a` at a workspace laid out as `plan` describes:
// chunk counters at offset 0, chunk records after them.
void bind_workspace(hack::DecodeArgs& a, const hack::DecodePlan& plan, void* ws) {
  a.counters = static_cast<int32_t*>(ws);
  a.partials = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + plan.record_offset);
  a.chunk = plan.chunk;
  a.splits = plan.splits;
}

hipError_t launch_attend(const hack_kv_layout& l, const hack::DecodeArgs& a, int batch, hipStream_t stream) {
  if (l.partition == 128) return hack::launch_decode128(l, a, batch, stream);
  return hack::launch_decode(l, a, batch, hack::MODE_ATTEND, stream);
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device; guarded by g_scratch_mu

__global__ void zero_words_kernel(int32_t* p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// Device address of the current device's `scratch`.  The first call on a device looks
// it up and clears its counters with a kernel on `stream` (a kernel rather than a
// memset, so that a caller may capture it in a graph).  Returns nullptr on failure.
void* scratch_for_current_device(hipStream_t stream) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
    hipLaunchKernelGGL(zero_words_kernel, dim3(64), dim3(256), 0, stream, static_cast<int32_t*>(p),
                       kScratchCounters);
    if (hipGetLastError() != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

hack_status hack_kv_layout_make(hack_kv_layout* out, int32_t head_dim, int32_t num_kv_heads,
                                int32_t kv_bits, int32_t partition, int32_t page_tokens,
                                int32_t qp_bits, int32_t rounding, uint64_t seed) {
  if (!out) return HACK_ERR_INVALID_ARGUMENT;
  hack_kv_layout l;
  std::memset(&l, 0, sizeof(l));
  l.head_dim = head_dim;
  l.num_kv_heads = num_kv_heads;
  l.kv_bits = kv_bits;
  l.partition = partition;
  l.page_tokens = page_tokens;
  l.qp_bits = qp_bits;
  l.rounding = rounding;
  l.seed = seed;
  l.sum_bytes = sum_width(kv_bits, partition);
  if (!layout_ok(&l)) return HACK_ERR_INVALID_ARGUMENT;
  *out = l;
  return HACK_OK;
}

hack_status hack_kv_layout_set_sums(hack_kv_layout* layout, int32_t cached) {
  if (!layout_ok(layout) || !(cached == 0 || cached == 1)) return HACK_ERR_INVALID_ARGUMENT;
  layout->sum_bytes = cached ? sum_width(layout->kv_bits, layout->partition) : 0;
  return HACK_OK;
}

int64_t hack_kv_bytes(const hack_kv_layout* l, int64_t count, int32_t section) {
  if (!layout_ok(l) || count < 0) return -1;
  const int64_t d = l->head_dim, H = l->num_kv_heads, pt = l->page_tokens, pi = l->partition;
  const int64_t P = d / pi;
  switch (section) {
    case HACK_K_CODES: return count * H * pt * (d * l->kv_bits / 8);
    case HACK_K_META: return count * H * pt * P * 4;
    case HACK_K_SUMS: return count * H * pt * P * l->sum_bytes;
    case HACK_V_CODES: return count * H * (pt / pi) * d * (pi * l->kv_bits / 8);
    case HACK_V_META: return count * H * (pt / pi) * d * 4;
    case HACK_V_SUMS: return count * H * (pt / pi) * d * l->sum_bytes;
    case HACK_V_TAIL: return count * H * pi * d * 2;
    default: return -1;
  }
}

hack_status hack_quantize(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* k_dev,
                          const void* v_dev, const int32_t* seq_lens_dev, int32_t batch, int32_t max_len,
                          hipStream_t stream) {
  if (!layout_ok(layout) || !k_dev || !v_dev || !seq_lens_dev || batch < 0 || max_len < 0)
    return HACK_ERR_INVALID_ARGUMENT;
  const int64_t cap = cache_capacity(layout, cache, batch);
  if (cap < 0) return HACK_ERR_INVALID_ARGUMENT;
  if (max_len > cap) return HACK_ERR_CAPACITY;
  if (batch == 0 || max_len == 0) return HACK_OK;
  // V blocks are one workgroup (partitions >= 64) or a fixed group of threads each: the
  // grid must fit its 2^31 - 1 limit
  if ((int64_t)batch * layout->num_kv_heads * ((max_len + layout->partition - 1) / layout->partition) > INT32_MAX)
    return HACK_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  return from_hip(hack::launch_quantize(*layout, make_view(layout, cache), static_cast<const __half*>(k_dev),
                                        static_cast<const __half*>(v_dev), seq_lens_dev, batch, max_len, stream));
}

hack_status hack_append(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* k_new_dev,
                        const void* v_new_dev, int32_t* seq_lens_dev, int32_t batch, int32_t max_len,
                        int32_t tail_mode, hipStream_t stream) {
  if (!layout_ok(layout) || !k_new_dev || !v_new_dev || !seq_lens_dev || batch < 0 || max_len < 0)
    return HACK_ERR_INVALID_ARGUMENT;
  if (!(tail_mode == HACK_TAIL_FP16 || tail_mode == HACK_TAIL_REQUANT || tail_mode == HACK_TAIL_DEQUANT)) return HACK_ERR_INVALID_ARGUMENT;
  const int64_t cap = cache_capacity(layout, cache, batch);
  if (cap < 0) return HACK_ERR_INVALID_ARGUMENT;
  if ((int64_t)max_len + 1 > cap) return HACK_ERR_CAPACITY;
  if (layout->num_kv_heads * layout->head_dim > 2048) return HACK_ERR_UNSUPPORTED;  // one workgroup per sequence
  if (batch == 0) return HACK_OK;
  (void)hipGetLastError();
  return from_hip(hack::launch_append(*layout, make_view(layout, cache), static_cast<const __half*>(k_new_dev),
                                      static_cast<const __half*>(v_new_dev), seq_lens_dev, batch, (int)cap,
                                      tail_mode, stream));
}

int64_t hack_decode_workspace_bytes(const hack_kv_layout* layout, int32_t batch, int32_t num_q_heads,
                                    int32_t max_len) {
  if (!layout_ok(layout) || batch < 0 || max_len < 0 || num_q_heads < 1 ||
      num_q_heads % layout->num_kv_heads != 0)
    return -1;
  return plan_attend(*layout, batch, num_q_heads, max_len).workspace_bytes;
}

static hack_status decode_common(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* q_dev,
                                 int32_t num_q_heads, const int32_t* seq_lens_dev, int32_t batch,
                                 int32_t max_len, hack::DecodeArgs& a, int64_t* cap_out) {
  if (!layout_ok(layout) || !q_dev || !seq_lens_dev || batch < 0 || max_len < 0)
    return HACK_ERR_INVALID_ARGUMENT;
  const hack_status sh = attention_shape(layout, num_q_heads);
  if (sh != HACK_OK) return sh;
  if (batch > kMaxGridYZ) return HACK_ERR_UNSUPPORTED;  // one grid row per sequence
  const int64_t cap = cache_capacity(layout, cache, batch);
  if (cap < 0) return HACK_ERR_INVALID_ARGUMENT;
  if (max_len > cap) return HACK_ERR_CAPACITY;
  // a decode span (four V blocks) must not cross a page
  if (cache->block_table_dev && layout->page_tokens % (4 * layout->partition) != 0) return HACK_ERR_UNSUPPORTED;
  std::memset(&a, 0, sizeof(a));
  a.c = make_view(layout, cache);
  a.q = static_cast<const __half*>(q_dev);
  a.lens = seq_lens_dev;
  a.num_q_heads = num_q_heads;
  a.group = num_q_heads / layout->num_kv_heads;
  a.max_len = max_len;
  a.qmax = (float)((1 << layout->qp_bits) - 1);
  a.inv_qmax = 1.0f / a.qmax;
  a.qoff = 1 << (layout->qp_bits - 1);
  a.qoff_f = (float)a.qoff;
  a.stochastic = layout->rounding == HACK_ROUND_STOCHASTIC;
  a.key_q = layout->seed ^ (3ull << 56);
  a.key_p = layout->seed ^ (4ull << 56);
  *cap_out = cap;
  return HACK_OK;
}

hack_status hack_attend_decode(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* q_dev,
                               int32_t num_q_heads, const int32_t* seq_lens_dev, int32_t batch, int32_t max_len,
                               int32_t tail_mode, float* out_dev, void* workspace_dev, int64_t workspace_bytes,
                               hipStream_t stream) {
  hack::DecodeArgs a;
  int64_t cap = 0;
  hack_status st = decode_common(layout, cache, q_dev, num_q_heads, seq_lens_dev, batch, max_len, a, &cap);
  if (st != HACK_OK) return st;
  if (!out_dev || !(tail_mode == HACK_TAIL_FP16 || tail_mode == HACK_TAIL_REQUANT || tail_mode == HACK_TAIL_DEQUANT))
    return HACK_ERR_INVALID_ARGUMENT;
  const hack::DecodePlan plan = plan_attend(*layout, batch, num_q_heads, max_len);
  if (!workspace_dev || workspace_bytes < plan.workspace_bytes) return HACK_ERR_WORKSPACE;
  if (batch == 0) return HACK_OK;
  a.out = out_dev;
  bind_workspace(a, plan, workspace_dev);
  a.tail_requant = tail_mode;  // 0: fp16 open block; 1, 2: its codes (re-quantized on append)
  (void)hipGetLastError();
  return from_hip(launch_attend(*layout, a, batch, stream));
}

hack_status hack_attend_decode_noalloc(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* q_dev,
                                       int32_t num_q_heads, const int32_t* seq_lens_dev, int32_t batch,
                                       int32_t max_len, int32_t tail_mode, float* out_dev, hipStream_t stream) {
  hack::DecodeArgs a;
  int64_t cap = 0;
  hack_status st = decode_common(layout, cache, q_dev, num_q_heads, seq_lens_dev, batch, max_len, a, &cap);
  if (st != HACK_OK) return st;
  if (!out_dev || !(tail_mode == HACK_TAIL_FP16 || tail_mode == HACK_TAIL_REQUANT || tail_mode == HACK_TAIL_DEQUANT))
    return HACK_ERR_INVALID_ARGUMENT;
  const hack::DecodePlan plan = plan_attend(*layout, batch, num_q_heads, max_len);
  if (plan.counter_bytes > kScratchCounterBytes || plan.workspace_bytes - plan.record_offset > kScratchRecordBytes)
    return HACK_ERR_WORKSPACE;
  if (batch == 0) return HACK_OK;
  (void)hipGetLastError();
  uint8_t* ws = static_cast<uint8_t*>(scratch_for_current_device(stream));
  if (!ws) return HACK_ERR_HIP;
  a.out = out_dev;
  a.counters = reinterpret_cast<int32_t*>(ws);
  a.partials = reinterpret_cast<float*>(ws + kScratchCounterBytes);
  a.chunk = plan.chunk;
  a.splits = plan.splits;
  a.tail_requant = tail_mode;
  return from_hip(launch_attend(*layout, a, batch, stream));
}

hack_status hack_decode_step(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* k_new_dev,
                             const void* v_new_dev, const void* q_dev, int32_t num_q_heads,
                             const int32_t* seq_lens_in_dev, int32_t* seq_lens_out_dev, int32_t batch,
                             int32_t max_len, int32_t tail_mode, float* out_dev, void* workspace_dev,
                             int64_t workspace_bytes, hipStream_t stream) {
  hack::DecodeArgs a;
  int64_t cap = 0;
  if (max_len < 0 || max_len == INT32_MAX) return HACK_ERR_INVALID_ARGUMENT;
  // validated as a decode over max_len + 1 tokens
  hack_status st = decode_common(layout, cache, q_dev, num_q_heads, seq_lens_in_dev, batch, max_len + 1, a, &cap);
  if (st != HACK_OK) return st;
  if (!k_new_dev || !v_new_dev || !seq_lens_out_dev || !out_dev || seq_lens_out_dev == seq_lens_in_dev ||
      !(tail_mode == HACK_TAIL_FP16 || tail_mode == HACK_TAIL_REQUANT || tail_mode == HACK_TAIL_DEQUANT))
    return HACK_ERR_INVALID_ARGUMENT;
  const hack::DecodePlan plan = plan_attend(*layout, batch, num_q_heads, max_len + 1);
  if (!workspace_dev || workspace_bytes < plan.workspace_bytes) return HACK_ERR_WORKSPACE;
  if (batch == 0) return HACK_OK;
  a.out = out_dev;
  bind_workspace(a, plan, workspace_dev);
  a.tail_requant = tail_mode;  // 0: fp16 open block; 1, 2: its codes (re-quantized on append)
  a.k_new = static_cast<const __half*>(k_new_dev);
  a.v_new = static_cast<const __half*>(v_new_dev);
  a.lens_out = seq_lens_out_dev;
  a.capacity = (int)cap;
  a.stochastic = layout->rounding == HACK_ROUND_STOCHASTIC;
  a.key_k = layout->seed ^ (1ull << 56);
  a.key_v = layout->seed ^ (2ull << 56);
  (void)hipGetLastError();
  // In the fused launch every workgroup whose chunk holds the new token appends it.
  // That is safe while those workgroups write identical bytes computed from the fp16
  // originals (FP16, REQUANT).  In DEQUANT mode the append reads the open block's codes
  // back and rewrites them, so when a kv group is split over several workgroups (more
  // than four query heads) one of them could requantize a block another has already
  // requantized.  That case, like partition 128 (whose attention kernel does not
  // append), runs the append as its own kernel first.
  const bool separate_append = layout->partition == 128 || (tail_mode == HACK_TAIL_DEQUANT && plan.head_groups > 1);
  if (separate_append) {
    // The new lengths start as a copy of the old ones, the append kernel writes the
    // token and bumps them, and the attention reads them (three operations on the
    // stream instead of one launch).
    if (layout->num_kv_heads * layout->head_dim > 2048) return HACK_ERR_UNSUPPORTED;  // one append workgroup
    hipError_t e = hipMemcpyAsync(seq_lens_out_dev, seq_lens_in_dev, (size_t)batch * sizeof(int32_t),
                                  hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess)
      e = hack::launch_append(*layout, a.c, a.k_new, a.v_new, seq_lens_out_dev, batch, (int)cap, tail_mode, stream);
    if (e != hipSuccess) return from_hip(e);
    a.lens = seq_lens_out_dev;
    a.k_new = nullptr;
    a.v_new = nullptr;
    a.lens_out = nullptr;
  }
  return from_hip(launch_attend(*layout, a, batch, stream));
}

hack_status hack_attend_prefill(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* q_dev,
                                int32_t num_q_heads, int32_t batch, int32_t len, int32_t causal, float* out_dev,
                                hipStream_t stream) {
  if (!layout_ok(layout) || !q_dev || !out_dev || batch < 0 || len < 0) return HACK_ERR_INVALID_ARGUMENT;
  const hack_status sh = attention_shape(layout, num_q_heads);
  if (sh != HACK_OK) return sh;
  if (layout->sum_bytes == 0) return HACK_ERR_UNSUPPORTED;  // prefill reads cached sums
  if (batch > kMaxGridYZ) return HACK_ERR_UNSUPPORTED;  // one grid plane per sequence
  const int64_t cap = cache_capacity(layout, cache, batch);
  if (cap < 0) return HACK_ERR_INVALID_ARGUMENT;
  if (len > cap) return HACK_ERR_CAPACITY;
  if (batch == 0 || len == 0) return HACK_OK;
  (void)hipGetLastError();
  return from_hip(hack::launch_prefill(*layout, make_view(layout, cache), static_cast<const __half*>(q_dev),
                                       num_q_heads, batch, len, causal != 0, out_dev, stream));
}

hack_status hack_project_qkv(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* e_dev,
                             const void* w_dev, int32_t num_q_heads, int32_t hidden, int32_t batch, int32_t len,
                             void* q_out_dev, hipStream_t stream) {
  if (!layout_ok(layout) || !e_dev || !w_dev || !q_out_dev || batch < 0 || len < 0 || hidden <= 0)
    return HACK_ERR_INVALID_ARGUMENT;
  if (num_q_heads < 1 || num_q_heads % layout->num_kv_heads != 0) return HACK_ERR_INVALID_ARGUMENT;
  if (layout->head_dim != 128 || hidden % 64 != 0) return HACK_ERR_UNSUPPORTED;
  const int64_t cap = cache_capacity(layout, cache, batch);
  if (cap < 0) return HACK_ERR_INVALID_ARGUMENT;
  if (len > cap) return HACK_ERR_CAPACITY;
  const int64_t tiles = (int64_t)batch * ((len + 255) / 256) * ((num_q_heads + 2 * layout->num_kv_heads + 1) / 2);
  if (tiles > INT32_MAX) return HACK_ERR_UNSUPPORTED;  // one workgroup per tile in a 1-D grid
  if (batch == 0 || len == 0) return HACK_OK;
  hack::ProjectArgs a;
  std::memset(&a, 0, sizeof(a));
  a.c = make_view(layout, cache);
  a.e = static_cast<const __half*>(e_dev);
  a.w = static_cast<const __half*>(w_dev);
  a.q = static_cast<__half*>(q_out_dev);
  a.batch = batch;
  a.len = len;
  a.hidden = hidden;
  a.q_heads = num_q_heads;
  a.kv_heads = layout->num_kv_heads;
  (void)hipGetLastError();
  return from_hip(hack::launch_project(*layout, a, stream));
}

hack_status hack_prefill_from_embeddings(const hack_kv_layout* layout, const hack_kv_cache* cache,
                                         const void* e_dev, const void* w_dev, int32_t num_q_heads, int32_t hidden,
                                         int32_t batch, int32_t len, int32_t causal, void* q_out_dev,
                                         float* out_dev, hipStream_t stream) {
  if (!layout_ok(layout) || !out_dev) return HACK_ERR_INVALID_ARGUMENT;
  // the attention's own checks first, so that nothing is launched for a shape it rejects
  if (num_q_heads < 1 || num_q_heads % layout->num_kv_heads != 0) return HACK_ERR_INVALID_ARGUMENT;
  const hack_status sh = attention_shape(layout, num_q_heads);
  if (sh != HACK_OK) return sh;
  if (layout->sum_bytes == 0 || batch > kMaxGridYZ) return HACK_ERR_UNSUPPORTED;
  hack_status st = hack_project_qkv(layout, cache, e_dev, w_dev, num_q_heads, hidden, batch, len, q_out_dev, stream);
  if (st != HACK_OK) return st;
  return hack_attend_prefill(layout, cache, q_out_dev, num_q_heads, batch, len, causal, out_dev, stream);
}

const char* hack_status_string(hack_status status) {
  switch (status) {
    case HACK_OK: return "ok";
    case HACK_ERR_INVALID_ARGUMENT: return "invalid argument";
    case HACK_ERR_UNSUPPORTED: return "unsupported format or shape";
    case HACK_ERR_CAPACITY: return "length exceeds the cache capacity";
    case HACK_ERR_WORKSPACE: return "workspace missing or too small";
    case HACK_ERR_HIP: return "HIP launch failure";
    default: return "unknown status";
  }
}

hack_status hack_debug_qk_products(const hack_kv_layout* layout, const hack_kv_cache* cache, const void* q_dev,
                                   int32_t num_q_heads, const int32_t* seq_lens_dev, int32_t batch,
                                   int32_t max_len, uint8_t* q_codes_dev, float* q_meta_dev,
                                   int32_t* products_dev, hipStream_t stream) {
  hack::DecodeArgs a;
  int64_t cap = 0;
  hack_status st = decode_common(layout, cache, q_dev, num_q_heads, seq_lens_dev, batch, max_len, a, &cap);
  if (st != HACK_OK) return st;
  if (layout->sum_bytes == 0) return HACK_ERR_UNSUPPORTED;  // the exports read cached sums
  if (layout->partition == 128) return HACK_ERR_UNSUPPORTED;  // exports of the matrix-core kernel only
  if (!q_codes_dev || !q_meta_dev || !products_dev) return HACK_ERR_INVALID_ARGUMENT;
  if (batch == 0) return HACK_OK;
  const hack::DecodePlan plan = hack::plan_decode(*layout, batch, num_q_heads, max_len);
  a.chunk = plan.chunk;
  a.splits = plan.splits;
  a.dbg_qcodes = q_codes_dev;
  a.dbg_qmeta = q_meta_dev;
  a.dbg_prod = products_dev;
  (void)hipGetLastError();
  return from_hip(hack::launch_decode(*layout, a, batch, hack::MODE_QK, stream));
}

hack_status hack_debug_pv_products(const hack_kv_layout* layout, const hack_kv_cache* cache,
                                   const uint8_t* p_codes_dev, const float* p_meta_dev, int32_t num_q_heads,
                                   const int32_t* seq_lens_dev, int32_t batch, int32_t max_len,
                                   int32_t* products_dev, float* out_dev, hipStream_t stream) {
  hack::DecodeArgs a;
  int64_t cap = 0;
  // the query is not read in this mode; pass any non-null pointer through validation
  hack_status st = decode_common(layout, cache, p_codes_dev, num_q_heads, seq_lens_dev, batch, max_len, a, &cap);
  if (st != HACK_OK) return st;
  if (layout->sum_bytes == 0) return HACK_ERR_UNSUPPORTED;  // the exports read cached sums
  if (layout->partition == 128) return HACK_ERR_UNSUPPORTED;  // exports of the matrix-core kernel only
  if (!p_meta_dev || !products_dev || !out_dev) return HACK_ERR_INVALID_ARGUMENT;
  if (batch == 0) return HACK_OK;
  const int span = 4 * layout->partition;
  a.q = nullptr;
  a.chunk = ((max_len + span - 1) / span) * span;
  if (a.chunk == 0) a.chunk = span;
  a.splits = 1;
  a.out = out_dev;
  a.dbg_prod = products_dev;
  a.dbg_pcodes = p_codes_dev;
  a.dbg_pmeta = p_meta_dev;
  (void)hipGetLastError();
  return from_hip(hack::launch_decode(*layout, a, batch, hack::MODE_PV, stream));
}

}  // extern "C"

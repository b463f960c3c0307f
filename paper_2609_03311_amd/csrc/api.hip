// api.hip -- host side of the C ABI declared in include/dopr.h: argument
// validation, store layout, workspace sizing and kernel launches.  Nothing
// here allocates device memory; every device buffer comes from the caller,
// except the fixed scratch array below that dopr_prefix_attn_noalloc uses.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.hpp"

using namespace dopr;

// Scratch of dopr_prefix_attn_noalloc: the attention plan of one call.  The
// code object holds one copy per device that loads it, for the life of the
// process.  In host code `scratch` names a host-side stand-in, not device
// memory: the device address comes from hipGetSymbolAddress (scratch_ptr
// below) and only that address is ever handed to a kernel.
static __device__ __align__(256) char scratch[dopr::kNoAllocScratchBytes];

namespace {

thread_local std::string g_last_error;

dopr_status_t fail(dopr_status_t s, const std::string &msg) {
  g_last_error = std::string(dopr_status_str(s)) + ": " + msg;
  return s;
}

dopr_status_t hip_fail(hipError_t e, const char *what) {
  return fail(DOPR_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

dopr_status_t ok() {
  g_last_error.clear();
  return DOPR_OK;
}

bool aligned16(const void *p) {
  return (reinterpret_cast<uintptr_t>(p) & 15) == 0;
}

hipStream_t as_stream(void *s) { return static_cast<hipStream_t>(s); }

struct StoreLayout {
  size_t len_off = 0, off_off = 0, kmax_off = 0, payload_off = 0, total = 0;
  size_t payload_canonical = 0;
  int32_t max_len = 0;
};

// Offsets of the pool sections; optionally the per-document block offsets.
dopr_status_t layout_store(const dopr_store_desc_t *d, StoreLayout *lay,
                           std::vector<int64_t> *doc_off) {
  if (!d) return fail(DOPR_ERR_INVALID_ARG, "desc is NULL");
  if (d->n_docs < 0 || d->n_docs > INT32_MAX)
    return fail(DOPR_ERR_INVALID_ARG, "n_docs must be in [0, 2^31)");
  if (d->n_docs > 0 && !d->doc_len)
    return fail(DOPR_ERR_INVALID_ARG, "doc_len is NULL");
  if (d->n_layers < 1 || d->n_kv_heads < 1)
    return fail(DOPR_ERR_INVALID_ARG, "n_layers and n_kv_heads must be >= 1");
  if (d->head_dim != 128 && d->head_dim != 64)
    return fail(DOPR_ERR_UNSUPPORTED, "head_dim must be 128 or 64");
  size_t off = align_up(sizeof(int32_t) * kStatusWords, kAlign);
  lay->len_off = off;
  off = align_up(off + sizeof(int32_t) * (size_t)d->n_docs, kAlign);
  lay->off_off = off;
  off = align_up(off + sizeof(int64_t) * (size_t)d->n_docs, kAlign);
  lay->kmax_off = off;
  off = align_up(off + sizeof(float) * (size_t)d->n_docs * d->n_layers *
                           d->n_kv_heads,
                 kAlign);
  lay->payload_off = off;
  int64_t elems = 0;
  size_t canon = 0;
  int32_t max_len = 0;
  if (doc_off) doc_off->assign((size_t)d->n_docs, -1);
  for (int64_t i = 0; i < d->n_docs; ++i) {
    const int32_t L = d->doc_len[i];
    if (L < -1)
      return fail(DOPR_ERR_INVALID_ARG,
                  "doc_len entries must be >= 0, or -1 (not resident)");
    if (L < 0) continue;
    if (doc_off) (*doc_off)[i] = elems;
    elems += (int64_t)d->n_layers *
             layer_block_elems(L, d->n_kv_heads, d->head_dim);
    canon += (size_t)L * d->n_layers * d->n_kv_heads * d->head_dim * 2 * 2;
    if (L > max_len) max_len = L;
  }
  lay->total = off + sizeof(uint16_t) * (size_t)elems;
  lay->payload_canonical = canon;
  lay->max_len = max_len;
  return DOPR_OK;
}

bool uses_stream_kernel(int32_t variant, const dopr_store *st);

// Rows per work item: long items for the full layer (the block kernels and
// the pass kernel stage a document's prefix once per item and walk the item
// in passes), and 32 for the one-wave-per-unit score kernel that the
// automatic choice takes when every prefix is at most kScoreRowsMaxLen
// slots.
int32_t default_rows_per_item(int32_t variant, bool score_only,
                              int32_t max_len, int32_t n_rep) {
  if (score_only)
    return (variant == 0 || variant == 5) && max_len <= kScoreRowsMaxLen
               ? 32
               : 2048;
  (void)n_rep;
  return 2048;
}

// The full layer runs the pass kernel for variant 8 and, in the automatic
// choice and the self-check mode, unless every prefix is short at head size
// 128 (at most 96 slots: two 4-wave blocks per CU keep it resident, and the
// pass kernel's per-pass costs outweigh its savings there).  Its plan then
// holds k^ of every token.
bool uses_stream_kernel(int32_t variant, const dopr_store *st) {
  if (variant == 8) return true;
  if (variant != 0 && variant != 5) return false;
  return !(st->head_dim == 128 && st->max_len <= kShortPrefix128);
}

// Validation shared by the workspace query and the attention call.
dopr_status_t check_attn(const dopr_store *st, const dopr_attn_args_t *a,
                         PlanShape *shape, int32_t *n_rep,
                         bool score_only = false) {
  if (!st) return fail(DOPR_ERR_INVALID_ARG, "store is NULL");
  if (!a) return fail(DOPR_ERR_INVALID_ARG, "args is NULL");
  if (a->n_pairs < 0) return fail(DOPR_ERR_INVALID_ARG, "n_pairs < 0");
  if (a->n_q_heads < 1 || a->n_q_heads % st->n_kv_heads)
    return fail(DOPR_ERR_INVALID_ARG,
                "n_q_heads must be a positive multiple of n_kv_heads");
  if (a->max_tokens < 1 || a->max_tokens > (1 << 20))
    return fail(DOPR_ERR_INVALID_ARG, "max_tokens must be in [1, 2^20]");
  if (a->total_tokens < a->n_pairs)
    return fail(DOPR_ERR_INVALID_ARG,
                "total_tokens must be >= n_pairs (every T_p >= 1)");
  *n_rep = a->n_q_heads / st->n_kv_heads;
  const int64_t stacked = score_only ? a->n_pairs : a->total_tokens;
  if (stacked * (int64_t)(*n_rep) > INT32_MAX)
    return fail(DOPR_ERR_UNSUPPORTED,
                "stacked rows (tokens, or pairs in score mode) * n_rep must "
                "be < 2^31");
  if (a->kernel_variant < 0 || a->kernel_variant > 8 ||
      a->kernel_variant == 7)
    return fail(DOPR_ERR_INVALID_ARG, "kernel_variant must be in 0..6 or 8");
  if (!(a->softmax_scale > 0.f) || !std::isfinite(a->softmax_scale))
    return fail(DOPR_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
  if (!(a->rope_theta > 1.f) || !std::isfinite(a->rope_theta))
    return fail(DOPR_ERR_INVALID_ARG, "rope_theta must be finite and > 1");
  if (!(a->rms_eps >= 0.f) || !std::isfinite(a->rms_eps))
    return fail(DOPR_ERR_INVALID_ARG, "rms_eps must be finite and >= 0");
  shape->n_pairs = a->n_pairs;
  shape->n_rep = *n_rep;
  shape->max_tokens = a->max_tokens;
  if (a->rows_per_item != 0) {
    if (score_only)
      return fail(DOPR_ERR_INVALID_ARG,
                  "rows_per_item must be 0 for last-layer scoring");
    // near-equal cuts of >= 32 rows each keep every item non-empty
    if (a->rows_per_item < 64 || a->rows_per_item > (1 << 20) ||
        a->rows_per_item % 32)
      return fail(DOPR_ERR_INVALID_ARG,
                  "rows_per_item must be 0 or a multiple of 32 in "
                  "[64, 2^20]");
  }
  if (a->queue_order < 0 || a->queue_order > 2)
    return fail(DOPR_ERR_INVALID_ARG, "queue_order must be 0, 1 or 2");
  shape->rows_per_item =
      a->rows_per_item ? a->rows_per_item
                       : default_rows_per_item(a->kernel_variant, score_only,
                                               st->max_len, *n_rep);
  // work units (item, kv head) are numbered in 32 bits by the scheduler's
  // queues: the plan's item capacity times the kv heads must stay below
  // 2^31
  const int64_t rows = stacked * (int64_t)(*n_rep);
  const int64_t items_cap =
      a->n_pairs + (rows + shape->rows_per_item - 1) / shape->rows_per_item +
      1;
  if (items_cap * (int64_t)st->n_kv_heads > INT32_MAX)
    return fail(DOPR_ERR_UNSUPPORTED,
                "too many work units (pairs and items times kv heads must be "
                "< 2^31)");
  shape->n_docs = st->n_docs;
  shape->total_tokens = a->total_tokens;
  shape->max_len = st->max_len;
  shape->n_kv_heads = st->n_kv_heads;
  shape->head_dim = st->head_dim;
  shape->score_only = score_only;
  shape->stream = !score_only && uses_stream_kernel(a->kernel_variant, st);
  return DOPR_OK;
}

dopr_status_t check_device(const dopr_store *st) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != st->device)
    return fail(DOPR_ERR_INVALID_ARG,
                "current device differs from the store's device");
  return DOPR_OK;
}

}  // namespace

extern "C" {

const char *dopr_status_str(dopr_status_t s) {
  switch (s) {
    case DOPR_OK: return "DOPR_OK";
    case DOPR_ERR_INVALID_ARG: return "DOPR_ERR_INVALID_ARG";
    case DOPR_ERR_UNSUPPORTED: return "DOPR_ERR_UNSUPPORTED";
    case DOPR_ERR_DOC_RANGE: return "DOPR_ERR_DOC_RANGE";
    case DOPR_ERR_WORKSPACE: return "DOPR_ERR_WORKSPACE";
    case DOPR_ERR_HIP: return "DOPR_ERR_HIP";
    case DOPR_ERR_SEQLEN: return "DOPR_ERR_SEQLEN";
  }
  return "DOPR_ERR_UNKNOWN";
}

const char *dopr_last_error(void) { return g_last_error.c_str(); }

dopr_status_t dopr_store_bytes(const dopr_store_desc_t *desc,
                               size_t *pool_bytes, size_t *payload_bytes) {
  if (!pool_bytes) return fail(DOPR_ERR_INVALID_ARG, "pool_bytes is NULL");
  StoreLayout lay;
  dopr_status_t s = layout_store(desc, &lay, nullptr);
  if (s != DOPR_OK) return s;
  *pool_bytes = lay.total;
  if (payload_bytes) *payload_bytes = lay.payload_canonical;
  return ok();
}

dopr_status_t dopr_store_create(const dopr_store_desc_t *desc, void *pool,
                                size_t pool_bytes, void *stream,
                                dopr_store_t *out) {
  if (!out) return fail(DOPR_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  StoreLayout lay;
  std::vector<int64_t> doc_off;
  dopr_status_t s = layout_store(desc, &lay, &doc_off);
  if (s != DOPR_OK) return s;
  if (!pool) return fail(DOPR_ERR_INVALID_ARG, "pool is NULL");
  if (reinterpret_cast<uintptr_t>(pool) % kAlign)
    return fail(DOPR_ERR_INVALID_ARG, "pool must be 256-byte aligned");
  if (pool_bytes < lay.total)
    return fail(DOPR_ERR_WORKSPACE,
                "pool holds " + std::to_string(pool_bytes) + " bytes, store needs " +
                    std::to_string(lay.total));
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  dopr_store *st = new (std::nothrow) dopr_store{};
  if (!st) return fail(DOPR_ERR_INVALID_ARG, "host allocation failed");
  char *base = static_cast<char *>(pool);
  st->n_layers = desc->n_layers;
  st->n_kv_heads = desc->n_kv_heads;
  st->head_dim = desc->head_dim;
  st->n_docs = desc->n_docs;
  st->pool = base;
  st->pool_bytes = pool_bytes;
  st->d_status = reinterpret_cast<int32_t *>(base);
  st->d_len = reinterpret_cast<int32_t *>(base + lay.len_off);
  st->d_off = reinterpret_cast<int64_t *>(base + lay.off_off);
  st->d_kmax = reinterpret_cast<float *>(base + lay.kmax_off);
  st->d_payload = reinterpret_cast<uint16_t *>(base + lay.payload_off);
  st->max_len = lay.max_len;
  st->device = dev;
  hipStream_t hs = as_stream(stream);
  e = hipMemsetAsync(st->d_status, 0, sizeof(int32_t) * kStatusWords, hs);
  if (e == hipSuccess && desc->n_docs > 0)
    e = hipMemcpyAsync(st->d_len, desc->doc_len,
                       sizeof(int32_t) * (size_t)desc->n_docs,
                       hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && desc->n_docs > 0)
    e = hipMemcpyAsync(st->d_off, doc_off.data(),
                       sizeof(int64_t) * (size_t)desc->n_docs,
                       hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && desc->n_docs > 0)
    e = hipMemsetAsync(st->d_kmax, 0,
                       sizeof(float) * (size_t)desc->n_docs * desc->n_layers *
                           desc->n_kv_heads,
                       hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) {
    delete st;
    return hip_fail(e, "store index upload");
  }
  *out = st;
  return ok();
}

dopr_status_t dopr_store_put(dopr_store_t st, int32_t layer, int64_t n,
                             const int32_t *doc_ids,
                             const int64_t *src_cu_slots, const void *k_src,
                             const void *v_src, void *stream) {
  if (!st) return fail(DOPR_ERR_INVALID_ARG, "store is NULL");
  if (layer < 0 || layer >= st->n_layers)
    return fail(DOPR_ERR_INVALID_ARG, "layer out of range");
  if (n < 0 || n > INT32_MAX) return fail(DOPR_ERR_INVALID_ARG, "bad n");
  if (n == 0) return ok();
  if (!doc_ids || !src_cu_slots || !k_src || !v_src)
    return fail(DOPR_ERR_INVALID_ARG, "NULL buffer");
  if (!aligned16(k_src) || !aligned16(v_src))
    return fail(DOPR_ERR_INVALID_ARG, "k_src/v_src must be 16-byte aligned");
  dopr_status_t s = check_device(st);
  if (s != DOPR_OK) return s;
  hipError_t e = launch_store_put(*st, layer, n, doc_ids, src_cu_slots,
                                  static_cast<const uint16_t *>(k_src),
                                  static_cast<const uint16_t *>(v_src),
                                  as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "store_put launch");
  return ok();
}

dopr_status_t dopr_store_copy_docs(dopr_store_t dst, dopr_store_t src,
                                   void *stream) {
  if (!dst || !src) return fail(DOPR_ERR_INVALID_ARG, "store is NULL");
  if (dst->n_docs != src->n_docs || dst->n_layers != src->n_layers ||
      dst->n_kv_heads != src->n_kv_heads || dst->head_dim != src->head_dim)
    return fail(DOPR_ERR_INVALID_ARG,
                "stores differ in n_docs, n_layers, n_kv_heads or head_dim");
  if (dst->pool < src->pool + src->pool_bytes &&
      src->pool < dst->pool + dst->pool_bytes)
    return fail(DOPR_ERR_INVALID_ARG, "store pools overlap");
  if (dst->device != src->device)
    return fail(DOPR_ERR_INVALID_ARG, "stores live on different devices");
  dopr_status_t s = check_device(dst);
  if (s != DOPR_OK) return s;
  hipError_t e = launch_store_copy(*dst, *src, as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "store_copy launch");
  return ok();
}

dopr_status_t dopr_store_destroy(dopr_store_t st) {
  delete st;
  return ok();
}

dopr_status_t dopr_prefix_attn_workspace(dopr_store_t st,
                                         const dopr_attn_args_t *args,
                                         size_t *bytes) {
  if (!bytes) return fail(DOPR_ERR_INVALID_ARG, "bytes is NULL");
  PlanShape shape;
  int32_t n_rep = 0;
  dopr_status_t s = check_attn(st, args, &shape, &n_rep);
  if (s != DOPR_OK) return s;
  *bytes = plan_bytes(shape);
  return ok();
}

}  // extern "C"

namespace {

// Device address of `scratch` on device `dev`, looked up once per device
// (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

dopr_status_t scratch_ptr(int dev, void **out) {
  if (dev < 0 || dev >= kMaxDevices)
    return fail(DOPR_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || reinterpret_cast<uintptr_t>(p) % kAlign)
      return fail(DOPR_ERR_HIP, "scratch address is NULL or misaligned");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DOPR_OK;
}

// The attention call in both modes: every online row (head == NULL) or the
// score token's rows with the fused score head.  no_alloc: the plan goes to
// the library's scratch array instead of the caller's workspace; the
// automatic kernel choice then keeps to the block kernels (the pass kernel's
// k^ buffer grows with the batch), and variant 8 is taken only when asked for.
dopr_status_t run_attention(dopr_store_t st, int32_t layer,
                            const dopr_attn_args_t *a,
                            const dopr_score_head_t *head, void *stream,
                            bool no_alloc = false) {
  const bool score = head != nullptr;
  PlanShape shape;
  int32_t n_rep = 0;
  dopr_status_t s = check_attn(st, a, &shape, &n_rep, score);
  if (s != DOPR_OK) return s;
  if (no_alloc) {
    if (a->workspace || a->workspace_bytes)
      return fail(DOPR_ERR_INVALID_ARG,
                  "workspace must be NULL with 0 bytes: the no-alloc call "
                  "uses the library's scratch");
    shape.stream = a->kernel_variant == 8;
  }
  if (layer < 0 || layer >= st->n_layers)
    return fail(DOPR_ERR_INVALID_ARG, "layer out of range");
  if (score) {
    if (!(head->rms_eps >= 0.f) || !std::isfinite(head->rms_eps))
      return fail(DOPR_ERR_INVALID_ARG,
                  "head rms_eps must be finite and >= 0");
  }
  if (a->n_pairs == 0) return ok();
  if (!a->doc_ids || !a->cu_seqlens || !a->q || !a->k || !a->v ||
      (!a->out && !score) || (!a->workspace && !no_alloc))
    return fail(DOPR_ERR_INVALID_ARG, "NULL buffer");
  if (!a->q_norm_w != !a->k_norm_w)
    return fail(DOPR_ERR_INVALID_ARG,
                "q_norm_w and k_norm_w must both be given or both be NULL");
  if (!aligned16(a->q) || !aligned16(a->k) || !aligned16(a->v) ||
      !aligned16(a->out) || !aligned16(a->q_norm_w) || !aligned16(a->k_norm_w))
    return fail(DOPR_ERR_INVALID_ARG,
                "q, k, v, out and norm weights must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(a->rope_inv_freq) % 4)
    return fail(DOPR_ERR_INVALID_ARG, "rope_inv_freq must be 4-byte aligned");
  if (score) {
    if (!head->norm_w || !head->w_head || !head->score)
      return fail(DOPR_ERR_INVALID_ARG, "NULL score-head buffer");
    if (!aligned16(head->norm_w) || !aligned16(head->w_head))
      return fail(DOPR_ERR_INVALID_ARG,
                  "head norm_w and w_head must be 16-byte aligned");
  }
  const size_t need = plan_bytes(shape);
  void *ws = a->workspace;
  if (no_alloc) {
    if (need > kNoAllocScratchBytes)
      return fail(DOPR_ERR_WORKSPACE,
                  "the call needs " + std::to_string(need) +
                      " bytes of scratch; the no-alloc entry point holds " +
                      std::to_string(kNoAllocScratchBytes) +
                      " (use dopr_prefix_attn with a workspace)");
  } else {
    if (reinterpret_cast<uintptr_t>(a->workspace) % kAlign)
      return fail(DOPR_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    if (a->workspace_bytes < need)
      return fail(DOPR_ERR_WORKSPACE,
                  "workspace holds " + std::to_string(a->workspace_bytes) +
                      " bytes, needs " + std::to_string(need));
  }
  s = check_device(st);
  if (s != DOPR_OK) return s;
  if (no_alloc) {
    s = scratch_ptr(st->device, &ws);
    if (s != DOPR_OK) return s;
  }
  const Plan plan = plan_carve(ws, shape);
  AttnCall call{st, layer, a, n_rep, head};
  hipStream_t hs = as_stream(stream);
  hipError_t e = launch_plan(call, plan, shape, hs);
  if (e != hipSuccess) return hip_fail(e, "scheduler launch");
  e = launch_attention(call, plan, shape, hs);
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  return ok();
}

}  // namespace

extern "C" {

dopr_status_t dopr_prefix_attn(dopr_store_t st, int32_t layer,
                               const dopr_attn_args_t *a, void *stream) {
  return run_attention(st, layer, a, nullptr, stream);
}

dopr_status_t dopr_prefix_attn_noalloc(dopr_store_t st, int32_t layer,
                                       const dopr_attn_args_t *a,
                                       void *stream) {
  return run_attention(st, layer, a, nullptr, stream, true);
}

dopr_status_t dopr_prefix_attn_score_workspace(dopr_store_t st,
                                               const dopr_attn_args_t *args,
                                               size_t *bytes) {
  if (!bytes) return fail(DOPR_ERR_INVALID_ARG, "bytes is NULL");
  PlanShape shape;
  int32_t n_rep = 0;
  dopr_status_t s = check_attn(st, args, &shape, &n_rep, true);
  if (s != DOPR_OK) return s;
  *bytes = plan_bytes(shape);
  return ok();
}

dopr_status_t dopr_prefix_attn_score(dopr_store_t st, int32_t layer,
                                     const dopr_attn_args_t *args,
                                     const dopr_score_head_t *head,
                                     void *stream) {
  if (!head) return fail(DOPR_ERR_INVALID_ARG, "head is NULL");
  return run_attention(st, layer, args, head, stream);
}

}  // extern "C"

namespace {

// Shapes and checks of a decoder-layer call; on success *ls and *shape
// describe the layer buffers and the attention plan.
dopr_status_t check_layer(dopr_store_t st, const dopr_attn_args_t *b,
                          const dopr_layer_args_t *l, LayerShape *ls,
                          PlanShape *shape, int32_t *n_rep) {
  dopr_status_t s = check_attn(st, b, shape, n_rep);
  if (s != DOPR_OK) return s;
  if (!l) return fail(DOPR_ERR_INVALID_ARG, "layer args are NULL");
  if (st->head_dim != kHeadDim)
    return fail(DOPR_ERR_UNSUPPORTED,
                "the decoder layer is built for head_dim 128");
  if (l->hidden < 8 || l->hidden % 8 || l->intermediate < 8 ||
      l->intermediate % 8)
    return fail(DOPR_ERR_INVALID_ARG,
                "hidden and intermediate must be multiples of 8, >= 8");
  if (b->q || b->k || b->v || b->out)
    return fail(DOPR_ERR_INVALID_ARG,
                "q, k, v and out must be NULL: the layer forms them");
  *ls = LayerShape{b->total_tokens, l->hidden, l->intermediate,
                   b->n_q_heads, st->n_kv_heads};
  return DOPR_OK;
}

size_t layer_bytes(const LayerShape &ls, const PlanShape &shape) {
  return layer_carve(nullptr, ls).bytes + plan_bytes(shape);
}

}  // namespace

extern "C" {

dopr_status_t dopr_decoder_layer_workspace(dopr_store_t st,
                                           const dopr_attn_args_t *batch,
                                           const dopr_layer_args_t *lw,
                                           size_t *bytes) {
  if (!bytes) return fail(DOPR_ERR_INVALID_ARG, "bytes is NULL");
  LayerShape ls;
  PlanShape shape;
  int32_t n_rep = 0;
  dopr_status_t s = check_layer(st, batch, lw, &ls, &shape, &n_rep);
  if (s != DOPR_OK) return s;
  *bytes = layer_bytes(ls, shape);
  return ok();
}

dopr_status_t dopr_decoder_layer(dopr_store_t st, int32_t layer,
                                 const dopr_attn_args_t *b,
                                 const dopr_layer_args_t *l, void *stream) {
  LayerShape ls;
  PlanShape shape;
  int32_t n_rep = 0;
  dopr_status_t s = check_layer(st, b, l, &ls, &shape, &n_rep);
  if (s != DOPR_OK) return s;
  if (layer < 0 || layer >= st->n_layers)
    return fail(DOPR_ERR_INVALID_ARG, "layer out of range");
  if (b->n_pairs == 0) return ok();
  if (!b->doc_ids || !b->cu_seqlens || !b->q_norm_w || !b->k_norm_w ||
      !b->workspace || !l->attn_norm_w || !l->w_q || !l->w_k || !l->w_v ||
      !l->w_o || !l->mlp_norm_w || !l->w_gate || !l->w_up || !l->w_down ||
      !l->x || !l->y)
    return fail(DOPR_ERR_INVALID_ARG, "NULL buffer");
  const void *al[] = {b->q_norm_w, b->k_norm_w, l->attn_norm_w, l->w_q,
                      l->w_k,      l->w_v,      l->w_o,         l->mlp_norm_w,
                      l->w_gate,   l->w_up,     l->w_down,      l->x,
                      l->y};
  for (const void *p : al)
    if (!aligned16(p))
      return fail(DOPR_ERR_INVALID_ARG,
                  "weights, x and y must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(b->workspace) % kAlign)
    return fail(DOPR_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  const size_t need = layer_bytes(ls, shape);
  if (b->workspace_bytes < need)
    return fail(DOPR_ERR_WORKSPACE,
                "workspace holds " + std::to_string(b->workspace_bytes) +
                    " bytes, needs " + std::to_string(need));
  s = check_device(st);
  if (s != DOPR_OK) return s;
  const LayerWs w = layer_carve(b->workspace, ls);
  dopr_attn_args_t a = *b;  // the attention of this layer
  a.q = w.q;
  a.k = w.k;
  a.v = w.v;
  a.out = w.att;
  a.workspace = w.plan;
  a.workspace_bytes = plan_bytes(shape);
  const Plan plan = plan_carve(w.plan, shape);
  AttnCall call{st, layer, &a, n_rep};
  hipStream_t hs = as_stream(stream);
  int g = launch_layer_pre(ls, l, w, b->rms_eps, hs);
  if (g != 0)
    return g < 0 ? hip_fail(hipGetLastError(), "layer launch")
                 : fail(DOPR_ERR_HIP, std::string("hipBLASLt: ") +
                                          gemm_status_str(g));
  hipError_t e = launch_plan(call, plan, shape, hs);
  if (e != hipSuccess) return hip_fail(e, "scheduler launch");
  e = launch_attention(call, plan, shape, hs);
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  g = launch_layer_post(ls, l, w, b->rms_eps, hs);
  if (g != 0)
    return g < 0 ? hip_fail(hipGetLastError(), "layer launch")
                 : fail(DOPR_ERR_HIP, std::string("hipBLASLt: ") +
                                          gemm_status_str(g));
  return ok();
}

dopr_status_t dopr_score_logits(const dopr_score_args_t *a, void *stream) {
  if (!a) return fail(DOPR_ERR_INVALID_ARG, "args is NULL");
  if (a->n_pairs < 0) return fail(DOPR_ERR_INVALID_ARG, "n_pairs < 0");
  if (a->width < 8 || a->width % 8)
    return fail(DOPR_ERR_INVALID_ARG, "width must be a multiple of 8, >= 8");
  if (a->h_row_stride < a->width || a->h_row_stride % 8)
    return fail(DOPR_ERR_INVALID_ARG,
                "h_row_stride must be >= width and a multiple of 8");
  if (!(a->rms_eps >= 0.f) || !std::isfinite(a->rms_eps))
    return fail(DOPR_ERR_INVALID_ARG, "rms_eps must be finite and >= 0");
  if (a->n_pairs == 0) return ok();
  if (!a->h || !a->norm_w || !a->w_head || !a->score)
    return fail(DOPR_ERR_INVALID_ARG, "NULL buffer");
  if (!aligned16(a->h) || !aligned16(a->norm_w) || !aligned16(a->w_head))
    return fail(DOPR_ERR_INVALID_ARG, "h, norm_w, w_head must be 16-byte aligned");
  hipError_t e = launch_score(a, as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "score launch");
  return ok();
}

dopr_status_t dopr_group_pairs(dopr_store_t st, int32_t n_pairs,
                               const int32_t *doc_ids, void *workspace,
                               size_t workspace_bytes, int32_t *n_groups,
                               int32_t *n_valid, int32_t *group_doc,
                               int32_t *group_ptr, int32_t *pair_order,
                               void *stream) {
  if (!st) return fail(DOPR_ERR_INVALID_ARG, "store is NULL");
  if (!n_groups || !n_valid)
    return fail(DOPR_ERR_INVALID_ARG, "n_groups/n_valid is NULL");
  if (n_pairs < 0) return fail(DOPR_ERR_INVALID_ARG, "n_pairs < 0");
  *n_groups = 0;
  *n_valid = 0;
  if (n_pairs == 0) return ok();
  if (!doc_ids || !workspace || !group_doc || !group_ptr || !pair_order)
    return fail(DOPR_ERR_INVALID_ARG, "NULL buffer");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(DOPR_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  dopr_status_t s = check_device(st);
  if (s != DOPR_OK) return s;
  dopr_attn_args_t a{};
  a.n_pairs = n_pairs;
  a.n_q_heads = st->n_kv_heads;
  a.max_tokens = 1;
  a.total_tokens = n_pairs;
  a.doc_ids = doc_ids;
  a.cu_seqlens = nullptr;
  a.rope_theta = 1e6f;
  a.softmax_scale = 1.f;
  PlanShape shape{n_pairs,     1,          1, 2048,
                  st->n_docs,  (int64_t)n_pairs, st->max_len,
                  st->n_kv_heads};
  const size_t need = plan_bytes(shape);
  if (workspace_bytes < need)
    return fail(DOPR_ERR_WORKSPACE, "workspace too small for grouping");
  const Plan plan = plan_carve(workspace, shape);
  AttnCall call{st, 0, &a, 1};
  hipStream_t hs = as_stream(stream);
  hipError_t e = launch_plan(call, plan, shape, hs);
  if (e != hipSuccess) return hip_fail(e, "scheduler launch");
  int64_t totals[4] = {0, 0, 0, 0};
  e = hipMemcpyAsync(totals, plan.counters + kCounters, sizeof(totals),
                     hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return hip_fail(e, "grouping readback");
  const int32_t nv = (int32_t)(totals[0] & 0xffffffff);
  const int32_t ng = (int32_t)(totals[0] >> 32);
  if (nv > 0)
    e = hipMemcpyAsync(pair_order, plan.pair_order, sizeof(int32_t) * nv,
                       hipMemcpyDeviceToDevice, hs);
  if (e == hipSuccess && ng > 0)
    e = hipMemcpyAsync(group_doc, plan.group_doc, sizeof(int32_t) * ng,
                       hipMemcpyDeviceToDevice, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(group_ptr, plan.group_ptr, sizeof(int32_t) * (ng + 1),
                       hipMemcpyDeviceToDevice, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return hip_fail(e, "grouping copy-out");
  *n_groups = ng;
  *n_valid = nv;
  return ok();
}

dopr_status_t dopr_gather_prefix(dopr_store_t st, int32_t layer, int32_t n,
                                 const int32_t *doc_ids,
                                 const int64_t *out_cu_slots, void *k_out,
                                 void *v_out, void *stream) {
  if (!st) return fail(DOPR_ERR_INVALID_ARG, "store is NULL");
  if (layer < 0 || layer >= st->n_layers)
    return fail(DOPR_ERR_INVALID_ARG, "layer out of range");
  if (n < 0) return fail(DOPR_ERR_INVALID_ARG, "n < 0");
  if (n == 0) return ok();
  if (!doc_ids || !out_cu_slots || !k_out || !v_out)
    return fail(DOPR_ERR_INVALID_ARG, "NULL buffer");
  if (!aligned16(k_out) || !aligned16(v_out))
    return fail(DOPR_ERR_INVALID_ARG, "k_out/v_out must be 16-byte aligned");
  dopr_status_t s = check_device(st);
  if (s != DOPR_OK) return s;
  hipError_t e = launch_gather(*st, layer, n, doc_ids, out_cu_slots,
                               static_cast<uint16_t *>(k_out),
                               static_cast<uint16_t *>(v_out),
                               as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "gather launch");
  return ok();
}

}  // extern "C"

namespace {

// Host checks shared by the salience entry points; `full` adds those of the
// attention part (heads, p, q, k); `ptrs` the buffer checks (not for a
// workspace query).
dopr_status_t check_salience(const dopr_salience_args_t *a, bool full,
                             bool ptrs = true) {
  if (!a) return fail(DOPR_ERR_INVALID_ARG, "args is NULL");
  if (a->n_docs < 0) return fail(DOPR_ERR_INVALID_ARG, "n_docs < 0");
  if (a->max_doclen < 1 || a->max_doclen > kSalienceMaxLen)
    return fail(a->max_doclen > kSalienceMaxLen ? DOPR_ERR_UNSUPPORTED
                                                : DOPR_ERR_INVALID_ARG,
                "max_doclen must be in [1, 4096]");
  if (a->total_tokens < 0 || a->total_tokens > INT32_MAX)
    return fail(DOPR_ERR_INVALID_ARG, "total_tokens must be in [0, 2^31)");
  if (a->selected && (a->total_select < 0 || a->total_select > INT32_MAX))
    return fail(DOPR_ERR_INVALID_ARG, "total_select must be in [0, 2^31)");
  if (full) {
    if (a->n_q_heads < 1 || a->n_kv_heads < 1 ||
        a->n_q_heads % a->n_kv_heads)
      return fail(DOPR_ERR_INVALID_ARG,
                  "n_q_heads must be a positive multiple of n_kv_heads");
    if (a->top_p < 1 || a->top_p > kSalienceMaxP)
      return fail(a->top_p > kSalienceMaxP ? DOPR_ERR_UNSUPPORTED
                                           : DOPR_ERR_INVALID_ARG,
                  "top_p must be in [1, 64]");
    // the row pass scales each chunk's largest logit once: a positive
    // scale keeps it the largest scaled logit
    if (!(a->softmax_scale > 0.f) || !std::isfinite(a->softmax_scale))
      return fail(DOPR_ERR_INVALID_ARG,
                  "softmax_scale must be finite and > 0");
  }
  if (a->n_docs == 0 || !ptrs) return ok();
  if (!a->cu_doclens || !a->u)
    return fail(DOPR_ERR_INVALID_ARG, "cu_doclens and u are required");
  if (a->selected && !a->cu_select)
    return fail(DOPR_ERR_INVALID_ARG, "selected needs cu_select");
  if (full) {
    if (!a->q || !a->k) return fail(DOPR_ERR_INVALID_ARG, "q and k are required");
    if (!aligned16(a->q) || !aligned16(a->k))
      return fail(DOPR_ERR_INVALID_ARG, "q and k must be 16-byte aligned");
    if (a->attn_mean && (reinterpret_cast<uintptr_t>(a->attn_mean) & 15))
      return fail(DOPR_ERR_INVALID_ARG, "attn_mean must be 16-byte aligned");
  }
  return ok();
}

struct SalienceWs {
  size_t lse_bytes = 0, kn_bytes = 0, abar_bytes = 0, total = 0;
  int32_t chunk = 0;  // documents per pass
};

SalienceWs salience_ws(const dopr_salience_args_t *a) {
  SalienceWs w;
  const size_t M = (size_t)a->max_doclen;
  w.lse_bytes = align_up(sizeof(float) * (size_t)a->n_q_heads *
                             (size_t)a->total_tokens, kAlign);
  w.kn_bytes = align_up(sizeof(float) * kKeyNormParts * (size_t)a->n_docs *
                            (size_t)a->n_kv_heads, kAlign);
  if (a->attn_mean) {
    w.chunk = a->n_docs;
  } else {
    const size_t per = sizeof(float) * M * M;
    size_t c = kSalienceAbarBudget / per;
    if (c < 1) c = 1;
    if (c > (size_t)a->n_docs) c = (size_t)a->n_docs;
    w.chunk = (int32_t)c;
    w.abar_bytes = align_up(per * c, kAlign);
  }
  w.total = w.lse_bytes + w.kn_bytes + w.abar_bytes;
  return w;
}

TopkParams topk_params(const dopr_salience_args_t *a) {
  TopkParams t;
  t.cu = a->cu_doclens;
  t.cs = a->cu_select;
  t.u = a->u;
  t.selected = a->selected;
  t.max_len = a->max_doclen;
  t.total_tokens = a->total_tokens;
  t.total_select = a->total_select;
  t.status = a->status;
  return t;
}

}  // namespace

extern "C" {

dopr_status_t dopr_salience_workspace(const dopr_salience_args_t *args,
                                      size_t *bytes) {
  if (!bytes) return fail(DOPR_ERR_INVALID_ARG, "bytes is NULL");
  dopr_status_t s = check_salience(args, true, false);
  if (s != DOPR_OK) return s;
  *bytes = args->n_docs == 0 ? 0 : salience_ws(args).total;
  return ok();
}

dopr_status_t dopr_salience(const dopr_salience_args_t *a, void *stream) {
  dopr_status_t s = check_salience(a, true);
  if (s != DOPR_OK) return s;
  if (a->n_docs == 0) return ok();
  SalienceWs w = salience_ws(a);
  // the least workspace holds the row statistics and one document's Abar;
  // more room lets more documents share a pass
  const size_t per = sizeof(float) * (size_t)a->max_doclen * a->max_doclen;
  const size_t fixed = w.lse_bytes + w.kn_bytes;
  const size_t least = fixed + (a->attn_mean ? 0 : per);
  if (!a->workspace || a->workspace_bytes < least)
    return fail(DOPR_ERR_WORKSPACE,
                "workspace needs at least " + std::to_string(least) +
                    " bytes");
  if (!a->attn_mean)
    w.chunk = (int32_t)std::min<size_t>(
        (size_t)a->n_docs, (a->workspace_bytes - fixed) / per);
  if (reinterpret_cast<uintptr_t>(a->workspace) % kAlign)
    return fail(DOPR_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  char *base = static_cast<char *>(a->workspace);
  SalienceParams p;
  p.q = static_cast<const uint16_t *>(a->q);
  p.k = static_cast<const uint16_t *>(a->k);
  p.cu = a->cu_doclens;
  p.n_docs = a->n_docs;
  p.d0 = 0;
  p.hq = a->n_q_heads;
  p.hkv = a->n_kv_heads;
  p.n_rep = a->n_q_heads / a->n_kv_heads;
  p.max_len = a->max_doclen;
  p.top_p = a->top_p;
  p.total_tokens = a->total_tokens;
  p.c = a->softmax_scale * 1.4426950408889634f;
  p.inv_hq = 1.0f / (float)a->n_q_heads;
  p.lse2 = reinterpret_cast<float *>(base);
  p.kmax = reinterpret_cast<float *>(base + w.lse_bytes);
  p.abar = a->attn_mean ? a->attn_mean
                        : reinterpret_cast<float *>(base + fixed);
  p.abar_stride = (int64_t)a->max_doclen * a->max_doclen;
  p.u = a->u;
  p.status = a->status;
  // q heads per row-LSE sweep: two where the group allows (four q heads'
  // fragments plus the key fragments no longer fit two waves per SIMD)
  const int hr = p.n_rep % 2 == 0 ? 2 : 1;
  const int pm = a->top_p <= 8 ? 8 : a->top_p <= 16 ? 16
               : a->top_p <= 32 ? 32 : 64;
  hipStream_t hs = as_stream(stream);
  hipError_t e = launch_salience_check(p, hs);
  if (e == hipSuccess) e = launch_key_norms(p, hs);
  for (int32_t d0 = 0; e == hipSuccess && d0 < a->n_docs; d0 += w.chunk) {
    p.d0 = d0;
    const int32_t nd = std::min(w.chunk, a->n_docs - d0);
    e = launch_salience_chunk(p, nd, hr, pm, hs);
  }
  if (e == hipSuccess && a->selected)
    e = launch_topk(topk_params(a), a->n_docs, hs);
  if (e != hipSuccess) return hip_fail(e, "salience launch");
  return ok();
}

dopr_status_t dopr_select_top_k(const dopr_salience_args_t *a, void *stream) {
  dopr_status_t s = check_salience(a, false);
  if (s != DOPR_OK) return s;
  if (a->n_docs == 0 || !a->selected) return ok();
  hipError_t e = launch_topk(topk_params(a), a->n_docs, as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "top-k launch");
  return ok();
}

dopr_status_t dopr_check_status(dopr_store_t st, void *stream) {
  if (!st) return fail(DOPR_ERR_INVALID_ARG, "store is NULL");
  hipStream_t hs = as_stream(stream);
  int32_t code = 0;
  hipError_t e = hipStreamSynchronize(hs);
  if (e == hipSuccess)
    e = hipMemcpy(&code, st->d_status + kStatusFirstError, sizeof(code),
                  hipMemcpyDeviceToHost);
  const int32_t zero = 0;
  if (e == hipSuccess)
    e = hipMemcpy(st->d_status + kStatusFirstError, &zero, sizeof(zero),
                  hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "status readback");
  if (code != 0)
    return fail((dopr_status_t)code, "deferred device-side error");
  return ok();
}

}  // extern "C"

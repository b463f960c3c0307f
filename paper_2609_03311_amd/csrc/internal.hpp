// internal.hpp -- shared declarations of the DoPR HIP library (not part of
// the public ABI; the public contract is include/dopr.h).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "dopr.h"

namespace dopr {

// Head sizes: 128 (Qwen3, Llama 3) and 64 (Llama 3.2 1B).  Everything sized
// for the largest uses kHeadDim; per-call code takes the store's head_dim.
constexpr int kHeadDim = 128;
constexpr int kAlign = 256;
// Longest prefix for which last-layer scoring runs one wave per 32-row work
// unit (the kernel variant and the planner's item size both follow it).
constexpr int32_t kScoreRowsMaxLen = 512;

// The attention's reference-free softmax serves a work unit when every
// logit (log2 units) lies in [-kNoRefBound, kNoRefBound].
constexpr float kNoRefBound = 64.f;

// Largest attention plan dopr_prefix_attn_noalloc lays out in the library's
// own scratch array (one copy per device).
constexpr size_t kNoAllocScratchBytes = DOPR_NOALLOC_SCRATCH_BYTES;

// Longest prefix for which the automatic choice at head size 128 runs two
// 4-wave blocks per CU (96 slots resident each) instead of the pass kernel.
constexpr int32_t kShortPrefix128 = 96;

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
__host__ __device__ inline int32_t pad8(int32_t n) { return (n + 7) & ~7; }

// Device status words at the head of every store pool.
enum StatusSlot { kStatusFirstError = 0, kStatusWords = 64 };

// Store layout inside the caller's pool:
//   [status words | doc_len int32[n_docs] | doc_off int64[n_docs] |
//    kmax fp32[n_docs][n_layers][Hkv] | payload]
// kmax holds an upper bound on the L2 norm of every stored key of a
// document's (layer, kv head) slice (0 when L = 0); the attention kernel uses
// it to bound logits.
// Each resident document owns one contiguous block of the payload; for layer
// l and kv head g the block holds
//   K  [L][D]   at  blk + l*Hkv*D*(L+Lp) + g*L*D
//   Vt [D][Lp]  at  blk + l*Hkv*D*(L+Lp) + Hkv*L*D + g*D*Lp
// with Lp = L rounded up to 8 (V is stored transposed so the PV contraction
// over keys reads 16-byte runs; the pad columns are zero).
struct StoreView {
  const int32_t *doc_len;  // [n_docs], -1 = not resident
  const int64_t *doc_off;  // [n_docs], element offset of the doc block
  float *kmax;             // [n_docs][n_layers][Hkv] key-norm bound
  uint16_t *payload;
  int64_t n_docs;
  int32_t n_layers, n_kv_heads, head_dim;
};

__host__ __device__ inline int64_t layer_block_elems(int32_t L, int32_t hkv,
                                                     int32_t D) {
  return (int64_t)hkv * D * ((int64_t)L + pad8(L));
}
__host__ __device__ inline int64_t k_offset(int64_t blk, int32_t L, int32_t hkv,
                                            int32_t layer, int32_t g,
                                            int32_t D) {
  return blk + layer * layer_block_elems(L, hkv, D) + (int64_t)g * L * D;
}
__host__ __device__ inline int64_t vt_offset(int64_t blk, int32_t L,
                                             int32_t hkv, int32_t layer,
                                             int32_t g, int32_t D) {
  return blk + layer * layer_block_elems(L, hkv, D) + (int64_t)hkv * L * D +
         (int64_t)g * D * pad8(L);
}

}  // namespace dopr

struct dopr_store {
  int32_t n_layers, n_kv_heads, head_dim;
  int64_t n_docs;
  char *pool;
  size_t pool_bytes;
  int32_t *d_status;
  int32_t *d_len;
  int64_t *d_off;
  float *d_kmax;
  uint16_t *d_payload;
  int32_t max_len;  // largest L over resident documents
  int device;
  dopr::StoreView view() const {
    return {d_len, d_off, d_kmax, d_payload, n_docs, n_layers, n_kv_heads,
            head_dim};
  }
};

namespace dopr {

// ---------------------------------------------------------------------------
// Groups with more pairs than this are put in pair order by a sort (one
// block per group) instead of a scan of the group per pair.
constexpr int32_t kBigGroup = 256;
// Cost classes of work units for the longest-first order: floor(log2) of
// stacked rows x (prefix slots + 32).
constexpr int32_t kCostBuckets = 40;

// The plan's int64 totals.
enum Total {
  kTotDocs = 0,   // (distinct docs << 32) | valid pairs
  kTotRows = 1,   // stacked rows of the valid pairs
  kTotItems = 2,  // work items
  kTotUnits = 3,  // 1 if the queues follow the longest-first order, else 0
  kTotals = 4
};

// Work unit handed out as the `slot`-th claim of queue `queue` (0..7):
// queue q serves the units w with w % 8 == q, in natural order (w = q +
// 8 * slot) when qorder is null, else costliest class first as the
// planner's qorder lists them; n_work when the queue is empty.
__device__ __forceinline__ int64_t unit_at(const int32_t *qorder, int queue,
                                           int64_t slot, int64_t n_work) {
  if (!qorder) {
    const int64_t w = queue + 8 * slot;
    return w < n_work ? w : n_work;
  }
  const int64_t per = n_work / 8, rem = n_work % 8;
  const int64_t n_q = per + (queue < rem ? 1 : 0);
  if (slot >= n_q) return n_work;
  const int64_t start = queue * per + (queue < rem ? queue : rem);
  return qorder[start + slot];
}

// The same in 32 bits: argument validation keeps every unit number (and
// n_work) below 2^31.
__device__ __forceinline__ int unit_at32(const int32_t *qorder, int queue,
                                         int slot, int n_work) {
  if (!qorder) {
    // slot >= the queue's unit count, tested without forming q + 8 * slot
    if (slot >= (n_work - queue + 7) / 8) return n_work;
    return queue + 8 * slot;
  }
  const int per = n_work / 8, rem = n_work % 8;
  const int n_q = per + (queue < rem ? 1 : 0);
  if (slot >= n_q) return n_work;
  const int start = queue * per + (queue < rem ? queue : rem);
  return qorder[start + slot];
}

// Per-call plan built on the device by the grouping kernels (workspace).
enum Counter {
  kCntValid = 0,     // pairs with a valid, resident document
  kCntGroups = 1,    // distinct documents among them
  kCntItems = 2,     // attention work items
  kCntInvalid = 3,   // pairs whose outputs must be zeroed
  kCntRows = 4,      // stacked rows (tokens * n_rep) of valid pairs (low)
  kCntFix = 5,       // work units queued for the exact (SAFE) pass
  kCntBig = 6,       // groups of more than kBigGroup pairs (ordered apart)
  kCounters = 16
};

struct Plan {
  int32_t *counters;    // [kCounters]
  int32_t *cnt;         // [n_docs]   pairs per document
  int32_t *fill;        // [n_docs]   placement cursor per document
  int64_t *doc_scan;    // [n_docs]   (has_pairs << 32 | count), scanned
  int64_t *blk;         // scan block sums
  int32_t *pair_flag;   // [P] 1 = valid, 0 = skip, 2 = zero outputs
  int32_t *invalid;     // [P] pairs whose outputs are zeroed
  int32_t *tmp_order;   // [P]
  int32_t *pair_order;  // [P]
  int4 *big;            // [P / (kBigGroup + 1) + 1] groups of more than
                        // kBigGroup pairs: (first slot, pairs, doc, group)
  int32_t *qorder;      // [items_cap * Hkv] work units by queue (w % 8),
                        // costliest class first within each queue, unit
                        // order within a class (when totals[kTotUnits]
                        // is 1)
  uint8_t *item_cls;    // [items_cap] cost class of each item's group
  int32_t *group_doc;   // [P]
  int32_t *group_ptr;   // [P+1]
  int64_t *prow;        // [P+1] stacked-row offsets, sorted pair order
  int64_t *item_scan;   // [P+1] work items per group, scanned
  int32_t *blk_pair;    // [blk_cap] sorted pair owning row 32*b
  int4 *items;          // [items_cap] (group, row0, row1, first sorted pair)
  int32_t *fix;         // [items_cap * Hkv] work units for the SAFE pass
  int4 *spair;          // [P+1] sorted pair: (tok0, T, first stacked row)
  int2 *utok;           // [stacked tokens] (batch token, position)
  float *part;          // [P][Hq][3] score-head partial sums (score mode)
  float *kown;          // [2] bounds on |k^| (own keys) and |q^|: sqrt(D) max|w|
                        // (0 when there is no QK-norm: no bound is known)
  uint16_t *unit_w;     // [D] bf16 ones: the gains when there is no QK-norm
  float2 *rope;         // [rope_pos][D/2] (cos, sin)
  uint16_t *kh;         // [Hkv][Ntok][D] own keys k^ (pass kernel), or NULL
  int4 *units;          // [items_cap * Hkv][2] work units (pass kernel):
                        // (row0, row1, first pair, L or -1 when over the
                        // logit bound), (K offset lo, hi, V^T offset lo, hi)
  uint16_t *zero;       // 256 zero bytes (streaming kernel loads past row ends)
  int32_t items_cap;
  int32_t blk_cap;
  int32_t rope_pos;
  int64_t scan_blocks_cap;
};

// score_only: one stacked token per pair (its score token, the last one)
// instead of all T_p.
struct PlanShape {
  int32_t n_pairs, n_rep, max_tokens, rows_per_item;
  int64_t n_docs, total_tokens;
  int32_t max_len, n_kv_heads;
  int32_t head_dim = kHeadDim;
  bool score_only = false;
  bool stream = false;  // the pass kernel runs: room for k^ of every token
                        // and the work-unit table
};

size_t plan_bytes(const PlanShape &s);
Plan plan_carve(void *ws, const PlanShape &s);

// Launchers (return hipError_t of the last launch).
hipError_t launch_store_put(const dopr_store &st, int32_t layer, int64_t n,
                            const int32_t *doc_ids, const int64_t *src_cu,
                            const uint16_t *k, const uint16_t *v,
                            hipStream_t s);
hipError_t launch_gather(const dopr_store &st, int32_t layer, int32_t n,
                         const int32_t *doc_ids, const int64_t *out_cu,
                         uint16_t *k, uint16_t *v, hipStream_t s);
hipError_t launch_store_copy(const dopr_store &dst, const dopr_store &src,
                             hipStream_t s);

struct AttnCall {
  const dopr_store *st;
  int32_t layer;
  const dopr_attn_args_t *a;
  int32_t n_rep;
  const dopr_score_head_t *head = nullptr;  // score mode (last layer)
};
hipError_t launch_plan(const AttnCall &c, const Plan &plan,
                       const PlanShape &shape, hipStream_t s);
hipError_t launch_attention(const AttnCall &c, const Plan &plan,
                            const PlanShape &shape, hipStream_t s);
hipError_t launch_score(const dopr_score_args_t *a, hipStream_t s);
// width: the score head's input width, n_q_heads * head_dim.
hipError_t launch_score_reduce(const Plan &pl, int32_t n_pairs, int32_t n_q_heads,
                               int32_t width, const dopr_score_head_t *head,
                               hipStream_t s);

// ---------------------------------------------------------------------------
// Decoder layer around the attention (layer.hip).
constexpr int64_t kMlpChunk = 32768;               // MLP tokens per chunk
constexpr size_t kGemmWorkspace = size_t(64) << 20;  // hipBLASLt workspace

struct LayerShape {
  int64_t ntok;
  int32_t hidden, inter, hq, hkv;
};

struct LayerWs {
  uint16_t *h;    // [Ntok][W]   RMSNorm(x), later RMSNorm(x2)
  uint16_t *q;    // [Ntok][Hq][D]
  uint16_t *k;    // [Ntok][Hkv][D]
  uint16_t *v;    // [Ntok][Hkv][D]
  uint16_t *att;  // [Ntok][Hq][D] attention rows
  uint16_t *gu;   // [chunk][2I]  gate | up
  uint16_t *act;  // [chunk][I]   SiLU(gate) * up
  void *gemm_ws;
  size_t gemm_ws_bytes;
  int64_t chunk;
  void *plan;     // the attention plan follows the layer's buffers
  size_t bytes;   // layer buffers before the plan
};

LayerWs layer_carve(void *base, const LayerShape &s);
// Return 0, -1 for a HIP launch error, or a hipBLASLt status.
int launch_layer_pre(const LayerShape &s, const dopr_layer_args_t *l,
                     const LayerWs &w, float eps, hipStream_t st);
int launch_layer_post(const LayerShape &s, const dopr_layer_args_t *l,
                      const LayerWs &w, float eps, hipStream_t st);
const char *gemm_status_str(int s);

// Offline salience selection (salience.hip).
constexpr int kSalienceMaxLen = 4096;   // longest document (LDS sort bound)
constexpr int kSalienceMaxP = 64;       // largest top-p (register list bound)
constexpr size_t kSalienceAbarBudget = size_t(1) << 30;  // scratch bytes

struct SalienceParams {
  const uint16_t *q, *k;     // [Ntok, Hq, D], [Ntok, Hkv, D]
  const int32_t *cu;         // [n_docs + 1]
  int32_t n_docs, d0;        // all docs; first doc of this launch
  int32_t hq, hkv, n_rep, max_len, top_p;
  int64_t total_tokens;
  float c;                   // softmax_scale * log2(e)
  float inv_hq;
  float *lse2;               // [Hq][Ntok] log2-domain row log-sum-exp
  float *kmax;               // [n_docs][Hkv][kKeyNormParts] partial maxima
                             // of the key norms per document
  float *abar;               // doc d - d0 at (d - d0) * abar_stride
  int64_t abar_stride;       // max_len * max_len
  float *u;                  // [Ntok]
  int32_t *status;           // deferred error word, or NULL
};

struct TopkParams {
  const int32_t *cu, *cs;    // [n_docs + 1] token and selection offsets
  const float *u;
  int32_t *selected;
  int32_t max_len;
  int64_t total_tokens, total_select;
  int32_t *status;
};

hipError_t launch_salience_check(const SalienceParams &p, hipStream_t s);
hipError_t launch_key_norms(const SalienceParams &p, hipStream_t s);
constexpr int kKeyNormParts = 8;  // partial maxima per (document, kv head)
hipError_t launch_salience_chunk(const SalienceParams &p, int32_t n_docs,
                                 int hr, int pm, hipStream_t s);
hipError_t launch_topk(const TopkParams &p, int32_t n_docs, hipStream_t s);

// Record a deferred error code in a status word (first error wins).
__device__ inline void raise_status(int32_t *status, int32_t code) {
  atomicCAS(status, 0, code);
}

}  // namespace dopr

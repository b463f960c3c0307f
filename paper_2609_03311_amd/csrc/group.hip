// group.hip -- per-batch scheduling of the online attention (integer work).
//
// Online, every candidate pair retrieves its document's prefix states
// (Sec. 3.4).  Pairs that name the same document are grouped so that one
// workgroup serves all of them and the document's prefix is read once per
// group: this is the paper's cross-query reuse of a document's prefix
// (Sec. 3.3, Sec. 4.5.2) applied inside one batch.  Everything here runs on
// the device with no host synchronisation:
//   1. validate each pair (doc id range/residency, token range) and count
//      pairs per document;
//   2. exclusive scan over the doc-id space -> first slot and group index
//      of every document (a counting sort: groups come out in ascending doc
//      id, the canonical order);
//   3. place pairs into their document's slots, then order each group's
//      members by pair index (stable, deterministic);
//   4. stacked-row offsets (T_p * n_rep rows per pair, in grouped order;
//      n_rep rows -- the score token's -- in score mode);
//   5. split each group's rows into work items of bounded size, and a
//      table from every 32-row block to the pair owning its first row;
//   6. the rotary cos/sin table for positions 0 .. max_L + max_tokens - 1.
#include <cmath>

#include "internal.hpp"

namespace dopr {
namespace {

constexpr int kScanThreads = 1024;
constexpr int kScanTile = 2 * kScanThreads;
constexpr int kThreads = 256;

enum NextSlots { kNextQueues = 16 };  // 8 XCD queues + the SAFE pass

inline unsigned blocks_for(int64_t n, int t) {
  int64_t b = (n + t - 1) / t;
  return (unsigned)(b < 1 ? 1 : b);
}

// Exclusive block-wide scan of two values per thread (1024 threads).
// Returns the prefix of the thread's first value; *block_total gets the sum.
__device__ int64_t block_scan2(int64_t a0, int64_t a1, int64_t *block_total) {
  __shared__ int64_t wsum[kScanThreads / 64 + 1];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int64_t t = a0 + a1;
  int64_t x = t;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int64_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) wsum[wid] = x;
  __syncthreads();
  if (wid == 0) {
    constexpr int nw = kScanThreads / 64;
    int64_t w = lane < nw ? wsum[lane] : 0;
    int64_t s = w;
#pragma unroll
    for (int off = 1; off < nw; off <<= 1) {
      int64_t y = __shfl_up(s, off, 64);
      if (lane >= off) s += y;
    }
    if (lane < nw) wsum[lane] = s - w;
    if (lane == nw - 1) wsum[nw] = s;
  }
  __syncthreads();
  const int64_t prefix = wsum[wid] + x - t;
  *block_total = wsum[kScanThreads / 64];
  __syncthreads();
  return prefix;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(
    const int64_t *data, int64_t n, int64_t *blk) {
  const int64_t i0 = (int64_t)blockIdx.x * kScanTile + 2 * threadIdx.x;
  const int64_t a0 = i0 < n ? data[i0] : 0;
  const int64_t a1 = i0 + 1 < n ? data[i0 + 1] : 0;
  int64_t tot;
  block_scan2(a0, a1, &tot);
  if (threadIdx.x == 0) blk[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_top(int64_t *blk,
                                                           int64_t nb,
                                                           int64_t *total) {
  int64_t carry = 0;
  for (int64_t base = 0; base < nb; base += kScanTile) {
    const int64_t i0 = base + 2 * threadIdx.x;
    const int64_t a0 = i0 < nb ? blk[i0] : 0;
    const int64_t a1 = i0 + 1 < nb ? blk[i0 + 1] : 0;
    int64_t tot;
    const int64_t pre = block_scan2(a0, a1, &tot);
    if (i0 < nb) blk[i0] = carry + pre;
    if (i0 + 1 < nb) blk[i0 + 1] = carry + pre + a0;
    carry += tot;
  }
  if (threadIdx.x == 0) *total = carry;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_apply(
    int64_t *data, int64_t n, const int64_t *blk) {
  const int64_t i0 = (int64_t)blockIdx.x * kScanTile + 2 * threadIdx.x;
  const int64_t a0 = i0 < n ? data[i0] : 0;
  const int64_t a1 = i0 + 1 < n ? data[i0 + 1] : 0;
  int64_t tot;
  const int64_t pre = block_scan2(a0, a1, &tot) + blk[blockIdx.x];
  if (i0 < n) data[i0] = pre;
  if (i0 + 1 < n) data[i0 + 1] = pre + a0;
}

// Arrays up to this many values are scanned by one block walking them tile
// by tile (k_scan_top on the data itself): one launch instead of three.
constexpr int64_t kScanOneBlock = 8 * kScanTile;

// In-place exclusive scan of n int64 values; the grand total goes to *total.
hipError_t exclusive_scan(int64_t *data, int64_t n, int64_t *blk,
                          int64_t *total, hipStream_t s) {
  if (n <= kScanOneBlock) {
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kScanThreads), 0, s, data,
                       n, total);
    return hipGetLastError();
  }
  const unsigned nb = blocks_for(n, kScanTile);
  hipLaunchKernelGGL(k_scan_reduce, dim3(nb), dim3(kScanThreads), 0, s, data,
                     n, blk);
  hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kScanThreads), 0, s, blk,
                     (int64_t)nb, total);
  hipLaunchKernelGGL(k_scan_apply, dim3(nb), dim3(kScanThreads), 0, s, data,
                     n, blk);
  return hipGetLastError();
}

struct PlanArgs {
  const int32_t *doc_ids, *cu, *doc_len;
  int64_t n_docs, total_tokens;
  int32_t n_pairs, n_rep, max_tokens, rows_per_item;
  int32_t *status;
  bool score_only;
  bool exact_items;
};

__global__ __launch_bounds__(kThreads) void k_plan_init(Plan pl, int64_t n_docs,
                                                        int64_t *totals,
                                                        int32_t *next) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n_docs) {
    pl.cnt[i] = 0;
    pl.fill[i] = 0;
  }
  if (i < kCounters) pl.counters[i] = 0;
  if (i < 64) reinterpret_cast<int32_t *>(pl.zero)[i] = 0;
  if (i < kTotals) totals[i] = 0;
  if (i < kNextQueues) next[i] = 0;
}

// Step 1: validate every pair and count pairs per document.
__global__ __launch_bounds__(kThreads) void k_pair_meta(Plan pl, PlanArgs a) {
  const int32_t p = blockIdx.x * kThreads + threadIdx.x;
  if (p >= a.n_pairs) return;
  if (a.cu) {  // grouping-only calls pass no token ranges
    if (p == 0 && a.cu[0] != 0) raise_status(a.status, DOPR_ERR_SEQLEN);
    if (p == a.n_pairs - 1 && (int64_t)a.cu[a.n_pairs] != a.total_tokens)
      raise_status(a.status, DOPR_ERR_SEQLEN);
    const int64_t t0 = a.cu[p], t1 = a.cu[p + 1];
    const bool well = t0 >= 0 && t1 >= t0 + 1 && t1 <= a.total_tokens &&
                      t1 - t0 <= a.max_tokens;
    if (!well) {
      raise_status(a.status, DOPR_ERR_SEQLEN);
      pl.pair_flag[p] = 0;
      return;
    }
  }
  const int32_t d = a.doc_ids[p];
  if (d < 0 || (int64_t)d >= a.n_docs || a.doc_len[d] < 0) {
    raise_status(a.status, DOPR_ERR_DOC_RANGE);
    pl.pair_flag[p] = 2;
    pl.invalid[atomicAdd(&pl.counters[kCntInvalid], 1)] = p;
    return;
  }
  pl.pair_flag[p] = 1;
  atomicAdd(&pl.cnt[d], 1);
}

__global__ __launch_bounds__(kThreads) void k_doc_pack(Plan pl, int64_t n_docs) {
  const int64_t d = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (d >= n_docs) return;
  const int32_t c = pl.cnt[d];
  pl.doc_scan[d] = c > 0 ? ((int64_t)1 << 32) | (int64_t)c : 0;
}

// Step 3a: each valid pair takes a slot in its document's range (arbitrary
// order within the range; fixed by k_rank).
__global__ __launch_bounds__(kThreads) void k_place(Plan pl, PlanArgs a) {
  const int32_t p = blockIdx.x * kThreads + threadIdx.x;
  if (p >= a.n_pairs || pl.pair_flag[p] != 1) return;
  const int32_t d = a.doc_ids[p];
  const int32_t slot = (int32_t)(pl.doc_scan[d] & 0xffffffff) +
                       atomicAdd(&pl.fill[d], 1);
  pl.tmp_order[slot] = p;
}

// Step 3b + 4: rank each pair within its group by pair index, write the
// canonical order, the group table and the pair's stacked-row count.
__global__ __launch_bounds__(kThreads) void k_rank(Plan pl, PlanArgs a,
                                                   const int64_t *totals) {
  const int32_t i = blockIdx.x * kThreads + threadIdx.x;
  const int32_t n_valid = (int32_t)(totals[kTotDocs] & 0xffffffff);
  const int32_t n_groups = (int32_t)(totals[kTotDocs] >> 32);
  if (i > a.n_pairs) return;
  if (i >= n_valid) {
    pl.prow[i] = 0;
    if (i == n_valid) pl.group_ptr[n_groups] = n_valid;
    return;
  }
  const int32_t v = pl.tmp_order[i];
  const int32_t d = a.doc_ids[v];
  const int64_t packed = pl.doc_scan[d];
  const int32_t s0 = (int32_t)(packed & 0xffffffff);
  const int32_t c = pl.cnt[d];
  if (c > kBigGroup) {
    // ordered by k_rank_big instead (a scan per pair would cost c^2)
    if (i == s0)
      pl.big[atomicAdd(&pl.counters[kCntBig], 1)] =
          make_int4(s0, c, d, (int32_t)(packed >> 32));
    return;
  }
  int32_t rank = 0;
  for (int32_t k = s0; k < s0 + c; ++k) rank += pl.tmp_order[k] < v;
  pl.pair_order[s0 + rank] = v;
  const int64_t T = a.cu && !a.score_only ? (int64_t)(a.cu[v + 1] - a.cu[v])
                                           : 1;
  pl.prow[s0 + rank] = T * a.n_rep;
  if (rank == 0) {
    const int32_t gi = (int32_t)(packed >> 32);
    pl.group_doc[gi] = d;
    pl.group_ptr[gi] = s0;
  }
}

// Step 3b for groups of more than kBigGroup pairs, one block per group: the
// group's slots are sorted by pair index in LDS in tiles of kSortTile
// (bitonic), and a pair's rank is its index in its tile plus the number of
// smaller pair indices in each other tile (binary search; pair indices are
// distinct).  Writes the canonical order, the stacked-row counts and the
// group table, as k_rank does for the others.
constexpr int32_t kSortTile = 16384;

__global__ __launch_bounds__(1024) void k_rank_big(Plan pl, PlanArgs a) {
  __shared__ int32_t key[kSortTile];
  const int32_t nb = pl.counters[kCntBig];
  for (int32_t b = blockIdx.x; b < nb; b += gridDim.x) {
    const int4 g = pl.big[b];
    const int32_t s0 = g.x, c = g.y;
    if (threadIdx.x == 0) {
      pl.group_doc[g.w] = g.z;
      pl.group_ptr[g.w] = s0;
    }
    const int32_t n_tiles = (c + kSortTile - 1) / kSortTile;
    for (int32_t k = 0; k < n_tiles; ++k) {
      const int32_t base = s0 + k * kSortTile;
      const int32_t n = c - k * kSortTile < kSortTile ? c - k * kSortTile
                                                      : kSortTile;
      int32_t N = 1;
      while (N < n) N <<= 1;
      __syncthreads();  // the previous tile's writes are done
      for (int32_t t = threadIdx.x; t < N; t += blockDim.x)
        key[t] = t < n ? pl.tmp_order[base + t] : INT32_MAX;
      __syncthreads();
      for (int32_t size = 2; size <= N; size <<= 1)
        for (int32_t stride = size >> 1; stride > 0; stride >>= 1) {
          for (int32_t t = threadIdx.x; t < N / 2; t += blockDim.x) {
            const int32_t lo = 2 * t - (t & (stride - 1));
            const int32_t hi = lo + stride;
            const bool up = (lo & size) == 0;
            const int32_t x = key[lo], y = key[hi];
            if ((x > y) == up) {
              key[lo] = y;
              key[hi] = x;
            }
          }
          __syncthreads();
        }
      for (int32_t t = threadIdx.x; t < n; t += blockDim.x)
        pl.tmp_order[base + t] = key[t];
    }
    __syncthreads();  // every sorted tile is visible to the block
    for (int32_t e = threadIdx.x; e < c; e += blockDim.x) {
      const int32_t k = e / kSortTile;
      const int32_t v = pl.tmp_order[s0 + e];
      int32_t rank = e - k * kSortTile;
      for (int32_t k2 = 0; k2 < n_tiles; ++k2) {
        if (k2 == k) continue;
        int32_t lo = s0 + k2 * kSortTile;
        int32_t hi = lo + (c - k2 * kSortTile < kSortTile ? c - k2 * kSortTile
                                                          : kSortTile);
        const int32_t start = lo;
        while (lo < hi) {  // first slot not below v
          const int32_t mid = (lo + hi) >> 1;
          if (pl.tmp_order[mid] < v) lo = mid + 1; else hi = mid;
        }
        rank += lo - start;
      }
      pl.pair_order[s0 + rank] = v;
      const int64_t T = a.cu && !a.score_only
                            ? (int64_t)(a.cu[v + 1] - a.cu[v])
                            : 1;
      pl.prow[s0 + rank] = T * a.n_rep;
    }
  }
}

// Step 5a: work items per group.
__global__ __launch_bounds__(kThreads) void k_items_count(Plan pl, PlanArgs a,
                                                          const int64_t *totals) {
  const int32_t g = blockIdx.x * kThreads + threadIdx.x;
  const int32_t n_groups = (int32_t)(totals[kTotDocs] >> 32);
  if (g > a.n_pairs) return;
  if (g >= n_groups) {
    pl.item_scan[g] = 0;
    return;
  }
  const int64_t rows = pl.prow[pl.group_ptr[g + 1]] - pl.prow[pl.group_ptr[g]];
  pl.item_scan[g] = (rows + a.rows_per_item - 1) / a.rows_per_item;
}

// The longest-first cost class of a document group: kCostBuckets - 1 -
// floor(log2(stacked rows * (prefix slots + 32))), clamped to the buckets
// (0 = costliest).
__device__ __forceinline__ uint8_t cost_class(int64_t rows, int32_t L) {
  const int64_t cost = rows * ((int64_t)L + 32);
  const int b = cost > 0 ? 63 - __clzll((unsigned long long)cost) : 0;
  return (uint8_t)(kCostBuckets - 1 - (b < kCostBuckets ? b : kCostBuckets - 1));
}

// Step 5b: split a group's rows into items, boundaries on multiples of 32
// rows: near-equal items (the block kernels, which walk an item in passes),
// or, with exact_items, items of exactly rows_per_item rows and a shorter
// last one (the streaming kernel serves an item in one pass, so no item
// may exceed it).  One wave per group, its lanes taking the items in turn:
// a hot document's group has hundreds of items, each with its own search.
// The waves stride over the groups, so the grid stays bounded.
__global__ __launch_bounds__(kThreads) void k_items_emit(Plan pl, PlanArgs a,
                                                         const int64_t *totals) {
  const int64_t wave0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * kThreads) >> 6;
  const int lane = threadIdx.x & 63;
  const int32_t n_groups = (int32_t)(totals[kTotDocs] >> 32);
  if (wave0 == 0 && lane == 0 && totals[kTotItems] > pl.items_cap)
    raise_status(a.status, DOPR_ERR_SEQLEN);
  for (int64_t gw = wave0; gw < n_groups; gw += n_waves) {
    const int32_t g = (int32_t)gw;
    const int64_t first = pl.item_scan[g];
    const int64_t n_it = pl.item_scan[g + 1] - first;
    const int64_t base = pl.prow[pl.group_ptr[g]];
    const int64_t R = pl.prow[pl.group_ptr[g + 1]] - base;
    const uint8_t cls = cost_class(R, a.doc_len[pl.group_doc[g]]);
    for (int64_t it = lane; it < n_it; it += 64) {
      const int64_t idx = first + it;
      if (idx >= pl.items_cap) break;
      pl.item_cls[idx] = cls;
      const int64_t b0 =
          a.exact_items ? base + it * a.rows_per_item
                        : base + ((it * R / n_it) & ~(int64_t)31);
      const int64_t b1 =
          it + 1 < n_it
              ? (a.exact_items ? base + (it + 1) * a.rows_per_item
                               : base + (((it + 1) * R / n_it) & ~(int64_t)31))
              : base + R;
      // the item's first sorted pair: the last of the group's pairs whose
      // stacked rows start at or before b0
      int32_t lo = pl.group_ptr[g], hi = pl.group_ptr[g + 1] - 1;
      while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (pl.prow[mid] <= b0) lo = mid; else hi = mid - 1;
      }
      pl.items[idx] = make_int4(g, (int32_t)b0, (int32_t)b1, lo);
    }
  }
}

// Step 5c: owner of the first row of every 32-row block, so a row finds
// its pair with one lookup and a short forward scan.
__global__ __launch_bounds__(kThreads) void k_blk_pair(Plan pl,
                                                       const int64_t *totals) {
  const int32_t s = blockIdx.x * kThreads + threadIdx.x;
  const int32_t n_valid = (int32_t)(totals[kTotDocs] & 0xffffffff);
  if (s >= n_valid) return;
  int64_t b0 = (pl.prow[s] + 31) >> 5, b1 = (pl.prow[s + 1] + 31) >> 5;
  if (b1 > pl.blk_cap) b1 = pl.blk_cap;
  for (int64_t b = b0; b < b1; ++b) pl.blk_pair[b] = s;
}

// Step 5d: per sorted pair (first token, token count, first stacked row),
// with a sentinel row count after the last pair, and per stacked token u
// (token-major: u = stacked row / n_rep) its (batch token, position in
// pair), positions descending within a pair (score mode: the last token
// only, so u is the sorted pair index).  One workgroup per sorted pair.
__global__ __launch_bounds__(kThreads) void k_token_table(Plan pl, PlanArgs a,
                                                          const int64_t *totals) {
  const int32_t s = blockIdx.x;
  const int32_t n_valid = (int32_t)(totals[kTotDocs] & 0xffffffff);
  if (s > n_valid) return;
  if (s == n_valid) {
    if (threadIdx.x == 0)
      pl.spair[s] = make_int4(0, 0, (int32_t)totals[kTotRows], 0);
    return;
  }
  const int32_t pr = pl.pair_order[s];
  const int32_t tok0 = a.cu[pr], T = a.cu[pr + 1] - tok0;
  const int64_t r0 = pl.prow[s];
  if (threadIdx.x == 0) pl.spair[s] = make_int4(tok0, T, (int32_t)r0, 0);
  // A pair's tokens are stacked last position first: the first pass over
  // the pair then holds its latest tokens (which see every own key) and the
  // short final pass of an item its earliest ones (which see few).
  const int64_t u0 = r0 / a.n_rep;
  const int32_t stacked = a.score_only ? 1 : T;
  for (int32_t j = threadIdx.x; j < stacked; j += kThreads)
    pl.utok[u0 + j] = make_int2(tok0 + (T - 1 - j), T - 1 - j);
}

// Bounds on the norms of every own key k^ and every query q^, each of the
// form RoPE(RMSNorm(x) * w): an RMS-normed vector has norm <= sqrt(D), the
// gain scales it by at most max|w|, rotation keeps it, and bf16 rounding
// adds at most 2^-8.  bound[0] is for keys (w_k), bound[1] for queries.
// Without QK-norm (no gains) no bound is known: both are written as 0 and
// unit_w gets the unit gains the attention kernel multiplies by.  One
// thread per head dim (blockDim.x = D, 64 or 128).
__global__ __launch_bounds__(128) void k_norm_bound(const uint16_t *kw,
                                                    const uint16_t *qw,
                                                    float *bound,
                                                    uint16_t *unit_w) {
  __shared__ float red[2][2];
  if (!kw) unit_w[threadIdx.x] = 0x3F80;  // bf16 1.0
  float a = 0.f, b = 0.f;
  if (kw) a = fabsf(__uint_as_float((uint32_t)kw[threadIdx.x] << 16));
  if (qw) b = fabsf(__uint_as_float((uint32_t)qw[threadIdx.x] << 16));
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a = fmaxf(a, __shfl_xor(a, off, 64));
    b = fmaxf(b, __shfl_xor(b, off, 64));
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = a;
    red[1][threadIdx.x >> 6] = b;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    const float m = blockDim.x > 64
                        ? fmaxf(red[threadIdx.x][0], red[threadIdx.x][1])
                        : red[threadIdx.x][0];
    bound[threadIdx.x] = m * sqrtf((float)blockDim.x) * 1.01f;
  }
}

// Work units of the pass kernel, one per (item, kv head): the item's rows
// and first pair, the document's prefix length and the element offsets of
// its K and V^T slices for this layer and head; a unit whose logits the
// norm bounds cannot keep within the reference-free range (the kernels'
// kNoRefBound) is marked with L = -1 and left to the exact pass.
__global__ __launch_bounds__(kThreads) void k_unit_table(
    Plan pl, StoreView sv, int32_t layer, float c, float no_ref_bound,
    const int64_t *totals) {
  const int64_t w = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t n_items = totals[kTotItems] < pl.items_cap
                              ? totals[kTotItems]
                              : pl.items_cap;
  if (w >= n_items * sv.n_kv_heads) return;
  const int32_t item = (int32_t)(w / sv.n_kv_heads);
  const int32_t g = (int32_t)(w % sv.n_kv_heads);
  const int4 it = pl.items[item];
  const int32_t doc = pl.group_doc[it.x];
  const int32_t L = sv.doc_len[doc];
  const int64_t blk = sv.doc_off[doc];
  const float kb = fmaxf(
      pl.kown[0],
      sv.kmax[((int64_t)doc * sv.n_layers + layer) * sv.n_kv_heads + g]);
  const bool over = c * pl.kown[1] * kb * 1.001f > no_ref_bound;
  const int64_t ko = k_offset(blk, L, sv.n_kv_heads, layer, g, sv.head_dim);
  const int64_t vo = vt_offset(blk, L, sv.n_kv_heads, layer, g, sv.head_dim);
  pl.units[2 * w] = make_int4(it.y, it.z, it.w, over ? -1 : L);
  pl.units[2 * w + 1] = make_int4((int32_t)(uint32_t)ko, (int32_t)(ko >> 32),
                                  (int32_t)(uint32_t)vo, (int32_t)(vo >> 32));
}

// Step 5f: the longest-first order of the work-unit queues.  Unit w =
// item * Hkv + kv head goes to queue w % 8, which the blocks b with
// b % 8 == queue serve; blocks are dealt round-robin to the 8 XCDs, so with
// 8 kv heads each head's prefix K/V is read through one XCD's L2.  Within
// a queue, units are handed out by the cost class of their document group
// (floor(log2(group rows * (L + 32)))), costliest first, so long groups
// start early and short ones fill the tail, and in unit order within a
// class: the items of one group stay adjacent and share its prefix in L2,
// and the queues still walk the items in step.  This pays only while the
// CUs get few units each: with many, the blocks' finishing times even out
// by themselves, and the queues keep the natural order (w = queue + 8 *
// slot), which the kernels take when totals[kTotUnits] is 0.
//
// One block of 8 waves sorts stably: wave q takes queue q's units (w = q
// + 8 s), counts them per class in its lanes (lane c holds class c), scans
// the counts into cursors and walks the units again, placing each one at
// its class's cursor; the classes of a 64-unit chunk are grouped with
// ballots, so each step costs a few instructions per distinct class.
constexpr int kOrderWaves = 8;
static_assert(kCostBuckets <= 64, "one lane per cost class");
// Longest-first only while the CUs average at most this many units each.
constexpr int64_t kLptUnitsPerCu = 128;
// Units one sort takes (128 per CU on 256 CUs); beyond it the queues keep
// the natural order.
constexpr int32_t kOrderMaxUnits = 32768;

__global__ __launch_bounds__(kOrderWaves * 64) void k_unit_order(
    Plan pl, int32_t hkv, int64_t lpt_units, int64_t *totals) {
  __shared__ uint8_t cls_s[kOrderMaxUnits];  // item classes
  const int64_t n_items = totals[kTotItems] < pl.items_cap
                              ? totals[kTotItems]
                              : pl.items_cap;
  const int64_t n64 = n_items * hkv;
  const bool ordered = n64 > 0 && n64 <= lpt_units && n64 <= kOrderMaxUnits;
  if (threadIdx.x == 0) totals[kTotUnits] = ordered ? 1 : 0;
  if (!ordered) return;  // block-uniform
  const int n = (int)n64;
  for (int i = threadIdx.x; i < (int)n_items; i += kOrderWaves * 64)
    cls_s[i] = pl.item_cls[i];
  __syncthreads();
  const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
  const uint64_t lt = (1ull << lane) - 1;
  const int per = n / 8, rem = n % 8;
  const int n_q = per + (q < rem ? 1 : 0);
  const int start = q * per + (q < rem ? q : rem);
  // counts per class
  int cnt = 0;
  for (int s0 = 0; s0 < n_q; s0 += 64) {
    const int slot = s0 + lane;
    const int cls = slot < n_q ? cls_s[(q + 8 * slot) / hkv] : -1;
    uint64_t todo = __ballot(cls >= 0);
    while (todo) {  // wave-uniform
      const int k = __builtin_amdgcn_readlane(cls, __builtin_ctzll(todo));
      const uint64_t m = __ballot(cls == k);
      if (lane == k) cnt += __popcll(m);
      todo &= ~m;
    }
  }
  // cursors: start of the queue + the counts of the costlier classes
  int incl = cnt;
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  int cur = start + incl - cnt;
  // placement, in unit order within each class
  for (int s0 = 0; s0 < n_q; s0 += 64) {
    const int slot = s0 + lane;
    const int w = q + 8 * slot;
    const int cls = slot < n_q ? cls_s[w / hkv] : -1;
    uint64_t todo = __ballot(cls >= 0);
    while (todo) {  // wave-uniform
      const int k = __builtin_amdgcn_readlane(cls, __builtin_ctzll(todo));
      const uint64_t m = __ballot(cls == k);
      const int b0 = __builtin_amdgcn_readlane(cur, k);
      if (cls == k) pl.qorder[b0 + __popcll(m & lt)] = w;
      if (lane == k) cur += __popcll(m);
      todo &= ~m;
    }
  }
}

// Step 6: rotary table, (cos, sin)(pos * omega_i) for i < half = D/2, in
// double, stored as float; omega_i = theta^(-2i/D), or the caller's
// inv_freq[i].
__global__ __launch_bounds__(kThreads) void k_rope_table(float2 *tab,
                                                         int32_t n_pos,
                                                         int32_t half,
                                                         double log_theta,
                                                         const float *inv_freq) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= (int64_t)n_pos * half) return;
  const int32_t pos = (int32_t)(e / half), i = (int32_t)(e % half);
  const double freq =
      inv_freq ? (double)inv_freq[i]
               : exp(-(double)i / (double)half * log_theta);
  double sn, cs;
  sincos((double)pos * freq, &sn, &cs);
  tab[e] = make_float2((float)cs, (float)sn);
}

}  // namespace

// ---------------------------------------------------------------------------

namespace {
struct Carver {
  char *base;
  size_t off = 0;
  template <class T>
  T *take(int64_t n) {
    T *p = reinterpret_cast<T *>(base ? base + off : nullptr);
    off = align_up(off + sizeof(T) * (size_t)(n > 0 ? n : 1), kAlign);
    return p;
  }
};

Plan carve(void *ws, const PlanShape &s, size_t *bytes) {
  Carver c{static_cast<char *>(ws)};
  Plan pl{};
  const int64_t P = s.n_pairs;
  pl.counters = c.take<int32_t>(kCounters + kTotals * 2 + kNextQueues);
  pl.cnt = c.take<int32_t>(s.n_docs);
  pl.fill = c.take<int32_t>(s.n_docs);
  pl.doc_scan = c.take<int64_t>(s.n_docs);
  const int64_t stacked = s.score_only ? P : s.total_tokens;
  const int64_t rows = stacked * s.n_rep;
  // (the item capacity; argument validation keeps cap * n_kv_heads < 2^31)
  const int64_t cap = P + (rows + s.rows_per_item - 1) / s.rows_per_item + 1;
  const int64_t hkv = s.n_kv_heads > 0 ? s.n_kv_heads : 1;
  const int64_t scan_n = s.n_docs > P + 1 ? s.n_docs : P + 1;
  pl.scan_blocks_cap = (scan_n + kScanTile - 1) / kScanTile;
  pl.blk = c.take<int64_t>(pl.scan_blocks_cap);
  pl.pair_flag = c.take<int32_t>(P);
  pl.invalid = c.take<int32_t>(P);
  pl.tmp_order = c.take<int32_t>(P);
  pl.pair_order = c.take<int32_t>(P);
  pl.big = c.take<int4>(P / (kBigGroup + 1) + 1);
  pl.group_doc = c.take<int32_t>(P);
  pl.group_ptr = c.take<int32_t>(P + 1);
  pl.prow = c.take<int64_t>(P + 1);
  pl.item_scan = c.take<int64_t>(P + 1);
  pl.items_cap = (int32_t)cap;
  pl.items = c.take<int4>(cap);
  pl.blk_cap = (int32_t)((rows + 31) / 32 + 1);
  pl.blk_pair = c.take<int32_t>(pl.blk_cap);
  pl.fix = c.take<int32_t>(cap * (s.n_kv_heads > 0 ? s.n_kv_heads : 1));
  pl.qorder = c.take<int32_t>(cap * hkv);
  pl.item_cls = c.take<uint8_t>(cap);
  pl.spair = c.take<int4>(P + 1);
  pl.utok = c.take<int2>(stacked);
  pl.part = s.score_only ? c.take<float>(P * s.n_rep * s.n_kv_heads * 3)
                         : nullptr;
  pl.kown = c.take<float>(2);
  pl.unit_w = c.take<uint16_t>(kHeadDim);
  pl.rope_pos = s.max_len + s.max_tokens;
  pl.rope = c.take<float2>((int64_t)pl.rope_pos * (s.head_dim / 2));
  pl.zero = c.take<uint16_t>(128);
  pl.kh = s.stream ? c.take<uint16_t>(s.total_tokens * s.n_kv_heads *
                                      s.head_dim)
                   : nullptr;
  pl.units = s.stream ? c.take<int4>(cap * 2 * (s.n_kv_heads > 0
                                                    ? s.n_kv_heads
                                                    : 1))
                      : nullptr;
  *bytes = c.off;
  return pl;
}
}  // namespace

// Totals and queue cursors live right after the int32 counters.
int64_t *plan_totals(const Plan &pl) {
  return reinterpret_cast<int64_t *>(pl.counters + kCounters);
}
int32_t *plan_next(const Plan &pl) {
  return pl.counters + kCounters + kTotals * 2;
}

size_t plan_bytes(const PlanShape &s) {
  size_t b = 0;
  carve(nullptr, s, &b);
  return b;
}

Plan plan_carve(void *ws, const PlanShape &s) {
  size_t b = 0;
  return carve(ws, s, &b);
}

hipError_t launch_plan(const AttnCall &c, const Plan &pl,
                       const PlanShape &shape, hipStream_t s) {
  const dopr_attn_args_t *a = c.a;
  PlanArgs pa{a->doc_ids,        a->cu_seqlens,      c.st->d_len,
              c.st->n_docs,      a->total_tokens,    a->n_pairs,
              c.n_rep,           a->max_tokens,      shape.rows_per_item,
              c.st->d_status,    shape.score_only, false};
  int64_t *totals = plan_totals(pl);
  const int64_t P = a->n_pairs;
  const int64_t init_n = c.st->n_docs > kCounters ? c.st->n_docs : kCounters;
  hipLaunchKernelGGL(k_plan_init, dim3(blocks_for(init_n, kThreads)),
                     dim3(kThreads), 0, s, pl, c.st->n_docs, totals,
                     plan_next(pl));
  hipLaunchKernelGGL(k_pair_meta, dim3(blocks_for(P, kThreads)),
                     dim3(kThreads), 0, s, pl, pa);
  hipLaunchKernelGGL(k_doc_pack, dim3(blocks_for(c.st->n_docs, kThreads)),
                     dim3(kThreads), 0, s, pl, c.st->n_docs);
  hipError_t e = exclusive_scan(pl.doc_scan, c.st->n_docs, pl.blk,
                                totals + kTotDocs, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_place, dim3(blocks_for(P, kThreads)), dim3(kThreads),
                     0, s, pl, pa);
  hipLaunchKernelGGL(k_rank, dim3(blocks_for(P + 1, kThreads)),
                     dim3(kThreads), 0, s, pl, pa, totals);
  {
    const int64_t cap = P / (kBigGroup + 1) + 1;
    hipLaunchKernelGGL(k_rank_big, dim3((unsigned)(cap < 256 ? cap : 256)),
                       dim3(1024), 0, s, pl, pa);
  }
  e = exclusive_scan(pl.prow, P + 1, pl.blk, totals + kTotRows, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_items_count, dim3(blocks_for(P + 1, kThreads)),
                     dim3(kThreads), 0, s, pl, pa, totals);
  e = exclusive_scan(pl.item_scan, P + 1, pl.blk, totals + kTotItems, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_items_emit,
                     dim3(std::min(blocks_for(P * 64, kThreads), 65536u)),
                     dim3(kThreads), 0, s, pl, pa, totals);
  hipLaunchKernelGGL(k_blk_pair, dim3(blocks_for(P, kThreads)),
                     dim3(kThreads), 0, s, pl, totals);
  if (a->cu_seqlens)
    hipLaunchKernelGGL(k_token_table, dim3((unsigned)(P + 1)),
                       dim3(kThreads), 0, s, pl, pa, totals);
  const int32_t D = c.st->head_dim;
  hipLaunchKernelGGL(k_norm_bound, dim3(1), dim3(D), 0, s,
                     static_cast<const uint16_t *>(a->k_norm_w),
                     static_cast<const uint16_t *>(a->q_norm_w), pl.kown,
                     pl.unit_w);
  int dev = 0, n_cu = 0;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int64_t lpt_units = a->queue_order == 1   ? 0
                            : a->queue_order == 2 ? kOrderMaxUnits
                                                  : kLptUnitsPerCu * n_cu;
  hipLaunchKernelGGL(k_unit_order, dim3(1), dim3(kOrderWaves * 64), 0, s, pl,
                     c.st->n_kv_heads, lpt_units, totals);
  if (pl.units) {
    const int64_t n_units = (int64_t)pl.items_cap * c.st->n_kv_heads;
    hipLaunchKernelGGL(k_unit_table, dim3(blocks_for(n_units, kThreads)),
                       dim3(kThreads), 0, s, pl, c.st->view(), c.layer,
                       a->softmax_scale * 1.4426950408889634f, kNoRefBound,
                       totals);
  }
  const double log_theta = std::log((double)a->rope_theta);
  hipLaunchKernelGGL(k_rope_table,
                     dim3(blocks_for((int64_t)pl.rope_pos * (D / 2),
                                     kThreads)),
                     dim3(kThreads), 0, s, pl.rope, pl.rope_pos, D / 2,
                     log_theta, a->rope_inv_freq);
  return hipGetLastError();
}

}  // namespace dopr

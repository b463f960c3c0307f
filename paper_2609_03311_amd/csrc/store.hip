// store.hip -- filling and reading back the HBM prefix store.
//
// The store holds, per resident document d and layer l, the prefix K/V
// states of its L_d slots (Sec. 3.3: computed offline, query-independent).
// Keys are kept row-major [L][D]; values are kept transposed [D][Lp] so the
// attention kernel's PV contraction (over keys) reads contiguous 16-byte
// runs.  These kernels run offline (ingest) or in tests only.
#include "internal.hpp"

namespace dopr {
namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;  // slots per transpose tile

__device__ bool doc_ok(const StoreView &sv, int32_t d) {
  return d >= 0 && (int64_t)d < sv.n_docs && sv.doc_len[d] >= 0;
}

// One workgroup per (document i, kv head g).
__global__ __launch_bounds__(kThreads) void k_store_put(
    StoreView sv, int32_t *status, int32_t layer, const int32_t *doc_ids,
    const int64_t *src_cu, const uint16_t *ksrc, const uint16_t *vsrc) {
  const int64_t i = blockIdx.x;
  const int g = blockIdx.y, hkv = sv.n_kv_heads;
  const int32_t d = doc_ids[i];
  const int64_t s0 = src_cu[i], s1 = src_cu[i + 1];
  if (!doc_ok(sv, d) || s1 - s0 != sv.doc_len[d]) {
    if (threadIdx.x == 0 && g == 0) raise_status(status, DOPR_ERR_DOC_RANGE);
    return;
  }
  const int32_t L = sv.doc_len[d], Lp = pad8(L);
  const int D = sv.head_dim, G = D / 8;  // 16-byte granules per row
  const int64_t blk = sv.doc_off[d];
  uint16_t *K = sv.payload + k_offset(blk, L, hkv, layer, g, D);
  uint16_t *VT = sv.payload + vt_offset(blk, L, hkv, layer, g, D);

  // Copy K and track the largest key norm of the slice (G lanes per row, a
  // power of two dividing 64, so a row's lanes run the loop together).
  float norm2_max = 0.f;
  for (int64_t gi = threadIdx.x; gi < (int64_t)L * G; gi += kThreads) {
    const int64_t row = gi / G;
    const int c = gi % G;
    const uint4 *src = reinterpret_cast<const uint4 *>(
        ksrc + ((s0 + row) * hkv + g) * D);
    const uint4 u = src[c];
    reinterpret_cast<uint4 *>(K + row * D)[c] = u;
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float lo = __uint_as_float(w[i] << 16);
      const float hi = __uint_as_float(w[i] & 0xffff0000u);
      ss = fmaf(lo, lo, ss);
      ss = fmaf(hi, hi, ss);
    }
    for (int off = 1; off < G; off <<= 1) ss += __shfl_xor(ss, off, 64);
    norm2_max = fmaxf(norm2_max, ss);
  }
  __shared__ float red[kThreads / 64];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1)
    norm2_max = fmaxf(norm2_max, __shfl_xor(norm2_max, off, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = norm2_max;
  __syncthreads();
  if (threadIdx.x == 0) {
    float m = 0.f;
    for (int w2 = 0; w2 < kThreads / 64; ++w2) m = fmaxf(m, red[w2]);
    // relative slack covers the fp32 rounding of the sum and the sqrt
    sv.kmax[((int64_t)d * sv.n_layers + layer) * hkv + g] =
        sqrtf(m) * 1.0001f;
  }

  __shared__ uint16_t tile[kTile][kHeadDim + 2];
  for (int t0 = 0; t0 < Lp; t0 += kTile) {
    for (int gi = threadIdx.x; gi < kTile * G; gi += kThreads) {
      const int r = gi / G, c = gi % G, slot = t0 + r;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (slot < L)
        val = reinterpret_cast<const uint4 *>(
            vsrc + ((s0 + slot) * hkv + g) * D)[c];
      uint32_t *dst = reinterpret_cast<uint32_t *>(&tile[r][c * 8]);
      dst[0] = val.x; dst[1] = val.y; dst[2] = val.z; dst[3] = val.w;
    }
    __syncthreads();
    // eight slots of one head dim per thread, one 16-byte store (t0 and
    // Lp are multiples of 8, so a run is wholly inside or past the row)
    for (int e = threadIdx.x; e < D * (kTile / 8); e += kThreads) {
      const int dd = e / (kTile / 8), r = 8 * (e % (kTile / 8)),
                slot = t0 + r;
      if (slot < Lp) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          w[i] = (uint32_t)tile[r + 2 * i][dd] |
                 ((uint32_t)tile[r + 2 * i + 1][dd] << 16);
        *reinterpret_cast<uint4 *>(VT + (int64_t)dd * Lp + slot) =
            make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
    __syncthreads();
  }
}

// Inverse of k_store_put into canonical [slots][Hkv][D] rows.
__global__ __launch_bounds__(kThreads) void k_gather(
    StoreView sv, int32_t *status, int32_t layer, const int32_t *doc_ids,
    const int64_t *out_cu, uint16_t *kout, uint16_t *vout) {
  const int64_t i = blockIdx.x;
  const int g = blockIdx.y, hkv = sv.n_kv_heads;
  const int32_t d = doc_ids[i];
  const int64_t o0 = out_cu[i], o1 = out_cu[i + 1];
  if (!doc_ok(sv, d) || o1 - o0 != sv.doc_len[d]) {
    if (threadIdx.x == 0 && g == 0) raise_status(status, DOPR_ERR_DOC_RANGE);
    return;
  }
  const int32_t L = sv.doc_len[d], Lp = pad8(L);
  const int D = sv.head_dim, G = D / 8;
  const int64_t blk = sv.doc_off[d];
  const uint16_t *K = sv.payload + k_offset(blk, L, hkv, layer, g, D);
  const uint16_t *VT = sv.payload + vt_offset(blk, L, hkv, layer, g, D);
  for (int64_t gi = threadIdx.x; gi < (int64_t)L * G; gi += kThreads) {
    const int64_t row = gi / G;
    const int c = gi % G;
    reinterpret_cast<uint4 *>(kout + ((o0 + row) * hkv + g) * D)[c] =
        reinterpret_cast<const uint4 *>(K + row * D)[c];
  }
  for (int64_t e = threadIdx.x; e < (int64_t)L * D; e += kThreads) {
    const int64_t slot = e / D;
    const int dd = e % D;
    vout[((o0 + slot) * hkv + g) * D + dd] = VT[(int64_t)dd * Lp + slot];
  }
}

// Copy every document resident in both stores with the same prefix length:
// its whole payload block (all layers and kv heads, laid out identically
// in both pools) and its key-norm bounds.  Documents resident in only one
// store are left alone; one resident in both with different lengths raises
// DOC_RANGE on dst and is skipped.  Grid-strided over documents, one
// workgroup per document at a time, four 16-byte moves in flight per lane.
__global__ __launch_bounds__(kThreads) void k_store_copy(StoreView dst,
                                                         int32_t *dst_status,
                                                         StoreView src) {
  const int64_t nk = (int64_t)dst.n_layers * dst.n_kv_heads;
  for (int64_t d = blockIdx.x; d < dst.n_docs; d += gridDim.x) {
    const int32_t L = dst.doc_len[d], Ls = src.doc_len[d];
    if (L < 0 || Ls < 0) continue;
    if (L != Ls) {
      if (threadIdx.x == 0) raise_status(dst_status, DOPR_ERR_DOC_RANGE);
      continue;
    }
    const int64_t n16 =
        (int64_t)dst.n_layers *
        layer_block_elems(L, dst.n_kv_heads, dst.head_dim) / 8;
    const uint4 *s = reinterpret_cast<const uint4 *>(src.payload +
                                                     src.doc_off[d]);
    uint4 *t = reinterpret_cast<uint4 *>(dst.payload + dst.doc_off[d]);
    int64_t e = threadIdx.x;
    for (; e + 3 * kThreads < n16; e += 4 * kThreads) {
      const uint4 a = s[e], b = s[e + kThreads], c = s[e + 2 * kThreads],
                  f = s[e + 3 * kThreads];
      t[e] = a;
      t[e + kThreads] = b;
      t[e + 2 * kThreads] = c;
      t[e + 3 * kThreads] = f;
    }
    for (; e < n16; e += kThreads) t[e] = s[e];
    for (int64_t k = threadIdx.x; k < nk; k += kThreads)
      dst.kmax[d * nk + k] = src.kmax[d * nk + k];
  }
}

}  // namespace

hipError_t launch_store_copy(const dopr_store &dst, const dopr_store &src,
                             hipStream_t s) {
  if (dst.n_docs == 0) return hipSuccess;
  const int64_t grid = dst.n_docs < 4096 ? dst.n_docs : 4096;
  hipLaunchKernelGGL(k_store_copy, dim3((unsigned)grid), dim3(kThreads), 0,
                     s, dst.view(), dst.d_status, src.view());
  return hipGetLastError();
}

hipError_t launch_store_put(const dopr_store &st, int32_t layer, int64_t n,
                            const int32_t *doc_ids, const int64_t *src_cu,
                            const uint16_t *k, const uint16_t *v,
                            hipStream_t s) {
  if (n == 0) return hipSuccess;
  dim3 grid((unsigned)n, (unsigned)st.n_kv_heads);
  hipLaunchKernelGGL(k_store_put, grid, dim3(kThreads), 0, s, st.view(),
                     st.d_status, layer, doc_ids, src_cu, k, v);
  return hipGetLastError();
}

hipError_t launch_gather(const dopr_store &st, int32_t layer, int32_t n,
                         const int32_t *doc_ids, const int64_t *out_cu,
                         uint16_t *k, uint16_t *v, hipStream_t s) {
  if (n == 0) return hipSuccess;
  dim3 grid((unsigned)n, (unsigned)st.n_kv_heads);
  hipLaunchKernelGGL(k_gather, grid, dim3(kThreads), 0, s, st.view(),
                     st.d_status, layer, doc_ids, out_cu, k, v);
  return hipGetLastError();
}

}  // namespace dopr

// attn.hip -- online prefix attention of DoPR on gfx950 (MFMA bf16).
//
// Online reranking injects a document's stored prefix states as a
// pre-filled K/V cache and runs only the query and score tokens (Sec. 3.4);
// those tokens see the document only through its prefix states and attend
// causally among themselves (Sec. 3.2.2).  Per layer and kv head g this is
//   out[j,h] = softmax(scale * q^[j,h] . [K_d[g] ; k^[0..j,g]]) . [V_d[g] ; v[0..j,g]]
// with q^/k^ the per-head RMS-normed, rotary-embedded online projections at
// positions L_d + j.
//
// Work decomposition.  The scheduler (group.hip) orders pairs by document
// and cuts each document's stacked rows (token j x q-head of the group,
// token-major) into work items.  A workgroup takes one (item, kv head): every
// row of the item shares the document, so each 32-key chunk of the
// document's prefix is staged in LDS once and consumed by all 4 waves (the
// per-document reuse across queries, expressed on-chip).  Each wave owns
// NQB x 32 rows per pass.  Own keys are staged per pair (normed, rotated)
// in the same LDS buffers and masked per row: same pair and key <= row.
//
// MFMA orientation (v_mfma_f32_32x32x16_bf16, A 32x16, B 16x32, C 32x32):
//   S^T[key][q] = K[key][:] . Q^T[:][q]    A = K (LDS), B = Q^T (registers)
//   O^T[d][q]  += V^T[d][key] . P^T[key][q] A = V^T (LDS), B = P^T (registers)
// so a lane owns one query column: the softmax row statistics are lane-local
// plus one exchange with lane^32, and the probabilities feed PV without a
// transpose.  A-operand rows are read in the order perm32(m) so that lane
// half hf's 16 accumulator registers hold 16 consecutive keys (S) or 16
// consecutive head dims (O): key = 16*hf + i, d = 32*db + 16*hf + i.
#include <cmath>

#include "internal.hpp"

namespace dopr {

int64_t *plan_totals(const Plan &pl);
int32_t *plan_next(const Plan &pl);

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int D = kHeadDim;
constexpr int KC = 32;       // keys per staged chunk
constexpr int WAVES = 4;
constexpr int THREADS = WAVES * 64;
constexpr int kTotItems = 2;  // index into the plan totals
constexpr float kLn2 = 0.69314718055994530942f;

struct AttnParams {
  const uint16_t *q, *k, *v, *qw, *kw;
  const int32_t *cu;
  const int32_t *doc_len;
  const int64_t *doc_off;
  const uint16_t *payload;
  const int32_t *pair_order, *group_doc, *group_ptr;
  const int64_t *prow;
  const int4 *items;
  const int64_t *totals;
  int32_t *next;
  const float2 *rope;
  uint16_t *out;
  float *lse;
  int32_t items_cap, Hq, Hkv, n_rep, layer;
  float eps, c;  // c = softmax_scale * log2(e)
};

// Row order of A operands: MFMA row m -> source row, chosen so that C
// register i of lane half hf corresponds to source row 16*hf + i.
__device__ __forceinline__ int perm32(int m) {
  return ((m >> 2) & 1) * 16 + (m >> 3) * 4 + (m & 3);
}
// XOR swizzles of 16-byte granules in the LDS tiles (bank-conflict-free
// A-operand reads and cooperative writes).
__device__ __forceinline__ int swz_k(int row) {
  return (row & 3) | ((row >> 2) & 4) | ((row << 1) & 8);
}
__device__ __forceinline__ int swz_v(int row) {
  return ((row >> 2) & 1) | ((row >> 3) & 2);
}
__device__ __forceinline__ int sk_off(int row, int gr) {
  return row * D + ((gr ^ swz_k(row)) << 3);
}
__device__ __forceinline__ int svt_off(int d, int gr) {
  return d * KC + ((gr ^ swz_v(d)) << 3);
}

__device__ __forceinline__ void unpack8(const uint4 &u, float *f) {
  f[0] = __uint_as_float(u.x << 16);
  f[1] = __uint_as_float(u.x & 0xffff0000u);
  f[2] = __uint_as_float(u.y << 16);
  f[3] = __uint_as_float(u.y & 0xffff0000u);
  f[4] = __uint_as_float(u.z << 16);
  f[5] = __uint_as_float(u.z & 0xffff0000u);
  f[6] = __uint_as_float(u.w << 16);
  f[7] = __uint_as_float(u.w & 0xffff0000u);
}

__device__ __forceinline__ bf16x8 to_bf16x8(const float *f) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)f[e];
  return r;
}

__device__ __forceinline__ uint4 as_uint4(const bf16x8 &b) {
  return __builtin_bit_cast(uint4, b);
}

// Largest s in [lo, hi) with prow[s] <= r (prow[lo] <= r < prow[hi]).
__device__ __forceinline__ int find_pair(const int64_t *prow, int lo, int hi,
                                         int64_t r) {
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (prow[mid] <= r) lo = mid; else hi = mid;
  }
  return lo;
}

// q^ = RoPE_pos(RMSNorm(q) * w) in the B-operand layout: lane half hf holds
// head dims 16*s + 8*hf + e of its query column (s = k-step 0..7); the
// rotate-half partner of dim i < 64 is dim i + 64, i.e. k-step s + 4 of the
// same lane.
__device__ __forceinline__ void q_fragments(const uint16_t *qrow,
                                            const uint16_t *w,
                                            const float2 *rope_row, int hf,
                                            float eps, bf16x8 *qf) {
  float x[8][8];
#pragma unroll
  for (int s = 0; s < 8; ++s)
    unpack8(*reinterpret_cast<const uint4 *>(qrow + 16 * s + 8 * hf), x[s]);
  float ss = 0.f;
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(x[s][e], x[s][e], ss);
  ss += __shfl_xor(ss, 32, 64);
  const float inv = rsqrtf(ss * (1.0f / D) + eps);
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    float wv[8];
    unpack8(*reinterpret_cast<const uint4 *>(w + 16 * s + 8 * hf), wv);
#pragma unroll
    for (int e = 0; e < 8; ++e) x[s][e] *= inv * wv[e];
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const float4 *cs4 =
        reinterpret_cast<const float4 *>(rope_row + 16 * s + 8 * hf);
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const float4 t = cs4[e2];  // (cos, sin) of dims 2*e2, 2*e2 + 1
      const float c0 = t.x, s0 = t.y, c1 = t.z, s1 = t.w;
      const int e = 2 * e2;
      float a = x[s][e], b = x[s + 4][e];
      x[s][e] = fmaf(a, c0, -b * s0);
      x[s + 4][e] = fmaf(b, c0, a * s0);
      a = x[s][e + 1];
      b = x[s + 4][e + 1];
      x[s][e + 1] = fmaf(a, c1, -b * s1);
      x[s + 4][e + 1] = fmaf(b, c1, a * s1);
    }
  }
#pragma unroll
  for (int s = 0; s < 8; ++s) qf[s] = to_bf16x8(x[s]);
}

// Stage 32 prefix keys (rows c0..c0+31 of K [L][D]) and the matching
// columns of V^T [D][Lp] into LDS; rows past L / Lp are zero.
__device__ __forceinline__ void stage_prefix(const uint16_t *Kp,
                                             const uint16_t *VTp, int L, int Lp,
                                             int c0, uint16_t *sK,
                                             uint16_t *sVT) {
  const uint4 zero = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int gi = threadIdx.x + THREADS * r;
    const int kk = gi >> 4, gr = gi & 15;
    uint4 val = zero;
    if (c0 + kk < L)
      val = *reinterpret_cast<const uint4 *>(Kp + (int64_t)(c0 + kk) * D +
                                             gr * 8);
    *reinterpret_cast<uint4 *>(sK + sk_off(kk, gr)) = val;
  }
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int gi = threadIdx.x + THREADS * r;
    const int d = gi >> 2, gr = gi & 3;
    const int key0 = c0 + 8 * gr;
    uint4 val = zero;
    if (key0 < Lp)
      val = *reinterpret_cast<const uint4 *>(VTp + (int64_t)d * Lp + key0);
    *reinterpret_cast<uint4 *>(sVT + svt_off(d, gr)) = val;
  }
}

// Stage 32 own keys j = c0..c0+31 of one pair: k^ = RoPE_{L+j}(RMSNorm(k) *
// w) into sK, v transposed into sVT.  Thread (kk = t/8, sub = t%8) handles
// head dims 8*sub..8*sub+7 and 64+8*sub..64+8*sub+7 (rotate-half partners).
__device__ __forceinline__ void stage_own(const AttnParams &P, int64_t tok0,
                                          int Tp, int c0, int g, int L,
                                          uint16_t *sK, uint16_t *sVT) {
  const int kk = threadIdx.x >> 3, sub = threadIdx.x & 7;
  const int jk = c0 + kk;
  const bool valid = jk < Tp;
  float x[16], vv[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) x[e] = vv[e] = 0.f;
  if (valid) {
    const int64_t rowoff = ((tok0 + jk) * P.Hkv + g) * (int64_t)D;
    unpack8(*reinterpret_cast<const uint4 *>(P.k + rowoff + 8 * sub), x);
    unpack8(*reinterpret_cast<const uint4 *>(P.k + rowoff + 64 + 8 * sub),
            x + 8);
    unpack8(*reinterpret_cast<const uint4 *>(P.v + rowoff + 8 * sub), vv);
    unpack8(*reinterpret_cast<const uint4 *>(P.v + rowoff + 64 + 8 * sub),
            vv + 8);
  }
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < 16; ++e) ss = fmaf(x[e], x[e], ss);
  ss += __shfl_xor(ss, 1, 64);
  ss += __shfl_xor(ss, 2, 64);
  ss += __shfl_xor(ss, 4, 64);
  if (valid) {
    const float inv = rsqrtf(ss * (1.0f / D) + P.eps);
    float w0[8], w1[8];
    unpack8(*reinterpret_cast<const uint4 *>(P.kw + 8 * sub), w0);
    unpack8(*reinterpret_cast<const uint4 *>(P.kw + 64 + 8 * sub), w1);
    const float2 *cs = P.rope + (int64_t)(L + jk) * kRopeHalf + 8 * sub;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float a = x[e] * inv * w0[e], b = x[8 + e] * inv * w1[e];
      const float2 t = cs[e];
      x[e] = fmaf(a, t.x, -b * t.y);
      x[8 + e] = fmaf(b, t.x, a * t.y);
    }
  }
  *reinterpret_cast<uint4 *>(sK + sk_off(kk, sub)) = as_uint4(to_bf16x8(x));
  *reinterpret_cast<uint4 *>(sK + sk_off(kk, sub + 8)) =
      as_uint4(to_bf16x8(x + 8));
  const bf16x8 v0 = to_bf16x8(vv), v1 = to_bf16x8(vv + 8);
  const int gr = kk >> 3, in = kk & 7;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int d0 = 8 * sub + e, d1 = 64 + 8 * sub + e;
    reinterpret_cast<__bf16 *>(sVT)[svt_off(d0, gr) + in] = v0[e];
    reinterpret_cast<__bf16 *>(sVT)[svt_off(d1, gr) + in] = v1[e];
  }
}

struct RowInfo {
  int64_t tok;
  int32_t s, j, head;
  bool valid;
};

// One 32-key chunk against one 32-query block: S^T = K Q^T, mask, online
// softmax update, O^T += V^T P^T.
template <bool OWN>
__device__ __forceinline__ void attend_chunk(const uint16_t *sK,
                                             const uint16_t *sVT,
                                             const bf16x8 *qf, floatx16 *acc,
                                             float &m, float &l, int lq, int hf,
                                             float c, int c0, int L,
                                             const RowInfo &ri, int s_cur) {
  floatx16 S;
#pragma unroll
  for (int i = 0; i < 16; ++i) S[i] = 0.f;
  const int krow = perm32(lq);
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const bf16x8 a =
        *reinterpret_cast<const bf16x8 *>(sK + sk_off(krow, 2 * s + hf));
    S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], S, 0, 0, 0);
  }
  const float NEG = -INFINITY;
  float mx = NEG;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int key = c0 + 16 * hf + i;
    const bool ok = OWN ? (ri.s == s_cur && key <= ri.j) : (key < L);
    S[i] = ok ? S[i] : NEG;
    mx = fmaxf(mx, S[i]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float mnew = fmaxf(m, mx * c);
  const float muse = mnew == NEG ? 0.f : mnew;
  const float alpha = __builtin_amdgcn_exp2f(m - muse);
  float p[16], psum = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    p[i] = __builtin_amdgcn_exp2f(fmaf(S[i], c, -muse));
    psum += p[i];
  }
  l = fmaf(l, alpha, psum);
  m = mnew;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[db][i] *= alpha;
  const bf16x8 pb0 = to_bf16x8(p), pb1 = to_bf16x8(p + 8);
  const int vrow = perm32(lq);
#pragma unroll
  for (int db = 0; db < 4; ++db) {
    const int d = 32 * db + vrow;
    const bf16x8 a0 =
        *reinterpret_cast<const bf16x8 *>(sVT + svt_off(d, 2 * hf));
    const bf16x8 a1 =
        *reinterpret_cast<const bf16x8 *>(sVT + svt_off(d, 2 * hf + 1));
    acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, pb0, acc[db], 0, 0, 0);
    acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, pb1, acc[db], 0, 0, 0);
  }
}

template <int NQB>
__global__ __launch_bounds__(THREADS) void k_prefix_attn(AttnParams P) {
  __shared__ __attribute__((aligned(16))) uint16_t sK[KC * D];
  __shared__ __attribute__((aligned(16))) uint16_t sVT[D * KC];
  __shared__ int s_w;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lq = lane & 31, hf = lane >> 5;
  const int queue = blockIdx.x & 7;
  int64_t n_items = P.totals[kTotItems];
  if (n_items > P.items_cap) n_items = P.items_cap;
  const int64_t n_work = n_items * P.Hkv;
  constexpr int PASS = WAVES * NQB * 32;

  for (;;) {
    if (threadIdx.x == 0) s_w = atomicAdd(&P.next[queue], 1);
    __syncthreads();
    const int64_t w = queue + 8 * (int64_t)s_w;
    __syncthreads();
    if (w >= n_work) break;
    const int item = (int)(w / P.Hkv), g = (int)(w % P.Hkv);
    const int4 it = P.items[item];
    const int group = it.x, row0 = it.y, row1 = it.z;
    const int doc = P.group_doc[group];
    const int L = P.doc_len[doc], Lp = pad8(L);
    const int64_t blk = P.doc_off[doc];
    const uint16_t *Kp =
        P.payload + k_offset(blk, L, P.Hkv, P.layer, g);
    const uint16_t *VTp =
        P.payload + vt_offset(blk, L, P.Hkv, P.layer, g);
    const int sp0 = P.group_ptr[group], sp1 = P.group_ptr[group + 1];

    for (int pass0 = row0; pass0 < row1; pass0 += PASS) {
      RowInfo ri[NQB];
      bf16x8 qf[NQB][8];
      floatx16 acc[NQB][4];
      float m[NQB], l[NQB];
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        const int r = pass0 + (wave * NQB + qb) * 32 + lq;
        const bool valid = r < row1;
        const int rc = valid ? r : row1 - 1;
        const int s = find_pair(P.prow, sp0, sp1, rc);
        const int pr = P.pair_order[s];
        const int rr = rc - (int)P.prow[s];
        const int j = rr / P.n_rep, rep = rr - j * P.n_rep;
        ri[qb].s = s;
        ri[qb].j = j;
        ri[qb].tok = (int64_t)P.cu[pr] + j;
        ri[qb].head = g * P.n_rep + rep;
        ri[qb].valid = valid;
        q_fragments(P.q + (ri[qb].tok * P.Hq + ri[qb].head) * D, P.qw,
                    P.rope + (int64_t)(L + j) * kRopeHalf, hf, P.eps,
                    qf[qb]);
        m[qb] = -INFINITY;
        l[qb] = 0.f;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[qb][db][i] = 0.f;
      }

      // Document prefix: every row sees all L slots.
      for (int c0 = 0; c0 < L; c0 += KC) {
        __syncthreads();
        stage_prefix(Kp, VTp, L, Lp, c0, sK, sVT);
        __syncthreads();
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb)
          attend_chunk<false>(sK, sVT, qf[qb], acc[qb], m[qb], l[qb], lq, hf,
                              P.c, c0, L, ri[qb], 0);
      }

      // Own causal keys, pair by pair over the pairs this pass touches.
      const int pass_end = pass0 + PASS < row1 ? pass0 + PASS : row1;
      const int s_lo = find_pair(P.prow, sp0, sp1, pass0);
      const int s_hi = find_pair(P.prow, sp0, sp1, pass_end - 1);
      for (int s = s_lo; s <= s_hi; ++s) {
        const int pr = P.pair_order[s];
        const int64_t tok0 = P.cu[pr];
        const int Tp = P.cu[pr + 1] - P.cu[pr];
        const int64_t srow0 = P.prow[s], srow1 = P.prow[s + 1];
        const int64_t hi_row = (srow1 < pass_end ? srow1 : pass_end) - 1;
        const int jmax = (int)((hi_row - srow0) / P.n_rep);
        for (int c0 = 0; c0 <= jmax; c0 += KC) {
          __syncthreads();
          stage_own(P, tok0, Tp, c0, g, L, sK, sVT);
          __syncthreads();
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb) {
            const bool need = ri[qb].s == s && ri[qb].j >= c0;
            if (__any(need))
              attend_chunk<true>(sK, sVT, qf[qb], acc[qb], m[qb], l[qb], lq,
                                 hf, P.c, c0, L, ri[qb], s);
          }
        }
      }

      // Normalise and write O (bf16) and the natural-log LSE.
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        const float lt = l[qb] + __shfl_xor(l[qb], 32, 64);
        if (!ri[qb].valid) continue;
        const float inv = 1.0f / lt;
        uint16_t *orow = P.out + (ri[qb].tok * P.Hq + ri[qb].head) * D;
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          float o[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) o[i] = acc[qb][db][i] * inv;
          uint4 *dst = reinterpret_cast<uint4 *>(orow + 32 * db + 16 * hf);
          dst[0] = as_uint4(to_bf16x8(o));
          dst[1] = as_uint4(to_bf16x8(o + 8));
        }
        if (P.lse && hf == 0)
          P.lse[ri[qb].tok * P.Hq + ri[qb].head] =
              (m[qb] + __log2f(lt)) * kLn2;
      }
    }
  }
}

// Pairs whose document is out of range or not resident: zero outputs and
// -inf LSE (their token range was validated by the scheduler).
__global__ __launch_bounds__(256) void k_zero_invalid(
    const int32_t *counters, const int32_t *invalid, const int32_t *cu,
    int32_t Hq, uint16_t *out, float *lse) {
  const int32_t n_inv = counters[kCntInvalid];
  for (int32_t idx = blockIdx.x; idx < n_inv; idx += gridDim.x) {
    const int32_t p = invalid[idx];
    const int64_t t0 = cu[p], t1 = cu[p + 1];
    const int64_t n16 = (t1 - t0) * Hq * D / 8;
    uint4 *o = reinterpret_cast<uint4 *>(out + t0 * Hq * D);
    for (int64_t e = threadIdx.x; e < n16; e += blockDim.x)
      o[e] = make_uint4(0, 0, 0, 0);
    if (lse)
      for (int64_t e = threadIdx.x; e < (t1 - t0) * Hq; e += blockDim.x)
        lse[t0 * Hq + e] = -INFINITY;
  }
}

template <int NQB>
hipError_t launch_variant(const AttnParams &p, hipStream_t s) {
  int dev = 0, n_cu = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_prefix_attn<NQB>,
                                                   THREADS, 0);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  // Persistent grid, a multiple of 8 so block b always serves queue b % 8
  // (consecutive blocks are dispatched round-robin over the 8 XCDs).
  unsigned grid = (unsigned)(n_cu * per_cu);
  grid = (grid + 7) / 8 * 8;
  hipLaunchKernelGGL(k_prefix_attn<NQB>, dim3(grid), dim3(THREADS), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnCall &c, const Plan &pl,
                            const PlanShape &shape, hipStream_t s) {
  const dopr_attn_args_t *a = c.a;
  const dopr_store &st = *c.st;
  AttnParams p{};
  p.q = static_cast<const uint16_t *>(a->q);
  p.k = static_cast<const uint16_t *>(a->k);
  p.v = static_cast<const uint16_t *>(a->v);
  p.qw = static_cast<const uint16_t *>(a->q_norm_w);
  p.kw = static_cast<const uint16_t *>(a->k_norm_w);
  p.cu = a->cu_seqlens;
  p.doc_len = st.d_len;
  p.doc_off = st.d_off;
  p.payload = st.d_payload;
  p.pair_order = pl.pair_order;
  p.group_doc = pl.group_doc;
  p.group_ptr = pl.group_ptr;
  p.prow = pl.prow;
  p.items = pl.items;
  p.totals = plan_totals(pl);
  p.next = plan_next(pl);
  p.rope = pl.rope;
  p.out = static_cast<uint16_t *>(a->out);
  p.lse = a->lse;
  p.items_cap = pl.items_cap;
  p.Hq = a->n_q_heads;
  p.Hkv = st.n_kv_heads;
  p.n_rep = c.n_rep;
  p.layer = c.layer;
  p.eps = a->rms_eps;
  p.c = a->softmax_scale * 1.4426950408889634f;

  hipError_t e;
  if (a->timing_begin) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->timing_begin), s);
    if (e != hipSuccess) return e;
  }
  switch (a->kernel_variant) {
    case 2: e = launch_variant<2>(p, s); break;
    default: e = launch_variant<1>(p, s); break;
  }
  if (e != hipSuccess) return e;
  if (a->timing_end) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->timing_end), s);
    if (e != hipSuccess) return e;
  }
  const unsigned zgrid = (unsigned)(a->n_pairs < 1024 ? (a->n_pairs > 0 ? a->n_pairs : 1) : 1024);
  hipLaunchKernelGGL(k_zero_invalid, dim3(zgrid), dim3(256), 0, s,
                     pl.counters, pl.invalid, a->cu_seqlens, a->n_q_heads,
                     p.out, a->lse);
  (void)shape;
  return hipGetLastError();
}

}  // namespace dopr

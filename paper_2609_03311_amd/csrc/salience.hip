// salience.hip -- offline salience selection (Sec. 3.2.1, used by the
// offline compression of Sec. 3.3).
//
// For one document of n tokens with final-layer queries q^ [n, Hq, D] and
// keys k^ [n, Hkv, D] (as they enter the attention product):
//   A_h[j, i] = softmax_i(scale * q^_h[j] . k^_g[i]),  i <= j,  g = h / n_rep
//   Abar      = (1/Hq) sum_h A_h                     (rows attend, columns
//                                                      are attended)
//   u_i       = mean of the m = min(p, n - i) largest Abar[j, i], j >= i
//   selected  = the K positions with the largest u (ties: lower position),
//               written in ascending position order.
//
// Four kernels, each a plain pass over its data:
//   k_row_lse     per (row block of 128, kv head): the log2-domain
//                 log-sum-exp of every row of every q head of the group
//                 (scaled logits; one flash-style sweep over the visible
//                 keys with a running maximum).
//   k_mean_attn   per (row block, key block) of 128 x 128 on or below the
//                 diagonal: every head's probabilities exp2(S - lse2),
//                 summed over heads in head order, times 1/Hq, stored as
//                 fp32 row-major [n, n] (only i <= j is written).
// In both attention kernels the key blocks strictly below the diagonal,
// which every row of the block sees whole, take a path without masks or
// branches inside the head or sub-tile loops, so that one sub-tile's
// exponentials can be scheduled against the next sub-tile's products.
//   k_col_topp    per strip of 64 columns: each lane keeps the PM largest
//                 values of its column in a sorted register list while four
//                 waves stream interleaved rows; the lists are merged and
//                 the top m averaged.
//   k_topk        per document: bitonic sort of (u, position) keys in LDS,
//                 then an ordered compaction of the chosen positions.
//
// Both attention kernels form S = K Q^T with the 32x32x16 bf16 MFMA in the
// same operand layout and the same k order, so the logits they see are the
// same fp32 values.  A-operand (key) rows are read in the order perm(m) so
// that lane half hf's 16 accumulators hold 16 consecutive keys 16 hf + i
// for the lane's query column.
#include <cmath>
#include <type_traits>

#include "internal.hpp"

namespace dopr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int D = kHeadDim;
constexpr int kRowBlock = 128;   // rows per unit (4 waves x 32)
constexpr int kKeyBlock = 128;   // keys per mean-attention unit
constexpr int kStrip = 64;       // columns per top-p strip

__device__ __forceinline__ int perm(int m) {
  return ((m >> 2) & 1) * 16 + (m >> 3) * 4 + (m & 3);
}
// XOR swizzle of the 16-byte granules of a K row staged in LDS, so the rows
// read together by a quarter wave fall on distinct bank groups.
__device__ __forceinline__ int swz(int row) {
  return (row & 3) | ((row >> 2) & 4) | ((row << 1) & 8);
}

struct Doc {
  int64_t t0;
  int32_t n;
  bool ok;
};

__device__ __forceinline__ Doc doc_at(const SalienceParams &P, int d) {
  Doc r;
  const int32_t a = P.cu[d], b = P.cu[d + 1];
  r.t0 = a;
  r.n = b - a;
  r.ok = a >= 0 && r.n >= 1 && r.n <= P.max_len && b <= P.total_tokens;
  return r;
}

__device__ __forceinline__ bf16x8 ld8(const uint16_t *p) {
  return *reinterpret_cast<const bf16x8 *>(p);
}

// ---------------------------------------------------------------------------
// Keys are staged in LDS in blocks of 128 rows (32 KB), double-buffered so a
// block's direct global->LDS loads overlap the products on the previous one.
constexpr int kLdsK = kKeyBlock * D;  // bf16 elements (swizzled rows)

// Keys key0 .. key0+127 of kv head g into `dst`: each lane writes 16 bytes of
// a 1 KB block (4 key rows), fetching the global granule that the swizzled
// layout puts in its slot, so slot p of row r holds granule p ^ swz(r).
// Rows past the document's end repeat row n-1 (masked by the causal test).
template <int WAVES = 4>
__device__ __forceinline__ void stage_keys(const SalienceParams &P,
                                           const Doc &doc, int key0, int g,
                                           uint16_t *dst) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int b = wave; b < kKeyBlock / 4; b += WAVES) {
    const int row = 4 * b + (lane >> 4), p = lane & 15;
    const int key = min(key0 + row, doc.n - 1);
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void *)(
            P.k + ((doc.t0 + key) * P.hkv + g) * D + ((p ^ swz(row)) << 3)),
        (__attribute__((address_space(3))) void *)(dst + b * 512), 16, 0, 0);
  }
}

__device__ __forceinline__ void wait_vmem() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// The A-operand fragments of key sub-tile st (keys 32 st .. 32 st + 31 of
// the staged block, row order perm) for lane half hf.
__device__ __forceinline__ void key_frags(const uint16_t *kbuf, int st,
                                          int kr, int hf, bf16x8 (&kf)[8]) {
  const int row = 32 * st + kr;
#pragma unroll
  for (int s = 0; s < 8; ++s)
    kf[s] = ld8(kbuf + row * D + (((2 * s + hf) ^ swz(row)) << 3));
}

// ---------------------------------------------------------------------------
// Largest key norm of each (document, kv head), as kKeyNormParts partial
// maxima over interleaved 64-row slices.  grid (docs, kv heads, parts);
// 16 lanes per key row (16 bytes each), four rows per wave and step, four
// steps in flight.
__global__ __launch_bounds__(256) void k_key_norm(SalienceParams P) {
  __shared__ float wmax[4];
  const int d = blockIdx.x, g = blockIdx.y, part = blockIdx.z;
  const Doc doc = doc_at(P, d);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane & 15, r0 = 4 * wave + (lane >> 4);  // 16 rows a step
  float mx = 0.f;
  if (doc.ok) {
    for (int i0 = 64 * part; i0 < doc.n; i0 += 64 * kKeyNormParts) {
      float ss[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + 16 * u + r0;
        ss[u] = 0.f;
        if (i < doc.n) {
          const uint4 w = *reinterpret_cast<const uint4 *>(
              P.k + ((doc.t0 + i) * P.hkv + g) * D + 8 * sub);
          const uint32_t v[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float lo = __uint_as_float(v[e] << 16);
            const float hi = __uint_as_float(v[e] & 0xffff0000u);
            ss[u] = fmaf(lo, lo, fmaf(hi, hi, ss[u]));
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
#pragma unroll
        for (int off = 8; off > 0; off >>= 1)
          ss[u] += __shfl_xor(ss[u], off, 64);
        mx = fmaxf(mx, ss[u]);
      }
    }
  }
#pragma unroll
  for (int off = 16; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  if (lane == 0) wmax[wave] = mx;
  __syncthreads();
  if (threadIdx.x == 0)
    P.kmax[((int64_t)d * P.hkv + g) * kKeyNormParts + part] =
        sqrtf(fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3])));
}

// Row log-sum-exp.  grid (row blocks of 128, kv head, docs); each wave owns
// 32 rows and keeps the HR q heads of the group in registers while the
// document's keys 0 .. (last row of the block) stream through LDS, one
// 128-key block at a time, shared by the block's four waves.  Per row and
// head the sum of 2^(logit - m) over the visible keys (scaled logits in log2
// units) with one of two references m:
//   - fixed: m = c |q^_j| max_i |k^_i| bounds every logit of the row from
//     above (Cauchy-Schwarz), and from below by -m, so with m <= 60 every
//     term lies in [2^-120, 1] and no maximum is tracked at all;
//   - running: the exact running maximum, for waves where some row's bound
//     exceeds 60.
// The two lane halves are combined at the end.
constexpr float kFixedRefMax = 60.f;
// row blocks (of 128) from which the LSE sweep groups three per block
constexpr int kLseGroupMinBlocks = 6;

// Sum and maximum of a tile's 16 values per lane in four interleaved
// partials, so the adds (or maxima) form chains of four, not one chain of
// sixteen behind the exponentials.
__device__ __forceinline__ float sum16(const float (&e)[16]) {
  float a[4] = {e[0], e[1], e[2], e[3]};
#pragma unroll
  for (int i = 4; i < 16; ++i) a[i & 3] += e[i];
  return (a[0] + a[1]) + (a[2] + a[3]);
}
__device__ __forceinline__ float max16(const floatx16 &x) {
  float a[4] = {x[0], x[1], x[2], x[3]};
#pragma unroll
  for (int i = 4; i < 16; ++i) a[i & 3] = fmaxf(a[i & 3], x[i]);
  return fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
}

// grid (row groups, kv heads, documents), longest rows first.  A block of
// WAVES waves covers RBS = WAVES / 4 consecutive row blocks (four waves of
// 32 rows each) and stages each key block once for all of them.  Groups
// are aligned to the last row block, so a partial group holds the
// shortest rows; its waves below row block 0 load clamped rows and
// compute nothing.  Four waves: two blocks per CU in 256 registers; twelve:
// one block per CU, three waves per SIMD in 168 registers.
template <int HR, int WAVES>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(
    WAVES == 4 ? 2 : 3, WAVES == 4 ? 2 : 3))) void k_row_lse(SalienceParams P) {
  constexpr int RBS = WAVES / 4;
  __shared__ __attribute__((aligned(16))) uint16_t ks[2][kLdsK];
  const int d = P.d0 + blockIdx.z;
  const Doc doc = doc_at(P, d);
  if (!doc.ok) return;
  const int nb_doc = (doc.n + kRowBlock - 1) / kRowBlock;
  const int top = (P.max_len + kRowBlock - 1) / kRowBlock - 1 -
                  RBS * (int)blockIdx.x;
  if (top - RBS + 1 >= nb_doc) return;  // block-uniform, before barriers
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int hf = lane >> 5, lq = lane & 31;
  const int rb = top - RBS + 1 + (wave >> 2);  // this wave's row block
  const int row0 = rb * kRowBlock + (wave & 3) * 32;
  const bool active = rb >= 0 && row0 < doc.n;
  const int g = blockIdx.y;
  const int j = row0 + lq;
  const int jl = min(max(j, 0), doc.n - 1);
  const int last = min(row0 + 31, doc.n - 1);
  const int64_t qrow = (doc.t0 + jl) * P.hq;
  const int kr = perm(lq);
  const int n_kb = min(top, nb_doc - 1) + 1;  // key blocks 0 .. the last

  float kmax = 0.f;
#pragma unroll
  for (int i = 0; i < kKeyNormParts; ++i)
    kmax = fmaxf(kmax, P.kmax[((int64_t)d * P.hkv + g) * kKeyNormParts + i]);
  for (int h0 = 0; h0 < P.n_rep; h0 += HR) {
    const int hbase = g * P.n_rep + h0;
    bf16x8 qf[HR][8];
    float m[HR], l[HR];
    bool fits = true;
#pragma unroll
    for (int r = 0; r < HR; ++r) {
      l[r] = 0.f;
      // (a wave past the document's end loads its clamped rows too: it
      // computes below the diagonal and stores nothing)
      float ss = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        qf[r][s] = ld8(P.q + (qrow + hbase + r) * D + 16 * s + 8 * hf);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = (float)qf[r][s][e];
          ss = fmaf(x, x, ss);
        }
      }
      ss += __shfl_xor(ss, 32, 64);
      m[r] = P.c * sqrtf(ss) * kmax;
      fits = fits && m[r] <= kFixedRefMax;
    }
    // wave-uniform choice of the reference
    const bool fixed = __all(fits);
    if (!fixed) {
#pragma unroll
      for (int r = 0; r < HR; ++r) m[r] = -INFINITY;
    }
    if (h0 > 0) __syncthreads();  // the previous heads are done with ks[0]
    stage_keys<WAVES>(P, doc, 0, g, ks[0]);
    for (int kb = 0; kb < n_kb; ++kb) {
      wait_vmem();
      __syncthreads();  // block kb staged; every wave done with the other
      if (kb + 1 < n_kb)
        stage_keys<WAVES>(P, doc, (kb + 1) * kKeyBlock, g, ks[(kb + 1) & 1]);
      // past this wave's diagonal, or a row block outside the document
      // (wave-uniform; the block's barriers are all above)
      if (RBS > 1 && (kb > rb || rb >= nb_doc)) continue;
      const uint16_t *kbuf = ks[kb & 1];
      const int key0 = kb * kKeyBlock;
      // below the diagonal every row sees all 128 keys: four sub-tiles in
      // straight-line code (no masks, no branches), the same arithmetic as
      // the masked path with every key visible; the next sub-tile's
      // fragments are read once the last head's products have consumed
      // the current ones
      auto full_block = [&](auto fixed_ref) {
        constexpr bool FIXED = decltype(fixed_ref)::value;
        bf16x8 kf[8];
        key_frags(kbuf, 0, kr, hf, kf);
#pragma unroll
        for (int st = 0; st < 4; ++st) {
#pragma unroll
          for (int r = 0; r < HR; ++r) {
            floatx16 S;
#pragma unroll
            for (int i = 0; i < 16; ++i) S[i] = 0.f;
#pragma unroll
            for (int s = 0; s < 8; ++s)
              S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[r][s], S,
                                                          0, 0, 0);
            if (r == HR - 1 && st + 1 < 4)
              key_frags(kbuf, st + 1, kr, hf, kf);
            if (FIXED) {
              float e[16];
#pragma unroll
              for (int i = 0; i < 16; ++i)
                e[i] = __builtin_amdgcn_exp2f(fmaf(S[i], P.c, -m[r]));
              l[r] += sum16(e);
            } else {
              const float mn = fmaxf(m[r], max16(S) * P.c);
              float e[16];
#pragma unroll
              for (int i = 0; i < 16; ++i)
                e[i] = __builtin_amdgcn_exp2f(fmaf(S[i], P.c, -mn));
              l[r] = l[r] * __builtin_amdgcn_exp2f(m[r] - mn) + sum16(e);
              m[r] = mn;
            }
          }
        }
      };
      if (kb < rb) {
        if (fixed)
          full_block(std::true_type{});
        else
          full_block(std::false_type{});
        continue;
      }
      if (!active) continue;
      const int nt = min(4, (last - key0) / 32 + 1);
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        if (st >= nt) break;
        const int row = 32 * st + kr;
        bf16x8 kf[8];
#pragma unroll
        for (int s = 0; s < 8; ++s)
          kf[s] = ld8(kbuf + row * D + (((2 * s + hf) ^ swz(row)) << 3));
        // keys of this sub-tile past the wave's first row need the mask
        const bool masked = key0 + 32 * st + 31 > row0;
        const int lim = j - key0 - 32 * st - 16 * hf;  // visible: i <= lim
#pragma unroll
        for (int r = 0; r < HR; ++r) {
          floatx16 S;
#pragma unroll
          for (int i = 0; i < 16; ++i) S[i] = 0.f;
#pragma unroll
          for (int s = 0; s < 8; ++s)
            S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[r][s], S,
                                                        0, 0, 0);
          // the scale c > 0 commutes with the max, so it is applied once
          // to the chunk's max and fused into each exponent's argument
          floatx16 x;
#pragma unroll
          for (int i = 0; i < 16; ++i)
            x[i] = masked && i > lim ? -INFINITY : S[i];
          const float mn = fixed ? m[r] : fmaxf(m[r], max16(x) * P.c);
          if (mn > -INFINITY) {
            float e[16];
#pragma unroll
            for (int i = 0; i < 16; ++i)
              e[i] = __builtin_amdgcn_exp2f(fmaf(x[i], P.c, -mn));
            l[r] = l[r] * __builtin_amdgcn_exp2f(m[r] - mn) + sum16(e);
            m[r] = mn;
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < HR; ++r) {
      const float mo = __shfl_xor(m[r], 32, 64);
      const float lo = __shfl_xor(l[r], 32, 64);
      const float mn = fmaxf(m[r], mo);
      // every row sees at least its own key, so mn is finite
      const float tot = l[r] * __builtin_amdgcn_exp2f(m[r] - mn) +
                        lo * __builtin_amdgcn_exp2f(mo - mn);
      if (active && hf == 0 && j < doc.n)
        P.lse2[(int64_t)(hbase + r) * P.total_tokens + doc.t0 + j] =
            mn + log2f(tot);
    }
  }
}

// ---------------------------------------------------------------------------
// Head-averaged attention.  Unit (rb, kb), kb <= rb, covers rows rb*128 ..
// +127 and keys kb*128 .. +127, with a code path of its own for the units
// below the diagonal (kb < rb: every row sees all 128 keys, no masks and
// no branches in the head loop, so a sub-tile's exponentials can overlap
// the next sub-tile's products) and for the diagonal units (kb == rb,
// causal masks).  Each kv head's 128 key rows are staged in
// LDS with direct global->LDS loads, double-buffered so the next kv head's
// keys arrive while the current one is used.  Each wave walks the q heads
// one at a time; a sub-tile's key fragments are read from LDS while the
// previous sub-tile's exponentials run, and the next head's q fragments
// (into the registers of the current head's, after its last product) while
// the last sub-tile's run.
template <bool DIAG>
__device__ __forceinline__ void mean_attn_unit(const SalienceParams &P,
                                               const Doc &doc, int d, int rb,
                                               int kb,
                                               uint16_t (&ks)[2][kLdsK]) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int hf = lane >> 5, lq = lane & 31;
  const int row0 = rb * kRowBlock + wave * 32;
  const bool active = row0 < doc.n;
  const int j = row0 + lq;
  const int jl = min(j, doc.n - 1);
  const int key0 = kb * kKeyBlock;
  // key sub-tiles 0 .. nt-1 hold a key some row of this wave can see
  const int last_row = min(row0 + 31, doc.n - 1);
  const int nt = active ? min(4, (last_row - key0) / 32 + 1) : 0;
  const int64_t qrow = (doc.t0 + jl) * P.hq;
  const int64_t lcol = doc.t0 + jl;
  const int kr = perm(lq);

  floatx16 acc[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[s][i] = 0.f;

  bf16x8 qf[8];
  float L = 0.f, L_next = 0.f;
  auto load_q = [&](int h) {
#pragma unroll
    for (int s = 0; s < 8; ++s)
      qf[s] = ld8(P.q + (qrow + h) * D + 16 * s + 8 * hf);
    L_next = P.lse2[(int64_t)h * P.total_tokens + lcol];
  };
  stage_keys(P, doc, key0, 0, ks[0]);
  // below the diagonal a wave past the document's end (rows clamped to
  // its last row) computes anyway and stores nothing, keeping the head
  // loop free of branches
  if (!DIAG || active) load_q(0);
  int g_cur = 0;
  for (int h = 0; h < P.hq; ++h) {
    // on a new kv head, wait for its keys (and for every wave to be done
    // with the other buffer), then start the next kv head's keys
    const int g = h / P.n_rep;
    if (h == 0 || g != g_cur) {
      wait_vmem();
      __syncthreads();
      if (g + 1 < P.hkv) stage_keys(P, doc, key0, g + 1, ks[(g + 1) & 1]);
      g_cur = g;
    }
    const uint16_t *kbuf = ks[g & 1];
    L = L_next;
    const int hn = h + 1 < P.hq ? h + 1 : h;  // the last head reloads its own
    if (!DIAG) {
      bf16x8 kf[8];
      key_frags(kbuf, 0, kr, hf, kf);
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        floatx16 S;
#pragma unroll
        for (int i = 0; i < 16; ++i) S[i] = 0.f;
#pragma unroll
        for (int s = 0; s < 8; ++s)
          S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[s], S, 0, 0,
                                                      0);
        if (st + 1 < 4)
          key_frags(kbuf, st + 1, kr, hf, kf);
        else
          load_q(hn);
#pragma unroll
        for (int i = 0; i < 16; ++i)
          acc[st][i] += __builtin_amdgcn_exp2f(fmaf(S[i], P.c, -L));
      }
    } else {
      if (!active) continue;
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        if (st >= nt) break;
        bf16x8 kf[8];
        key_frags(kbuf, st, kr, hf, kf);
        floatx16 S;
#pragma unroll
        for (int i = 0; i < 16; ++i) S[i] = 0.f;
#pragma unroll
        for (int s = 0; s < 8; ++s)
          S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[s], S, 0, 0,
                                                      0);
        const int lim = j - key0 - 32 * st - 16 * hf;  // visible: i <= lim
#pragma unroll
        for (int i = 0; i < 16; ++i)
          acc[st][i] += i <= lim ? __builtin_amdgcn_exp2f(fmaf(S[i], P.c, -L))
                                 : 0.f;
      }
      load_q(hn);
    }
  }
  if (!active || j >= doc.n) return;
  float *out = P.abar + (int64_t)(d - P.d0) * P.abar_stride +
               (int64_t)j * P.max_len;
  const bool vec = (P.max_len & 3) == 0;  // rows 16-byte aligned
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    if (st >= nt) break;
    const int i0 = key0 + 32 * st + 16 * hf;
    float v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = acc[st][i] * P.inv_hq;
    if (vec && i0 + 16 <= j + 1) {
#pragma unroll
      for (int c = 0; c < 4; ++c)
        *reinterpret_cast<float4 *>(out + i0 + 4 * c) =
            make_float4(v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]);
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (i0 + i <= j) out[i0 + i] = v[i];
    }
  }
}

// grid (units, docs): the nb diagonal units first (their waves see 1 to 4
// sub-tiles, so they are kept out of the launch's tail), then the units
// below the diagonal, unit nb + t with t = rb (rb - 1) / 2 + kb.
__global__ __launch_bounds__(256, 2) void k_mean_attn(SalienceParams P,
                                                      int32_t nb) {
  __shared__ __attribute__((aligned(16))) uint16_t ks[2][kLdsK];
  const int d = P.d0 + blockIdx.y;
  const Doc doc = doc_at(P, d);
  if (!doc.ok) return;
  if ((int)blockIdx.x < nb) {  // block-uniform
    const int rb = blockIdx.x;
    if (rb * kRowBlock >= doc.n) return;  // before any barrier
    mean_attn_unit<true>(P, doc, d, rb, rb, ks);
  } else {
    const int t = blockIdx.x - nb;
    int rb = (int)((sqrtf(8.f * t + 1.f) + 1.f) * 0.5f);
    while (rb * (rb - 1) / 2 > t) --rb;
    while ((rb + 1) * rb / 2 <= t) ++rb;
    const int kb = t - rb * (rb - 1) / 2;
    if (rb * kRowBlock >= doc.n) return;  // before any barrier
    mean_attn_unit<false>(P, doc, d, rb, kb, ks);
  }
}

// ---------------------------------------------------------------------------
// Column top-p means.  grid (strips of 64 columns, docs); the 4 waves of a
// block stream rows j = c0 + w, c0 + w + 4, ... of the strip; lane l keeps
// the PM largest values of column c0 + l (descending, -1 = empty) and the
// lists are merged through LDS at the end.
template <int PM>
__device__ __forceinline__ void insert(float (&L)[PM], float v) {
#pragma unroll
  for (int k = 0; k < PM; ++k) {
    const float hi = fmaxf(L[k], v);
    v = fminf(L[k], v);
    L[k] = hi;
  }
}

template <int PM>
__global__ __launch_bounds__(256) void k_col_topp(SalienceParams P) {
  __shared__ float merge[3][PM][kStrip];
  const int d = P.d0 + blockIdx.y;
  const Doc doc = doc_at(P, d);
  if (!doc.ok) return;
  const int c0 = blockIdx.x * kStrip;
  if (c0 >= doc.n) return;  // block-uniform, before the barrier
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = c0 + lane;
  const bool col = c < doc.n;
  const float *base = P.abar + (int64_t)(d - P.d0) * P.abar_stride +
                      (col ? c : c0);
  float L[PM];
#pragma unroll
  for (int k = 0; k < PM; ++k) L[k] = -1.f;
  constexpr int U = 8;
  int j = c0 + wave;
  for (; j + 4 * (U - 1) < doc.n; j += 4 * U) {
    float v[U];
#pragma unroll
    for (int x = 0; x < U; ++x)
      v[x] = base[(int64_t)(j + 4 * x) * P.max_len];
#pragma unroll
    for (int x = 0; x < U; ++x) {
      const float w = (col && j + 4 * x >= c) ? v[x] : -1.f;
      if (__any(w > L[PM - 1])) insert(L, w);
    }
  }
  for (; j < doc.n; j += 4) {
    const float v = base[(int64_t)j * P.max_len];
    const float w = (col && j >= c) ? v : -1.f;
    if (__any(w > L[PM - 1])) insert(L, w);
  }
  if (wave > 0) {
#pragma unroll
    for (int k = 0; k < PM; ++k) merge[wave - 1][k][lane] = L[k];
  }
  __syncthreads();
  if (wave != 0 || !col) return;
  for (int w = 0; w < 3; ++w)
    for (int k = 0; k < PM; ++k) {
      const float v = merge[w][k][lane];
      if (__any(v > L[PM - 1])) insert(L, v);
    }
  const int m = min(P.top_p, doc.n - c);
  float sum = 0.f;
#pragma unroll
  for (int k = 0; k < PM; ++k)
    if (k < m) sum += L[k];
  P.u[doc.t0 + c] = sum / (float)m;
}

// ---------------------------------------------------------------------------
// Validation of the document and selection offsets (one thread per doc).
__global__ __launch_bounds__(256) void k_check(SalienceParams P) {
  const int d = blockIdx.x * 256 + threadIdx.x;
  if (d >= P.n_docs) return;
  if (!doc_at(P, d).ok || (d == P.n_docs - 1 &&
                           P.cu[d + 1] != P.total_tokens))
    raise_status(P.status, DOPR_ERR_SEQLEN);
}

}  // namespace

// ---------------------------------------------------------------------------
// Top-K selection.  One block per document; keys (orderable u bits << 32 |
// ~position) sorted descending by a bitonic network in LDS, the first K
// positions flagged and compacted in position order.
namespace {

constexpr int kTopkThreads = 1024;

__device__ __forceinline__ uint32_t orderable(float f) {
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__global__ __launch_bounds__(kTopkThreads) void k_topk(TopkParams P) {
  __shared__ uint64_t key[kSalienceMaxLen];
  __shared__ uint8_t flag[kSalienceMaxLen];
  __shared__ int32_t wsum[kTopkThreads / 64];
  const int d = blockIdx.x;
  const int32_t a = P.cu[d], b = P.cu[d + 1];
  const int32_t n = b - a;
  if (a < 0 || n < 1 || n > P.max_len || b > P.total_tokens) {
    if (threadIdx.x == 0 && P.status) raise_status(P.status, DOPR_ERR_SEQLEN);
    return;
  }
  const int32_t sa = P.cs[d], sb = P.cs[d + 1];
  const int32_t K = sb - sa;
  if (sa < 0 || K < 0 || K > n || sb > P.total_select) {
    if (threadIdx.x == 0 && P.status) raise_status(P.status, DOPR_ERR_SEQLEN);
    return;
  }
  if (K == 0) return;
  int32_t *out = P.selected + sa;
  if (K == n) {
    for (int i = threadIdx.x; i < n; i += kTopkThreads) out[i] = i;
    return;
  }
  int N2 = 1;
  while (N2 < n) N2 <<= 1;
  const float *u = P.u + a;
  for (int i = threadIdx.x; i < N2; i += kTopkThreads)
    key[i] = i < n ? ((uint64_t)orderable(u[i]) << 32) | (uint32_t)~i : 0ull;
  __syncthreads();
  for (int k = 2; k <= N2; k <<= 1)
    for (int s = k >> 1; s > 0; s >>= 1) {
      for (int i = threadIdx.x; i < N2; i += kTopkThreads) {
        const int x = i ^ s;
        if (x > i) {
          const uint64_t p = key[i], q = key[x];
          const bool desc = (i & k) == 0;
          if (desc ? p < q : p > q) {
            key[i] = q;
            key[x] = p;
          }
        }
      }
      __syncthreads();
    }
  for (int i = threadIdx.x; i < n; i += kTopkThreads) flag[i] = 0;
  __syncthreads();
  for (int r = threadIdx.x; r < K; r += kTopkThreads)
    flag[~(uint32_t)key[r]] = 1;
  __syncthreads();
  // ordered compaction: thread t owns positions [t*per, (t+1)*per)
  const int per = (n + kTopkThreads - 1) / kTopkThreads;
  const int p0 = threadIdx.x * per;
  int cnt = 0;
  for (int i = p0; i < min(p0 + per, n); ++i) cnt += flag[i];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = cnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int before = incl - cnt;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  for (int i = p0; i < min(p0 + per, n); ++i)
    if (flag[i]) out[before++] = i;
}

}  // namespace

hipError_t launch_salience_chunk(const SalienceParams &p, int32_t n_docs,
                                 int hr, int pm, hipStream_t s) {
  if (n_docs == 0) return hipSuccess;
  const int nb = (p.max_len + kRowBlock - 1) / kRowBlock;
  const dim3 g_lse(nb, p.hkv, n_docs);
  const dim3 g_att(nb * (nb + 1) / 2, n_docs);
  const dim3 g_col((p.max_len + kStrip - 1) / kStrip, n_docs);
  // long documents: three row blocks per block at three waves per SIMD
  // (one q head per sweep); short ones keep enough blocks with one row
  // block each
  if (nb >= kLseGroupMinBlocks) {
    hipLaunchKernelGGL((k_row_lse<1, 12>), dim3((nb + 2) / 3, p.hkv, n_docs),
                       dim3(768), 0, s, p);
  } else if (hr == 2) {
    hipLaunchKernelGGL((k_row_lse<2, 4>), g_lse, dim3(256), 0, s, p);
  } else {
    hipLaunchKernelGGL((k_row_lse<1, 4>), g_lse, dim3(256), 0, s, p);
  }
  hipLaunchKernelGGL(k_mean_attn, g_att, dim3(256), 0, s, p, (int32_t)nb);
  if (pm == 8)
    hipLaunchKernelGGL(k_col_topp<8>, g_col, dim3(256), 0, s, p);
  else if (pm == 16)
    hipLaunchKernelGGL(k_col_topp<16>, g_col, dim3(256), 0, s, p);
  else if (pm == 32)
    hipLaunchKernelGGL(k_col_topp<32>, g_col, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(k_col_topp<64>, g_col, dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_key_norms(const SalienceParams &p, hipStream_t s) {
  if (p.n_docs == 0) return hipSuccess;
  hipLaunchKernelGGL(k_key_norm,
                     dim3((unsigned)p.n_docs, (unsigned)p.hkv, kKeyNormParts),
                     dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_salience_check(const SalienceParams &p, hipStream_t s) {
  if (p.n_docs == 0 || !p.status) return hipSuccess;
  hipLaunchKernelGGL(k_check, dim3((p.n_docs + 255) / 256), dim3(256), 0, s,
                     p);
  return hipGetLastError();
}

hipError_t launch_topk(const TopkParams &p, int32_t n_docs, hipStream_t s) {
  if (n_docs == 0) return hipSuccess;
  hipLaunchKernelGGL(k_topk, dim3(n_docs), dim3(kTopkThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace dopr

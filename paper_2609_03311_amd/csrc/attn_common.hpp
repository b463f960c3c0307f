// attn_common.hpp -- device building blocks shared by the attention
// kernels (attn.hip: block kernels, last-layer scoring; stream.hip: the
// streaming kernel): operand layouts and swizzles, the q^ and k^
// prologues, and the MFMA/softmax steps of one 32-key chunk.  Internal to
// the library.
#pragma once

#include <cmath>

#include "internal.hpp"

namespace dopr {

int64_t *plan_totals(const Plan &pl);
int32_t *plan_next(const Plan &pl);

// Arguments of the attention kernels.
struct AttnParams {
  const uint16_t *q, *k, *v, *qw, *kw;
  const int32_t *doc_len;
  const int64_t *doc_off;
  const float *kmax;
  const uint16_t *payload;
  const int32_t *group_doc, *blk_pair;
  const int4 *items;
  const int4 *spair;  // sorted pair: (tok0, T, first stacked row)
  const int2 *utok;   // stacked token: (batch token, position in pair)
  const int64_t *totals;
  int32_t *next;
  int32_t *counters;
  int32_t *fix;
  const float *kown;
  const float2 *rope;
  uint16_t *out;
  float *lse;
  // score mode: output row of sorted pair s is pair_order[s]; the epilogue
  // adds the score head's partial sums (h^2, g*w_yes*h, g*w_no*h) per row
  const int32_t *pair_order;
  float *part;
  const uint16_t *head_norm_w, *head_w;
  // pass kernel: precomputed own keys k^ [Hkv][Ntok][D], a zero page and
  // the work-unit table
  const uint16_t *kh, *zero;
  const int4 *units;
  int64_t ntok;
  // work units of each queue, costliest first (see unit_at)
  const int32_t *qorder;
  int32_t items_cap, Hq, Hkv, n_rep, layer, n_layers;
  int32_t flag_all;  // queue every unit for the SAFE pass (self-check mode)
  int32_t norm;      // per-head RMSNorm of q and k (0: no QK-norm, unit gains)
  float eps, c;      // c = softmax_scale * log2(e)
};

// Arguments of k_own_khat (k^ of every online token, for the streaming
// kernel).
struct KhatParams {
  const uint16_t *k, *kw;
  const int32_t *doc_ids, *pair_order, *doc_len;
  const int4 *spair;
  const int64_t *totals;
  const float2 *rope;
  uint16_t *kh;
  int64_t ntok;
  int32_t Hkv;
  float eps;
  int32_t norm;
};

// stream.hip: k_own_khat, then the streaming kernel (head size D).
hipError_t launch_stream(int D, const AttnParams &p, const KhatParams &kp,
                         int32_t n_pairs, hipStream_t s);

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int KC = 32;      // keys per MFMA chunk
constexpr int kFixQueue = 8;  // cursor slot of the fixup pass
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kTau = 8.0f;       // SAFE mode: lazy-rescale threshold
constexpr float kHeadroom = 80.f;  // reference <= first max + 80 (log2)
constexpr float kLoOk = 0x1p-90f, kHiOk = 0x1p100f;
// Fix-up list entries: work unit index, plus this bit when the unit was not
// computed by the fast pass (its logit bound exceeds kNoRefBound); those
// run the bounded-reference mode first, the others the exact mode.
constexpr int32_t kFixUnscored = 1 << 30;
// Prefix chunks resident in LDS per head size: the one-block-per-CU shape
// fills the CU's LDS (D = 128: 8 chunks, 256 slots; D = 64: 16 chunks),
// the two-blocks-per-CU shape half of it (3 chunks at D = 128; at D = 64
// 8 chunks, so a 256-slot prefix stays resident in both blocks and the
// two blocks' independent barriers let one's memory waits overlap the
// other's products).
constexpr int big_chunks(int d) { return d == 128 ? 8 : 16; }
constexpr int small_chunks(int d) { return d == 128 ? 3 : 8; }



// Up to 160 KB: the whole LDS of a CU.  Keys and values live in 32-key
// chunk blocks of 64*D bytes -- K [32 keys][D] and V^T [D][32 keys], 16-byte
// granules XOR-swizzled -- so prefix chunks and own-key chunks share one
// layout and one set of per-lane read offsets.  The own-key chunk is
// double-buffered; at item boundaries (no own chunk in flight) its first
// words carry the work index broadcast and the per-wave overflow flags.
template <int D, int NCHK>
struct Smem {
  static constexpr int PSEG = NCHK * KC;  // prefix slots resident at once
  uint16_t pk[NCHK][KC * D];  // prefix K chunks
  uint16_t pv[NCHK][D * KC];  // prefix V^T chunks
  uint16_t ok[2][KC * D];     // own k^
  uint16_t ov[2][D * KC];     // own v^T
  __device__ int *words() { return reinterpret_cast<int *>(ok[0]); }
};

__device__ __forceinline__ int perm32(int m) {
  return ((m >> 2) & 1) * 16 + (m >> 3) * 4 + (m & 3);
}
// XOR swizzles of 16-byte granules: the 16 rows read together by a quarter
// wave (perm32 of lanes 0..15 or 16..31) land on 16 distinct bank groups.
// A K row is 256 B at D = 128 (16 granules) and 128 B at D = 64 (8, so two
// rows share a 256-byte bank line).
template <int D>
__device__ __forceinline__ int swz(int row) {
  if constexpr (D == 128)
    return (row & 3) | ((row >> 2) & 4) | ((row << 1) & 8);
  else
    return ((row >> 1) & 1) | ((row >> 1) & 2) | ((row >> 2) & 4);
}
__device__ __forceinline__ int swz_v(int row) {
  return ((row >> 2) & 1) | ((row >> 3) & 2);
}
// Element offsets inside a chunk block: K row `key` (0..31), granule gr
// (0..D/8-1); V^T row d (0..D-1), granule g (0..3, keys 8g..8g+7).
template <int D>
__device__ __forceinline__ int kc_off(int key, int gr) {
  return key * D + ((gr ^ swz<D>(key)) << 3);
}
__device__ __forceinline__ int vc_off(int d, int g) {
  return d * KC + ((g ^ swz_v(d)) << 3);
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

// A zero the compiler cannot see through: offsetting a loop-invariant load
// by it keeps the load (and its unpacked values) inside the loop instead of
// hoisting them and holding the registers for the whole kernel.
__device__ __forceinline__ int opaque_zero() {
  int z;
  asm volatile("s_mov_b32 %0, 0" : "=s"(z));
  return z;
}

// Materialise a finished value here: an empty asm that "modifies" it stops
// the compiler from sinking its computation (and the inputs it keeps alive)
// down to the first use.
__device__ __forceinline__ void pin(bf16x8 &x) {
  uint4 u = __builtin_bit_cast(uint4, x);
  asm volatile("" : "+v"(u.x), "+v"(u.y), "+v"(u.z), "+v"(u.w));
  x = __builtin_bit_cast(bf16x8, u);
}

// acc + sum of squares of 8 packed bf16 values (products exact in fp32).
__device__ __forceinline__ float sumsq8(const uint4 &u, float acc) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2 p = __builtin_bit_cast(bf16x2, w[i]);
    acc = __builtin_amdgcn_fdot2_f32_bf16(p, p, acc, false);
  }
  return acc;
}

// Sorted pair owning stacked row r: the owner of r's 32-row block, then a
// short forward scan (wave-uniform when r is).
__device__ __forceinline__ int find_pair(const AttnParams &P, int r) {
  int s = P.blk_pair[r >> 5];
  while (P.spair[s + 1].z <= r) ++s;
  return s;
}

// c * q^ with q^ = RoPE_pos(RMSNorm(q) * w), in the B-operand layout: lane
// half hf holds head dims 16*s + 8*hf + e of its query column (k-step
// s = 0..D/16-1); the rotate-half partner of dim i < D/2 is dim i + D/2 =
// k-step s + D/32, same lane.  c = softmax_scale * log2(e).  The raw row
// stays packed until the norm is known; the rotation then runs one k-step
// pair at a time, each finished fragment pinned in place so the compiler
// does not keep the step's inputs alive until the first product.
template <int D>
__device__ __forceinline__ void q_fragments(const uint16_t *qrow,
                                            const uint16_t *w,
                                            const float2 *rope_row, int hf,
                                            float eps, float c, bool norm,
                                            bf16x8 *qf) {
  constexpr int NS = D / 16, HS = NS / 2;
  // every load is issued up front (one round trip to memory): the raw row,
  // the gains (packed) and this lane's D/4 (cos, sin) pairs
  uint4 raw[NS], wr[NS];
  float4 cs[4 * HS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    raw[s] = *reinterpret_cast<const uint4 *>(qrow + 16 * s + 8 * hf);
  w += opaque_zero();
#pragma unroll
  for (int s = 0; s < NS; ++s)
    wr[s] = *reinterpret_cast<const uint4 *>(w + 16 * s + 8 * hf);
#pragma unroll
  for (int s = 0; s < HS; ++s)
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2)
      cs[4 * s + e2] =
          reinterpret_cast<const float4 *>(rope_row + 16 * s + 8 * hf)[e2];
  // sum of squares straight from the packed pairs (v_dot2), so the
  // unpacked row is not kept alive until the rotation
  float ss = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) ss = sumsq8(raw[s], ss);
  ss += __shfl_xor(ss, 32, 64);
  const float inv = norm ? c * rsqrtf(ss * (1.0f / D) + eps) : c;
#pragma unroll
  for (int s = 0; s < HS; ++s) {
    float x0[8], x1[8], w0[8], w1[8];
    unpack8(raw[s], x0);
    unpack8(raw[s + HS], x1);
    unpack8(wr[s], w0);
    unpack8(wr[s + HS], w1);
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const float4 t = cs[4 * s + e2];  // (cos, sin) of dims 2e2, 2e2 + 1
      const int e = 2 * e2;
      float a = x0[e] * (inv * w0[e]), b = x1[e] * (inv * w1[e]);
      x0[e] = fmaf(a, t.x, -b * t.y);
      x1[e] = fmaf(b, t.x, a * t.y);
      a = x0[e + 1] * (inv * w0[e + 1]);
      b = x1[e + 1] * (inv * w1[e + 1]);
      x0[e + 1] = fmaf(a, t.z, -b * t.w);
      x1[e + 1] = fmaf(b, t.z, a * t.w);
    }
    qf[s] = to_bf16x8(x0);
    qf[s + HS] = to_bf16x8(x1);
    pin(qf[s]);
    pin(qf[s + HS]);
  }
}

// ---- q^ with the rotary pairs and gains shared across a token's lanes ----
// When n_rep is a multiple of 4 (of 2), the four lanes of a quad (the two
// lanes of a pair) hold query heads of one token and the same half of the
// head dims, so they need the same (cos, sin) pairs and gains.  Each lane
// loads its share; the multiplies that use a value read it from the owning
// lane through a DPP broadcast within the quad folded into the instruction
// (the compiler's DPP moves are not folded into these users, so the
// operations are written out).  Every product and sum is the one
// q_fragments forms, in the same order and rounding: fma(cos, a, sin * -b)
// and fma(cos, b, sin * a).  s_nop 4 covers the wait states a DPP read
// needs after a vector write of its source or of EXEC.
//
// Source codes: K = 0..3 reads quad lane K (quad_perm [K,K,K,K]); K = 4, 5
// reads pair lane K - 4 (quad_perm [p,p,p+2,p+2]).
#define DPP_Q(A, B, C, E) \
  " quad_perm:[" #A "," #B "," #C "," #E "] row_mask:0xf bank_mask:0xf"
#define DPP_ROT(A, B, C, E)                                     \
  "s_nop 4\n\t"                                                 \
  "v_mul_f32_dpp %0, %9, -%5" DPP_Q(A, B, C, E) "\n\t"          \
  "v_mul_f32_dpp %1, %9, %4" DPP_Q(A, B, C, E) "\n\t"           \
  "v_fmac_f32_dpp %0, %8, %4" DPP_Q(A, B, C, E) "\n\t"          \
  "v_fmac_f32_dpp %1, %8, %5" DPP_Q(A, B, C, E) "\n\t"          \
  "v_mul_f32_dpp %2, %11, -%7" DPP_Q(A, B, C, E) "\n\t"         \
  "v_mul_f32_dpp %3, %11, %6" DPP_Q(A, B, C, E) "\n\t"          \
  "v_fmac_f32_dpp %2, %10, %6" DPP_Q(A, B, C, E) "\n\t"         \
  "v_fmac_f32_dpp %3, %10, %7" DPP_Q(A, B, C, E)
#define DPP_UNPACK(A, B, C, E)                                  \
  "s_nop 4\n\t"                                                 \
  "v_mul_u32_u24_dpp %0, %8, %12" DPP_Q(A, B, C, E) "\n\t"      \
  "v_and_b32_dpp %1, %8, %13" DPP_Q(A, B, C, E) "\n\t"          \
  "v_mul_u32_u24_dpp %2, %9, %12" DPP_Q(A, B, C, E) "\n\t"      \
  "v_and_b32_dpp %3, %9, %13" DPP_Q(A, B, C, E) "\n\t"          \
  "v_mul_u32_u24_dpp %4, %10, %12" DPP_Q(A, B, C, E) "\n\t"     \
  "v_and_b32_dpp %5, %10, %13" DPP_Q(A, B, C, E) "\n\t"         \
  "v_mul_u32_u24_dpp %6, %11, %12" DPP_Q(A, B, C, E) "\n\t"     \
  "v_and_b32_dpp %7, %11, %13" DPP_Q(A, B, C, E)

// (x0[e], x1[e]) and (x0[e+1], x1[e+1]) rotated by source K's pairs t =
// (cos_e, sin_e, cos_e+1, sin_e+1); a and b are the normed, scaled inputs.
template <int K>
__device__ __forceinline__ void rot_pairs_shared(const float4 &t, float a0,
                                                 float b0, float a1, float b1,
                                                 float &x0a, float &x1a,
                                                 float &x0b, float &x1b) {
#define DPP_ROT_ASM(A, B, C, E)                                              \
  asm volatile(DPP_ROT(A, B, C, E)                                           \
               : "=&v"(x0a), "=&v"(x1a), "=&v"(x0b), "=&v"(x1b)              \
               : "v"(a0), "v"(b0), "v"(a1), "v"(b1), "v"(t.x), "v"(t.y),     \
                 "v"(t.z), "v"(t.w))
  if constexpr (K == 0) DPP_ROT_ASM(0, 0, 0, 0);
  else if constexpr (K == 1) DPP_ROT_ASM(1, 1, 1, 1);
  else if constexpr (K == 2) DPP_ROT_ASM(2, 2, 2, 2);
  else if constexpr (K == 3) DPP_ROT_ASM(3, 3, 3, 3);
  else if constexpr (K == 4) DPP_ROT_ASM(0, 0, 2, 2);
  else DPP_ROT_ASM(1, 1, 3, 3);
#undef DPP_ROT_ASM
}

// Source K's packed bf16 gains u, unpacked as unpack8 does.
template <int K>
__device__ __forceinline__ void unpack8_shared(const uint4 &u, uint32_t c16,
                                               uint32_t hi, float *f) {
  uint32_t r[8];
#define DPP_UNPACK_ASM(A, B, C, E)                                           \
  asm volatile(DPP_UNPACK(A, B, C, E)                                        \
               : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]),         \
                 "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])          \
               : "v"(u.x), "v"(u.y), "v"(u.z), "v"(u.w), "v"(c16), "v"(hi))
  // (u24 product by 65536: the low half shifted up, the high half dropped)
  if constexpr (K == 0) DPP_UNPACK_ASM(0, 0, 0, 0);
  else if constexpr (K == 1) DPP_UNPACK_ASM(1, 1, 1, 1);
  else if constexpr (K == 2) DPP_UNPACK_ASM(2, 2, 2, 2);
  else if constexpr (K == 3) DPP_UNPACK_ASM(3, 3, 3, 3);
  else if constexpr (K == 4) DPP_UNPACK_ASM(0, 0, 2, 2);
  else DPP_UNPACK_ASM(1, 1, 3, 3);
#undef DPP_UNPACK_ASM
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = __uint_as_float(r[i]);
}

// The source as a value that is constant once the caller's loops are
// unrolled.
__device__ __forceinline__ void rot_pairs_at(int k, const float4 &t, float a0,
                                             float b0, float a1, float b1,
                                             float &x0a, float &x1a,
                                             float &x0b, float &x1b) {
  switch (k) {
    case 0: rot_pairs_shared<0>(t, a0, b0, a1, b1, x0a, x1a, x0b, x1b); break;
    case 1: rot_pairs_shared<1>(t, a0, b0, a1, b1, x0a, x1a, x0b, x1b); break;
    case 2: rot_pairs_shared<2>(t, a0, b0, a1, b1, x0a, x1a, x0b, x1b); break;
    case 3: rot_pairs_shared<3>(t, a0, b0, a1, b1, x0a, x1a, x0b, x1b); break;
    case 4: rot_pairs_shared<4>(t, a0, b0, a1, b1, x0a, x1a, x0b, x1b); break;
    default: rot_pairs_shared<5>(t, a0, b0, a1, b1, x0a, x1a, x0b, x1b);
  }
}

__device__ __forceinline__ void unpack8_at(int k, const uint4 &u,
                                           uint32_t c16, uint32_t hi,
                                           float *f) {
  switch (k) {
    case 0: unpack8_shared<0>(u, c16, hi, f); break;
    case 1: unpack8_shared<1>(u, c16, hi, f); break;
    case 2: unpack8_shared<2>(u, c16, hi, f); break;
    case 3: unpack8_shared<3>(u, c16, hi, f); break;
    case 4: unpack8_shared<4>(u, c16, hi, f); break;
    default: unpack8_shared<5>(u, c16, hi, f);
  }
}

// q_fragments with the sharing above among GROUP = 4 or 2 lanes; qk = the
// lane's place in its group.  Lane qk loads gain vectors s = qk*NS/GROUP ..
// + NS/GROUP - 1 and, of every k-step pair s, the rotary float4s
// e2 = qk*4/GROUP .. + 4/GROUP - 1 (q_fragments' numbering), so the
// group's loads of one k-step cover contiguous bytes of the row.
template <int D, int GROUP>
__device__ __forceinline__ void q_fragments_shared(const uint16_t *qrow,
                                                   const uint16_t *w,
                                                   const float2 *rope_row,
                                                   int hf, int qk, float eps,
                                                   float c, bool norm,
                                                   bf16x8 *qf) {
  constexpr int NS = D / 16, HS = NS / 2, GW = NS / GROUP, EW = 4 / GROUP;
  constexpr int BASE = GROUP == 4 ? 0 : 4;  // source codes of the group
  uint4 raw[NS], wr[GW];
  float4 cs[HS * EW];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    raw[s] = *reinterpret_cast<const uint4 *>(qrow + 16 * s + 8 * hf);
  w += opaque_zero();
#pragma unroll
  for (int m = 0; m < GW; ++m)
    wr[m] = *reinterpret_cast<const uint4 *>(w + 16 * (qk * GW + m) + 8 * hf);
#pragma unroll
  for (int s = 0; s < HS; ++s)
#pragma unroll
    for (int m = 0; m < EW; ++m)
      cs[s * EW + m] = reinterpret_cast<const float4 *>(
          rope_row + 16 * s + 8 * hf)[qk * EW + m];
  float ss = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) ss = sumsq8(raw[s], ss);
  ss += __shfl_xor(ss, 32, 64);
  const float inv = norm ? c * rsqrtf(ss * (1.0f / D) + eps) : c;
  const uint32_t c16 = 65536u + opaque_zero(), hi = 0xffff0000u + opaque_zero();
#pragma unroll
  for (int s = 0; s < HS; ++s) {
    float x0[8], x1[8], w0[8], w1[8];
    unpack8(raw[s], x0);
    unpack8(raw[s + HS], x1);
    unpack8_at(BASE + s / GW, wr[s % GW], c16, hi, w0);
    unpack8_at(BASE + (s + HS) / GW, wr[(s + HS) % GW], c16, hi, w1);
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const int e = 2 * e2;
      const float a0 = x0[e] * (inv * w0[e]);
      const float b0 = x1[e] * (inv * w1[e]);
      const float a1 = x0[e + 1] * (inv * w0[e + 1]);
      const float b1 = x1[e + 1] * (inv * w1[e + 1]);
      rot_pairs_at(BASE + e2 / EW, cs[s * EW + e2 % EW], a0, b0, a1, b1,
                   x0[e], x1[e], x0[e + 1], x1[e + 1]);
    }
    qf[s] = to_bf16x8(x0);
    qf[s + HS] = to_bf16x8(x1);
    pin(qf[s]);
    pin(qf[s + HS]);
  }
}

// q^ for a lane whose token is shared by the lanes of its quad (n_rep a
// multiple of 4) or pair (n_rep even), else q_fragments.
template <int D>
__device__ __forceinline__ void q_fragments_any(const uint16_t *qrow,
                                                const uint16_t *w,
                                                const float2 *rope_row, int hf,
                                                int lane, int n_rep, float eps,
                                                float c, bool norm,
                                                bf16x8 *qf) {
  if ((n_rep & 3) == 0)
    q_fragments_shared<D, 4>(qrow, w, rope_row, hf, lane & 3, eps, c, norm,
                             qf);
  else if ((n_rep & 1) == 0)
    q_fragments_shared<D, 2>(qrow, w, rope_row, hf, lane & 1, eps, c, norm,
                             qf);
  else
    q_fragments<D>(qrow, w, rope_row, hf, eps, c, norm, qf);
}
#undef DPP_UNPACK
#undef DPP_ROT
#undef DPP_Q

// Stage prefix slots [seg0, seg0 + n) of kv head g into LDS with direct
// global->LDS loads (no registers): lane i of a wave writes bytes
// [16i, 16i+16) of the wave's 1 KB LDS block, so each lane fetches the
// global granule that the swizzled layout puts in its slot.  K rows past n
// are left stale (their logits are masked by a select).  V^T columns past
// the stored ones (up to the chunk end) are zeroed instead: masked keys
// must multiply a finite value.  The store's pad columns [L, Lp) are zero.
template <int WAVES, int D, int NCHK>
__device__ __forceinline__ void stage_prefix(const uint16_t *Kp,
                                             const uint16_t *VTp, int L,
                                             int seg0, int n,
                                             Smem<D, NCHK> &sm) {
  constexpr int PSEG = Smem<D, NCHK>::PSEG;
  const int Lp = pad8(L);
  constexpr int G = D / 8;       // granules per K row
  constexpr int RPB = 64 / G;    // K rows per 1 KB block
  constexpr int VB = D / 16;     // 1 KB V^T blocks per chunk
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // K: 1 KB block b = rows RPB*b .. RPB*b + RPB-1, lane -> (row, physical
  // granule)
  const int kblocks = (unsigned)(n + RPB - 1) / RPB;
  uint16_t *pk = sm.pk[0];
  for (int b = wave; b < kblocks; b += WAVES) {
    const int r = RPB * b + (unsigned)lane / G, p = (unsigned)lane % G;
    if (r < n) {
      const int gr = p ^ swz<D>(r & 31);
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void *)(
              Kp + (int64_t)(seg0 + r) * D + gr * 8),
          (__attribute__((address_space(3))) void *)(pk + b * 512), 16, 0, 0);
    }
  }
  // V^T: 1 KB block b = chunk b / VB, rows d = 16 (b % VB) .. + 15, four
  // granules of 8 keys each
  const int lp = Lp - seg0 < PSEG ? Lp - seg0 : PSEG;  // stored columns
  const int vblocks = ((n + KC - 1) / KC) * VB;
  uint16_t *pv = sm.pv[0];
  for (int b = wave; b < vblocks; b += WAVES) {
    const int d = 16 * ((unsigned)b % VB) + (lane >> 2), p = lane & 3;
    const int key = KC * ((unsigned)b / VB) + 8 * (p ^ swz_v(d));
    if (key < lp)
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void *)(
              VTp + (int64_t)d * Lp + seg0 + key),
          (__attribute__((address_space(3))) void *)(pv + b * 512), 16, 0, 0);
    else
      *reinterpret_cast<uint4 *>(pv + b * 512 + lane * 8) =
          make_uint4(0, 0, 0, 0);
  }
}

// Wait for this wave's direct-to-LDS (and other vector-memory) loads.
__device__ __forceinline__ void wait_vmem() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// One own-key chunk: 32 keys of one pair starting at key c0 (wave-uniform).
struct OwnStep {
  int s;      // sorted pair index
  int c0;     // first own key of the chunk
  int tok0;   // the pair's first batch token
  int T;      // the pair's token count
  int srow0;  // the pair's first stacked row
};

// Sum over the N = 4 or 8 lanes Nk..Nk+N-1 (every lane gets the same
// value): the two quad butterflies, then for N = 8 the other quad through
// row_half_mirror (DPP, no LDS round trip).  The additions pair the same
// values as a butterfly over lane ^ 1, ^ 2 (, ^ 4).
template <int N>
__device__ __forceinline__ float sum_lanes(float x) {
  x += __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0xB1, 0xF,
                                      0xF, false));
  x += __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x4E, 0xF,
                                      0xF, false));
  if constexpr (N == 8)
    x += __builtin_bit_cast(
        float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x141,
                                        0xF, 0xF, false));
  return x;
}

// k^ = RoPE(RMSNorm(k) * w) for one lane's share of a key row: head dims
// 8*sub .. 8*sub+7 (a0) and their rotate-half partners D/2 + 8*sub .. (a1),
// with the row's D/16 lanes adjacent (the norm's sum of squares is reduced
// over them).  g0/g1 are the gains of the same dims, r0..r3 the (cos, sin)
// pairs of the key's position.  Invalid rows give zeros (and add zero to
// the reduction).  Every kernel that forms k^ calls this, so the staged,
// streamed and precomputed values agree bit for bit.
template <int D>
__device__ __forceinline__ void khat_part(const uint4 &a0, const uint4 &a1,
                                          const uint4 &g0, const uint4 &g1,
                                          const float4 &r0, const float4 &r1,
                                          const float4 &r2, const float4 &r3,
                                          bool valid, float eps, bool norm,
                                          float *x) {
  float ss = valid ? sumsq8(a1, sumsq8(a0, 0.f)) : 0.f;
  if (valid) {
    unpack8(a0, x);
    unpack8(a1, x + 8);
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) x[e] = 0.f;
  }
  ss = sum_lanes<D / 16>(ss);
  if (valid) {
    const float inv = norm ? rsqrtf(ss * (1.0f / D) + eps) : 1.f;
    float w0[8], w1[8];
    unpack8(g0, w0);
    unpack8(g1, w1);
    const float cs[16] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w,
                          r2.x, r2.y, r2.z, r2.w, r3.x, r3.y, r3.z, r3.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float a = x[e] * inv * w0[e], b = x[8 + e] * inv * w1[e];
      const float co = cs[2 * e], si = cs[2 * e + 1];
      x[e] = fmaf(a, co, -b * si);
      x[8 + e] = fmaf(b, co, a * si);
    }
  }
}

// Raw k/v rows and rotary factors of one own-key chunk, held in registers
// between the prefetch and the LDS stage.  NSUB = D/16 threads share a key:
// thread t handles key kk = (t / NSUB) % 32, head dims 8*sub..8*sub+7
// (sub = t % NSUB) and their rotate-half partners D/2+8*sub..D/2+8*sub+7,
// so a role takes 2*D threads.  When the block has 4*D threads or more the
// first 2*D stage k^ and the next 2*D stage v (one register set, two
// roles); otherwise (4 waves at D = 128) each of the first 2*D threads
// stages both.
template <int WAVES, int D>
struct OwnGeo {
  static constexpr int NSUB = D / 16;
  static constexpr int ROLE = 2 * D;
  static constexpr bool SPLIT = WAVES * 64 >= 2 * ROLE;
  static constexpr int ACTIVE = SPLIT ? 2 * ROLE : ROLE;
};

struct OwnRegs {
  uint4 a0, a1;            // k (or v in the value role)
  uint4 b0, b1;            // v when one thread has both roles
  float4 r0, r1, r2, r3;   // (cos, sin) of the key's position
  bool valid;
};

template <int WAVES, int D>
__device__ __forceinline__ bool key_role() {
  return !OwnGeo<WAVES, D>::SPLIT || threadIdx.x < OwnGeo<WAVES, D>::ROLE;
}
template <int WAVES, int D>
__device__ __forceinline__ bool value_role() {
  return !OwnGeo<WAVES, D>::SPLIT || threadIdx.x >= OwnGeo<WAVES, D>::ROLE;
}

template <int WAVES, int D>
__device__ __forceinline__ void own_load(const AttnParams &P, const OwnStep &o,
                                         int g, int L, OwnRegs &r) {
  using Geo = OwnGeo<WAVES, D>;
  // thread indices are recomputed here (opaque offset) rather than hoisted
  // out of the kernel's loops with their derived addresses
  const int t = threadIdx.x + opaque_zero();
  const int kk = ((unsigned)t / Geo::NSUB) & 31, sub = (unsigned)t % Geo::NSUB;
  const int jk = o.c0 + kk;
  r.valid = t < Geo::ACTIVE && jk < o.T;
  if (r.valid) {
    const int64_t off = ((int64_t)(o.tok0 + jk) * P.Hkv + g) * D;
    if (key_role<WAVES, D>()) {
      r.a0 = *reinterpret_cast<const uint4 *>(P.k + off + 8 * sub);
      r.a1 = *reinterpret_cast<const uint4 *>(P.k + off + D / 2 + 8 * sub);
      const float4 *cq = reinterpret_cast<const float4 *>(
          P.rope + (int64_t)(L + jk) * (D / 2) + 8 * sub);
      r.r0 = cq[0];
      r.r1 = cq[1];
      r.r2 = cq[2];
      r.r3 = cq[3];
    }
    if (!Geo::SPLIT) {
      r.b0 = *reinterpret_cast<const uint4 *>(P.v + off + 8 * sub);
      r.b1 = *reinterpret_cast<const uint4 *>(P.v + off + D / 2 + 8 * sub);
    } else if (value_role<WAVES, D>()) {
      r.a0 = *reinterpret_cast<const uint4 *>(P.v + off + 8 * sub);
      r.a1 = *reinterpret_cast<const uint4 *>(P.v + off + D / 2 + 8 * sub);
    }
  }
}

// k^ = RoPE(RMSNorm(k) * w) into sm.ok; v transposed into sm.ov.  Rows of
// keys past the pair's end are zero.
template <int WAVES, int D, int NCHK>
__device__ __forceinline__ void own_stage(const AttnParams &P,
                                          const OwnRegs &r,
                                          Smem<D, NCHK> &sm, int buf) {
  using Geo = OwnGeo<WAVES, D>;
  if (threadIdx.x >= Geo::ACTIVE) return;
  const int t = threadIdx.x + opaque_zero();
  const int kk = ((unsigned)t / Geo::NSUB) & 31, sub = (unsigned)t % Geo::NSUB;
  if (key_role<WAVES, D>()) {
    // the gains first: their load overlaps the norm's reduction
    const uint4 g0 = *reinterpret_cast<const uint4 *>(P.kw + 8 * sub);
    const uint4 g1 =
        *reinterpret_cast<const uint4 *>(P.kw + D / 2 + 8 * sub);
    float x[16];
    khat_part<D>(r.a0, r.a1, g0, g1, r.r0, r.r1, r.r2, r.r3, r.valid, P.eps,
                 P.norm != 0, x);
    *reinterpret_cast<uint4 *>(sm.ok[buf] + kc_off<D>(kk, sub)) =
        as_uint4(to_bf16x8(x));
    *reinterpret_cast<uint4 *>(sm.ok[buf] + kc_off<D>(kk, sub + Geo::NSUB)) =
        as_uint4(to_bf16x8(x + 8));
  }
  if (value_role<WAVES, D>()) {
    // a pure transpose: the bf16 halves are stored as they are (keys past
    // the pair's end are written as zeros)
    const uint4 &v0 = Geo::SPLIT ? r.a0 : r.b0;
    const uint4 &v1 = Geo::SPLIT ? r.a1 : r.b1;
    const uint32_t h[8] = {r.valid ? v0.x : 0u, r.valid ? v0.y : 0u,
                           r.valid ? v0.z : 0u, r.valid ? v0.w : 0u,
                           r.valid ? v1.x : 0u, r.valid ? v1.y : 0u,
                           r.valid ? v1.z : 0u, r.valid ? v1.w : 0u};
    // rows d = 8*sub + e and D/2 + 8*sub + e, column kk: the swizzle of
    // row d depends only on e >= 4 and sub (not on adding D/2), so two base
    // addresses serve all 16 stores (the rest are constant offsets)
    const int gr = kk >> 3, in = kk & 7;
    uint16_t *ov = sm.ov[buf];
    const int b0 = vc_off(8 * sub, gr) + in, b1 = vc_off(8 * sub + 4, gr) + in;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int base = (e < 4 ? b0 + e * KC : b1 + (e - 4) * KC);
      const uint32_t lo = h[e >> 1], hi = h[4 + (e >> 1)];
      ov[base] = (uint16_t)((e & 1) ? lo >> 16 : lo);
      ov[base + (D / 2) * KC] = (uint16_t)((e & 1) ? hi >> 16 : hi);
    }
  }
}

// Softmax state of one query block (per lane: one query column), log2
// units.  m is the reference subtracted from the logits: 0 in mode 0; in
// mode 1 fixed at the first visible chunk (+inf before); in mode 2 (SAFE)
// the running maximum (-inf before).
template <int D>
struct Acc {
  floatx16 o[D / 32];
  float m, l;
};

// Per-lane element offsets of the MFMA A-operand fragments inside a chunk
// block, the same for every chunk: K fragment s (k-step s: head dims
// 16s + 8hf .. + 7 of key row perm32(lq)) and V^T fragment f = (db, t)
// (head-dim row 32db + perm32(lq), keys 16hf + 8t .. + 7).  The V^T
// offsets differ by whole rows across db, so two registers hold them.
template <int D>
struct Frag {
  int k[D / 16], v[2];
};
template <int D>
__device__ __forceinline__ Frag<D> frag_offsets(int lq, int hf) {
  Frag<D> f;
  const int row = perm32(lq);
#pragma unroll
  for (int s = 0; s < D / 16; ++s) f.k[s] = kc_off<D>(row, 2 * s + hf);
  f.v[0] = vc_off(row, 2 * hf);
  f.v[1] = vc_off(row, 2 * hf + 1);
  return f;
}

// K fragments are read RA at a time ahead of the QK products, and V^T
// fragments RA at a time ahead of the PV products, so LDS latency overlaps
// MFMA and VALU work (RA trades registers for latency hiding).
constexpr int RA = 4;

// S^T = K Q^T for one 32-key chunk (logits in log2 units: q^ carries the
// scale).
template <int NQB, int D>
__device__ __forceinline__ void qk_part(const uint16_t *kblk,
                                        const Frag<D> &fo,
                                        const bf16x8 (*qf)[D / 16],
                                        floatx16 *S) {
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
    for (int i = 0; i < 16; ++i) S[qb][i] = 0.f;
#pragma unroll
  for (int s0 = 0; s0 < D / 16; s0 += RA) {
    bf16x8 kf[RA];
#pragma unroll
    for (int s = 0; s < RA; ++s)
      kf[s] = *reinterpret_cast<const bf16x8 *>(kblk + fo.k[s0 + s]);
#pragma unroll
    for (int s = 0; s < RA; ++s)
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb)
        S[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[qb][s0 + s],
                                                        S[qb], 0, 0, 0);
  }
}

// V^T fragments f0 .. f0 + RA - 1 of a chunk, f = (db, t).
template <int D>
__device__ __forceinline__ void v_read(const uint16_t *vblk,
                                       const Frag<D> &fo, int f0,
                                       bf16x8 *vf) {
#pragma unroll
  for (int f = f0; f < f0 + RA; ++f)
    vf[f - f0] = *reinterpret_cast<const bf16x8 *>(
        vblk + (f >> 1) * (32 * KC) + fo.v[f & 1]);
}

// Weights of one chunk's logits into pb (bf16), updating each row's
// normaliser (and reference, rescaling O, in modes 1 and 2).
// MODE 0: no mask; MODE 1: key index (0..31 within the chunk) must be
// <= lim[qb] (a per-row limit, < 0 hides every key of the chunk).
// SMX 0: weights exp2(S); 1: exp2(S - m), m fixed at the first visible
// chunk to min(B, max + 80); 2: exact running maximum.
template <int MODE, int NQB, int SMX, int D>
__device__ __forceinline__ void softmax_part(floatx16 *S, Acc<D> *acc, int hf,
                                             float B, const int *lim,
                                             bf16x8 (*pb)[2]) {
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    if (MODE == 1) {
      // key 16 hf + i is visible when i <= lim - 16 hf (comparing the
      // immediate i, so no register holds each lane's key indices)
      const int li = lim[qb] - 16 * hf;
#pragma unroll
      for (int i = 0; i < 16; ++i) S[qb][i] = i <= li ? S[qb][i] : -INFINITY;
    }
    Acc<D> &A = acc[qb];
    if (SMX == 2) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[qb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const bool need = mx > A.m + kTau;
      const float mnew = need ? mx : A.m;
      const float alpha = need ? __builtin_amdgcn_exp2f(A.m - mnew) : 1.0f;
      A.l *= alpha;
      A.m = mnew;
      if (__any(need)) {
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) A.o[db][i] *= alpha;
      }
    } else if (SMX == 1 && __any(A.m == INFINITY)) {
      // first chunk with visible keys: fix the row's reference
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[qb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (A.m == INFINITY && mx > -INFINITY) A.m = fminf(B, mx + kHeadroom);
    }
    float p[16];
    if (SMX == 0) {
#pragma unroll
      for (int i = 0; i < 16; ++i) p[i] = __builtin_amdgcn_exp2f(S[qb][i]);
    } else {
      const float muse = A.m == -INFINITY || A.m == INFINITY ? 0.f : A.m;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        p[i] = __builtin_amdgcn_exp2f(S[qb][i] - muse);
    }
    pb[qb][0] = to_bf16x8(p);
    pb[qb][1] = to_bf16x8(p + 8);
    // The normaliser sums the same bf16 weights the PV product uses, two at
    // a time (v_dot2 with (1, 1)), so the output is an exact weighted mean.
    const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8 &w = pb[qb][t];
      A.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 0, 1),
                                            one, A.l, false);
      A.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 2, 3),
                                            one, A.l, false);
      A.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 4, 5),
                                            one, A.l, false);
      A.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 6, 7),
                                            one, A.l, false);
    }
  }
}

// O^T += V^T P^T for one chunk; vf holds the first RA V^T fragments.
template <int NQB, int D>
__device__ __forceinline__ void pv_part(const uint16_t *vblk,
                                        const Frag<D> &fo, bf16x8 *vf,
                                        Acc<D> *acc, const bf16x8 (*pb)[2]) {
#pragma unroll
  for (int f0 = 0; f0 < D / 16; f0 += RA) {
    if (f0 > 0) v_read(vblk, fo, f0, vf);
#pragma unroll
    for (int f = f0; f < f0 + RA; ++f)
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb)
        acc[qb].o[f >> 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            vf[f - f0], pb[qb][f & 1], acc[qb].o[f >> 1], 0, 0, 0);
  }
}

// One 32-key chunk for NQB query blocks: S^T = K Q^T, weights, O^T += V^T P^T
// (the first V^T fragments are read before the weights are formed).
template <int MODE, int NQB, int SMX, int D>
__device__ __forceinline__ void attend(const uint16_t *kblk,
                                       const uint16_t *vblk,
                                       const Frag<D> &fo,
                                       const bf16x8 (*qf)[D / 16],
                                       Acc<D> *acc, int hf, float B,
                                       const int *lim) {
  floatx16 S[NQB];
  qk_part<NQB, D>(kblk, fo, qf, S);
  bf16x8 vf[RA];
  v_read<D>(vblk, fo, 0, vf);
  bf16x8 pb[NQB][2];
  softmax_part<MODE, NQB, SMX, D>(S, acc, hf, B, lim, pb);
  pv_part<NQB, D>(vblk, fo, vf, acc, pb);
}

}  // namespace
}  // namespace dopr

// attn.hip -- online prefix attention of DoPR on gfx950 (MFMA bf16).
//
// Online reranking injects a document's stored prefix states as a
// pre-filled K/V cache and runs only the query and score tokens (Sec. 3.4);
// those tokens see the document only through its prefix states and attend
// causally among themselves (Sec. 3.2.2).  Per layer and kv head g:
//   out[j,h] = softmax(scale * q^[j,h] . [K_d[g] ; k^[0..j,g]]) . [V_d[g] ; v[0..j,g]]
// with q^/k^ the per-head RMS-normed, rotary-embedded online projections at
// positions L_d + j.
//
// Work decomposition.  The scheduler (group.hip) orders pairs by document
// and cuts each document's stacked rows (token j x q-head of the kv group,
// token-major) into work items.  A workgroup takes one (item, kv head) from
// an XCD-local queue.  Every row of an item shares the document, so the
// document's prefix for head g (up to 256 slots: K 64 KB + V^T 64 KB) is
// staged in LDS once per item, with direct global->LDS loads, and every pass
// of every wave reads it from there with no barrier: one HBM read of the
// prefix per document group, reused on-chip across all the queries that
// retrieved the document.  Longer prefixes are streamed through the same
// buffer in 256-slot segments.  A pass gives each wave NQB x 32 rows; the
// rows' own keys are normed/rotated cooperatively into a small LDS chunk
// (the next chunk's raw k/v is prefetched into registers while the current
// one is consumed) and masked per row: same pair and key <= row.
//
// MFMA orientation (v_mfma_f32_32x32x16_bf16, A 32x16, B 16x32, C 32x32):
//   S^T[key][q] = K[key][:] . Q^T[:][q]    A = K (LDS), B = Q^T (registers)
//   O^T[d][q]  += V^T[d][key] . P^T[key][q] A = V^T (LDS), B = P^T (registers)
// A lane owns one query column, so row statistics are lane-local plus one
// exchange with lane ^ 32 and the probabilities feed PV without a transpose.
// A-operand rows are read in the order perm32(m) so lane half hf's 16
// accumulator registers hold 16 consecutive keys (S) or head dims (O):
// key = 16*hf + i, d = 32*db + 16*hf + i.  With NQB = 2 every K/V fragment
// read from LDS feeds two MFMAs.
//
// Softmax without a running maximum.  Every key a row can see has a known
// norm bound (stored prefix keys: a per-slice maximum written when the store
// is filled; own keys: an RMS-normed vector has norm <= sqrt(D), times the
// largest gain), so by Cauchy-Schwarz the row's scaled logits are <= a bound
// B.  The row uses the fixed reference m = min(B, first chunk's max + 80) (in
// log2 units): exp2(s*c - m) is then never large, and the row's largest term
// is >= 2^-80, so the normaliser l = sum exp2(...) stays in a safe range
// without the per-chunk max reduction and accumulator rescale of the usual
// online softmax.  A work unit in which some row ends with l outside
// [2^-90, 2^100] (only possible for extreme key norms) is queued and
// recomputed by a second launch of the same kernel in SAFE mode, which
// tracks the running max exactly.
#include <cmath>

#include "internal.hpp"

namespace dopr {

int64_t *plan_totals(const Plan &pl);
int32_t *plan_next(const Plan &pl);

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int D = kHeadDim;
constexpr int KC = 32;      // keys per MFMA chunk
constexpr int PSEG = 256;   // prefix slots resident in LDS at once
constexpr int kTotItems = 2;
constexpr int kFixQueue = 8;  // cursor slot of the fixup pass
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kTau = 8.0f;       // SAFE mode: lazy-rescale threshold
constexpr float kHeadroom = 80.f;  // reference <= first max + 80 (log2)
constexpr float kLoOk = 0x1p-90f, kHiOk = 0x1p100f;

struct AttnParams {
  const uint16_t *q, *k, *v, *qw, *kw;
  const int32_t *cu;
  const int32_t *doc_len;
  const int64_t *doc_off;
  const float *kmax;
  const uint16_t *payload;
  const int32_t *pair_order, *group_doc, *group_ptr, *blk_pair;
  const int64_t *prow;
  const int4 *items;
  const int64_t *totals;
  int32_t *next;
  int32_t *counters;
  int32_t *fix;
  const float *kown;
  const float2 *rope;
  uint16_t *out;
  float *lse;
  int32_t items_cap, Hq, Hkv, n_rep, layer, n_layers;
  int32_t flag_all;  // queue every unit for the SAFE pass (self-check mode)
  float eps, c;      // c = softmax_scale * log2(e)
};

// 160 KB: the whole LDS of a CU.  The own-key chunk is double-buffered; at
// item boundaries (no own chunk in flight) its first words carry the work
// index broadcast and the per-wave overflow flags.
struct Smem {
  uint16_t pk[PSEG * D];      // prefix K   [key][D]    (granules swizzled)
  uint16_t pvt[D * PSEG];     // prefix V^T [d][key]    (row stride PSEG)
  uint16_t ok[2][KC * D];     // own k^     [key][D]
  uint16_t ovt[2][D * KC];    // own v^T    [d][key]
  __device__ int *words() { return reinterpret_cast<int *>(ok[0]); }
};

__device__ __forceinline__ int perm32(int m) {
  return ((m >> 2) & 1) * 16 + (m >> 3) * 4 + (m & 3);
}
// XOR swizzle of 16-byte granules: the 16 rows read together by a half
// wave (perm32 of lanes 0..15 or 16..31) land on 16 distinct bank groups.
__device__ __forceinline__ int swz(int row) {
  return (row & 3) | ((row >> 2) & 4) | ((row << 1) & 8);
}
__device__ __forceinline__ int swz_v(int row) {
  return ((row >> 2) & 1) | ((row >> 3) & 2);
}
__device__ __forceinline__ int pk_off(int key, int gr) {
  return key * D + ((gr ^ swz(key & 31)) << 3);
}
__device__ __forceinline__ int pvt_off(int d, int gr) {
  return d * PSEG + ((gr ^ swz(d & 31)) << 3);
}
__device__ __forceinline__ int ok_off(int key, int gr) {
  return key * D + ((gr ^ swz(key)) << 3);
}
__device__ __forceinline__ int ovt_off(int d, int gr) {
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

// Sorted pair owning stacked row r: the owner of r's 32-row block, then a
// short forward scan.
__device__ __forceinline__ int find_pair(const AttnParams &P, int r) {
  int s = P.blk_pair[r >> 5];
  while (P.prow[s + 1] <= r) ++s;
  return s;
}

struct RowInfo {
  int64_t tok;
  int32_t s, j, head;
  bool valid;
};

// q^ = RoPE_pos(RMSNorm(q) * w) in the B-operand layout: lane half hf holds
// head dims 16*s + 8*hf + e of its query column (k-step s = 0..7); the
// rotate-half partner of dim i < 64 is dim i + 64 = k-step s + 4, same lane.
// Returns an upper bound on |q^| after rounding to bf16.
__device__ __forceinline__ float q_fragments(const uint16_t *qrow,
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
  float n2 = 0.f;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const float4 *cs4 =
        reinterpret_cast<const float4 *>(rope_row + 16 * s + 8 * hf);
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const float4 t = cs4[e2];  // (cos, sin) of dims 2*e2 and 2*e2 + 1
      const int e = 2 * e2;
      float a = x[s][e], b = x[s + 4][e];
      x[s][e] = fmaf(a, t.x, -b * t.y);
      x[s + 4][e] = fmaf(b, t.x, a * t.y);
      n2 = fmaf(a, a, fmaf(b, b, n2));  // rotation preserves the norm
      a = x[s][e + 1];
      b = x[s + 4][e + 1];
      x[s][e + 1] = fmaf(a, t.z, -b * t.w);
      x[s + 4][e + 1] = fmaf(b, t.z, a * t.w);
      n2 = fmaf(a, a, fmaf(b, b, n2));
    }
  }
#pragma unroll
  for (int s = 0; s < 8; ++s) qf[s] = to_bf16x8(x[s]);
  n2 += __shfl_xor(n2, 32, 64);
  return sqrtf(n2) * 1.01f;  // bf16 rounding (2^-8) and fp32 slack
}

// Stage prefix slots [seg0, seg0 + n) of kv head g into LDS with direct
// global->LDS loads (no registers): lane i of a wave writes bytes
// [16i, 16i+16) of the wave's 1 KB LDS block, so each lane fetches the
// global granule that the swizzled layout puts in its slot.  K rows past n
// are left stale (their logits are masked by a select).  V^T columns from
// Lp up to the next multiple of 32 are zeroed (masked keys must multiply a
// finite value); the store's own pad columns [L, Lp) are zero already.
template <int WAVES>
__device__ __forceinline__ void stage_prefix(const uint16_t *Kp,
                                             const uint16_t *VTp, int Lp,
                                             int seg0, int n, Smem &sm) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // K: 1 KB block b = rows 4b..4b+3, lane -> (row, physical granule)
  const int kblocks = (n + 3) >> 2;
  for (int b = wave; b < kblocks; b += WAVES) {
    const int r = 4 * b + (lane >> 4), p = lane & 15;
    if (r < n) {
      const int gr = p ^ swz(r & 31);
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void *)(
              Kp + (int64_t)(seg0 + r) * D + gr * 8),
          (__attribute__((address_space(3))) void *)(sm.pk + b * 512), 16, 0,
          0);
    }
  }
  // V^T: 1 KB block b = rows d = 2b, 2b+1 (32 granules of 8 keys each)
  const int lp = Lp - seg0 < PSEG ? Lp - seg0 : PSEG;  // stored columns
  const int gl = lp >> 3;
  for (int b = wave; b < D / 2; b += WAVES) {
    const int d = 2 * b + (lane >> 5), p = lane & 31;
    const int gr = p ^ swz(d & 31);
    if (gr < gl)
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void *)(
              VTp + (int64_t)d * Lp + seg0 + 8 * gr),
          (__attribute__((address_space(3))) void *)(sm.pvt + b * 512), 16,
          0, 0);
  }
  const int gc = ((n + 31) & ~31) >> 3;  // granules through the chunk end
  for (int e = threadIdx.x; e < D * 4; e += WAVES * 64) {
    const int d = e >> 2, gr = gl + (e & 3);
    if (gr < gc)
      *reinterpret_cast<uint4 *>(sm.pvt + pvt_off(d, gr)) =
          make_uint4(0, 0, 0, 0);
  }
}

// Wait for this wave's direct-to-LDS (and other vector-memory) loads.
__device__ __forceinline__ void wait_vmem() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Own-key chunk: raw k/v rows and rotary factors of 32 online tokens of one
// pair, held in registers between the prefetch and the LDS stage.  Thread
// (kk = t / 8, sub = t % 8) of the first 256 threads handles head dims
// 8*sub..8*sub+7 and their rotate-half partners 64+8*sub..64+8*sub+7.
struct OwnRegs {
  uint4 k0, k1, v0, v1;
  float4 r0, r1, r2, r3;
  bool valid;
};

struct OwnStep {
  int s;      // sorted pair index
  int c0;     // first own key of the chunk
  int pr;     // pair index
  int64_t tok0;
  int T;
};

__device__ __forceinline__ void own_load(const AttnParams &P, const OwnStep &o,
                                         int g, int L, OwnRegs &r) {
  const int kk = (threadIdx.x >> 3) & 31, sub = threadIdx.x & 7;
  const int jk = o.c0 + kk;
  r.valid = threadIdx.x < 256 && jk < o.T;
  if (r.valid) {
    const int64_t off = ((o.tok0 + jk) * P.Hkv + g) * (int64_t)D;
    r.k0 = *reinterpret_cast<const uint4 *>(P.k + off + 8 * sub);
    r.k1 = *reinterpret_cast<const uint4 *>(P.k + off + 64 + 8 * sub);
    r.v0 = *reinterpret_cast<const uint4 *>(P.v + off + 8 * sub);
    r.v1 = *reinterpret_cast<const uint4 *>(P.v + off + 64 + 8 * sub);
    const float4 *cq = reinterpret_cast<const float4 *>(
        P.rope + (int64_t)(L + jk) * kRopeHalf + 8 * sub);
    r.r0 = cq[0];
    r.r1 = cq[1];
    r.r2 = cq[2];
    r.r3 = cq[3];
  }
}

// k^ = RoPE(RMSNorm(k) * w) into sm.ok; v transposed into sm.ovt.  Rows of
// keys past the pair's end are zero.
__device__ __forceinline__ void own_stage(const AttnParams &P,
                                          const OwnRegs &r, Smem &sm,
                                          int buf) {
  if (threadIdx.x >= 256) return;
  const int kk = threadIdx.x >> 3, sub = threadIdx.x & 7;
  float x[16], vv[16];
  if (r.valid) {
    unpack8(r.k0, x);
    unpack8(r.k1, x + 8);
    unpack8(r.v0, vv);
    unpack8(r.v1, vv + 8);
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) x[e] = vv[e] = 0.f;
  }
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < 16; ++e) ss = fmaf(x[e], x[e], ss);
  ss += __shfl_xor(ss, 1, 64);
  ss += __shfl_xor(ss, 2, 64);
  ss += __shfl_xor(ss, 4, 64);
  if (r.valid) {
    const float inv = rsqrtf(ss * (1.0f / D) + P.eps);
    float w0[8], w1[8];
    unpack8(*reinterpret_cast<const uint4 *>(P.kw + 8 * sub), w0);
    unpack8(*reinterpret_cast<const uint4 *>(P.kw + 64 + 8 * sub), w1);
    const float cs[16] = {r.r0.x, r.r0.y, r.r0.z, r.r0.w, r.r1.x, r.r1.y,
                          r.r1.z, r.r1.w, r.r2.x, r.r2.y, r.r2.z, r.r2.w,
                          r.r3.x, r.r3.y, r.r3.z, r.r3.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float a = x[e] * inv * w0[e], b = x[8 + e] * inv * w1[e];
      const float co = cs[2 * e], si = cs[2 * e + 1];
      x[e] = fmaf(a, co, -b * si);
      x[8 + e] = fmaf(b, co, a * si);
    }
  }
  *reinterpret_cast<uint4 *>(sm.ok[buf] + ok_off(kk, sub)) =
      as_uint4(to_bf16x8(x));
  *reinterpret_cast<uint4 *>(sm.ok[buf] + ok_off(kk, sub + 8)) =
      as_uint4(to_bf16x8(x + 8));
  const bf16x8 v0 = to_bf16x8(vv), v1 = to_bf16x8(vv + 8);
  const int gr = kk >> 3, in = kk & 7;
  __bf16 *ovt = reinterpret_cast<__bf16 *>(sm.ovt[buf]);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    ovt[ovt_off(8 * sub + e, gr) + in] = v0[e];
    ovt[ovt_off(64 + 8 * sub + e, gr) + in] = v1[e];
  }
}

// Softmax state of one query block (per lane: one query column).
//   fast mode: m = fixed reference (+inf until the row sees a key), mb = the
//   row's logit bound (log2 units);  SAFE mode: m = running reference.
struct Acc {
  floatx16 o[4];
  float m, l, mb;
};

// MODE 0: interior prefix chunk (no mask); 1: last prefix chunk (keys >=
// lim masked); 2: own-key chunk (same pair and key <= row).
template <int MODE, int NQB, bool SAFE>
__device__ __forceinline__ void attend(const uint16_t *kbase, int krow0,
                                       const uint16_t *vt_rows, bool own_lds,
                                       int vt_gr0, const bf16x8 (*qf)[8],
                                       Acc *acc, int lq, int hf, float c,
                                       int key0, int lim, const RowInfo *ri,
                                       int s_cur) {
  const int krow = perm32(lq);
  // K fragments are read RA at a time ahead of the QK products, and the
  // first RA V^T fragments before the softmax, so LDS latency overlaps MFMA
  // and VALU work instead of stalling each product (the sched barriers pin
  // the order; RA trades registers for latency hiding).
  constexpr int RA = NQB == 2 ? 8 : 4;
  floatx16 S[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
    for (int i = 0; i < 16; ++i) S[qb][i] = 0.f;
#pragma unroll
  for (int s0 = 0; s0 < 8; s0 += RA) {
    bf16x8 kf[RA];
#pragma unroll
    for (int s = 0; s < RA; ++s) {
      const int gr = 2 * (s0 + s) + hf;
      const int off = own_lds ? ok_off(krow, gr) : pk_off(krow0 + krow, gr);
      kf[s] = *reinterpret_cast<const bf16x8 *>(kbase + off);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < RA; ++s)
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb)
        S[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[qb][s0 + s],
                                                        S[qb], 0, 0, 0);
  }
  const int vrow = perm32(lq);
  bf16x8 vf[8];
  auto vread = [&](int f) {  // fragment f = (db, t) = (f / 2, f % 2)
    const int d = 32 * (f >> 1) + vrow;
    const int gr = vt_gr0 + 2 * hf + (f & 1);
    const int off = own_lds ? ovt_off(d, gr) : pvt_off(d, gr);
    vf[f] = *reinterpret_cast<const bf16x8 *>(vt_rows + off);
  };
#pragma unroll
  for (int f = 0; f < RA; ++f) vread(f);
  __builtin_amdgcn_sched_barrier(0);
  bf16x8 pb[NQB][2];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    if (MODE != 0) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = key0 + 16 * hf + i;
        const bool ok = MODE == 1 ? key < lim
                                  : (ri[qb].s == s_cur && key <= ri[qb].j);
        S[qb][i] = ok ? S[qb][i] : -INFINITY;
      }
    }
    Acc &A = acc[qb];
    if (SAFE) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[qb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mxs = mx * c;
      const bool need = mxs > A.m + kTau;
      const float mnew = need ? mxs : A.m;
      const float alpha = need ? __builtin_amdgcn_exp2f(A.m - mnew) : 1.0f;
      A.l *= alpha;
      A.m = mnew;
      if (__any(need)) {
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) A.o[db][i] *= alpha;
      }
    } else if (__any(A.m == INFINITY)) {
      // first chunk with visible keys: fix the row's reference
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[qb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (A.m == INFINITY && mx > -INFINITY)
        A.m = fminf(A.mb, fmaf(mx, c, kHeadroom));
    }
    const float muse = A.m == -INFINITY ? 0.f : A.m;
    float p[16];
#pragma unroll
    for (int i = 0; i < 16; ++i)
      p[i] = __builtin_amdgcn_exp2f(fmaf(S[qb][i], c, -muse));
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
#pragma unroll
  for (int f = 0; f < 8; ++f) {
    if (f + RA < 8 && f % RA == 0) {
#pragma unroll
      for (int g2 = 0; g2 < RA; ++g2) vread(f + RA + g2);
    }
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb)
      acc[qb].o[f >> 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          vf[f], pb[qb][f & 1], acc[qb].o[f >> 1], 0, 0, 0);
  }
}

template <int WAVES, int NQB, bool SAFE>
__global__ __launch_bounds__(WAVES * 64) __attribute__((
    amdgpu_waves_per_eu(WAVES / 4, WAVES / 4))) void k_prefix_attn(AttnParams P) {
  constexpr int PASS = WAVES * NQB * 32;
  __shared__ __attribute__((aligned(16))) Smem sm;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lq = lane & 31, hf = lane >> 5;
  const int queue = SAFE ? kFixQueue : (blockIdx.x & 7);
  int64_t n_work;
  if (SAFE) {
    n_work = P.counters[kCntFix];
  } else {
    int64_t n_items = P.totals[kTotItems];
    if (n_items > P.items_cap) n_items = P.items_cap;
    n_work = n_items * P.Hkv;
  }
  const float kown = *P.kown;

  for (;;) {
    if (threadIdx.x == 0) sm.words()[0] = atomicAdd(&P.next[queue], 1);
    __syncthreads();
    const int slot = sm.words()[0];
    int64_t w = SAFE ? (int64_t)slot : queue + 8 * (int64_t)slot;
    if (w >= n_work) break;
    bool wave_bad = false;
    if (SAFE) w = P.fix[w];
    const int item = (int)(w / P.Hkv), g = (int)(w % P.Hkv);
    const int4 it = P.items[item];
    const int group = it.x, row0 = it.y, row1 = it.z;
    const int doc = P.group_doc[group];
    const int L = P.doc_len[doc], Lp = pad8(L);
    const int64_t blk = P.doc_off[doc];
    const uint16_t *Kp = P.payload + k_offset(blk, L, P.Hkv, P.layer, g);
    const uint16_t *VTp = P.payload + vt_offset(blk, L, P.Hkv, P.layer, g);
    const float kbound = fmaxf(
        kown, P.kmax[((int64_t)doc * P.n_layers + P.layer) * P.Hkv + g]);
    const int n_seg = (L + PSEG - 1) / PSEG;
    const bool resident = n_seg <= 1;
    if (resident && L > 0) stage_prefix<WAVES>(Kp, VTp, Lp, 0, L, sm);

    for (int pass0 = row0; pass0 < row1; pass0 += PASS) {
      const int pass_end = pass0 + PASS < row1 ? pass0 + PASS : row1;
      RowInfo ri[NQB];
      bf16x8 qf[NQB][8];
      Acc acc[NQB];
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        const int r = pass0 + (wave * NQB + qb) * 32 + lq;
        ri[qb].valid = r < row1;
        const int rc = ri[qb].valid ? r : row1 - 1;
        const int s = find_pair(P, rc);
        const int pr = P.pair_order[s];
        const int rr = rc - (int)P.prow[s];
        const int j = rr / P.n_rep, rep = rr - j * P.n_rep;
        ri[qb].s = s;
        ri[qb].j = j;
        ri[qb].tok = (int64_t)P.cu[pr] + j;
        ri[qb].head = g * P.n_rep + rep;
        const float qn = q_fragments(
            P.q + (ri[qb].tok * P.Hq + ri[qb].head) * D, P.qw,
            P.rope + (int64_t)(L + j) * kRopeHalf, hf, P.eps, qf[qb]);
        __builtin_amdgcn_sched_barrier(0);
        acc[qb].m = SAFE ? -INFINITY : INFINITY;
        acc[qb].mb = qn * kbound * P.c * 1.001f;
        acc[qb].l = 0.f;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[qb].o[db][i] = 0.f;
      }

      const int s_lo = find_pair(P, pass0);
      const int s_hi = find_pair(P, pass_end - 1);
      OwnStep os;
      os.s = s_lo;
      os.c0 = 0;
      os.pr = P.pair_order[s_lo];
      os.tok0 = P.cu[os.pr];
      os.T = P.cu[os.pr + 1] - P.cu[os.pr];
      OwnRegs orr;
      if (n_seg == 0) own_load(P, os, g, L, orr);

      // Document prefix: every row sees all L slots.
      for (int sg = 0; sg < n_seg; ++sg) {
        const int seg0 = sg * PSEG;
        const int n = L - seg0 < PSEG ? L - seg0 : PSEG;
        if (!resident) {
          __syncthreads();
          stage_prefix<WAVES>(Kp, VTp, Lp, seg0, n, sm);
        }
        wait_vmem();
        __syncthreads();
        // the first own chunk lands while the prefix is consumed
        if (sg == 0) own_load(P, os, g, L, orr);
        const int n_full = n >> 5;
        for (int ck = 0; ck < n_full; ++ck)
          attend<0, NQB, SAFE>(sm.pk, ck * KC, sm.pvt, false, ck * 4, qf, acc,
                               lq, hf, P.c, 0, 0, ri, 0);
        if (n & 31)
          attend<1, NQB, SAFE>(sm.pk, n_full * KC, sm.pvt, false, n_full * 4,
                               qf, acc, lq, hf, P.c, n_full * KC, n, ri, 0);
      }

      // Own causal keys, pair by pair, chunk by chunk, double-buffered: the
      // next chunk's raw k/v are loaded while the current one is consumed,
      // then normed/rotated into the other buffer; one barrier per chunk.
      __syncthreads();  // the previous pass's last own chunk is consumed
      own_stage(P, orr, sm, 0);
      __syncthreads();
      int buf = 0;
      while (os.s <= s_hi) {
        // next step: next chunk of this pair, else first chunk of the next
        const int64_t srow0 = P.prow[os.s], srow1 = P.prow[os.s + 1];
        const int64_t hi_row = (srow1 < pass_end ? srow1 : pass_end) - 1;
        const int jmax = (int)((hi_row - srow0) / P.n_rep);
        OwnStep nx = os;
        if (os.c0 + KC <= jmax) {
          nx.c0 = os.c0 + KC;
        } else {
          nx.s = os.s + 1;
          nx.c0 = 0;
          if (nx.s <= s_hi) {
            nx.pr = P.pair_order[nx.s];
            nx.tok0 = P.cu[nx.pr];
            nx.T = P.cu[nx.pr + 1] - P.cu[nx.pr];
          }
        }
        const bool more = nx.s <= s_hi;
        if (more) own_load(P, nx, g, L, orr);
        bool need = false;
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb)
          need = need || (ri[qb].s == os.s && ri[qb].j >= os.c0);
        if (__any(need))  // wave-uniform: skip chunks no row of the wave sees
          attend<2, NQB, SAFE>(sm.ok[buf], 0, sm.ovt[buf], true, 0, qf, acc,
                               lq, hf, P.c, os.c0, 0, ri, os.s);
        if (more) own_stage(P, orr, sm, buf ^ 1);
        __syncthreads();
        buf ^= 1;
        os = nx;
      }

      // Normalise; write O (bf16) and the natural-log LSE.
      bool bad = false;
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        const float lt = acc[qb].l + __shfl_xor(acc[qb].l, 32, 64);
        if (!ri[qb].valid) continue;
        bad = bad || !(lt >= kLoOk && lt <= kHiOk);
        const float inv = 1.0f / lt;
        uint16_t *orow = P.out + (ri[qb].tok * P.Hq + ri[qb].head) * D;
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          float o[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) o[i] = acc[qb].o[db][i] * inv;
          uint4 *dst = reinterpret_cast<uint4 *>(orow + 32 * db + 16 * hf);
          dst[0] = as_uint4(to_bf16x8(o));
          dst[1] = as_uint4(to_bf16x8(o + 8));
        }
        if (P.lse && hf == 0)
          P.lse[ri[qb].tok * P.Hq + ri[qb].head] =
              (acc[qb].m + __log2f(lt)) * kLn2;
      }
      wave_bad = wave_bad || __any(bad) || P.flag_all;
    }
    __syncthreads();  // every wave is done with this item's LDS
    if (!SAFE) {
      if (lane == 0) sm.words()[1 + wave] = wave_bad;
      __syncthreads();
      if (threadIdx.x == 0) {
        bool any_bad = false;
        for (int i = 0; i < WAVES; ++i) any_bad = any_bad || sm.words()[1 + i];
        if (any_bad) P.fix[atomicAdd(&P.counters[kCntFix], 1)] = (int32_t)w;
      }
      __syncthreads();
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

// Exact mode: queue every work unit for the SAFE pass.
__global__ __launch_bounds__(256) void k_queue_all(const int64_t *totals,
                                                   int32_t items_cap,
                                                   int32_t hkv,
                                                   int32_t *counters,
                                                   int32_t *fix) {
  int64_t n_items = totals[kTotItems];
  if (n_items > items_cap) n_items = items_cap;
  const int64_t n = n_items * hkv;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * 256)
    fix[i] = (int32_t)i;
  if (blockIdx.x == 0 && threadIdx.x == 0) counters[kCntFix] = (int32_t)n;
}

template <int WAVES, int NQB, bool SAFE>
hipError_t launch_variant(const AttnParams &p, hipStream_t s, int max_grid) {
  int dev = 0, n_cu = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
      &per_cu, k_prefix_attn<WAVES, NQB, SAFE>, WAVES * 64, 0);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  // Persistent grid, a multiple of 8 so block b always serves queue b % 8
  // (consecutive blocks are dispatched round-robin over the 8 XCDs).
  unsigned grid = (unsigned)(n_cu * per_cu);
  grid = (grid + 7) / 8 * 8;
  if (max_grid > 0 && grid > (unsigned)max_grid) grid = (unsigned)max_grid;
  hipLaunchKernelGGL((k_prefix_attn<WAVES, NQB, SAFE>), dim3(grid),
                     dim3(WAVES * 64), 0, s, p);
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
  p.kmax = st.d_kmax;
  p.payload = st.d_payload;
  p.pair_order = pl.pair_order;
  p.group_doc = pl.group_doc;
  p.group_ptr = pl.group_ptr;
  p.blk_pair = pl.blk_pair;
  p.prow = pl.prow;
  p.items = pl.items;
  p.totals = plan_totals(pl);
  p.next = plan_next(pl);
  p.counters = pl.counters;
  p.fix = pl.fix;
  p.kown = pl.kown;
  p.rope = pl.rope;
  p.out = static_cast<uint16_t *>(a->out);
  p.lse = a->lse;
  p.items_cap = pl.items_cap;
  p.Hq = a->n_q_heads;
  p.Hkv = st.n_kv_heads;
  p.n_rep = c.n_rep;
  p.layer = c.layer;
  p.n_layers = st.n_layers;
  p.eps = a->rms_eps;
  p.c = a->softmax_scale * 1.4426950408889634f;

  hipError_t e;
  if (a->timing_begin) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->timing_begin), s);
    if (e != hipSuccess) return e;
  }
  const bool exact = a->kernel_variant >= 4;
  p.flag_all = a->kernel_variant == 5;
  switch (a->kernel_variant) {
    case 1:
    case 5: e = launch_variant<4, 2, false>(p, s, 0); break;
    case 2: e = launch_variant<8, 1, false>(p, s, 0); break;
    case 4:
      hipLaunchKernelGGL(k_queue_all, dim3(256), dim3(256), 0, s, p.totals,
                         p.items_cap, p.Hkv, p.counters, p.fix);
      e = hipGetLastError();
      break;
    default: e = launch_variant<4, 1, false>(p, s, 0); break;  // 0, 3
  }
  if (e != hipSuccess) return e;
  // Work units flagged by the fast pass (normally none) are recomputed with
  // the exact running maximum; in exact mode that is every unit.
  e = launch_variant<4, 1, true>(p, s, exact ? 0 : 64);
  if (e != hipSuccess) return e;
  if (a->timing_end) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->timing_end), s);
    if (e != hipSuccess) return e;
  }
  const unsigned zgrid =
      (unsigned)(a->n_pairs < 1024 ? (a->n_pairs > 0 ? a->n_pairs : 1) : 1024);
  hipLaunchKernelGGL(k_zero_invalid, dim3(zgrid), dim3(256), 0, s,
                     pl.counters, pl.invalid, a->cu_seqlens, a->n_q_heads,
                     p.out, a->lse);
  (void)shape;
  return hipGetLastError();
}

}  // namespace dopr

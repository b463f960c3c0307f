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
// one is consumed) and masked per row: same pair and key <= row.  With 8
// waves (two per SIMD) one wave's MFMA work overlaps the other's softmax
// and memory latency; the kernel is written to fit 256 registers per lane.
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
// Softmax without a running maximum.  q^ is scaled by softmax_scale *
// log2(e) before it is rounded to bf16, so the products are logits in log2
// units.  Every key a row can see has a known norm bound (stored prefix
// keys: a per-slice maximum written when the store is filled; own keys and
// queries: an RMS-normed vector has norm <= sqrt(D), times the largest
// gain), so by Cauchy-Schwarz every logit of a work unit lies in [-B, B].
// When B <= 64 the weights are exp2(logit) directly: no term exceeds 2^64
// and the largest is >= 2^-64, so the normaliser is safe with no reference
// at all.  Otherwise a row uses the fixed reference m = min(B, its first
// chunk's max + 80): terms stay <= 2^0 or bounded and the largest is
// >= 2^-80, with no per-chunk max reduction or accumulator rescale.  A work
// unit in which some row still ends with l outside [2^-90, 2^100] (only
// possible for extreme key norms) is queued and recomputed by a second
// launch of the same kernel in SAFE mode, which tracks the running max
// exactly.
#include <cmath>

#include "attn_common.hpp"

namespace dopr {
namespace {

// The passes of one work unit (an item for one kv head) with softmax mode
// SMX fixed, so every loop below is straight-line code over one set of
// accumulators.  Returns whether some row of this wave left the range the
// fast modes guarantee (the unit is then recomputed in SAFE mode).
template <int WAVES, int NQB, int SMX, bool SCORE, int D, int NCHK>
__device__ __forceinline__ bool run_unit(const AttnParams &P,
                                         Smem<D, NCHK> &sm, const Frag<D> &fo,
                                         int g, int row0, int row1, int L,
                                         int Lp, const uint16_t *Kp,
                                         const uint16_t *VTp, float B) {
  constexpr int PASS = WAVES * NQB * 32;
  constexpr int PSEG = Smem<D, NCHK>::PSEG;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lq = lane & 31, hf = lane >> 5;
  const int n_seg = (L + PSEG - 1) / PSEG;
  const bool resident = n_seg <= 1;
  bool wave_bad = false;

  // (batch token, position) of this lane's rows, loaded one pass ahead so
  // a pass starts with one round trip to memory (q rows, rotary factors)
  int2 tj_next[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int r = row0 + (wave * NQB + qb) * 32 + lq;
    tj_next[qb] = P.utok[(r < row1 ? r : row1 - 1) / P.n_rep];
  }
  for (int pass0 = row0; pass0 < row1; pass0 += PASS) {
    const int pass_end = pass0 + PASS < row1 ? pass0 + PASS : row1;
    // Rows of this lane: batch token, position in the pair, q head.
    int tokq[NQB], head[NQB];
    bool valid[NQB];
    bf16x8 qf[NQB][D / 16];
    Acc<D> acc[NQB];
    // a wave whose rows all lie past the item's end (the tail pass of an
    // item) computes nothing; it still stages and meets the barriers
    const bool live = pass0 + wave * NQB * 32 < row1;
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const int r = pass0 + (wave * NQB + qb) * 32 + lq;
      valid[qb] = r < row1;
      const int rc = valid[qb] ? r : row1 - 1;
      const int u = rc / P.n_rep;
      const int2 tj = tj_next[qb];
      tokq[qb] = tj.x;
      head[qb] = g * P.n_rep + (rc - u * P.n_rep);
      if (live) {
        const uint16_t *qrow = P.q + ((int64_t)tokq[qb] * P.Hq + head[qb]) * D;
        const float2 *rrow = P.rope + (int64_t)(L + tj.y) * (D / 2);
        q_fragments_any<D>(qrow, P.qw, rrow, hf, lq, P.n_rep, P.eps, P.c,
                           P.norm != 0, qf[qb]);
      }
      acc[qb].m = SMX == 2 ? -INFINITY : (SMX == 1 ? INFINITY : 0.f);
      acc[qb].l = 0.f;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[qb].o[db][i] = 0.f;
    }

    // next pass's rows
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const int r = pass0 + PASS + (wave * NQB + qb) * 32 + lq;
      tj_next[qb] = P.utok[(r < row1 ? r : row1 - 1) / P.n_rep];
    }
    const int s_hi = find_pair(P, pass_end - 1);
    OwnStep os;
    os.s = find_pair(P, pass0);
    os.c0 = 0;
    {
      const int4 sp = P.spair[os.s];
      os.tok0 = sp.x;
      os.T = sp.y;
      os.srow0 = sp.z;
    }
    OwnRegs orr;

    // Document prefix: every row sees all L slots.
    for (int sg = 0; sg < n_seg; ++sg) {
      const int seg0 = sg * PSEG;
      const int n = L - seg0 < PSEG ? L - seg0 : PSEG;
      if (!resident) {
        __syncthreads();
        stage_prefix<WAVES, D, NCHK>(Kp, VTp, L, seg0, n, sm);
      }
      wait_vmem();
      __syncthreads();
      const int n_full = live ? n >> 5 : 0;
      for (int ck = 0; ck < n_full; ++ck)
        attend<0, NQB, SMX, D>(sm.pk[ck], sm.pv[ck], fo, qf, acc, hf, B,
                               nullptr);
      if (live && (n & 31)) {
        int lim[NQB];
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) lim[qb] = (n & 31) - 1;
        attend<1, NQB, SMX, D>(sm.pk[n_full], sm.pv[n_full], fo, qf, acc,
                               hf, B, lim);
      }
    }

    // Own causal keys, pair by pair, chunk by chunk, double-buffered: the
    // next chunk's raw k/v are loaded while the current one is consumed,
    // then normed/rotated into the other buffer; one barrier per chunk.
    // (The first chunk is loaded only here: its registers are not held
    // through the prefix products.)
    own_load<WAVES, D>(P, os, g, L, orr);
    __syncthreads();  // the previous pass's last own chunk is consumed
    own_stage<WAVES, D, NCHK>(P, orr, sm, 0);
    __syncthreads();
    int buf = 0;
    while (os.s <= s_hi) {
      // next step: next chunk of this pair, else first chunk of the next.
      // Positions are stacked in descending order, so the pass's latest
      // position of this pair is at its first row in the pass.
      const int srow0 = os.srow0;
      const int lo_row = srow0 > pass0 ? srow0 : pass0;
      const int jmax = os.T - 1 - (lo_row - srow0) / P.n_rep;
      OwnStep nx = os;
      if (os.c0 + KC <= jmax) {
        nx.c0 = os.c0 + KC;
      } else {
        nx.s = os.s + 1;
        nx.c0 = 0;
        if (nx.s <= s_hi) {
          const int4 sp = P.spair[nx.s];
          nx.tok0 = sp.x;
          nx.T = sp.y;
          nx.srow0 = sp.z;
        }
      }
      const bool more = nx.s <= s_hi;
      if (more) own_load<WAVES, D>(P, nx, g, L, orr);
      // per row: last visible key of this chunk (same pair, key <= row)
      int lim[NQB];
      bool need = false;
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        const int jr = tokq[qb] - os.tok0;
        lim[qb] = (unsigned)jr < (unsigned)os.T ? jr - os.c0 : -1;
        need = need || (valid[qb] && lim[qb] >= 0);
      }
      if (__any(need))  // wave-uniform: skip chunks no row of the wave sees
        attend<1, NQB, SMX, D>(sm.ok[buf], sm.ov[buf], fo, qf, acc, hf, B,
                               lim);
      if (more) own_stage<WAVES, D, NCHK>(P, orr, sm, buf ^ 1);
      __syncthreads();
      buf ^= 1;
      os = nx;
    }

    // Normalise; write O (bf16) and the natural-log LSE.
    bool bad = false;
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const float lt = acc[qb].l + __shfl_xor(acc[qb].l, 32, 64);
      if (!valid[qb]) continue;
      bad = bad || !(lt >= kLoOk && lt <= kHiOk);
      const float inv = 1.0f / lt;
      // (score mode stacks one token per pair: stacked token u is the
      // sorted pair, whose output row is the pair's index)
      const int64_t orow =
          (int64_t)(SCORE ? P.pair_order[(pass0 + (wave * NQB + qb) * 32 +
                                          lq) / P.n_rep]
                          : tokq[qb]) * P.Hq + head[qb];
      uint16_t *op = P.out + orow * D;
      float ss = 0.f, sy = 0.f, sn = 0.f;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        float o[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) o[i] = acc[qb].o[db][i] * inv;
        const uint4 h0 = as_uint4(to_bf16x8(o)), h1 = as_uint4(to_bf16x8(o + 8));
        if (!SCORE || P.out) {
          uint4 *dst = reinterpret_cast<uint4 *>(op + 32 * db + 16 * hf);
          dst[0] = h0;
          dst[1] = h1;
        }
        if (SCORE) {
          // the head reads the bf16 row, as it would from memory: lane
          // dims 32*db + 16*hf + 0..15 of q head head[qb] (the opaque
          // offset keeps each slice's weight loads in its own iteration)
          const int64_t c0 =
              (int64_t)head[qb] * D + 32 * db + 16 * hf + opaque_zero();
          const int64_t W = (int64_t)P.Hq * D;
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            float hv[8], gv[8], yv[8], nv[8];
            unpack8(half ? h1 : h0, hv);
            unpack8(*reinterpret_cast<const uint4 *>(P.head_norm_w + c0 +
                                                     8 * half), gv);
            unpack8(*reinterpret_cast<const uint4 *>(P.head_w + c0 +
                                                     8 * half), yv);
            unpack8(*reinterpret_cast<const uint4 *>(P.head_w + W + c0 +
                                                     8 * half), nv);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              ss = fmaf(hv[e], hv[e], ss);
              const float gh = gv[e] * hv[e];
              sy = fmaf(gh, yv[e], sy);
              sn = fmaf(gh, nv[e], sn);
            }
          }
        }
      }
      if (SCORE) {
        ss += __shfl_xor(ss, 32, 64);
        sy += __shfl_xor(sy, 32, 64);
        sn += __shfl_xor(sn, 32, 64);
        if (hf == 0) {
          float *pp = P.part + orow * 3;
          pp[0] = ss;
          pp[1] = sy;
          pp[2] = sn;
        }
      }
      if (P.lse && hf == 0)
        P.lse[orow] = (acc[qb].m + __log2f(lt)) * kLn2;
    }
    wave_bad = wave_bad || __any(bad);
  }
  return wave_bad;
}

// Waves per SIMD: a block's waves spread over the CU's 4 SIMDs, and two
// blocks share a CU when the LDS block fits in half of it (160 KB).
constexpr int waves_per_simd(int waves, int d, int nchk) {
  return (waves / 4) * ((nchk + 2) * 2 * KC * d * 2 <= 81920 ? 2 : 1);
}

template <int WAVES, int NQB, bool SAFE, bool SCORE, int D, int NCHK>
__global__ __launch_bounds__(WAVES * 64) __attribute__((amdgpu_waves_per_eu(
    waves_per_simd(WAVES, D, NCHK),
    waves_per_simd(WAVES, D, NCHK)))) void k_prefix_attn(AttnParams P) {
  __shared__ __attribute__((aligned(16))) Smem<D, NCHK> sm;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lq = lane & 31, hf = lane >> 5;
  const int queue = SAFE ? kFixQueue : (blockIdx.x & 7);
  int64_t n_work;
  const int32_t *qo = nullptr;
  if (SAFE) {
    n_work = P.counters[kCntFix];
  } else {
    int64_t n_items = P.totals[kTotItems];
    if (n_items > P.items_cap) n_items = P.items_cap;
    n_work = n_items * P.Hkv;
    if (P.totals[kTotUnits]) qo = P.qorder;
  }
  const Frag<D> fo = frag_offsets<D>(lq, hf);

  for (;;) {
    if (threadIdx.x == 0) sm.words()[0] = atomicAdd(&P.next[queue], 1);
    __syncthreads();
    const int slot = sm.words()[0];
    int64_t w = SAFE ? (int64_t)slot : unit_at(qo, queue, slot, n_work);
    if (w >= n_work) break;
    bool wave_bad = false;
    bool unscored = false;
    if (SAFE) {
      w = P.fix[w];
      unscored = (w & kFixUnscored) != 0;
      w &= ~(int64_t)kFixUnscored;
    }
    const int item = (int)(w / P.Hkv), g = (int)(w % P.Hkv);
    const int4 it = P.items[item];
    const int row0 = it.y, row1 = it.z;
    const int doc = P.group_doc[it.x];
    const int L = P.doc_len[doc], Lp = pad8(L);
    const int64_t blk = P.doc_off[doc];
    const uint16_t *Kp = P.payload + k_offset(blk, L, P.Hkv, P.layer, g, D);
    const uint16_t *VTp =
        P.payload + vt_offset(blk, L, P.Hkv, P.layer, g, D);
    // every logit of this unit lies in [-B, B] (log2 units).  Without
    // QK-norm no bound is known (kown = 0, so B = 0): the unit runs the
    // no-reference mode anyway, and a row whose normaliser leaves the range
    // that mode serves exactly is caught by the check after the pass and
    // recomputed by the exact pass.
    const float kbound = fmaxf(
        P.kown[0], P.kmax[((int64_t)doc * P.n_layers + P.layer) * P.Hkv + g]);
    const float B = P.c * P.kown[1] * kbound * 1.001f;
    const int n_seg = (L + Smem<D, NCHK>::PSEG - 1) / Smem<D, NCHK>::PSEG;
    const bool resident = n_seg <= 1;
    if (!SAFE) {
      if (B <= kNoRefBound) {
        if (resident && L > 0)
          stage_prefix<WAVES, D, NCHK>(Kp, VTp, L, 0, L, sm);
        wave_bad = run_unit<WAVES, NQB, 0, SCORE, D, NCHK>(
                       P, sm, fo, g, row0, row1, L, Lp, Kp, VTp, B) ||
                   P.flag_all;
      }
      __syncthreads();  // every wave is done with this item's LDS
      if (lane == 0) sm.words()[1 + wave] = wave_bad;
      __syncthreads();
      if (threadIdx.x == 0) {
        bool any_bad = false;
        for (int i = 0; i < WAVES; ++i) any_bad = any_bad || sm.words()[1 + i];
        if (B > kNoRefBound)
          P.fix[atomicAdd(&P.counters[kCntFix], 1)] = (int32_t)w | kFixUnscored;
        else if (any_bad)
          P.fix[atomicAdd(&P.counters[kCntFix], 1)] = (int32_t)w;
      }
      __syncthreads();
    } else {
      if (resident && L > 0)
        stage_prefix<WAVES, D, NCHK>(Kp, VTp, L, 0, L, sm);
      // (self-check mode sends every unit to the exact mode)
      bool exact = !unscored || P.flag_all;
      if (!exact) {
        wave_bad = run_unit<WAVES, NQB, 1, SCORE, D, NCHK>(
            P, sm, fo, g, row0, row1, L, Lp, Kp, VTp, B);
        __syncthreads();
        if (lane == 0) sm.words()[1 + wave] = wave_bad;
        __syncthreads();
        for (int i = 0; i < WAVES; ++i) exact = exact || sm.words()[1 + i];
        __syncthreads();
      }
      if (exact)
        run_unit<WAVES, NQB, 2, SCORE, D, NCHK>(P, sm, fo, g, row0, row1, L,
                                                Lp, Kp, VTp, B);
      __syncthreads();  // every wave is done with this item's LDS
    }
  }
}

// ---------------------------------------------------------------------------
// Last-layer scoring with one wave per work unit.  A score work unit holds
// the score-token rows of the pairs of one document for one kv head, a few
// rows (n_rep per pair), so a block-wide unit leaves most of the block idle
// behind barriers while the prefix is staged.  Here every wave takes its own
// unit (items cut at about 32 rows; the planner's 32-row-aligned cut can
// leave an item empty or up to 63 rows long, which the wave then walks as
// 32-row tiles) and streams it with no block barrier, so a CU has eight
// units in flight and their memory waits overlap:
//   - prefix K and V^T fragments are loaded straight from the store into
//     MFMA operand registers (the store keeps V transposed, so both are
//     16-byte runs per lane);
//   - own keys are normed and rotated in registers by the lane that holds
//     the key's fragments, with the arithmetic of own_stage;
//   - own values are transposed through the wave's own 8 KB LDS slice in
//     the chunk-block layout, then read as V^T fragments.
// The chunk sequence and every operand value equal those of the full path,
// so a score row comes out bit-identical to the full path's row.

// x of lane ^ 32, through the lane-swap instruction (no LDS round trip):
// the swap of a value with itself leaves the lower half's values in [0]
// and the upper half's in [1], each in both halves.
__device__ __forceinline__ float xor32(float x, int hf) {
  const auto r = __builtin_amdgcn_permlane32_swap(
      __builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, x), false,
      false);
  return __builtin_bit_cast(float, hf ? r[0] : r[1]);
}

// k^ = RoPE(RMSNorm(k) * w) of key row `krow` in the A-operand layout: lane
// half hf holds the head-dim groups sub = 2 s' + hf (s' < D/32) and their
// rotate-half partners, as kf[s'] and kf[s' + D/32].  The norm's sum of
// squares is formed per group and added in the order of own_stage's lane
// reduction, so the values equal the staged ones bit for bit.  Invalid keys
// give zero rows.  The gains come from the block's LDS copy `kw`; the
// rotary factors are loaded for half of the groups at a time.
template <int D>
__device__ __forceinline__ void k_group(const uint4 &a0, const uint4 &a1,
                                        const uint16_t *kw, const float4 *cs,
                                        float inv, int sub, bool valid,
                                        bf16x8 &lo, bf16x8 &hi) {
  float x[16];
  if (valid) {
    unpack8(a0, x);
    unpack8(a1, x + 8);
    float w0[8], w1[8];
    unpack8(*reinterpret_cast<const uint4 *>(kw + 8 * sub), w0);
    unpack8(*reinterpret_cast<const uint4 *>(kw + D / 2 + 8 * sub), w1);
    const float c[16] = {cs[0].x, cs[0].y, cs[0].z, cs[0].w,
                         cs[1].x, cs[1].y, cs[1].z, cs[1].w,
                         cs[2].x, cs[2].y, cs[2].z, cs[2].w,
                         cs[3].x, cs[3].y, cs[3].z, cs[3].w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float a = x[e] * inv * w0[e], b = x[8 + e] * inv * w1[e];
      const float co = c[2 * e], si = c[2 * e + 1];
      x[e] = fmaf(a, co, -b * si);
      x[8 + e] = fmaf(b, co, a * si);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) x[e] = 0.f;
  }
  lo = to_bf16x8(x);
  hi = to_bf16x8(x + 8);
}

template <int D>
__device__ __forceinline__ void own_k_fragments(const AttnParams &P,
                                                const uint16_t *krow,
                                                const float2 *rope_row,
                                                const uint16_t *kw,
                                                bool valid, int hf,
                                                bf16x8 *kf) {
  constexpr int NG = D / 32;  // groups per lane half
  constexpr int NH = NG / 2;  // groups per rotary-factor batch
  uint4 a0[NG], a1[NG];
  float4 cs[NH][4];
  if (valid) {
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      const int sub = 2 * s + hf;
      a0[s] = *reinterpret_cast<const uint4 *>(krow + 8 * sub);
      a1[s] = *reinterpret_cast<const uint4 *>(krow + D / 2 + 8 * sub);
    }
#pragma unroll
    for (int s = 0; s < NH; ++s)
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2)
        cs[s][e2] =
            reinterpret_cast<const float4 *>(rope_row + 8 * (2 * s + hf))[e2];
  }
  // group sums, then pairs of adjacent groups (this half's group 2s' with
  // the other half's 2s' + 1), then the pair sums in a balanced tree
  float y[NG];
#pragma unroll
  for (int s = 0; s < NG; ++s) {
    const float own = valid ? sumsq8(a1[s], sumsq8(a0[s], 0.f)) : 0.f;
    y[s] = own + xor32(own, hf);
  }
  float ss;
  if constexpr (NG == 4)
    ss = (y[0] + y[1]) + (y[2] + y[3]);
  else
    ss = y[0] + y[1];
  const float inv = P.norm ? rsqrtf(ss * (1.0f / D) + P.eps) : 1.f;
#pragma unroll
  for (int s = 0; s < NH; ++s)
    k_group<D>(a0[s], a1[s], kw, cs[s], inv, 2 * s + hf, valid, kf[s],
               kf[s + NG]);
  // second batch of rotary factors (the first batch's registers are free)
  if (valid) {
    const float2 *rr = rope_row + opaque_zero();
#pragma unroll
    for (int s = 0; s < NH; ++s)
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2)
        cs[s][e2] = reinterpret_cast<const float4 *>(
            rr + 8 * (2 * (s + NH) + hf))[e2];
  }
#pragma unroll
  for (int s = NH; s < NG; ++s)
    k_group<D>(a0[s], a1[s], kw, cs[s - NH], inv, 2 * s + hf, valid, kf[s],
               kf[s + NG]);
}

// v of own keys c0 .. c0 + 31 of a pair, transposed into the wave's V^T
// chunk block: lane i takes keys 4m .. 4m + 3 (m = i % 8) and head dims
// D/8 * (i / 8) .. + D/8 - 1, and writes four keys of one head dim per
// 8-byte store.  Keys past the pair's end are written as zeros.
template <int D>
__device__ __forceinline__ void own_v_transpose(const AttnParams &P,
                                                const uint16_t *v0, int64_t
                                                key_stride, int nvalid,
                                                uint16_t *ov) {
  constexpr int DL = D / 8;  // head dims per lane
  // (lane offsets from an opaque zero: formed per call, not held across
  // the caller's loops)
  const int lane = (threadIdx.x & 63) + opaque_zero();
  const int m = lane & 7, d0 = DL * (lane >> 3);
  uint4 r[4][DL / 8];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int h = 0; h < DL / 8; ++h)
      r[k][h] = 4 * m + k < nvalid
                    ? *reinterpret_cast<const uint4 *>(
                          v0 + (int64_t)(4 * m + k) * key_stride + d0 + 8 * h)
                    : make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int h = 0; h < DL / 8; ++h) {
    const uint32_t w[4][4] = {{r[0][h].x, r[0][h].y, r[0][h].z, r[0][h].w},
                              {r[1][h].x, r[1][h].y, r[1][h].z, r[1][h].w},
                              {r[2][h].x, r[2][h].y, r[2][h].z, r[2][h].w},
                              {r[3][h].x, r[3][h].y, r[3][h].z, r[3][h].w}};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int d = d0 + 8 * h + e;
      uint32_t k4[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        k4[k] = (e & 1) ? w[k][e >> 1] >> 16 : w[k][e >> 1] & 0xffffu;
      const uint2 pk = make_uint2(k4[0] | (k4[1] << 16), k4[2] | (k4[3] << 16));
      *reinterpret_cast<uint2 *>(ov + vc_off(d, m >> 1) + 4 * (m & 1)) = pk;
    }
  }
}

// One 32-key chunk from operand registers, in the order of attend: S^T =
// K Q^T over the k-steps (qk_regs), then the weights and O^T += V^T P^T over
// the V^T fragments (pv_regs).  Two calls, so that a caller can free the K
// fragments before it gathers the V^T ones.
template <int D>
__device__ __forceinline__ void qk_regs(const bf16x8 *kf,
                                        const bf16x8 (*qf)[D / 16],
                                        floatx16 *S) {
#pragma unroll
  for (int i = 0; i < 16; ++i) S[0][i] = 0.f;
#pragma unroll
  for (int s = 0; s < D / 16; ++s)
    S[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[0][s], S[0], 0,
                                                   0, 0);
}

template <int MODE, int D>
__device__ __forceinline__ void pv_regs(floatx16 *S, const bf16x8 *vf,
                                        Acc<D> *acc, int hf,
                                        const int *lim) {
  bf16x8 pb[1][2];
  softmax_part<MODE, 1, 0, D>(S, acc, hf, 0.f, lim, pb);
#pragma unroll
  for (int f = 0; f < D / 16; ++f)
    acc[0].o[f >> 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
        vf[f], pb[0][f & 1], acc[0].o[f >> 1], 0, 0, 0);
}

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(
    2, 2))) void k_score_rows(AttnParams P) {
  __shared__ __attribute__((aligned(16))) uint16_t sov[4][D * KC];
  __shared__ __attribute__((aligned(16))) uint16_t skw[D];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // the k gains, once per block (the block's only barrier)
  if (threadIdx.x < D / 8)
    reinterpret_cast<uint4 *>(skw)[threadIdx.x] =
        reinterpret_cast<const uint4 *>(P.kw)[threadIdx.x];
  __syncthreads();
  const int queue = blockIdx.x & 7;
  const int64_t n_items64 = P.totals[kTotItems];
  const int n_items = n_items64 < P.items_cap ? (int)n_items64 : P.items_cap;
  // (32-bit unit numbers: below 2^31 by argument validation)
  const int n_work = n_items * P.Hkv;
  const int32_t *qo = P.totals[kTotUnits] ? P.qorder : nullptr;
  uint16_t *ov = sov[wave];

  for (;;) {
    int slot = 0;
    if (lane == 0) slot = atomicAdd(&P.next[queue], 1);
    slot = __builtin_amdgcn_readfirstlane(slot);
    const int w = unit_at32(qo, queue, slot, n_work);
    if (w >= n_work) break;
    const int item = w / P.Hkv, g = w % P.Hkv;
    const int4 it = P.items[item];
    const int doc = P.group_doc[it.x];
    const int L = P.doc_len[doc], Lp = pad8(L);
    const int64_t blk = P.doc_off[doc];
    const uint16_t *Kp = P.payload + k_offset(blk, L, P.Hkv, P.layer, g, D);
    const uint16_t *VTp =
        P.payload + vt_offset(blk, L, P.Hkv, P.layer, g, D);
    const float kbound = fmaxf(
        P.kown[0], P.kmax[((int64_t)doc * P.n_layers + P.layer) * P.Hkv + g]);
    const float B = P.c * P.kown[1] * kbound * 1.001f;
    // a unit over the bound is left to the exact pass.  Every lane runs the
    // same path to the end of the unit (no early continue: the unit loop
    // must leave the queue with the whole wave, and the one queue push is
    // made by lane 0 after a wave-wide vote)
    const bool unscored = B > kNoRefBound;
    bool bad = false;
    for (int t0 = it.y; !unscored && t0 < it.z; t0 += 32) {
      const int t1 = t0 + 32 < it.z ? t0 + 32 : it.z;
      // the lane's row, head-dim and fragment offsets, formed per tile from
      // an opaque lane index (held across the kernel they are spilled)
      const int lt_ = lane + opaque_zero();
      const int lq = lt_ & 31, hf = lt_ >> 5, prow = perm32(lq);
      const Frag<D> fo = frag_offsets<D>(lq, hf);
      // this lane's row: stacked token u is the sorted pair
      const int r = t0 + lq;
      const bool valid = r < t1;
      const int rc = valid ? r : t1 - 1;
      const int u = rc / P.n_rep;
      const int head = g * P.n_rep + (rc - u * P.n_rep);
      const int2 tj = P.utok[u];
      bf16x8 qf[1][D / 16];
      {
        const uint16_t *qrow = P.q + ((int64_t)tj.x * P.Hq + head) * D;
        const float2 *rrow = P.rope + (int64_t)(L + tj.y) * (D / 2);
        q_fragments_any<D>(qrow, P.qw, rrow, hf, lq, P.n_rep, P.eps, P.c,
                           P.norm != 0, qf[0]);
      }
      Acc<D> acc[1];
      acc[0].m = 0.f;
      acc[0].l = 0.f;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[0].o[db][i] = 0.f;

      // prefix chunks: K rows past L are clamped (their logits are masked),
      // V^T granules past the stored columns are zero
      // (at D = 128 the V^T fragments are gathered after the QK products,
      // so the K fragments' registers are free again: fewer spills)
      for (int c0 = 0; c0 < L; c0 += KC) {
        floatx16 S[1];
        bf16x8 kf[D / 16], vf[D / 16];
        const int krow = c0 + prow < L ? c0 + prow : L - 1;
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
          kf[s] = *reinterpret_cast<const bf16x8 *>(
              Kp + (int64_t)krow * D + 16 * s + 8 * hf);
        if constexpr (D == 128) qk_regs<D>(kf, qf, S);
        // (the row offsets are formed here, per chunk, from an opaque
        // zero: hoisted out of the loop they would hold four 64-bit
        // addresses across the whole tile)
        const int vrow = prow + opaque_zero();
#pragma unroll
        for (int f = 0; f < D / 16; ++f) {
          const int key = c0 + 16 * hf + 8 * (f & 1);
          vf[f] = key < Lp ? *reinterpret_cast<const bf16x8 *>(
                                 VTp + (int64_t)(32 * (f >> 1) + vrow) * Lp +
                                 key)
                           : bf16x8{};
        }
        if constexpr (D != 128) qk_regs<D>(kf, qf, S);
        if (c0 + KC <= L) {
          pv_regs<0, D>(S, vf, acc, hf, nullptr);
        } else {
          const int lim[1] = {L - c0 - 1};
          pv_regs<1, D>(S, vf, acc, hf, lim);
        }
      }

      // own keys, pair by pair: a score row sees every own key of its pair
      const int s_lo = t0 / P.n_rep, s_hi = (t1 - 1) / P.n_rep;
      for (int s = s_lo; s <= s_hi; ++s) {
        const int4 sp = P.spair[s];
        const int tok0 = sp.x, T = sp.y;
        for (int c0 = 0; c0 < T; c0 += KC) {
          const int lim[1] = {valid && u == s ? T - 1 - c0 : -1};
          const int jk = c0 + prow;
          floatx16 S[1];
          {
            bf16x8 kf[D / 16];
            own_k_fragments<D>(
                P,
                P.k + ((int64_t)(tok0 + (jk < T ? jk : T - 1)) * P.Hkv + g) * D,
                P.rope + (int64_t)(L + jk) * (D / 2), skw, jk < T, hf, kf);
            qk_regs<D>(kf, qf, S);
          }
          own_v_transpose<D>(P, P.v + ((int64_t)(tok0 + c0) * P.Hkv + g) * D,
                             (int64_t)P.Hkv * D, T - c0, ov);
          // the slice's stores land before the fragment reads (one wave)
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          bf16x8 vf[D / 16];
#pragma unroll
          for (int f = 0; f < D / 16; ++f)
            vf[f] = *reinterpret_cast<const bf16x8 *>(
                ov + (f >> 1) * (32 * KC) + fo.v[f & 1]);
          pv_regs<1, D>(S, vf, acc, hf, lim);
          // every fragment read has returned before the next transpose
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
      }

      // Normalise; O (bf16) if requested, the head's partial sums, LSE.
      const float lt = acc[0].l + xor32(acc[0].l, hf);
      if (valid) {
        bad = bad || !(lt >= kLoOk && lt <= kHiOk);
        const float inv = 1.0f / lt;
        const int64_t orow = (int64_t)P.pair_order[u] * P.Hq + head;
        uint16_t *op = P.out ? P.out + orow * D : nullptr;
        float ss = 0.f, sy = 0.f, sn = 0.f;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          float o[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) o[i] = acc[0].o[db][i] * inv;
          const uint4 h0 = as_uint4(to_bf16x8(o)),
                      h1 = as_uint4(to_bf16x8(o + 8));
          if (op) {
            uint4 *dst = reinterpret_cast<uint4 *>(op + 32 * db + 16 * hf);
            dst[0] = h0;
            dst[1] = h1;
          }
          // (the opaque offset keeps each slice's weight loads in its own
          // iteration instead of all of them in flight at once)
          const int64_t c0 =
              (int64_t)head * D + 32 * db + 16 * hf + opaque_zero();
          const int64_t W = (int64_t)P.Hq * D;
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            float hv[8], gv[8], yv[8], nv[8];
            unpack8(half ? h1 : h0, hv);
            unpack8(*reinterpret_cast<const uint4 *>(P.head_norm_w + c0 +
                                                     8 * half), gv);
            unpack8(*reinterpret_cast<const uint4 *>(P.head_w + c0 +
                                                     8 * half), yv);
            unpack8(*reinterpret_cast<const uint4 *>(P.head_w + W + c0 +
                                                     8 * half), nv);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              ss = fmaf(hv[e], hv[e], ss);
              const float gh = gv[e] * hv[e];
              sy = fmaf(gh, yv[e], sy);
              sn = fmaf(gh, nv[e], sn);
            }
          }
        }
        ss += xor32(ss, hf);
        sy += xor32(sy, hf);
        sn += xor32(sn, hf);
        if (hf == 0) {
          float *pp = P.part + orow * 3;
          pp[0] = ss;
          pp[1] = sy;
          pp[2] = sn;
          if (P.lse) P.lse[orow] = (acc[0].m + __log2f(lt)) * kLn2;
        }
      }
    }
    const bool push = unscored || P.flag_all || __any(bad);
    if (push && lane == 0)
      P.fix[atomicAdd(&P.counters[kCntFix], 1)] =
          (int32_t)w | (unscored ? kFixUnscored : 0);
  }
}

// Pairs whose document is out of range or not resident: zero outputs and
// -inf LSE (their token range was validated by the scheduler).  With no
// token ranges (score mode) pair p owns row p; out may then be NULL.
__global__ __launch_bounds__(256) void k_zero_invalid(
    const int32_t *counters, const int32_t *invalid, const int32_t *cu,
    int32_t Hq, int32_t D, uint16_t *out, float *lse) {
  const int32_t n_inv = counters[kCntInvalid];
  for (int32_t idx = blockIdx.x; idx < n_inv; idx += gridDim.x) {
    const int32_t p = invalid[idx];
    const int64_t t0 = cu ? cu[p] : p, t1 = cu ? cu[p + 1] : p + 1;
    const int64_t n16 = (t1 - t0) * Hq * D / 8;
    uint4 *o = reinterpret_cast<uint4 *>(out + t0 * Hq * D);
    if (out)
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

template <int WAVES, int NQB, bool SAFE, bool SCORE, int D,
          int NCHK = big_chunks(D)>
hipError_t launch_variant(const AttnParams &p, hipStream_t s, int max_grid) {
  int dev = 0, n_cu = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
      &per_cu, k_prefix_attn<WAVES, NQB, SAFE, SCORE, D, NCHK>, WAVES * 64,
      0);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  // Persistent grid, a multiple of 8 so block b always serves queue b % 8
  // (consecutive blocks are dispatched round-robin over the 8 XCDs).
  unsigned grid = (unsigned)(n_cu * per_cu);
  grid = (grid + 7) / 8 * 8;
  if (max_grid > 0 && grid > (unsigned)max_grid) grid = (unsigned)max_grid;
  hipLaunchKernelGGL((k_prefix_attn<WAVES, NQB, SAFE, SCORE, D, NCHK>),
                     dim3(grid), dim3(WAVES * 64), 0, s, p);
  return hipGetLastError();
}

// One-wave-per-unit score kernel: a persistent grid of 4-wave blocks, as
// many as fit (two per CU), a multiple of 8 so block b serves queue b % 8.
template <int D>
hipError_t launch_score_rows(const AttnParams &p, hipStream_t s) {
  int dev = 0, n_cu = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_score_rows<D>,
                                                   256, 0);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  const unsigned grid = (unsigned)((n_cu * per_cu + 7) / 8 * 8);
  hipLaunchKernelGGL(k_score_rows<D>, dim3(grid), dim3(256), 0, s, p);
  return hipGetLastError();
}

// The fast pass in tile shape shape_v (1, 2, 3, 6; 7 the one-wave-per-unit
// score kernel; 4 queues every unit for the exact pass instead), then the
// exact pass over the queued units.
template <int D>
hipError_t launch_passes(const AttnParams &p, const KhatParams &kp,
                         int32_t n_pairs, int shape_v, bool score,
                         hipStream_t s) {
  hipError_t e;
  switch (shape_v) {
    case 8: e = launch_stream(D, p, kp, n_pairs, s); break;
    case 7: e = launch_score_rows<D>(p, s); break;
    case 1: e = launch_variant<4, 2, false, false, D>(p, s, 0); break;
    case 3: e = launch_variant<4, 1, false, false, D>(p, s, 0); break;
    case 6:
      e = score ? launch_variant<4, 1, false, true, D, small_chunks(D)>(p, s, 0)
                : launch_variant<4, 1, false, false, D, small_chunks(D)>(p, s,
                                                                         0);
      break;
    case 4:
      hipLaunchKernelGGL(k_queue_all, dim3(256), dim3(256), 0, s, p.totals,
                         p.items_cap, p.Hkv, p.counters, p.fix);
      e = hipGetLastError();
      break;
    default:  // 2
      e = score ? launch_variant<8, 1, false, true, D>(p, s, 0)
                : launch_variant<8, 1, false, false, D>(p, s, 0);
      break;
  }
  if (e != hipSuccess) return e;
  // Work units the fast pass flagged or left unscored (normally none) are
  // computed here; in exact mode that is every unit.
  return score ? launch_variant<4, 1, true, true, D>(p, s, 0)
               : launch_variant<4, 1, true, false, D>(p, s, 0);
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
  p.norm = a->q_norm_w != nullptr;
  p.qw = p.norm ? static_cast<const uint16_t *>(a->q_norm_w) : pl.unit_w;
  p.kw = p.norm ? static_cast<const uint16_t *>(a->k_norm_w) : pl.unit_w;
  p.doc_len = st.d_len;
  p.doc_off = st.d_off;
  p.kmax = st.d_kmax;
  p.payload = st.d_payload;
  p.group_doc = pl.group_doc;
  p.blk_pair = pl.blk_pair;
  p.items = pl.items;
  p.spair = pl.spair;
  p.utok = pl.utok;
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
  p.kh = pl.kh;
  p.zero = pl.zero;
  p.units = pl.units;
  p.qorder = pl.qorder;
  p.ntok = a->total_tokens;
  KhatParams kp{};
  kp.k = p.k;
  kp.kw = p.kw;
  kp.doc_ids = a->doc_ids;
  kp.pair_order = pl.pair_order;
  kp.doc_len = st.d_len;
  kp.spair = pl.spair;
  kp.totals = p.totals;
  kp.rope = pl.rope;
  kp.kh = pl.kh;
  kp.ntok = a->total_tokens;
  kp.Hkv = st.n_kv_heads;
  kp.eps = a->rms_eps;
  kp.norm = p.norm;

  hipError_t e;
  if (a->timing_begin) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->timing_begin), s);
    if (e != hipSuccess) return e;
  }
  p.flag_all = a->kernel_variant == 5;
  const bool score = c.head != nullptr;
  if (score) {
    p.pair_order = pl.pair_order;
    p.part = pl.part;
    p.head_norm_w = static_cast<const uint16_t *>(c.head->norm_w);
    p.head_w = static_cast<const uint16_t *>(c.head->w_head);
  }
  // Tile shape.  Automatic: for score rows, one wave per work unit (shape
  // 7) unless some prefix is longer than kScoreRowsMaxLen (each 32-row unit
  // streams its whole prefix, so long prefixes shared by many pairs are
  // cheaper staged once per item by shape 6).  For full rows the pass kernel
  // (shape 8) when the plan holds k^ of every token; without that buffer two
  // 4-wave blocks per CU (half the LDS each: 96 prefix slots resident at
  // D = 128, 256 at D = 64) when every prefix fits, else one 8-wave block per
  // CU with 256 (512) slots resident.  Variants 2 and 6 keep the block-wide
  // kernels for score rows (1, 3 and 8 map to 6).
  const int D = st.head_dim;
  int shape_v = a->kernel_variant;
  if (shape_v == 0 || shape_v == 5)
    shape_v = score ? (st.max_len <= kScoreRowsMaxLen ? 7 : 6)
              : pl.kh ? 8
              : st.max_len <= small_chunks(D) * KC ? 6
                                                   : 2;
  static_assert(small_chunks(128) * KC == kShortPrefix128,
                "short prefixes are those two blocks per CU keep resident");
  if (score && (shape_v == 1 || shape_v == 3 || shape_v >= 8)) shape_v = 6;
  if (shape_v >= 8 && !pl.kh) return hipErrorInvalidValue;
  e = D == 128 ? launch_passes<128>(p, kp, a->n_pairs, shape_v, score, s)
               : launch_passes<64>(p, kp, a->n_pairs, shape_v, score, s);
  if (e != hipSuccess) return e;
  if (a->timing_end) {
    e = hipEventRecord(static_cast<hipEvent_t>(a->timing_end), s);
    if (e != hipSuccess) return e;
  }
  const unsigned zgrid =
      (unsigned)(a->n_pairs < 1024 ? (a->n_pairs > 0 ? a->n_pairs : 1) : 1024);
  hipLaunchKernelGGL(k_zero_invalid, dim3(zgrid), dim3(256), 0, s,
                     pl.counters, pl.invalid, score ? nullptr : a->cu_seqlens,
                     a->n_q_heads, D, p.out, a->lse);
  if (score) {
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_score_reduce(pl, a->n_pairs, a->n_q_heads,
                               a->n_q_heads * D, c.head, s);
  }
  (void)shape;
  return hipGetLastError();
}

}  // namespace dopr


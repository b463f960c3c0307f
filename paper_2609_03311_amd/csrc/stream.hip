// stream.hip -- the pass kernel of the full online layer (the automatic
// choice unless every prefix is at most 96 slots at head size 128) and the
// k^ precompute it reads.  Built as its own
// translation unit with the compiler's common-code sinking off: that
// transformation would merge stores of different unit fields into one
// through a pointer and move wave-uniform state to scratch memory.
#include "attn_common.hpp"

namespace dopr {
namespace {

// ---------------------------------------------------------------------------
// k^ precompute.  One block per sorted pair: RMSNorm, gain and rotation of
// every online key of the pair at positions L + j, for every kv head, with
// the arithmetic of the block kernels' own-key staging (own_stage), rounded
// to bf16 and written as k^ [Hkv][Ntok][D].  The pass kernel then copies
// own keys like prefix keys, and a pair's keys are normed once per batch
// instead of once per pass that reads them.
constexpr int kKhatRowsPerStep = 2;

template <int D>
__global__ __launch_bounds__(256) void k_own_khat(KhatParams P) {
  constexpr int NSUB = D / 16, ROWS = 256 / NSUB;
  const int s = blockIdx.x;
  const int n_valid = (int)(P.totals[kTotDocs] & 0xffffffff);
  if (s >= n_valid) return;
  const int4 sp = P.spair[s];
  const int tok0 = sp.x, T = sp.y;
  const int L = P.doc_len[P.doc_ids[P.pair_order[s]]];
  const int t = threadIdx.x;
  const int sub = t % NSUB;
  const uint4 g0 = *reinterpret_cast<const uint4 *>(P.kw + 8 * sub);
  const uint4 g1 = *reinterpret_cast<const uint4 *>(P.kw + D / 2 + 8 * sub);
  const int64_t n_rows = (int64_t)T * P.Hkv;
  // KB rows per thread and step, every row's loads issued before the first
  // is used (the stores of one step cannot be moved above the next step's
  // loads by the compiler, so one row per step leaves one load in flight)
  constexpr int KB = kKhatRowsPerStep;
  for (int64_t r0 = t / NSUB; r0 < n_rows; r0 += KB * ROWS) {
    uint4 a0[KB], a1[KB];
    const float4 *cq[KB];
    int j[KB], g[KB];
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int64_t rr = r0 + k * ROWS < n_rows ? r0 + k * ROWS : r0;
      j[k] = (int)(rr / P.Hkv);
      g[k] = (int)(rr % P.Hkv);
      const uint16_t *kr = P.k + ((int64_t)(tok0 + j[k]) * P.Hkv + g[k]) * D;
      a0[k] = *reinterpret_cast<const uint4 *>(kr + 8 * sub);
      a1[k] = *reinterpret_cast<const uint4 *>(kr + D / 2 + 8 * sub);
      cq[k] = reinterpret_cast<const float4 *>(
          P.rope + (int64_t)(L + j[k]) * (D / 2) + 8 * sub);
    }
    float4 c[KB][4];
#pragma unroll
    for (int k = 0; k < KB; ++k)
#pragma unroll
      for (int i = 0; i < 4; ++i) c[k][i] = cq[k][i];
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      if (k > 0 && r0 + k * ROWS >= n_rows) break;
      float x[16];
      khat_part<D>(a0[k], a1[k], g0, g1, c[k][0], c[k][1], c[k][2], c[k][3],
                   true, P.eps, P.norm != 0, x);
      uint16_t *o = P.kh + ((int64_t)g[k] * P.ntok + tok0 + j[k]) * D;
      *reinterpret_cast<uint4 *>(o + 8 * sub) = as_uint4(to_bf16x8(x));
      *reinterpret_cast<uint4 *>(o + D / 2 + 8 * sub) =
          as_uint4(to_bf16x8(x + 8));
    }
  }
}

__device__ __forceinline__ int rfl(int x) {
  return __builtin_amdgcn_readfirstlane(x);
}

// Loads of read-only plan and store metadata at wave-uniform indices, made
// through the constant address space so they become scalar loads.
template <class T>
__device__ __forceinline__ T cld(const T *p, int64_t i) {
  return ((const __attribute__((address_space(4))) T *)p)[i];
}

// Own-V rows: 16-byte granule swizzle that puts the four keys one
// transposing read takes per lane group on four different 64-byte bank
// ranges (a row is 256 B at D = 128, 128 B at D = 64).
template <int D>
__device__ __forceinline__ int swvo(int r) {
  if constexpr (D == 128)
    return (r & 3) << 2;
  else
    return ((r >> 1) & 1) << 2;
}

// A lane-derived index formed again where it is used, at head size 64, where
// the pass kernel runs in 128 registers: per-lane pointers the compiler would
// otherwise hoist to the kernel's start (and spill) are rebuilt per use.  At
// 128 the plain index keeps the schedule it has.
template <int D>
__device__ __forceinline__ int lane_here(int x) {
  if constexpr (D == 64)
    return x + opaque_zero();
  else
    return x;
}


// Per-phase cycle counters of the pass kernel, compiled in only for the
// measurement library (-DDOPR_PASS_TIMERS): each wave adds the s_memtime
// cycles between consecutive marks to the total of the phase the mark
// closes, and adds its totals to a device array when it exits.  In the
// product library the marks are empty.
enum PassPhase {
  kPtUnit,        // unit hand-over (the claimed unit read from LDS)
  kPtStage,       // the resident prefix's loads issued
  kPtSearch,      // the pass's pair records found
  kPtOwnIssue,    // the first two own chunks' loads issued
  kPtQ,           // q rows loaded and q^ formed
  kPtWaitLoads,   // waiting for the pass's loads
  kPtBarrierPre,  // the barrier before the products
  kPtPrefix,      // prefix chunks
  kPtOwnCompute,  // own chunks: products
  kPtOwnBarrier,  // own chunks: the two barriers per chunk
  kPtOwnLoads,    // own chunks: next chunk's loads issued and waited for
  kPtEpilogue,    // normalise and store O and the LSE
  kPtPassEnd,     // the barrier at the end of a pass
  kPtUnitEnd,     // the next unit's claim and the hand-over
  kPtUnits,       // count: units
  kPtPasses,      // count: passes
  kPtTailCycles,  // cycles of passes with at most 32 rows
  kPtTails,       // count: such passes
  kPtSlots
};
#ifdef DOPR_PASS_TIMERS
__device__ unsigned long long g_pass_phase[8][kPtSlots];
#define PT_NOW() ((int64_t)__builtin_amdgcn_s_memtime())
#define PT_DECL()                    \
  int64_t pt_acc[kPtSlots] = {};     \
  int64_t pt_last = PT_NOW(), pt_pass = pt_last
#define PT_MARK(k)                   \
  do {                               \
    const int64_t pt_t = PT_NOW();   \
    pt_acc[k] += pt_t - pt_last;     \
    pt_last = pt_t;                  \
  } while (0)
#define PT_COUNT(k) (pt_acc[k] += 1)
#define PT_PASS_START() (pt_pass = PT_NOW())
#define PT_PASS_END(rows)                   \
  do {                                      \
    if ((rows) <= 32) {                     \
      pt_acc[kPtTailCycles] += pt_last - pt_pass; \
      pt_acc[kPtTails] += 1;                \
    }                                       \
  } while (0)
#define PT_FLUSH(wave, lane)                                          \
  do {                                                                \
    if ((lane) == 0)                                                  \
      for (int pt_i = 0; pt_i < kPtSlots; ++pt_i)                     \
        atomicAdd(&g_pass_phase[wave][pt_i],                          \
                  (unsigned long long)pt_acc[pt_i]);                  \
  } while (0)
#else
#define PT_DECL() ((void)0)
#define PT_MARK(k) ((void)0)
#define PT_COUNT(k) ((void)0)
#define PT_PASS_START() ((void)0)
#define PT_PASS_END(rows) ((void)0)
#define PT_FLUSH(wave, lane) ((void)0)
#endif

template <int N>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Block barrier for LDS traffic only: outstanding global loads and stores
// keep flowing through it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// V^T fragments of an own chunk from v rows [32][D] in LDS, by gfx950's
// transposing LDS read (4 keys of one head dim per lane and read, two
// reads per fragment).  Issued through inline assembly: the compiler
// would otherwise wait for every outstanding direct-to-LDS load in
// flight before each of these reads.  The results are not ready until
// lgkm_ready() has run on them.  vaddr is this lane's LDS byte address
// (row 16*hf + e, column perm32(16*(lq/16) + 4q) of the lane's (e, q) role
// in its 16-lane group); ex selects the row swizzle.
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

template <int D, int OFF>
__device__ __forceinline__ u32x2 ds_tr(uint32_t vaddr) {
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
               : "=v"(r)
               : "v"(vaddr), "n"(OFF));
  return r;
}

template <int D>
__device__ __forceinline__ void own_v_frags(uint32_t vaddr, int ex, int f0,
                                            u32x4 *vf) {
  // fragment f = (db = f / 2, t = f % 2): keys 8t .. 8t + 7 of this lane's
  // half, head dims 32 db + perm32(lq)
#pragma unroll
  for (int f = 0; f < RA; ++f) {
    const int ff = f0 + f, db = ff >> 1, t = ff & 1;
    const uint32_t a = vaddr + 2 * 32 * (db ^ ex);
    u32x2 lo, hi;
    if (t == 0) {
      lo = ds_tr<D, 0>(a);
      hi = ds_tr<D, 2 * 4 * D>(a);
    } else {
      lo = ds_tr<D, 2 * 8 * D>(a);
      hi = ds_tr<D, 2 * 12 * D>(a);
    }
    vf[f] = u32x4{lo.x, lo.y, hi.x, hi.y};
  }
}

// Wait for this wave's LDS reads; the fragments are tied to the wait so
// no use of them moves above it.
__device__ __forceinline__ void lgkm_ready(u32x4 *vf) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(vf[0]), "+v"(vf[1]), "+v"(vf[2]), "+v"(vf[3])
               :
               : "memory");
}

// One own-key chunk: S^T = K Q^T from the K rows, weights with per-row key
// limits, O^T += V^T P^T with V^T from the transposing reads.
template <int D>
__device__ __forceinline__ void attend_own(const uint16_t *kblk,
                                           uint32_t vaddr, int ex,
                                           const Frag<D> &fo,
                                           const bf16x8 (*qf)[D / 16],
                                           Acc<D> *acc, int hf,
                                           const int *lim) {
  floatx16 S[1];
  qk_part<1, D>(kblk, fo, qf, S);
  u32x4 vf[RA];
  own_v_frags<D>(vaddr, ex, 0, vf);
  bf16x8 pb[1][2];
  softmax_part<1, 1, 0, D>(S, acc, hf, 0.f, lim, pb);
  lgkm_ready(vf);
#pragma unroll
  for (int f0 = 0; f0 < D / 16; f0 += RA) {
    if (f0 > 0) {
      own_v_frags<D>(vaddr, ex, f0, vf);
      lgkm_ready(vf);
    }
#pragma unroll
    for (int f = f0; f < f0 + RA; ++f)
      acc[0].o[f >> 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          __builtin_bit_cast(bf16x8, vf[f - f0]), pb[0][f & 1],
          acc[0].o[f >> 1], 0, 0, 0);
  }
}

// ---------------------------------------------------------------------------
// Pass kernel (full layer).  A work unit is one item of one document's
// stacked rows (up to rows_per_item, 2048 by default) for one kv head,
// walked in passes of 256 rows, one 32-row tile per wave of the 8-wave
// block.  The document's prefix (up to 256 slots) is staged in LDS once
// per unit and read by every pass with no barrier, as
// in the block kernels; what differs is everything around it:
//   - own keys come precomputed (k_own_khat), so an own chunk is a plain
//     copy: K rows and raw v rows go straight to LDS with direct loads into
//     two slots, and the PV product reads v with gfx950's transposing LDS
//     read; a pass's first two own chunks are issued before its prefix
//     products, later ones while the chunk before them is consumed;
//   - the pass's q rows load while the prefix and first own chunks are in
//     flight, so one memory latency covers all of them;
//   - wave 0 claims the next unit while the current one is in progress and
//     hands it to the other waves through a small LDS table.
// Per row the chunk order and operand values are those of the block
// kernels, so the outputs are bit-identical to theirs.  Only the
// reference-free softmax (mode 0) runs here: units over the logit bound
// and units with a normaliser out of range go to the exact pass.
//
// Loop exits are wave- or block-uniform: the unit loop ends on the unit
// wave 0 published in LDS (read after a barrier), the pass loop on
// wave-uniform unit fields, the pair search on a ballot, and the own-chunk
// loop on positions taken from the pair records with readlane.

// A work unit as wave 0 found it (every field wave-uniform).
struct PUnit {
  int w, g, row0, row1, s_lo, L;
  int64_t koff, vtoff;
};

// Words of the unit hand-over at the start of own slot 0 (free at unit
// boundaries): [0] = 1 when the last unit needs the exact pass, [1..8] the
// waves' flags, [16..] the next unit.
constexpr int kWordUnit = 16;

// Work unit w from the plan's unit table, read by wave 0 with one vector
// load (lane i holds word i of the unit's two records).
__device__ __forceinline__ int unit_words(const AttnParams &P, int w,
                                          int lane) {
  return lane < 8 ? reinterpret_cast<const int *>(P.units)[8 * (int64_t)w +
                                                           lane]
                  : 0;
}

__device__ __forceinline__ PUnit unit_from_words(int w, int x) {
  PUnit u;
  u.w = w;
  u.g = 0;
  u.row0 = __builtin_amdgcn_readlane(x, 0);
  u.row1 = __builtin_amdgcn_readlane(x, 1);
  u.s_lo = __builtin_amdgcn_readlane(x, 2);
  u.L = __builtin_amdgcn_readlane(x, 3);
  u.koff = (int64_t)(uint32_t)__builtin_amdgcn_readlane(x, 4) |
           ((int64_t)__builtin_amdgcn_readlane(x, 5) << 32);
  u.vtoff = (int64_t)(uint32_t)__builtin_amdgcn_readlane(x, 6) |
            ((int64_t)__builtin_amdgcn_readlane(x, 7) << 32);
  return u;
}

// Wave 0 (uniform): finish a claim -- the queue slot `slot` (already
// taken) and the unit's table words x.  Units over the logit bound are
// handed to the exact pass unscored and replaced by further claims (rare:
// those waits are not hidden).  w = -1 past the end of the queue.
__device__ PUnit pass_claim_finish(const AttnParams &P, const int32_t *qo,
                                   int queue, int64_t n_work, int lane,
                                   int slot, int x) {
  for (;;) {
    const int64_t w = unit_at(qo, queue, slot, n_work);
    if (w >= n_work) {
      PUnit u{};
      u.w = -1;
      return u;
    }
    PUnit u = unit_from_words((int)w, x);
    if (u.L >= 0) {
      u.g = (int)(w % P.Hkv);
      return u;
    }
    int s2 = 0;
    if (lane == 0) {
      P.fix[atomicAdd(&P.counters[kCntFix], 1)] = (int32_t)w | kFixUnscored;
      s2 = atomicAdd(&P.next[queue], 1);
    }
    slot = rfl(s2);
    const int64_t w2 = unit_at(qo, queue, slot, n_work);
    x = w2 < n_work ? unit_words(P, (int)w2, lane) : 0;
  }
}

// The hand-over words are written and read with LDS instructions the
// compiler does not see: as plain LDS accesses to memory that direct loads
// also target, each would first wait for every outstanding vector memory
// operation of the wave, the output stores included.  The slot holding
// them has no direct load in flight whenever they are accessed.
__device__ __forceinline__ void lds_put(uint32_t addr, int v) {
  asm volatile("ds_write_b32 %0, %1" ::"v"(addr), "v"(v) : "memory");
}
__device__ __forceinline__ int lds_get(uint32_t addr) {
  int v;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)"
               : "=v"(v)
               : "v"(addr)
               : "memory");
  return v;
}

__device__ __forceinline__ void unit_put(uint32_t wd, const PUnit &u) {
  lds_put(wd + 0, u.w);
  lds_put(wd + 4, u.g);
  lds_put(wd + 8, u.row0);
  lds_put(wd + 12, u.row1);
  lds_put(wd + 16, u.s_lo);
  lds_put(wd + 20, u.L);
  lds_put(wd + 24, (int)(uint32_t)u.koff);
  lds_put(wd + 28, (int)(u.koff >> 32));
  lds_put(wd + 32, (int)(uint32_t)u.vtoff);
  lds_put(wd + 36, (int)(u.vtoff >> 32));
}

__device__ __forceinline__ PUnit unit_get(uint32_t wd) {
  PUnit u;
  u.w = rfl(lds_get(wd + 0));
  u.g = rfl(lds_get(wd + 4));
  u.row0 = rfl(lds_get(wd + 8));
  u.row1 = rfl(lds_get(wd + 12));
  u.s_lo = rfl(lds_get(wd + 16));
  u.L = rfl(lds_get(wd + 20));
  u.koff = (int64_t)(uint32_t)rfl(lds_get(wd + 24)) |
           ((int64_t)rfl(lds_get(wd + 28)) << 32);
  u.vtoff = (int64_t)(uint32_t)rfl(lds_get(wd + 32)) |
            ((int64_t)rfl(lds_get(wd + 36)) << 32);
  return u;
}

// Own-chunk position: pair pi of the unit (its record in lane pi of the
// wave's pair-record registers), keys k0 .. k0 + 31.
struct OwnPos {
  int pi, k0, tok0, T, jmax;
};

__device__ __forceinline__ void own_at(OwnPos &o, int pi, int rtok,
                                       int rT, int rj) {
  o.pi = pi;
  o.k0 = 0;
  o.tok0 = __builtin_amdgcn_readlane(rtok, pi);
  o.T = __builtin_amdgcn_readlane(rT, pi);
  o.jmax = __builtin_amdgcn_readlane(rj, pi);
}

// Next own chunk of the unit; false past the last one.
__device__ __forceinline__ bool own_next(OwnPos &o, int np, int rtok, int rT,
                                         int rj) {
  o.k0 = rfl(o.k0 + KC);
  if (o.k0 <= o.jmax) return true;
  if (o.pi + 1 >= np) return false;
  own_at(o, o.pi + 1, rtok, rT, rj);
  return true;
}

// This wave's share of the direct loads of one own chunk: K rows (k^,
// swizzled as prefix K) into kslot, raw v rows into vslot.
template <int D>
__device__ __forceinline__ void own_dma(const AttnParams &P, int g,
                                        const OwnPos &o, uint16_t *kslot,
                                        uint16_t *vslot, int wave, int lane) {
  constexpr int G = D / 8, RPB = 64 / G;
  constexpr int HALF = KC * D * 2 / 1024;  // 1 KB blocks of K (and of V)
  constexpr int PER = 2 * HALF / 8;         // per wave
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int b = wave * PER + i;
    const bool isv = b >= HALF;
    const int kb = isv ? b - HALF : b;
    const int r = RPB * kb + lane / G, p = lane % G;
    const int j = o.k0 + r;
    const uint16_t *src;
    uint16_t *dst;
    if (!isv) {
      const int gr = p ^ swz<D>(r);
      src = j < o.T ? P.kh + ((int64_t)g * P.ntok + o.tok0 + j) * D + 8 * gr
                    : P.zero;
      dst = kslot + kb * 512;
    } else {
      const int gr = p ^ swvo<D>(r);
      src = j < o.T ? P.v + ((int64_t)(o.tok0 + j) * P.Hkv + g) * D + 8 * gr
                    : P.zero;
      dst = vslot + kb * 512;
    }
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void *)src,
        (__attribute__((address_space(3))) void *)dst, 16, 0, 0);
  }
}

// At head size 64 a 256-slot prefix and the own slots take 80 KB, so two
// blocks share a CU (four waves per SIMD within 128 registers): the two
// blocks' passes are in independent phases, and each hides the other's
// waits.  At 128 the 256-slot prefix fills the LDS: one block per CU.
template <int D>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(
    D == 64 ? 4 : 2, D == 64 ? 4 : 2))) void k_pass_attn(AttnParams P) {
  constexpr int NCHK = D == 64 ? small_chunks(D) : big_chunks(D);
  using SM = Smem<D, NCHK>;
  constexpr int PSEG = SM::PSEG;
  constexpr int OWN_DMA = 2 * (KC * D * 2 / 1024) / 8;  // per wave, chunk
  __shared__ __attribute__((aligned(16))) SM sm;
  // (the wave index is uniform by construction; saying so keeps every
  // branch on it scalar and every value derived from it in scalar
  // registers)
  const int lane = threadIdx.x & 63, wave = rfl(threadIdx.x >> 6);
  const int lq = lane & 31, hf = lane >> 5;
  const int queue = blockIdx.x & 7;
  int64_t n_items = P.totals[kTotItems];
  if (n_items > P.items_cap) n_items = P.items_cap;
  const int64_t n_work = n_items * P.Hkv;
  const int32_t *qo = P.totals[kTotUnits] ? P.qorder : nullptr;
  const int n_valid = (int)(cld(P.totals, kTotDocs) & 0xffffffff);
  // rows per pass: one 32-row tile per wave, and at most 64 pairs (a pair
  // has n_rep rows per token, and one pair record per lane)
  const int PR = P.n_rep >= 4 ? 256 : 64 * P.n_rep;
  const Frag<D> fo = frag_offsets<D>(lq, hf);
  const int e4 = (lane >> 2) & 3, q4 = lane & 3;
  const int ex = D == 128 ? e4 : (e4 >> 1);
  // own-V transposing reads: byte address of this lane's part in slot b
  const uint32_t v_lane_b =
      2u * (uint32_t)((16 * hf + e4) * D +
                      perm32(16 * ((lane >> 4) & 1) + 4 * q4));
  const uint32_t ov0 =
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)
          sm.ov[0];
  const uint32_t ov1 =
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)
          sm.ov[1];
  // hand-over words: LDS byte address of the start of own slot 0
  const uint32_t wd =
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)
          sm.ok[0];

  PT_DECL();
  if (wave == 0) {
    int slot = 0;
    if (lane == 0) slot = atomicAdd(&P.next[queue], 1);
    slot = rfl(slot);
    const int64_t w = unit_at(qo, queue, slot, n_work);
    const int x = w < n_work ? unit_words(P, (int)w, lane) : 0;
    const PUnit u0 = pass_claim_finish(P, qo, queue, n_work, lane, slot, x);
    if (lane == 0) unit_put(wd + 4 * kWordUnit, u0);
  }
  lds_barrier();

  for (;;) {
    const PUnit u = unit_get(wd + 4 * kWordUnit);
    if (u.w < 0) break;
    lds_barrier();  // every wave has the unit before slot 0 is refilled
    PT_MARK(kPtUnit);
    PT_COUNT(kPtUnits);
    // wave 0 claims the next unit: the atomic is issued here, its table
    // words read once the first pass's loads are in, and used at the end
    int next_slot = 0, next_x = 0;
    if (wave == 0 && lane == 0) next_slot = atomicAdd(&P.next[queue], 1);

    const uint16_t *Kp = P.payload + u.koff;
    const uint16_t *VTp = P.payload + u.vtoff;
    const int n_seg = (u.L + PSEG - 1) / PSEG;
    const bool resident = n_seg <= 1;
    // a prefix that fits stays in LDS for every pass of the unit
    if (resident && u.L > 0) stage_prefix<8, D, NCHK>(Kp, VTp, u.L, 0, u.L, sm);
    bool wave_bad = false;
    int s_first = u.s_lo;
    PT_MARK(kPtStage);
    for (int pass0 = u.row0; pass0 < u.row1; pass0 += PR) {
      PT_PASS_START();
      PT_COUNT(kPtPasses);
      const int pass_end = pass0 + PR < u.row1 ? pass0 + PR : u.row1;
      // the pass's first pair: the last pair starting at or before pass0
      const int lane_p = lane_here<D>(lane);
      for (;;) {
        const int si = s_first + lane_p;
        const int z = si < n_valid ? P.spair[si].z : 0x7fffffff;
        const uint64_t le = __ballot(z <= pass0);
        const int k = 63 - __clzll(le);  // highest such lane (lane 0 is)
        s_first = rfl(s_first + k);
        if (k < 63) break;
      }
      // pair records, lane i: the pass's i-th pair (tok0, T, latest
      // position in the pass; positions are stacked latest first)
      const int si = s_first + lane_p;
      int4 rec = make_int4(0, 0, pass_end, 0);
      if (si < n_valid) rec = P.spair[si];
      const bool in = si < n_valid && rec.z < pass_end;
      const int np = __popcll(__ballot(in));
      const int lo_row = rec.z > pass0 ? rec.z : pass0;
      const int rtok = rec.x, rT = rec.y;
      const int rj = rec.y - 1 - (lo_row - rec.z) / P.n_rep;

      PT_MARK(kPtSearch);
      // the pass's first two own chunks
      OwnPos o0, o1, o2;
      own_at(o0, 0, rtok, rT, rj);
      own_dma<D>(P, u.g, o0, sm.ok[0], sm.ov[0], wave, lane_here<D>(lane));
      o1 = o0;
      bool has1 = own_next(o1, np, rtok, rT, rj);
      if (has1)
        own_dma<D>(P, u.g, o1, sm.ok[1], sm.ov[1], wave, lane_here<D>(lane));

      PT_MARK(kPtOwnIssue);
      // this wave's rows and q^
      const int r = pass0 + wave * 32 + lq;
      const bool valid = wave * 32 < PR && r < pass_end;
      const bool live = wave * 32 < PR && pass0 + wave * 32 < pass_end;
      const int rc = valid ? r : pass_end - 1;
      const int ut = rc / P.n_rep;
      const int head = u.g * P.n_rep + (rc - ut * P.n_rep);
      bf16x8 qf[1][D / 16];
      int tokq = 0;
      if (live) {
        const int2 tj = P.utok[ut];
        tokq = tj.x;
        const uint16_t *qrow = P.q + ((int64_t)tokq * P.Hq + head) * D;
        const float2 *rrow = P.rope + (int64_t)(u.L + tj.y) * (D / 2);
        q_fragments_any<D>(qrow, P.qw, rrow, lane_here<D>(hf),
                           lane_here<D>(lane), P.n_rep, P.eps, P.c,
                           P.norm != 0, qf[0]);
      }
      Acc<D> acc[1];
      acc[0].m = 0.f;
      acc[0].l = 0.f;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[0].o[db][i] = 0.f;
      // wave 0: the next unit's table words (its atomic has returned)
      if (wave == 0 && pass0 == u.row0) {
        next_slot = rfl(next_slot);
        const int64_t w = unit_at(qo, queue, next_slot, n_work);
        if (w < n_work) next_x = unit_words(P, (int)w, lane);
      }

      PT_MARK(kPtQ);
      // document prefix: every row sees all L slots
      wait_vmem();
      PT_MARK(kPtWaitLoads);
      lds_barrier();
      PT_MARK(kPtBarrierPre);
      for (int sg = 0; sg < n_seg; ++sg) {
        const int seg0 = sg * PSEG;
        const int n = u.L - seg0 < PSEG ? u.L - seg0 : PSEG;
        if (!resident) {
          __syncthreads();
          stage_prefix<8, D, NCHK>(Kp, VTp, u.L, seg0, n, sm);
          wait_vmem();
          __syncthreads();
        }
        const int n_full = live ? n >> 5 : 0;
        for (int ck = 0; ck < n_full; ++ck)
          attend<0, 1, 0, D>(sm.pk[ck], sm.pv[ck], fo, qf, acc, hf, 0.f,
                             nullptr);
        if (live && (n & 31)) {
          const int lim[1] = {(n & 31) - 1};
          attend<1, 1, 0, D>(sm.pk[n_full], sm.pv[n_full], fo, qf, acc, hf,
                             0.f, lim);
        }
      }

      PT_MARK(kPtPrefix);
      // own keys: chunk c in slot c % 2; chunk c + 2 is loaded into that
      // slot once every wave is done with chunk c
      int b = 0;
      for (;;) {
        const int jr = tokq - o0.tok0;
        const int lim[1] = {(unsigned)jr < (unsigned)o0.T ? jr - o0.k0 : -1};
        if (__any(valid && lim[0] >= 0))
          attend_own<D>(sm.ok[b], (b ? ov1 : ov0) + v_lane_b, ex, fo, qf,
                        acc, hf, lim);
        PT_MARK(kPtOwnCompute);
        if (!has1) break;
        o2 = o1;
        const bool has2 = own_next(o2, np, rtok, rT, rj);
        lds_barrier();  // every wave is done with slot b
        PT_MARK(kPtOwnBarrier);
        if (has2) {
          own_dma<D>(P, u.g, o2, sm.ok[b], sm.ov[b], wave,
                     lane_here<D>(lane));
          vm_wait<OWN_DMA>();  // this wave's loads of chunk c + 1 are in
        } else {
          vm_wait<0>();
        }
        PT_MARK(kPtOwnLoads);
        lds_barrier();  // every wave's loads of chunk c + 1 are in
        PT_MARK(kPtOwnBarrier);
        o0 = o1;
        o1 = o2;
        has1 = has2;
        b ^= 1;
      }

      // normalise; write O (bf16) and the natural-log LSE
      bool bad = false;
      const float lt = acc[0].l + __shfl_xor(acc[0].l, 32, 64);
      if (valid) {
        bad = !(lt >= kLoOk && lt <= kHiOk);
        const float inv = 1.0f / lt;
        const int64_t orow = (int64_t)tokq * P.Hq + head;
        uint16_t *op = P.out + orow * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          float o[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) o[i] = acc[0].o[db][i] * inv;
          uint4 *dst = reinterpret_cast<uint4 *>(op + 32 * db + 16 * hf);
          dst[0] = as_uint4(to_bf16x8(o));
          dst[1] = as_uint4(to_bf16x8(o + 8));
        }
        if (P.lse && hf == 0) P.lse[orow] = __log2f(lt) * kLn2;
      }
      wave_bad = wave_bad || __any(bad);
      PT_MARK(kPtEpilogue);
      lds_barrier();  // the own slots are free for the next pass
      PT_MARK(kPtPassEnd);
      PT_PASS_END(pass_end - pass0);
    }

    PUnit nu{};
    if (wave == 0)
      nu = pass_claim_finish(P, qo, queue, n_work, lane, next_slot, next_x);
    // hand-over: the waves' range flags and the next unit
    if (lane == 0) lds_put(wd + 4 * (1 + wave), wave_bad);
    if (wave == 0 && lane == 0) unit_put(wd + 4 * kWordUnit, nu);
    lds_barrier();
    if (threadIdx.x == 0) {
      bool any_bad = P.flag_all != 0;
      for (int i = 0; i < 8; ++i)
        any_bad = any_bad || lds_get(wd + 4 * (1 + i));
      if (any_bad) P.fix[atomicAdd(&P.counters[kCntFix], 1)] = u.w;
    }
    PT_MARK(kPtUnitEnd);
  }
  PT_FLUSH(wave, lane);
}

}  // namespace

// The pass kernel: k^ of every token first, then 8-wave blocks, one per CU
// at head size 128 (the prefix and two own slots fill the LDS) and two at
// 64, a multiple of 8 blocks so block b serves queue b % 8.
#ifdef DOPR_PASS_TIMERS
// The measurement library's phase totals, [8 waves][kPtSlots], summed over
// every block since the last reset; reset != 0 clears them afterwards.
extern "C" int dopr_pass_phase_read(unsigned long long *out, int reset) {
  hipError_t e = hipMemcpyFromSymbol(out, HIP_SYMBOL(g_pass_phase),
                                     sizeof(g_pass_phase));
  if (e == hipSuccess && reset) {
    static const unsigned long long zero[8][kPtSlots] = {};
    e = hipMemcpyToSymbol(HIP_SYMBOL(g_pass_phase), zero, sizeof(zero));
  }
  return (int)e;
}
#endif

hipError_t launch_stream(int D, const AttnParams &p, const KhatParams &kp,
                         int32_t n_pairs, hipStream_t s) {
  int dev = 0, n_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const unsigned grid = (unsigned)((n_cu + 7) / 8 * 8);
  if (D == 128) {
    if (n_pairs > 0)
      hipLaunchKernelGGL(k_own_khat<128>, dim3((unsigned)n_pairs), dim3(256),
                         0, s, kp);
    hipLaunchKernelGGL(k_pass_attn<128>, dim3(grid), dim3(512), 0, s, p);
  } else {
    if (n_pairs > 0)
      hipLaunchKernelGGL(k_own_khat<64>, dim3((unsigned)n_pairs), dim3(256),
                         0, s, kp);
    hipLaunchKernelGGL(k_pass_attn<64>, dim3(2 * grid), dim3(512), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace dopr

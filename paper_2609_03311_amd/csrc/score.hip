// score.hip -- relevance score read off the score token (Sec. 3.2.3).
//
// The paper feeds the score token's hidden state to a lightweight MLP head;
// here the head is RMSNorm followed by a two-row (yes, no) linear map and
// the score is the log-odds l_yes - l_no.  One workgroup per pair: a single
// streaming pass accumulates sum(h^2), sum(g*h*w_yes) and sum(g*h*w_no),
// then applies 1/rms once (the norm is a common scalar factor).
//
// In last-layer scoring the attention epilogue already produced those three
// sums per (pair, q head); k_score_reduce adds a pair's heads in head order
// (deterministic) and applies the norm.
#include "internal.hpp"

namespace dopr {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ void unpack8f(const uint4 &u, float *f) {
  f[0] = __uint_as_float(u.x << 16);
  f[1] = __uint_as_float(u.x & 0xffff0000u);
  f[2] = __uint_as_float(u.y << 16);
  f[3] = __uint_as_float(u.y & 0xffff0000u);
  f[4] = __uint_as_float(u.z << 16);
  f[5] = __uint_as_float(u.z & 0xffff0000u);
  f[6] = __uint_as_float(u.w << 16);
  f[7] = __uint_as_float(u.w & 0xffff0000u);
}

__global__ __launch_bounds__(kThreads) void k_score(dopr_score_args_t a) {
  __shared__ float red[3][kThreads / 64];
  const int W = a.width;
  const uint16_t *h = static_cast<const uint16_t *>(a.h);
  const uint16_t *nw = static_cast<const uint16_t *>(a.norm_w);
  const uint16_t *wy = static_cast<const uint16_t *>(a.w_head);
  const uint16_t *wn = wy + W;
  for (int32_t p = blockIdx.x; p < a.n_pairs; p += gridDim.x) {
    int64_t row = p;
    if (a.row_index) row = a.row_index[p];
    else if (a.cu_seqlens) row = (int64_t)a.cu_seqlens[p + 1] - 1;
    const uint16_t *x = h + row * a.h_row_stride;
    float ss = 0.f, dy = 0.f, dn = 0.f;
    for (int e = threadIdx.x * 8; e < W; e += kThreads * 8) {
      float xv[8], gv[8], yv[8], nv[8];
      unpack8f(*reinterpret_cast<const uint4 *>(x + e), xv);
      unpack8f(*reinterpret_cast<const uint4 *>(nw + e), gv);
      unpack8f(*reinterpret_cast<const uint4 *>(wy + e), yv);
      unpack8f(*reinterpret_cast<const uint4 *>(wn + e), nv);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ss = fmaf(xv[i], xv[i], ss);
        const float gx = gv[i] * xv[i];
        dy = fmaf(gx, yv[i], dy);
        dn = fmaf(gx, nv[i], dn);
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      ss += __shfl_xor(ss, off, 64);
      dy += __shfl_xor(dy, off, 64);
      dn += __shfl_xor(dn, off, 64);
    }
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    if (lane == 0) {
      red[0][wid] = ss;
      red[1][wid] = dy;
      red[2][wid] = dn;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      float S = 0.f, Y = 0.f, N = 0.f;
      for (int w = 0; w < kThreads / 64; ++w) {
        S += red[0][w];
        Y += red[1][w];
        N += red[2][w];
      }
      const float inv = rsqrtf(S / (float)W + a.rms_eps);
      const float ly = Y * inv, ln = N * inv;
      if (a.logits) {
        a.logits[2 * (int64_t)p] = ly;
        a.logits[2 * (int64_t)p + 1] = ln;
      }
      a.score[p] = ly - ln;
    }
    __syncthreads();
  }
}

// One thread per pair.  Pairs the scheduler did not accept (bad doc id or
// token range) have h = 0, hence logits and score 0.
__global__ __launch_bounds__(kThreads) void k_score_reduce(
    const float *part, const int32_t *pair_flag, int32_t n_pairs, int32_t hq,
    float width, float eps, float *logits, float *score) {
  const int32_t p = blockIdx.x * kThreads + threadIdx.x;
  if (p >= n_pairs) return;
  float ly = 0.f, ln = 0.f;
  if (pair_flag[p] == 1) {
    float S = 0.f, Y = 0.f, N = 0.f;
    const float *pp = part + (int64_t)p * hq * 3;
    for (int32_t h = 0; h < hq; ++h) {
      S += pp[3 * h];
      Y += pp[3 * h + 1];
      N += pp[3 * h + 2];
    }
    const float inv = rsqrtf(S / width + eps);
    ly = Y * inv;
    ln = N * inv;
  }
  if (logits) {
    logits[2 * (int64_t)p] = ly;
    logits[2 * (int64_t)p + 1] = ln;
  }
  score[p] = ly - ln;
}

}  // namespace

hipError_t launch_score_reduce(const Plan &pl, int32_t n_pairs,
                               int32_t n_q_heads, int32_t width,
                               const dopr_score_head_t *head, hipStream_t s) {
  if (n_pairs == 0) return hipSuccess;
  const unsigned grid = (unsigned)((n_pairs + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(k_score_reduce, dim3(grid), dim3(kThreads), 0, s,
                     pl.part, pl.pair_flag, n_pairs, n_q_heads,
                     (float)width, head->rms_eps, head->logits,
                     head->score);
  return hipGetLastError();
}

hipError_t launch_score(const dopr_score_args_t *a, hipStream_t s) {
  if (a->n_pairs == 0) return hipSuccess;
  const unsigned grid = (unsigned)(a->n_pairs < 65536 ? a->n_pairs : 65536);
  hipLaunchKernelGGL(k_score, dim3(grid), dim3(kThreads), 0, s, *a);
  return hipGetLastError();
}

}  // namespace dopr

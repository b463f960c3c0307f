// layer.hip -- one decoder layer of the online pass around the prefix
// attention.
//
// Online, only the query tokens and the score token run through the
// reranker, and every layer's attention also sees the document's stored
// prefix states (Sec. 3.4).  The layer is the Qwen3 decoder layer the paper
// builds on:
//   h  = RMSNorm(x) * g_attn
//   q, k, v = h Wq^T, h Wk^T, h Wv^T          (hipBLASLt, fp32 accumulate)
//   a  = prefix attention of q, k, v          (attn.hip)
//   x2 = x + a Wo^T                           (residual in the GEMM epilogue)
//   h2 = RMSNorm(x2) * g_mlp
//   y  = x2 + (SiLU(h2 Wg^T) * (h2 Wu^T)) Wd^T
// The projections are plain GEMMs (hipBLASLt); the norms and the SiLU gate
// are the hand-written kernels here.  The MLP runs over tokens in chunks so
// its intermediate activations stay small.
#include <hipblaslt/hipblaslt.h>

#include <cmath>
#include <map>
#include <mutex>
#include <tuple>

#include "internal.hpp"

namespace dopr {
namespace {

constexpr int kNormRowsPerBlock = 4;  // one wave per row

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

// fp32 -> bf16, round to nearest even (inputs are finite)
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint4 pack8(const float *f) {
  return make_uint4(bf16_bits(f[0]) | (bf16_bits(f[1]) << 16),
                    bf16_bits(f[2]) | (bf16_bits(f[3]) << 16),
                    bf16_bits(f[4]) | (bf16_bits(f[5]) << 16),
                    bf16_bits(f[6]) | (bf16_bits(f[7]) << 16));
}

// y = RMSNorm(x) * w per row of W elements (W a multiple of 8), fp32 math.
// One wave per row: a first pass sums the squares, a second (cache-hot)
// pass scales and rounds.
__global__ __launch_bounds__(64 * kNormRowsPerBlock) void k_rmsnorm_rows(
    const uint16_t *x, const uint16_t *w, int64_t rows, int32_t W, float eps,
    uint16_t *y) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kNormRowsPerBlock + (threadIdx.x >> 6);
  if (r >= rows) return;
  const uint16_t *xr = x + r * W;
  float ss = 0.f;
  for (int c = lane * 8; c < W; c += 512) {
    float f[8];
    unpack8(*reinterpret_cast<const uint4 *>(xr + c), f);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
  const float inv = rsqrtf(ss / (float)W + eps);
  uint16_t *yr = y + r * W;
  for (int c = lane * 8; c < W; c += 512) {
    float f[8], g[8];
    unpack8(*reinterpret_cast<const uint4 *>(xr + c), f);
    unpack8(*reinterpret_cast<const uint4 *>(w + c), g);
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = g[e] * (f[e] * inv);
    *reinterpret_cast<uint4 *>(yr + c) = pack8(f);
  }
}

// a = SiLU(g) * u with g = gu[:, 0:I] and u = gu[:, I:2I] (row stride 2I),
// fp32 math; SiLU(g) = g / (1 + e^-g).
__global__ __launch_bounds__(256) void k_swiglu(const uint16_t *gu,
                                                int64_t rows, int32_t I,
                                                uint16_t *a) {
  const int64_t per_row = I / 8;
  const int64_t n = rows * per_row;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / per_row, c = (i - r * per_row) * 8;
    float g[8], u[8];
    unpack8(*reinterpret_cast<const uint4 *>(gu + r * 2 * I + c), g);
    unpack8(*reinterpret_cast<const uint4 *>(gu + r * 2 * I + I + c), u);
#pragma unroll
    for (int e = 0; e < 8; ++e) g[e] = g[e] / (1.0f + __expf(-g[e])) * u[e];
    *reinterpret_cast<uint4 *>(a + r * I + c) = pack8(g);
  }
}

// ---------------------------------------------------------------------------
// Row-major Y[M][N] = X[M][K] W[N][K]^T (+ R[M][N]) through hipBLASLt.  In
// its column-major terms D (N x M) = op(A) B + beta C with A = W viewed as a
// K x N matrix, transposed, B = X viewed as K x M, and C = R (or D itself
// when R is Y, in place).

struct GemmKey {
  int dev;
  int64_t m, n, k, ldx, ldy;
  bool acc;
  bool operator<(const GemmKey &o) const {
    return std::tie(dev, m, n, k, ldx, ldy, acc) <
           std::tie(o.dev, o.m, o.n, o.k, o.ldx, o.ldy, o.acc);
  }
};

struct GemmAlgo {
  hipblasLtMatmulAlgo_t algo;
  size_t ws;
};

std::mutex g_mu;
hipblasLtHandle_t g_handle[64] = {};
std::map<GemmKey, GemmAlgo> g_algos;

hipblasStatus_t handle_for(int dev, hipblasLtHandle_t *h) {
  if (dev < 0 || dev >= 64) return HIPBLAS_STATUS_INVALID_VALUE;
  if (!g_handle[dev]) {
    const hipblasStatus_t s = hipblasLtCreate(&g_handle[dev]);
    if (s != HIPBLAS_STATUS_SUCCESS) return s;
  }
  *h = g_handle[dev];
  return HIPBLAS_STATUS_SUCCESS;
}

struct Descs {
  hipblasLtMatmulDesc_t op = nullptr;
  hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
  ~Descs() {
    if (c) hipblasLtMatrixLayoutDestroy(c);
    if (b) hipblasLtMatrixLayoutDestroy(b);
    if (a) hipblasLtMatrixLayoutDestroy(a);
    if (op) hipblasLtMatmulDescDestroy(op);
  }
};

hipblasStatus_t gemm_xwt(int64_t M, int64_t N, int64_t K, const uint16_t *X,
                         int64_t ldx, const uint16_t *Wt, const uint16_t *R,
                         uint16_t *Y, int64_t ldy, void *ws, size_t ws_bytes,
                         hipStream_t stream) {
  const bool accumulate = R != nullptr;
  if (M == 0) return HIPBLAS_STATUS_SUCCESS;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return HIPBLAS_STATUS_INTERNAL_ERROR;
  Descs d;
  hipblasStatus_t s =
      hipblasLtMatmulDescCreate(&d.op, HIPBLAS_COMPUTE_32F, HIP_R_32F);
  if (s != HIPBLAS_STATUS_SUCCESS) return s;
  const hipblasOperation_t ta = HIPBLAS_OP_T, tb = HIPBLAS_OP_N;
  s = hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_TRANSA, &ta,
                                      sizeof(ta));
  if (s != HIPBLAS_STATUS_SUCCESS) return s;
  s = hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_TRANSB, &tb,
                                      sizeof(tb));
  if (s != HIPBLAS_STATUS_SUCCESS) return s;
  if ((s = hipblasLtMatrixLayoutCreate(&d.a, HIP_R_16BF, K, N, K)) !=
          HIPBLAS_STATUS_SUCCESS ||
      (s = hipblasLtMatrixLayoutCreate(&d.b, HIP_R_16BF, K, M, ldx)) !=
          HIPBLAS_STATUS_SUCCESS ||
      (s = hipblasLtMatrixLayoutCreate(&d.c, HIP_R_16BF, N, M, ldy)) !=
          HIPBLAS_STATUS_SUCCESS)
    return s;
  GemmAlgo ga{};
  {
    std::lock_guard<std::mutex> lock(g_mu);
    hipblasLtHandle_t h = nullptr;
    s = handle_for(dev, &h);
    if (s != HIPBLAS_STATUS_SUCCESS) return s;
    const GemmKey key{dev, M, N, K, ldx, ldy, accumulate};
    auto it = g_algos.find(key);
    if (it == g_algos.end()) {
      hipblasLtMatmulPreference_t pref = nullptr;
      s = hipblasLtMatmulPreferenceCreate(&pref);
      if (s != HIPBLAS_STATUS_SUCCESS) return s;
      const uint64_t max_ws = ws_bytes;
      s = hipblasLtMatmulPreferenceSetAttribute(
          pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &max_ws,
          sizeof(max_ws));
      hipblasLtMatmulHeuristicResult_t res[1];
      int got = 0;
      if (s == HIPBLAS_STATUS_SUCCESS)
        s = hipblasLtMatmulAlgoGetHeuristic(h, d.op, d.a, d.b, d.c, d.c, pref,
                                            1, res, &got);
      hipblasLtMatmulPreferenceDestroy(pref);
      if (s != HIPBLAS_STATUS_SUCCESS) return s;
      if (got < 1 || res[0].state != HIPBLAS_STATUS_SUCCESS)
        return HIPBLAS_STATUS_NOT_SUPPORTED;
      it = g_algos.emplace(key, GemmAlgo{res[0].algo, res[0].workspaceSize})
               .first;
    }
    ga = it->second;
    if (ga.ws > ws_bytes) return HIPBLAS_STATUS_INVALID_VALUE;
    const float alpha = 1.f, beta = accumulate ? 1.f : 0.f;
    s = hipblasLtMatmul(h, d.op, &alpha, Wt, d.a, X, d.b, &beta,
                        accumulate ? R : Y, d.c, Y, d.c, &ga.algo, ws,
                        ws_bytes, stream);
  }
  return s;
}

}  // namespace

// Workspace of the layer (on top of the attention plan).
LayerWs layer_carve(void *base, const LayerShape &s) {
  char *p = static_cast<char *>(base);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char *r = p ? p + off : nullptr;
    off = align_up(off + (bytes ? bytes : 1), kAlign);
    return r;
  };
  LayerWs w{};
  const size_t e = sizeof(uint16_t);
  w.h = reinterpret_cast<uint16_t *>(take(e * s.ntok * s.hidden));
  w.q = reinterpret_cast<uint16_t *>(take(e * s.ntok * s.hq * kHeadDim));
  w.k = reinterpret_cast<uint16_t *>(take(e * s.ntok * s.hkv * kHeadDim));
  w.v = reinterpret_cast<uint16_t *>(take(e * s.ntok * s.hkv * kHeadDim));
  w.att = reinterpret_cast<uint16_t *>(take(e * s.ntok * s.hq * kHeadDim));
  w.chunk = s.ntok < kMlpChunk ? s.ntok : kMlpChunk;
  w.gu = reinterpret_cast<uint16_t *>(take(e * w.chunk * 2 * s.inter));
  w.act = reinterpret_cast<uint16_t *>(take(e * w.chunk * s.inter));
  w.gemm_ws = take(kGemmWorkspace);
  w.gemm_ws_bytes = kGemmWorkspace;
  w.plan = take(0);  // the attention plan starts here
  w.bytes = off;
  return w;
}

const char *gemm_status_str(int s) {
  switch (static_cast<hipblasStatus_t>(s)) {
    case HIPBLAS_STATUS_SUCCESS: return "success";
    case HIPBLAS_STATUS_NOT_INITIALIZED: return "not initialized";
    case HIPBLAS_STATUS_ALLOC_FAILED: return "allocation failed";
    case HIPBLAS_STATUS_INVALID_VALUE: return "invalid value";
    case HIPBLAS_STATUS_MAPPING_ERROR: return "mapping error";
    case HIPBLAS_STATUS_EXECUTION_FAILED: return "execution failed";
    case HIPBLAS_STATUS_INTERNAL_ERROR: return "internal error";
    case HIPBLAS_STATUS_NOT_SUPPORTED: return "not supported";
    case HIPBLAS_STATUS_ARCH_MISMATCH: return "architecture mismatch";
    case HIPBLAS_STATUS_HANDLE_IS_NULLPTR: return "null handle";
    case HIPBLAS_STATUS_INVALID_ENUM: return "invalid enum";
    default: return "unknown status";
  }
}

int launch_layer_pre(const LayerShape &s, const dopr_layer_args_t *l,
                     const LayerWs &w, float eps, hipStream_t st) {
  const unsigned nb = (unsigned)((s.ntok + kNormRowsPerBlock - 1) /
                                 kNormRowsPerBlock);
  if (s.ntok > 0)
    hipLaunchKernelGGL(k_rmsnorm_rows, dim3(nb), dim3(64 * kNormRowsPerBlock),
                       0, st, static_cast<const uint16_t *>(l->x),
                       static_cast<const uint16_t *>(l->attn_norm_w), s.ntok,
                       s.hidden, eps, w.h);
  if (hipGetLastError() != hipSuccess) return -1;
  const int64_t hq = (int64_t)s.hq * kHeadDim, hk = (int64_t)s.hkv * kHeadDim;
  hipblasStatus_t g = gemm_xwt(s.ntok, hq, s.hidden, w.h, s.hidden,
                               static_cast<const uint16_t *>(l->w_q), nullptr,
                               w.q, hq, w.gemm_ws, w.gemm_ws_bytes, st);
  if (g == HIPBLAS_STATUS_SUCCESS)
    g = gemm_xwt(s.ntok, hk, s.hidden, w.h, s.hidden,
                 static_cast<const uint16_t *>(l->w_k), nullptr, w.k, hk,
                 w.gemm_ws, w.gemm_ws_bytes, st);
  if (g == HIPBLAS_STATUS_SUCCESS)
    g = gemm_xwt(s.ntok, hk, s.hidden, w.h, s.hidden,
                 static_cast<const uint16_t *>(l->w_v), nullptr, w.v, hk,
                 w.gemm_ws, w.gemm_ws_bytes, st);
  return g == HIPBLAS_STATUS_SUCCESS ? 0 : (int)g;
}

int launch_layer_post(const LayerShape &s, const dopr_layer_args_t *l,
                      const LayerWs &w, float eps, hipStream_t st) {
  uint16_t *y = static_cast<uint16_t *>(l->y);
  const int64_t hq = (int64_t)s.hq * kHeadDim;
  // x2 = x + a Wo^T, written to y (the residual enters as C)
  hipblasStatus_t g = gemm_xwt(s.ntok, s.hidden, hq, w.att, hq,
                               static_cast<const uint16_t *>(l->w_o),
                               static_cast<const uint16_t *>(l->x), y,
                               s.hidden, w.gemm_ws, w.gemm_ws_bytes, st);
  if (g != HIPBLAS_STATUS_SUCCESS) return (int)g;
  // h2 = RMSNorm(x2) for every token (into h, free after the projections)
  const unsigned nb = (unsigned)((s.ntok + kNormRowsPerBlock - 1) /
                                 kNormRowsPerBlock);
  if (s.ntok > 0)
    hipLaunchKernelGGL(k_rmsnorm_rows, dim3(nb), dim3(64 * kNormRowsPerBlock),
                       0, st, y, static_cast<const uint16_t *>(l->mlp_norm_w),
                       s.ntok, s.hidden, eps, w.h);
  if (hipGetLastError() != hipSuccess) return -1;
  // MLP over token chunks: gate and up side by side, SiLU gate, down with
  // the residual accumulated in place
  for (int64_t t0 = 0; t0 < s.ntok; t0 += w.chunk) {
    const int64_t m = s.ntok - t0 < w.chunk ? s.ntok - t0 : w.chunk;
    const uint16_t *h2 = w.h + t0 * s.hidden;
    g = gemm_xwt(m, s.inter, s.hidden, h2, s.hidden,
                 static_cast<const uint16_t *>(l->w_gate), nullptr, w.gu,
                 2 * s.inter, w.gemm_ws, w.gemm_ws_bytes, st);
    if (g == HIPBLAS_STATUS_SUCCESS)
      g = gemm_xwt(m, s.inter, s.hidden, h2, s.hidden,
                   static_cast<const uint16_t *>(l->w_up), nullptr,
                   w.gu + s.inter, 2 * s.inter, w.gemm_ws, w.gemm_ws_bytes,
                   st);
    if (g != HIPBLAS_STATUS_SUCCESS) return (int)g;
    const int64_t n8 = m * (s.inter / 8);
    const unsigned gb = (unsigned)((n8 + 255) / 256 < 8192 ? (n8 + 255) / 256
                                                           : 8192);
    hipLaunchKernelGGL(k_swiglu, dim3(gb), dim3(256), 0, st, w.gu, m,
                       s.inter, w.act);
    if (hipGetLastError() != hipSuccess) return -1;
    g = gemm_xwt(m, s.hidden, s.inter, w.act, s.inter,
                 static_cast<const uint16_t *>(l->w_down),
                 y + t0 * s.hidden, y + t0 * s.hidden, s.hidden, w.gemm_ws,
                 w.gemm_ws_bytes, st);
    if (g != HIPBLAS_STATUS_SUCCESS) return (int)g;
  }
  return 0;
}

}  // namespace dopr

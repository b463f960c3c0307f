// vector_rates.hip -- issue cost of the exponential against a plain
// multiply-add on one GPU, for the softmax cost model of the attention and
// salience kernels.
//
//   hipcc --offload-arch=gfx950 -O3 -o vector_rates vector_rates.hip
//   ./vector_rates
//
// 2048 blocks of four waves each run 4096 iterations of eight independent
// v_exp_f32, of eight independent v_fma_f32, of both interleaved, of four
// independent 32x32x16 bf16 MFMAs, or of those MFMAs with two exponentials
// of the same wave after each; the time of one launch gives the cycles one
// SIMD spends per wave instruction at 2.4 GHz.  The results are summed into one store
// per thread so nothing is left unused.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <vector>
#define CHECK(x) do { hipError_t e = (x); if (e != hipSuccess) { printf("HIP error %s at %d\n", hipGetErrorString(e), __LINE__); return 1; } } while (0)
constexpr int ITERS = 4096;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

// Four independent 32x32x16 bf16 MFMA chains per iteration; with EXP, eight
// exponentials of the same wave between them.
template <bool EXP>
__device__ __forceinline__ float mfma_loop(float seed) {
  bf16x8 a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(seed * (e + 1));
    b[e] = (__bf16)(1.0f / (e + 2));
  }
  floatx16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  float x0 = seed, x1 = seed + 1, x2 = seed + 2, x3 = seed + 3;
  float x4 = seed + 4, x5 = seed + 5, x6 = seed + 6, x7 = seed + 7;
  for (int i = 0; i < ITERS; ++i) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    if (EXP) { asm volatile("v_exp_f32 %0, %0" : "+v"(x0)); asm volatile("v_exp_f32 %0, %0" : "+v"(x1)); }
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    if (EXP) { asm volatile("v_exp_f32 %0, %0" : "+v"(x2)); asm volatile("v_exp_f32 %0, %0" : "+v"(x3)); }
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    if (EXP) { asm volatile("v_exp_f32 %0, %0" : "+v"(x4)); asm volatile("v_exp_f32 %0, %0" : "+v"(x5)); }
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
    if (EXP) { asm volatile("v_exp_f32 %0, %0" : "+v"(x6)); asm volatile("v_exp_f32 %0, %0" : "+v"(x7)); }
  }
  float r = x0 + x1 + x2 + x3 + x4 + x5 + x6 + x7;
  for (int i = 0; i < 16; ++i) r += c0[i] + c1[i] + c2[i] + c3[i];
  return r;
}

template <int KIND>
__global__ __launch_bounds__(256) void k(float *out, float seed) {
  if (KIND == 3 || KIND == 4) {
    out[blockIdx.x * 256 + threadIdx.x] =
        KIND == 4 ? mfma_loop<true>(seed) : mfma_loop<false>(seed);
    return;
  }
  float a0 = seed + threadIdx.x, a1 = a0 + 1, a2 = a0 + 2, a3 = a0 + 3;
  float a4 = a0 + 4, a5 = a0 + 5, a6 = a0 + 6, a7 = a0 + 7;
  float b = 0.5f;
  for (int i = 0; i < ITERS; ++i) {
    if (KIND == 0 || KIND == 2) {
      asm volatile("v_exp_f32 %0, %0" : "+v"(a0)); asm volatile("v_exp_f32 %0, %0" : "+v"(a1));
      asm volatile("v_exp_f32 %0, %0" : "+v"(a2)); asm volatile("v_exp_f32 %0, %0" : "+v"(a3));
      asm volatile("v_exp_f32 %0, %0" : "+v"(a4)); asm volatile("v_exp_f32 %0, %0" : "+v"(a5));
      asm volatile("v_exp_f32 %0, %0" : "+v"(a6)); asm volatile("v_exp_f32 %0, %0" : "+v"(a7));
    }
    if (KIND == 1 || KIND == 2) {
      asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(a0) : "v"(b)); asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(a1) : "v"(b));
      asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(a2) : "v"(b)); asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(a3) : "v"(b));
      asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(a4) : "v"(b)); asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(a5) : "v"(b));
      asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(a6) : "v"(b)); asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(a7) : "v"(b));
    }
  }
  out[blockIdx.x * 256 + threadIdx.x] = a0 + a1 + a2 + a3 + a4 + a5 + a6 + a7;
}
int main() {
  const int blocks = 256 * 8;  // 8 blocks of 4 waves per CU: 8 waves per SIMD
  float *out;
  CHECK(hipMalloc(&out, sizeof(float) * blocks * 256));
  hipEvent_t a, b;
  CHECK(hipEventCreate(&a)); CHECK(hipEventCreate(&b));
  const char *name[5] = {"exp", "fma", "exp+fma", "mfma", "mfma+exp"};
  for (int rep = 0; rep < 2; ++rep)
  for (int kind = 0; kind < 5; ++kind) {
    auto launch = [&]() {
      if (kind == 0) hipLaunchKernelGGL(k<0>, dim3(blocks), dim3(256), 0, 0, out, 0.01f);
      if (kind == 1) hipLaunchKernelGGL(k<1>, dim3(blocks), dim3(256), 0, 0, out, 0.01f);
      if (kind == 2) hipLaunchKernelGGL(k<2>, dim3(blocks), dim3(256), 0, 0, out, 0.01f);
      if (kind == 3) hipLaunchKernelGGL(k<3>, dim3(blocks), dim3(256), 0, 0, out, 0.01f);
      if (kind == 4) hipLaunchKernelGGL(k<4>, dim3(blocks), dim3(256), 0, 0, out, 0.01f);
    };
    launch();
    CHECK(hipDeviceSynchronize());
    CHECK(hipEventRecord(a));
    launch();
    CHECK(hipEventRecord(b));
    CHECK(hipEventSynchronize(b));
    float ms; CHECK(hipEventElapsedTime(&ms, a, b));
    // per SIMD at 2.4 GHz over 1024 SIMDs: cycles per wave instruction of
    // the loop's kind (exp, fma: 8 per iteration; mfma: 4 per iteration)
    const double waves = blocks * 4.0;
    const double per_iter = kind < 3 ? 8.0 : 4.0;
    const double cyc = ms * 1e-3 * 2.4e9 * 1024.0 / (waves * ITERS * per_iter);
    printf("%-8s %8.3f ms  %.1f cycles per wave instruction (%s)\n",
           name[kind], ms, cyc,
           kind < 3 ? "each kind" : kind == 4 ? "per MFMA, 2 exps each"
                                              : "per MFMA");
  }
  CHECK(hipFree(out));
  return 0;
}

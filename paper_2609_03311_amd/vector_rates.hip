// vector_rates.hip -- issue cost of the exponential against a plain
// multiply-add on one GPU, for the softmax cost model of the attention and
// salience kernels.
//
//   hipcc --offload-arch=gfx950 -O3 -o vector_rates vector_rates.hip
//   ./vector_rates
//
// 2048 blocks of four waves (eight waves per SIMD) each run 4096 iterations
// of eight independent v_exp_f32, of eight independent v_fma_f32, or of
// both interleaved; the time of one launch gives the cycles one SIMD spends
// per wave instruction at 2.4 GHz.  The results are summed into one store
// per thread so nothing is left unused.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <vector>
#define CHECK(x) do { hipError_t e = (x); if (e != hipSuccess) { printf("HIP error %s at %d\n", hipGetErrorString(e), __LINE__); return 1; } } while (0)
constexpr int ITERS = 4096;
template <int KIND>
__global__ __launch_bounds__(256) void k(float *out, float seed) {
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
  const char *name[3] = {"exp", "fma", "exp+fma"};
  for (int rep = 0; rep < 2; ++rep)
  for (int kind = 0; kind < 3; ++kind) {
    auto launch = [&]() {
      if (kind == 0) hipLaunchKernelGGL(k<0>, dim3(blocks), dim3(256), 0, 0, out, 0.01f);
      if (kind == 1) hipLaunchKernelGGL(k<1>, dim3(blocks), dim3(256), 0, 0, out, 0.01f);
      if (kind == 2) hipLaunchKernelGGL(k<2>, dim3(blocks), dim3(256), 0, 0, out, 0.01f);
    };
    launch();
    CHECK(hipDeviceSynchronize());
    CHECK(hipEventRecord(a));
    launch();
    CHECK(hipEventRecord(b));
    CHECK(hipEventSynchronize(b));
    float ms; CHECK(hipEventElapsedTime(&ms, a, b));
    const double waves = blocks * 4.0, instr = waves * ITERS * 8;
    // wave instructions per SIMD per cycle at 2.4 GHz over 1024 SIMDs
    const double per_simd_cycle = instr / 1024.0 / (ms * 1e-3 * 2.4e9);
    printf("%-8s %8.3f ms  %.4f wave-instr of each kind per SIMD-cycle (%.1f cycles each)\n",
           name[kind], ms, per_simd_cycle, 1.0 / per_simd_cycle);
  }
  CHECK(hipFree(out));
  return 0;
}

// Matrix-core ceiling of the GPU: the best rate of dense 32x32x16 bf16 MFMA
// instructions (the shape the prefill and influence kernels use) with operands
// in registers and four independent accumulators per wave, over a sweep of
// waves per SIMD.  Nothing but the instructions and the loop runs, so this is
// the practical roof for MFMA-bound kernels on this GPU (the published
// 2.5 PFLOP/s assumes the peak clock, which the part does not hold under a
// full matrix load).  Prints one line per configuration and a final
// "best <TFLOP/s>" line.  With an argument S > 0 it then keeps the 2-waves-
// per-SIMD configuration running for about S seconds (for sampling the board
// power and clock under a pure matrix load) and prints "hold <TFLOP/s>".
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// MFMA steps per SIMD in every configuration (about 4 ms of work, so clock
// ramp-up and launch spread do not decide the result).
constexpr int kStepsPerSimd = 65536;

__global__ void __launch_bounds__(256) mfma_loop(float* out, float seed, int iters) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<__bf16>(seed * float(threadIdx.x + i));
    b[i] = static_cast<__bf16>(seed * float(i - int(threadIdx.x)));
  }
  f32x16 acc[4] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;   // keeps the products
}

int main(int argc, char** argv) {
  const double hold_s = argc > 1 ? std::atof(argv[1]) : 0.0;
  const int max_blocks = 4096;
  float* out = nullptr;
  if (hipMalloc(&out, sizeof(float) * max_blocks * 256) != hipSuccess) {
    std::fprintf(stderr, "allocation failed\n");
    return 1;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0) != hipSuccess || cus < 1) return 1;
  double best = 0.0;
  for (int per_simd : {1, 2, 4, 8, 16}) {
    const int blocks = cus * per_simd;                // 4 waves per block = one per SIMD
    const int iters = kStepsPerSimd / per_simd;
    if (blocks > max_blocks) break;
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return 1;
    hipLaunchKernelGGL(mfma_loop, dim3(blocks), dim3(256), 0, 0, out, 1e-3f, iters);
    float ms_best = 1e30f;
    for (int r = 0; r < 5; ++r) {
      (void)hipEventRecord(e0);
      hipLaunchKernelGGL(mfma_loop, dim3(blocks), dim3(256), 0, 0, out, 1e-3f, iters);
      (void)hipEventRecord(e1);
      if (hipEventSynchronize(e1) != hipSuccess) return 1;
      float ms = 0.0f;
      (void)hipEventElapsedTime(&ms, e0, e1);
      ms_best = ms < ms_best ? ms : ms_best;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    const double flops = double(blocks) * 4 /* waves */ * iters * 4 /* chains */ * 2.0 * 32 * 32 * 16;
    const double tf = flops / (ms_best / 1e3) / 1e12;
    std::printf("waves per SIMD %2d: %8.1f TFLOP/s\n", per_simd, tf);
    best = tf > best ? tf : best;
  }
  std::printf("best %.1f\n", best);
  if (hold_s > 0.0) {
    const int blocks = cus * 2, iters = kStepsPerSimd / 2;
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return 1;
    double flops = 0.0, ms_total = 0.0;
    while (ms_total < hold_s * 1e3) {
      (void)hipEventRecord(e0);
      hipLaunchKernelGGL(mfma_loop, dim3(blocks), dim3(256), 0, 0, out, 1e-3f, iters);
      (void)hipEventRecord(e1);
      if (hipEventSynchronize(e1) != hipSuccess) return 1;
      float ms = 0.0f;
      (void)hipEventElapsedTime(&ms, e0, e1);
      ms_total += ms;
      flops += double(blocks) * 4 * iters * 4 * 2.0 * 32 * 32 * 16;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    std::printf("hold %.1f\n", flops / (ms_total / 1e3) / 1e12);
  }
  (void)hipFree(out);
  return 0;
}

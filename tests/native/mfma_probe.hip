// mfma_probe.hip -- test-only probe (part of libqgprobe.so, not of libqgemm.so).
//
// Issue rates of the matrix instructions an exact NVFP4 GEMM can run on:
// the K = 16 FP8 instruction (v_mfma_f32_32x32x16_fp8_fp8, the operand shape
// of one NVFP4 16-block), the fp16 instruction the W4A4 kernels use
// (v_mfma_f32_32x32x16_f16) and the K = 64 fp8 / fp4 instruction
// (v_mfma_scale_f32_32x32x64_f8f6f4). Each wave runs NACC independent
// 32 x 32 accumulators for `iters` rounds, one wave per SIMD (four per
// workgroup), on all-ones operands, so every accumulator element ends at
// iters * K exactly: the host checks that, then divides the flops by the
// kernel time. Bounded loops, no memory traffic besides the final store.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef int v8i __attribute__((ext_vector_type(8)));

constexpr int NACC = 8;

// which: 0 = fp8 K=16, 1 = f16 K=16, 2 = fp8 K=64, 3 = fp4 K=64
template <int WHICH>
__global__ void __launch_bounds__(256) k_mfma_rate(float* out, int iters) {
  v16f acc[NACC];
#pragma unroll
  for (int a = 0; a < NACC; ++a)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[a][v] = 0.0f;
  const long ones8 = 0x3838383838383838l;                    // eight E4M3 1.0
  const v8h onesh = {1, 1, 1, 1, 1, 1, 1, 1};
  const v8i ones8x32 = {0x38383838, 0x38383838, 0x38383838, 0x38383838,
                        0x38383838, 0x38383838, 0x38383838, 0x38383838};
  const v8i ones4x64 = {0x22222222, 0x22222222, 0x22222222, 0x22222222, 0, 0, 0, 0};  // E2M1 1.0 = 0x2
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int a = 0; a < NACC; ++a) {
      if (WHICH == 0) acc[a] = __builtin_amdgcn_mfma_f32_32x32x16_fp8_fp8(ones8, ones8, acc[a], 0, 0, 0);
      if (WHICH == 1) acc[a] = __builtin_amdgcn_mfma_f32_32x32x16_f16(onesh, onesh, acc[a], 0, 0, 0);
      if (WHICH == 2) acc[a] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ones8x32, ones8x32, acc[a], 0, 0, 0, 0, 0, 0);
      if (WHICH == 3) acc[a] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ones4x64, ones4x64, acc[a], 4, 4, 0, 127, 0, 127);
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int a = 0; a < NACC; ++a)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[a][v];
  // every element equals iters * K: the sum over the lane's 16 x NACC values
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

extern "C" int qgp_mfma_rate(int which, float* out, int blocks, int iters, float* ms) {
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return -1;
  auto launch = [&]() {
    if (which == 0) hipLaunchKernelGGL(k_mfma_rate<0>, dim3(blocks), dim3(256), 0, 0, out, iters);
    else if (which == 1) hipLaunchKernelGGL(k_mfma_rate<1>, dim3(blocks), dim3(256), 0, 0, out, iters);
    else if (which == 2) hipLaunchKernelGGL(k_mfma_rate<2>, dim3(blocks), dim3(256), 0, 0, out, iters);
    else hipLaunchKernelGGL(k_mfma_rate<3>, dim3(blocks), dim3(256), 0, 0, out, iters);
  };
  launch();                                 // warm-up (clocks, code object)
  hipEventRecord(e0, 0);
  launch();
  hipEventRecord(e1, 0);
  hipEventSynchronize(e1);
  hipEventElapsedTime(ms, e0, e1);
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  return (int)hipGetLastError();
}

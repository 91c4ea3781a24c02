// cvt_probe.hip -- test-only probe library (not part of libqgemm.so).
//
// Compares the library's hardware float -> E2M1 / E4M3 encoders (hw_e2m1x8,
// hw_e4m3x4 in csrc/common.hpp, built on v_cvt_scalef32_pk_fp4_f32 and
// v_cvt_scalef32_pk_fp8_f32) with its integer encoders (checked against the
// CPU oracle on every fp32 input) over all 2^32 fp32 bit patterns, and reports
// how the hardware E2M1 -> fp16 conversion treats a scale that is not a power
// of two. Every kernel is a bounded grid-stride loop over a fixed index
// range; outputs are a handful of counters.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

using namespace qg;

// The library's hardware encoders (hw_e2m1x8 / hw_e4m3x4) against its integer
// encoders on every fp32 input. Each thread converts 8 (resp. 4) inputs spaced
// `stride` apart. counts[0] = mismatches, counts[1] = mismatches on finite
// inputs; first[0..7] = some mismatching inputs, first[8..15] = hardware codes.
__device__ inline void note(unsigned long long* counts, uint32_t* first, uint32_t u, uint32_t h) {
  const unsigned long long c = atomicAdd(&counts[0], 1ull);
  if ((u & 0x7F800000u) != 0x7F800000u) atomicAdd(&counts[1], 1ull);
  if (c < 8) { first[c] = u; first[8 + c] = h; }
}

__global__ void k_probe_fp4(unsigned long long* counts, uint32_t* first) {
  const uint64_t nthreads = (uint64_t)gridDim.x * blockDim.x;   // 2^20
  const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  // 2^32 inputs = nthreads * 8 lanes-of-work * 512 rounds
  for (uint64_t r = 0; r < (1ull << 32) / (nthreads * 8); ++r) {
    float y[8];
    uint32_t u[8];
    for (int j = 0; j < 8; ++j) {
      u[j] = (uint32_t)(((r * 8 + j) * nthreads) + t);
      y[j] = u2f(u[j]);
    }
    const uint32_t hw = hw_e2m1x8(y);
    for (int j = 0; j < 8; ++j) {
      const uint32_t h = (hw >> (4 * j)) & 0xFu;
      if (h != enc_e2m1(y[j])) note(counts, first, u[j], h);
    }
  }
}

__global__ void k_probe_fp8(unsigned long long* counts, uint32_t* first) {
  const uint64_t nthreads = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (uint64_t r = 0; r < (1ull << 32) / (nthreads * 4); ++r) {
    float y[4];
    uint32_t u[4];
    for (int j = 0; j < 4; ++j) {
      u[j] = (uint32_t)(((r * 4 + j) * nthreads) + t);
      y[j] = u2f(u[j]);
    }
    const uint32_t hw = hw_e4m3x4(y);
    for (int j = 0; j < 4; ++j) {
      const uint32_t h = (hw >> (8 * j)) & 0xFFu;
      if (h != enc_e4m3(y[j])) note(counts, first, u[j], h);
    }
  }
}

// For every E2M1 code and every E4M3 block-scale code: the fp16 results of
// v_cvt_scalef32_pk_f16_fp4 with (a) scale 1.0 and (b) the block scale passed
// as the fp32 scale operand. out[(s * 16 + c) * 2 + {0,1}] = fp16 bits.
__global__ void k_probe_f16_scale(uint16_t* out) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= 256 * 16) return;
  const uint32_t s = (uint32_t)t >> 4, c = (uint32_t)t & 15u;
  const float sc = dec_e4m3(s);
  const v2h a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 0);
  const v2h b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, sc, 0);
  out[2 * t] = __builtin_bit_cast(uint16_t, (_Float16)a[0]);
  out[2 * t + 1] = __builtin_bit_cast(uint16_t, (_Float16)b[0]);
}

// The GEMM kernels' E4M3 block-scale decoders on every code: for code c
// (0..255) placed in byte position b (0..3) of a dword,
//   f32[4 c + b] = v_cvt_pk_f32_fp8 (hardware, the W4A16 weight-pool kernels),
//   and, for c < 128 (block scales are magnitudes),
//   ref[4 c + b] = dec_e4m3_scale (the W4A16 split-K kernel),
//   h16[4 c + b] = e4m3x4_to_f16x4 (the W4A4 kernels; v_cvt_scalef32_pk_f16_fp8).
__global__ void k_probe_scale_decoders(float* f32, float* ref, uint16_t* h16) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= 256 * 4) return;
  const uint32_t c = (uint32_t)t >> 2, b = (uint32_t)t & 3u;
  const uint32_t d = c << (8 * b);
  const v2f lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)d, false), hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)d, true);
  f32[t] = (b == 0) ? lo[0] : (b == 1) ? lo[1] : (b == 2) ? hi[0] : hi[1];
  if (c >= 128u) return;
  ref[t] = dec_e4m3_scale(d >> (8 * b));
  const uint2 h = e4m3x4_to_f16x4(d);
  const uint32_t w = (b < 2) ? h.x : h.y;
  h16[t] = (uint16_t)((b & 1) ? (w >> 16) : (w & 0xFFFFu));
}

extern "C" int qgp_probe_cvt(int which, unsigned long long* counts, uint32_t* first) {
  // 4096 x 256 = 2^20 threads; the loops above cover exactly [0, 2^32)
  if (which == 0)
    hipLaunchKernelGGL(k_probe_fp4, dim3(4096), dim3(256), 0, 0, counts, first);
  else
    hipLaunchKernelGGL(k_probe_fp8, dim3(4096), dim3(256), 0, 0, counts, first);
  return (int)hipGetLastError();
}

extern "C" int qgp_probe_f16_scale(uint16_t* out) {
  hipLaunchKernelGGL(k_probe_f16_scale, dim3(16), dim3(256), 0, 0, out);
  return (int)hipGetLastError();
}

extern "C" int qgp_probe_scale_decoders(float* f32, float* ref, uint16_t* h16) {
  hipLaunchKernelGGL(k_probe_scale_decoders, dim3(4), dim3(256), 0, 0, f32, ref, h16);
  return (int)hipGetLastError();
}

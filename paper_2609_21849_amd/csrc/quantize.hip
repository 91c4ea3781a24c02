// quantize.hip -- activation/weight quantizers and dequantizers (gfx950).
//
// Dynamic per-tensor quantization of bf16 tensors to FP8 E4M3 and to NVFP4
// (E2M1 elements, E4M3 scale per 16 consecutive elements, fp32 tensor
// scale), the run-time activation quantization that the paper's recipe
// relies on for its speed-up on compute-bound stages (Sec. 4, quantization
// paragraph; Table 2). The same kernels quantize weights offline (PTQ).
//
// A tensor-wide scale needs the tensor-wide max before any element can be
// coded, so one call is a short chain on the caller's stream:
//   k_fill       : zero the fp32 scale slot (a kernel, not a memset, so the
//                  chain can be captured in a HIP graph)
//   k_amax       : max |x| as integer max of bf16 magnitude bits, wave
//                  reduction, one atomicMax per workgroup on the slot (the
//                  bit pattern of a non-negative float orders like the float)
//   k_finalize   : slot (amax bits) -> decode scale s or s_t, in place
//   k_quant_*    : each thread codes 16 elements with the finished scale
// Stream order separates the kernels; nothing waits on the host.
#include "common.hpp"
#include "kernels.hpp"

namespace qg {

__global__ void k_fill_u32(uint32_t* p, uint32_t v) { *p = v; }

// ---------------------------------------------------------------- amax
// Rows of `cols` bf16 elements, `ldx` apart. VEC: rows are 16-byte aligned
// and cols % 8 == 0, so each step reads 8 elements with one 16-byte load.
template <bool VEC>
__global__ void __launch_bounds__(256) k_amax(const uint16_t* __restrict__ x, int64_t rows,
                                              int64_t cols, int64_t ldx, uint32_t* slot) {
  uint32_t m = 0;
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
    const uint16_t* xr = x + r * ldx;
    if (VEC) {
      const int64_t units = cols >> 3;
      for (int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x; u < units;
           u += (int64_t)gridDim.x * 256) {
        const uint4 v = *reinterpret_cast<const uint4*>(xr + u * 8);
        const uint32_t w0 = v.x & 0x7FFF7FFFu, w1 = v.y & 0x7FFF7FFFu;
        const uint32_t w2 = v.z & 0x7FFF7FFFu, w3 = v.w & 0x7FFF7FFFu;
        m = max(m, max(max(w0 & 0xFFFFu, w0 >> 16), max(w1 & 0xFFFFu, w1 >> 16)));
        m = max(m, max(max(w2 & 0xFFFFu, w2 >> 16), max(w3 & 0xFFFFu, w3 >> 16)));
      }
    } else {
      for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < cols;
           c += (int64_t)gridDim.x * 256)
        m = max(m, (uint32_t)(xr[c] & 0x7FFFu));
    }
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    m = max(max(part[0], part[1]), max(part[2], part[3]));
    if (m) atomicMax(slot, m << 16);  // bf16 magnitude bits -> fp32 bits
  }
}

// amax bits -> decode scale. divisor = 448 (FP8) or 2688 = 448 * 6 (NVFP4).
// Inf/NaN anywhere in the tensor leaves a NaN scale as the sentinel.
__global__ void k_finalize(uint32_t* slot, float divisor) {
  const uint32_t a = *slot;
  const float s = (a >= 0x7F800000u) ? __builtin_nanf("") : __fdiv_rn(u2f(a), divisor);
  *reinterpret_cast<float*>(slot) = s;
}

// ---------------------------------------------------------------- element access
// 16 consecutive bf16 of one row as fp32 (exact).
template <bool VEC>
__device__ inline void load16(const uint16_t* p, float (&v)[16]) {
  if (VEC) {
    const uint4 a = reinterpret_cast<const uint4*>(p)[0];
    const uint4 b = reinterpret_cast<const uint4*>(p)[1];
    const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      v[2 * i] = bf16_lo(w[i]);
      v[2 * i + 1] = bf16_hi(w[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = u2f((uint32_t)p[i] << 16);
  }
}

// ---------------------------------------------------------------- FP8
// One thread codes 16 consecutive elements of a row: q = E4M3(x * r), r = 1/s.
// CONTIG: the tensor is one dense run of n elements (ldx == cols); a thread
// owns elements [16 t, 16 t + 16) and the last thread may be partial.
// Otherwise rows are handled as units of 16 (VEC requires cols % 16 == 0).
template <bool VEC, bool CONTIG>
__global__ void __launch_bounds__(256) k_quant_fp8(const uint16_t* __restrict__ x, int64_t rows,
                                                   int64_t cols, int64_t ldx,
                                                   uint8_t* __restrict__ q,
                                                   const float* __restrict__ scale) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const float s = *scale;
  const float r = (s > 0.0f) ? __fdiv_rn(1.0f, s) : 0.0f;
  int64_t src, dst, cnt;
  if (CONTIG) {
    const int64_t n = rows * cols;
    src = dst = t * 16;
    if (src >= n) return;
    cnt = min((int64_t)16, n - src);
  } else {
    const int64_t upr = (cols + 15) >> 4;
    const int64_t row = t / upr, u = t - row * upr;
    if (row >= rows) return;
    src = row * ldx + u * 16;
    dst = row * cols + u * 16;
    cnt = min((int64_t)16, cols - u * 16);
  }
  if (VEC && cnt == 16) {
    float v[16];
    load16<true>(x + src, v);
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = enc_e4m3(__fmul_rn(v[4 * i], r)) | (enc_e4m3(__fmul_rn(v[4 * i + 1], r)) << 8) |
             (enc_e4m3(__fmul_rn(v[4 * i + 2], r)) << 16) |
             (enc_e4m3(__fmul_rn(v[4 * i + 3], r)) << 24);
    *reinterpret_cast<uint4*>(q + dst) = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
    for (int64_t i = 0; i < cnt; ++i)
      q[dst + i] = (uint8_t)enc_e4m3(__fmul_rn(u2f((uint32_t)x[src + i] << 16), r));
  }
}

// ---------------------------------------------------------------- NVFP4
// One thread per 16-element block: block max, E4M3 block scale, then the 16
// E2M1 codes packed into 8 bytes (element 2i in the low nibble).
template <bool VEC, bool CONTIG>
__global__ void __launch_bounds__(256) k_quant_nvfp4(const uint16_t* __restrict__ x, int64_t rows,
                                                     int64_t cols, int64_t ldx,
                                                     uint8_t* __restrict__ q,
                                                     uint8_t* __restrict__ bscale,
                                                     const float* __restrict__ tscale) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t bpr = cols >> 4;
  int64_t src;
  if (CONTIG) {
    if (t >= rows * bpr) return;
    src = t * 16;
  } else {
    const int64_t row = t / bpr, b = t - row * bpr;
    if (row >= rows) return;
    src = row * ldx + b * 16;
  }
  float v[16];
  load16<VEC>(x + src, v);
  uint32_t amax_bits = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) amax_bits = max(amax_bits, f2u(v[i]) & 0x7FFFFFFFu);
  const float s_t = *tscale;
  const float d_t = __fmul_rn(6.0f, s_t);
  const float vb = (d_t > 0.0f) ? __fdiv_rn(u2f(amax_bits), d_t) : 0.0f;
  const uint32_t sb = enc_e4m3(vb);
  const float S = __fmul_rn(dec_e4m3(sb), s_t);
  const float r = (S > 0.0f) ? __fdiv_rn(1.0f, S) : 0.0f;
  uint32_t w[2] = {0u, 0u};
#pragma unroll
  for (int i = 0; i < 16; ++i) w[i >> 3] |= enc_e2m1(__fmul_rn(v[i], r)) << (4 * (i & 7));
  *reinterpret_cast<uint2*>(q + t * 8) = make_uint2(w[0], w[1]);
  bscale[t] = (uint8_t)sb;
}

// ---------------------------------------------------------------- dequant
// out = fl(e4m3(q) * s)  or  fl(fl(e2m1(q) * e4m3(s_b)) * s_t), as fp32 or
// RNE bf16; one thread per 16 consecutive elements of the dense tensor.
template <bool F32OUT>
__device__ inline void store16(void* out, int64_t e, const float (&v)[16], int64_t cnt, bool vec) {
  if (F32OUT) {
    float* o = reinterpret_cast<float*>(out) + e;
    if (vec && cnt == 16) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        reinterpret_cast<float4*>(o)[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
    } else {
      for (int64_t i = 0; i < cnt; ++i) o[i] = v[i];
    }
  } else {
    uint16_t* o = reinterpret_cast<uint16_t*>(out) + e;
    if (vec && cnt == 16) {
      uint32_t w[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) w[i] = f32_to_bf16(v[2 * i]) | (f32_to_bf16(v[2 * i + 1]) << 16);
      reinterpret_cast<uint4*>(o)[0] = make_uint4(w[0], w[1], w[2], w[3]);
      reinterpret_cast<uint4*>(o)[1] = make_uint4(w[4], w[5], w[6], w[7]);
    } else {
      for (int64_t i = 0; i < cnt; ++i) o[i] = (uint16_t)f32_to_bf16(v[i]);
    }
  }
}

template <bool F32OUT>
__global__ void __launch_bounds__(256) k_dequant_fp8(const uint8_t* __restrict__ q, int64_t n,
                                                     const float* __restrict__ scale, void* out,
                                                     bool vec) {
  const int64_t e = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 16;
  if (e >= n) return;
  const int64_t cnt = min((int64_t)16, n - e);
  const float s = *scale;
  float v[16];
  if (vec && cnt == 16) {
    const uint4 c = *reinterpret_cast<const uint4*>(q + e);
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = __fmul_rn(dec_e4m3((w[i >> 2] >> (8 * (i & 3))) & 0xFFu), s);
  } else {
    for (int64_t i = 0; i < cnt; ++i) v[i] = __fmul_rn(dec_e4m3(q[e + i]), s);
  }
  store16<F32OUT>(out, e, v, cnt, vec);
}

template <bool F32OUT>
__global__ void __launch_bounds__(256) k_dequant_nvfp4(const uint8_t* __restrict__ q,
                                                       const uint8_t* __restrict__ bscale,
                                                       int64_t nblocks,
                                                       const float* __restrict__ tscale,
                                                       void* out, bool vec) {
  const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (b >= nblocks) return;
  const float s_t = *tscale;
  const float sb = dec_e4m3(bscale[b]);
  const uint2 c = *reinterpret_cast<const uint2*>(q + b * 8);
  const uint32_t w[2] = {c.x, c.y};
  float v[16];
#pragma unroll
  for (int i = 0; i < 16; ++i)
    v[i] = __fmul_rn(__fmul_rn(dec_e2m1((w[i >> 3] >> (4 * (i & 7))) & 0xFu), sb), s_t);
  store16<F32OUT>(out, b * 16, v, 16, vec);
}

// ---------------------------------------------------------------- launchers
static inline unsigned grid_for(int64_t threads) { return (unsigned)((threads + 255) / 256); }

hipError_t launch_quantize(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ldx,
                           uint8_t* codes, uint8_t* bscale, float* tscale, hipStream_t st) {
  uint32_t* slot = reinterpret_cast<uint32_t*>(tscale);
  hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(1), 0, st, slot, 0u);
  if (rows == 0 || cols == 0) return hipGetLastError();
  const bool contig = (ldx == cols);
  const bool aligned = (reinterpret_cast<uintptr_t>(x) % 16 == 0);
  // amax
  {
    const int64_t r_eff = contig ? 1 : rows;
    const int64_t c_eff = contig ? rows * cols : cols;
    const bool vec = aligned && (c_eff % 8 == 0) && (contig || ldx % 8 == 0);
    const int64_t per_row = vec ? c_eff / 8 : c_eff;
    unsigned gx = (unsigned)std::min<int64_t>(std::max<int64_t>(1, (per_row + 255) / 256), 4096);
    unsigned gy = (unsigned)std::min<int64_t>(r_eff, 65535);
    if ((int64_t)gx * gy > 8192) gx = std::max<unsigned>(1u, 8192u / gy);
    if (vec)
      hipLaunchKernelGGL(k_amax<true>, dim3(gx, gy), dim3(256), 0, st, x, r_eff, c_eff, contig ? c_eff : ldx, slot);
    else
      hipLaunchKernelGGL(k_amax<false>, dim3(gx, gy), dim3(256), 0, st, x, r_eff, c_eff, contig ? c_eff : ldx, slot);
  }
  hipLaunchKernelGGL(k_finalize, dim3(1), dim3(1), 0, st, slot, fmt == 1 ? 448.0f : 2688.0f);
  if (fmt == 1) {
    const bool qal = (reinterpret_cast<uintptr_t>(codes) % 16 == 0);
    if (contig) {
      const bool vec = aligned && qal;
      const unsigned g = grid_for((rows * cols + 15) / 16);
      if (vec) hipLaunchKernelGGL((k_quant_fp8<true, true>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, tscale);
      else hipLaunchKernelGGL((k_quant_fp8<false, true>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, tscale);
    } else {
      const bool vec = aligned && qal && (ldx % 8 == 0) && (cols % 16 == 0);
      const unsigned g = grid_for(rows * ((cols + 15) / 16));
      if (vec) hipLaunchKernelGGL((k_quant_fp8<true, false>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, tscale);
      else hipLaunchKernelGGL((k_quant_fp8<false, false>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, tscale);
    }
  } else {
    const unsigned g = grid_for(rows * (cols / 16));
    const bool vec = aligned && (contig || ldx % 8 == 0);
    if (contig) {
      if (vec) hipLaunchKernelGGL((k_quant_nvfp4<true, true>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, bscale, tscale);
      else hipLaunchKernelGGL((k_quant_nvfp4<false, true>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, bscale, tscale);
    } else {
      if (vec) hipLaunchKernelGGL((k_quant_nvfp4<true, false>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, bscale, tscale);
      else hipLaunchKernelGGL((k_quant_nvfp4<false, false>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, bscale, tscale);
    }
  }
  return hipGetLastError();
}

hipError_t launch_dequant(int fmt, const uint8_t* codes, const uint8_t* bscale, const float* tscale,
                          int64_t rows, int64_t cols, void* out, bool f32out, hipStream_t st) {
  const int64_t n = rows * cols;
  if (n == 0) return hipSuccess;
  if (fmt == 1) {
    const bool vec = (reinterpret_cast<uintptr_t>(codes) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(out) % 16 == 0);
    const unsigned g = grid_for((n + 15) / 16);
    if (f32out) hipLaunchKernelGGL(k_dequant_fp8<true>, dim3(g), dim3(256), 0, st, codes, n, tscale, out, vec);
    else hipLaunchKernelGGL(k_dequant_fp8<false>, dim3(g), dim3(256), 0, st, codes, n, tscale, out, vec);
  } else {
    const int64_t nb = n / 16;
    const unsigned g = grid_for(nb);
    const bool vec = (reinterpret_cast<uintptr_t>(out) % 16 == 0);
    if (f32out) hipLaunchKernelGGL(k_dequant_nvfp4<true>, dim3(g), dim3(256), 0, st, codes, bscale, nb, tscale, out, vec);
    else hipLaunchKernelGGL(k_dequant_nvfp4<false>, dim3(g), dim3(256), 0, st, codes, bscale, nb, tscale, out, vec);
  }
  return hipGetLastError();
}

}  // namespace qg

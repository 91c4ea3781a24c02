// quantize.hip -- activation/weight quantizers and dequantizers (gfx950).
//
// Dynamic per-tensor quantization of bf16 tensors to FP8 E4M3 and to NVFP4
// (E2M1 elements, E4M3 scale per 16 consecutive elements, fp32 tensor
// scale), the run-time activation quantization that the paper's recipe
// relies on for its speed-up on compute-bound stages (Sec. 4, quantization
// paragraph; Table 2). The same kernels quantize weights offline (PTQ).
//
// A tensor-wide scale needs the tensor-wide max before any element can be
// coded. A small tensor (at most 3072 units of 16 elements) is quantized in
// one launch (k_quant_small); a dense one of at most 3 Mi elements in two
// (k_amax_slots, k_quant_dense_slots: the maxima handed over inside the code
// buffer); any other is a short chain on the caller's stream:
//   k_amax_dense / : max |x| as an integer max of bf16 magnitude bits (the
//   k_amax_partial   bit pattern of a non-negative value orders like the
//                    value); one partial per workgroup, parked in the code
//                    buffer that the last kernel overwrites anyway
//   k_finalize     : max of the partials -> decode scale s or s_t
//   k_quant_*      : code the elements with the finished scale
// Stream order separates the kernels; nothing waits on the host.
#include "common.hpp"
#include "kernels.hpp"
#include "quant_plan.hpp"

namespace qg {

__global__ void k_fill_u32(uint32_t* p, uint32_t v) { *p = v; }

// ---------------------------------------------------------------- amax
// Rows of `cols` bf16 elements, `ldx` apart. VEC: rows are 16-byte aligned
// and cols % 8 == 0, so each step reads 8 elements with one 16-byte load.
// Each workgroup writes the bf16 magnitude bits of its max to partial[id];
// there are no atomics, so thousands of workgroups do not serialise on one
// address. k_finalize reduces the partials.
template <bool VEC>
__global__ void __launch_bounds__(256) k_amax_partial(const uint16_t* __restrict__ x, int64_t rows,
                                                      int64_t cols, int64_t ldx,
                                                      uint32_t* __restrict__ partial) {
  uint32_t m = 0;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
    const uint16_t* xr = x + r * ldx;
    if (VEC) {
      const int64_t units = cols >> 3;
      const uint4* xv = reinterpret_cast<const uint4*>(xr);
      int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
      for (; u + 3 * stride < units; u += 4 * stride) {
        const uint4 v0 = xv[u], v1 = xv[u + stride], v2 = xv[u + 2 * stride], v3 = xv[u + 3 * stride];
        const uint32_t w[16] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w,
                          v2.x, v2.y, v2.z, v2.w, v3.x, v3.y, v3.z, v3.w};
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const uint32_t t = w[i] & 0x7FFF7FFFu;
          m = max(m, max(t & 0xFFFFu, t >> 16));
        }
      }
      for (; u < units; u += stride) {
        const uint4 v = xv[u];
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t t = w[i] & 0x7FFF7FFFu;
          m = max(m, max(t & 0xFFFFu, t >> 16));
        }
      }
    } else {
      for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < cols; c += stride)
        m = max(m, (uint32_t)(xr[c] & 0x7FFFu));
    }
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0)
    partial[blockIdx.y * gridDim.x + blockIdx.x] = max(max(part[0], part[1]), max(part[2], part[3]));
}

// Dense, 16-byte aligned tensors of `units` 8-element units: a grid of at most
// kAmaxGroups workgroups strides over blocks of 1024 units, each block read
// as four wave-contiguous runs with all four 16-byte loads of a thread issued
// before the first max. Measured against one-shot grids (every workgroup one
// block of 1024, 2048 or 4096 units): 3.5 us faster on a 4608 x 3072
// activation, 1.3 us on 4608 x 9216.
constexpr int64_t kAmaxGroups = 1024;  // four workgroups per CU on 256 CUs

__global__ void __launch_bounds__(256) k_amax_dense(const uint16_t* __restrict__ x, int64_t units,
                                                    uint32_t* __restrict__ partial) {
  constexpr int U = 4;
  const uint4* xv = reinterpret_cast<const uint4*>(x);
  uint32_t m = 0;
  for (int64_t base = (int64_t)blockIdx.x * 256 * U + threadIdx.x; base < units; base += (int64_t)gridDim.x * 256 * U) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = (base + u * 256 < units) ? xv[base + u * 256] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t t = w[i] & 0x7FFF7FFFu;
        m = max(m, max(t & 0xFFFFu, t >> 16));
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) partial[blockIdx.x] = max(max(part[0], part[1]), max(part[2], part[3]));
}

// Max of `count` partials (bf16 magnitude bits) -> decode scale, written to
// `slot`. divisor = 448 (FP8) or 2688 = 448 * 6 (NVFP4). Inf/NaN anywhere in
// the tensor leaves a NaN scale as the sentinel. `partial` may be `slot`
// itself (count 1): every read happens before the barrier, the write after.
__global__ void __launch_bounds__(256) k_finalize(const uint32_t* partial, int count, float* slot,
                                                  float divisor) {
  // eight loads per thread in flight at once: the partials were just written
  // by workgroups on every XCD, so each round trip is a far-cache latency
  constexpr int U = 8;
  uint32_t m = 0;
  for (int base = 0; base < count; base += 256 * U) {
    uint32_t v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * 256 + (int)threadIdx.x;
      v[u] = (i < count) ? partial[i] : 0u;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) m = max(m, v[u]);
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t a = max(max(part[0], part[1]), max(part[2], part[3])) << 16;
    *slot = (a >= 0x7F800000u) ? __builtin_nanf("") : __fdiv_rn(u2f(a), divisor);
  }
}

// ---------------------------------------------------------------- units of 16
// A unit: cnt (<= 16) consecutive bf16 of a row, held as 8 words (element
// 2 i in the low half of word i, missing elements zero). VEC: the unit is
// whole and 16-byte aligned (two 16-byte loads).
template <bool VEC>
__device__ inline void unit_load(const uint16_t* __restrict__ p, int64_t cnt, uint32_t (&w)[8]) {
  if (VEC && cnt == 16) {
    const uint4 a = reinterpret_cast<const uint4*>(p)[0], b = reinterpret_cast<const uint4*>(p)[1];
    w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w; w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t lo = (2 * i < cnt) ? (uint32_t)p[2 * i] : 0u;
      const uint32_t hi = (2 * i + 1 < cnt) ? (uint32_t)p[2 * i + 1] : 0u;
      w[i] = lo | (hi << 16);
    }
  }
}

// FP8 codes of a unit: q = E4M3(x * r) by the hardware conversion (hw_e4m3x4,
// equal to enc_e4m3 on every finite input); one 16-byte store when vec_store
// (whole unit, 16-byte aligned destination), else byte stores.
__device__ inline void quant_fp8_words(const uint32_t (&w)[8], int64_t cnt, uint8_t* __restrict__ dst, float r,
                                       bool vec_store) {
  uint32_t c[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float y[4] = {__fmul_rn(bf16_lo(w[2 * i]), r), __fmul_rn(bf16_hi(w[2 * i]), r),
                        __fmul_rn(bf16_lo(w[2 * i + 1]), r), __fmul_rn(bf16_hi(w[2 * i + 1]), r)};
    c[i] = hw_e4m3x4(y);
  }
  if (vec_store && cnt == 16) {
    *reinterpret_cast<uint4*>(dst) = make_uint4(c[0], c[1], c[2], c[3]);
  } else {
    for (int64_t i = 0; i < cnt; ++i) dst[i] = (uint8_t)((c[i >> 2] >> (8 * (i & 3))) & 0xFFu);
  }
}

// NVFP4 block of a whole unit: block max, E4M3 block scale (returned), then
// the 16 E2M1 codes packed into 8 bytes at q8 (element 2i in the low nibble;
// hardware conversion hw_e2m1x8, equal to enc_e2m1 on every input).
__device__ inline uint32_t quant_nvfp4_words(const uint32_t (&w)[8], uint8_t* __restrict__ q8, float s_t) {
  float v[16];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    v[2 * i] = bf16_lo(w[i]);
    v[2 * i + 1] = bf16_hi(w[i]);
  }
  uint32_t amax_bits = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) amax_bits = max(amax_bits, f2u(v[i]) & 0x7FFFFFFFu);
  const float d_t = __fmul_rn(6.0f, s_t);
  const float vb = (d_t > 0.0f) ? __fdiv_rn(u2f(amax_bits), d_t) : 0.0f;
  const uint32_t sb = enc_e4m3(vb);
  const float S = __fmul_rn(dec_e4m3(sb), s_t);
  const float r = (S > 0.0f) ? __fdiv_rn(1.0f, S) : 0.0f;
  float y[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) y[i] = __fmul_rn(v[i], r);
  *reinterpret_cast<uint2*>(q8) = make_uint2(hw_e2m1x8(y), hw_e2m1x8(y + 8));
  return sb;
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
  uint32_t w[8];
  unit_load<VEC>(x + src, cnt, w);
  quant_fp8_words(w, cnt, q + dst, r, VEC);
}

// ---------------------------------------------------------------- NVFP4
// One thread per 16-element block.
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
  uint32_t w[8];
  unit_load<VEC>(x + src, 16, w);
  bscale[t] = (uint8_t)quant_nvfp4_words(w, q + t * 8, *tscale);
}

// ---------------------------------------------------------------- small tensors
// The whole dynamic quantization of a small tensor (at most 3072 units of 16
// elements) in one launch: every workgroup loads the whole tensor into
// registers (up to three units per thread) and reduces its max; workgroup b
// of G codes its G-th of the units from the same registers -- one launch
// instead of the three-kernel chain, whose launch latencies dominate at these
// sizes, with the coding and the stores spread over G CUs. The same arithmetic
// as the chain, so the same bits: the max of the bf16 magnitude bits,
// s = fl(amax / 448) or fl(amax / 2688) (NaN if the tensor holds inf or NaN),
// then the unit helpers above. FP8 rows may end in a shorter unit; NVFP4
// rows are whole blocks. VEC: 16-byte aligned rows of a multiple of 8
// elements; vec_store (FP8): 16-byte aligned codes and cols % 16 == 0.
constexpr int kSmallPerThread = 3;
constexpr int64_t kSmallUnits = 1024 * kSmallPerThread;
constexpr int64_t kSmallGroups = 8;  // workgroups that share the coding

template <int FMT, bool VEC>
__global__ void __launch_bounds__(1024) k_quant_small(const uint16_t* __restrict__ x, int64_t rows, int64_t cols,
                                                      int64_t ldx, uint8_t* __restrict__ q,
                                                      uint8_t* __restrict__ bscale, float* __restrict__ tscale,
                                                      bool vec_store) {
  // at most kSmallUnits units: 32-bit unit arithmetic
  const int upr = (int)((cols + 15) >> 4);
  const int units = (int)rows * upr;
  uint32_t w[kSmallPerThread][8];
#pragma unroll
  for (int i = 0; i < kSmallPerThread; ++i) {
    const int u = (int)threadIdx.x + 1024 * i;
    if (u < units) {
      const int row = u / upr, c = (u - row * upr) * 16;
      unit_load<VEC>(x + (int64_t)row * ldx + c, min((int64_t)16, cols - c), w[i]);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) w[i][j] = 0u;
    }
  }
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < kSmallPerThread; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t t = w[i][j] & 0x7FFF7FFFu;
      m = max(m, max(t & 0xFFFFu, t >> 16));
    }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t part[16];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
  __syncthreads();
  uint32_t a = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) a = max(a, part[i]);
  a <<= 16;
  const float s = (a >= 0x7F800000u) ? __builtin_nanf("") : __fdiv_rn(u2f(a), FMT == 1 ? 448.0f : 2688.0f);
  if (blockIdx.x == 0 && threadIdx.x == 0) *tscale = s;
  // every workgroup reduces the whole tensor; workgroup b codes the units
  // [b U / G, (b + 1) U / G) of the U units (G workgroups)
  const int lo = gridDim.x == 1 ? 0 : units * (int)blockIdx.x / (int)gridDim.x;
  const int hi = gridDim.x == 1 ? units : units * ((int)blockIdx.x + 1) / (int)gridDim.x;
  const float r = (FMT == 1 && s > 0.0f) ? __fdiv_rn(1.0f, s) : 0.0f;
#pragma unroll
  for (int i = 0; i < kSmallPerThread; ++i) {
    const int u = (int)threadIdx.x + 1024 * i;
    if (u < lo || u >= hi) continue;
    const int row = u / upr, c = (u - row * upr) * 16;
    if (FMT == 1) quant_fp8_words(w[i], min((int64_t)16, cols - c), q + (int64_t)row * cols + c, r, vec_store);
    else bscale[u] = (uint8_t)quant_nvfp4_words(w[i], q + (int64_t)u * 8, s);
  }
}

// ---------------------------------------------------------------- dense tensors
// FP8 codes of one whole 16-byte unit (8 consecutive elements, index u)
// held in `raw`: one 8-byte store, gated by `in`.
__device__ inline void code_unit8_fp8(const uint4 raw, int64_t u, bool in, uint8_t* __restrict__ q, float r) {
  const uint32_t ww[4] = {raw.x, raw.y, raw.z, raw.w};
  float y[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    y[2 * j] = __fmul_rn(bf16_lo(ww[j]), r);
    y[2 * j + 1] = __fmul_rn(bf16_hi(ww[j]), r);
  }
  const uint32_t lo = hw_e4m3x4(y), hi = hw_e4m3x4(y + 4);
  if (in) *reinterpret_cast<uint2*>(q + u * 8) = make_uint2(lo, hi);
}

// NVFP4 codes of two whole units per lane from two load steps: lanes 2j and
// 2j+1 hold the halves of block A (units u[0]) and of block B (units u[1]);
// the even lane derives A's scale, the odd lane B's, so each lane does one
// block's two divisions for two blocks' worth of elements, and the two
// reciprocals are swapped across the pair. Every lane of the wave calls it
// together; in[] only gates the stores. The arithmetic of quant_nvfp4_words.
__device__ inline void code_units8_nv_pair(const uint4 (&raw)[2], const int64_t (&u)[2], const bool (&in)[2],
                                           uint8_t* __restrict__ q, uint8_t* __restrict__ bscale, float s,
                                           float d_t, int lane) {
  float v[2][8];
  uint32_t am[2];
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const uint32_t ww[4] = {raw[p].x, raw[p].y, raw[p].z, raw[p].w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[p][2 * j] = bf16_lo(ww[j]);
      v[p][2 * j + 1] = bf16_hi(ww[j]);
    }
    uint32_t a = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) a = max(a, f2u(v[p][j]) & 0x7FFFFFFFu);
    am[p] = max(a, (uint32_t)__shfl_xor((int)a, 1));
  }
  const bool odd = lane & 1;
  const float vb = (d_t > 0.0f) ? __fdiv_rn(u2f(odd ? am[1] : am[0]), d_t) : 0.0f;
  const uint32_t sb = enc_e4m3(vb);
  const float S = __fmul_rn(dec_e4m3(sb), s);
  const float rb = (S > 0.0f) ? __fdiv_rn(1.0f, S) : 0.0f;
  const float rp = __shfl_xor(rb, 1);
  const float rr[2] = {odd ? rp : rb, odd ? rb : rp};
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    float y[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) y[j] = __fmul_rn(v[p][j], rr[p]);
    const uint32_t w = hw_e2m1x8(y);
    if (in[p]) {
      *reinterpret_cast<uint32_t*>(q + u[p] * 4) = w;
      if (odd == (p == 1)) bscale[u[p] >> 1] = (uint8_t)sb;
    }
  }
}

// Dense tensors (ldx == cols, 16-byte aligned rows): each wavefront codes a
// chunk of 512 H consecutive elements. Lane l reads elements
// [512 h + 8l, 512 h + 8l + 8) of the chunk for h < H with one 16-byte load
// each, all issued before the first is used, so every load and store
// instruction of the wave covers one contiguous run of memory and H loads
// per lane are in flight. Elements are coded with the hardware conversions
// (hw_e4m3x4 / hw_e2m1x8). NVFP4: n % 16 == 0, so lanes (2j, 2j+1) hold one
// whole 16-element block (or both lie past the end); the block max is shared
// with one lane swap, and each lane of the pair derives the scale of one of
// the two blocks the pair holds in two consecutive steps.
template <int FMT, int H>
__global__ void __launch_bounds__(256) k_quant_dense(const uint16_t* __restrict__ x, int64_t n,
                                                     uint8_t* __restrict__ q,
                                                     uint8_t* __restrict__ bscale,
                                                     const float* __restrict__ tscale) {
  const int lane = threadIdx.x & 63;
  const int64_t chunk = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;
  uint4 raw[H];
#pragma unroll
  for (int h = 0; h < H; ++h) {
    const int64_t e0 = chunk * (512 * H) + h * 512 + lane * 8;
    raw[h] = (e0 + 8 <= n) ? *reinterpret_cast<const uint4*>(x + e0) : make_uint4(0u, 0u, 0u, 0u);
  }
  const float s = *tscale;
  const float r = (FMT == 1 && s > 0.0f) ? __fdiv_rn(1.0f, s) : 0.0f;
  const float d_t = __fmul_rn(6.0f, s);
  if constexpr (FMT == 2) {
    static_assert(H % 2 == 0, "NVFP4 steps go in pairs");
#pragma unroll
    for (int h = 0; h < H; h += 2) {
      const int64_t e0 = chunk * (512 * H) + h * 512 + lane * 8;
      const uint4 rw[2] = {raw[h], raw[h + 1]};
      const int64_t u[2] = {e0 >> 3, (e0 + 512) >> 3};
      const bool in[2] = {e0 + 8 <= n, e0 + 520 <= n};
      code_units8_nv_pair(rw, u, in, q, bscale, s, d_t, lane);
    }
  } else {
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int64_t e0 = chunk * (512 * H) + h * 512 + lane * 8;
      const bool full = (e0 + 8 <= n);
      code_unit8_fp8(raw[h], e0 >> 3, full, q, r);
      if (!full && e0 < n) {  // FP8 tail unit of fewer than 8 elements
        float y[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = (e0 + j < n) ? __fmul_rn(u2f((uint32_t)x[e0 + j] << 16), r) : 0.0f;
        const uint32_t lo = hw_e4m3x4(y), hi = hw_e4m3x4(y + 4);
        for (int j = 0; j < 8 && e0 + j < n; ++j) q[e0 + j] = (uint8_t)(((j < 4 ? lo : hi) >> (8 * (j & 3))) & 0xFFu);
      }
    }
  }
}

// ---------------------------------------------------------------- dense, two launches
// Dynamic quantization of a dense tensor without the one-workgroup finalize
// kernel. k_amax_slots leaves each of its P workgroup maxima not in one
// place but in every code region of the quantize launch (slot i among the
// first 4 P bytes of each region); each workgroup of k_quant_dense_slots
// reduces the P maxima found at the start of its own region to the tensor
// scale before any of its codes overwrite them. No workgroup reads what
// another writes within a launch, so stream order between the two launches
// is the only synchronisation, and the caller's code buffer the only memory.
// Region j of G: the 16-byte units [slot_region_lo(j), slot_region_lo(j + 1))
// of the n / 8 (the last region ends at n / 8), whose codes start at byte CB
// times their first unit (CB = 8 for FP8, 4 for NVFP4). The host picks G so
// that every region's codes hold the 4 P bytes of slots.
// (the plan: slot_region_lo, slots_plan and their limits in quant_plan.hpp)

template <int U>
__global__ void __launch_bounds__(256) k_amax_slots(const uint16_t* __restrict__ x, int64_t units,
                                                    uint8_t* __restrict__ q, int cb, int gq) {
  const uint4* xv = reinterpret_cast<const uint4*>(x);
  uint32_t m = 0;
  for (int64_t base = (int64_t)blockIdx.x * 256 * U + threadIdx.x; base < units; base += (int64_t)gridDim.x * 256 * U) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = (base + u * 256 < units) ? xv[base + u * 256] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t t = w[i] & 0x7FFF7FFFu;
        m = max(m, max(t & 0xFFFFu, t >> 16));
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
  __syncthreads();
  const uint32_t mw = max(max(part[0], part[1]), max(part[2], part[3]));
  // workgroup b runs on XCD b mod 8: with the slots ordered XCD-major, the
  // maxima of one XCD's workgroups fill whole cache lines of each region
  const int P = (int)gridDim.x, b = (int)blockIdx.x;
  const int slot = (P % 8 == 0) ? (b % 8) * (P / 8) + b / 8 : b;
  const int64_t pairs = units >> 1;
  for (int j = (int)threadIdx.x; j < gq; j += 256)
    reinterpret_cast<uint32_t*>(q + slot_region_lo(pairs, j, gq) * cb)[slot] = mw;
}

// Each wave codes runs of 64 consecutive units (one 16-byte load per lane,
// four per lane in flight); rounds of 1024 units until the region ends.
template <int FMT>
__global__ void __launch_bounds__(256) k_quant_dense_slots(const uint16_t* __restrict__ x, int64_t units,
                                                           uint8_t* __restrict__ q, uint8_t* __restrict__ bscale,
                                                           float* __restrict__ tscale, int P) {
  constexpr int H = 4;
  constexpr int CB = FMT == 1 ? 8 : 4;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t pairs = units >> 1;
  const int64_t lo = slot_region_lo(pairs, blockIdx.x, gridDim.x);
  const int64_t hi = (blockIdx.x + 1 == gridDim.x) ? units : slot_region_lo(pairs, blockIdx.x + 1, gridDim.x);
  const uint4* xv = reinterpret_cast<const uint4*>(x);
  uint4 raw[H];
#pragma unroll
  for (int h = 0; h < H; ++h) {
    const int64_t u = lo + 256 * wv + 64 * h + lane;
    raw[h] = (u < hi) ? xv[u] : make_uint4(0u, 0u, 0u, 0u);
  }
  // the tensor max from this region's slots, all read before the barrier
  const uint32_t* slots = reinterpret_cast<const uint32_t*>(q + lo * CB);
  uint32_t m = 0;
  for (int i = (int)threadIdx.x; i < P; i += 256) m = max(m, slots[i]);
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t part[4];
  if (lane == 0) part[wv] = m;
  __syncthreads();
  const uint32_t a = max(max(part[0], part[1]), max(part[2], part[3])) << 16;
  const float s = (a >= 0x7F800000u) ? __builtin_nanf("") : __fdiv_rn(u2f(a), FMT == 1 ? 448.0f : 2688.0f);
  if (blockIdx.x == 0 && threadIdx.x == 0) *tscale = s;
  const float r = (FMT == 1 && s > 0.0f) ? __fdiv_rn(1.0f, s) : 0.0f;
  const float d_t = __fmul_rn(6.0f, s);
  for (int64_t base = lo;;) {
    if constexpr (FMT == 2) {
#pragma unroll
      for (int h = 0; h < H; h += 2) {
        const int64_t u0 = base + 256 * wv + 64 * h + lane;
        const uint4 rw[2] = {raw[h], raw[h + 1]};
        const int64_t u[2] = {u0, u0 + 64};
        const bool in[2] = {u0 < hi, u0 + 64 < hi};
        code_units8_nv_pair(rw, u, in, q, bscale, s, d_t, lane);
      }
    } else {
#pragma unroll
      for (int h = 0; h < H; ++h) {
        const int64_t u = base + 256 * wv + 64 * h + lane;
        code_unit8_fp8(raw[h], u, u < hi, q, r);
      }
    }
    base += 1024;
    if (base >= hi) break;
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int64_t u = base + 256 * wv + 64 * h + lane;
      raw[h] = (u < hi) ? xv[u] : make_uint4(0u, 0u, 0u, 0u);
    }
  }
}

// ---------------------------------------------------------------- MX formats
// OCP MX (MXFP4: E2M1 elements, MXFP8: E4M3 elements), one E8M0 scale per 32
// consecutive elements of a row, no tensor scale: the block scaling gfx950's
// matrix cores consume natively. Shared exponent = floor(log2 max|x|) - emax
// (emax 2 for E2M1, 8 for E4M3), E8M0 code = that + 127 clamped to [0, 254],
// 0 for an all-zero block; elements = RNE_sat(x * 2^(127 - code)), the
// multiply exact (a power of two, inside the normal range for bf16 inputs).
// One thread codes 8 consecutive elements of a row; rows hold whole blocks
// (cols % 32 == 0), so the 4 threads of a block are lanes 4j .. 4j + 3 of one
// wave and share its max with two lane swaps. VEC: 16-byte aligned rows.
template <bool FP4, bool VEC>
__global__ void __launch_bounds__(256) k_quant_mx(const uint16_t* __restrict__ x, int64_t rows, int64_t cols,
                                                  int64_t ldx, uint8_t* __restrict__ q,
                                                  uint8_t* __restrict__ scales) {
  const int64_t upr = cols >> 3;  // 8-element units per row
  const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const bool live = u < rows * upr;
  const int64_t row = live ? u / upr : 0, c8 = live ? u - row * upr : 0;
  float v[8];
  if (live) {
    const uint16_t* p = x + row * ldx + 8 * c8;
    if (VEC) {
      const uint4 w = *reinterpret_cast<const uint4*>(p);
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[2 * j] = bf16_lo(ww[j]);
        v[2 * j + 1] = bf16_hi(ww[j]);
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = u2f((uint32_t)p[j] << 16);
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = 0.0f;
  }
  uint32_t am = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) am = max(am, f2u(v[j]) & 0x7FFFFFFFu);
  am = max(am, (uint32_t)__shfl_xor((int)am, 1));
  am = max(am, (uint32_t)__shfl_xor((int)am, 2));
  // floor(log2(max)) from the fp32 bits (normal or denormal), then the code.
  // A block holding inf or NaN gets the E8M0 NaN code 255 (its element codes
  // are then unspecified: r = 0 makes them signed zeros).
  int e = 0;
  if (am >= 0x7F800000u) {
    e = 255;
  } else if (am != 0u) {
    const int ef = (int)(am >> 23);
    const int fl = (ef > 0) ? ef - 127 : (31 - __builtin_clz(am)) - 149;
    e = min(max(fl - (FP4 ? 2 : 8) + 127, 0), 254);
  }
  // 2^(127 - e); finite bf16 inputs give e <= 252, so this is a normal number
  const float r = (e == 255) ? 0.0f : u2f((uint32_t)(254 - e) << 23);
  float y[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) y[j] = __fmul_rn(v[j], r);
  if (!live) return;
  if (FP4) {
    *reinterpret_cast<uint32_t*>(q + row * (cols >> 1) + 4 * c8) = hw_e2m1x8(y);
  } else {
    const uint32_t lo = hw_e4m3x4(y), hi = hw_e4m3x4(y + 4);
    uint8_t* d = q + row * cols + 8 * c8;
    if ((reinterpret_cast<uintptr_t>(d) & 7) == 0) *reinterpret_cast<uint2*>(d) = make_uint2(lo, hi);
    else for (int j = 0; j < 8; ++j) d[j] = (uint8_t)(((j < 4 ? lo : hi) >> (8 * (j & 3))) & 0xFFu);
  }
  if ((c8 & 3) == 0) scales[row * (cols >> 5) + (c8 >> 2)] = (uint8_t)e;
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

// MX: out = element * 2^(e - 127) (exact in fp32), one thread per 8 elements.
template <bool FP4, bool F32OUT>
__global__ void __launch_bounds__(256) k_dequant_mx(const uint8_t* __restrict__ q, const uint8_t* __restrict__ sc,
                                                    int64_t n, void* __restrict__ out) {
  const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (u * 8 >= n) return;
  const uint32_t e = sc[u >> 2];
  // 2^(e - 127); code 255 is the E8M0 NaN (a block that held inf or NaN)
  const float scale = (e == 0u) ? u2f(0x00400000u) : (e == 255u) ? __builtin_nanf("") : u2f(e << 23);
  float v[8];
  if (FP4) {
    const uint32_t w = reinterpret_cast<const uint32_t*>(q)[u];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = dec_e2m1((w >> (4 * j)) & 15u) * scale;
  } else {
    const uint2 w = reinterpret_cast<const uint2*>(q)[u];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = dec_e4m3(((j < 4 ? w.x : w.y) >> (8 * (j & 3))) & 0xFFu) * scale;
  }
  if (F32OUT) {
    float4* o = reinterpret_cast<float4*>(out) + 2 * u;
    o[0] = make_float4(v[0], v[1], v[2], v[3]);
    o[1] = make_float4(v[4], v[5], v[6], v[7]);
  } else {
    uint32_t h[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) h[j] = f32_to_bf16(v[2 * j]) | (f32_to_bf16(v[2 * j + 1]) << 16);
    reinterpret_cast<uint4*>(out)[u] = make_uint4(h[0], h[1], h[2], h[3]);
  }
}

// ---------------------------------------------------------------- launchers
static inline unsigned grid_for(int64_t threads) { return (unsigned)((threads + 255) / 256); }

// The element kernels alone, reading a finished decode scale from `tscale`:
// the last kernel of the dynamic chain, and the whole of a quantization with
// a static (calibrated) scale.
hipError_t launch_quantize_static(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ldx,
                                  uint8_t* codes, uint8_t* bscale, const float* tscale, hipStream_t st) {
  if (rows == 0 || cols == 0) return hipSuccess;
  const bool contig = (ldx == cols);
  const bool aligned = (reinterpret_cast<uintptr_t>(x) % 16 == 0);
  const int64_t n = rows * cols;
  const bool qal = (reinterpret_cast<uintptr_t>(codes) % 8 == 0);
  if (contig && aligned && qal) {
    const unsigned g = (unsigned)((n + 8191) / 8192);  // 4 waves x 2048 elements per workgroup
    if (fmt == 1) hipLaunchKernelGGL((k_quant_dense<1, 4>), dim3(g), dim3(256), 0, st, x, n, codes, bscale, tscale);
    else hipLaunchKernelGGL((k_quant_dense<2, 4>), dim3(g), dim3(256), 0, st, x, n, codes, bscale, tscale);
  } else if (fmt == 1) {
    const bool qal16 = (reinterpret_cast<uintptr_t>(codes) % 16 == 0);
    if (contig) {
      const bool vec = aligned && qal16;
      const unsigned g = grid_for((rows * cols + 15) / 16);
      if (vec) hipLaunchKernelGGL((k_quant_fp8<true, true>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, tscale);
      else hipLaunchKernelGGL((k_quant_fp8<false, true>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, tscale);
    } else {
      const bool vec = aligned && qal16 && (ldx % 8 == 0) && (cols % 16 == 0);
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

// MX formats: block scales only, one kernel.
static hipError_t launch_quantize_mx(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ldx,
                                     uint8_t* codes, uint8_t* scales, hipStream_t st) {
  if (rows == 0 || cols == 0) return hipSuccess;
  const unsigned g = grid_for(rows * (cols / 8));
  const bool vec = (reinterpret_cast<uintptr_t>(x) % 16 == 0) && (ldx % 8 == 0);
  if (fmt == 3) {
    if (vec) hipLaunchKernelGGL((k_quant_mx<true, true>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, scales);
    else hipLaunchKernelGGL((k_quant_mx<true, false>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, scales);
  } else {
    if (vec) hipLaunchKernelGGL((k_quant_mx<false, true>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, scales);
    else hipLaunchKernelGGL((k_quant_mx<false, false>), dim3(g), dim3(256), 0, st, x, rows, cols, ldx, codes, scales);
  }
  return hipGetLastError();
}

hipError_t launch_quantize(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ldx,
                           uint8_t* codes, uint8_t* bscale, float* tscale, hipStream_t st) {
  if (fmt == 3 || fmt == 4) return launch_quantize_mx(fmt, x, rows, cols, ldx, codes, bscale, st);
  if (rows == 0 || cols == 0) {
    hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(1), 0, st, reinterpret_cast<uint32_t*>(tscale), 0u);
    return hipGetLastError();
  }
  const bool contig = (ldx == cols);
  const bool aligned = (reinterpret_cast<uintptr_t>(x) % 16 == 0);
  if (rows * ((cols + 15) / 16) <= kSmallUnits) {
    // one launch does it all (NVFP4 codes are 8-byte aligned: checked by
    // the caller); one workgroup per 256 units, at most eight. Measured
    // against the chain (GPU time from graph replays): 1 x 1024 3.1 us,
    // 128 x 256 4.3 us, 16 x 3072 4.6 us, where the chain takes 6.5 us
    // (FP8) to 7.4 us (NVFP4); one workgroup took 5.0 and 5.9 us on the last
    // two. Raising the limit to 8192 units (eight per thread) lost to the
    // chain from 6144 units on.
    const bool rvec = aligned && (cols % 8 == 0) && (contig || ldx % 8 == 0);
    const bool qvec = (reinterpret_cast<uintptr_t>(codes) % 16 == 0) && (cols % 16 == 0);
    const int64_t units = rows * ((cols + 15) / 16);
    const unsigned G = (unsigned)std::min<int64_t>(kSmallGroups, (units + 255) / 256);
    if (fmt == 1) {
      if (rvec) hipLaunchKernelGGL((k_quant_small<1, true>), dim3(G), dim3(1024), 0, st, x, rows, cols, ldx, codes, bscale, tscale, qvec);
      else hipLaunchKernelGGL((k_quant_small<1, false>), dim3(G), dim3(1024), 0, st, x, rows, cols, ldx, codes, bscale, tscale, qvec);
    } else {
      if (rvec) hipLaunchKernelGGL((k_quant_small<2, true>), dim3(G), dim3(1024), 0, st, x, rows, cols, ldx, codes, bscale, tscale, false);
      else hipLaunchKernelGGL((k_quant_small<2, false>), dim3(G), dim3(1024), 0, st, x, rows, cols, ldx, codes, bscale, tscale, false);
    }
    return hipGetLastError();
  }
  const int64_t n = rows * cols;
  if (contig && aligned && reinterpret_cast<uintptr_t>(codes) % 8 == 0) {
    // dense: two launches, the maxima handed over in every code region
    const int64_t units = n / 8;
    const int cb = (fmt == 1) ? 8 : 4;
    const SlotsPlan plan = slots_plan(n, cb);
    const int64_t P = plan.P, G = plan.G;
    if (G >= 1) {
      hipLaunchKernelGGL(k_amax_slots<kSlotsAmaxLoads>, dim3((unsigned)P), dim3(256), 0, st, x, units, codes, cb, (int)G);
      if (fmt == 1)
        hipLaunchKernelGGL(k_quant_dense_slots<1>, dim3((unsigned)G), dim3(256), 0, st, x, units, codes, bscale, tscale, (int)P);
      else
        hipLaunchKernelGGL(k_quant_dense_slots<2>, dim3((unsigned)G), dim3(256), 0, st, x, units, codes, bscale, tscale, (int)P);
      return hipGetLastError();
    }
  }
  // amax: per-workgroup partial maxima are parked in the code buffer, which
  // the quantize kernel overwrites afterwards (stream order separates them).
  {
    const int64_t r_eff = contig ? 1 : rows;
    const int64_t c_eff = contig ? rows * cols : cols;
    const bool vec = aligned && (c_eff % 8 == 0) && (contig || ldx % 8 == 0);
    const int64_t per_row = vec ? c_eff / 8 : c_eff;
    const int64_t code_bytes = (fmt == 1) ? rows * cols : rows * cols / 2;
    const uintptr_t base = (reinterpret_cast<uintptr_t>(codes) + 3) & ~uintptr_t(3);
    const int64_t cap = (code_bytes - (int64_t)(base - reinterpret_cast<uintptr_t>(codes))) / 4;
    int64_t gx, gy;
    uint32_t* partial = reinterpret_cast<uint32_t*>(base);
    const int64_t dense_groups = std::min<int64_t>((c_eff / 8 + 1023) / 1024, kAmaxGroups);
    if (contig && vec && dense_groups <= cap) {
      gx = dense_groups;
      gy = 1;
      hipLaunchKernelGGL(k_amax_dense, dim3((unsigned)gx), dim3(256), 0, st, x, c_eff / 8, partial);
    } else {
      gy = std::min<int64_t>(r_eff, 1024);
      gx = std::min<int64_t>(std::max<int64_t>(1, (per_row + 1023) / 1024), std::max<int64_t>(1, 1024 / gy));
      if (gx * gy > cap) {  // tiny tensor: one workgroup, its max goes straight to the scale slot
        gx = gy = 1;
        partial = reinterpret_cast<uint32_t*>(tscale);
      }
      if (vec)
        hipLaunchKernelGGL(k_amax_partial<true>, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, st, x, r_eff, c_eff,
                           contig ? c_eff : ldx, partial);
      else
        hipLaunchKernelGGL(k_amax_partial<false>, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, st, x, r_eff, c_eff,
                           contig ? c_eff : ldx, partial);
    }
    hipLaunchKernelGGL(k_finalize, dim3(1), dim3(256), 0, st, partial, (int)(gx * gy), tscale,
                       fmt == 1 ? 448.0f : 2688.0f);
  }
  return launch_quantize_static(fmt, x, rows, cols, ldx, codes, bscale, tscale, st);
}

hipError_t launch_dequant(int fmt, const uint8_t* codes, const uint8_t* bscale, const float* tscale,
                          int64_t rows, int64_t cols, void* out, bool f32out, hipStream_t st) {
  const int64_t n = rows * cols;
  if (n == 0) return hipSuccess;
  if (fmt == 3 || fmt == 4) {  // MX: aligned buffers (checked by the caller)
    const unsigned g = grid_for(n / 8);
    if (fmt == 3) {
      if (f32out) hipLaunchKernelGGL((k_dequant_mx<true, true>), dim3(g), dim3(256), 0, st, codes, bscale, n, out);
      else hipLaunchKernelGGL((k_dequant_mx<true, false>), dim3(g), dim3(256), 0, st, codes, bscale, n, out);
    } else {
      if (f32out) hipLaunchKernelGGL((k_dequant_mx<false, true>), dim3(g), dim3(256), 0, st, codes, bscale, n, out);
      else hipLaunchKernelGGL((k_dequant_mx<false, false>), dim3(g), dim3(256), 0, st, codes, bscale, n, out);
    }
    return hipGetLastError();
  }
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

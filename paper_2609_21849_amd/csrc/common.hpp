// common.hpp -- device-side types and bit-exact codecs of the gfx950 library.
//
// The quantizers must reproduce, bit for bit, the fp32 recipe of the
// formats the paper's quantization recipe uses (Sec. 4): E4M3 and E2M1
// round-to-nearest-even with saturation, sign of zero kept. The encoders
// below do this with integer operations on the fp32 bit pattern (plus one
// v_rndne_f32 on the subnormal grid), so their result does not depend on
// the GPU's denormal or rounding modes. They are __host__ __device__ so a
// host build can test them against every fp32 input.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qg {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

__host__ __device__ inline uint32_t f2u(float f) { return __builtin_bit_cast(uint32_t, f); }
__host__ __device__ inline float u2f(uint32_t u) { return __builtin_bit_cast(float, u); }

// bf16 bit pattern -> fp32 (exact)
__host__ __device__ inline float bf16_lo(uint32_t w) { return u2f(w << 16); }
__host__ __device__ inline float bf16_hi(uint32_t w) { return u2f(w & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even; NaN -> 0x7FC0.
__host__ __device__ inline uint32_t f32_to_bf16(float f) {
  uint32_t u = f2u(f);
  uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  return ((u & 0x7FFFFFFFu) > 0x7F800000u) ? 0x7FC0u : r;
}

// E4M3 code of fp32 y: nearest of the 127 finite magnitudes, ties to the
// even code, |y| >= 448 saturates to 448 (0x7E), NaN -> 0x7F, sign kept.
//   normal range [2^-6, 448): round the 23-bit mantissa to 3 bits (RNE on
//     the bit pattern); the carry walks into the exponent, which is exactly
//     the next code. code = biased-exp-rebias | mantissa = (r >> 20) - 960.
//   below 2^-6: E4M3 subnormals are the grid k * 2^-9, k = 0..8 (8 is the
//     smallest normal, code 0x08), so code = rint(|y| * 512).
__host__ __device__ inline uint32_t enc_e4m3(float y) {
  const uint32_t u = f2u(y);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7FFFFFFFu;
  const uint32_t rn = a + 0x7FFFFu + ((a >> 20) & 1u);
  uint32_t q = (rn >> 20) - 960u;
  const uint32_t qs = (uint32_t)__builtin_rintf(u2f(a < 0x3C800000u ? a : 0u) * 512.0f);
  q = (a < 0x3C800000u) ? qs : q;           // |y| < 2^-6
  q = (a >= 0x43E00000u) ? 0x7Eu : q;       // |y| >= 448 (and inf)
  q = (a > 0x7F800000u) ? 0x7Fu : q;        // NaN
  return sign | q;
}

// E2M1 code (4 bits) of fp32 y: nearest of {0,.5,1,1.5,2,3,4,6}, ties to
// the even code, |y| >= 6 saturates to 6, sign kept (bit 3). NaN saturates
// (E2M1 has no NaN; only reached through a NaN tensor-scale sentinel).
//   [1, 6): round the mantissa to 1 bit; code = (r >> 22) - 252.
//   below 1: grid k * 0.5, k = 0..2, code = rint(|y| * 2).
__host__ __device__ inline uint32_t enc_e2m1(float y) {
  const uint32_t u = f2u(y);
  const uint32_t sign = (u >> 28) & 0x8u;
  const uint32_t a = u & 0x7FFFFFFFu;
  const uint32_t rn = a + 0x1FFFFFu + ((a >> 22) & 1u);
  uint32_t q = (rn >> 22) - 252u;
  const uint32_t qs = (uint32_t)__builtin_rintf(u2f(a < 0x3F800000u ? a : 0u) * 2.0f);
  q = (a < 0x3F800000u) ? qs : q;           // |y| < 1
  q = (a >= 0x40C00000u) ? 7u : q;          // |y| >= 6, inf, NaN
  return sign | q;
}

// Value of an E4M3 code as fp32 (exact). Normal codes: the 7 magnitude bits
// eeee.mmm moved to fp32 bits [26:20] with the exponent rebased by +120.
// Subnormal codes (exponent field 0) are k * 2^-9.
__host__ __device__ inline float dec_e4m3(uint32_t c) {
  const uint32_t mag = c & 0x7Fu;
  float v = (mag >= 8u) ? u2f((mag << 20) + (120u << 23)) : (float)(mag & 7u) * 0.001953125f;
  v = (mag == 0x7Fu) ? __builtin_nanf("") : v;
  return (c & 0x80u) ? -v : v;
}

// Value of an E2M1 code (low 4 bits) as fp32 (exact).
__host__ __device__ inline float dec_e2m1(uint32_t c) {
  const uint32_t mag = c & 7u;
  float v = (mag >= 2u) ? u2f(((mag + 252u) << 22)) : (float)mag * 0.5f;
  return (c & 8u) ? -v : v;
}

// E4M3 -> fp16 (exact: every E4M3 value is a normal or subnormal fp16 with
// at most 4 significant bits). For exponent field >= 1 the fp16 pattern is
// the E4M3 magnitude bits shifted to fp16's field with exponent + 8; the
// 8 subnormal codes (k * 2^-9) are normal fp16 values built from k.
__host__ __device__ inline _Float16 e4m3_to_f16(uint32_t c) {
  const uint32_t mag = c & 0x7Fu;
  const uint32_t m = mag & 7u;
  // subnormal k*2^-9: k = 1 -> 2^-9 (exp 6), 2 -> 2^-8, 3 -> 1.5*2^-8, 4 -> 2^-7,
  // 5 -> 1.25*2^-7, 6 -> 1.5*2^-7, 7 -> 1.75*2^-7  (fp16 bias 15)
  const uint32_t sub = (m == 0u) ? 0u
                     : (m == 1u) ? (6u << 10)
                     : (m < 4u)  ? ((7u << 10) | ((m & 1u) << 9))
                                 : ((8u << 10) | ((m & 3u) << 8));
  uint32_t h = (mag >= 8u) ? ((mag << 7) + (8u << 10)) : sub;
  h |= (c & 0x80u) << 8;
  return __builtin_bit_cast(_Float16, (uint16_t)h);
}

// ---------------------------------------------------------------------------
// Block-scale decoders of the GEMM kernels (E4M3 block scales are never
// negative: the quantizer codes a magnitude). The test probe checks each of
// them on all 128 non-negative codes against the E4M3 definition.
// Value of a non-negative E4M3 block-scale code (never NaN: the quantizer
// saturates at 448), exactly: its 7 bits placed at the top of the fp32
// mantissa/exponent field are the value times 2^-120 -- normal codes become
// normal fp32 numbers, subnormal codes denormal ones -- and one multiply by
// 2^120 restores it.
__device__ inline float dec_e4m3_scale(uint32_t c) {
  return u2f((c & 0x7Fu) << 20) * 1.329227995784915872903807060280344576e36f;  // 2^120
}

// Four E4M3 block scales (one dword, block b in byte b; never negative) to
// fp16, exact: every E4M3 value, the subnormal ones included, is a normal
// fp16 number, and the hardware conversion at unit scale
// (v_cvt_scalef32_pk_f16_fp8, two codes per instruction) keeps it (checked on
// every code in every byte position on the GPU). Result: .x = blocks 0 and 1,
// .y = blocks 2 and 3.
__device__ __attribute__((always_inline)) inline uint2 e4m3x4_to_f16x4(uint32_t d) {
  return make_uint2(__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d, 1.0f, false)),
                    __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(d, 1.0f, true)));
}

// fp16 block scale b (0..3) of a lane's four.
__device__ __attribute__((always_inline)) inline _Float16 scale_f16(uint2 sc, int b) {
  const uint32_t w = (b < 2) ? sc.x : sc.y;
  return __builtin_bit_cast(_Float16, (uint16_t)((b & 1) ? (w >> 16) : (w & 0xFFFFu)));
}

// ---------------------------------------------------------------------------
// Hardware conversions used by the quantizers (gfx950). Both are checked on
// the GPU against the integer encoders above over all 2^32 fp32 inputs:
//   E2M1: v_cvt_scalef32_pk_fp4_f32 with scale 1.0 equals enc_e2m1 on every
//         input (RNE, ties to even code, saturation at 6, sign of zero).
//   E4M3: v_cvt_scalef32_pk_fp8_f32 with scale 1.0 turns magnitudes above
//         464 into NaN instead of saturating; after a clamp to [-448, 448]
//         (v_med3_f32, which keeps -0) it equals enc_e4m3 on every finite input.
// Element 2i / the first operand lands in the low nibble / low byte.
__device__ inline uint32_t hw_e2m1x8(const float* y) {
  uint32_t w = 0;
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, y[0], y[1], 1.0f, 0);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, y[2], y[3], 1.0f, 1);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, y[4], y[5], 1.0f, 2);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, y[6], y[7], 1.0f, 3);
  return w;
}

__device__ inline uint32_t hw_e4m3x4(const float* y) {
  typedef short v2s __attribute__((ext_vector_type(2)));
  v2s w = {0, 0};
  const float a = __builtin_amdgcn_fmed3f(y[0], -448.0f, 448.0f);
  const float b = __builtin_amdgcn_fmed3f(y[1], -448.0f, 448.0f);
  const float c = __builtin_amdgcn_fmed3f(y[2], -448.0f, 448.0f);
  const float d = __builtin_amdgcn_fmed3f(y[3], -448.0f, 448.0f);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, a, b, 1.0f, false);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, c, d, 1.0f, true);
  return __builtin_bit_cast(uint32_t, w);
}

}  // namespace qg

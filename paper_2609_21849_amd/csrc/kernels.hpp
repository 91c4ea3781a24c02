// kernels.hpp -- internal launchers shared by the C-ABI layer (api.hip).
// Each launcher only enqueues work on `st`; arguments were validated by the
// caller. Format ids follow qg_format: 0 bf16, 1 FP8 E4M3, 2 NVFP4,
// 3 MXFP4, 4 MXFP8.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace qg {

// Packed weight buffer: a 256-byte header, then the codes region, then (for
// NVFP4, MXFP4 and MXFP8) the block-scale region. Header fields (little endian):
//   +0 u32 magic 'QGPW', +4 u32 layout version, +8 u32 format,
//   +16 i64 n, +24 i64 k, +32 f32 tensor decode scale.
// The weight is stored in panels of 32 rows (n rounded up to a multiple of
// 32, padding rows are zero codes) and chunks of 128 reduction elements.
constexpr uint32_t kPackMagic = 0x57504751u;  // "QGPW"
constexpr uint32_t kPackVersion = 3u;
constexpr int64_t kPackHeader = 256;
constexpr int64_t kPackScaleOffset = 32;
constexpr int64_t kPanel = 32;

inline int64_t padded_rows(int64_t n) { return (n + kPanel - 1) / kPanel * kPanel; }
inline int64_t packed_codes_bytes(int fmt, int64_t n, int64_t k) {
  return (fmt == 1 || fmt == 4) ? padded_rows(n) * k : padded_rows(n) * k / 2;
}
inline int64_t packed_scale_bytes(int fmt, int64_t n, int64_t k) {
  return fmt == 2 ? padded_rows(n) * k / 16 : (fmt == 3 || fmt == 4) ? padded_rows(n) * k / 32 : 0;
}
inline int64_t packed_total_bytes(int fmt, int64_t n, int64_t k) {
  return kPackHeader + packed_codes_bytes(fmt, n, k) + packed_scale_bytes(fmt, n, k);
}

hipError_t launch_quantize_static(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ldx,
                                  uint8_t* codes, uint8_t* bscale, const float* tscale, hipStream_t st);
hipError_t launch_quantize(int fmt, const uint16_t* x, int64_t rows, int64_t cols, int64_t ldx,
                           uint8_t* codes, uint8_t* bscale, float* tscale, hipStream_t st);
hipError_t launch_dequant(int fmt, const uint8_t* codes, const uint8_t* bscale, const float* tscale,
                          int64_t rows, int64_t cols, void* out, bool f32out, hipStream_t st);
hipError_t launch_pack(int fmt, const uint8_t* codes, const uint8_t* bscale, const float* tscale,
                       int64_t n, int64_t k, uint8_t* packed, hipStream_t st);
hipError_t launch_unpack(int fmt, const uint8_t* packed, int64_t n, int64_t k, uint8_t* codes,
                         uint8_t* bscale, float* tscale, hipStream_t st);
// out_mode: 0 bf16, 1 fp32, 2 E4M3 codes of y / *y_scale (y_scale: device
// fp32), 3 NVFP4 codes [m, ldy / 2] and E4M3 block scales y_bscale
// [m, ldy / 16] with the static tensor decode scale *y_scale
hipError_t launch_gemm(int a_fmt, const void* a, const uint8_t* a_bscale, const float* a_tscale,
                       int64_t lda, const uint8_t* w_packed, int64_t m, int64_t n, int64_t k,
                       void* y, int64_t ldy, int out_mode, const float* y_scale, uint8_t* y_bscale,
                       hipStream_t st);
// W8A8 linear from bf16 activations x [m, ldx] (16-byte aligned rows):
// the dynamic FP8 quantization of x inside the split-K GEMM; a_tscale
// receives the decode scale; out_mode 0 (bf16) or 1 (fp32)
hipError_t launch_linear_fp8(const uint16_t* x, int64_t ldx, float* a_tscale, const uint8_t* w_packed, int64_t m,
                             int64_t n, int64_t k, void* y, int64_t ldy, int out_mode, hipStream_t st);

}  // namespace qg

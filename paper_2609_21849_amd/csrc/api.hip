// api.hip -- the C ABI declared in include/qgemm.h.
//
// Every entry point validates its arguments on the host, then only enqueues
// kernels on the caller's stream. Nothing here allocates device memory or
// synchronises. A failed check returns before any HIP call, which is why
// these checks can be exercised on a machine without a GPU.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <limits>

#include "checks.hpp"
#include "kernels.hpp"
#include "log.hpp"
#include "qgemm.h"

namespace {

thread_local int g_last_hip_error = 0;

qg_status hip_status(hipError_t e) {
  if (e == hipSuccess) return QG_OK;
  g_last_hip_error = (int)e;
  return QG_ERR_HIP;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool valid_fmt(int f) {
  return f == QG_FMT_BF16 || f == QG_FMT_FP8_E4M3 || f == QG_FMT_NVFP4 || f == QG_FMT_MXFP4 || f == QG_FMT_MXFP8;
}

bool is_mx(int f) { return f == QG_FMT_MXFP4 || f == QG_FMT_MXFP8; }

// MX element codes: 4-byte stores / loads of 8 MXFP4 codes, 8-byte ones of
// 8 MXFP8 codes
uintptr_t mx_code_align(int f) { return f == QG_FMT_MXFP4 ? 4 : 8; }

constexpr int64_t kMaxDim = std::numeric_limits<int32_t>::max();
// qg_linear_fp8: every workgroup reduces the whole activation's max itself
constexpr int64_t kLinearFp8MaxElements = 65536;

}  // namespace

namespace qg {

qg_status check_quantize(qg_format fmt, const void* x, int64_t rows, int64_t cols, int64_t ldx,
                         const void* codes, const void* block_scales, const float* tensor_scale) {
  if (!valid_fmt(fmt)) return QG_ERR_INVALID_ARG;
  if (fmt == QG_FMT_BF16) return QG_ERR_UNSUPPORTED;
  if (rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return QG_ERR_INVALID_ARG;
  if (rows > 0 && ldx < cols) return QG_ERR_INVALID_ARG;
  const bool empty = (rows == 0 || cols == 0);
  if (is_mx(fmt)) {  // block scales only: no tensor scale
    if (tensor_scale != nullptr) return QG_ERR_INVALID_ARG;
    if (cols % 32 != 0) return QG_ERR_SHAPE;
    if (!empty && (x == nullptr || codes == nullptr || block_scales == nullptr || !aligned(x, 2) ||
                   !aligned(codes, fmt == QG_FMT_MXFP4 ? 4 : 1)))
      return QG_ERR_INVALID_ARG;
    return QG_OK;
  }
  if (tensor_scale == nullptr || !aligned(tensor_scale, 4)) return QG_ERR_INVALID_ARG;
  if (fmt == QG_FMT_NVFP4 && cols % 16 != 0) return QG_ERR_SHAPE;
  if (fmt == QG_FMT_FP8_E4M3 && block_scales != nullptr) return QG_ERR_INVALID_ARG;
  if (!empty) {
    if (x == nullptr || codes == nullptr || !aligned(x, 2)) return QG_ERR_INVALID_ARG;
    if (fmt == QG_FMT_NVFP4 && (block_scales == nullptr || !aligned(codes, 8))) return QG_ERR_INVALID_ARG;
  }
  return QG_OK;
}

qg_status check_gemm(qg_format a_fmt, const void* a, const void* a_block_scales, const float* a_tensor_scale,
                     int64_t lda, qg_format w_fmt, const void* w_packed, size_t w_packed_bytes, int64_t m,
                     int64_t n, int64_t k, const void* y, int64_t ldy, int y_esz) {
  if (!valid_fmt(a_fmt) || !valid_fmt(w_fmt)) return QG_ERR_INVALID_ARG;
  if (y_esz != 1 && y_esz != 2 && y_esz != 4) return QG_ERR_INVALID_ARG;
  const bool w8a8 = (a_fmt == QG_FMT_FP8_E4M3 && w_fmt == QG_FMT_FP8_E4M3);
  const bool w4a4 = (a_fmt == QG_FMT_NVFP4 && w_fmt == QG_FMT_NVFP4);
  const bool w4a16 = (a_fmt == QG_FMT_BF16 && w_fmt == QG_FMT_NVFP4);
  const bool mx4 = (a_fmt == QG_FMT_MXFP4 && w_fmt == QG_FMT_MXFP4);
  const bool mx8 = (a_fmt == QG_FMT_MXFP8 && w_fmt == QG_FMT_MXFP8);
  if (!(w8a8 || w4a4 || w4a16 || mx4 || mx8)) return QG_ERR_UNSUPPORTED;
  if (m < 0 || n < 0 || k < 0 || m > kMaxDim || n > kMaxDim || k > kMaxDim) return QG_ERR_INVALID_ARG;
  if (n % 16 != 0 || k % 128 != 0) return QG_ERR_SHAPE;
  if ((mx4 || mx8) && k % 256 != 0) return QG_ERR_SHAPE;
  if (m > 0 && lda < k) return QG_ERR_INVALID_ARG;
  if (m > 0 && ldy < n) return QG_ERR_INVALID_ARG;
  if (w_packed == nullptr || !aligned(w_packed, 256)) return QG_ERR_INVALID_ARG;
  if (w_packed_bytes < (size_t)packed_total_bytes((int)w_fmt, n, k)) return QG_ERR_BUFFER_TOO_SMALL;
  // operands are addressed with 32-bit byte offsets: every operand extent
  // (activation rows, their block scales, the packed weight) must stay below 2 GiB
  if (m > 0 && k > 0) {
    const int64_t esz2 = (w8a8 || mx8) ? 2 : ((w4a4 || mx4) ? 1 : 4);  // element size x 2
    const int64_t a_extent = ((m - 1) * lda + k) * esz2 / 2;
    if (a_extent > kMaxDim || (w4a4 && m * (lda / 16) > kMaxDim)) return QG_ERR_SHAPE;
  }
  if (packed_total_bytes((int)w_fmt, n, k) > kMaxDim) return QG_ERR_SHAPE;
  if (m > 0 && n > 0) {
    if (y == nullptr || !aligned(y, (uintptr_t)y_esz)) return QG_ERR_INVALID_ARG;
    if (k > 0) {
      if (a == nullptr) return QG_ERR_INVALID_ARG;
      if (w8a8 && (!aligned(a, 16) || lda % 16 != 0 || a_tensor_scale == nullptr || a_block_scales != nullptr))
        return QG_ERR_INVALID_ARG;
      // NVFP4 activations: rows of lda / 2 code bytes and lda / 16 scale bytes
      // (lda > k reads the first k columns of a wider tensor in place)
      if (w4a4 && (!aligned(a, 16) || lda % 128 != 0 || a_tensor_scale == nullptr || a_block_scales == nullptr ||
                   !aligned(a_block_scales, 8)))
        return QG_ERR_INVALID_ARG;
      if (w4a16 && (!aligned(a, 16) || lda % 8 != 0 || a_tensor_scale != nullptr || a_block_scales != nullptr))
        return QG_ERR_INVALID_ARG;
      if (mx4 && (!aligned(a, 16) || lda != k || a_tensor_scale != nullptr || a_block_scales == nullptr ||
                  !aligned(a_block_scales, 8)))
        return QG_ERR_INVALID_ARG;
      if (mx8 && (!aligned(a, 16) || lda != k || a_tensor_scale != nullptr || a_block_scales == nullptr ||
                  !aligned(a_block_scales, 4)))
        return QG_ERR_INVALID_ARG;
    }
  }
  return QG_OK;
}

qg_status status_of(hipError_t e) { return hip_status(e); }

void log_call(const char* fn, qg_status st, const char* fmt, ...) {
  char args[256];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(args, sizeof args, fmt, ap);
  va_end(ap);
  if (st == QG_ERR_HIP)
    std::fprintf(stderr, "[qgemm] %s(%s) -> %s (hipError %d: %s)\n", fn, args, qg_status_string(st),
                 g_last_hip_error, hipGetErrorString((hipError_t)g_last_hip_error));
  else
    std::fprintf(stderr, "[qgemm] %s(%s) -> %s\n", fn, args, qg_status_string(st));
}

}  // namespace qg

extern "C" {

const char* qg_status_string(qg_status s) {
  switch (s) {
    case QG_OK: return "ok";
    case QG_ERR_INVALID_ARG: return "invalid argument";
    case QG_ERR_UNSUPPORTED: return "unsupported format";
    case QG_ERR_SHAPE: return "shape breaks the layout contract";
    case QG_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case QG_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

int qg_last_hip_error(void) { return g_last_hip_error; }

int qg_abi_version(void) { return QG_ABI_VERSION; }

qg_status qg_quantize_act(qg_format fmt, const void* x, int64_t rows, int64_t cols, int64_t ldx,
                          void* codes, void* block_scales, float* tensor_scale, void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    const qg_status c = qg::check_quantize(fmt, x, rows, cols, ldx, codes, block_scales, tensor_scale);
    if (c != QG_OK) return c;
    return hip_status(qg::launch_quantize((int)fmt, reinterpret_cast<const uint16_t*>(x), rows, cols, ldx,
                                          reinterpret_cast<uint8_t*>(codes),
                                          reinterpret_cast<uint8_t*>(block_scales), tensor_scale,
                                          reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_quantize_act", st_, "fmt=%d rows=%lld cols=%lld ldx=%lld",
                 (int)fmt, (long long)rows, (long long)cols, (long long)ldx);
  return st_;
}

qg_status qg_quantize_act_static(qg_format fmt, const void* x, int64_t rows, int64_t cols, int64_t ldx,
                                 void* codes, void* block_scales, const float* tensor_scale, void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    if (!valid_fmt(fmt)) return QG_ERR_INVALID_ARG;
    if (fmt == QG_FMT_BF16 || is_mx(fmt)) return QG_ERR_UNSUPPORTED;
    if (rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return QG_ERR_INVALID_ARG;
    if (rows > 0 && ldx < cols) return QG_ERR_INVALID_ARG;
    if (tensor_scale == nullptr || !aligned(tensor_scale, 4)) return QG_ERR_INVALID_ARG;
    if (fmt == QG_FMT_NVFP4 && cols % 16 != 0) return QG_ERR_SHAPE;
    if (fmt == QG_FMT_FP8_E4M3 && block_scales != nullptr) return QG_ERR_INVALID_ARG;
    if (rows > 0 && cols > 0) {
      if (x == nullptr || codes == nullptr || !aligned(x, 2)) return QG_ERR_INVALID_ARG;
      if (fmt == QG_FMT_NVFP4 && (block_scales == nullptr || !aligned(codes, 8))) return QG_ERR_INVALID_ARG;
    }
    return hip_status(qg::launch_quantize_static((int)fmt, reinterpret_cast<const uint16_t*>(x), rows, cols, ldx,
                                                 reinterpret_cast<uint8_t*>(codes),
                                                 reinterpret_cast<uint8_t*>(block_scales), tensor_scale,
                                                 reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_quantize_act_static", st_, "fmt=%d rows=%lld cols=%lld ldx=%lld",
                 (int)fmt, (long long)rows, (long long)cols, (long long)ldx);
  return st_;
}

size_t qg_packed_bytes(qg_format fmt, int64_t n, int64_t k) {
  if (!valid_fmt(fmt) || fmt == QG_FMT_BF16) return 0;
  if (n < 0 || k < 0 || n > kMaxDim || k > kMaxDim || n % 16 != 0 || k % 128 != 0) return 0;
  if (is_mx(fmt) && k % 256 != 0) return 0;
  return (size_t)qg::packed_total_bytes((int)fmt, n, k);
}

static qg_status check_pack_args(qg_format fmt, const void* codes, const void* block_scales,
                                 const void* tensor_scale, int64_t n, int64_t k,
                                 const void* packed, size_t packed_bytes) {
  if (!valid_fmt(fmt)) return QG_ERR_INVALID_ARG;
  if (fmt == QG_FMT_BF16) return QG_ERR_UNSUPPORTED;
  if (n < 0 || k < 0 || n > kMaxDim || k > kMaxDim) return QG_ERR_INVALID_ARG;
  if (n % 16 != 0 || k % 128 != 0) return QG_ERR_SHAPE;
  if (is_mx(fmt) && k % 256 != 0) return QG_ERR_SHAPE;
  if (packed == nullptr || !aligned(packed, 256)) return QG_ERR_INVALID_ARG;
  // the MX formats have no tensor scale; the others carry one in the header
  if (is_mx(fmt) ? tensor_scale != nullptr : (tensor_scale == nullptr || !aligned(tensor_scale, 4)))
    return QG_ERR_INVALID_ARG;
  if (packed_bytes < (size_t)qg::packed_total_bytes((int)fmt, n, k)) return QG_ERR_BUFFER_TOO_SMALL;
  if (n > 0 && k > 0) {
    if (codes == nullptr || !aligned(codes, 16)) return QG_ERR_INVALID_ARG;
    if (fmt == QG_FMT_NVFP4 && (block_scales == nullptr || !aligned(block_scales, 8))) return QG_ERR_INVALID_ARG;
    if (is_mx(fmt) && block_scales == nullptr) return QG_ERR_INVALID_ARG;
  }
  if (fmt == QG_FMT_FP8_E4M3 && block_scales != nullptr) return QG_ERR_INVALID_ARG;
  return QG_OK;
}

qg_status qg_pack_weights(qg_format fmt, const void* codes, const void* block_scales,
                          const float* tensor_scale, int64_t n, int64_t k, void* packed,
                          size_t packed_bytes, void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    const qg_status s = check_pack_args(fmt, codes, block_scales, tensor_scale, n, k, packed, packed_bytes);
    if (s != QG_OK) return s;
    return hip_status(qg::launch_pack((int)fmt, reinterpret_cast<const uint8_t*>(codes),
                                      reinterpret_cast<const uint8_t*>(block_scales), tensor_scale, n,
                                      k, reinterpret_cast<uint8_t*>(packed),
                                      reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_pack_weights", st_, "fmt=%d n=%lld k=%lld packed_bytes=%zu",
                 (int)fmt, (long long)n, (long long)k, packed_bytes);
  return st_;
}

qg_status qg_unpack_weights(qg_format fmt, const void* packed, size_t packed_bytes, int64_t n,
                            int64_t k, void* codes, void* block_scales, float* tensor_scale,
                            void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    const qg_status s = check_pack_args(fmt, codes, block_scales, tensor_scale, n, k, packed, packed_bytes);
    if (s != QG_OK) return s;
    return hip_status(qg::launch_unpack((int)fmt, reinterpret_cast<const uint8_t*>(packed), n, k,
                                        reinterpret_cast<uint8_t*>(codes),
                                        reinterpret_cast<uint8_t*>(block_scales), tensor_scale,
                                        reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_unpack_weights", st_, "fmt=%d n=%lld k=%lld packed_bytes=%zu",
                 (int)fmt, (long long)n, (long long)k, packed_bytes);
  return st_;
}

qg_status qg_gemm(qg_format a_fmt, const void* a, const void* a_block_scales,
                  const float* a_tensor_scale, int64_t lda, qg_format w_fmt, const void* w_packed,
                  size_t w_packed_bytes, int64_t m, int64_t n, int64_t k, void* y, int64_t ldy,
                  qg_out_dtype y_dtype, void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    if (y_dtype != QG_OUT_BF16 && y_dtype != QG_OUT_F32) return QG_ERR_INVALID_ARG;
    const qg_status c = qg::check_gemm(a_fmt, a, a_block_scales, a_tensor_scale, lda, w_fmt, w_packed,
                                       w_packed_bytes, m, n, k, y, ldy, y_dtype == QG_OUT_F32 ? 4 : 2);
    if (c != QG_OK) return c;
    return hip_status(qg::launch_gemm((int)a_fmt, a, reinterpret_cast<const uint8_t*>(a_block_scales),
                                      a_tensor_scale, lda, reinterpret_cast<const uint8_t*>(w_packed), m,
                                      n, k, y, ldy, y_dtype == QG_OUT_F32 ? 1 : 0, nullptr, nullptr,
                                      reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_gemm", st_, "a_fmt=%d w_fmt=%d m=%lld n=%lld k=%lld lda=%lld ldy=%lld y_dtype=%d",
                 (int)a_fmt, (int)w_fmt, (long long)m, (long long)n, (long long)k, (long long)lda,
                 (long long)ldy, (int)y_dtype);
  return st_;
}

qg_status qg_linear_fp8(const void* x, int64_t ldx, float* a_tensor_scale, const void* w_packed,
                        size_t w_packed_bytes, int64_t m, int64_t n, int64_t k, void* y, int64_t ldy,
                        qg_out_dtype y_dtype, void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    if (y_dtype != QG_OUT_BF16 && y_dtype != QG_OUT_F32) return QG_ERR_INVALID_ARG;
    if (a_tensor_scale == nullptr || !aligned(a_tensor_scale, 4)) return QG_ERR_INVALID_ARG;
    if (m < 0 || n < 0 || k < 0 || m > kMaxDim || n > kMaxDim || k > kMaxDim) return QG_ERR_INVALID_ARG;
    if (n % 16 != 0 || k % 128 != 0) return QG_ERR_SHAPE;
    if (m * k > kLinearFp8MaxElements) return QG_ERR_SHAPE;
    if (m > 0 && (ldx < k || ldy < n)) return QG_ERR_INVALID_ARG;
    if (w_packed == nullptr || !aligned(w_packed, 256)) return QG_ERR_INVALID_ARG;
    if (w_packed_bytes < (size_t)qg::packed_total_bytes(QG_FMT_FP8_E4M3, n, k)) return QG_ERR_BUFFER_TOO_SMALL;
    if (qg::packed_total_bytes(QG_FMT_FP8_E4M3, n, k) > kMaxDim) return QG_ERR_SHAPE;
    if (m > 0 && k > 0) {
      if (x == nullptr || !aligned(x, 16) || ldx % 8 != 0) return QG_ERR_INVALID_ARG;
      if (((m - 1) * ldx + k) * 2 > kMaxDim) return QG_ERR_SHAPE;
    }
    if (m > 0 && n > 0 && (y == nullptr || !aligned(y, y_dtype == QG_OUT_F32 ? 4 : 2))) return QG_ERR_INVALID_ARG;
    return hip_status(qg::launch_linear_fp8(reinterpret_cast<const uint16_t*>(x), ldx, a_tensor_scale,
                                            reinterpret_cast<const uint8_t*>(w_packed), m, n, k, y, ldy,
                                            y_dtype == QG_OUT_F32 ? 1 : 0, reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_linear_fp8", st_, "m=%lld n=%lld k=%lld ldx=%lld ldy=%lld y_dtype=%d", (long long)m,
                 (long long)n, (long long)k, (long long)ldx, (long long)ldy, (int)y_dtype);
  return st_;
}

qg_status qg_gemm_quant(qg_format a_fmt, const void* a, const void* a_block_scales, const float* a_tensor_scale,
                        int64_t lda, qg_format w_fmt, const void* w_packed, size_t w_packed_bytes, int64_t m,
                        int64_t n, int64_t k, void* y_codes, int64_t ldy, const float* y_scale, void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    if (y_scale == nullptr || !aligned(y_scale, 4)) return QG_ERR_INVALID_ARG;
    const qg_status c = qg::check_gemm(a_fmt, a, a_block_scales, a_tensor_scale, lda, w_fmt, w_packed,
                                       w_packed_bytes, m, n, k, y_codes, ldy, 1);
    if (c != QG_OK) return c;
    return hip_status(qg::launch_gemm((int)a_fmt, a, reinterpret_cast<const uint8_t*>(a_block_scales),
                                      a_tensor_scale, lda, reinterpret_cast<const uint8_t*>(w_packed), m,
                                      n, k, y_codes, ldy, 2, y_scale, nullptr, reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_gemm_quant", st_, "a_fmt=%d w_fmt=%d m=%lld n=%lld k=%lld lda=%lld ldy=%lld",
                 (int)a_fmt, (int)w_fmt, (long long)m, (long long)n, (long long)k, (long long)lda,
                 (long long)ldy);
  return st_;
}

qg_status qg_gemm_quant_nvfp4(qg_format a_fmt, const void* a, const void* a_block_scales,
                              const float* a_tensor_scale, int64_t lda, qg_format w_fmt, const void* w_packed,
                              size_t w_packed_bytes, int64_t m, int64_t n, int64_t k, void* y_codes,
                              void* y_block_scales, int64_t ldy, const float* y_tensor_scale, void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    if (y_tensor_scale == nullptr || !aligned(y_tensor_scale, 4)) return QG_ERR_INVALID_ARG;
    // codes are written four bytes at a time, rows of ldy / 2 bytes
    const qg_status c = qg::check_gemm(a_fmt, a, a_block_scales, a_tensor_scale, lda, w_fmt, w_packed,
                                       w_packed_bytes, m, n, k, y_codes, ldy, 4);
    if (c != QG_OK) return c;
    if (a_fmt == QG_FMT_BF16) return QG_ERR_UNSUPPORTED;  // weight-only linears keep bf16 / fp32 outputs
    if (m > 0 && ldy % 16 != 0) return QG_ERR_INVALID_ARG;
    if (m > 0 && n > 0 && (y_block_scales == nullptr || !aligned(y_codes, 4))) return QG_ERR_INVALID_ARG;
    if (m > 0 && ((m - 1) * ldy + n) / 2 > kMaxDim) return QG_ERR_SHAPE;
    return hip_status(qg::launch_gemm((int)a_fmt, a, reinterpret_cast<const uint8_t*>(a_block_scales),
                                      a_tensor_scale, lda, reinterpret_cast<const uint8_t*>(w_packed), m,
                                      n, k, y_codes, ldy, 3, y_tensor_scale,
                                      reinterpret_cast<uint8_t*>(y_block_scales),
                                      reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_gemm_quant_nvfp4", st_, "a_fmt=%d w_fmt=%d m=%lld n=%lld k=%lld lda=%lld ldy=%lld",
                 (int)a_fmt, (int)w_fmt, (long long)m, (long long)n, (long long)k, (long long)lda,
                 (long long)ldy);
  return st_;
}

qg_status qg_dequant(qg_format fmt, const void* codes, const void* block_scales,
                     const float* tensor_scale, int64_t rows, int64_t cols, void* out,
                     qg_out_dtype out_dtype, void* stream) {
  const qg_status st_ = [&]() -> qg_status {
    if (!valid_fmt(fmt)) return QG_ERR_INVALID_ARG;
    if (fmt == QG_FMT_BF16) return QG_ERR_UNSUPPORTED;
    if (out_dtype != QG_OUT_BF16 && out_dtype != QG_OUT_F32) return QG_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return QG_ERR_INVALID_ARG;
    if (is_mx(fmt)) {
      if (tensor_scale != nullptr) return QG_ERR_INVALID_ARG;
      if (cols % 32 != 0) return QG_ERR_SHAPE;
      if (rows > 0 && cols > 0 &&
          (codes == nullptr || block_scales == nullptr || out == nullptr || !aligned(codes, mx_code_align(fmt)) ||
           !aligned(out, 16)))
        return QG_ERR_INVALID_ARG;
      return hip_status(qg::launch_dequant((int)fmt, reinterpret_cast<const uint8_t*>(codes),
                                           reinterpret_cast<const uint8_t*>(block_scales), nullptr, rows, cols,
                                           out, out_dtype == QG_OUT_F32, reinterpret_cast<hipStream_t>(stream)));
    }
    if (fmt == QG_FMT_NVFP4 && cols % 16 != 0) return QG_ERR_SHAPE;
    if (tensor_scale == nullptr || !aligned(tensor_scale, 4)) return QG_ERR_INVALID_ARG;
    if (fmt == QG_FMT_FP8_E4M3 && block_scales != nullptr) return QG_ERR_INVALID_ARG;
    if (rows > 0 && cols > 0) {
      if (codes == nullptr || out == nullptr || !aligned(out, out_dtype == QG_OUT_F32 ? 4 : 2))
        return QG_ERR_INVALID_ARG;
      if (fmt == QG_FMT_NVFP4 && (block_scales == nullptr || !aligned(codes, 8))) return QG_ERR_INVALID_ARG;
    }
    return hip_status(qg::launch_dequant((int)fmt, reinterpret_cast<const uint8_t*>(codes),
                                         reinterpret_cast<const uint8_t*>(block_scales), tensor_scale,
                                         rows, cols, out, out_dtype == QG_OUT_F32,
                                         reinterpret_cast<hipStream_t>(stream)));
  }();
  if (qg::log_enabled())
    qg::log_call("qg_dequant", st_, "fmt=%d rows=%lld cols=%lld out_dtype=%d",
                 (int)fmt, (long long)rows, (long long)cols, (int)out_dtype);
  return st_;
}

}  // extern "C"

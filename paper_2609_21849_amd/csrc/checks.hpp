// checks.hpp -- host-side argument checks of the C ABI, shared by the entry
// points that validate a whole batch of calls before enqueueing any of them.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qgemm.h"

namespace qg {

// The checks of qg_quantize_act (before anything is enqueued).
qg_status check_quantize(qg_format fmt, const void* x, int64_t rows, int64_t cols, int64_t ldx,
                         const void* codes, const void* block_scales, const float* tensor_scale);
// The checks of qg_gemm; y_esz = bytes per output element (1 FP8 codes, 2 bf16, 4 fp32).
qg_status check_gemm(qg_format a_fmt, const void* a, const void* a_block_scales, const float* a_tensor_scale,
                     int64_t lda, qg_format w_fmt, const void* w_packed, size_t w_packed_bytes, int64_t m,
                     int64_t n, int64_t k, const void* y, int64_t ldy, int y_esz);
// QG_OK for hipSuccess, else QG_ERR_HIP (the code is kept for qg_last_hip_error).
qg_status status_of(hipError_t e);

}  // namespace qg

/*
 * qgemm.h -- C ABI of the MI355X (gfx950) low-bit quantized-linear library.
 *
 * The library implements the quantized linear layers that the paper's
 * recipe puts on low-precision matrix units (Sec. 4, quantization paragraph;
 * effect in Table 2): post-training quantization of weights AND runtime
 * quantization of activations, in two formats the paper cites there:
 *
 *   FP8  : E4M3 codes (bias 7, largest finite 448, no infinities), one fp32
 *          decode scale per tensor:   x ~ e4m3(q) * s.
 *   NVFP4: E2M1 codes (0, .5, 1, 1.5, 2, 3, 4, 6 and negatives) in blocks of
 *          16 consecutive elements along a row, one E4M3 scale per block and
 *          one fp32 decode scale per tensor:  x ~ e2m1(q) * e4m3(s_b) * s_t.
 *
 * and a weight-only variant (bf16 activations times NVFP4 weights). Beside
 * them, the OCP Microscaling (MX v1.0) 4- and 8-bit formats, the block
 * scaling gfx950's matrix cores apply in hardware:
 *
 *   MXFP4: E2M1 codes in blocks of 32 consecutive elements along a row, one
 *          E8M0 scale (a power of two 2^(e-127), e in 0..254) per block and
 *          no tensor scale:                x ~ e2m1(q) * 2^(e-127).
 *   MXFP8: the same with E4M3 codes.
 *
 * MX is the hardware-native variant of the paper's 4-bit recipe (Sec. 4,
 * quantization paragraph: activation quantization onto 4-bit matrix units);
 * its numerics differ from NVFP4's (power-of-two scales per 32 instead of
 * E4M3 scales per 16), so it is a separate format, not an NVFP4 kernel.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every tensor pointer is a DEVICE pointer on the current HIP device.
 *    The caller allocates and owns every buffer; the library allocates
 *    nothing and keeps no state besides its loaded code objects.
 *  - Matrices are row-major. A "row" runs along the reduction dimension K of
 *    a linear layer: activations X are [M, K], weights W are [N, K] (the
 *    nn.Linear layout), outputs Y are [M, N].
 *  - bf16 data are 16-bit bfloat16 bit patterns; `ld*` arguments count
 *    elements between consecutive rows (>= the row length).
 *  - FP8 codes: one byte per element, dense [rows, cols].
 *  - NVFP4 codes: two per byte, dense [rows, cols/2]; element 2i of a row
 *    sits in the low nibble of byte i. Block scales: E4M3 bytes, dense
 *    [rows, cols/16]; block j covers elements 16j .. 16j+15 of its row.
 *  - MX codes: MXFP4 like NVFP4 codes, MXFP8 like FP8 codes. Block scales:
 *    E8M0 bytes, dense [rows, cols/32]; block j covers elements 32j .. 32j+31.
 *  - Tensor scales are single fp32 values in device memory (decode scales).
 *  - All work is enqueued on `stream` (a hipStream_t; NULL = the default
 *    stream) with no host synchronisation. Argument and shape checks run on
 *    the host before anything is enqueued and report through the return
 *    value; a failed check enqueues nothing. Errors of the HIP runtime are
 *    reported as QG_ERR_HIP (see qg_last_hip_error). Calls are thread-safe;
 *    calls whose buffers overlap must be ordered by the caller's streams.
 *  - Non-finite inputs are outside the contract: a tensor holding inf/NaN
 *    gets a NaN tensor scale (a sentinel a caller can test) and
 *    unspecified codes. The MX formats have no tensor scale: a block holding
 *    inf/NaN gets the E8M0 NaN code 255 as its block scale (the other blocks
 *    are unaffected), unspecified element codes, a NaN dequantization, and
 *    unspecified GEMM outputs wherever it takes part.
 *  - Debug logging: with the environment variable QG_LOG set (to anything
 *    but "" or "0") when the library is first used, every qg_status entry
 *    point writes one line to stderr with its name, its scalar arguments
 *    and the status it returns. Off by default.
 */
#ifndef QGEMM_H
#define QGEMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QG_ABI_VERSION 1

typedef enum qg_status {
    QG_OK = 0,
    QG_ERR_INVALID_ARG = 1,      /* null pointer, bad enum, negative size, ld too small */
    QG_ERR_UNSUPPORTED = 2,      /* format or format pair the library does not implement */
    QG_ERR_SHAPE = 3,            /* shape breaks the layout contract (e.g. K % 16 for NVFP4) */
    QG_ERR_BUFFER_TOO_SMALL = 4, /* a size argument is smaller than the data it must hold */
    QG_ERR_HIP = 5               /* the HIP runtime reported an error */
} qg_status;

typedef enum qg_format {
    QG_FMT_BF16 = 0,             /* unquantized bfloat16 */
    QG_FMT_FP8_E4M3 = 1,         /* E4M3 codes + per-tensor fp32 scale */
    QG_FMT_NVFP4 = 2,            /* E2M1 codes + E4M3 per-16 block scales + fp32 tensor scale */
    QG_FMT_MXFP4 = 3,            /* E2M1 codes + E8M0 per-32 block scales, no tensor scale */
    QG_FMT_MXFP8 = 4             /* E4M3 codes + E8M0 per-32 block scales, no tensor scale */
} qg_format;

typedef enum qg_out_dtype {
    QG_OUT_BF16 = 0,             /* round-to-nearest-even bfloat16 */
    QG_OUT_F32 = 1               /* IEEE binary32 */
} qg_out_dtype;

/*
 * qg_quantize_act -- dynamic quantization of a bf16 tensor (activations at
 * run time, weights offline before qg_pack_weights: the same arithmetic).
 * Paper: Sec. 4, quantization paragraph (activation quantization is what
 * lets the linears run on low-precision units; PTQ of weights).
 *
 *   fmt           QG_FMT_FP8_E4M3, QG_FMT_NVFP4, QG_FMT_MXFP4 or QG_FMT_MXFP8.
 *   x             bf16 [rows, ldx], the first `cols` of each row are used.
 *   codes         out: FP8/MXFP8 [rows, cols] bytes; NVFP4/MXFP4 [rows, cols/2]
 *                 bytes (MXFP4: 4-byte aligned).
 *   block_scales  out: NVFP4 [rows, cols/16] E4M3 bytes; MX [rows, cols/32]
 *                 E8M0 bytes; must be NULL for FP8.
 *   tensor_scale  out: one fp32 decode scale; must be NULL for the MX formats.
 *   A tensor of at most 3072 units of 16 elements (units per row:
 *   ceil(cols / 16)) is quantized by one launch, whose workgroups each
 *   reduce the whole tensor and code their share of it. A dense one
 *   (ldx == cols, 16-byte aligned x, 8-byte aligned codes, rows * cols a
 *   multiple of 8) of at most 3 Mi elements takes two launches: the first
 *   leaves its partial maxima in `codes`, the second reduces them and writes
 *   the codes over them. Any other tensor-wide max is reduced in two kernels
 *   whose partial results are parked in `codes` the same way, then a third
 *   codes the elements. Always x, codes, block_scales and tensor_scale must
 *   not overlap.
 *
 * Arithmetic (bit-exact; every step one IEEE binary32 operation, RNE):
 *   FP8  : a = max|x|; s = a/448; r = s>0 ? 1/s : 0; q = E4M3(x*r)
 *   NVFP4: a = max|x|; s_t = a/2688; d = 6*s_t; per block b:
 *          v = d>0 ? max_b|x|/d : 0; s_b = E4M3(v); S = e4m3(s_b)*s_t;
 *          r = S>0 ? 1/S : 0; q = E2M1(x*r)
 *   MX   : per block b: a_b = max_b|x|; e = a_b > 0 ? clamp(floor(log2 a_b)
 *          - emax + 127, 0, 254) : 0 (emax = 2 for E2M1, 8 for E4M3);
 *          q = E2M1 / E4M3(x * 2^(127-e)) (the product is exact). OCP MX
 *          v1.0, scale and element conversion; one kernel, no reduction
 *          across the tensor.
 *   E4M3()/E2M1() round to nearest, ties to the even code, saturate at
 *   +-448 / +-6, and keep the sign of zero.
 * Shapes: rows, cols >= 0; NVFP4 needs cols % 16 == 0, MX cols % 32 == 0
 * (QG_ERR_SHAPE). An empty tensor gets tensor_scale = 0 (none for MX).
 */
qg_status qg_quantize_act(qg_format fmt, const void *x, int64_t rows, int64_t cols, int64_t ldx,
                          void *codes, void *block_scales, float *tensor_scale, void *stream);

/*
 * qg_quantize_act_static -- quantization of a bf16 tensor with a static
 * (calibrated) decode scale instead of the tensor's own max: post-training
 * quantization with fixed activation ranges, which removes the tensor-wide
 * max reduction (for all but small tensors, two of the three kernels of
 * qg_quantize_act) from the run time. Paper: Sec. 4, quantization paragraph
 * (PTQ recipe).
 *
 *   fmt, x, rows, cols, ldx, codes, block_scales: as for qg_quantize_act.
 *   tensor_scale  in: the fp32 decode scale (FP8: s; NVFP4: s_t), e.g. the
 *                 value qg_quantize_act wrote for calibration data, or the
 *                 max of such values over several batches. It must be 0 or
 *                 a normal positive number (FP8), 0 or >= 2^-96 (NVFP4);
 *                 other values give unspecified codes. It is not written.
 * Arithmetic: the element (and, for NVFP4, block) steps of qg_quantize_act
 * with the given scale; elements beyond the calibrated range saturate to
 * +-448 (FP8) or to a block scale of 448 and codes of +-6 (NVFP4). With the
 * scale qg_quantize_act would derive, the codes are identical to its codes.
 * An empty tensor enqueues nothing. The MX formats have no tensor scale:
 * QG_ERR_UNSUPPORTED.
 */
qg_status qg_quantize_act_static(qg_format fmt, const void *x, int64_t rows, int64_t cols, int64_t ldx,
                                 void *codes, void *block_scales, const float *tensor_scale, void *stream);

/*
 * qg_packed_bytes -- size of the packed weight buffer for an [n, k] weight
 * in `fmt` (FP8, NVFP4, MXFP4 or MXFP8), or 0 when the shape breaks the GEMM
 * contract (n % 16, k % 128; MX k % 256) or the format is not packable.
 * Paper: Sec. 4, quantization and weight-streaming paragraphs (the bytes a
 * quantized layer occupies are the W of the streaming cost model below).
 * Host-only; touches no device memory.
 */
size_t qg_packed_bytes(qg_format fmt, int64_t n, int64_t k);

/*
 * qg_pack_weights -- offline re-layout of a quantized weight W [n, k] into
 * the order in which the GEMM's matrix-core operands consume it, plus a
 * small header holding the format, n, k and a copy of the tensor scale.
 * Paper: Sec. 4, quantization paragraph (PTQ weights are prepared once,
 * like the cached engines of Sec. 5).
 *
 *   codes, block_scales, tensor_scale: as written by qg_quantize_act
 *                 (block_scales NULL for FP8; tensor_scale NULL for MX).
 *   packed        out: qg_packed_bytes(fmt, n, k) bytes, 256-byte aligned.
 * The layout is private to this library version (qg_unpack_weights is its
 * exact inverse). Shapes: n % 16 == 0 and k % 128 == 0 (MX: k % 256), else
 * QG_ERR_SHAPE.
 */
qg_status qg_pack_weights(qg_format fmt, const void *codes, const void *block_scales,
                          const float *tensor_scale, int64_t n, int64_t k,
                          void *packed, size_t packed_bytes, void *stream);

/*
 * qg_unpack_weights -- inverse of qg_pack_weights: writes the canonical
 * codes, block scales (NVFP4, MX) and tensor scale (FP8, NVFP4) back out.
 * Paper: Sec. 4, quantization paragraph (the PTQ weight as quantized: the
 * formats above). For tests and for tools that need the weights in the
 * canonical layout. Arguments are checked as in qg_pack_weights
 * (packed_bytes < qg_packed_bytes(fmt, n, k): QG_ERR_BUFFER_TOO_SMALL). The
 * header sits in device memory and is not read on the host: fmt, n and k
 * must be those of the qg_pack_weights call, else the outputs are
 * unspecified. Outputs are dense like qg_quantize_act's (block_scales NULL
 * for FP8; tensor_scale NULL for MX).
 */
qg_status qg_unpack_weights(qg_format fmt, const void *packed, size_t packed_bytes,
                            int64_t n, int64_t k, void *codes, void *block_scales,
                            float *tensor_scale, void *stream);

/*
 * qg_gemm -- quantized linear layer Y = deq(A) . deq(W)^T.
 * Paper: Sec. 4, quantization paragraph; Table 2 (FP8 and NVFP4 linears of
 * the denoising transformer); weight-only NVFP4 for the small encoder path.
 *
 * Supported (a_fmt, w_fmt) pairs, else QG_ERR_UNSUPPORTED:
 *   (FP8_E4M3, FP8_E4M3)  W8A8:  a = codes [m, k] (lda = k), a_block_scales NULL
 *   (NVFP4,    NVFP4)     W4A4:  a = codes, rows of lda/2 bytes, and
 *                         a_block_scales, rows of lda/16 bytes (8-byte
 *                         aligned); lda >= k, lda % 128 == 0 (lda > k reads
 *                         the first k columns of a wider tensor in place)
 *   (BF16,     NVFP4)     W4A16: a = bf16 [m, lda], a_block_scales and a_tensor_scale NULL
 *   (MXFP4,    MXFP4)     MX W4A4: a = codes [m, k/2], a_block_scales [m, k/32]
 *                         (8-byte aligned, lda = k), a_tensor_scale NULL;
 *                         k % 256 == 0. The E8M0 block scales of both
 *                         operands are applied by the matrix instruction.
 *   (MXFP8,    MXFP8)     MX W8A8: a = codes [m, k], a_block_scales [m, k/32]
 *                         (4-byte aligned, lda = k), a_tensor_scale NULL;
 *                         k % 256 == 0.
 *   a_tensor_scale  device fp32 decode scale of A (FP8, NVFP4).
 *   w_packed        buffer written by qg_pack_weights for an [n, k] weight.
 *   y               out: [m, ldy] of y_dtype.
 * Result: y[i,j] = s_a * s_w * sum_k deq'(a)[i,k] deq'(w)[j,k] with fp32
 * accumulation (deq' = decoded codes times block scales; the tensor scales
 * are applied once at the end; MX has none), then rounded to y_dtype. Accuracy contract:
 * |y - y_exact| <= 1e-3 * sum_k |a w| plus the rounding of y to y_dtype.
 * Shapes: m, n, k >= 0; n % 16 == 0; k % 128 == 0; lda >= k, ldy >= n.
 * Operands are addressed with 32-bit byte offsets: the activation extent
 * ((m - 1) * lda + k elements), NVFP4 activation scales and the packed
 * weight must each stay below 2 GiB, else QG_ERR_SHAPE.
 */
qg_status qg_gemm(qg_format a_fmt, const void *a, const void *a_block_scales,
                  const float *a_tensor_scale, int64_t lda,
                  qg_format w_fmt, const void *w_packed, size_t w_packed_bytes,
                  int64_t m, int64_t n, int64_t k,
                  void *y, int64_t ldy, qg_out_dtype y_dtype, void *stream);

/*
 * qg_linear_fp8 -- W8A8 linear layer straight from bf16 activations: the
 * dynamic per-tensor FP8 quantization of qg_quantize_act done inside the
 * GEMM of qg_gemm, one launch instead of two, for activations small enough
 * that every workgroup reduces the whole tensor's max itself (few tokens:
 * the single FP8 linear, the small encoder's linears). Paper: Sec. 4,
 * quantization paragraph (activations quantized at run time for the FP8
 * linears; the encoder runs on few tokens).
 *   x               bf16 [m, ldx] activations, 16-byte aligned, ldx % 8 == 0,
 *                   ldx >= k; not modified.
 *   a_tensor_scale  out: device fp32, the decode scale s = fl(max|x| / 448)
 *                   (NaN when x holds inf or NaN, 0 for an empty x), the bits
 *                   qg_quantize_act writes for the same x.
 *   w_packed        an FP8 weight [n, k] as written by qg_pack_weights.
 *   y               out: [m, ldy] of y_dtype (bf16 or fp32).
 * Result: the activation codes are those of qg_quantize_act; y is the value
 * qg_gemm(FP8, FP8) returns for them, bit for bit where qg_gemm takes its
 * few-token (split-K) kernel, which is every shape with m <= 1024 and at
 * most two 32 x 64 tiles per compute unit; elsewhere within qg_gemm's
 * accuracy contract. Shapes: n % 16 == 0, k % 128 == 0, ldy >= n and
 * m * k <= 65536, else QG_ERR_SHAPE (a larger activation takes
 * qg_quantize_act and qg_gemm). x, a_tensor_scale and y must not overlap.
 */
qg_status qg_linear_fp8(const void *x, int64_t ldx, float *a_tensor_scale,
                        const void *w_packed, size_t w_packed_bytes,
                        int64_t m, int64_t n, int64_t k,
                        void *y, int64_t ldy, qg_out_dtype y_dtype, void *stream);

/*
 * qg_gemm_quant -- qg_gemm whose epilogue writes the output already
 * quantized to FP8 E4M3 with a static (calibrated) decode scale: the next
 * linear's activation operand, produced without the bf16 round trip through
 * memory and without a separate quantize kernel. Paper: Sec. 4, quantization
 * paragraph (activations quantized for the low-precision linears; PTQ with
 * calibrated ranges).
 *   a_fmt ... k   as for qg_gemm (every supported pair).
 *   y_codes       out: [m, ldy] E4M3 bytes (ldy >= n, any alignment).
 *   y_scale       in: device fp32 decode scale s_y of the output, 0 or a
 *                 normal positive number (e.g. the scale qg_quantize_act
 *                 derived for calibration data); not written.
 * Result: y_codes[i,j] = E4M3(fl(y[i,j] * r)) with r = s_y > 0 ? fl(1/s_y) : 0
 * and y[i,j] the fp32 value qg_gemm would round to its output type; E4M3()
 * rounds to nearest even and saturates at +-448, as in qg_quantize_act. With
 * the accuracy contract of qg_gemm, every code is a correct rounding of some
 * value within that contract's error of the exact product.
 */
qg_status qg_gemm_quant(qg_format a_fmt, const void *a, const void *a_block_scales,
                        const float *a_tensor_scale, int64_t lda,
                        qg_format w_fmt, const void *w_packed, size_t w_packed_bytes,
                        int64_t m, int64_t n, int64_t k,
                        void *y_codes, int64_t ldy, const float *y_scale, void *stream);

/*
 * qg_gemm_quant_nvfp4 -- qg_gemm whose epilogue writes the output quantized
 * to NVFP4 with a static (calibrated) tensor decode scale: the next linear's
 * 4-bit activation operand, produced without the bf16 round trip through
 * memory and without the three quantize kernels. Paper: Sec. 4, quantization
 * paragraph (NVFP4 activations for the low-precision linears; PTQ with
 * calibrated ranges).
 *   a_fmt ... k     as for qg_gemm; every pair but the weight-only one
 *                   (BF16, NVFP4), which returns QG_ERR_UNSUPPORTED.
 *   y_codes         out: rows of ldy/2 bytes, two E2M1 codes per byte
 *                   (element 2i in the low nibble); 4-byte aligned.
 *   y_block_scales  out: rows of ldy/16 bytes, one E4M3 scale per 16
 *                   consecutive elements of a row.
 *   ldy             elements between rows, >= n, ldy % 16 == 0 (as a W4A4
 *                   activation operand of a later qg_gemm, the rows then
 *                   need lda = ldy % 128 == 0, or ldy = n dense).
 *   y_tensor_scale  in: device fp32 tensor decode scale s_t of the output,
 *                   0 or >= 2^-96 (e.g. the scale qg_quantize_act derived for
 *                   calibration data); not written.
 * Result: the static NVFP4 quantization (qg_quantize_act_static) of the fp32
 * values y[i,j] that qg_gemm would round to its output type: per 16-block of
 * a row, s_b = E4M3(fl(max|y| / fl(6 s_t))), S = fl(e4m3(s_b) s_t),
 * r = S > 0 ? fl(1/S) : 0, q = E2M1(fl(y r)) (round to nearest even,
 * saturating). With the accuracy contract of qg_gemm, every block scale and
 * code is a correct rounding for some output within that contract's error of
 * the exact product.
 */
qg_status qg_gemm_quant_nvfp4(qg_format a_fmt, const void *a, const void *a_block_scales,
                              const float *a_tensor_scale, int64_t lda,
                              qg_format w_fmt, const void *w_packed, size_t w_packed_bytes,
                              int64_t m, int64_t n, int64_t k,
                              void *y_codes, void *y_block_scales, int64_t ldy,
                              const float *y_tensor_scale, void *stream);

/*
 * qg_dequant -- decode a quantized tensor to bf16 or fp32.
 * Paper: Sec. 4, quantization paragraph (the value a code stands for in each
 * cited format: the decode side of the quantizers above).
 *   FP8  : out = fl(e4m3(q) * s)
 *   NVFP4: out = fl(fl(e2m1(q) * e4m3(s_b)) * s_t)   (the inner product is exact)
 *   MX   : out = e2m1 / e4m3(q) * 2^(e-127)                  (exact in fp32)
 * bf16 output is the RNE rounding of that fp32 value. out is dense
 * [rows, cols]. NVFP4 needs cols % 16 == 0. MX needs cols % 32 == 0, a NULL
 * tensor_scale, 16-byte aligned out and codes aligned to 4 (MXFP4) or 8
 * (MXFP8) bytes.
 */
qg_status qg_dequant(qg_format fmt, const void *codes, const void *block_scales,
                     const float *tensor_scale, int64_t rows, int64_t cols,
                     void *out, qg_out_dtype out_dtype, void *stream);

/*
 * ---------------------------------------------------------------- weight streaming
 * Paper: Sec. 4, weight-streaming paragraph. A resident subset of the layer
 * weights stays in device memory; the other packed weights live in pinned
 * host memory and are copied into a few device buffers ("slots") ahead of
 * their GEMM, on a copy stream, so that the copies overlap the compute. Only
 * where the weight bytes come from changes: the outputs are bit-identical to
 * a run with every weight resident. The paper's model of the cost:
 *   lambda = L * M / W   (L: compute time between successive GEMMs, M: the
 *                         host-to-device rate, W: the layer's weight bytes);
 *   lambda >= 1 hides every copy; lambda < 1 adds up to Delta = (N-K) W / M
 *   (N layers, K overlapped); device memory cannot go below
 *   T_min = 2 W_max + A_max (two slots of the largest streamed layer plus
 *   the peak activation).
 */

/* One linear of a streamed run: optional activation quantization, then the
 * GEMM. Field meanings are those of qg_quantize_act and qg_gemm. */
typedef struct qg_stream_layer {
    const void *x;            /* bf16 [m, k] dense input (lda = k) */
    qg_format a_fmt;          /* BF16: x is the GEMM operand; else x is quantized first */
    void *a_codes;            /* quantize outputs (device), unused for BF16 */
    void *a_block_scales;
    float *a_tensor_scale;    /* NULL for MXFP4 */
    qg_format w_fmt;
    const void *w_packed;     /* resident: device buffer; streamed: host buffer (pinned for overlap) */
    size_t w_packed_bytes;
    int32_t resident;         /* nonzero: w_packed is device memory used in place */
    int64_t m, n, k;
    void *y;                  /* [m, n] output, ldy = n */
    qg_out_dtype y_dtype;
} qg_stream_layer;

/*
 * qg_run_layers -- enqueue one pass over `layers` in order. For every layer:
 * (quantize x on compute_stream), then, if it is streamed, the copy of its
 * packed weight into slot s = *slot_cursor (then s + 1 mod n_slots) on
 * copy_stream after slot_free[s] (the slot's previous GEMM), followed by
 * slot_ready[s]; the GEMM waits for slot_ready[s] on compute_stream and
 * records slot_free[s]. Nothing waits on the host.
 *   slots       n_slots device buffers of slot_bytes each, 256-byte aligned
 *               (slot_bytes >= every streamed layer's w_packed_bytes).
 *   slot_ready, slot_free  n_slots hipEvent_t each, created by the caller
 *               (hipEventDisableTiming is fine) and reused across calls.
 *   slot_cursor in/out: the slot the first streamed layer takes; repeated
 *               calls (one per step) keep the round robin going.
 *   compute_stream, copy_stream  hipStream_t (distinct for overlap).
 * Every layer's arguments are checked before anything is enqueued, with the
 * checks and status codes of qg_quantize_act and qg_gemm. n_slots must be
 * >= 1 when a layer is streamed.
 */
qg_status qg_run_layers(const qg_stream_layer *layers, int32_t n_layers,
                        void *const *slots, int32_t n_slots, size_t slot_bytes,
                        void *const *slot_ready, void *const *slot_free, int32_t *slot_cursor,
                        void *compute_stream, void *copy_stream);

/*
 * qg_stream_simulate -- the schedule qg_run_layers enqueues, as a
 * discrete-event model: layers in order, `steps` passes; the streamed
 * occurrences take the n_slots slots in turn; one copy engine at
 * h2d_bytes_per_s serves the copies in order; a copy starts once its slot's
 * previous layer has computed; a layer computes once the previous one has
 * finished and its weight is in place (compute_s[i] seconds).
 *   step_s  out: the duration of the last pass (the steady state for
 *           steps >= 3).
 * Pure host arithmetic (no GPU).
 */
qg_status qg_stream_simulate(int32_t n_layers, const double *w_bytes, const double *compute_s,
                             const uint8_t *resident, int32_t n_slots, double h2d_bytes_per_s,
                             int32_t steps, double *step_s);

/*
 * qg_stream_plan -- choose the resident layers for a device memory budget.
 * Device bytes of a plan = resident weights + n_slots x the largest streamed
 * weight + act_peak_bytes. The plan minimises the simulated step time
 * (qg_stream_simulate, 3 passes), then the device bytes: over every resident
 * subset for up to 16 layers; for more layers, for each slot size (every
 * layer above it resident) layers are made resident greedily by step time
 * saved per byte while they fit and copies are still exposed.
 *   resident_out  n_layers flags; step_s, device_bytes: of the chosen plan.
 * QG_ERR_BUFFER_TOO_SMALL when no plan fits (budget below T_min and below
 * the all-resident size). Pure host arithmetic (no GPU).
 */
qg_status qg_stream_plan(int32_t n_layers, const double *w_bytes, const double *compute_s, int32_t n_slots,
                         double h2d_bytes_per_s, double budget_bytes, double act_peak_bytes,
                         uint8_t *resident_out, double *step_s, double *device_bytes);

/* Human-readable name of a status code (static storage, never NULL). */
const char *qg_status_string(qg_status s);

/* The HIP error code behind the most recent QG_ERR_HIP on this thread (0 if none). */
int qg_last_hip_error(void);

/* QG_ABI_VERSION of the built library. */
int qg_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* QGEMM_H */

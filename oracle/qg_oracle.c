/*
 * qg_oracle.c -- CPU oracle for the low-bit quantized-linear hot path.
 *
 * TEST INFRASTRUCTURE ONLY. The product library neither includes, links nor
 * calls anything here; only the tests, the smoke check and the benchmark's
 * CPU-baseline leg load it. It shares no code, header, table or constant
 * generator with the HIP path.
 *
 * What it computes follows Sec. 4 of the paper ("Speed/Quality/Memory
 * Recipe", paragraph on quantization): post-training quantization of the
 * denoising transformer's weights AND activations to FP8 or NVFP4 so that
 * its linears run on low-precision matrix units (Table 2 gives the effect).
 * The formats are the two the paper cites there:
 *   FP8 E4M3 [Micikevicius et al. 2022]: 1 sign, 4 exponent bits (bias 7),
 *     3 mantissa bits, no infinities, NaN = S.1111.111, largest finite 448;
 *     used with one fp32 scale per tensor.
 *   NVFP4 [NVIDIA 2025]: E2M1 elements (values 0, .5, 1, 1.5, 2, 3, 4, 6 and
 *     their negatives) in blocks of 16 consecutive elements, each block with
 *     an E4M3 scale, plus one fp32 scale for the whole tensor.
 * Where the paper and its citations leave a step open (rounding of scales,
 * the tensor-scale constant, the exact fp32 operation order) the reading
 * used here is written next to the step and listed in the design notes.
 *
 * Precision: every step that the format definitions fix in fp32 is done as
 * one IEEE binary32 operation with round-to-nearest-even (build with
 * -ffp-contract=off, no -ffast-math, SSE arithmetic). Dequantized values are
 * exact in binary64, and the GEMM accumulates in binary64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define QO_OK 0
#define QO_ERR_NONFINITE 6
#define QO_ERR_SHAPE 3

/* ------------------------------------------------------------------ */
/* Codecs                                                             */
/* ------------------------------------------------------------------ */

/* E4M3 (OCP "fn" variant): value of an 8-bit code. */
double qo_e4m3_value(uint8_t code)
{
    int sign = code >> 7;
    int e = (code >> 3) & 15;
    int m = code & 7;
    double mag;
    if (e == 15 && m == 7)
        return NAN;
    if (e == 0)
        mag = ldexp((double)m / 8.0, -6);          /* subnormal: m/8 * 2^-6 */
    else
        mag = ldexp(1.0 + (double)m / 8.0, e - 7); /* normal: 1.m * 2^(e-7) */
    return sign ? -mag : mag;
}

/* E2M1: value of the low 4 bits of `code`. */
double qo_e2m1_value(uint8_t code)
{
    int sign = (code >> 3) & 1;
    int e = (code >> 1) & 3;
    int m = code & 1;
    double mag;
    if (e == 0)
        mag = 0.5 * m;                             /* subnormal: m * 0.5 */
    else
        mag = ldexp(1.0 + 0.5 * m, e - 1);         /* normal: 1.m * 2^(e-1) */
    return sign ? -mag : mag;
}

/*
 * Round-to-nearest-even onto the non-negative codes 0..max_code of a small
 * float format whose values increase with the code. Magnitudes at or above
 * the largest value saturate to it. A tie between two neighbours goes to the
 * even code (the one whose mantissa LSB is 0), which is what IEEE
 * round-half-to-even means for these formats. Comparing against the exact
 * midpoint (representable in binary64) keeps the decision exact.
 */
static int nearest_code(double a, int max_code, double (*value)(uint8_t))
{
    int lo = 0, hi = max_code;
    if (a >= value((uint8_t)max_code))
        return max_code;
    /* binary search for the largest code with value <= a */
    while (hi - lo > 1) {
        int mid = (lo + hi) / 2;
        if (value((uint8_t)mid) <= a)
            lo = mid;
        else
            hi = mid;
    }
    if (value((uint8_t)hi) <= a)
        return hi;
    {
        double vlo = value((uint8_t)lo), vhi = value((uint8_t)hi);
        double midpoint = 0.5 * (vlo + vhi);
        if (a < midpoint)
            return lo;
        if (a > midpoint)
            return hi;
        return (lo & 1) ? hi : lo;
    }
}

/* E4M3 encode of a finite fp32 value: RNE, saturating at 448, sign kept
 * (also for zero). NaN maps to the NaN code. */
uint8_t qo_e4m3_encode(float v)
{
    uint8_t sign = signbit(v) ? 0x80 : 0x00;
    if (isnan(v))
        return sign | 0x7F;
    return sign | (uint8_t)nearest_code(fabs((double)v), 0x7E, qo_e4m3_value);
}

/* E2M1 encode of a finite fp32 value: RNE, saturating at 6, sign kept. */
uint8_t qo_e2m1_encode(float v)
{
    uint8_t sign = signbit(v) ? 0x8 : 0x0;
    if (isnan(v))
        return sign | 0x7;
    return sign | (uint8_t)nearest_code(fabs((double)v), 7, qo_e2m1_value);
}

/* Array forms of the two encoders (used to test them on many inputs). */
void qo_e4m3_encode_array(const float *v, int64_t n, uint8_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = qo_e4m3_encode(v[i]);
}

void qo_e2m1_encode_array(const float *v, int64_t n, uint8_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = qo_e2m1_encode(v[i]);
}

static float bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* fp32 -> bf16 bits, round-to-nearest-even (NaN -> canonical quiet NaN). */
uint16_t qo_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        return 0x7FC0;
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

/* max |x| over a bf16 matrix; returns 0 when every element is finite. */
static int tensor_amax(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx, float *amax)
{
    float a = 0.0f;
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t c = 0; c < cols; ++c) {
            float v = fabsf(bf16_to_f32(x[r * ldx + c]));
            if (!isfinite(v))
                return QO_ERR_NONFINITE;
            if (v > a)
                a = v;
        }
    *amax = a;
    return QO_OK;
}

/* ------------------------------------------------------------------ */
/* FP8 E4M3 quantization with one per-tensor scale                    */
/* ------------------------------------------------------------------ */
/*
 * Steps (dynamic per-tensor scaling of a bf16 tensor, weights and
 * activations alike):
 *   a = max |x|                       (exact)
 *   s = fl(a / 448)                   decode scale: x ~ dec(q) * s
 *   r = s > 0 ? fl(1 / s) : 0         one correctly rounded reciprocal
 *   q = E4M3_RNE_sat(fl(x * r))
 * Output: codes [rows, cols] row-major, and s.
 */
/* The element step of FP8 quantization with a given decode scale s:
 * r = s > 0 ? fl(1/s) : 0;  q = E4M3_RNE_sat(fl(x * r)). */
static void quantize_fp8_core(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                              float s, uint8_t *codes)
{
    float r = (s > 0.0f) ? 1.0f / s : 0.0f;
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t c = 0; c < cols; ++c) {
            float y = bf16_to_f32(x[i * ldx + c]) * r;
            codes[i * cols + c] = qo_e4m3_encode(y);
        }
}

int qo_quantize_fp8(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                    uint8_t *codes, float *scale_out)
{
    float amax, s;
    int st = tensor_amax(x, rows, cols, ldx, &amax);
    if (st != QO_OK)
        return st;
    s = amax / 448.0f;
    quantize_fp8_core(x, rows, cols, ldx, s, codes);
    *scale_out = s;
    return QO_OK;
}

/*
 * Static (calibrated) scales: the decode scale comes from calibration data
 * instead of the tensor itself (post-training quantization with fixed
 * activation ranges). The element step is the one above; values beyond the
 * calibrated range saturate. The scale must be 0 or a normal positive fp32
 * (so that 1/s is finite); inputs must be finite.
 */
#define QO_ERR_INVALID 1
static int scale_ok(float s, float min_normal)
{
    return s == 0.0f || (isfinite(s) && s >= min_normal);
}

int qo_quantize_fp8_static(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                           float s, uint8_t *codes)
{
    float amax;
    int st;
    if (!scale_ok(s, 0x1p-126f))
        return QO_ERR_INVALID;
    st = tensor_amax(x, rows, cols, ldx, &amax);  /* finiteness check only */
    if (st != QO_OK)
        return st;
    quantize_fp8_core(x, rows, cols, ldx, s, codes);
    return QO_OK;
}

/* ------------------------------------------------------------------ */
/* NVFP4 quantization: E2M1 elements, E4M3 scale per 16, fp32 tensor  */
/* ------------------------------------------------------------------ */
/*
 * Two-level scaling of a bf16 tensor whose blocks are 16 consecutive
 * elements along a row (the reduction dimension K of a linear):
 *   a_t = max |x|
 *   s_t = fl(a_t / 2688)              2688 = 448 * 6: the largest block lands
 *                                      on the largest E4M3 scale value
 *   d_t = fl(6 * s_t)
 *   per block b: a_b = max |x| over the block
 *                v_b = d_t > 0 ? fl(a_b / d_t) : 0
 *                s_b = E4M3_RNE_sat(v_b)            (stored block scale)
 *                S   = fl(dec(s_b) * s_t)           (effective block scale)
 *                r   = S > 0 ? fl(1 / S) : 0
 *                q_k = E2M1_RNE_sat(fl(x_k * r))
 * Codes are packed two per byte, element 2i in the low nibble.
 * Outputs: codes [rows, cols/2], block scales [rows, cols/16], s_t.
 */
/* The block and element steps of NVFP4 quantization with a given tensor
 * decode scale s_t (everything after the tensor amax above). */
static void quantize_nvfp4_core(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                                float s_t, uint8_t *codes, uint8_t *block_scales)
{
    float d_t = 6.0f * s_t;
    for (int64_t i = 0; i < rows; ++i) {
        for (int64_t b = 0; b < cols / 16; ++b) {
            const uint16_t *xb = x + i * ldx + b * 16;
            float a_b = 0.0f, v_b, S, r;
            uint8_t s_b;
            for (int t = 0; t < 16; ++t) {
                float v = fabsf(bf16_to_f32(xb[t]));
                if (v > a_b)
                    a_b = v;
            }
            v_b = (d_t > 0.0f) ? a_b / d_t : 0.0f;
            s_b = qo_e4m3_encode(v_b);
            S = (float)qo_e4m3_value(s_b) * s_t;
            r = (S > 0.0f) ? 1.0f / S : 0.0f;
            block_scales[i * (cols / 16) + b] = s_b;
            for (int t = 0; t < 16; t += 2) {
                uint8_t lo = qo_e2m1_encode(bf16_to_f32(xb[t]) * r);
                uint8_t hi = qo_e2m1_encode(bf16_to_f32(xb[t + 1]) * r);
                codes[i * (cols / 2) + b * 8 + t / 2] = (uint8_t)(lo | (hi << 4));
            }
        }
    }
}

int qo_quantize_nvfp4(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                      uint8_t *codes, uint8_t *block_scales, float *tscale_out)
{
    float amax, s_t;
    int st;
    if (cols % 16 != 0)
        return QO_ERR_SHAPE;
    st = tensor_amax(x, rows, cols, ldx, &amax);
    if (st != QO_OK)
        return st;
    s_t = amax / 2688.0f;
    quantize_nvfp4_core(x, rows, cols, ldx, s_t, codes, block_scales);
    *tscale_out = s_t;
    return QO_OK;
}

/* Static tensor scale (see qo_quantize_fp8_static): s_t must be 0 or at
 * least 2^-96, which keeps every effective block scale's reciprocal finite. */
int qo_quantize_nvfp4_static(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                             float s_t, uint8_t *codes, uint8_t *block_scales)
{
    float amax;
    int st;
    if (cols % 16 != 0)
        return QO_ERR_SHAPE;
    if (!scale_ok(s_t, 0x1p-96f))
        return QO_ERR_INVALID;
    st = tensor_amax(x, rows, cols, ldx, &amax);  /* finiteness check only */
    if (st != QO_OK)
        return st;
    quantize_nvfp4_core(x, rows, cols, ldx, s_t, codes, block_scales);
    return QO_OK;
}

/*
 * The same block and element steps on fp32 values with a static tensor
 * decode scale: the NVFP4 quantization of a GEMM's fp32 output (before any
 * rounding to bf16), which a fused epilogue performs to hand the next
 * linear its 4-bit activation. Identical to quantize_nvfp4_core except
 * that the element values are read as fp32 (a bf16 value widened to fp32
 * gives the same codes). s_t must be 0 or at least 2^-96; inputs finite.
 */
int qo_quantize_nvfp4_static_f32(const float *x, int64_t rows, int64_t cols, int64_t ldx,
                                 float s_t, uint8_t *codes, uint8_t *block_scales)
{
    float d_t;
    if (cols % 16 != 0)
        return QO_ERR_SHAPE;
    if (!scale_ok(s_t, 0x1p-96f))
        return QO_ERR_INVALID;
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t k = 0; k < cols; ++k)
            if (!isfinite(x[i * ldx + k]))
                return QO_ERR_NONFINITE;
    d_t = 6.0f * s_t;
    for (int64_t i = 0; i < rows; ++i) {
        for (int64_t b = 0; b < cols / 16; ++b) {
            const float *xb = x + i * ldx + b * 16;
            float a_b = 0.0f, v_b, S, r;
            uint8_t s_b;
            for (int t = 0; t < 16; ++t) {
                float v = fabsf(xb[t]);
                if (v > a_b)
                    a_b = v;
            }
            v_b = (d_t > 0.0f) ? a_b / d_t : 0.0f;
            s_b = qo_e4m3_encode(v_b);
            S = (float)qo_e4m3_value(s_b) * s_t;
            r = (S > 0.0f) ? 1.0f / S : 0.0f;
            block_scales[i * (cols / 16) + b] = s_b;
            for (int t = 0; t < 16; t += 2) {
                uint8_t lo = qo_e2m1_encode(xb[t] * r);
                uint8_t hi = qo_e2m1_encode(xb[t + 1] * r);
                codes[i * (cols / 2) + b * 8 + t / 2] = (uint8_t)(lo | (hi << 4));
            }
        }
    }
    return QO_OK;
}

/* ------------------------------------------------------------------ */
/* MX formats (OCP Microscaling v1.0): the matrix-core-native block    */
/* scaling of gfx950, a variant beside the paper's NVFP4               */
/* ------------------------------------------------------------------ */
/*
 * Blocks of 32 consecutive elements along a row share one E8M0 scale (an
 * 8-bit power-of-two exponent, bias 127: value 2^(e - 127); 255 = NaN is
 * never produced); there is no tensor scale. Per the OCP Microscaling
 * Formats specification, section on conversion:
 *   a_b = max |x| over the block
 *   shared exponent E = floor(log2(a_b)) - emax_elem, where emax_elem is the
 *     exponent of the element format's largest normal number: 2 for E2M1
 *     (6 = 1.5 * 2^2), 8 for E4M3 (448 = 1.75 * 2^8)
 *   e = E + 127 clamped to [0, 254] (e = 0 for an all-zero block)
 *   q_k = element_RNE_sat(x_k / 2^(e - 127))
 * Readings where the specification leaves a choice: values above the
 * element format's largest normal saturate to it (E2M1 has no inf/NaN;
 * for E4M3 the same saturation as the FP8 recipe), ties round to the even
 * code, an all-zero block gets e = 0. Division by the power of two is exact
 * (bf16 inputs keep x / 2^(e-127) inside the binary32 normal range).
 * Outputs: codes (MXFP4: two per byte, element 2i in the low nibble;
 * MXFP8: one E4M3 byte per element) and E8M0 scales [rows, cols/32].
 */
double qo_e8m0_value(uint8_t e)
{
    if (e == 255)
        return NAN;
    return ldexp(1.0, (int)e - 127);
}

static uint8_t mx_scale_code(float a_b, int emax_elem)
{
    int ex, e;
    if (a_b == 0.0f)
        return 0;
    frexpf(a_b, &ex);          /* a_b = f * 2^ex, f in [0.5, 1): floor(log2 a_b) = ex - 1 */
    e = (ex - 1) - emax_elem + 127;
    if (e < 0)
        e = 0;
    if (e > 254)
        e = 254;
    return (uint8_t)e;
}

static int quantize_mx(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                       int fp4, uint8_t *codes, uint8_t *scales)
{
    float amax;
    int st;
    if (cols % 32 != 0)
        return QO_ERR_SHAPE;
    st = tensor_amax(x, rows, cols, ldx, &amax);  /* finiteness check only */
    if (st != QO_OK)
        return st;
    for (int64_t i = 0; i < rows; ++i) {
        for (int64_t b = 0; b < cols / 32; ++b) {
            const uint16_t *xb = x + i * ldx + b * 32;
            float a_b = 0.0f;
            uint8_t e;
            for (int t = 0; t < 32; ++t) {
                float v = fabsf(bf16_to_f32(xb[t]));
                if (v > a_b)
                    a_b = v;
            }
            e = mx_scale_code(a_b, fp4 ? 2 : 8);
            scales[i * (cols / 32) + b] = e;
            for (int t = 0; t < 32; ++t) {
                float y = ldexpf(bf16_to_f32(xb[t]), 127 - (int)e);
                if (fp4) {
                    uint8_t q = qo_e2m1_encode(y);
                    uint8_t *dst = &codes[i * (cols / 2) + b * 16 + t / 2];
                    if (t & 1)
                        *dst = (uint8_t)((*dst & 0x0F) | (q << 4));
                    else
                        *dst = q;
                } else {
                    codes[i * cols + b * 32 + t] = qo_e4m3_encode(y);
                }
            }
        }
    }
    return QO_OK;
}

int qo_quantize_mxfp4(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                      uint8_t *codes, uint8_t *scales)
{
    return quantize_mx(x, rows, cols, ldx, 1, codes, scales);
}

int qo_quantize_mxfp8(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                      uint8_t *codes, uint8_t *scales)
{
    return quantize_mx(x, rows, cols, ldx, 0, codes, scales);
}

/* Exact values (binary64): x = element(q) * 2^(e - 127). */
void qo_dequant_mxfp4_f64(const uint8_t *codes, const uint8_t *scales, int64_t rows, int64_t cols,
                          double *out)
{
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t c = 0; c < cols; ++c) {
            uint8_t byte = codes[i * (cols / 2) + c / 2];
            uint8_t q = (c & 1) ? (byte >> 4) : (byte & 15);
            out[i * cols + c] = qo_e2m1_value(q) * qo_e8m0_value(scales[i * (cols / 32) + c / 32]);
        }
}

void qo_dequant_mxfp8_f64(const uint8_t *codes, const uint8_t *scales, int64_t rows, int64_t cols,
                          double *out)
{
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t c = 0; c < cols; ++c)
            out[i * cols + c] = qo_e4m3_value(codes[i * cols + c]) * qo_e8m0_value(scales[i * (cols / 32) + c / 32]);
}

/* ------------------------------------------------------------------ */
/* Dequantization                                                     */
/* ------------------------------------------------------------------ */
/* Exact values (binary64): FP8 x = dec(q) * s. */
void qo_dequant_fp8_f64(const uint8_t *codes, int64_t n, float scale, double *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = qo_e4m3_value(codes[i]) * (double)scale;
}

/* Exact values (binary64): NVFP4 x = dec_e2m1(q) * dec_e4m3(s_b) * s_t. */
void qo_dequant_nvfp4_f64(const uint8_t *codes, const uint8_t *block_scales,
                          int64_t rows, int64_t cols, float tscale, double *out)
{
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t c = 0; c < cols; ++c) {
            uint8_t byte = codes[i * (cols / 2) + c / 2];
            uint8_t q = (c & 1) ? (byte >> 4) : (byte & 15);
            double sb = qo_e4m3_value(block_scales[i * (cols / 16) + c / 16]);
            out[i * cols + c] = qo_e2m1_value(q) * sb * (double)tscale;
        }
}

/* fp32 output of dequantization: the exact value above rounded once to
 * binary32 (the element-times-block-scale product is exact in binary32, so
 * this equals fl(fl(e2m1 * e4m3) * s_t) and fl(e4m3 * s)). */
void qo_dequant_fp8_f32(const uint8_t *codes, int64_t n, float scale, float *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = (float)(qo_e4m3_value(codes[i]) * (double)scale);
}

void qo_dequant_nvfp4_f32(const uint8_t *codes, const uint8_t *block_scales,
                          int64_t rows, int64_t cols, float tscale, float *out)
{
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t c = 0; c < cols; ++c) {
            uint8_t byte = codes[i * (cols / 2) + c / 2];
            uint8_t q = (c & 1) ? (byte >> 4) : (byte & 15);
            double sb = qo_e4m3_value(block_scales[i * (cols / 16) + c / 16]);
            out[i * cols + c] = (float)(qo_e2m1_value(q) * sb * (double)tscale);
        }
}

/* bf16 output of dequantization: RNE of the fp32 output. */
void qo_f32_to_bf16_array(const float *in, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = qo_f32_to_bf16(in[i]);
}

void qo_bf16_to_f64(const uint16_t *in, int64_t n, double *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = (double)bf16_to_f32(in[i]);
}

/* ------------------------------------------------------------------ */
/* Linear layer: Y = A . W^T on dequantized operands                   */
/* ------------------------------------------------------------------ */
/*
 * y[m,n] = sum_k a[m,k] * w[n,k] accumulated in binary64 over the exact
 * dequantized operands, together with the magnitude sum
 * b[m,n] = sum_k |a[m,k] * w[n,k]| that bounds the admissible error of a
 * device result (|y_dev - y| <= 1e-3 * b). Rows are independent and are
 * spread over OpenMP threads; each (m, n) is one plain loop over k.
 */
void qo_gemm_f64(const double *a, const double *w, int64_t m, int64_t n, int64_t k,
                 double *y, double *babs)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j) {
            double acc = 0.0, mag = 0.0;
            for (int64_t t = 0; t < k; ++t) {
                double p = a[i * k + t] * w[j * k + t];
                acc += p;
                mag += fabs(p);
            }
            y[i * n + j] = acc;
            if (babs)
                babs[i * n + j] = mag;
        }
}

/* Same as qo_gemm_f64 for a list of (row, column) pairs only, for outputs
 * of full-size problems where the whole product is out of reach. */
void qo_gemm_f64_sampled(const double *a, const double *w, int64_t k,
                         const int64_t *rows, const int64_t *colsn, int64_t count,
                         double *y, double *babs)
{
#pragma omp parallel for schedule(static)
    for (int64_t s = 0; s < count; ++s) {
        const double *ar = a + rows[s] * k;
        const double *wr = w + colsn[s] * k;
        double acc = 0.0, mag = 0.0;
        for (int64_t t = 0; t < k; ++t) {
            double p = ar[t] * wr[t];
            acc += p;
            mag += fabs(p);
        }
        y[s] = acc;
        babs[s] = mag;
    }
}

int qo_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Thread count of the parallel loops above (timing of the CPU baseline in
 * single-thread and all-core modes; the results do not depend on it). */
void qo_set_num_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}

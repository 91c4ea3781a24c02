/* Drives every entry point of the CPU oracle (oracle/qg_oracle.c, compiled
 * into this program) over small tensors with padded rows, random bf16 bit
 * patterns across the whole finite range, zeros, the extremes and a
 * non-finite input, so that a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer sees every loop and every branch of the codecs.
 * Exits 0 when every call returns the expected status; the sanitizers abort
 * on the first finding. Test infrastructure, built and run by
 * tests/test_oracle_sanitize.py. */
#include "../../oracle/qg_oracle.c"

#include <math.h>
#include <stdio.h>
#include <stdlib.h>

static uint64_t lcg = 0x243F6A8885A308D3ull;
static uint16_t rand_finite_bf16(void) {
    for (;;) {
        lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
        const uint16_t b = (uint16_t)(lcg >> 48);
        if (((b >> 7) & 0xFF) != 0xFF) return b;  /* exponent all ones: inf or NaN */
    }
}

static int fail(const char *what, int got, int want) {
    fprintf(stderr, "%s: status %d, expected %d\n", what, got, want);
    return 1;
}

int main(void) {
    const int64_t rows = 7, cols = 96, ldx = 100;  /* cols % 32 == 0; rows padded to ldx */
    uint16_t *x = malloc(sizeof(uint16_t) * rows * ldx);
    uint8_t *c8 = malloc(rows * cols), *c4 = malloc(rows * cols / 2);
    uint8_t *bs = malloc(rows * cols / 16), *ms = malloc(rows * cols / 32);
    double *d = malloc(sizeof(double) * rows * cols);
    float *f = malloc(sizeof(float) * rows * cols);
    uint8_t e[256];
    float s = 0.0f;
    int bad = 0;
    double sum = 0.0;

    for (int c = 0; c < 256; ++c)
        if (c != 0x7F && c != 0xFF) sum += qo_e4m3_value((uint8_t)c);  /* 0x7F, 0xFF: NaN */
    for (int c = 0; c < 16; ++c) sum += qo_e2m1_value((uint8_t)c);
    for (int c = 0; c < 255; ++c) sum += qo_e8m0_value((uint8_t)c) > 0.0;
    for (int c = 0; c < 256; ++c) f[c] = (float)(c - 128) * 3.7f;
    qo_e4m3_encode_array(f, 256, e);
    qo_e2m1_encode_array(f, 256, e);

    for (int pass = 0; pass < 4; ++pass) {
        for (int64_t i = 0; i < rows * ldx; ++i) x[i] = rand_finite_bf16();
        if (pass == 1) for (int64_t i = 0; i < rows * ldx; ++i) x[i] &= 0x80FF;     /* tiny and subnormal */
        if (pass == 2) for (int64_t i = 0; i < rows * ldx; ++i) x[i] = (i % 3) ? 0x0000 : 0x8000;  /* signed zeros */
        if (pass == 3) { x[5] = 0x7F7F; x[6] = 0xFF7F; x[7] = 0x0001; }          /* extremes */
        int st;
        if ((st = qo_quantize_fp8(x, rows, cols, ldx, c8, &s))) bad |= fail("fp8", st, 0);
        qo_dequant_fp8_f64(c8, rows * cols, s, d);
        qo_dequant_fp8_f32(c8, rows * cols, s, f);
        /* a static scale is 0 or at least 2^-126 (FP8) / 2^-96 (NVFP4); the
           dynamic scale of the tiny-value pass falls below and is rejected */
        int want = (s == 0.0f || s >= 0x1p-126f) ? 0 : 1;
        if ((st = qo_quantize_fp8_static(x, rows, cols, ldx, s, c8)) != want) bad |= fail("fp8 static", st, want);
        if ((st = qo_quantize_nvfp4(x, rows, cols, ldx, c4, bs, &s))) bad |= fail("nvfp4", st, 0);
        qo_dequant_nvfp4_f64(c4, bs, rows, cols, s, d);
        qo_dequant_nvfp4_f32(c4, bs, rows, cols, s, f);
        want = (s == 0.0f || s >= 0x1p-96f) ? 0 : 1;
        if ((st = qo_quantize_nvfp4_static(x, rows, cols, ldx, s, c4, bs)) != want) bad |= fail("nvfp4 static", st, want);
        if ((st = qo_quantize_mxfp4(x, rows, cols, ldx, c4, ms))) bad |= fail("mxfp4", st, 0);
        qo_dequant_mxfp4_f64(c4, ms, rows, cols, d);
        if ((st = qo_quantize_mxfp8(x, rows, cols, ldx, c8, ms))) bad |= fail("mxfp8", st, 0);
        qo_dequant_mxfp8_f64(c8, ms, rows, cols, d);
        for (int64_t i = 0; i < rows * cols; ++i) sum += isfinite(d[i]) ? d[i] : 0.0;
    }
    /* non-finite input: every quantizer reports it */
    x[3 * ldx + 17] = 0x7F80;
    int st;
    if ((st = qo_quantize_fp8(x, rows, cols, ldx, c8, &s)) != 6) bad |= fail("fp8 inf", st, 6);
    if ((st = qo_quantize_nvfp4(x, rows, cols, ldx, c4, bs, &s)) != 6) bad |= fail("nvfp4 inf", st, 6);
    if ((st = qo_quantize_mxfp4(x, rows, cols, ldx, c4, ms)) != 6) bad |= fail("mxfp4 inf", st, 6);
    x[3 * ldx + 17] = 0x7FC1;
    if ((st = qo_quantize_mxfp8(x, rows, cols, ldx, c8, ms)) != 6) bad |= fail("mxfp8 nan", st, 6);

    /* fp64 products, full and sampled */
    const int64_t m = 5, n = 7, k = 33;
    double *a = malloc(sizeof(double) * m * k), *w = malloc(sizeof(double) * n * k);
    double *y = malloc(sizeof(double) * m * n), *b = malloc(sizeof(double) * m * n);
    for (int64_t i = 0; i < m * k; ++i) a[i] = (double)((i * 37) % 11) - 5.0;
    for (int64_t i = 0; i < n * k; ++i) w[i] = (double)((i * 53) % 13) * 0.25 - 1.5;
    qo_gemm_f64(a, w, m, n, k, y, b);
    int64_t rr[3] = {0, 4, 2}, cc[3] = {6, 0, 3};
    double ys[3], bs3[3];
    qo_gemm_f64_sampled(a, w, k, rr, cc, 3, ys, bs3);
    for (int i = 0; i < 3; ++i)
        if (ys[i] != y[rr[i] * n + cc[i]] || bs3[i] != b[rr[i] * n + cc[i]]) { fprintf(stderr, "sampled %d\n", i); bad = 1; }
    uint16_t hb[4];
    const float hv[4] = {1.0f, -3.25f, 1e-40f, 65504.0f};
    for (int i = 0; i < 4; ++i) hb[i] = qo_f32_to_bf16(hv[i]);
    qo_f32_to_bf16_array(hv, 4, hb);
    qo_bf16_to_f64(hb, 4, d);
    printf("oracle sanitizer run done (checksum %.6g, threads %d)\n", sum + d[0], qo_num_threads());
    free(x); free(c8); free(c4); free(bs); free(ms); free(d); free(f); free(a); free(w); free(y); free(b);
    return bad;
}

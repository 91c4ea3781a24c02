"""GPU parity of qg_gemm with the CPU oracle: every output (or, at the full
transformer sizes, a large sample of outputs including the tile edges)
within |y - y_ref| <= 1e-3 * sum_k |a w| of the oracle's fp64 product over
the same quantized operands. Codes of both operands are checked bit-exact
on the way."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_21849_amd as q
import synth
from gpu_util import DEV, assert_quant_equal, check_linear, host, log, to_dev_bf16

pytestmark = pytest.mark.gpu

FP8, NVFP4, BF16 = q.QG_FMT_FP8_E4M3, q.QG_FMT_NVFP4, q.QG_FMT_BF16
KINDS = {"fp8": (FP8, FP8), "nvfp4": (NVFP4, NVFP4), "w4a16": (BF16, NVFP4)}


def run_linear(kind, x, w, out=q.QG_OUT_BF16, check_codes=True):
    a_fmt, w_fmt = KINDS[kind]
    xd, wd = to_dev_bf16(x), to_dev_bf16(w)
    wq = q.quantize(wd, w_fmt)
    packed = q.pack(wq)
    a = xd if a_fmt == BF16 else q.quantize(xd, a_fmt)
    y = q.linear(a, packed, w_fmt, w.shape[0], out_dtype=out)
    torch.cuda.synchronize()
    if check_codes:
        assert_quant_equal(wq, w)
        if a_fmt != BF16:
            assert_quant_equal(a, x)
    return y


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "w4a16"])
@pytest.mark.parametrize("m,n,k", [(1, 16, 128), (17, 48, 256), (64, 256, 256), (65, 128, 128),
                                   (300, 272, 384), (257, 512, 1024), (512, 768, 640), (100, 2080, 384),
                                   (129, 528, 1152)])
@pytest.mark.parametrize("out", [q.QG_OUT_F32, q.QG_OUT_BF16])
def test_small_full_parity(kind, m, n, k, out):
    log("gemm kind=%s m=%d n=%d k=%d out=%d" % (kind, m, n, k, out))
    x = synth.normal_bf16(m, k, 1.0, 11, 0)
    w = synth.normal_bf16(n, k, 0.02, 11, 1)
    y = run_linear(kind, x, w, out)
    ref = oracle.linear_reference(kind, x, w)
    # few reduction terms (K = 128 ... 1152): bf16 outputs are held to the
    # rounding window (a correct rounding of a value within the bound)
    check_linear(y, ref, literal=False)


E2M1_VALUES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def _exact_operand(rows, k, kind, rng, one_hot):
    """Values the format represents exactly with power-of-two tensor scales.

    FP8   : amax 1.75 (activations) or 7 (weights) -> s = 2^-8 / 2^-6, and every
            value times 1/s is an E4M3 value.
    NVFP4 : every 16-block holds +-5.25 and otherwise E2M1 values times 0.875;
            a_t = 5.25 = 2688 * 2^-9 -> s_t = 2^-9, each block scale is 448.
    """
    v = np.zeros((rows, k))
    if kind == "fp8":
        if one_hot:
            for i in range(rows):
                for b in range(k // 16):
                    v[i, 16 * b + rng.integers(16)] = rng.choice([-1.75, 1.75])
        else:
            v = rng.integers(-7, 8, size=(rows, k)).astype(np.float64)
            v[:, 0] = 7.0
    else:
        for i in range(rows):
            for b in range(k // 16):
                if not one_hot:
                    v[i, 16 * b:16 * b + 16] = rng.choice(E2M1_VALUES, 16) * rng.choice([-1, 1], 16) * 0.875
                v[i, 16 * b + rng.integers(16)] = rng.choice([-5.25, 5.25])
    x = synth.f32_to_bf16_bits(v.astype(np.float32))
    assert np.array_equal(synth.bf16_bits_to_f32(x), v.astype(np.float32))
    return x


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "w4a16"])
def test_structured_exact(kind):
    """Operands whose quantization is exact and whose tensor scales are powers
    of two; X has one nonzero per 16-block. Every product and partial sum is
    exact in fp32, so the fp32 output must equal the oracle bit for bit
    (catches any transposition or shuffle of operand or output layouts)."""
    m, n, k = 48, 64, 256
    rng = np.random.default_rng(12)
    x = _exact_operand(m, k, "fp8" if kind == "fp8" else "nvfp4", rng, one_hot=True)
    w = _exact_operand(n, k, "fp8" if kind == "fp8" else "nvfp4", rng, one_hot=False)
    y = run_linear(kind, x, w, q.QG_OUT_F32)
    ref = oracle.linear_reference(kind, x, w)
    got = host(y).astype(np.float64)
    assert np.array_equal(got, ref["y"]), np.argwhere(got != ref["y"])[:5]


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "w4a16"])
def test_row_of_output_independent_of_batch(kind):
    """Row m of a 16-row product equals the 1-row product of that row."""
    x = synth.normal_bf16(16, 1024, 1.0, 13, 0)
    w = synth.normal_bf16(3072, 1024, 0.02, 13, 1)
    a_fmt, w_fmt = KINDS[kind]
    wq = q.quantize(to_dev_bf16(w), w_fmt)
    packed = q.pack(wq)
    xd = to_dev_bf16(x)
    if a_fmt == BF16:
        y16 = q.linear(xd, packed, w_fmt, 3072, out_dtype=q.QG_OUT_F32)
        y1 = q.linear(xd[5:6], packed, w_fmt, 3072, out_dtype=q.QG_OUT_F32)
        torch.cuda.synchronize()
        assert torch.allclose(y16[5], y1[0], rtol=1e-5, atol=1e-6)
    else:
        a = q.quantize(xd, a_fmt)
        y16 = q.linear(a, packed, w_fmt, 3072, out_dtype=q.QG_OUT_F32)
        torch.cuda.synchronize()
        ref = oracle.linear_reference(kind, x, w)
        check_linear(y16, ref)


def test_deterministic():
    x = synth.normal_bf16(300, 1024, 1.0, 14, 0)
    w = synth.normal_bf16(512, 1024, 0.02, 14, 1)
    for kind in ("fp8", "nvfp4", "w4a16"):
        y1 = run_linear(kind, x, w, check_codes=False)
        y2 = run_linear(kind, x, w, check_codes=False)
        assert torch.equal(y1, y2), kind


def test_zero_k_and_empty_m():
    w = torch.zeros((16, 0), dtype=torch.bfloat16, device=DEV)
    for fmt in (FP8, NVFP4):
        nbytes = q.qg_packed_bytes(fmt, 16, 0)
        packed = torch.zeros(nbytes, dtype=torch.uint8, device=DEV)
        ts = torch.ones(1, dtype=torch.float32, device=DEV)
        y = torch.full((3, 16), 7.0, dtype=torch.float32, device=DEV)
        a = torch.zeros(16, dtype=torch.uint8, device=DEV)
        bs = torch.zeros(16, dtype=torch.uint8, device=DEV)
        q.qg_gemm(fmt, a, bs if fmt == NVFP4 else None, ts, 0, fmt, packed, nbytes, 3, 16, 0, y, 16, q.QG_OUT_F32)
        torch.cuda.synchronize()
        assert torch.count_nonzero(y) == 0
    # m = 0: nothing written, no error
    wq = q.quantize(to_dev_bf16(synth.normal_bf16(16, 128, 0.02, 1, 1)), FP8)
    packed = q.pack(wq)
    empty = q.QTensor(FP8, torch.zeros((0, 128), dtype=torch.uint8, device=DEV), None,
                      torch.ones(1, device=DEV), 0, 128)
    y = q.linear(empty, packed, FP8, 16)
    torch.cuda.synchronize()
    assert y.shape == (0, 16)


# ---------------------------------------------------------------- workload sizes
def _sample(m, n, count, seed):
    rng = np.random.default_rng(seed)
    rows = np.concatenate([[0, m - 1, 0, m - 1], rng.integers(0, m, count)])
    cols = np.concatenate([[0, 0, n - 1, n - 1], rng.integers(0, n, count)])
    return rows, cols


def test_single_fp8_linear_full():
    x = synth.normal_bf16(128, 256, 1.0, 0, 0)
    w = synth.normal_bf16(256, 256, 0.02, 0, 1)
    y = run_linear("fp8", x, w)
    log("fp8 128x256x256 max err/B", check_linear(y, oracle.linear_reference("fp8", x, w),
                                                  name="C1 fp8 w8a8 128x256x256 (every output)"))


def test_single_fp8_linear_full_f32():
    # the same configuration with fp32 output: the bound without any output rounding
    x = synth.normal_bf16(128, 256, 1.0, 0, 0)
    w = synth.normal_bf16(256, 256, 0.02, 0, 1)
    y = run_linear("fp8", x, w, q.QG_OUT_F32, check_codes=False)
    log("fp8 128x256x256 f32 max err/B", check_linear(y, oracle.linear_reference("fp8", x, w),
                                                      name="C1 fp8 w8a8 128x256x256 f32 (every output)"))


def test_single_nvfp4_linear_full():
    x = synth.normal_bf16(512, 3072, 1.0, 0, 0)
    w = synth.normal_bf16(3072, 3072, 0.02, 0, 1)
    y = run_linear("nvfp4", x, w)
    log("nvfp4 512x3072x3072 max err/B", check_linear(y, oracle.linear_reference("nvfp4", x, w),
                                                      name="C2 nvfp4 w4a4 512x3072x3072 (every output)"))


@pytest.mark.parametrize("kind", ["fp8", "nvfp4"])
@pytest.mark.parametrize("name", list(synth.DIT_LINEARS))
def test_dit_linear_sampled(kind, name):
    n, k = synth.DIT_LINEARS[name]
    m = synth.DIT_TOKENS
    log("dit %s %s m=%d n=%d k=%d" % (kind, name, m, n, k))
    tail = 0.001 if kind == "nvfp4" else 0.0
    x = synth.normal_bf16(m, k, 1.0, 0, 0, outlier_frac=tail, outlier_gain=50.0)
    w = synth.normal_bf16(n, k, 0.02, 0, 1)
    y = run_linear(kind, x, w)
    rows, cols = _sample(m, n, 3000, 1)
    ref = oracle.linear_reference(kind, x, w, rows=rows, cols=cols)
    cfg = "C3 fp8 w8a8" if kind == "fp8" else "C4 nvfp4 w4a4 heavy-tailed"
    log("  max err/B", check_linear(y, ref, rows, cols, name="%s %s %dx%dx%d (%d sampled)" % (cfg, name, m, n, k, rows.size)))


@pytest.mark.parametrize("kind", ["fp8", "nvfp4"])
@pytest.mark.parametrize("m,n,k", [(256, 3072, 1024), (512, 1024, 3072), (2048, 1024, 3072), (1530, 3072, 3072),
                                   (2300, 3072, 3072), (3072, 3072, 1024), (1000, 1008, 1152), (250, 2992, 768)])
def test_mid_m_linear_sampled(kind, m, n, k):
    # token counts between the small-M shapes and the transformer's (ragged
    # ones among them), on both sides of the tile-count thresholds that pick
    # the 64 x 128 kernels (FP8, W4A4) over the persistent 256 x 256 ones, and
    # FP8 split-K tilings 32 x 128 (1000 x 1008, nine chunks over eight waves)
    # and 32 x 96 (250 x 2992, six chunks: two waves without one)
    log("%s mid-m %dx%dx%d" % (kind, m, n, k))
    x = synth.normal_bf16(m, k, 1.0, 7, 0)
    w = synth.normal_bf16(n, k, 0.02, 7, 1)
    y = run_linear(kind, x, w, check_codes=False)
    rows, cols = _sample(m, n, 2000, 8)
    ref = oracle.linear_reference(kind, x, w, rows=rows, cols=cols)
    log("  max err/B", check_linear(y, ref, rows, cols))


@pytest.mark.parametrize("m,n,k,out", [(4600, 9200, 3072, q.QG_OUT_BF16), (4608, 3072, 1152, q.QG_OUT_F32),
                                       (4321, 3056, 640, q.QG_OUT_BF16), (4321, 3056, 640, q.QG_OUT_F32)])
def test_fp8_whole_round_tiles_sampled(m, n, k, out):
    # shapes the FP8 GEMM runs on 288 x 192 tiles (whole rounds of tiles):
    # ragged rows and columns (4321 leaves one valid row in the last tile
    # row, 3056 and 9200 a part-filled last weight panel), an odd number of
    # 128-wide chunks (K = 1152, 640), bf16 and fp32 outputs
    log("fp8 288x192 tiles %dx%dx%d out=%d" % (m, n, k, out))
    x = synth.normal_bf16(m, k, 1.0, 9, 0)
    w = synth.normal_bf16(n, k, 0.02, 9, 1)
    y = run_linear("fp8", x, w, out, check_codes=False)
    rows, cols = _sample(m, n, 2000, 10)
    # the last row and the last columns of every tile edge are sampled too
    rows = np.concatenate([rows, np.full(192, m - 1), np.resize(np.arange(0, m, 288), 192)])
    cols = np.concatenate([cols, np.arange(n - 192, n), np.resize(np.arange(191, n, 192), 192)])
    ref = oracle.linear_reference("fp8", x, w, rows=rows, cols=cols)
    log("  max err/B", check_linear(y, ref, rows, cols))


@pytest.mark.parametrize("m,n,k,out", [(4600, 9200, 3072, q.QG_OUT_BF16), (4608, 3072, 1152, q.QG_OUT_F32),
                                       (4321, 3056, 640, q.QG_OUT_BF16), (4321, 3056, 640, q.QG_OUT_F32),
                                       (1000, 8208, 640, q.QG_OUT_BF16)])
def test_nvfp4_ragged_large_sampled(m, n, k, out):
    # the persistent 256 x 256 W4A4 kernel at ragged sizes: rows and columns
    # that leave the last tile row and tile column part-filled (4321, 4600,
    # 1000 rows; 3056, 9200, 8208 columns, a part-filled last weight panel),
    # an odd number of 128-wide chunks (K = 1152, 640), bf16 and fp32
    # outputs, heavy-tailed activations
    log("nvfp4 ragged %dx%dx%d out=%d" % (m, n, k, out))
    x = synth.normal_bf16(m, k, 1.0, 11, 0, outlier_frac=0.001, outlier_gain=50.0)
    w = synth.normal_bf16(n, k, 0.02, 11, 1)
    y = run_linear("nvfp4", x, w, out, check_codes=False)
    rows, cols = _sample(m, n, 2000, 12)
    # the last row, the first row of every tile row and the last column of
    # every tile column are sampled too
    rows = np.concatenate([rows, np.full(192, m - 1), np.resize(np.arange(0, m, 256), 192)])
    cols = np.concatenate([cols, np.arange(n - 192, n), np.resize(np.arange(255, n, 256), 192)])
    ref = oracle.linear_reference("nvfp4", x, w, rows=rows, cols=cols)
    log("  max err/B", check_linear(y, ref, rows, cols))


@pytest.mark.parametrize("name", list(synth.ENCODER_LINEARS))
@pytest.mark.parametrize("m", synth.ENCODER_TOKENS)
def test_w4a16_encoder_full(name, m):
    n, k = synth.ENCODER_LINEARS[name]
    x = synth.normal_bf16(m, k, 1.0, 0, 0)
    w = synth.normal_bf16(n, k, 0.02, 0, 1)
    y = run_linear("w4a16", x, w)
    log("w4a16 %s m=%d max err/B" % (name, m),
        check_linear(y, oracle.linear_reference("w4a16", x, w),
                     name="C5 w4a16 %s %dx%dx%d (every output)" % (name, m, n, k)))


@pytest.mark.parametrize("m,k", [(1, 1024), (1, 3072), (2, 3072), (7, 1024), (8, 1024), (9, 1024), (16, 1024), (15, 3072)])
def test_w4a16_weight_pool_sampled(m, k):
    # a few activation rows against a very wide weight (a pool of stacked
    # encoder weights streamed once): the persistent streaming kernel, with a
    # ragged last panel group; sampled outputs against the oracle
    n = 70016
    log("w4a16 pool m=%d n=%d k=%d" % (m, n, k))
    x = synth.normal_bf16(m, k, 1.0, 5, 0)
    w = synth.normal_bf16(n, k, 0.02, 5, 1)
    y = run_linear("w4a16", x, w)
    rows, cols = _sample(m, n, 2000, 3)
    ref = oracle.linear_reference("w4a16", x, w, rows=rows, cols=cols)
    log("  max err/B", check_linear(y, ref, rows, cols))


@pytest.mark.parametrize("out", [q.QG_OUT_F32, q.QG_OUT_BF16])
def test_w4a16_one_row_wide_weight(out):
    # one activation row against a very wide weight (the matrix-vector
    # kernel): a half-filled last panel, heavy-tailed channels, subnormal and
    # near-underflow activations, a zero block; every output against the oracle
    n, k = 70032, 1024
    log("w4a16 one row n=%d k=%d out=%d" % (n, k, out))
    x = synth.normal_bf16(1, k, 1.0, 6, 0, synth.HEAVY_TAIL_FRAC, synth.HEAVY_TAIL_GAIN)
    x[0, 16:32] &= 0x807F                          # subnormals only
    x[0, 32:48] = (x[0, 32:48] & 0x807F) | 0x0080  # exponent field 1
    x[0, 48:64] = 0
    w = synth.normal_bf16(n, k, 0.02, 6, 1)
    y = run_linear("w4a16", x, w, out=out)
    log("  max err/B", check_linear(y, oracle.linear_reference("w4a16", x, w)))


@pytest.mark.parametrize("m,n,k,out", [(256, 65536, 1024, q.QG_OUT_BF16), (300, 16400, 1152, q.QG_OUT_F32),
                                       (4608, 3072, 3072, q.QG_OUT_BF16), (1000, 8208, 640, q.QG_OUT_BF16)])
def test_w4a16_many_tiles_sampled(m, n, k, out):
    # W4A16 past the ridge point with enough 256 x 256 tiles for the
    # persistent kernel: a pool-like wide weight, ragged rows and columns
    # (300, 1000 rows; 16400, 8208 columns), odd chunk counts (K = 1152, 640),
    # bf16 and fp32 outputs; heavy-tailed activations with subnormal and zero
    # blocks in some rows
    log("w4a16 many tiles %dx%dx%d out=%d" % (m, n, k, out))
    x = synth.normal_bf16(m, k, 1.0, 12, 0, synth.HEAVY_TAIL_FRAC, synth.HEAVY_TAIL_GAIN)
    x[1, 16:32] &= 0x807F
    x[2, 32:48] = 0
    w = synth.normal_bf16(n, k, 0.02, 12, 1)
    y = run_linear("w4a16", x, w, out, check_codes=False)
    rows, cols = _sample(m, n, 2000, 13)
    rows = np.concatenate([rows, [1, 2, m - 1], np.resize(np.arange(255, m, 256), 64)])
    cols = np.concatenate([cols, [0, n - 1, n // 2], np.resize(np.arange(n - 64, n), 64)])
    ref = oracle.linear_reference("w4a16", x, w, rows=rows, cols=cols)
    log("  max err/B", check_linear(y, ref, rows, cols))


@pytest.mark.parametrize("kind", ["fp8", "nvfp4"])
def test_linear_with_calibrated_activation_scale(kind):
    # static activation scale calibrated on other batches (the max of their
    # dynamic scales), applied to a new batch: quantize once with the given
    # scale, then the GEMM; reference = oracle static codes x oracle weights
    m, n, k = 300, 272, 384
    fmt = q.QG_FMT_FP8_E4M3 if kind == "fp8" else q.QG_FMT_NVFP4
    cal = [synth.normal_bf16(m, k, 1.0, 20 + i, 0) for i in range(3)]
    x = synth.normal_bf16(m, k, 1.3, 30, 0)          # wider than the calibration data: some saturation
    w = synth.normal_bf16(n, k, 0.02, 30, 1)
    if kind == "fp8":
        s = max(oracle.quantize_fp8(c)[1] for c in cal)
        qa = oracle.quantize_fp8_static(x, s)
        a_ref = oracle.dequant_fp8(qa, s)
        qw, sw = oracle.quantize_fp8(w)
        w_ref = oracle.dequant_fp8(qw, sw)
    else:
        s = max(oracle.quantize_nvfp4(c)[2] for c in cal)
        qa, ba = oracle.quantize_nvfp4_static(x, s)
        a_ref = oracle.dequant_nvfp4(qa, ba, s)
        qw, bw, sw = oracle.quantize_nvfp4(w)
        w_ref = oracle.dequant_nvfp4(qw, bw, sw)
    y_ref, b = oracle.gemm_f64(a_ref, w_ref)
    sd = torch.tensor([np.float32(s)], dtype=torch.float32, device=DEV)
    a = q.quantize(to_dev_bf16(x), fmt, static_scale=sd)
    packed = q.pack(q.quantize(to_dev_bf16(w), fmt))
    y = q.linear(a, packed, fmt, n, out_dtype=q.QG_OUT_F32)
    torch.cuda.synchronize()
    log("  static %s max err/B" % kind, check_linear(y, {"y": y_ref, "b": b}))

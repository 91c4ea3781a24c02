"""GPU parity of the quantizers, dequantizers and weight packer with the CPU
oracle: every code, block scale and tensor-scale bit must match."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2609_21849_amd as q
import synth
from gpu_util import DEV, assert_quant_equal, host, log, scale_of, to_dev_bf16

pytestmark = pytest.mark.gpu

FP8, NVFP4 = q.QG_FMT_FP8_E4M3, q.QG_FMT_NVFP4
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")

# (rows, cols, sigma, heavy_tail): workload operands plus small and ragged cases
SHAPES = [
    (1, 16, 1.0, False), (3, 48, 1.0, False), (37, 160, 1.0, False),
    (128, 256, 1.0, False), (256, 256, 0.02, False),          # single FP8 linear
    (512, 3072, 1.0, False), (3072, 3072, 0.02, False),        # single NVFP4 linear
    (4608, 3072, 1.0, False), (4608, 3072, 1.0, True),          # DiT activations (K = 3072)
    (4608, 9216, 1.0, True), (9216, 3072, 0.02, False),         # DiT down-proj input, QKV weight
    (3072, 9216, 0.02, False), (16, 1024, 1.0, False),          # down-proj weight, encoder tokens
]


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
@pytest.mark.parametrize("rows,cols,sigma,tail", SHAPES)
def test_quantize_bit_exact(fmt, rows, cols, sigma, tail):
    log("quantize fmt=%d shape=%dx%d tail=%s" % (fmt, rows, cols, tail))
    x = synth.normal_bf16(rows, cols, sigma, 0, 0, outlier_frac=0.001 if tail else 0.0, outlier_gain=50.0)
    qt = q.quantize(to_dev_bf16(x), fmt)
    torch.cuda.synchronize()
    assert_quant_equal(qt, x)


@pytest.mark.parametrize("rows,cols", [(5, 37), (2, 7), (1, 1), (9, 130)])
def test_fp8_ragged_columns(rows, cols):
    x = synth.normal_bf16(rows, cols, 1.0, 3, 0)
    qt = q.quantize(to_dev_bf16(x), FP8)
    torch.cuda.synchronize()
    assert_quant_equal(qt, x)


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
@pytest.mark.parametrize("rows,cols", [(192, 256), (193, 256), (99, 496), (100, 496), (1, 49152), (3, 16384)])
def test_small_tensor_path_boundary(fmt, rows, cols):
    # tensors of up to 3072 units of 16 elements are quantized by one
    # workgroup in one kernel, larger ones by the three-kernel chain: both
    # sides of the limit, bit-exact against the oracle
    x = synth.normal_bf16(rows, cols, 1.0, 8, 0, outlier_frac=0.001, outlier_gain=50.0)
    qt = q.quantize(to_dev_bf16(x), fmt)
    torch.cuda.synchronize()
    assert_quant_equal(qt, x)


@pytest.mark.parametrize("rows,cols", [(99, 487), (100, 487)])
def test_small_tensor_path_boundary_ragged_fp8(rows, cols):
    # FP8 rows that end in a short unit: 99 x 31 units (one workgroup),
    # 100 x 31 (the chain)
    x = synth.normal_bf16(rows, cols, 1.0, 9, 0)
    qt = q.quantize(to_dev_bf16(x), FP8)
    torch.cuda.synchronize()
    assert_quant_equal(qt, x)


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
@pytest.mark.parametrize("offset", [0, 1])
def test_strided_rows_past_the_small_limit(fmt, offset):
    # row stride 1280, 1024 columns, 600 rows (38400 units: the three-kernel
    # chain's per-row element kernels); offset 1 makes the rows 2-byte aligned
    # only (the scalar loads)
    full = synth.normal_bf16(600, 1280, 1.0, 10, 0, outlier_frac=0.001, outlier_gain=50.0)
    xd = to_dev_bf16(full)[:, offset:offset + 1024]
    qt = q.quantize(xd, fmt)
    torch.cuda.synchronize()
    assert_quant_equal(qt, np.ascontiguousarray(full[:, offset:offset + 1024]))


@pytest.mark.parametrize("fmt,rows,cols", [(FP8, 3073, 16), (NVFP4, 3073, 16), (FP8, 1001, 1000),
                                           (FP8, 600, 1024), (NVFP4, 600, 1024), (FP8, 512, 3072),
                                           (NVFP4, 512, 3072), (FP8, 1024, 3072), (NVFP4, 1025, 3072)])
@pytest.mark.parametrize("where", ["first", "last"])
def test_dense_two_launch_path(fmt, rows, cols, where):
    # dense tensors past the small limit: the amax launch hands its maxima to
    # every code region of the quantize launch (3073 x 16: 3073 units, just
    # past the small kernel; 1001 x 1000: an odd number of 8-element units;
    # 1024 x 3072: the largest such tensor, 1025 x 3072 the chain); the
    # tensor max sits in the first or the last region
    x = synth.normal_bf16(rows, cols, 1.0, 11, 0, outlier_frac=0.001, outlier_gain=20.0)
    if where == "first":
        x[0, 1] = 0xC300   # -128
    else:
        x[rows - 1, cols - 1] = 0x4300   # 128
    qt = q.quantize(to_dev_bf16(x), fmt)
    torch.cuda.synchronize()
    assert_quant_equal(qt, x)


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
def test_dense_two_launch_zero_and_reuse(fmt):
    # an all-zero dense tensor (scale 0, every code 0), then a tensor with a
    # much smaller max quantized into the same buffers, which hold the first
    # call's codes: every handed-over maximum must be the second call's
    rows, cols = 600, 1024
    z = np.zeros((rows, cols), np.uint16)
    qt = q.quantize(to_dev_bf16(z), fmt)
    torch.cuda.synchronize()
    assert_quant_equal(qt, z)
    big = synth.normal_bf16(rows, cols, 100.0, 12, 0)
    small = synth.normal_bf16(rows, cols, 0.01, 13, 0)
    for x in (big, small):
        xd = to_dev_bf16(x)
        q.qg_quantize_act(fmt, xd, rows, cols, cols, qt.codes, qt.block_scales, qt.tensor_scale)
        torch.cuda.synchronize()
        assert_quant_equal(qt, x)


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
def test_concurrent_calls_on_two_streams(fmt):
    # the dynamic quantizers keep no state of their own (their partial maxima
    # live in each call's code buffer), so calls on two streams may overlap:
    # a dense tensor on the two-launch path and one on the three-kernel chain,
    # each issued several times on its own stream
    xa = synth.normal_bf16(600, 1024, 1.0, 14, 0, outlier_frac=0.001, outlier_gain=50.0)
    xb = synth.normal_bf16(2048, 3072, 0.5, 15, 0, outlier_frac=0.001, outlier_gain=50.0)
    da, db = to_dev_bf16(xa), to_dev_bf16(xb)
    qa, qb = q.quantize(da, fmt), q.quantize(db, fmt)
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(4):
        q.qg_quantize_act(fmt, da, 600, 1024, 1024, qa.codes, qa.block_scales, qa.tensor_scale, stream=sa)
        q.qg_quantize_act(fmt, db, 2048, 3072, 3072, qb.codes, qb.block_scales, qb.tensor_scale, stream=sb)
    torch.cuda.synchronize()
    assert_quant_equal(qa, xa)
    assert_quant_equal(qb, xb)


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
def test_row_stride_larger_than_row(fmt):
    full = synth.normal_bf16(64, 400, 1.0, 4, 0)
    xd = to_dev_bf16(full)[:, :320]
    assert xd.stride(0) == 400
    qt = q.quantize(xd, fmt)
    torch.cuda.synchronize()
    assert_quant_equal(qt, np.ascontiguousarray(full[:, :320]))


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
def test_odd_row_stride_unaligned(fmt):
    """ldx not a multiple of 8 and a 2-byte-aligned base: the scalar load path."""
    full = synth.normal_bf16(33, 163, 1.0, 5, 0)
    xd = to_dev_bf16(full)[:, 1:161]
    qt = q.quantize(xd, fmt)
    torch.cuda.synchronize()
    assert_quant_equal(qt, np.ascontiguousarray(full[:, 1:161]))


def test_worked_examples():
    g = json.load(open(GOLDEN))
    x8 = synth.f32_to_bf16_bits(np.array(g["fp8"]["x"], np.float32))[None, :]
    q8 = q.quantize(to_dev_bf16(x8), FP8)
    x4 = synth.f32_to_bf16_bits(np.array(g["nvfp4"]["x"], np.float32))[None, :]
    q4 = q.quantize(to_dev_bf16(x4), NVFP4)
    torch.cuda.synchronize()
    assert host(q8.codes)[0].tolist() == g["fp8"]["codes"]
    assert scale_of(q8.tensor_scale) == np.float32(g["fp8"]["scale"])
    c = host(q4.codes)[0]
    codes = np.stack([c & 15, c >> 4], axis=1).reshape(-1).tolist()
    assert codes == g["nvfp4"]["element_codes"]
    assert host(q4.block_scales)[0].tolist() == g["nvfp4"]["block_scales"]
    assert scale_of(q4.tensor_scale) == np.float32(g["nvfp4"]["tensor_scale"])


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
def test_zero_tensor_and_empty(fmt):
    x = np.zeros((8, 64), np.uint16)
    x[3, 5] = 0x8000
    qt = q.quantize(to_dev_bf16(x), fmt)
    torch.cuda.synchronize()
    assert_quant_equal(qt, x)
    e = q.quantize(torch.empty((0, 64), dtype=torch.bfloat16, device=DEV), fmt)
    torch.cuda.synchronize()
    assert scale_of(e.tensor_scale) == 0.0


def test_tiny_blocks_get_subnormal_scales():
    """Rows scaled down by 2^-12 .. 2^-20 give E4M3-subnormal and zero block scales."""
    x = synth.normal_bf16(32, 256, 1.0, 6, 0)
    xf = synth.bf16_bits_to_f32(x).astype(np.float64)
    xf[8:] *= 2.0 ** -np.arange(12, 36)[:, None]
    xb = synth.f32_to_bf16_bits(xf.astype(np.float32))
    _, bs, _ = oracle.quantize_nvfp4(xb)
    assert (bs < 8).any() and (bs == 0).any()
    for fmt in (FP8, NVFP4):
        qt = q.quantize(to_dev_bf16(xb), fmt)
        torch.cuda.synchronize()
        assert_quant_equal(qt, xb)


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
@pytest.mark.parametrize("rows,cols,bad", [(4, 64, 0x7F80), (16, 3072, 0xFFC1), (600, 1024, 0x7F80),
                                            (600, 1024, 0xFFC1)])
def test_nonfinite_input_gives_nan_scale(fmt, rows, cols, bad):
    # +inf or a NaN anywhere: the single-launch small-tensor kernel (one
    # workgroup at 4 x 64, eight at 16 x 3072) and the two-launch dense path
    # (600 x 1024) both leave a NaN tensor scale
    x = synth.normal_bf16(rows, cols, 1.0, 7, 0)
    x[rows // 2, 9] = bad
    qt = q.quantize(to_dev_bf16(x), fmt)
    torch.cuda.synchronize()
    assert np.isnan(scale_of(qt.tensor_scale))


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
@pytest.mark.parametrize("out", [q.QG_OUT_F32, q.QG_OUT_BF16])
def test_dequant_bit_exact(fmt, out):
    x = synth.normal_bf16(96, 512, 1.0, 8, 0, outlier_frac=0.01, outlier_gain=50.0)
    qt = q.quantize(to_dev_bf16(x), fmt)
    d = q.dequantize(qt, out)
    torch.cuda.synchronize()
    kind = "f32" if out == q.QG_OUT_F32 else "bf16"
    if fmt == FP8:
        c, s = oracle.quantize_fp8(x)
        ref = oracle.dequant_fp8(c, s, out=kind)
    else:
        c, b, s = oracle.quantize_nvfp4(x)
        ref = oracle.dequant_nvfp4(c, b, s, out=kind)
    got = host(d) if out == q.QG_OUT_F32 else host(d.view(torch.int16)).view(np.uint16)
    assert got.dtype == ref.dtype
    assert np.array_equal(got.view(np.uint32 if out == q.QG_OUT_F32 else np.uint16),
                          ref.view(np.uint32 if out == q.QG_OUT_F32 else np.uint16))


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
@pytest.mark.parametrize("n,k", [(16, 128), (48, 384), (3072, 1024), (1024, 3072)])
def test_pack_unpack_roundtrip(fmt, n, k):
    w = synth.normal_bf16(n, k, 0.02, 9, 1)
    wq = q.quantize(to_dev_bf16(w), fmt)
    packed = q.pack(wq)
    back = q.unpack(packed, fmt, n, k)
    torch.cuda.synchronize()
    assert torch.equal(back.codes, wq.codes)
    if fmt == NVFP4:
        assert torch.equal(back.block_scales, wq.block_scales)
    assert torch.equal(back.tensor_scale, wq.tensor_scale)
    # the packed image is a permutation of the codes plus zero padding rows
    # (panels of 32 rows)
    codes = host(wq.codes)
    pad_rows = (-n) % 32
    body = host(packed)[256:256 + codes.size + pad_rows * codes.shape[1]]
    expect = np.concatenate([codes.reshape(-1), np.zeros(pad_rows * codes.shape[1], np.uint8)])
    assert np.array_equal(np.sort(body), np.sort(expect))


# ---------------------------------------------------------------- static (calibrated) scales
STATIC_SHAPES = [(1, 16), (37, 160), (512, 3072), (4608, 3072), (257, 400)]


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
@pytest.mark.parametrize("rows,cols", STATIC_SHAPES)
@pytest.mark.parametrize("factor", [1.0, 0.5, 0.3, 3.0, 0.0])
def test_static_quantize_bit_exact(fmt, rows, cols, factor):
    # the calibrated scale: the tensor's own dynamic scale (codes must equal
    # the dynamic codes), smaller ones (saturation beyond the calibrated
    # range), a larger one and zero
    log("static quantize fmt=%d shape=%dx%d factor=%g" % (fmt, rows, cols, factor))
    x = synth.normal_bf16(rows, cols, 1.0, 7, 0, outlier_frac=0.001, outlier_gain=50.0)
    if fmt == FP8:
        _, s_dyn = oracle.quantize_fp8(x)
    else:
        _, _, s_dyn = oracle.quantize_nvfp4(x)
    s = np.float32(s_dyn * np.float32(factor))
    sd = torch.tensor([s], dtype=torch.float32, device=DEV)
    qt = q.quantize(to_dev_bf16(x), fmt, static_scale=sd)
    torch.cuda.synchronize()
    assert scale_of(sd).view(np.uint32) == s.view(np.uint32)      # the scale is an input only
    if fmt == FP8:
        ref = oracle.quantize_fp8_static(x, s)
        nbad = int(np.count_nonzero(host(qt.codes) != ref))
        assert nbad == 0, "fp8 static codes differ at %d of %d" % (nbad, ref.size)
    else:
        rc, rb = oracle.quantize_nvfp4_static(x, s)
        assert int(np.count_nonzero(host(qt.codes) != rc)) == 0
        assert int(np.count_nonzero(host(qt.block_scales) != rb)) == 0


@pytest.mark.parametrize("fmt", [FP8, NVFP4])
def test_static_quantize_strided_rows(fmt):
    full = synth.normal_bf16(64, 400, 1.0, 8, 0)
    xd = to_dev_bf16(full)[:, :320]
    x = np.ascontiguousarray(full[:, :320])
    s = np.float32(0.004)
    qt = q.quantize(xd, fmt, static_scale=torch.tensor([s], device=DEV))
    torch.cuda.synchronize()
    if fmt == FP8:
        assert np.array_equal(host(qt.codes), oracle.quantize_fp8_static(x, s))
    else:
        rc, rb = oracle.quantize_nvfp4_static(x, s)
        assert np.array_equal(host(qt.codes), rc) and np.array_equal(host(qt.block_scales), rb)

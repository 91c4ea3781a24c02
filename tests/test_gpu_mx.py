"""GPU parity of the OCP MX path (MXFP4 / MXFP8 quantizer, dequantizer and
weight packing, the MXFP4 x MXFP4 and MXFP8 x MXFP8 GEMMs on the block-scaled
matrix instruction) with the CPU oracle: codes and E8M0 scales bit-exact, decoded
values bit-exact, GEMM outputs within |y - y_ref| <= 1e-3 * sum_k |a w| of the
oracle's fp64 product over the same quantized operands."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_21849_amd as q
import synth
from gpu_util import DEV, check_linear, host, log, to_dev_bf16

pytestmark = pytest.mark.gpu

MXFP4, MXFP8 = q.QG_FMT_MXFP4, q.QG_FMT_MXFP8
NAME = {MXFP4: "mxfp4", MXFP8: "mxfp8"}


def assert_mx_equal(qt, x_bits):
    codes, sc = oracle.quantize_mx(x_bits, NAME[qt.fmt])
    got = host(qt.codes)
    assert got.shape == codes.shape
    nbad = int(np.count_nonzero(got != codes))
    assert nbad == 0, "%s codes differ at %d of %d" % (NAME[qt.fmt], nbad, codes.size)
    nbs = int(np.count_nonzero(host(qt.block_scales) != sc))
    assert nbs == 0, "%s scales differ at %d of %d" % (NAME[qt.fmt], nbs, sc.size)
    assert qt.tensor_scale is None


def random_finite_bf16(rows, cols, seed):
    """Uniformly random finite bf16 bit patterns: every exponent from the
    subnormals to the largest finite value, both signs, exercising the scale
    clamp at both ends (plus whole zero blocks)."""
    w = synth.uniform_words(seed, 0, rows * cols)
    b = (w & np.uint64(0xFFFF)).astype(np.uint16)
    finite = (b & 0x7F80) != 0x7F80
    b = np.where(finite, b, b & 0x807F).reshape(rows, cols)   # inf/NaN -> subnormal
    b[0, :32] = 0                                              # an all-zero block
    b[-1, -32:] = 0x8000                                       # a block of -0
    # blocks whose largest magnitude lies below 2^-125 (bf16 exponent fields 0
    # and 1): a random block almost never does, and they need the code clamped at 0
    b[1, :32] &= 0x807F                                        # subnormals only
    b[2, 32:64] = (b[2, 32:64] & 0x807F) | 0x0080              # exponent field 1
    return b


SHAPES = [(1, 32, 1.0, False), (3, 64, 1.0, False), (37, 160, 1.0, False), (128, 256, 1.0, False),
          (4608, 3072, 1.0, True), (9216, 3072, 0.02, False), (3072, 9216, 0.02, False)]


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
@pytest.mark.parametrize("rows,cols,sigma,tail", SHAPES)
def test_mx_quantize_bit_exact(fmt, rows, cols, sigma, tail):
    log("mx quantize fmt=%d shape=%dx%d tail=%s" % (fmt, rows, cols, tail))
    x = synth.normal_bf16(rows, cols, sigma, 0, 0, outlier_frac=0.001 if tail else 0.0, outlier_gain=50.0)
    qt = q.quantize(to_dev_bf16(x), fmt)
    torch.cuda.synchronize()
    assert_mx_equal(qt, x)


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
def test_mx_quantize_every_exponent(fmt):
    x = random_finite_bf16(257, 1024, 21)
    qt = q.quantize(to_dev_bf16(x), fmt)
    torch.cuda.synchronize()
    assert_mx_equal(qt, x)
    sc = host(qt.block_scales)
    # zero blocks give code 0; the largest bf16 exponent (127) gives
    # 127 - emax + 127: 252 for E2M1 (emax 2), 246 for E4M3 (emax 8)
    assert sc.min() == 0 and sc.max() == (252 if fmt == MXFP4 else 246)


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
def test_mx_row_stride_and_unaligned_base(fmt):
    full = synth.normal_bf16(33, 330, 1.0, 5, 0)
    for lo in (0, 1):                           # 16-byte aligned rows, then the scalar path
        xd = to_dev_bf16(full)[:, lo:lo + 288]
        qt = q.quantize(xd, fmt)
        torch.cuda.synchronize()
        assert_mx_equal(qt, np.ascontiguousarray(full[:, lo:lo + 288]))


def test_mxfp8_unaligned_codes():
    x = synth.normal_bf16(9, 96, 1.0, 6, 0)
    buf = torch.full((9 * 96 + 8,), 0xAB, dtype=torch.uint8, device=DEV)
    bs = torch.empty((9, 3), dtype=torch.uint8, device=DEV)
    xd = to_dev_bf16(x)
    q.qg_quantize_act(MXFP8, xd, 9, 96, 96, buf[3:], bs, None)
    torch.cuda.synchronize()
    codes, sc = oracle.quantize_mx(x, "mxfp8")
    got = host(buf)
    assert np.array_equal(got[3:3 + codes.size].reshape(codes.shape), codes)
    assert np.all(got[:3] == 0xAB) and np.all(got[3 + codes.size:] == 0xAB)
    assert np.array_equal(host(bs), sc)


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
@pytest.mark.parametrize("out", [q.QG_OUT_F32, q.QG_OUT_BF16])
def test_mx_dequant_bit_exact(fmt, out):
    # every code with every finite scale (0 .. 254)
    rows, cols = 255, 256
    rng = np.random.default_rng(3)
    if fmt == MXFP4:
        codes = rng.integers(0, 256, (rows, cols // 2), dtype=np.uint8)
    else:
        codes = rng.integers(0, 256, (rows, cols), dtype=np.uint8)
        codes[(codes & 0x7F) == 0x7F] = 0x7E               # E4M3 NaN codes are outside the contract
    sc = np.repeat(np.arange(255, dtype=np.uint8)[:, None], cols // 32, axis=1)
    with np.errstate(over="ignore"):      # 6 * 2^127 and 448 * 2^127 round to inf in fp32
        ref = oracle.dequant_mx(codes, sc, NAME[fmt]).astype(np.float32)   # exact values, rounded to fp32
    qt = q.QTensor(fmt, torch.from_numpy(codes).to(DEV), torch.from_numpy(sc).to(DEV), None, rows, cols)
    d = q.dequantize(qt, out)
    torch.cuda.synchronize()
    if out == q.QG_OUT_F32:
        assert np.array_equal(host(d).view(np.uint32), ref.view(np.uint32))
    else:
        want = torch.from_numpy(ref).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(host(d.view(torch.int16)).view(np.uint16), want)


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
@pytest.mark.parametrize("n,k", [(16, 256), (48, 512), (80, 768), (3072, 3072)])
def test_mx_pack_unpack_roundtrip(fmt, n, k):
    w = synth.normal_bf16(n, k, 0.02, 9, 1)
    wq = q.quantize(to_dev_bf16(w), fmt)
    packed = q.pack(wq)
    back = q.unpack(packed, fmt, n, k)
    torch.cuda.synchronize()
    assert torch.equal(back.codes, wq.codes)
    assert torch.equal(back.block_scales, wq.block_scales)
    assert back.tensor_scale is None
    # codes region: a permutation of the codes plus zero padding rows
    codes = host(wq.codes)
    pad_rows = (-n) % 32
    body = host(packed)[256:256 + codes.size + pad_rows * codes.shape[1]]
    expect = np.concatenate([codes.reshape(-1), np.zeros(pad_rows * codes.shape[1], np.uint8)])
    assert np.array_equal(np.sort(body), np.sort(expect))


def run_mx_linear(x, w, out=q.QG_OUT_BF16, check_codes=True, fmt=MXFP4):
    xd, wd = to_dev_bf16(x), to_dev_bf16(w)
    wq = q.quantize(wd, fmt)
    packed = q.pack(wq)
    a = q.quantize(xd, fmt)
    y = q.linear(a, packed, fmt, w.shape[0], out_dtype=out)
    torch.cuda.synchronize()
    if check_codes:
        assert_mx_equal(wq, w)
        assert_mx_equal(a, x)
    return y


@pytest.mark.parametrize("m,n,k", [(1, 16, 256), (17, 48, 256), (64, 256, 512), (300, 272, 768),
                                   (257, 512, 1024), (512, 768, 1280), (100, 2080, 512), (129, 528, 2304)])
@pytest.mark.parametrize("out", [q.QG_OUT_F32, q.QG_OUT_BF16])
@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
def test_mx_gemm_small_full_parity(fmt, m, n, k, out):
    log("%s gemm m=%d n=%d k=%d out=%d" % (NAME[fmt], m, n, k, out))
    x = synth.normal_bf16(m, k, 1.0, 11, 0)
    w = synth.normal_bf16(n, k, 0.02, 11, 1)
    y = run_mx_linear(x, w, out, fmt=fmt)
    log("  max err/B", check_linear(y, oracle.linear_reference(NAME[fmt], x, w), literal=False))


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
def test_mx_gemm_zero_rows_and_blocks(fmt):
    # an all-zero activation row gives an exactly zero output row; zero blocks
    # (E8M0 code 0) elsewhere contribute nothing
    m, n, k = 40, 64, 512
    x = synth.normal_bf16(m, k, 1.0, 12, 0)
    x[5, :] = 0
    x[7, 64:160] = 0
    w = synth.normal_bf16(n, k, 0.02, 12, 1)
    w[3, :256] = 0
    y = run_mx_linear(x, w, q.QG_OUT_F32, fmt=fmt)
    assert not torch.any(y[5]).item()
    check_linear(y, oracle.linear_reference(NAME[fmt], x, w))


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
def test_mx_gemm_row_independent_of_batch(fmt):
    # the same activation row gives bit-identical outputs whatever the batch
    n, k = 512, 1024
    x = synth.normal_bf16(600, k, 1.0, 13, 0)
    w = synth.normal_bf16(n, k, 0.02, 13, 1)
    y_all = run_mx_linear(x, w, q.QG_OUT_F32, check_codes=False, fmt=fmt)
    y_one = run_mx_linear(x[299:300], w, q.QG_OUT_F32, check_codes=False, fmt=fmt)
    assert torch.equal(y_all[299:300], y_one)
    y_again = run_mx_linear(x, w, q.QG_OUT_F32, check_codes=False, fmt=fmt)
    assert torch.equal(y_all, y_again)


def _sample(m, n, count, seed):
    rng = np.random.default_rng(seed)
    rows = np.concatenate([[0, m - 1, 0, m - 1], rng.integers(0, m, count)])
    cols = np.concatenate([[0, 0, n - 1, n - 1], rng.integers(0, n, count)])
    return rows, cols


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
@pytest.mark.parametrize("name", list(synth.DIT_LINEARS))
def test_mx_dit_linear_sampled(fmt, name):
    n, k = synth.DIT_LINEARS[name]
    m = synth.DIT_TOKENS
    log("dit %s %s m=%d n=%d k=%d" % (NAME[fmt], name, m, n, k))
    x = synth.normal_bf16(m, k, 1.0, 0, 0, outlier_frac=0.001, outlier_gain=50.0)
    w = synth.normal_bf16(n, k, 0.02, 0, 1)
    y = run_mx_linear(x, w, fmt=fmt)
    rows, cols = _sample(m, n, 3000, 1)
    ref = oracle.linear_reference(NAME[fmt], x, w, rows=rows, cols=cols)
    log("  max err/B", check_linear(y, ref, rows, cols,
                                    name="%s %s %dx%dx%d heavy-tailed (%d sampled)" % (NAME[fmt], name, m, n, k, rows.size)))


@pytest.mark.parametrize("fmt", [MXFP4, MXFP8])
def test_mx_nonfinite_block_gets_nan_scale(fmt):
    """A block holding inf and a block holding NaN get the E8M0 NaN code 255
    and decode to NaN; every other block (MX has no tensor-wide reduction) is
    coded exactly as the oracle codes the same tensor with those two blocks
    zeroed (the oracle refuses non-finite input)."""
    rows, cols = 8, 256
    x = synth.normal_bf16(rows, cols, 1.0, 14, 0)
    x[2, 37] = 0x7F80          # +inf in block 1 of row 2
    x[5, 200] = 0xFFC1         # a NaN in block 6 of row 5
    qt = q.quantize(to_dev_bf16(x), fmt)
    d = q.dequantize(qt, q.QG_OUT_F32)
    torch.cuda.synchronize()
    sc = host(qt.block_scales)
    assert sc[2, 1] == 255 and sc[5, 6] == 255
    clean = x.copy()
    clean[2, 32:64] = 0
    clean[5, 192:224] = 0
    codes_ref, sc_ref = oracle.quantize_mx(clean, NAME[fmt])
    bad = np.zeros(sc_ref.shape, bool)
    bad[2, 1] = bad[5, 6] = True
    assert np.array_equal(sc[~bad], sc_ref[~bad])
    per = 16 if fmt == MXFP4 else 32                       # code bytes per block
    got = host(qt.codes).reshape(rows, cols // 32, per)
    want = codes_ref.reshape(rows, cols // 32, per)
    assert np.array_equal(got[~bad], want[~bad])
    dv = host(d)
    assert np.isnan(dv[2, 32:64]).all() and np.isnan(dv[5, 192:224]).all()
    ok = np.ones(dv.shape, bool)
    ok[2, 32:64] = ok[5, 192:224] = False
    assert np.isfinite(dv[ok]).all()

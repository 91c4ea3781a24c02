"""GPU parity of qg_gemm_quant: the GEMM epilogue writes its output as FP8
E4M3 codes with a static decode scale (the next linear's activation). Every
code must be a correct rounding (the static quantizer's E4M3(fl(y * r))) of
some value within the GEMM accuracy contract of the oracle's exact product,
i.e. lie between the codes of (y_ref - e) and (y_ref + e), e = 1e-3 sum|a w|."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_21849_amd as q
import synth
from gpu_util import DEV, check_codes, check_linear, check_nvfp4_codes, host, log, to_dev_bf16

pytestmark = pytest.mark.gpu

KINDS = {"fp8": (q.QG_FMT_FP8_E4M3, q.QG_FMT_FP8_E4M3), "nvfp4": (q.QG_FMT_NVFP4, q.QG_FMT_NVFP4),
         "w4a16": (q.QG_FMT_BF16, q.QG_FMT_NVFP4), "mxfp4": (q.QG_FMT_MXFP4, q.QG_FMT_MXFP4),
         "mxfp8": (q.QG_FMT_MXFP8, q.QG_FMT_MXFP8)}


def run(kind, x, w, s_y):
    a_fmt, w_fmt = KINDS[kind]
    xd, wd = to_dev_bf16(x), to_dev_bf16(w)
    packed = q.pack(q.quantize(wd, w_fmt))
    a = xd if a_fmt == q.QG_FMT_BF16 else q.quantize(xd, a_fmt)
    ys = torch.tensor([s_y], dtype=torch.float32, device=DEV)
    qt = q.linear_fp8_out(a, packed, w_fmt, w.shape[0], ys)
    y32 = q.linear(a, packed, w_fmt, w.shape[0], out_dtype=q.QG_OUT_F32)
    torch.cuda.synchronize()
    return host(qt.codes), host(y32)


@pytest.mark.parametrize("kind", list(KINDS))
@pytest.mark.parametrize("m,n,k", [(1, 16, 256), (37, 80, 512), (300, 272, 768), (129, 528, 1280),
                                   (250, 2992, 768)])
@pytest.mark.parametrize("sat", [1.0, 0.25])
def test_fp8_output_within_contract(kind, m, n, k, sat):
    log("gemm_quant %s m=%d n=%d k=%d sat=%.2f" % (kind, m, n, k, sat))
    x = synth.normal_bf16(m, k, 1.0, 21, 0)
    w = synth.normal_bf16(n, k, 0.02, 21, 1)
    ref = oracle.linear_reference(kind, x, w)
    # static scale from the exact output's range (sat < 1: part of it saturates)
    s_y = np.float32(sat * np.abs(ref["y"]).max() / 448.0)
    r = np.float32(1.0) / s_y
    codes, y32 = run(kind, x, w, float(s_y))
    unique = check_codes(codes, ref, float(r))
    log("  unique-rounding fraction %.4f" % unique)
    # consistency with the fp32 output of the same GEMM (not a parity claim:
    # both sides are this library): the epilogue is the quantizer's element
    # step on that value, here done by torch's e4m3fn cast after the clamp
    prod = torch.from_numpy(np.clip(y32 * r, -448.0, 448.0).astype(np.float32))
    want = prod.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes, want)


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "mxfp4", "w4a16"])
def test_fp8_output_transformer_shape_sampled(kind):
    # the persistent large-M kernel of each format (W8A8: 288 x 192 tiles;
    # W4A16: the bf16 kernel past the ridge point) writing FP8 codes
    m, (n, k) = synth.DIT_TOKENS, synth.DIT_LINEARS["qkv"]
    x = synth.normal_bf16(m, k, 1.0, 0, 0)
    w = synth.normal_bf16(n, k, 0.02, 0, 1)
    rng = np.random.default_rng(4)
    rows = np.concatenate([[0, m - 1, 0, m - 1], rng.integers(0, m, 3000)])
    cols = np.concatenate([[0, 0, n - 1, n - 1], rng.integers(0, n, 3000)])
    ref = oracle.linear_reference(kind, x, w, rows=rows, cols=cols)
    s_y = np.float32(np.abs(ref["y"]).max() / 448.0)
    codes, _ = run(kind, x, w, float(s_y))
    check_codes(codes, ref, float(np.float32(1.0) / s_y), rows, cols)


def test_zero_scale_and_empty_k():
    x = synth.normal_bf16(8, 256, 1.0, 3, 0)
    w = synth.normal_bf16(32, 256, 0.02, 3, 1)
    codes, _ = run("fp8", x, w, 0.0)
    assert np.all((codes & 0x7F) == 0)           # r = 0: signed zeros
    # k = 0: every output is an exact zero
    ys = torch.ones(1, dtype=torch.float32, device=DEV)
    wq = q.quantize(to_dev_bf16(synth.normal_bf16(16, 128, 0.02, 1, 1)), q.QG_FMT_FP8_E4M3)
    packed = q.pack(wq)
    out = torch.full((4, 16), 0x55, dtype=torch.uint8, device=DEV)
    a = torch.empty((4, 0), dtype=torch.uint8, device=DEV)
    q.qg_gemm_quant(q.QG_FMT_FP8_E4M3, a, None, ys, 0, q.QG_FMT_FP8_E4M3, packed, packed.numel(), 4, 16, 0,
                    out, 16, ys)
    torch.cuda.synchronize()
    assert not torch.any(out).item()


# ---------------------------------------------------------------- NVFP4 output (qg_gemm_quant_nvfp4)
NV_KINDS = ["fp8", "nvfp4", "mxfp4", "mxfp8"]


def run_nvfp4_out(kind, x, w, s_t):
    a_fmt, w_fmt = KINDS[kind]
    xd, wd = to_dev_bf16(x), to_dev_bf16(w)
    packed = q.pack(q.quantize(wd, w_fmt))
    a = q.quantize(xd, a_fmt)
    st = torch.tensor([s_t], dtype=torch.float32, device=DEV)
    qt = q.linear_nvfp4_out(a, packed, w_fmt, w.shape[0], st)
    y32 = q.linear(a, packed, w_fmt, w.shape[0], out_dtype=q.QG_OUT_F32)
    torch.cuda.synchronize()
    return host(qt.codes), host(qt.block_scales), host(y32)


def _nv_scale(ref, sat):
    # the tensor scale a calibration of this output would give (its max over
    # 2688), times `sat` (< 1: some blocks saturate)
    return np.float32(np.abs(ref["y"]).max() / 2688.0 * sat)


@pytest.mark.parametrize("kind", NV_KINDS)
@pytest.mark.parametrize("m,n,k", [(1, 16, 256), (37, 80, 512), (300, 272, 768), (129, 528, 1280),
                                   (250, 2992, 768)])
@pytest.mark.parametrize("sat", [1.0, 0.25])
def test_nvfp4_output_within_contract(kind, m, n, k, sat):
    log("gemm_quant_nvfp4 %s m=%d n=%d k=%d sat=%.2f" % (kind, m, n, k, sat))
    x = synth.normal_bf16(m, k, 1.0, 22, 0)
    w = synth.normal_bf16(n, k, 0.02, 22, 1)
    ref = oracle.linear_reference(kind, x, w)
    s_t = _nv_scale(ref, sat)
    codes, bs, y32 = run_nvfp4_out(kind, x, w, s_t)
    uniq = check_nvfp4_codes(codes, bs, ref, s_t)
    log("  block scales with a unique rounding: %.3f" % uniq)
    # consistency (not a parity claim): the epilogue quantizes exactly the
    # fp32 values the same kernel returns with fp32 output
    c2, b2 = oracle.quantize_nvfp4_static_f32(y32, s_t)
    assert np.array_equal(codes, c2) and np.array_equal(bs, b2)


@pytest.mark.parametrize("kind", ["fp8", "nvfp4"])
def test_nvfp4_output_transformer_shape_sampled_rows(kind):
    # the QKV linear at the transformer's token count (persistent 256 x 256
    # kernels); 48 whole output rows against the oracle
    m, (n, k) = synth.DIT_TOKENS, synth.DIT_LINEARS["qkv"]
    log("gemm_quant_nvfp4 %s %dx%dx%d" % (kind, m, n, k))
    x = synth.normal_bf16(m, k, 1.0, 23, 0)
    w = synth.normal_bf16(n, k, 0.02, 23, 1)
    rows = np.sort(np.random.default_rng(4).choice(m, 48, replace=False))
    rr, cc = np.repeat(rows, n), np.tile(np.arange(n), rows.size)
    ref = oracle.linear_reference(kind, x, w, rows=rr, cols=cc)
    ref = {"y": ref["y"].reshape(rows.size, n), "b": ref["b"].reshape(rows.size, n)}
    s_t = _nv_scale(ref, 1.0)
    codes, bs, y32 = run_nvfp4_out(kind, x, w, s_t)
    uniq = check_nvfp4_codes(codes[rows], bs[rows], ref, s_t)
    log("  block scales with a unique rounding: %.3f" % uniq)
    c2, b2 = oracle.quantize_nvfp4_static_f32(y32, s_t)
    assert np.array_equal(codes, c2) and np.array_equal(bs, b2)


def test_nvfp4_output_zero_k_and_scale():
    # k = 0: zero codes and zero block scales; s_t = 0: every block scale 0
    m, n = 5, 80
    packed = torch.zeros(q.qg_packed_bytes(q.QG_FMT_NVFP4, n, 0), dtype=torch.uint8, device=DEV)
    ts = torch.ones(1, dtype=torch.float32, device=DEV)
    codes = torch.full((m, n // 2), 0x55, dtype=torch.uint8, device=DEV)
    bs = torch.full((m, n // 16), 0x55, dtype=torch.uint8, device=DEV)
    a = torch.zeros(16, dtype=torch.uint8, device=DEV)
    q.qg_gemm_quant_nvfp4(q.QG_FMT_NVFP4, a, a, ts, 0, q.QG_FMT_NVFP4, packed, packed.numel(), m, n, 0, codes, bs,
                          n, ts)
    torch.cuda.synchronize()
    assert not codes.any().item() and not bs.any().item()
    x = synth.normal_bf16(40, 256, 1.0, 24, 0)
    w = synth.normal_bf16(64, 256, 0.02, 24, 1)
    c, b, _ = run_nvfp4_out("nvfp4", x, w, np.float32(0.0))
    assert not b.any() and np.all((c & 0x77) == 0)       # zero codes, signs kept


def test_w4a4_activation_row_pitch():
    # the first k columns of a wider NVFP4 tensor read in place (lda = 2k):
    # the same codes and scales a dense copy of the slice would carry
    m, n, k = 300, 272, 512
    x2 = synth.normal_bf16(m, 2 * k, 1.0, 25, 0)
    w = synth.normal_bf16(n, k, 0.02, 25, 1)
    wide = q.quantize(to_dev_bf16(x2), q.QG_FMT_NVFP4)
    packed = q.pack(q.quantize(to_dev_bf16(w), q.QG_FMT_NVFP4))
    for off in (0, k):  # left half, right half (codes + k/2 bytes, scales + k/16 bytes)
        y = torch.empty((m, n), dtype=torch.float32, device=DEV)
        q.qg_gemm(q.QG_FMT_NVFP4, wide.codes.data_ptr() + off // 2, wide.block_scales.data_ptr() + off // 16,
                  wide.tensor_scale, 2 * k, q.QG_FMT_NVFP4, packed, packed.numel(), m, n, k, y, n, q.QG_OUT_F32)
        torch.cuda.synchronize()
        qa, ba, sa = oracle.quantize_nvfp4(x2)
        qw, bw, sw = oracle.quantize_nvfp4(w)
        a_ref = oracle.dequant_nvfp4(np.ascontiguousarray(qa[:, off // 2:off // 2 + k // 2]),
                                     np.ascontiguousarray(ba[:, off // 16:off // 16 + k // 16]), sa)
        y_ref, b = oracle.gemm_f64(a_ref, oracle.dequant_nvfp4(qw, bw, sw))
        log("  lda slice at %d max err/B %.3e" % (off, check_linear(y, {"y": y_ref, "b": b})))

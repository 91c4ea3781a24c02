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
from gpu_util import DEV, check_codes, host, log, to_dev_bf16

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
@pytest.mark.parametrize("m,n,k", [(1, 16, 256), (37, 80, 512), (300, 272, 768), (129, 528, 1280)])
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


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "mxfp4"])
def test_fp8_output_transformer_shape_sampled(kind):
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

"""GPU parity of the transformer-block chain, linear by linear.

The four linears of one block run as a chain at the transformer's full
token count (M = 4608), data flowing through, exactly as the bench runs
them: QKV -> the V third of its output (attention stubbed; a strided view,
row pitch 9216) -> attention-out -> MLP-up -> GELU (torch glue) ->
MLP-down. Paper: Sec. 4, quantization paragraph; Table 2 (the linears whose
precision sets the step time).

For each linear, the activation operand's codes are compared bit for bit
with the oracle's quantization of the very bf16 tensor the GPU quantized,
and the output with the oracle's fp64 product over those operands (sampled
outputs, |y - y_ref| <= 1e-3 sum|a w|). A stage's input is the previous
stage's GPU output, which the previous check has just tied to the oracle;
the chain cannot be recomputed on the CPU from x0 alone because the next
quantization sees the bf16 rounding of a tolerance-checked product.

The static-scale chain writes the QKV and attention-out outputs as FP8 codes
in the GEMM epilogue (qg_gemm_quant), and attention-out reads the V third of
the QKV codes in place (row pitch 9216). Those codes are checked with the
rounding window: each must be a correct rounding of a value within the GEMM
contract of the oracle's exact product; the next linear is then checked
against the oracle on the decoded codes the GPU fed it."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import paper_2609_21849_amd as q
import synth
from gpu_util import (DEV, assert_quant_equal, check_codes, check_linear, check_nvfp4_codes, host, log, scale_of,
                      to_dev_bf16)

pytestmark = pytest.mark.gpu

M = synth.DIT_TOKENS
FMT = {"fp8": q.QG_FMT_FP8_E4M3, "nvfp4": q.QG_FMT_NVFP4, "mxfp4": q.QG_FMT_MXFP4, "mxfp8": q.QG_FMT_MXFP8}
NSAMPLE = 2000


@pytest.fixture(scope="module")
def block():
    x0 = synth.normal_bf16(M, 3072, 1.0, 60, 0)
    ws = {name: synth.normal_bf16(n, k, 0.02, 60, 1 + i) for i, (name, (n, k)) in enumerate(synth.DIT_LINEARS.items())}
    wd = {name: to_dev_bf16(w) for name, w in ws.items()}
    return x0, ws, wd


def bits_of(t: torch.Tensor) -> np.ndarray:
    """bf16 bit patterns of a (possibly strided) device tensor."""
    return host(t.contiguous().view(torch.int16)).view(np.uint16)


def sample(n, seed):
    rng = np.random.default_rng(seed)
    rows = np.concatenate([[0, M - 1, 0, M - 1], rng.integers(0, M, NSAMPLE)]).astype(np.int64)
    cols = np.concatenate([[0, 0, n - 1, n - 1], rng.integers(0, n, NSAMPLE)]).astype(np.int64)
    return rows, cols


def assert_codes(kind, a: q.QTensor, x_bits):
    if kind in ("fp8", "nvfp4"):
        assert_quant_equal(a, x_bits)
    else:
        codes, sc = oracle.quantize_mx(x_bits, kind)
        assert np.array_equal(host(a.codes), codes), kind
        assert np.array_equal(host(a.block_scales), sc), kind


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "mxfp4", "mxfp8"])
def test_dynamic_chain_each_linear_against_oracle(block, kind):
    x0, ws, wd = block
    fmt = FMT[kind]
    log("block chain %s M=%d" % (kind, M))
    packed = {name: q.pack(q.quantize(wd[name], fmt)) for name in ws}

    def stage(name, x_dev, x_bits, seed):
        n, k = synth.DIT_LINEARS[name]
        a = q.quantize(x_dev, fmt)            # a strided view is quantized in place (ldx = its row pitch)
        y = q.linear(a, packed[name], fmt, n)
        torch.cuda.synchronize()
        assert_codes(kind, a, x_bits)
        rows, cols = sample(n, seed)
        ref = oracle.linear_reference(kind, x_bits, ws[name], rows=rows, cols=cols)
        worst = check_linear(y, ref, rows, cols, name="chain %s %s %dx%dx%d (%d sampled)" % (kind, name, M, n, k, rows.size))
        log("  %s max err/B %.3e" % (name, worst))
        return y

    h = stage("qkv", to_dev_bf16(x0), x0, 61)
    v = h[:, 6144:9216]
    assert v.stride(0) == 9216
    a = stage("attn_out", v, bits_of(v), 62)
    u = F.gelu(stage("mlp_up", a, bits_of(a), 63), approximate="tanh")
    stage("mlp_down", u, bits_of(u), 64)


def _fp8_weight(w_bits):
    qw, sw = oracle.quantize_fp8(w_bits)
    return qw, sw


def _ref_on_codes(a_codes, s_a, w_codes, s_w, rows, cols):
    """Oracle product of FP8 codes the GPU fed a linear with the oracle's weight codes."""
    ur, ri = np.unique(rows, return_inverse=True)
    uc, ci = np.unique(cols, return_inverse=True)
    y, b = oracle.gemm_f64_sampled(oracle.dequant_fp8(a_codes[ur], s_a), oracle.dequant_fp8(w_codes[uc], s_w), ri, ci)
    return {"y": y, "b": b}


def test_static_fused_chain_each_linear_against_oracle(block):
    x0, ws, wd = block
    FP8 = q.QG_FMT_FP8_E4M3
    log("block chain fp8 static + fused epilogue quantization M=%d" % M)
    packed = {name: q.pack(q.quantize(wd[name], FP8)) for name in ws}
    wq = {name: _fp8_weight(w) for name, w in ws.items()}
    # calibration: the dynamic scales of a chain run on another batch
    xc = to_dev_bf16(synth.normal_bf16(M, 3072, 1.0, 65, 0))
    c0 = q.quantize(xc, FP8)
    hc = q.linear(c0, packed["qkv"], FP8, 9216)
    cv = q.quantize(hc[:, 6144:9216], FP8)
    ac = q.linear(cv, packed["attn_out"], FP8, 3072)
    ca = q.quantize(ac, FP8)
    uc = F.gelu(q.linear(ca, packed["mlp_up"], FP8, 9216), approximate="tanh")
    cu = q.quantize(uc, FP8)
    torch.cuda.synchronize()
    cal = {key: t.tensor_scale.clone() for key, t in (("x0", c0), ("v", cv), ("a", ca), ("u", cu))}
    s = {key: scale_of(t) for key, t in cal.items()}

    # QKV: static input quantization, output codes with the V scale
    a0 = q.quantize(to_dev_bf16(x0), FP8, static_scale=cal["x0"])
    qkv_codes = torch.empty((M, 9216), dtype=torch.uint8, device=DEV)
    q.qg_gemm_quant(FP8, a0.codes, None, a0.tensor_scale, 3072, FP8, packed["qkv"], packed["qkv"].numel(),
                    M, 9216, 3072, qkv_codes, 9216, cal["v"])
    # attention-out reads the V third of the QKV codes in place (row pitch 9216)
    ao_codes = torch.empty((M, 3072), dtype=torch.uint8, device=DEV)
    q.qg_gemm_quant(FP8, qkv_codes.data_ptr() + 6144, None, cal["v"], 9216, FP8, packed["attn_out"],
                    packed["attn_out"].numel(), M, 3072, 3072, ao_codes, 3072, cal["a"])
    y_up = q.linear(q.QTensor(FP8, ao_codes, None, cal["a"], M, 3072), packed["mlp_up"], FP8, 9216)
    u = F.gelu(y_up, approximate="tanh")
    au = q.quantize(u, FP8, static_scale=cal["u"])
    y = q.linear(au, packed["mlp_down"], FP8, 3072)
    torch.cuda.synchronize()

    a0_ref = oracle.quantize_fp8_static(x0, s["x0"])
    assert np.array_equal(host(a0.codes), a0_ref)
    rows, cols = sample(9216, 66)
    ref = _ref_on_codes(a0_ref, s["x0"], *wq["qkv"], rows, cols)
    r_v = np.float32(1.0) / s["v"]
    uniq = check_codes(host(qkv_codes), ref, r_v, rows, cols)
    log("  qkv fused FP8 codes within the contract (%.3f unique roundings)" % uniq)

    codes_v = np.ascontiguousarray(host(qkv_codes)[:, 6144:9216])
    rows, cols = sample(3072, 67)
    ref = _ref_on_codes(codes_v, s["v"], *wq["attn_out"], rows, cols)
    uniq = check_codes(host(ao_codes), ref, np.float32(1.0) / s["a"], rows, cols)
    log("  attn_out (V slice at row pitch 9216) fused FP8 codes within the contract (%.3f unique)" % uniq)

    rows, cols = sample(9216, 68)
    ref = _ref_on_codes(host(ao_codes), s["a"], *wq["mlp_up"], rows, cols)
    log("  mlp_up max err/B %.3e" % check_linear(y_up, ref, rows, cols,
                                                 name="chain fp8 static-fused mlp_up %dx9216x3072 (%d sampled)" % (M, rows.size)))

    u_bits = bits_of(u)
    au_ref = oracle.quantize_fp8_static(u_bits, s["u"])
    assert np.array_equal(host(au.codes), au_ref)
    rows, cols = sample(3072, 69)
    ref = _ref_on_codes(au_ref, s["u"], *wq["mlp_down"], rows, cols)
    log("  mlp_down max err/B %.3e" % check_linear(y, ref, rows, cols,
                                                   name="chain fp8 static-fused mlp_down %dx3072x9216 (%d sampled)" % (M, rows.size)))


def test_static_fused_nvfp4_chain_each_linear_against_oracle(block):
    """The NVFP4 chain with calibrated tensor scales: QKV and attention-out
    write NVFP4 codes and block scales in their epilogues, attention-out
    reads the V third of the QKV codes in place (row pitch 9216 elements:
    codes + 3072 bytes, block scales + 384 bytes). Whole sampled rows (the
    block scales span 16 columns) are held to the NVFP4 rounding window; the
    next linear is checked on the decoded codes the GPU fed it."""
    x0, ws, wd = block
    NV = q.QG_FMT_NVFP4
    log("block chain nvfp4 static + fused epilogue quantization M=%d" % M)
    packed = {name: q.pack(q.quantize(wd[name], NV)) for name in ws}
    wq = {name: oracle.quantize_nvfp4(w) for name, w in ws.items()}
    xc = to_dev_bf16(synth.normal_bf16(M, 3072, 1.0, 65, 0))
    c0 = q.quantize(xc, NV)
    hc = q.linear(c0, packed["qkv"], NV, 9216)
    cv = q.quantize(hc[:, 6144:9216], NV)
    ac = q.linear(cv, packed["attn_out"], NV, 3072)
    ca = q.quantize(ac, NV)
    uc = F.gelu(q.linear(ca, packed["mlp_up"], NV, 9216), approximate="tanh")
    cu = q.quantize(uc, NV)
    torch.cuda.synchronize()
    cal = {key: t.tensor_scale.clone() for key, t in (("x0", c0), ("v", cv), ("a", ca), ("u", cu))}
    s = {key: scale_of(t) for key, t in cal.items()}

    a0 = q.quantize(to_dev_bf16(x0), NV, static_scale=cal["x0"])
    qkv = (torch.empty((M, 4608), dtype=torch.uint8, device=DEV), torch.empty((M, 576), dtype=torch.uint8, device=DEV))
    q.qg_gemm_quant_nvfp4(NV, a0.codes, a0.block_scales, a0.tensor_scale, 3072, NV, packed["qkv"],
                          packed["qkv"].numel(), M, 9216, 3072, qkv[0], qkv[1], 9216, cal["v"])
    ao = (torch.empty((M, 1536), dtype=torch.uint8, device=DEV), torch.empty((M, 192), dtype=torch.uint8, device=DEV))
    q.qg_gemm_quant_nvfp4(NV, qkv[0].data_ptr() + 3072, qkv[1].data_ptr() + 384, cal["v"], 9216, NV,
                          packed["attn_out"], packed["attn_out"].numel(), M, 3072, 3072, ao[0], ao[1], 3072, cal["a"])
    y_up = q.linear(q.QTensor(NV, ao[0], ao[1], cal["a"], M, 3072), packed["mlp_up"], NV, 9216)
    u = F.gelu(y_up, approximate="tanh")
    au = q.quantize(u, NV, static_scale=cal["u"])
    y = q.linear(au, packed["mlp_down"], NV, 3072)
    torch.cuda.synchronize()

    def ref_rows(a_codes, a_bs, s_a, name, rows):
        n = synth.DIT_LINEARS[name][0]
        qw, bw, sw = wq[name]
        y_ref, b = oracle.gemm_f64(oracle.dequant_nvfp4(a_codes[rows], a_bs[rows], s_a), oracle.dequant_nvfp4(qw, bw, sw))
        return {"y": y_ref.reshape(rows.size, n), "b": b.reshape(rows.size, n)}

    rng = np.random.default_rng(70)
    a0c, a0b = oracle.quantize_nvfp4_static(x0, s["x0"])
    assert np.array_equal(host(a0.codes), a0c) and np.array_equal(host(a0.block_scales), a0b)
    rows = np.sort(rng.choice(M, 24, replace=False))
    uniq = check_nvfp4_codes(host(qkv[0])[rows], host(qkv[1])[rows], ref_rows(a0c, a0b, s["x0"], "qkv", rows), s["v"])
    log("  qkv fused NVFP4 output within the contract (%.3f unique block scales)" % uniq)

    vc = np.ascontiguousarray(host(qkv[0])[:, 3072:4608])
    vb = np.ascontiguousarray(host(qkv[1])[:, 384:576])
    rows = np.sort(rng.choice(M, 24, replace=False))
    uniq = check_nvfp4_codes(host(ao[0])[rows], host(ao[1])[rows], ref_rows(vc, vb, s["v"], "attn_out", rows), s["a"])
    log("  attn_out (V slice, row pitch 9216) fused NVFP4 output within the contract (%.3f unique)" % uniq)

    rows, cols = sample(9216, 71)
    aoc, aob = host(ao[0]), host(ao[1])
    qw, bw, sw = wq["mlp_up"]
    ur, ri = np.unique(rows, return_inverse=True)
    uc_, ci = np.unique(cols, return_inverse=True)
    yr, b = oracle.gemm_f64_sampled(oracle.dequant_nvfp4(aoc[ur], aob[ur], s["a"]),
                                    oracle.dequant_nvfp4(qw[uc_], bw[uc_], sw), ri, ci)
    log("  mlp_up max err/B %.3e" % check_linear(y_up, {"y": yr, "b": b}, rows, cols,
                                                 name="chain nvfp4 static-fused mlp_up %dx9216x3072 (%d sampled)" % (M, rows.size)))
    u_bits = bits_of(u)
    auc, aub = oracle.quantize_nvfp4_static(u_bits, s["u"])
    assert np.array_equal(host(au.codes), auc) and np.array_equal(host(au.block_scales), aub)
    rows, cols = sample(3072, 72)
    qw, bw, sw = wq["mlp_down"]
    ur, ri = np.unique(rows, return_inverse=True)
    uc_, ci = np.unique(cols, return_inverse=True)
    yr, b = oracle.gemm_f64_sampled(oracle.dequant_nvfp4(auc[ur], aub[ur], s["u"]),
                                    oracle.dequant_nvfp4(qw[uc_], bw[uc_], sw), ri, ci)
    log("  mlp_down max err/B %.3e" % check_linear(y, {"y": yr, "b": b}, rows, cols,
                                                   name="chain nvfp4 static-fused mlp_down %dx3072x9216 (%d sampled)" % (M, rows.size)))

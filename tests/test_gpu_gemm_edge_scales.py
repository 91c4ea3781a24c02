"""GEMMs whose operands carry E4M3-subnormal and zero NVFP4 block scales.

Rows of the activations and of the weights are scaled down by 2^-12 ...
2^-35 (one factor per row, cycling), so that, against a tensor scale set by
the rows left at full size, their block scales run through normal, subnormal
(codes 1..7, k * 2^-9) and zero (code 0) E4M3 values. Every kernel that
decodes block scales is driven through such operands at a workload shape:
the persistent 256 x 256 W4A4 kernel (transformer linear), the small-token
W4A4 kernels (512 x 3072 x 3072), and the W4A16 split-K, few-row streaming,
one-row matrix-vector and large-M kernels. Outputs are checked against the
oracle: fp32 outputs with the literal bound |y - y_ref| <= 1e-3 sum|a w|,
bf16 outputs with the rounding window (a correct rounding of a value within
that bound: the shrunken rows keep only a few nonzero terms, where the bf16
rounding alone can exceed the bound); rows whose block scales are all zero
must come out exactly zero."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_21849_amd as q
import synth
from gpu_util import check_linear, log, to_dev_bf16

pytestmark = pytest.mark.gpu

NV, BF16 = q.QG_FMT_NVFP4, q.QG_FMT_BF16


def shrink_rows(bits: np.ndarray, first: int) -> np.ndarray:
    """Rows first.. multiplied by 2^-(12 + (i - first) % 24)."""
    v = synth.bf16_bits_to_f32(bits).astype(np.float64)
    r = np.arange(bits.shape[0] - first)
    v[first:] *= (2.0 ** -(12 + r % 24))[:, None]
    return synth.f32_to_bf16_bits(v.astype(np.float32))


def scale_classes(bits: np.ndarray) -> dict:
    _, bs, _ = oracle.quantize_nvfp4(bits)
    return {"normal": int(np.count_nonzero(bs >= 8)), "subnormal": int(np.count_nonzero((bs >= 1) & (bs < 8))),
            "zero": int(np.count_nonzero(bs == 0))}


def sample(m, n, count, seed, extra_rows=()):
    rng = np.random.default_rng(seed)
    rows = np.concatenate([[0, m - 1, 0, m - 1], list(extra_rows), rng.integers(0, m, count)])
    cols = np.concatenate([[0, 0, n - 1, n - 1], rng.integers(0, n, len(extra_rows) + count)])
    return rows.astype(np.int64), cols.astype(np.int64)


def run(kind, x, w, out):
    xd, wd = to_dev_bf16(x), to_dev_bf16(w)
    packed = q.pack(q.quantize(wd, NV))
    a = xd if kind == "w4a16" else q.quantize(xd, NV)
    y = q.linear(a, packed, NV, w.shape[0], out_dtype=out)
    torch.cuda.synchronize()
    return y


@pytest.mark.parametrize("m,n,k,label", [(4608, 3072, 3072, "256x256 kernel, transformer attn-out"),
                                         (512, 3072, 3072, "small-token kernel, 512x3072x3072"),
                                         (96, 1024, 3072, "small-token kernel, few rows")])
@pytest.mark.parametrize("out", [q.QG_OUT_F32, q.QG_OUT_BF16])
def test_w4a4_subnormal_and_zero_block_scales(m, n, k, label, out):
    log("w4a4 edge scales %s %dx%dx%d out=%d" % (label, m, n, k, out))
    x = shrink_rows(synth.normal_bf16(m, k, 1.0, 50, 0, outlier_frac=0.001, outlier_gain=50.0), m // 4)
    w = shrink_rows(synth.normal_bf16(n, k, 0.02, 50, 1), n // 4)
    cx, cw = scale_classes(x), scale_classes(w)
    log("  activation block scales", cx, "weight block scales", cw)
    assert min(cx.values()) > 0 and min(cw.values()) > 0
    y = run("nvfp4", x, w, out)
    # the first shrunken rows of each 24-row cycle span normal -> zero scales
    extra = [m // 4 + i for i in range(24)]
    rows, cols = sample(m, n, 3000, 51, extra)
    ref = oracle.linear_reference("nvfp4", x, w, rows=rows, cols=cols)
    log("  max err/B", check_linear(y, ref, rows, cols, literal=False,
                                    name="nvfp4 w4a4 subnormal/zero block scales %dx%dx%d %s" % (m, n, k, "f32" if out else "bf16")))
    # an activation row whose block scales are all zero gives a zero output row
    _, bs, _ = oracle.quantize_nvfp4(x)
    zero_rows = np.flatnonzero((bs == 0).all(axis=1))
    assert zero_rows.size > 0
    assert not torch.any(y[torch.as_tensor(zero_rows, device=y.device)]).item()


@pytest.mark.parametrize("m,n,k,label", [(256, 3072, 1024, "split-K, two panels per workgroup"),
                                         (16, 1024, 3072, "split-K, direct activation fragments"),
                                         (16, 70016, 1024, "few-row streaming kernel"),
                                         (1, 70016, 1024, "one-row matrix-vector kernel"),
                                         (1100, 512, 1024, "large-M kernel")])
@pytest.mark.parametrize("out", [q.QG_OUT_F32, q.QG_OUT_BF16])
def test_w4a16_subnormal_and_zero_block_scales(m, n, k, label, out):
    log("w4a16 edge scales %s %dx%dx%d out=%d" % (label, m, n, k, out))
    x = synth.normal_bf16(m, k, 1.0, 52, 0)
    if m > 4:
        x = shrink_rows(x, m // 2)
    w = shrink_rows(synth.normal_bf16(n, k, 0.02, 52, 1), n // 4)
    cw = scale_classes(w)
    log("  weight block scales", cw)
    assert min(cw.values()) > 0
    y = run("w4a16", x, w, out)
    if m * n <= 400_000:
        ref = oracle.linear_reference("w4a16", x, w)
        rows = cols = None
    else:
        rows, cols = sample(m, n, 3000, 53)
        # and the output columns of the shrunken weight rows of the first cycle
        rows = np.concatenate([rows, np.arange(24) % m]).astype(np.int64)
        cols = np.concatenate([cols, n // 4 + np.arange(24)]).astype(np.int64)
        ref = oracle.linear_reference("w4a16", x, w, rows=rows, cols=cols)
    log("  max err/B", check_linear(y, ref, rows, cols, literal=False,
                                    name="w4a16 subnormal/zero block scales %dx%dx%d %s" % (m, n, k, "f32" if out else "bf16")))
    # a weight row whose block scales are all zero gives a zero output column
    _, bs, _ = oracle.quantize_nvfp4(w)
    zero_cols = np.flatnonzero((bs == 0).all(axis=1))
    assert zero_cols.size > 0
    assert not torch.any(y[:, torch.as_tensor(zero_cols, device=y.device)]).item()

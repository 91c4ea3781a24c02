"""GPU parity over seeded random shapes: every GEMM path that the dispatch
can choose for few to a few hundred tokens (split-K FP8 and NVFP4 tilings,
the W4A16 split-K / stream / direct kernels, the fused FP8 linear), each
output against the oracle's exact product of the same quantized operands.
The shapes are drawn across the dispatch boundaries (M from 1 to 700, N a
multiple of 16 up to 2400, K a multiple of 128 up to 2048), so a tiling
rule that mishandles a ragged edge or a row/column bound shows up here."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_21849_amd as q
import synth
from gpu_util import check_linear, host, log, to_dev_bf16

pytestmark = pytest.mark.gpu

FP8, NVFP4, BF16 = q.QG_FMT_FP8_E4M3, q.QG_FMT_NVFP4, q.QG_FMT_BF16
KINDS = {"fp8": (FP8, FP8), "nvfp4": (NVFP4, NVFP4), "w4a16": (BF16, NVFP4)}


def _shapes(seed, count):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        m = int(rng.choice([rng.integers(1, 33), rng.integers(33, 257), rng.integers(257, 701)]))
        n = 16 * int(rng.integers(1, 151))
        k = 128 * int(rng.integers(1, 17))
        out.append((m, n, k))
    return out


SHAPES = _shapes(2026, 14)


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "w4a16"])
@pytest.mark.parametrize("m,n,k", SHAPES)
def test_random_shape_parity(kind, m, n, k):
    log("random shape kind=%s m=%d n=%d k=%d" % (kind, m, n, k))
    seed = (m * 7919 + n * 31 + k) % 1000
    x = synth.normal_bf16(m, k, 1.0, seed, 0, outlier_frac=0.002, outlier_gain=30.0)
    w = synth.normal_bf16(n, k, 0.02, seed, 1)
    a_fmt, w_fmt = KINDS[kind]
    xd = to_dev_bf16(x)
    packed = q.pack(q.quantize(to_dev_bf16(w), w_fmt))
    a = xd if a_fmt == BF16 else q.quantize(xd, a_fmt)
    y = q.linear(a, packed, w_fmt, n, out_dtype=q.QG_OUT_F32)
    torch.cuda.synchronize()
    ref = oracle.linear_reference(kind, x, w)
    check_linear(y, ref)
    if kind == "fp8" and m * k <= 65536:
        # the one-launch linear (these draws all take a split-K tiling that
        # qg_gemm shares): the same output bits
        yf, _ = q.linear_fp8(xd, packed, n, q.QG_OUT_F32)
        torch.cuda.synchronize()
        assert np.array_equal(host(yf).view(np.uint32), host(y).view(np.uint32))


def _large_shapes(seed, count):
    rng = np.random.default_rng(seed)
    return [(int(rng.integers(701, 3300)), 16 * int(rng.integers(40, 260)), 128 * int(rng.integers(1, 25)))
            for _ in range(count)]


def _edge_samples(m, n, count, seed):
    # random outputs plus the rows and columns at every 256-, 288- and
    # 192-wide tile edge (the large kernels' tilings)
    rng = np.random.default_rng(seed)
    er = sorted({min(v, m - 1) for t in (256, 288, 64, 32) for b in range(t, m + t, t) for v in (b - 1, b)} | {0})
    ec = sorted({min(v, n - 1) for t in (256, 192, 128, 32) for b in range(t, n + t, t) for v in (b - 1, b)} | {0})
    rows = np.concatenate([rng.integers(0, m, count), rng.choice(er, count), rng.integers(0, m, len(ec))])
    cols = np.concatenate([rng.choice(ec, count), rng.integers(0, n, count), np.array(ec)])
    return rows, cols


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "w4a16"])
@pytest.mark.parametrize("m,n,k", _large_shapes(2027, 6))
def test_random_large_shape_parity(kind, m, n, k):
    # the many-token kernels (256 x 256, 288 x 192, 64 x 128 tiles and the
    # W4A16 direct kernel) at ragged sizes, on sampled outputs at tile edges
    log("random large shape kind=%s m=%d n=%d k=%d" % (kind, m, n, k))
    seed = (m * 131 + n * 17 + k) % 1000
    x = synth.normal_bf16(m, k, 1.0, seed, 0, outlier_frac=0.002, outlier_gain=30.0)
    w = synth.normal_bf16(n, k, 0.02, seed, 1)
    a_fmt, w_fmt = KINDS[kind]
    xd = to_dev_bf16(x)
    packed = q.pack(q.quantize(to_dev_bf16(w), w_fmt))
    a = xd if a_fmt == BF16 else q.quantize(xd, a_fmt)
    y = q.linear(a, packed, w_fmt, n, out_dtype=q.QG_OUT_BF16)
    torch.cuda.synchronize()
    rows, cols = _edge_samples(m, n, 600, seed)
    # bf16 outputs held to the rounding window (short reductions leave many
    # outputs within a rounding step of the bound)
    check_linear(y, oracle.linear_reference(kind, x, w, rows, cols), rows, cols, literal=False)

"""Helpers shared by the GPU parity tests: moving the seeded bf16 bit
patterns to the device and comparing device results with the oracle."""
import sys

import numpy as np
import torch

import oracle
import paper_2609_21849_amd as q
import synth

DEV = torch.device("cuda:0")


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev_bf16(x_bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.array(x_bits, dtype=np.uint16, copy=True, order="C").view(np.int16)).view(torch.bfloat16).to(DEV)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def scale_of(t: torch.Tensor) -> np.float32:
    return np.float32(host(t)[0])


def assert_quant_equal(qt: q.QTensor, x_bits: np.ndarray):
    """Codes, block scales and tensor-scale bits must equal the oracle's."""
    if qt.fmt == q.QG_FMT_FP8_E4M3:
        codes, s = oracle.quantize_fp8(x_bits)
        got = host(qt.codes)
        assert got.shape == codes.shape
        nbad = int(np.count_nonzero(got != codes))
        assert nbad == 0, "fp8 codes differ at %d of %d" % (nbad, codes.size)
    else:
        codes, bs, s = oracle.quantize_nvfp4(x_bits)
        got = host(qt.codes)
        nbad = int(np.count_nonzero(got != codes))
        assert nbad == 0, "nvfp4 codes differ at %d of %d" % (nbad, codes.size)
        nbs = int(np.count_nonzero(host(qt.block_scales) != bs))
        assert nbs == 0, "nvfp4 block scales differ at %d of %d" % (nbs, bs.size)
    got_s = scale_of(qt.tensor_scale)
    assert got_s.view(np.uint32) == np.float32(s).view(np.uint32), (got_s, s)


def check_linear(y_dev: torch.Tensor, ref: dict, rows=None, cols=None, tol=1e-3):
    """|y - y_ref| <= tol * sum|a w| everywhere (or at the sampled outputs).

    fp32 outputs get exactly that bound. A bf16 output v' = bf16(v) of an
    fp32 value v within the bound adds the output rounding:
    |v' - y_ref| <= 2^-9 |v| + |v - y_ref| <= 2^-9 |y_ref| + (1 + 2^-9) tol * b.
    """
    y = host(y_dev.float()).astype(np.float64)
    if rows is not None:
        y = y[rows, cols]
    err = np.abs(y - ref["y"])
    bound = tol * ref["b"]
    if y_dev.dtype == torch.bfloat16:
        bound = (1 + 2.0 ** -9) * bound + 2.0 ** -9 * np.abs(ref["y"])
    worst = float(np.max(err / np.maximum(ref["b"], 1e-300)))
    assert np.all(err <= bound), "max err / sum|aw| = %.3e" % worst
    return worst

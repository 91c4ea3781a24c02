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


def order_key(codes: np.ndarray) -> np.ndarray:
    """E4M3 codes (sign-magnitude) to integers in value order (-0 and +0 equal)."""
    c = codes.astype(np.int32)
    mag = c & 0x7F
    return np.where(c & 0x80, -mag, mag)


def check_codes(codes, ref, r, rows=None, cols=None, tol=1e-3):
    y, b = ref["y"], ref["b"]
    e = tol * b * (1 + 2.0 ** -20) + 1e-300
    lo = oracle.e4m3_encode_array(((y - e) * r).astype(np.float32))
    hi = oracle.e4m3_encode_array(((y + e) * r).astype(np.float32))
    got = codes if rows is None else codes[rows, cols]
    k, klo, khi = order_key(got), order_key(lo), order_key(hi)
    bad = np.count_nonzero((k < klo) | (k > khi))
    assert bad == 0, "%d of %d codes outside the contract" % (bad, k.size)
    # most codes are the unique rounding (the window holds one code)
    return float(np.mean(klo == khi))


# max err / sum|a w| per named workload case, written out at the end of the
# session when QG_PARITY_LOG names a file (tests/conftest.py)
MARGINS = {}


def bf16_rne(v: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value, ties to even, in one
    rounding (no pass through fp32); returned as float64. bf16 keeps 8
    significant bits, so ulp(v) = 2^(floor(log2 |v|) - 7)."""
    v = np.asarray(v, dtype=np.float64)
    out = np.zeros_like(v)
    nz = (v != 0) & np.isfinite(v)
    e = np.floor(np.log2(np.abs(v[nz])))
    # log2 can land one off at exact powers of two: fix the exponent so that
    # 2^e <= |v| < 2^(e+1)
    e = np.where(np.abs(v[nz]) < 2.0 ** e, e - 1, e)
    e = np.where(np.abs(v[nz]) >= 2.0 ** (e + 1), e + 1, e)
    e = np.maximum(e, -133.0)                           # bf16 subnormal grid below 2^-126
    ulp = 2.0 ** (np.maximum(e, -126.0) - 7)
    out[nz] = np.rint(v[nz] / ulp) * ulp                 # exact scaling, rint ties to even
    out[~np.isfinite(v)] = v[~np.isfinite(v)]
    return out


def check_linear(y_dev: torch.Tensor, ref: dict, rows=None, cols=None, tol=1e-3, literal=True, name=None):
    """The GEMM accuracy contract against the oracle's exact product y_ref,
    at every output (or at the sampled ones), with b = sum_k |a w|:

      fp32 output: |y - y_ref| <= tol * b.
      bf16 output: y must be the round-to-nearest-even bf16 of some value
        within tol * b of y_ref, i.e. bf16(y_ref - tol b) <= y <=
        bf16(y_ref + tol b) (rounding is monotone); and, with literal=True,
        |y - y_ref| <= tol * b itself at every output where the correctly
        rounded exact product bf16(y_ref) meets that bound. Where it does not
        (|y_ref| large against b, so that the bf16 rounding alone, up to
        2^-8 |y|, exceeds tol * b) no bf16 output can meet it; those outputs
        are counted in the recorded margins.
    literal=False is for unit cases with few reduction terms, where many
    outputs sit within a bf16 rounding step of the bound and the GEMM's own
    fp32 error may legitimately flip the rounding across it.
    """
    y = host(y_dev.float()).astype(np.float64)
    if rows is not None:
        y = y[rows, cols]
    yr, b = ref["y"], ref["b"]
    err = np.abs(y - yr)
    bound = tol * b
    worst = float(np.max(err / np.maximum(b, 1e-300))) if err.size else 0.0
    unreachable = 0
    if y_dev.dtype == torch.bfloat16:
        lo, hi = bf16_rne(yr - bound), bf16_rne(yr + bound)
        nbad = int(np.count_nonzero((y < lo) | (y > hi)))
        assert nbad == 0, "%d outputs are not a bf16 rounding of a value within the bound (max err/B %.3e)" % (nbad, worst)
        reach = np.abs(bf16_rne(yr) - yr) <= bound
        unreachable = int(np.count_nonzero(~reach))
        if literal:
            nlit = int(np.count_nonzero(err[reach] > bound[reach]))
            assert nlit == 0, "%d outputs beyond %.0e sum|aw| (max err/B %.3e)" % (nlit, tol, worst)
    else:
        assert np.all(err <= bound), "max err / sum|aw| = %.3e" % worst
    if name is not None:
        MARGINS[name] = {"max_err_over_sum_abs_aw": worst, "bound": tol, "outputs_checked": int(err.size),
                         "dtype": str(y_dev.dtype).replace("torch.", ""),
                         "outputs_where_bf16_rounding_alone_exceeds_bound": unreachable}
    return worst


def _f32_down(x):
    v = np.asarray(x, dtype=np.float64).astype(np.float32)
    return np.where(v.astype(np.float64) > x, np.nextafter(v, np.float32(-np.inf)), v).astype(np.float32)


def _f32_up(x):
    v = np.asarray(x, dtype=np.float64).astype(np.float32)
    return np.where(v.astype(np.float64) < x, np.nextafter(v, np.float32(np.inf)), v).astype(np.float32)


def _e2m1_key(c):
    c = c.astype(np.int32)
    mag = c & 7
    return np.where(c & 8, -mag, mag)


def check_nvfp4_codes(codes, bscales, ref, s_t, tol=1e-3):
    """NVFP4 output of a GEMM epilogue against the oracle's exact product
    y_ref (rows of whole 16-blocks): every block scale and code must be a
    correct rounding (the static NVFP4 steps in fp32) for some output y' with
    |y' - y_ref| <= tol * sum|a w| elementwise. Sound bounds: the block scale
    lies between the scales of the smallest and largest possible block max,
    and, given the block scale actually chosen, each code lies between the
    codes of the smallest and largest possible element. Returns the share of
    blocks whose scale window holds a single code."""
    y, b = ref["y"], ref["b"]
    rows, n = y.shape
    e = tol * b * (1 + 2.0 ** -20) + 1e-300
    s_t = np.float32(s_t)
    d = np.float32(np.float32(6.0) * s_t)
    lo_abs = np.maximum(np.abs(y) - e, 0.0).reshape(rows, n // 16, 16).max(axis=2)
    hi_abs = (np.abs(y) + e).reshape(rows, n // 16, 16).max(axis=2)
    if d > 0:
        v_lo, v_hi = _f32_down(lo_abs) / d, _f32_up(hi_abs) / d
    else:
        v_lo = v_hi = np.zeros_like(lo_abs, dtype=np.float32)
    sb_lo = oracle.e4m3_encode_array(v_lo.astype(np.float32))
    sb_hi = oracle.e4m3_encode_array(v_hi.astype(np.float32))
    bad = np.count_nonzero((bscales < sb_lo) | (bscales > sb_hi))
    assert bad == 0, "%d of %d block scales outside the contract" % (bad, bscales.size)
    S = (oracle.e4m3_table()[bscales].astype(np.float32) * s_t).astype(np.float32)
    r = np.where(S > 0, np.float32(1.0) / np.where(S > 0, S, np.float32(1.0)), np.float32(0.0)).astype(np.float32)
    rr = np.repeat(r, 16, axis=1)
    c_lo = oracle.e2m1_encode_array((_f32_down(y - e) * rr).astype(np.float32))
    c_hi = oracle.e2m1_encode_array((_f32_up(y + e) * rr).astype(np.float32))
    got = np.empty((rows, n), dtype=np.uint8)
    got[:, 0::2] = codes & 0xF
    got[:, 1::2] = codes >> 4
    k, klo, khi = _e2m1_key(got), _e2m1_key(c_lo), _e2m1_key(c_hi)
    badc = np.count_nonzero((k < klo) | (k > khi))
    assert badc == 0, "%d of %d codes outside the contract" % (badc, k.size)
    return float(np.mean(sb_lo == sb_hi))

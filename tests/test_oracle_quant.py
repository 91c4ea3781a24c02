"""Pins for the oracle's FP8 and NVFP4 quantizers and dequantizers (CPU only).

What pins them, none of it the oracle's own arithmetic retyped:
  * hand-derived worked examples (tests/golden/worked_examples.json);
  * a closed form: tensors built as exact dequantized values, whose scales are
    then exact, must quantize back to the codes they were built from;
  * invariants of the recipe: scaling by 2^k, sign symmetry, row permutation,
    block maxima landing on the top code, all-zero and non-finite tensors;
  * the formats' rounding-error bounds on random data;
  * torch's float8_e4m3fn decoder for FP8 dequantization.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")
E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0])


def _torch_e4m3(codes: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(codes, np.uint8)).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def _bf16(v) -> np.ndarray:
    x = np.asarray(v, dtype=np.float32)
    b = synth.f32_to_bf16_bits(x)
    assert np.array_equal(synth.bf16_bits_to_f32(b), x), "input must be exact in bf16"
    return b


def _unpack(codes: np.ndarray) -> np.ndarray:
    out = np.empty((codes.shape[0], codes.shape[1] * 2), dtype=np.uint8)
    out[:, 0::2] = codes & 15
    out[:, 1::2] = codes >> 4
    return out


# ------------------------------------------------------------ worked examples
def test_fp8_worked_example():
    g = json.load(open(GOLDEN))["fp8"]
    codes, s = oracle.quantize_fp8(_bf16(g["x"])[None, :])
    assert s == np.float32(g["scale"])
    assert codes[0].tolist() == g["codes"]


def test_nvfp4_worked_example():
    g = json.load(open(GOLDEN))["nvfp4"]
    codes, bs, st = oracle.quantize_nvfp4(_bf16(g["x"])[None, :])
    assert st == np.float32(g["tensor_scale"])
    assert bs[0].tolist() == g["block_scales"]
    assert _unpack(codes)[0].tolist() == g["element_codes"]


# ------------------------------------------------------------ closed form
def _nvfp4_image(rows, cols, p, seed):
    """A tensor that is exactly the dequantization of chosen codes/scales.

    Block scales are random E4M3 values in [2^-6, 448] with one block at 448,
    and every block holds a +-6 element, so a_b = 6*dec(s_b)*2^p. The tensor
    scale is then s_t = 6*448*2^p/2688 = 2^p exactly, v_b = dec(s_b) exactly,
    and the quantizer must give back exactly the chosen codes and scales.
    """
    rng = np.random.default_rng(seed)
    nb = cols // 16
    sb = rng.integers(0x08, 0x7F, size=(rows, nb)).astype(np.uint8)   # normal E4M3 codes 2^-6..448
    sb[0, 0] = 0x7E
    q = rng.integers(0, 16, size=(rows, cols)).astype(np.uint8)
    pos = rng.integers(0, 16, size=(rows, nb))
    for r in range(rows):
        for b in range(nb):
            q[r, b * 16 + pos[r, b]] = 7 | (8 * rng.integers(0, 2))
    scale = _torch_e4m3(sb) * 2.0 ** p
    x = E2M1[q] * np.repeat(scale, 16, axis=1)
    return _bf16(x), q, sb


@pytest.mark.parametrize("p", [-12, -3, 0, 5])
def test_nvfp4_quantize_inverts_exact_dequant(p):
    x, q, sb = _nvfp4_image(8, 128, p, seed=100 + p)
    codes, bs, st = oracle.quantize_nvfp4(x)
    assert st == np.float32(2.0 ** p)
    assert np.array_equal(bs, sb)
    got = _unpack(codes)
    # -0 and +0 both dequantize to 0; the quantizer keeps the sign of x, and x = -0.0 where q == 8
    assert np.array_equal(got, q)


def test_fp8_quantize_inverts_exact_dequant():
    rng = np.random.default_rng(5)
    q = rng.integers(0, 256, size=(16, 64)).astype(np.uint8)
    q[(q & 0x7F) == 0x7F] = 0x7E                       # no NaN codes
    q[0, 0] = 0x7E                                     # amax = 448 * s
    s = 2.0 ** -4
    x = _bf16(_torch_e4m3(q) * s)
    codes, scale = oracle.quantize_fp8(x)
    assert scale == np.float32(s)
    assert np.array_equal(codes, q)


# ------------------------------------------------------------ invariants
def _data(rows=32, cols=256, seed=0, sigma=1.0, frac=0.0):
    return synth.normal_bf16(rows, cols, sigma, seed, 0, outlier_frac=frac, outlier_gain=50.0)


def _scale_bf16(x, k):
    return _bf16(synth.bf16_bits_to_f32(x).astype(np.float64) * 2.0 ** k)


@pytest.mark.parametrize("k", [-7, 3])
def test_power_of_two_scaling(k):
    x = _data()
    xs = _scale_bf16(x, k)
    c8, s8 = oracle.quantize_fp8(x)
    c8s, s8s = oracle.quantize_fp8(xs)
    assert np.array_equal(c8, c8s) and s8s == np.float32(s8 * 2.0 ** k)
    c4, b4, t4 = oracle.quantize_nvfp4(x)
    c4s, b4s, t4s = oracle.quantize_nvfp4(xs)
    assert np.array_equal(c4, c4s) and np.array_equal(b4, b4s) and t4s == np.float32(t4 * 2.0 ** k)


def test_sign_symmetry():
    x = _data(seed=3)
    xn = x ^ np.uint16(0x8000)
    c8, s8 = oracle.quantize_fp8(x)
    c8n, s8n = oracle.quantize_fp8(xn)
    assert s8 == s8n and np.array_equal(c8n, c8 ^ 0x80)
    c4, b4, t4 = oracle.quantize_nvfp4(x)
    c4n, b4n, t4n = oracle.quantize_nvfp4(xn)
    assert t4 == t4n and np.array_equal(b4, b4n) and np.array_equal(c4n, c4 ^ 0x88)


def test_row_permutation():
    x = _data(seed=4)
    perm = np.random.default_rng(0).permutation(x.shape[0])
    c8, _ = oracle.quantize_fp8(x)
    c8p, _ = oracle.quantize_fp8(x[perm])
    assert np.array_equal(c8p, c8[perm])
    c4, b4, _ = oracle.quantize_nvfp4(x)
    c4p, b4p, _ = oracle.quantize_nvfp4(x[perm])
    assert np.array_equal(c4p, c4[perm]) and np.array_equal(b4p, b4[perm])


def test_block_max_lands_on_top_code():
    """The largest element of a block maps into [5.625, 6.375] before rounding
    whenever its block scale is a normal E4M3 value, so it encodes to +-6; the
    tensor's largest element encodes to +-448 in FP8."""
    x = _data(rows=64, cols=512, seed=6, frac=0.01)
    xf = synth.bf16_bits_to_f32(x)
    c4, b4, _ = oracle.quantize_nvfp4(x)
    e = _unpack(c4)
    checked = 0
    for r in range(x.shape[0]):
        for b in range(x.shape[1] // 16):
            if b4[r, b] < 0x08:
                continue
            blk = np.abs(xf[r, b * 16:(b + 1) * 16])
            j = int(blk.argmax())
            assert e[r, b * 16 + j] & 7 == 7
            checked += 1
    assert checked > 1000
    c8, _ = oracle.quantize_fp8(x)
    i = np.unravel_index(np.abs(xf).argmax(), xf.shape)
    assert c8[i] & 0x7F == 0x7E


def test_zero_tensor_and_signed_zeros():
    x = np.zeros((4, 32), dtype=np.uint16)
    x[1, 3] = 0x8000                                   # -0.0
    c8, s8 = oracle.quantize_fp8(x)
    assert s8 == 0.0 and c8[1, 3] == 0x80 and np.count_nonzero(c8) == 1
    c4, b4, t4 = oracle.quantize_nvfp4(x)
    assert t4 == 0.0 and not b4.any()
    assert _unpack(c4)[1, 3] == 8 and np.count_nonzero(_unpack(c4)) == 1


@pytest.mark.parametrize("bad", [0x7F80, 0xFF80, 0x7FC0])
def test_non_finite_rejected(bad):
    x = _data(rows=2, cols=32)
    x[1, 5] = bad
    with pytest.raises(oracle.NonFiniteInput):
        oracle.quantize_fp8(x)
    with pytest.raises(oracle.NonFiniteInput):
        oracle.quantize_nvfp4(x)


# ------------------------------------------------------------ error bounds
def test_fp8_error_bound():
    """|x - deq| <= half an E4M3 step at x*r: 2^-4 relative in the normal range,
    2^-10 * s absolute in the subnormal range (plus fp32 rounding of x*r)."""
    x = _data(rows=64, cols=256, seed=8)
    xf = synth.bf16_bits_to_f32(x).astype(np.float64)
    c, s = oracle.quantize_fp8(x)
    d = oracle.dequant_fp8(c, s)
    bound = np.maximum(np.abs(xf) * 2.0 ** -4, 2.0 ** -10 * float(s)) * (1 + 2 ** -20)
    assert np.all(np.abs(xf - d) <= bound)


def test_nvfp4_error_bound():
    """Within a block with effective scale S, elements below 6*S round to the
    E2M1 grid (error <= half a step: 0.25*S below 2*S, 0.5*S below 4*S, 1*S
    above); the block max may saturate at 6*S, at most 6.375*S - 6*S away."""
    x = _data(rows=32, cols=256, seed=9, frac=0.01)
    xf = synth.bf16_bits_to_f32(x).astype(np.float64)
    c, b, t = oracle.quantize_nvfp4(x)
    d = oracle.dequant_nvfp4(c, b, t)
    S = np.repeat(_torch_e4m3(b) * float(t), 16, axis=1)
    a = np.abs(xf)
    step_half = np.where(a < 2 * S, 0.25 * S, np.where(a < 4 * S, 0.5 * S, 1.0 * S))
    bound = np.maximum(step_half, a - 6 * S) * (1 + 2 ** -18)
    assert np.all(np.abs(xf - d) <= bound + 1e-300)


def test_dequant_fp8_matches_torch_decoder():
    rng = np.random.default_rng(11)
    c = rng.integers(0, 256, size=(8, 64)).astype(np.uint8)
    c[(c & 0x7F) == 0x7F] = 0
    s = np.float32(0.0137)
    d64 = oracle.dequant_fp8(c, s)
    assert np.array_equal(d64, _torch_e4m3(c) * float(s))
    d32 = oracle.dequant_fp8(c, s, out="f32")
    assert np.array_equal(d32, (_torch_e4m3(c) * float(s)).astype(np.float32))


def test_dequant_nvfp4_table():
    rng = np.random.default_rng(12)
    q = rng.integers(0, 16, size=(4, 64)).astype(np.uint8)
    packed = (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8)
    sb = rng.integers(0, 0x7F, size=(4, 4)).astype(np.uint8)
    t = np.float32(0.00390625)
    d = oracle.dequant_nvfp4(packed, sb, t)
    ref = E2M1[q] * np.repeat(_torch_e4m3(sb), 16, axis=1) * float(t)
    assert np.array_equal(d, ref)
    bf = oracle.dequant_nvfp4(packed, sb, t, out="bf16")
    assert np.array_equal(synth.bf16_bits_to_f32(bf), torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16).float().numpy())

"""Pins of the oracle's OCP MX quantizers (MXFP4: E2M1 elements, MXFP8: E4M3
elements; one E8M0 power-of-two scale per 32 elements, no tensor scale).

Independent references: the E2M1 value list of the format definition, torch's
float8_e4m3fn decoder for E4M3 values, an exhaustive nearest-value search in
exact rational arithmetic (ties to the even code) for the element codes, the
closed form of the shared exponent for constructed blocks, and invariants.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth

E2M1 = [Fraction(v) for v in ("0", "1/2", "1", "3/2", "2", "3", "4", "6")]
E4M3 = [Fraction(float(v)) for v in torch.arange(0, 127, dtype=torch.uint8).view(torch.float8_e4m3fn).float()]
EMAX = {"mxfp4": 2, "mxfp8": 8}


def _bits(values):
    return synth.f32_to_bf16_bits(np.asarray(values, dtype=np.float32))


def _nearest_code(v: Fraction, table):
    """Code (sign in the top bit of the format) of the nearest table value to
    v, ties to the even code, saturating at the largest value."""
    a = abs(v)
    best, best_d = 0, None
    for c, t in enumerate(table):
        d = abs(a - t)
        if best_d is None or d < best_d or (d == best_d and c % 2 == 0 and best % 2 == 1):
            best, best_d = c, d
    return best


def _reference(xblock_f32, fmt):
    """Scale code and element codes of one 32-element block, from the spec."""
    a = max(abs(Fraction(float(v))) for v in xblock_f32)
    if a == 0:
        e = 0
    else:
        p = 0
        while Fraction(2) ** (p + 1) <= a:
            p += 1
        while Fraction(2) ** p > a:
            p -= 1
        e = min(max(p - EMAX[fmt] + 127, 0), 254)
    scale = Fraction(2) ** (e - 127)
    table = E2M1 if fmt == "mxfp4" else E4M3
    sign_bit = 8 if fmt == "mxfp4" else 0x80
    codes = []
    for v in xblock_f32:
        fv = Fraction(float(v))
        c = _nearest_code(fv / scale, table)
        neg = np.signbit(np.float32(v))
        codes.append(c | (sign_bit if neg else 0))
    return e, codes


def _unpack(codes, fmt):
    if fmt == "mxfp8":
        return codes
    out = np.empty((codes.shape[0], codes.shape[1] * 2), dtype=np.uint8)
    out[:, 0::2] = codes & 15
    out[:, 1::2] = codes >> 4
    return out


def test_e8m0_values():
    t = oracle.e8m0_table()
    assert np.isnan(t[255])
    assert np.array_equal(t[:255], np.ldexp(1.0, np.arange(255) - 127))


@pytest.mark.parametrize("fmt", ["mxfp4", "mxfp8"])
@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_codes_match_exhaustive_rational_reference(fmt, seed):
    # wide dynamic range across blocks: sigma 10^(-3..3) per block, some zeros
    rng = np.random.default_rng(seed)
    rows, blocks = 4, 6
    vals = rng.normal(0, 1, (rows, blocks, 32)) * (10.0 ** rng.uniform(-3, 3, (rows, blocks, 1)))
    vals[0, 0, :] = 0.0
    vals[1, 1, :5] = 0.0
    x = _bits(vals.reshape(rows, blocks * 32))
    xf = synth.bf16_bits_to_f32(x).reshape(rows, blocks, 32)
    codes, scales = oracle.quantize_mx(x, fmt)
    el = _unpack(codes, fmt).reshape(rows, blocks, 32)
    for i in range(rows):
        for b in range(blocks):
            e, ref = _reference(xf[i, b], fmt)
            assert scales[i, b] == e, (i, b, scales[i, b], e)
            assert list(el[i, b]) == ref, (i, b)


@pytest.mark.parametrize("fmt", ["mxfp4", "mxfp8"])
@pytest.mark.parametrize("p", [-20, -3, 0, 1, 7, 30])
def test_shared_exponent_closed_form(fmt, p):
    # a block whose max is 1.5 * 2^p: e = p - emax + 127
    v = np.full(32, 0.25 * 2.0 ** p, dtype=np.float64)
    v[7] = -1.5 * 2.0 ** p
    _, scales = oracle.quantize_mx(_bits(v.reshape(1, 32)), fmt)
    assert scales[0, 0] == p - EMAX[fmt] + 127


@pytest.mark.parametrize("fmt", ["mxfp4", "mxfp8"])
def test_representable_blocks_round_trip(fmt):
    # element values times 2^(e-127) with the block max at the format maximum
    # (so the shared exponent lands on e): dequant(quantize(x)) == x exactly
    rng = np.random.default_rng(7)
    table = np.array([float(t) for t in (E2M1 if fmt == "mxfp4" else E4M3)])
    rows = []
    for e in (100, 120, 127, 140):
        el = rng.choice(table, 32) * rng.choice([-1.0, 1.0], 32)
        el[0] = table[-1]
        rows.append(el * 2.0 ** (e - 127))
    x = _bits(np.array(rows))
    assert np.array_equal(synth.bf16_bits_to_f32(x), np.array(rows, dtype=np.float32))
    codes, scales = oracle.quantize_mx(x, fmt)
    assert list(scales[:, 0]) == [100, 120, 127, 140]
    assert np.array_equal(oracle.dequant_mx(codes, scales, fmt), np.array(rows))


@pytest.mark.parametrize("fmt", ["mxfp4", "mxfp8"])
def test_power_of_two_scaling_and_sign_symmetry(fmt):
    x = synth.normal_bf16(8, 128, 1.0, 9, 0)
    c1, s1 = oracle.quantize_mx(x, fmt)
    c2, s2 = oracle.quantize_mx(_bits(synth.bf16_bits_to_f32(x) * 2.0 ** 5), fmt)
    assert np.array_equal(c1, c2) and np.array_equal(s2.astype(int), s1.astype(int) + 5)
    c3, s3 = oracle.quantize_mx(_bits(-synth.bf16_bits_to_f32(x)), fmt)
    sign = np.uint8(0x88) if fmt == "mxfp4" else np.uint8(0x80)
    e1 = _unpack(c1, fmt)
    e3 = _unpack(c3, fmt)
    sb = 8 if fmt == "mxfp4" else 0x80
    assert np.array_equal(s1, s3)
    assert np.array_equal(e3, e1 ^ sb)
    del sign


@pytest.mark.parametrize("fmt", ["mxfp4", "mxfp8"])
def test_tiny_blocks_clamp_the_scale_code_at_zero(fmt):
    # block maxima below 2^(emax - 127) (bf16 subnormals and the smallest
    # normals) would need a negative code: it clamps to 0 and the elements
    # are coded at the scale 2^-127 (exact rational reference)
    rng = np.random.default_rng(11)
    rows = []
    for top in (2.0 ** -133, 2.0 ** -130, 1.5 * 2.0 ** -127, 1.5 * 2.0 ** -126, 1.75 * 2.0 ** -120):
        v = rng.uniform(-1.0, 1.0, 32) * top
        v[3] = -top                                     # the largest magnitude is negative
        rows.append(v)
    x = _bits(np.array(rows))
    xf = synth.bf16_bits_to_f32(x)
    codes, scales = oracle.quantize_mx(x, fmt)
    el = _unpack(codes, fmt)
    for i in range(len(rows)):
        e, ref = _reference(xf[i], fmt)
        assert scales[i, 0] == e and list(el[i]) == ref, (i, scales[i, 0], e)
    assert scales[:4, 0].tolist() == [0, 0, 0, 0] if fmt == "mxfp4" else scales[:, 0].tolist() == [0] * 5


def test_zero_block_and_signed_zero():
    x = _bits(np.array([[0.0] * 31 + [-0.0]]))
    c, s = oracle.quantize_mx(x, "mxfp4")
    assert s[0, 0] == 0 and c[0, 15] == 0x80 and not c[0, :15].any()

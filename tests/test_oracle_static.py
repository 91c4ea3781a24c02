"""Pins of the oracle's static-scale quantizers (calibrated activation scales).

The static path is the dynamic recipe with the tensor decode scale given
instead of derived from the tensor's own max (post-training quantization
with fixed activation ranges). Pins: equality with the already-pinned
dynamic path at the dynamic scale; closed forms for saturation beyond the
calibrated range and for a zero scale; torch's float8_e4m3fn cast for the
in-range FP8 codes; invariance under x -> 2x, s -> 2s.
"""
import numpy as np
import pytest
import torch

import oracle
import synth


def _bits(values):
    return synth.f32_to_bf16_bits(np.asarray(values, dtype=np.float32))


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("shape", [(1, 16), (7, 48), (64, 256)])
def test_static_equals_dynamic_at_dynamic_scale(seed, shape):
    x = synth.normal_bf16(shape[0], shape[1], 1.0, seed, 0, outlier_frac=0.05, outlier_gain=30.0)
    q, s = oracle.quantize_fp8(x)
    assert np.array_equal(oracle.quantize_fp8_static(x, s), q)
    qn, bn, st = oracle.quantize_nvfp4(x)
    c2, b2 = oracle.quantize_nvfp4_static(x, st)
    assert np.array_equal(c2, qn) and np.array_equal(b2, bn)


def test_fp8_static_saturates_and_matches_torch_in_range():
    # s = 2^-3: r = 8 exactly, so x * r is exact and codes are E4M3(8 x)
    s = np.float32(0.125)
    rng = np.random.default_rng(3)
    vals = np.concatenate([rng.normal(0.0, 10.0, 4000), [60.0, -60.0, 57.5, -57.0, 100.0, 1e4, -1e4]])
    x = _bits(vals)
    q = oracle.quantize_fp8_static(x.reshape(1, -1), s).reshape(-1)
    y = synth.bf16_bits_to_f32(x).astype(np.float64) * 8.0
    inr = np.abs(y) < 464.0
    ref = torch.from_numpy(y[inr].astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(q[inr], ref)
    # beyond the calibrated range: the largest finite E4M3 with the sign of x
    sat = ~inr
    assert sat.sum() >= 4
    assert np.array_equal(q[sat], np.where(y[sat] > 0, 0x7E, 0xFE).astype(np.uint8))


def test_nvfp4_static_saturates_closed_form():
    # s_t = 1/2688: d_t = 6 s_t = 1/448. A block of +-10: v_b = 4480 saturates to
    # 448 (0x7E), S = 448 s_t = 1/6, r = 6, x r = +-60 saturates to +-6 (code 7).
    s_t = np.float32(1.0) / np.float32(2688.0)
    blk = np.array([10.0, -10.0] * 8, dtype=np.float32)
    x = _bits(np.concatenate([blk, blk]).reshape(1, 32))
    codes, bs = oracle.quantize_nvfp4_static(x, s_t)
    assert np.array_equal(bs, np.array([[0x7E, 0x7E]], dtype=np.uint8))
    assert np.array_equal(codes, np.full((1, 16), 0x7 | (0xF << 4), dtype=np.uint8))


def test_static_zero_scale_gives_signed_zeros():
    x = _bits([[1.5, -2.0, 0.25, -0.0] * 4])
    q = oracle.quantize_fp8_static(x, 0.0)
    assert np.array_equal(q[0], np.array([0x00, 0x80, 0x00, 0x80] * 4, dtype=np.uint8))
    c, b = oracle.quantize_nvfp4_static(x, 0.0)
    assert np.array_equal(b, np.zeros((1, 1), dtype=np.uint8))
    assert np.array_equal(c[0], np.array([0x80] * 8, dtype=np.uint8))


@pytest.mark.parametrize("seed", [4, 5])
def test_static_scale_invariance(seed):
    x = synth.normal_bf16(8, 64, 1.0, seed, 0)
    x2 = _bits(synth.bf16_bits_to_f32(x) * 2.0)
    for s in (np.float32(0.01), np.float32(0.003)):
        assert np.array_equal(oracle.quantize_fp8_static(x, s), oracle.quantize_fp8_static(x2, np.float32(2 * s)))
        c1, b1 = oracle.quantize_nvfp4_static(x, s)
        c2, b2 = oracle.quantize_nvfp4_static(x2, np.float32(2 * s))
        assert np.array_equal(c1, c2) and np.array_equal(b1, b2)


def test_static_rejects_bad_scales_and_nonfinite():
    x = synth.normal_bf16(2, 16, 1.0, 0, 0)
    for bad in (-1.0, float("nan"), float("inf"), 1e-40):
        with pytest.raises(ValueError):
            oracle.quantize_fp8_static(x, bad)
    with pytest.raises(ValueError):
        oracle.quantize_nvfp4_static(x, 1e-30)
    xn = x.copy()
    xn[0, 3] = 0x7F80
    with pytest.raises(oracle.NonFiniteInput):
        oracle.quantize_fp8_static(xn, 0.01)


def test_static_scale_validity_boundaries():
    # FP8: 0 or a normal fp32 (>= 2^-126), so that 1/s is finite. NVFP4: 0 or
    # >= 2^-96, so that 1/(dec(s_b) s_t) is finite for the smallest block
    # scale code (2^-9). Both sides of each boundary, and the next float down.
    x = synth.normal_bf16(2, 16, 1.0, 0, 0)
    oracle.quantize_fp8_static(x, np.float32(2.0 ** -126))
    oracle.quantize_nvfp4_static(x, np.float32(2.0 ** -96))
    for bad in (2.0 ** -127, np.nextafter(np.float32(2.0 ** -126), np.float32(0))):
        with pytest.raises(ValueError):
            oracle.quantize_fp8_static(x, np.float32(bad))
    for bad in (2.0 ** -97, np.nextafter(np.float32(2.0 ** -96), np.float32(0))):
        with pytest.raises(ValueError):
            oracle.quantize_nvfp4_static(x, np.float32(bad))


# ---------------------------------------------------------------- static NVFP4 on fp32 values
@pytest.mark.parametrize("seed", [0, 1])
def test_nvfp4_static_f32_equals_bf16_path_on_bf16_values(seed):
    # bf16 values widened to fp32 exactly: the fp32 entry point must give the
    # codes of the (pinned) bf16 entry point, scale for scale
    x = synth.normal_bf16(33, 256, 1.0, seed, 0, outlier_frac=0.05, outlier_gain=40.0)
    x[3, :16] = 0
    x[4, 16:32] &= 0x807F                                  # subnormal-only block
    xf = synth.bf16_bits_to_f32(x)
    _, _, s_dyn = oracle.quantize_nvfp4(x)
    for s in (s_dyn, np.float32(s_dyn * 0.3), np.float32(s_dyn * 3.0), np.float32(0.0)):
        c1, b1 = oracle.quantize_nvfp4_static(x, s)
        c2, b2 = oracle.quantize_nvfp4_static_f32(xf, s)
        assert np.array_equal(c1, c2) and np.array_equal(b1, b2)


def test_nvfp4_static_f32_worked_example():
    # s_t = fl(1/6): d = fl(6 s_t) = 1 and the block max 6 gives v = 6, an
    # E4M3 value (1.5 x 2^2: code 0x4C), so S = fl(6 s_t) = 1 and r = 1: each
    # code is E2M1 of the fp32 value itself. The values sit one fp32 ulp on
    # either side of the E2M1 midpoints (0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5)
    # or on them (ties to the even code), which bf16 inputs cannot do.
    y = np.array([6.0, 1.2500001, 1.2499999, -0.2500001, 0.25, 0.7499999, 0.75, 1.75,
                  2.5, 2.5000002, 3.4999998, 3.5, 4.9999995, 5.0, 5.0000005, -6.0], dtype=np.float32)
    # codes: 6 -> 7; 1.2500001 -> 1.5 (3); 1.2499999 -> 1 (2); -0.2500001 -> -0.5 (9);
    # 0.25 tie -> 0 (0); 0.7499999 -> 0.5 (1); 0.75 tie -> 1 (2); 1.75 tie -> 2 (4);
    # 2.5 tie -> 2 (4); 2.5000002 -> 3 (5); 3.4999998 -> 3 (5); 3.5 tie -> 4 (6);
    # 4.9999995 -> 4 (6); 5 tie -> 4 (6); 5.0000005 -> 6 (7); -6 -> -6 (15)
    want = [7, 3, 2, 9, 0, 1, 2, 4, 4, 5, 5, 6, 6, 6, 7, 15]
    s_t = np.float32(1.0) / np.float32(6.0)
    assert np.float32(6.0) * s_t == np.float32(1.0)
    c, b = oracle.quantize_nvfp4_static_f32(y.reshape(1, 16), s_t)
    assert b.tolist() == [[0x4C]]
    assert c.reshape(-1).tolist() == [want[2 * i] | (want[2 * i + 1] << 4) for i in range(8)]


def test_nvfp4_static_f32_saturates_and_refuses():
    # beyond the calibrated range: block scale 448, codes +-6
    y = np.full((1, 16), 1e6, dtype=np.float32)
    y[0, 1::2] = -1e6
    c, b = oracle.quantize_nvfp4_static_f32(y, np.float32(2.0 ** -10))
    assert b.tolist() == [[0x7E]] and c.reshape(-1).tolist() == [0xF7] * 8
    with pytest.raises(oracle.NonFiniteInput):
        oracle.quantize_nvfp4_static_f32(np.array([[np.inf] + [0.0] * 15], np.float32), np.float32(1.0))
    with pytest.raises(ValueError):
        oracle.quantize_nvfp4_static_f32(np.zeros((1, 16), np.float32), np.float32(2.0 ** -100))

"""Pins for the oracle's E4M3 / E2M1 codecs (CPU only).

Each test checks the oracle against something other than itself: the value
table the format definitions fix, torch's independent float8_e4m3fn decoder
and caster, and a brute-force nearest-value search written here.
"""
import math

import numpy as np
import pytest
import torch

import oracle

E2M1_MAGNITUDES = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]   # fixed by the NVFP4 element format


def test_e2m1_table_matches_format():
    vals = [oracle.e2m1_value(c) for c in range(16)]
    assert vals[:8] == E2M1_MAGNITUDES
    assert vals[8:] == [-v for v in E2M1_MAGNITUDES]
    assert math.copysign(1.0, vals[8]) == -1.0          # code 8 is -0


def test_e4m3_constants():
    t = oracle.e4m3_table()
    assert t[0x7E] == 448.0                              # largest finite
    assert t[0x08] == 2.0 ** -6                          # smallest normal
    assert t[0x01] == 2.0 ** -9                          # smallest subnormal
    assert math.isnan(t[0x7F]) and math.isnan(t[0xFF])   # the only NaNs, no infinities
    assert np.isfinite(t[[c for c in range(256) if c not in (0x7F, 0xFF)]]).all()
    pos = t[:0x7F]
    assert len(pos) == 127 and np.all(np.diff(pos) > 0)  # 127 finite non-negative values, increasing
    assert math.copysign(1.0, t[0x80]) == -1.0


def test_e4m3_decode_matches_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = oracle.e4m3_table()
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(ours))
    assert np.array_equal(ref[~nan], ours[~nan])
    assert np.array_equal(np.signbit(ref[~nan]), np.signbit(ours[~nan]))


@pytest.mark.parametrize("fmt", ["e4m3", "e2m1"])
def test_roundtrip_every_representable_value(fmt):
    if fmt == "e4m3":
        codes = [c for c in range(256) if c not in (0x7F, 0xFF)]
        val, enc = oracle.e4m3_value, oracle.e4m3_encode
    else:
        codes = list(range(16))
        val, enc = oracle.e2m1_value, oracle.e2m1_encode
    for c in codes:
        assert enc(val(c)) == c, (fmt, c)


@pytest.mark.parametrize("fmt", ["e4m3", "e2m1"])
def test_ties_go_to_even_code(fmt):
    if fmt == "e4m3":
        top, val, enc = 0x7E, oracle.e4m3_value, oracle.e4m3_encode
    else:
        top, val, enc = 7, oracle.e2m1_value, oracle.e2m1_encode
    for c in range(top):
        mid = 0.5 * (val(c) + val(c + 1))
        assert float(np.float32(mid)) == mid             # every midpoint is an fp32 value
        even = c if c % 2 == 0 else c + 1
        assert enc(mid) == even, (fmt, c, mid)
        sign = 0x80 if fmt == "e4m3" else 0x8
        assert enc(-mid) == sign | even
        # one fp32 ulp either side of the midpoint decides by distance
        lo = np.nextafter(np.float32(mid), np.float32(0))
        hi = np.nextafter(np.float32(mid), np.float32(1e9))
        assert enc(float(lo)) == c and enc(float(hi)) == c + 1


def _brute_force(v: np.ndarray, mags: np.ndarray, sign_bit: int) -> np.ndarray:
    """Nearest magnitude by exhaustive distance, ties to the even code, saturating."""
    a = np.abs(v.astype(np.float64))
    d = np.abs(a[:, None] - mags[None, :])
    best = d.min(axis=1, keepdims=True)
    cand = d == best
    idx = np.arange(len(mags))
    # among equal distances prefer the even code
    score = np.where(cand, np.where(idx % 2 == 0, 0, 1), 9)
    code = score.argmin(axis=1)
    code = np.where(a >= mags[-1], len(mags) - 1, code)
    return (code | np.where(np.signbit(v), sign_bit, 0)).astype(np.uint8)


def _probe_values(mags: np.ndarray) -> np.ndarray:
    rng = np.random.default_rng(1234)
    bits = rng.integers(0, 2 ** 32, size=1 << 18, dtype=np.uint64).astype(np.uint32)
    v = bits.view(np.float32)
    v = v[np.isfinite(v)]
    # dense coverage of the interesting range: scaled uniform magnitudes
    u = (rng.random(1 << 18) * mags[-1] * 1.2).astype(np.float32)
    # every midpoint and neighbouring value +-4 ulps, and the grid points themselves
    pts = np.concatenate([mags, 0.5 * (mags[1:] + mags[:-1])]).astype(np.float32)
    near = [pts]
    cur_lo, cur_hi = pts.copy(), pts.copy()
    for _ in range(4):
        cur_lo = np.nextafter(cur_lo, np.float32(-1e30))
        cur_hi = np.nextafter(cur_hi, np.float32(1e30))
        near += [cur_lo, cur_hi]
    near = np.concatenate(near)
    allv = np.concatenate([v, u, -u, near, -near, np.array([0.0, -0.0, 1e-45, -1e-45, 3e38, -3e38], np.float32)])
    return allv.astype(np.float32)


def test_e4m3_encode_brute_force():
    mags = oracle.e4m3_table()[:0x7F]
    v = _probe_values(mags)
    assert np.array_equal(oracle.e4m3_encode_array(v), _brute_force(v, mags, 0x80))


def test_e2m1_encode_brute_force():
    mags = np.array(E2M1_MAGNITUDES)
    v = _probe_values(mags)
    assert np.array_equal(oracle.e2m1_encode_array(v), _brute_force(v, mags, 0x8))


def test_e4m3_encode_matches_torch_cast_below_464():
    """torch's float8_e4m3fn cast rounds to nearest-even but does not saturate
    (it turns magnitudes >= 464 into NaN), so compare where it is defined."""
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 2 ** 32, size=1 << 21, dtype=np.uint64).astype(np.uint32)
    v = bits.view(np.float32)
    v = np.concatenate([v, (rng.random(1 << 20) * 470 - 235).astype(np.float32)])
    v = v[np.isfinite(v) & (np.abs(v) < 464)]
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(oracle.e4m3_encode_array(v), ref)


def test_saturation():
    assert oracle.e4m3_encode(464.0) == 0x7E
    assert oracle.e4m3_encode(1e30) == 0x7E
    assert oracle.e4m3_encode(-1e30) == 0xFE
    assert oracle.e2m1_encode(7.0) == 0x7
    assert oracle.e2m1_encode(-1000.0) == 0xF

"""The rounding helper of the GPU parity checks (tests/gpu_util.py:
bf16_rne, one round-to-nearest-even of a float64 value to bf16) against the
oracle's fp32 -> bf16 rounding on random fp32 inputs, where one rounding and
two agree, and on exact ties between neighbouring bf16 values."""
import numpy as np

import oracle
import synth
from gpu_util import bf16_rne


def test_bf16_rne_equals_oracle_rounding_of_fp32():
    rng = np.random.default_rng(1)
    v = rng.integers(0, 2 ** 32, 1_000_000, dtype=np.uint64).astype(np.uint32).view(np.float32)
    v = v[np.isfinite(v) & (np.abs(v) < 3.0e38)]
    want = synth.bf16_bits_to_f32(oracle.to_bf16(v)).astype(np.float64)
    assert np.array_equal(bf16_rne(v.astype(np.float64)), want)


def test_bf16_rne_ties_go_to_even():
    a = synth.bf16_bits_to_f32(np.arange(0x3F80, 0x3FA0, dtype=np.uint16)).astype(np.float64)
    mid = (a[:-1] + a[1:]) / 2
    even = np.where(np.arange(mid.size) % 2 == 0, a[:-1], a[1:])
    assert np.array_equal(bf16_rne(mid), even)
    assert np.array_equal(bf16_rne(-mid), -even)
    assert bf16_rne(np.array([0.0]))[0] == 0.0

"""Pins for the oracle's linear layer Y = A . W^T (CPU only).

Checked against: exact rational arithmetic (fractions) on tiny shapes, torch's
float64 matmul, dyadic special cases whose result is an exact integer, and
the permutation/linearity structure of the product.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth


def test_tiny_bruteforce_exact_rational():
    rng = np.random.default_rng(0)
    for m, n, k in [(1, 1, 16), (3, 4, 32), (4, 2, 64)]:
        a = rng.standard_normal((m, k)) * 3
        w = rng.standard_normal((n, k)) * 0.1
        y, b = oracle.gemm_f64(a, w)
        for i in range(m):
            for j in range(n):
                exact = sum(Fraction(a[i, t]) * Fraction(w[j, t]) for t in range(k))
                mag = sum(abs(Fraction(a[i, t]) * Fraction(w[j, t])) for t in range(k))
                assert abs(Fraction(y[i, j]) - exact) <= Fraction(k) * Fraction(2) ** -52 * mag
                assert abs(Fraction(b[i, j]) - mag) <= Fraction(k) * Fraction(2) ** -52 * mag


def test_matches_torch_float64_matmul():
    rng = np.random.default_rng(1)
    a = rng.standard_normal((37, 96))
    w = rng.standard_normal((29, 96))
    y, b = oracle.gemm_f64(a, w)
    ref = (torch.from_numpy(a) @ torch.from_numpy(w).T).numpy()
    refb = (torch.from_numpy(np.abs(a)) @ torch.from_numpy(np.abs(w)).T).numpy()
    assert np.allclose(y, ref, rtol=0, atol=1e-12 * refb.max())
    assert np.allclose(b, refb, rtol=1e-13, atol=0)


def test_dyadic_inputs_give_exact_integers():
    rng = np.random.default_rng(2)
    a = rng.integers(-12, 13, size=(8, 256)).astype(np.float64) / 2     # E2M1-like values
    w = rng.integers(-12, 13, size=(16, 256)).astype(np.float64) / 2
    y, _ = oracle.gemm_f64(a, w)
    exact = (a * 2).astype(np.int64) @ (w * 2).astype(np.int64).T
    assert np.array_equal(y * 4, exact.astype(np.float64))


def test_sampled_matches_full():
    rng = np.random.default_rng(3)
    a = rng.standard_normal((20, 48))
    w = rng.standard_normal((30, 48))
    y, b = oracle.gemm_f64(a, w)
    rows = rng.integers(0, 20, 50)
    cols = rng.integers(0, 30, 50)
    ys, bs = oracle.gemm_f64_sampled(a, w, rows, cols)
    assert np.array_equal(ys, y[rows, cols]) and np.array_equal(bs, b[rows, cols])


def test_k_block_permutation_and_scale_linearity():
    """Permuting K jointly in both operands keeps the product (up to fp64
    rounding); scaling an operand's tensor scale by 2^j scales Y exactly."""
    x = synth.normal_bf16(8, 64, 1.0, 0, 0)
    wt = synth.normal_bf16(12, 64, 0.02, 0, 1)
    ref = oracle.linear_reference("nvfp4", x, wt)
    perm = np.random.default_rng(4).permutation(4)
    kp = np.concatenate([np.arange(16) + 16 * p for p in perm])
    got = oracle.linear_reference("nvfp4", x[:, kp], wt[:, kp])
    assert np.allclose(got["y"], ref["y"], rtol=0, atol=1e-13 * ref["b"].max())
    a = oracle.dequant_nvfp4(ref["a_codes"], ref["a_bscales"], ref["a_scale"])
    w2 = oracle.dequant_nvfp4(ref["w_codes"], ref["w_bscales"], np.float32(ref["w_scale"] * 4))
    y2, _ = oracle.gemm_f64(a, w2)
    assert np.array_equal(y2, ref["y"] * 4)


@pytest.mark.parametrize("kind", ["fp8", "nvfp4", "w4a16"])
def test_linear_reference_consistent(kind):
    """End-to-end reference: quantize, dequantize, product; sampled == full."""
    x = synth.normal_bf16(16, 128, 1.0, 0, 0)
    wt = synth.normal_bf16(32, 128, 0.02, 0, 1)
    full = oracle.linear_reference(kind, x, wt)
    rows = np.array([0, 5, 15, 7])
    cols = np.array([31, 0, 9, 9])
    smp = oracle.linear_reference(kind, x, wt, rows=rows, cols=cols)
    assert np.array_equal(smp["y"], full["y"][rows, cols])
    # quantization error vs the unquantized product stays within what the formats allow
    xf = synth.bf16_bits_to_f32(x).astype(np.float64)
    wf = synth.bf16_bits_to_f32(wt).astype(np.float64)
    exact, mag = oracle.gemm_f64(xf, wf)
    rel = {"fp8": 0.13, "nvfp4": 0.6, "w4a16": 0.35}[kind]
    assert np.all(np.abs(full["y"] - exact) <= rel * mag)

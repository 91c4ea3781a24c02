"""Seeded synthetic tensors shared by the oracle side and the device side.

This module only draws numbers: it holds none of the quantization or GEMM
arithmetic. Both the CPU oracle and the HIP path read the exact same bf16 bit
patterns produced here, so any disagreement between them is theirs, not the
generator's.

Recipe (counter-based, reproducible on any machine):
  * stream key  = splitmix64(seed * 0x100000001B3 + stream)
  * word i      = splitmix64(key + i * 0x9E3779B97F4A7C15)
  * normal i    = Box-Muller on words (2i, 2i+1) in float64, cosine branch
  * value       = sigma * normal, rounded float64 -> float32 (RNE) -> bf16 (RNE)
  * heavy tail  = n_out = max(1, round(frac * K)) input channels picked by a
                  seeded Fisher-Yates shuffle are multiplied by `gain` before
                  the float32 rounding; the same channels in every row.

bf16 tensors are returned as numpy uint16 arrays of bit patterns.
"""
from __future__ import annotations

import os

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_MASK = (1 << 64) - 1


def _splitmix64_py(z: int) -> int:
    z &= _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def _splitmix64_np(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * _M1
    z = z ^ (z >> np.uint64(27))
    z = z * _M2
    return z ^ (z >> np.uint64(31))


def stream_key(seed: int, stream: int) -> int:
    return _splitmix64_py(seed * 0x100000001B3 + stream)


def uniform_words(seed: int, stream: int, count: int, offset: int = 0) -> np.ndarray:
    """`count` raw 64-bit words of the (seed, stream) sequence starting at `offset`."""
    key = np.uint64(stream_key(seed, stream))
    idx = np.arange(offset, offset + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _splitmix64_np(key + idx * _GOLDEN)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    out = rounded.astype(np.uint16)
    out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_chunk(seed: int, stream: int, start: int, out: np.ndarray) -> None:
    n = out.size
    scale = 2.0 ** -53
    w = uniform_words(seed, stream, 2 * n, offset=2 * start)
    u1 = ((w[0::2] >> np.uint64(11)).astype(np.float64) + 1.0) * scale  # (0, 1]
    u2 = (w[1::2] >> np.uint64(11)).astype(np.float64) * scale          # [0, 1)
    out[:] = np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)


def normal_f64(seed: int, stream: int, count: int) -> np.ndarray:
    """`count` standard normals (float64) from the counter-based stream.

    Chunks are independent (counter-based), so they are filled by a thread
    pool; the result does not depend on the number of threads.
    """
    out = np.empty(count, dtype=np.float64)
    chunk = 1 << 20
    starts = list(range(0, count, chunk))
    if len(starts) <= 1:
        _normal_chunk(seed, stream, 0, out)
        return out
    from concurrent.futures import ThreadPoolExecutor
    workers = max(1, min(16, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(lambda s0: _normal_chunk(seed, stream, s0, out[s0:s0 + chunk]), starts))
    return out


def outlier_channels(seed: int, stream: int, k: int, frac: float) -> np.ndarray:
    """Seeded Fisher-Yates pick of max(1, round(frac*k)) distinct channel indices."""
    n_out = max(1, int(round(frac * k)))
    perm = list(range(k))
    words = uniform_words(seed, stream, k)
    for i in range(k - 1, 0, -1):
        j = int(words[k - 1 - i] % np.uint64(i + 1))
        perm[i], perm[j] = perm[j], perm[i]
    return np.array(sorted(perm[k - n_out:]), dtype=np.int64)


def normal_bf16(rows: int, cols: int, sigma: float, seed: int, stream: int,
                outlier_frac: float = 0.0, outlier_gain: float = 1.0,
                outlier_stream: int = 2) -> np.ndarray:
    """bf16 bit patterns [rows, cols] of sigma * N(0,1), optional heavy-tail channels."""
    v = normal_f64(seed, stream, rows * cols).reshape(rows, cols) * sigma
    if outlier_frac > 0.0:
        ch = outlier_channels(seed, outlier_stream, cols, outlier_frac)
        v[:, ch] *= outlier_gain
    return f32_to_bf16_bits(v.astype(np.float32))


# Workloads with the shapes of the paper's denoising transformer at a 1024^2
# image (4096 latent + 512 text tokens, hidden 3072) and of the small text
# encoder (hidden 1024, FFN 3072).
DIT_TOKENS = 4608
DIT_LINEARS = {            # name: (N, K) for Y[M,N] = X[M,K] . W[N,K]^T
    "qkv": (9216, 3072),
    "attn_out": (3072, 3072),
    "mlp_up": (9216, 3072),
    "mlp_down": (3072, 9216),
}
ENCODER_LINEARS = {"up": (3072, 1024), "down": (1024, 3072)}
ENCODER_TOKENS = (1, 16, 256, 512)
SIGMA_X = 1.0
SIGMA_W = 0.02
HEAVY_TAIL_FRAC = 0.001
HEAVY_TAIL_GAIN = 50.0
STREAM_X, STREAM_W, STREAM_OUTLIER = 0, 1, 2

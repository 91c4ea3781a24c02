"""CPU oracle for the quantized-linear hot path (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product library never loads it.

The arithmetic lives in ``qg_oracle.c`` (plain C, built with gcc); this module
only builds that file and marshals numpy arrays. bf16 tensors are numpy uint16
arrays of bit patterns, codes and block scales are uint8 arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "qg_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

GCC_FLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
             "-fopenmp", "-fPIC", "-shared", "-Wall"]


def build(force: bool = True) -> str:
    """Compile qg_oracle.c into liboracle.so next to it."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", *GCC_FLAGS, "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        L.qo_e4m3_value.restype = ctypes.c_double
        L.qo_e4m3_value.argtypes = [ctypes.c_uint8]
        L.qo_e2m1_value.restype = ctypes.c_double
        L.qo_e2m1_value.argtypes = [ctypes.c_uint8]
        L.qo_e4m3_encode.restype = ctypes.c_uint8
        L.qo_e4m3_encode.argtypes = [ctypes.c_float]
        L.qo_e2m1_encode.restype = ctypes.c_uint8
        L.qo_e2m1_encode.argtypes = [ctypes.c_float]
        L.qo_e4m3_encode_array.argtypes = [P, I64, P]
        L.qo_e2m1_encode_array.argtypes = [P, I64, P]
        L.qo_f32_to_bf16.restype = ctypes.c_uint16
        L.qo_f32_to_bf16.argtypes = [ctypes.c_float]
        L.qo_quantize_fp8.restype = ctypes.c_int
        L.qo_quantize_fp8.argtypes = [P, I64, I64, I64, P, P]
        L.qo_quantize_nvfp4.restype = ctypes.c_int
        L.qo_quantize_nvfp4.argtypes = [P, I64, I64, I64, P, P, P]
        L.qo_e8m0_value.restype = ctypes.c_double
        L.qo_e8m0_value.argtypes = [ctypes.c_uint8]
        L.qo_quantize_mxfp4.restype = ctypes.c_int
        L.qo_quantize_mxfp4.argtypes = [P, I64, I64, I64, P, P]
        L.qo_quantize_mxfp8.restype = ctypes.c_int
        L.qo_quantize_mxfp8.argtypes = [P, I64, I64, I64, P, P]
        L.qo_dequant_mxfp4_f64.argtypes = [P, P, I64, I64, P]
        L.qo_dequant_mxfp8_f64.argtypes = [P, P, I64, I64, P]
        L.qo_quantize_fp8_static.restype = ctypes.c_int
        L.qo_quantize_fp8_static.argtypes = [P, I64, I64, I64, ctypes.c_float, P]
        L.qo_quantize_nvfp4_static.restype = ctypes.c_int
        L.qo_quantize_nvfp4_static.argtypes = [P, I64, I64, I64, ctypes.c_float, P, P]
        L.qo_quantize_nvfp4_static_f32.restype = ctypes.c_int
        L.qo_quantize_nvfp4_static_f32.argtypes = [P, I64, I64, I64, ctypes.c_float, P, P]
        L.qo_dequant_fp8_f64.argtypes = [P, I64, ctypes.c_float, P]
        L.qo_dequant_nvfp4_f64.argtypes = [P, P, I64, I64, ctypes.c_float, P]
        L.qo_dequant_fp8_f32.argtypes = [P, I64, ctypes.c_float, P]
        L.qo_dequant_nvfp4_f32.argtypes = [P, P, I64, I64, ctypes.c_float, P]
        L.qo_f32_to_bf16_array.argtypes = [P, I64, P]
        L.qo_bf16_to_f64.argtypes = [P, I64, P]
        L.qo_gemm_f64.argtypes = [P, P, I64, I64, I64, P, P]
        L.qo_gemm_f64_sampled.argtypes = [P, P, I64, P, P, I64, P, P]
        L.qo_num_threads.restype = ctypes.c_int
        L.qo_set_num_threads.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


class NonFiniteInput(ValueError):
    """The oracle refuses tensors holding inf or NaN."""


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


# ---------------------------------------------------------------- codecs
def e4m3_value(code: int) -> float:
    return lib().qo_e4m3_value(int(code) & 0xFF)


def e2m1_value(code: int) -> float:
    return lib().qo_e2m1_value(int(code) & 0xF)


def e4m3_encode(v: float) -> int:
    return lib().qo_e4m3_encode(float(np.float32(v)))


def e2m1_encode(v: float) -> int:
    return lib().qo_e2m1_encode(float(np.float32(v)))


def e4m3_encode_array(v: np.ndarray) -> np.ndarray:
    x = _c(v, np.float32)
    o = np.empty(x.shape, dtype=np.uint8)
    lib().qo_e4m3_encode_array(_ptr(x), x.size, _ptr(o))
    return o


def e2m1_encode_array(v: np.ndarray) -> np.ndarray:
    x = _c(v, np.float32)
    o = np.empty(x.shape, dtype=np.uint8)
    lib().qo_e2m1_encode_array(_ptr(x), x.size, _ptr(o))
    return o


E4M3_TABLE = None
E2M1_TABLE = None


def e4m3_table() -> np.ndarray:
    global E4M3_TABLE
    if E4M3_TABLE is None:
        E4M3_TABLE = np.array([e4m3_value(c) for c in range(256)], dtype=np.float64)
    return E4M3_TABLE


def e2m1_table() -> np.ndarray:
    global E2M1_TABLE
    if E2M1_TABLE is None:
        E2M1_TABLE = np.array([e2m1_value(c) for c in range(16)], dtype=np.float64)
    return E2M1_TABLE


# ---------------------------------------------------------------- quantizers
def quantize_fp8(x_bf16: np.ndarray):
    """bf16 bits [R, K] -> (codes uint8 [R, K], decode scale float32)."""
    x = _c(x_bf16, np.uint16)
    r, k = x.shape
    codes = np.empty((r, k), dtype=np.uint8)
    s = np.zeros(1, dtype=np.float32)
    st = lib().qo_quantize_fp8(_ptr(x), r, k, k, _ptr(codes), _ptr(s))
    if st == 6:
        raise NonFiniteInput("tensor holds inf or NaN")
    assert st == 0, st
    return codes, np.float32(s[0])


def quantize_nvfp4(x_bf16: np.ndarray):
    """bf16 bits [R, K] -> (codes uint8 [R, K/2], block scales uint8 [R, K/16], s_t float32)."""
    x = _c(x_bf16, np.uint16)
    r, k = x.shape
    if k % 16:
        raise ValueError("NVFP4 needs K % 16 == 0")
    codes = np.empty((r, k // 2), dtype=np.uint8)
    bs = np.empty((r, k // 16), dtype=np.uint8)
    s = np.zeros(1, dtype=np.float32)
    st = lib().qo_quantize_nvfp4(_ptr(x), r, k, k, _ptr(codes), _ptr(bs), _ptr(s))
    if st == 6:
        raise NonFiniteInput("tensor holds inf or NaN")
    assert st == 0, st
    return codes, bs, np.float32(s[0])


# ---------------------------------------------------------------- dequantization
def dequant_fp8(codes: np.ndarray, scale, out: str = "f64") -> np.ndarray:
    c = _c(codes, np.uint8)
    if out == "f64":
        y = np.empty(c.shape, dtype=np.float64)
        lib().qo_dequant_fp8_f64(_ptr(c), c.size, float(scale), _ptr(y))
        return y
    y = np.empty(c.shape, dtype=np.float32)
    lib().qo_dequant_fp8_f32(_ptr(c), c.size, float(scale), _ptr(y))
    return y if out == "f32" else to_bf16(y)


def dequant_nvfp4(codes: np.ndarray, block_scales: np.ndarray, tscale, out: str = "f64") -> np.ndarray:
    c = _c(codes, np.uint8)
    b = _c(block_scales, np.uint8)
    rows, k = c.shape[0], c.shape[1] * 2
    assert b.shape == (rows, k // 16)
    if out == "f64":
        y = np.empty((rows, k), dtype=np.float64)
        lib().qo_dequant_nvfp4_f64(_ptr(c), _ptr(b), rows, k, float(tscale), _ptr(y))
        return y
    y = np.empty((rows, k), dtype=np.float32)
    lib().qo_dequant_nvfp4_f32(_ptr(c), _ptr(b), rows, k, float(tscale), _ptr(y))
    return y if out == "f32" else to_bf16(y)


def to_bf16(y32: np.ndarray) -> np.ndarray:
    y = _c(y32, np.float32)
    o = np.empty(y.shape, dtype=np.uint16)
    lib().qo_f32_to_bf16_array(_ptr(y), y.size, _ptr(o))
    return o


def bf16_to_f64(x_bf16: np.ndarray) -> np.ndarray:
    x = _c(x_bf16, np.uint16)
    y = np.empty(x.shape, dtype=np.float64)
    lib().qo_bf16_to_f64(_ptr(x), x.size, _ptr(y))
    return y


# ---------------------------------------------------------------- linear layer
def gemm_f64(a: np.ndarray, w: np.ndarray):
    """(y, b) with y = a . w^T in fp64 and b = sum_k |a w| for dequantized operands."""
    a = _c(a, np.float64)
    w = _c(w, np.float64)
    m, k = a.shape
    n, k2 = w.shape
    assert k == k2
    y = np.empty((m, n), dtype=np.float64)
    b = np.empty((m, n), dtype=np.float64)
    lib().qo_gemm_f64(_ptr(a), _ptr(w), m, n, k, _ptr(y), _ptr(b))
    return y, b


def gemm_f64_sampled(a: np.ndarray, w: np.ndarray, rows: np.ndarray, cols: np.ndarray):
    """y[s], b[s] for output (rows[s], cols[s]) of a . w^T."""
    a = _c(a, np.float64)
    w = _c(w, np.float64)
    rows = _c(rows, np.int64)
    cols = _c(cols, np.int64)
    k = a.shape[1]
    assert w.shape[1] == k and rows.shape == cols.shape
    y = np.empty(rows.shape, dtype=np.float64)
    b = np.empty(rows.shape, dtype=np.float64)
    lib().qo_gemm_f64_sampled(_ptr(a), _ptr(w), k, _ptr(rows), _ptr(cols), rows.size, _ptr(y), _ptr(b))
    return y, b


def num_threads() -> int:
    return lib().qo_num_threads()


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops (results do not depend on it)."""
    lib().qo_set_num_threads(int(n))


# ---------------------------------------------------------------- end-to-end references
def quantize_fp8_static(x_bf16: np.ndarray, s):
    """bf16 bits [R, K] and a calibrated decode scale s -> codes uint8 [R, K]."""
    x = _c(x_bf16, np.uint16)
    r, k = x.shape
    codes = np.empty((r, k), dtype=np.uint8)
    st = lib().qo_quantize_fp8_static(_ptr(x), r, k, k, float(np.float32(s)), _ptr(codes))
    if st == 6:
        raise NonFiniteInput("tensor holds inf or NaN")
    if st == 1:
        raise ValueError("scale must be 0 or a normal positive fp32")
    assert st == 0, st
    return codes


def quantize_nvfp4_static(x_bf16: np.ndarray, s_t):
    """bf16 bits [R, K] and a calibrated tensor decode scale s_t ->
    (codes uint8 [R, K/2], block scales uint8 [R, K/16])."""
    x = _c(x_bf16, np.uint16)
    r, k = x.shape
    if k % 16:
        raise ValueError("NVFP4 needs K % 16 == 0")
    codes = np.empty((r, k // 2), dtype=np.uint8)
    bs = np.empty((r, k // 16), dtype=np.uint8)
    st = lib().qo_quantize_nvfp4_static(_ptr(x), r, k, k, float(np.float32(s_t)), _ptr(codes), _ptr(bs))
    if st == 6:
        raise NonFiniteInput("tensor holds inf or NaN")
    if st == 1:
        raise ValueError("scale must be 0 or at least 2^-96")
    assert st == 0, st
    return codes, bs


def quantize_nvfp4_static_f32(y_f32: np.ndarray, s_t):
    """fp32 values [R, K] (a GEMM's fp32 output) and a static tensor decode
    scale s_t -> (codes uint8 [R, K/2], block scales uint8 [R, K/16]): the
    static NVFP4 steps on fp32 inputs."""
    y = _c(y_f32, np.float32)
    r, k = y.shape
    if k % 16:
        raise ValueError("NVFP4 needs K % 16 == 0")
    codes = np.empty((r, k // 2), dtype=np.uint8)
    bs = np.empty((r, k // 16), dtype=np.uint8)
    st = lib().qo_quantize_nvfp4_static_f32(_ptr(y), r, k, k, float(np.float32(s_t)), _ptr(codes), _ptr(bs))
    if st == 6:
        raise NonFiniteInput("tensor holds inf or NaN")
    if st == 1:
        raise ValueError("scale must be 0 or at least 2^-96")
    assert st == 0, st
    return codes, bs


def e8m0_table():
    """Values of the 255 finite E8M0 scale codes (code 255 is NaN)."""
    return np.array([lib().qo_e8m0_value(c) for c in range(256)])


def quantize_mx(x_bf16: np.ndarray, fmt: str):
    """bf16 bits [R, K] -> (codes, E8M0 scales uint8 [R, K/32]) for fmt in
    {"mxfp4", "mxfp8"} (OCP MX, blocks of 32 along K, no tensor scale)."""
    x = _c(x_bf16, np.uint16)
    r, k = x.shape
    if k % 32:
        raise ValueError("MX formats need K % 32 == 0")
    codes = np.zeros((r, k // 2) if fmt == "mxfp4" else (r, k), dtype=np.uint8)
    sc = np.empty((r, k // 32), dtype=np.uint8)
    fn = lib().qo_quantize_mxfp4 if fmt == "mxfp4" else lib().qo_quantize_mxfp8
    st = fn(_ptr(x), r, k, k, _ptr(codes), _ptr(sc))
    if st == 6:
        raise NonFiniteInput("tensor holds inf or NaN")
    assert st == 0, st
    return codes, sc


def dequant_mx(codes: np.ndarray, scales: np.ndarray, fmt: str) -> np.ndarray:
    """Exact (binary64) values of MX codes."""
    c = _c(codes, np.uint8)
    s = _c(scales, np.uint8)
    rows = c.shape[0]
    k = c.shape[1] * 2 if fmt == "mxfp4" else c.shape[1]
    y = np.empty((rows, k), dtype=np.float64)
    fn = lib().qo_dequant_mxfp4_f64 if fmt == "mxfp4" else lib().qo_dequant_mxfp8_f64
    fn(_ptr(c), _ptr(s), rows, k, _ptr(y))
    return y


def linear_reference(kind: str, x_bf16: np.ndarray, w_bf16: np.ndarray, rows=None, cols=None):
    """Oracle for one quantized linear Y = X . W^T.

    kind = "fp8"   : both operands FP8 E4M3, per-tensor scales (W8A8)
           "nvfp4" : both operands NVFP4 (W4A4)
           "w4a16" : X stays bf16, W is NVFP4
           "mxfp4" / "mxfp8": both operands in the OCP MX format (E2M1 / E4M3
                     elements, E8M0 scale per 32, no tensor scale)
    Returns dict with quantized operands, y (fp64) and b = sum|a w| for the
    full product, or for the (rows[s], cols[s]) samples when given.
    """
    out = {}
    if kind == "fp8":
        qa, sa = quantize_fp8(x_bf16)
        qw, sw = quantize_fp8(w_bf16)
        out.update(a_codes=qa, a_scale=sa, w_codes=qw, w_scale=sw)
        deq_a = lambda idx: dequant_fp8(qa[idx], sa)
        deq_w = lambda idx: dequant_fp8(qw[idx], sw)
    elif kind in ("nvfp4", "w4a16"):
        qw, bw, sw = quantize_nvfp4(w_bf16)
        out.update(w_codes=qw, w_bscales=bw, w_scale=sw)
        deq_w = lambda idx: dequant_nvfp4(qw[idx], bw[idx], sw)
        if kind == "nvfp4":
            qa, ba, sa = quantize_nvfp4(x_bf16)
            out.update(a_codes=qa, a_bscales=ba, a_scale=sa)
            deq_a = lambda idx: dequant_nvfp4(qa[idx], ba[idx], sa)
        else:
            deq_a = lambda idx: bf16_to_f64(x_bf16[idx])
    elif kind in ("mxfp4", "mxfp8"):
        qa, sa = quantize_mx(x_bf16, kind)
        qw, sw = quantize_mx(w_bf16, kind)
        out.update(a_codes=qa, a_bscales=sa, w_codes=qw, w_bscales=sw)
        deq_a = lambda idx: dequant_mx(qa[idx], sa[idx], kind)
        deq_w = lambda idx: dequant_mx(qw[idx], sw[idx], kind)
    else:
        raise ValueError(kind)
    if rows is None:
        all_m = np.arange(x_bf16.shape[0])
        all_n = np.arange(w_bf16.shape[0])
        y, b = gemm_f64(deq_a(all_m), deq_w(all_n))
    else:
        rows = np.asarray(rows, dtype=np.int64)
        cols = np.asarray(cols, dtype=np.int64)
        ur, ri = np.unique(rows, return_inverse=True)
        uc, ci = np.unique(cols, return_inverse=True)
        y, b = gemm_f64_sampled(deq_a(ur), deq_w(uc), ri, ci)
    out.update(y=y, b=b)
    return out

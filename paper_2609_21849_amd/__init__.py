"""MI355X (gfx950) low-bit quantized linear layers: Python binding of libqgemm.so.

The functions named ``qg_*`` mirror the C ABI in ``include/qgemm.h`` one to
one and only marshal arguments: torch tensors become device pointers, None
becomes NULL, and the stream defaults to torch's current stream. Every step
of the computation runs in the HIP kernels of ``libqgemm.so``; if the library
is missing this module raises instead of computing anything elsewhere.

A few helpers below (``quantize``, ``pack``, ``linear`` ...) allocate the
output tensors with torch and then call the same entry points.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libqgemm.so")

QG_FMT_BF16, QG_FMT_FP8_E4M3, QG_FMT_NVFP4, QG_FMT_MXFP4, QG_FMT_MXFP8 = 0, 1, 2, 3, 4
MX_FORMATS = (QG_FMT_MXFP4, QG_FMT_MXFP8)
QG_OUT_BF16, QG_OUT_F32 = 0, 1
QG_OK = 0
STATUS_NAMES = {0: "QG_OK", 1: "QG_ERR_INVALID_ARG", 2: "QG_ERR_UNSUPPORTED", 3: "QG_ERR_SHAPE",
                4: "QG_ERR_BUFFER_TOO_SMALL", 5: "QG_ERR_HIP"}
EXPORTS = ["qg_quantize_act", "qg_quantize_act_static", "qg_packed_bytes", "qg_pack_weights", "qg_unpack_weights", "qg_gemm",
           "qg_linear_fp8",
           "qg_gemm_quant", "qg_gemm_quant_nvfp4", "qg_dequant", "qg_run_layers", "qg_stream_simulate", "qg_stream_plan", "qg_status_string",
           "qg_last_hip_error", "qg_abi_version"]


class StreamLayer(ctypes.Structure):
    """qg_stream_layer of include/qgemm.h."""
    _fields_ = [("x", ctypes.c_void_p), ("a_fmt", ctypes.c_int), ("a_codes", ctypes.c_void_p),
                ("a_block_scales", ctypes.c_void_p), ("a_tensor_scale", ctypes.c_void_p),
                ("w_fmt", ctypes.c_int), ("w_packed", ctypes.c_void_p), ("w_packed_bytes", ctypes.c_size_t),
                ("resident", ctypes.c_int32), ("m", ctypes.c_int64), ("n", ctypes.c_int64), ("k", ctypes.c_int64),
                ("y", ctypes.c_void_p), ("y_dtype", ctypes.c_int)]


class QGError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s" % (where, STATUS_NAMES.get(status, status)))


_lib = None


def lib() -> ctypes.CDLL:
    """Load libqgemm.so; raise loudly when it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libqgemm.so is not built (run `python -m paper_2609_21849_amd.build` "
                              "or __graft_entry__.build()); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
        L.qg_quantize_act.restype = I32
        L.qg_quantize_act.argtypes = [I32, P, I64, I64, I64, P, P, P, P]
        L.qg_quantize_act_static.restype = I32
        L.qg_quantize_act_static.argtypes = [I32, P, I64, I64, I64, P, P, P, P]
        L.qg_packed_bytes.restype = SZ
        L.qg_packed_bytes.argtypes = [I32, I64, I64]
        L.qg_pack_weights.restype = I32
        L.qg_pack_weights.argtypes = [I32, P, P, P, I64, I64, P, SZ, P]
        L.qg_unpack_weights.restype = I32
        L.qg_unpack_weights.argtypes = [I32, P, SZ, I64, I64, P, P, P, P]
        L.qg_gemm.restype = I32
        L.qg_gemm.argtypes = [I32, P, P, P, I64, I32, P, SZ, I64, I64, I64, P, I64, I32, P]
        L.qg_linear_fp8.restype = I32
        L.qg_linear_fp8.argtypes = [P, I64, P, P, SZ, I64, I64, I64, P, I64, I32, P]
        L.qg_gemm_quant.restype = I32
        L.qg_gemm_quant.argtypes = [I32, P, P, P, I64, I32, P, SZ, I64, I64, I64, P, I64, P, P]
        L.qg_gemm_quant_nvfp4.restype = I32
        L.qg_gemm_quant_nvfp4.argtypes = [I32, P, P, P, I64, I32, P, SZ, I64, I64, I64, P, P, I64, P, P]
        L.qg_dequant.restype = I32
        L.qg_dequant.argtypes = [I32, P, P, P, I64, I64, P, I32, P]
        D, U8 = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_uint8)
        L.qg_run_layers.restype = I32
        L.qg_run_layers.argtypes = [ctypes.POINTER(StreamLayer), ctypes.c_int32, ctypes.POINTER(P), ctypes.c_int32, SZ,
                                    ctypes.POINTER(P), ctypes.POINTER(P), ctypes.POINTER(ctypes.c_int32), P, P]
        L.qg_stream_simulate.restype = I32
        L.qg_stream_simulate.argtypes = [ctypes.c_int32, D, D, U8, ctypes.c_int32, ctypes.c_double, ctypes.c_int32, D]
        L.qg_stream_plan.restype = I32
        L.qg_stream_plan.argtypes = [ctypes.c_int32, D, D, ctypes.c_int32, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_double, U8, D, D]
        L.qg_status_string.restype = ctypes.c_char_p
        L.qg_status_string.argtypes = [I32]
        L.qg_last_hip_error.restype = I32
        L.qg_abi_version.restype = I32
        _lib = L
    return _lib


def _p(t) -> int | None:
    """Device pointer of a CUDA tensor (or an int pointer, passed as given);
    None -> NULL. A tensor in host memory is refused: the kernels would
    dereference its address on the GPU."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not getattr(t, "is_cuda", False):
        raise ValueError("expected a CUDA tensor, got one on %s" % (getattr(t, "device", type(t).__name__),))
    return t.data_ptr()


def _need(t, name: str, dtype, shape=None, device=None, dense: bool = True) -> None:
    """Checks a tensor argument of the allocating helpers: on the GPU, of
    `dtype`, of `shape` (if given), on `device` (if given), and dense
    (contiguous) or at least unit-stride along its rows. The C ABI sees only
    pointers and sizes, so a wrong element type or shape would otherwise
    become an out-of-bounds access on the GPU."""
    if t is None or not getattr(t, "is_cuda", False):
        raise ValueError("%s: expected a CUDA tensor, got %r" % (name, getattr(t, "device", t)))
    if t.dtype != dtype:
        raise ValueError("%s: expected dtype %s, got %s" % (name, dtype, t.dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s: expected shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if device is not None and t.device != device:
        raise ValueError("%s: on %s, expected %s" % (name, t.device, device))
    if dense and not t.is_contiguous():
        raise ValueError("%s: expected a contiguous tensor" % name)
    if not dense and (t.dim() != 2 or t.stride(1) != 1):
        raise ValueError("%s: expected a 2-D tensor with unit stride along its rows" % name)


def _need_q(q) -> None:
    """Checks a QTensor: codes, block scales and tensor scale of the shapes
    and types its format defines, all on one GPU."""
    import torch
    if not isinstance(q, QTensor):
        raise ValueError("expected a QTensor, got %s" % type(q).__name__)
    r, c = q.rows, q.cols
    code_cols = c if q.fmt in (QG_FMT_FP8_E4M3, QG_FMT_MXFP8) else c // 2
    _need(q.codes, "codes", torch.uint8, (r, code_cols))
    dev = q.codes.device
    if q.fmt == QG_FMT_FP8_E4M3:
        if q.block_scales is not None:
            raise ValueError("FP8 tensors have no block scales")
    else:
        _need(q.block_scales, "block_scales", torch.uint8, (r, c // (32 if q.fmt in MX_FORMATS else 16)), dev)
    if q.fmt in MX_FORMATS:
        if q.tensor_scale is not None:
            raise ValueError("MX tensors have no tensor scale")
    else:
        _need(q.tensor_scale, "tensor_scale", torch.float32, None, dev)
        if q.tensor_scale.numel() < 1:
            raise ValueError("tensor_scale: expected one element")


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, where: str) -> None:
    if status != QG_OK:
        raise QGError(status, where)


# ---------------------------------------------------------------- the C ABI, one to one
def qg_quantize_act(fmt, x, rows, cols, ldx, codes, block_scales, tensor_scale, stream=None, check=True):
    s = lib().qg_quantize_act(fmt, _p(x), rows, cols, ldx, _p(codes), _p(block_scales), _p(tensor_scale), _stream(stream))
    if check:
        _check(s, "qg_quantize_act")
    return s


def qg_quantize_act_static(fmt, x, rows, cols, ldx, codes, block_scales, tensor_scale, stream=None, check=True):
    s = lib().qg_quantize_act_static(fmt, _p(x), rows, cols, ldx, _p(codes), _p(block_scales), _p(tensor_scale),
                                     _stream(stream))
    if check:
        _check(s, "qg_quantize_act_static")
    return s


def qg_packed_bytes(fmt, n, k) -> int:
    return lib().qg_packed_bytes(fmt, n, k)


def qg_pack_weights(fmt, codes, block_scales, tensor_scale, n, k, packed, packed_bytes, stream=None, check=True):
    s = lib().qg_pack_weights(fmt, _p(codes), _p(block_scales), _p(tensor_scale), n, k, _p(packed), packed_bytes, _stream(stream))
    if check:
        _check(s, "qg_pack_weights")
    return s


def qg_unpack_weights(fmt, packed, packed_bytes, n, k, codes, block_scales, tensor_scale, stream=None, check=True):
    s = lib().qg_unpack_weights(fmt, _p(packed), packed_bytes, n, k, _p(codes), _p(block_scales), _p(tensor_scale), _stream(stream))
    if check:
        _check(s, "qg_unpack_weights")
    return s


def qg_gemm(a_fmt, a, a_block_scales, a_tensor_scale, lda, w_fmt, w_packed, w_packed_bytes, m, n, k,
            y, ldy, y_dtype, stream=None, check=True):
    s = lib().qg_gemm(a_fmt, _p(a), _p(a_block_scales), _p(a_tensor_scale), lda, w_fmt, _p(w_packed),
                      w_packed_bytes, m, n, k, _p(y), ldy, y_dtype, _stream(stream))
    if check:
        _check(s, "qg_gemm")
    return s


def qg_linear_fp8(x, ldx, a_tensor_scale, w_packed, w_packed_bytes, m, n, k, y, ldy, y_dtype, stream=None,
                  check=True):
    s = lib().qg_linear_fp8(_p(x), ldx, _p(a_tensor_scale), _p(w_packed), w_packed_bytes, m, n, k, _p(y), ldy,
                            y_dtype, _stream(stream))
    if check:
        _check(s, "qg_linear_fp8")
    return s


def qg_gemm_quant(a_fmt, a, a_block_scales, a_tensor_scale, lda, w_fmt, w_packed, w_packed_bytes, m, n, k,
                  y_codes, ldy, y_scale, stream=None, check=True):
    s = lib().qg_gemm_quant(a_fmt, _p(a), _p(a_block_scales), _p(a_tensor_scale), lda, w_fmt, _p(w_packed),
                            w_packed_bytes, m, n, k, _p(y_codes), ldy, _p(y_scale), _stream(stream))
    if check:
        _check(s, "qg_gemm_quant")
    return s


def qg_gemm_quant_nvfp4(a_fmt, a, a_block_scales, a_tensor_scale, lda, w_fmt, w_packed, w_packed_bytes, m, n, k,
                        y_codes, y_block_scales, ldy, y_tensor_scale, stream=None, check=True):
    s = lib().qg_gemm_quant_nvfp4(a_fmt, _p(a), _p(a_block_scales), _p(a_tensor_scale), lda, w_fmt, _p(w_packed),
                                  w_packed_bytes, m, n, k, _p(y_codes), _p(y_block_scales), ldy,
                                  _p(y_tensor_scale), _stream(stream))
    if check:
        _check(s, "qg_gemm_quant_nvfp4")
    return s


def linear_nvfp4_out(a, w_packed, w_fmt: int, n: int, y_tensor_scale, stream=None) -> "QTensor":
    """Y = A . W^T written as NVFP4 codes and E4M3 block scales with the static
    tensor decode scale y_tensor_scale (a one-element fp32 CUDA tensor): the
    next linear's 4-bit activation."""
    import torch
    m, k, a_fmt, a_data, a_bs, a_ts, lda, dev = _operands(a, w_packed)
    _need(y_tensor_scale, "y_tensor_scale", torch.float32, None, dev)
    codes = torch.empty((m, n // 2), dtype=torch.uint8, device=dev)
    bs = torch.empty((m, n // 16), dtype=torch.uint8, device=dev)
    qg_gemm_quant_nvfp4(a_fmt, a_data, a_bs, a_ts, lda, w_fmt, w_packed, w_packed.numel(), m, n, k, codes, bs, n,
                        y_tensor_scale, stream)
    return QTensor(QG_FMT_NVFP4, codes, bs, y_tensor_scale, m, n)


def linear_fp8(x, w_packed, n: int, out_dtype: int = QG_OUT_BF16, stream=None):
    """Y = Q(x) . W^T from a bf16 activation x [m, k] (rows 16-byte aligned):
    the FP8 activation quantization inside the GEMM. Returns (y, the
    activation's decode scale as a one-element fp32 tensor)."""
    import torch
    _need(x, "x", torch.bfloat16, dense=False)
    _need(w_packed, "w_packed", torch.uint8, None, x.device)
    m, k = x.shape
    ts = torch.empty(1, dtype=torch.float32, device=x.device)
    y = torch.empty((m, n), dtype=torch.float32 if out_dtype == QG_OUT_F32 else torch.bfloat16, device=x.device)
    ldx = x.stride(0) if m > 1 else k
    qg_linear_fp8(x, ldx, ts, w_packed, w_packed.numel(), m, n, k, y, n, out_dtype, stream)
    return y, ts


def linear_fp8_out(a, w_packed, w_fmt: int, n: int, y_scale, stream=None) -> "QTensor":
    """Y = A . W^T written as FP8 E4M3 codes with the static decode scale
    y_scale (a one-element fp32 CUDA tensor): the next linear's activation."""
    import torch
    m, k, a_fmt, a_data, a_bs, a_ts, lda, dev = _operands(a, w_packed)
    _need(y_scale, "y_scale", torch.float32, None, dev)
    codes = torch.empty((m, n), dtype=torch.uint8, device=dev)
    qg_gemm_quant(a_fmt, a_data, a_bs, a_ts, lda, w_fmt, w_packed, w_packed.numel(), m, n, k, codes, n, y_scale,
                  stream)
    return QTensor(QG_FMT_FP8_E4M3, codes, None, y_scale, m, n)


def _doubles(v):
    arr = (ctypes.c_double * max(1, len(v)))(*[float(x) for x in v])
    return arr


def qg_run_layers(layers, slots, slot_bytes, slot_ready, slot_free, slot_cursor, compute_stream=None,
                  copy_stream=None, check=True):
    """layers: sequence of StreamLayer; slots: device pointers (ints or
    tensors); slot_ready / slot_free: hipEvent_t handles (ints, e.g.
    torch.cuda.Event.cuda_event); slot_cursor: a ctypes.c_int32, updated."""
    arr = (StreamLayer * max(1, len(layers)))(*layers)
    n_slots = len(slots)
    sp = (ctypes.c_void_p * max(1, n_slots))(*[_p(t) for t in slots])
    rp = (ctypes.c_void_p * max(1, n_slots))(*slot_ready)
    fp = (ctypes.c_void_p * max(1, n_slots))(*slot_free)
    s = lib().qg_run_layers(arr, len(layers), sp, n_slots, slot_bytes, rp, fp, ctypes.byref(slot_cursor),
                            _stream(compute_stream), _stream(copy_stream))
    if check:
        _check(s, "qg_run_layers")
    return s


def qg_stream_simulate(w_bytes, compute_s, resident, n_slots, h2d_bytes_per_s, steps=3, check=True):
    """Returns (status, step seconds of the last pass)."""
    n = len(w_bytes)
    res = (ctypes.c_uint8 * max(1, n))(*[1 if r else 0 for r in resident])
    out = ctypes.c_double(0.0)
    s = lib().qg_stream_simulate(n, _doubles(w_bytes), _doubles(compute_s), res, n_slots, h2d_bytes_per_s, steps,
                                 ctypes.byref(out))
    if check:
        _check(s, "qg_stream_simulate")
    return s, out.value


def qg_stream_plan(w_bytes, compute_s, n_slots, h2d_bytes_per_s, budget_bytes, act_peak_bytes, check=True):
    """Returns (status, resident flags, step seconds, device bytes)."""
    n = len(w_bytes)
    res = (ctypes.c_uint8 * max(1, n))()
    t, b = ctypes.c_double(0.0), ctypes.c_double(0.0)
    s = lib().qg_stream_plan(n, _doubles(w_bytes), _doubles(compute_s), n_slots, h2d_bytes_per_s, budget_bytes,
                             act_peak_bytes, res, ctypes.byref(t), ctypes.byref(b))
    if check:
        _check(s, "qg_stream_plan")
    return s, [int(res[i]) for i in range(n)], t.value, b.value


def qg_dequant(fmt, codes, block_scales, tensor_scale, rows, cols, out, out_dtype, stream=None, check=True):
    s = lib().qg_dequant(fmt, _p(codes), _p(block_scales), _p(tensor_scale), rows, cols, _p(out), out_dtype, _stream(stream))
    if check:
        _check(s, "qg_dequant")
    return s


def qg_status_string(status: int) -> str:
    return lib().qg_status_string(status).decode()


def qg_last_hip_error() -> int:
    return lib().qg_last_hip_error()


def qg_abi_version() -> int:
    return lib().qg_abi_version()


# ---------------------------------------------------------------- allocating helpers
@dataclass
class QTensor:
    """A quantized tensor on the GPU: codes, block scales (NVFP4, MX) and the
    fp32 tensor scale (None for the MX formats, which have none)."""
    fmt: int
    codes: "object"
    block_scales: "object"
    tensor_scale: "object"
    rows: int
    cols: int


def quantize(x, fmt: int, stream=None, static_scale=None) -> QTensor:
    """Quantize a [rows, cols] bf16 CUDA tensor (row stride may exceed cols).
    With static_scale (a one-element fp32 CUDA tensor holding a calibrated
    decode scale) the scale is used as given instead of derived from x."""
    import torch
    _need(x, "x", torch.bfloat16, dense=False)
    rows, cols = x.shape
    dev = x.device
    if static_scale is not None:
        _need(static_scale, "static_scale", torch.float32, None, dev)
        if static_scale.numel() < 1:
            raise ValueError("static_scale: expected one element")
    if fmt == QG_FMT_FP8_E4M3:
        codes = torch.empty((rows, cols), dtype=torch.uint8, device=dev)
        bs = None
    elif fmt in MX_FORMATS:
        codes = torch.empty((rows, cols if fmt == QG_FMT_MXFP8 else cols // 2), dtype=torch.uint8, device=dev)
        bs = torch.empty((rows, cols // 32), dtype=torch.uint8, device=dev)
    else:
        codes = torch.empty((rows, cols // 2), dtype=torch.uint8, device=dev)
        bs = torch.empty((rows, cols // 16), dtype=torch.uint8, device=dev)
    ldx = x.stride(0) if rows > 1 else cols   # a size-1 dimension may carry any stride
    if fmt in MX_FORMATS:
        qg_quantize_act(fmt, x, rows, cols, ldx, codes, bs, None, stream)
        return QTensor(fmt, codes, bs, None, rows, cols)
    if static_scale is not None:
        qg_quantize_act_static(fmt, x, rows, cols, ldx, codes, bs, static_scale, stream)
        return QTensor(fmt, codes, bs, static_scale, rows, cols)
    ts = torch.empty(1, dtype=torch.float32, device=dev)
    qg_quantize_act(fmt, x, rows, cols, ldx, codes, bs, ts, stream)
    return QTensor(fmt, codes, bs, ts, rows, cols)


def pack(q: QTensor, stream=None):
    """Pack a quantized weight [n, k] for qg_gemm; returns a uint8 CUDA tensor."""
    import torch
    _need_q(q)
    nbytes = qg_packed_bytes(q.fmt, q.rows, q.cols)
    if nbytes == 0:
        raise QGError(3, "qg_packed_bytes")
    packed = torch.empty(nbytes, dtype=torch.uint8, device=q.codes.device)
    qg_pack_weights(q.fmt, q.codes, q.block_scales, q.tensor_scale, q.rows, q.cols, packed, nbytes, stream)
    return packed


def unpack(packed, fmt: int, n: int, k: int, stream=None) -> QTensor:
    import torch
    _need(packed, "packed", torch.uint8)
    dev = packed.device
    if fmt == QG_FMT_FP8_E4M3:
        codes, bs = torch.empty((n, k), dtype=torch.uint8, device=dev), None
    elif fmt in MX_FORMATS:
        codes = torch.empty((n, k if fmt == QG_FMT_MXFP8 else k // 2), dtype=torch.uint8, device=dev)
        bs = torch.empty((n, k // 32), dtype=torch.uint8, device=dev)
    else:
        codes = torch.empty((n, k // 2), dtype=torch.uint8, device=dev)
        bs = torch.empty((n, k // 16), dtype=torch.uint8, device=dev)
    ts = None if fmt in MX_FORMATS else torch.empty(1, dtype=torch.float32, device=dev)
    qg_unpack_weights(fmt, packed, packed.numel(), n, k, codes, bs, ts, stream)
    return QTensor(fmt, codes, bs, ts, n, k)


def _operands(a, w_packed):
    """(m, k, a_fmt, data, block scales, tensor scale, lda, device) of a
    linear's activation operand, checked, and the packed weight checked."""
    import torch
    if isinstance(a, QTensor):
        _need_q(a)
        dev = a.codes.device
        out = (a.rows, a.cols, a.fmt, a.codes, a.block_scales, a.tensor_scale, a.cols, dev)
    else:
        _need(a, "a", torch.bfloat16, dense=False)
        m, k = a.shape
        dev = a.device
        out = (m, k, QG_FMT_BF16, a, None, None, a.stride(0) if m > 1 else k, dev)
    _need(w_packed, "w_packed", torch.uint8, None, dev)
    return out


def linear(a, w_packed, w_fmt: int, n: int, out_dtype: int = QG_OUT_BF16, y=None, stream=None):
    """Y = A . W^T for a quantized A (QTensor) or a bf16 A (torch tensor)."""
    import torch
    m, k, a_fmt, a_data, a_bs, a_ts, lda, dev = _operands(a, w_packed)
    if out_dtype not in (QG_OUT_BF16, QG_OUT_F32):
        raise ValueError("out_dtype must be QG_OUT_BF16 or QG_OUT_F32")
    ydt = torch.float32 if out_dtype == QG_OUT_F32 else torch.bfloat16
    if y is None:
        y = torch.empty((m, n), dtype=ydt, device=dev)
    else:
        _need(y, "y", ydt, (m, n), dev, dense=False)
    ldy = y.stride(0) if m > 1 else n
    qg_gemm(a_fmt, a_data, a_bs, a_ts, lda, w_fmt, w_packed, w_packed.numel(), m, n, k, y, ldy, out_dtype, stream)
    return y


def dequantize(q: QTensor, out_dtype: int = QG_OUT_F32, stream=None):
    import torch
    _need_q(q)
    out = torch.empty((q.rows, q.cols), dtype=torch.float32 if out_dtype == QG_OUT_F32 else torch.bfloat16,
                      device=q.codes.device)
    qg_dequant(q.fmt, q.codes, q.block_scales, q.tensor_scale, q.rows, q.cols, out, out_dtype, stream)
    return out

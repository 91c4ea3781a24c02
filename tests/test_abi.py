"""C-ABI checks that need no GPU: the library loads, exports every function
include/qgemm.h declares, and rejects bad arguments on the host with the
documented status codes before any HIP call.

Every call below is built to FAIL validation (fake pointers are never
dereferenced), so the tests are also safe on a machine with a GPU.
"""
import ctypes
import os
import re

import pytest

import paper_2609_21849_amd as q

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qgemm.h")

OK, INVALID, UNSUP, SHAPE, SMALL = 0, 1, 2, 3, 4
FP8, NVFP4, BF16 = q.QG_FMT_FP8_E4M3, q.QG_FMT_NVFP4, q.QG_FMT_BF16
P = 0x10000  # a fake, 64 KiB-aligned "device pointer" that validation never dereferences


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qg_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 9
    L = ctypes.CDLL(q.LIB_PATH)
    for name in names:
        assert hasattr(L, name), name
    assert sorted(names) == sorted(q.EXPORTS)


def test_abi_version_and_status_strings():
    assert q.qg_abi_version() == 1
    for s in range(6):
        assert q.qg_status_string(s)
    assert q.qg_status_string(OK) == "ok"
    assert q.qg_last_hip_error() == 0


def test_packed_bytes():
    assert q.qg_packed_bytes(FP8, 256, 256) == 256 + 256 * 256
    assert q.qg_packed_bytes(NVFP4, 3072, 3072) == 256 + 3072 * 3072 // 2 + 3072 * 3072 // 16
    assert q.qg_packed_bytes(NVFP4, 0, 0) == 256
    assert q.qg_packed_bytes(FP8, 24, 256) == 0      # n % 16
    assert q.qg_packed_bytes(FP8, 256, 192) == 0     # k % 128
    assert q.qg_packed_bytes(BF16, 256, 256) == 0
    assert q.qg_packed_bytes(7, 256, 256) == 0


def _quant(fmt, x=P, rows=4, cols=32, ldx=32, codes=P, bs=P, ts=P):
    return q.qg_quantize_act(fmt, x, rows, cols, ldx, codes, bs, ts, stream=0, check=False)


def test_quantize_validation():
    assert _quant(9) == INVALID
    assert _quant(BF16) == UNSUP
    assert _quant(NVFP4, cols=24, ldx=24) == SHAPE
    assert _quant(NVFP4, ts=None) == INVALID
    assert _quant(NVFP4, x=None) == INVALID
    assert _quant(NVFP4, bs=None) == INVALID
    assert _quant(NVFP4, codes=P + 4) == INVALID          # codes need 8-byte alignment
    assert _quant(NVFP4, ldx=16) == INVALID               # ldx < cols
    assert _quant(NVFP4, rows=-1) == INVALID
    assert _quant(FP8, bs=P) == INVALID                   # FP8 has no block scales
    assert _quant(FP8, bs=None, x=P + 1) == INVALID       # bf16 needs 2-byte alignment
    assert _quant(FP8, bs=None, ts=P + 2) == INVALID


def _quant_static(fmt, x=P, rows=4, cols=32, ldx=32, codes=P, bs=P, ts=P):
    return q.qg_quantize_act_static(fmt, x, rows, cols, ldx, codes, bs, ts, stream=0, check=False)


def test_static_quantize_validation():
    assert _quant_static(9) == INVALID
    assert _quant_static(BF16) == UNSUP
    assert _quant_static(NVFP4, cols=24, ldx=24) == SHAPE
    assert _quant_static(NVFP4, ts=None) == INVALID
    assert _quant_static(NVFP4, x=None) == INVALID
    assert _quant_static(NVFP4, bs=None) == INVALID
    assert _quant_static(NVFP4, codes=P + 4) == INVALID
    assert _quant_static(NVFP4, ldx=16) == INVALID
    assert _quant_static(FP8, bs=P) == INVALID
    assert _quant_static(FP8, bs=None, ts=P + 2) == INVALID


def _pack(fmt, codes=P, bs=P, ts=P, n=32, k=128, packed=P, nbytes=1 << 20, unpack=False):
    if unpack:
        return q.qg_unpack_weights(fmt, packed, nbytes, n, k, codes, bs, ts, stream=0, check=False)
    return q.qg_pack_weights(fmt, codes, bs, ts, n, k, packed, nbytes, stream=0, check=False)


@pytest.mark.parametrize("unpack", [False, True])
def test_pack_validation(unpack):
    assert _pack(5, unpack=unpack) == INVALID
    assert _pack(BF16, unpack=unpack) == UNSUP
    assert _pack(NVFP4, n=24, unpack=unpack) == SHAPE
    assert _pack(NVFP4, k=64, unpack=unpack) == SHAPE
    assert _pack(NVFP4, nbytes=100, unpack=unpack) == SMALL
    assert _pack(NVFP4, packed=P + 128, unpack=unpack) == INVALID     # 256-byte alignment
    assert _pack(NVFP4, codes=P + 8, unpack=unpack) == INVALID
    assert _pack(NVFP4, bs=None, unpack=unpack) == INVALID
    assert _pack(FP8, unpack=unpack) == INVALID                       # FP8 with block scales
    assert _pack(NVFP4, ts=None, unpack=unpack) == INVALID


def _gemm(a_fmt=NVFP4, w_fmt=NVFP4, a=P, abs_=P, ats=P, lda=256, wp=P, wbytes=1 << 24,
          m=32, n=64, k=256, y=P, ldy=64, yd=0):
    return q.qg_gemm(a_fmt, a, abs_, ats, lda, w_fmt, wp, wbytes, m, n, k, y, ldy, yd, stream=0, check=False)


def test_gemm_validation():
    assert _gemm(a_fmt=7) == INVALID
    assert _gemm(yd=3) == INVALID
    assert _gemm(a_fmt=FP8, w_fmt=NVFP4) == UNSUP
    assert _gemm(a_fmt=NVFP4, w_fmt=FP8) == UNSUP
    assert _gemm(a_fmt=BF16, w_fmt=BF16) == UNSUP
    assert _gemm(a_fmt=BF16, w_fmt=FP8) == UNSUP
    assert _gemm(n=40) == SHAPE
    assert _gemm(k=200, lda=200) == SHAPE
    assert _gemm(m=-1) == INVALID
    assert _gemm(ldy=32) == INVALID
    assert _gemm(lda=128) == INVALID
    assert _gemm(wbytes=1000) == SMALL
    assert _gemm(wp=P + 16) == INVALID
    assert _gemm(wp=None) == INVALID
    assert _gemm(y=None) == INVALID
    assert _gemm(a=None) == INVALID
    assert _gemm(abs_=None) == INVALID                                   # W4A4 needs A block scales
    assert _gemm(lda=320) == INVALID                                     # W4A4 row pitch % 128
    assert _gemm(lda=512) not in (INVALID, SHAPE)                        # a slice of a wider tensor
    assert _gemm(m=70000, lda=65536) == SHAPE                            # scales + codes above 2 GiB
    assert _gemm(a_fmt=FP8, w_fmt=FP8, abs_=None, a=P + 8) == INVALID     # 16-byte alignment
    # operand extents above 2 GiB (32-bit buffer offsets)
    assert _gemm(a_fmt=FP8, w_fmt=FP8, abs_=None, m=70000, lda=32768, k=32768) == SHAPE
    assert _gemm(a_fmt=BF16, abs_=None, ats=None, m=40000, lda=32768, k=32768) == SHAPE
    assert _gemm(a_fmt=FP8, w_fmt=FP8, abs_=None, ats=None) == INVALID
    assert _gemm(a_fmt=FP8, w_fmt=FP8) == INVALID                         # FP8 A has no block scales
    assert _gemm(a_fmt=BF16, abs_=None, ats=P) == INVALID                 # bf16 A has no scales
    assert _gemm(a_fmt=BF16, abs_=None, ats=None, lda=260) == INVALID      # lda % 8


def test_dequant_validation():
    def dq(fmt, codes=P, bs=P, ts=P, rows=4, cols=32, out=P, od=0):
        return q.qg_dequant(fmt, codes, bs, ts, rows, cols, out, od, stream=0, check=False)
    assert dq(8) == INVALID
    assert dq(BF16) == UNSUP
    assert dq(NVFP4, cols=20) == SHAPE
    assert dq(NVFP4, od=5) == INVALID
    assert dq(NVFP4, ts=None) == INVALID
    assert dq(NVFP4, bs=None) == INVALID
    assert dq(NVFP4, out=None) == INVALID
    assert dq(FP8) == INVALID                                            # FP8 with block scales
    assert dq(NVFP4, out=P + 2, od=1) == INVALID                          # fp32 out alignment


MXFP4, MXFP8 = q.QG_FMT_MXFP4, q.QG_FMT_MXFP8


def test_mx_packed_bytes():
    # header + E2M1 codes + one E8M0 scale per 32 elements
    assert q.qg_packed_bytes(MXFP4, 64, 256) == 256 + 64 * 256 // 2 + 64 * 256 // 32
    assert q.qg_packed_bytes(MXFP4, 48, 512) == 256 + 64 * 512 // 2 + 64 * 512 // 32   # 32-row panels
    assert q.qg_packed_bytes(MXFP4, 64, 128) == 0     # MXFP4 weights need k % 256
    assert q.qg_packed_bytes(MXFP8, 64, 256) == 256 + 64 * 256 + 64 * 256 // 32
    assert q.qg_packed_bytes(MXFP8, 64, 384) == 0     # MX weights need k % 256


def test_mx_quantize_validation():
    assert _quant(MXFP4) == INVALID                                   # MX has no tensor scale
    assert _quant(MXFP8) == INVALID
    assert _quant(MXFP4, ts=None, cols=48, ldx=48) == SHAPE           # cols % 32
    assert _quant(MXFP8, ts=None, cols=16, ldx=16) == SHAPE
    assert _quant(MXFP4, ts=None, bs=None) == INVALID                 # block scales required
    assert _quant(MXFP4, ts=None, codes=P + 2) == INVALID             # 4-byte code stores
    assert _quant(MXFP4, ts=None, x=None) == INVALID
    assert _quant(MXFP4, ts=None, x=P + 1) == INVALID
    assert _quant(MXFP8, ts=None, ldx=16) == INVALID                  # ldx < cols
    assert _quant_static(MXFP4) == UNSUP                              # no static MX scale
    assert _quant_static(MXFP8, ts=None) == UNSUP


@pytest.mark.parametrize("unpack", [False, True])
def test_mx_pack_validation(unpack):
    assert _pack(MXFP8, ts=None, k=384, unpack=unpack) == SHAPE       # k % 256
    assert _pack(MXFP8, k=256, unpack=unpack) == INVALID              # no tensor scale
    assert _pack(MXFP4, ts=None, k=128, unpack=unpack) == SHAPE       # k % 256
    assert _pack(MXFP4, ts=None, n=24, k=256, unpack=unpack) == SHAPE
    assert _pack(MXFP4, k=256, unpack=unpack) == INVALID              # no tensor scale
    assert _pack(MXFP4, ts=None, bs=None, k=256, unpack=unpack) == INVALID
    assert _pack(MXFP4, ts=None, k=256, nbytes=4000, unpack=unpack) == SMALL


def test_mx_gemm_validation():
    mx = dict(a_fmt=MXFP4, w_fmt=MXFP4, ats=None)
    assert _gemm(a_fmt=MXFP4, w_fmt=NVFP4, ats=None) == UNSUP
    assert _gemm(a_fmt=NVFP4, w_fmt=MXFP4) == UNSUP
    assert _gemm(a_fmt=MXFP8, w_fmt=MXFP4, ats=None) == UNSUP
    assert _gemm(a_fmt=MXFP8, w_fmt=MXFP8, ats=None, k=384, lda=384) == SHAPE
    assert _gemm(a_fmt=MXFP8, w_fmt=MXFP8) == INVALID                 # no tensor scale
    assert _gemm(a_fmt=MXFP8, w_fmt=MXFP8, ats=None, abs_=P + 2) == INVALID   # 4-byte aligned scales
    assert _gemm(a_fmt=MXFP8, w_fmt=MXFP8, ats=None, lda=512) == INVALID      # dense codes
    assert _gemm(a_fmt=BF16, w_fmt=MXFP4, abs_=None, ats=None) == UNSUP
    assert _gemm(**mx, k=384, lda=384) == SHAPE                       # k % 256
    assert _gemm(a_fmt=MXFP4, w_fmt=MXFP4) == INVALID                 # MX A has no tensor scale
    assert _gemm(**mx, abs_=None) == INVALID                          # A block scales required
    assert _gemm(**mx, abs_=P + 4) == INVALID                         # 8-byte aligned scales
    assert _gemm(**mx, lda=512) == INVALID                            # dense codes
    assert _gemm(**mx, a=P + 8) == INVALID
    assert _gemm(**mx, m=70000, k=65536, lda=65536) == SHAPE          # codes above 2 GiB


def test_mx_dequant_validation():
    def dq(fmt, codes=P, bs=P, ts=None, rows=4, cols=64, out=P, od=1):
        return q.qg_dequant(fmt, codes, bs, ts, rows, cols, out, od, stream=0, check=False)
    assert dq(MXFP4, ts=P) == INVALID                                 # no tensor scale
    assert dq(MXFP4, cols=48) == SHAPE
    assert dq(MXFP8, cols=16) == SHAPE
    assert dq(MXFP4, bs=None) == INVALID
    assert dq(MXFP4, out=None) == INVALID
    assert dq(MXFP4, out=P + 8) == INVALID                            # 16-byte stores
    assert dq(MXFP4, codes=P + 2) == INVALID                          # 4-byte code loads
    assert dq(MXFP8, codes=P + 4) == INVALID                          # 8-byte code loads


def test_gemm_quant_validation():
    def gq(a_fmt=FP8, w_fmt=FP8, abs_=None, ats=P, lda=256, y=P, ldy=64, ys=P, m=32, n=64, k=256, wbytes=1 << 24):
        return q.qg_gemm_quant(a_fmt, P, abs_, ats, lda, w_fmt, P, wbytes, m, n, k, y, ldy, ys, stream=0, check=False)
    assert gq(ys=None) == INVALID                      # the output's decode scale is required
    assert gq(ys=P + 2) == INVALID
    assert gq(a_fmt=FP8, w_fmt=NVFP4) == UNSUP
    assert gq(n=40) == SHAPE
    assert gq(ldy=32) == INVALID                       # ldy < n
    assert gq(y=None) == INVALID
    assert gq(wbytes=100) == SMALL
    assert gq(ats=None) == INVALID                     # the GEMM's own operand checks


def test_gemm_quant_nvfp4_validation():
    def gq(a_fmt=NVFP4, w_fmt=NVFP4, abs_=P, ats=P, lda=256, y=P, ybs=P, ldy=64, ys=P, m=32, n=64, k=256,
           wbytes=1 << 24):
        return q.qg_gemm_quant_nvfp4(a_fmt, P, abs_, ats, lda, w_fmt, P, wbytes, m, n, k, y, ybs, ldy, ys,
                                     stream=0, check=False)
    assert gq(ys=None) == INVALID                      # the output's tensor scale is required
    assert gq(ys=P + 2) == INVALID
    assert gq(ybs=None) == INVALID                     # block scales out
    assert gq(y=P + 2) == INVALID                      # 4-byte aligned codes
    assert gq(ldy=72) == INVALID                       # ldy % 16
    assert gq(ldy=32) == INVALID                       # ldy < n
    assert gq(a_fmt=BF16, abs_=None, ats=None) == UNSUP  # weight-only: bf16 / fp32 outputs only
    assert gq(a_fmt=FP8, w_fmt=NVFP4) == UNSUP
    assert gq(n=40) == SHAPE
    assert gq(wbytes=100) == SMALL
    assert gq(ats=None) == INVALID                     # the GEMM's own operand checks
    assert gq(m=0) == OK and gq(n=0, ldy=0) == OK      # nothing to do

"""The quantizers code elements with gfx950's conversion instructions
(csrc/common.hpp: hw_e2m1x8, hw_e4m3x4). These tests run those exact device
functions on all 2^32 fp32 inputs and require them to equal the library's
integer encoders -- which tests/test_encoder_exhaustive.py ties to the CPU
oracle on the same 2^32 inputs. The GEMM's W4A4 dequantization relies on
v_cvt_scalef32_pk_f16_fp4 returning the exact E2M1 values at scale 1.0."""
import ctypes
import os

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

LIB = os.path.join(os.path.dirname(__file__), "native", "libqgprobe.so")


def _probe():
    if not os.path.exists(LIB):
        pytest.fail("tests/native/libqgprobe.so is not built (__graft_entry__.build())")
    return ctypes.CDLL(LIB)


@pytest.mark.parametrize("which,name", [(0, "e2m1"), (1, "e4m3")])
def test_hw_encoder_equals_integer_encoder_on_all_fp32(which, name):
    L = _probe()
    counts = torch.zeros(2, dtype=torch.int64, device="cuda")
    first = torch.zeros(16, dtype=torch.int32, device="cuda")
    assert L.qgp_probe_cvt(which, ctypes.c_void_p(counts.data_ptr()), ctypes.c_void_p(first.data_ptr())) == 0
    torch.cuda.synchronize()
    c = counts.cpu().tolist()
    f = first.cpu().numpy().view(np.uint32)
    print(name, "mismatches (all, finite):", c, [hex(v) for v in f[:8]], flush=True)
    assert c[1] == 0, "finite mismatches %d, e.g. inputs %s -> hw %s" % (c[1], [hex(v) for v in f[:4]], [hex(v) for v in f[8:12]])


def test_f16_conversion_of_e2m1_is_exact_at_unit_scale():
    L = _probe()
    out = torch.zeros(8192, dtype=torch.int16, device="cuda")
    assert L.qgp_probe_f16_scale(ctypes.c_void_p(out.data_ptr())) == 0
    torch.cuda.synchronize()
    o = out.cpu().numpy().view(np.float16).astype(np.float64).reshape(256, 16, 2)
    assert np.array_equal(o[:, :, 0], np.broadcast_to(oracle.e2m1_table(), (256, 16)))


def test_block_scale_decoders_on_every_code():
    """The E4M3 block-scale decoders the GEMM kernels use, on every code and
    in every byte position, against the oracle's E4M3 table: the hardware
    v_cvt_pk_f32_fp8 (W4A16 weight-pool and large-M kernels) on all 256 codes
    (the two NaN codes give NaN), and on the 128 non-negative codes (block
    scales are magnitudes) the bit-move decoder of the split-K W4A16 kernel
    (fp32; the E4M3 subnormal codes 1..7 pass through fp32 subnormals) and the
    hardware v_cvt_scalef32_pk_f16_fp8 at unit scale of the W4A4 kernels (fp16,
    four per dword)."""
    L = _probe()
    f32 = torch.full((1024,), 12345.0, dtype=torch.float32, device="cuda")
    ref = torch.full((1024,), 12345.0, dtype=torch.float32, device="cuda")
    h16 = torch.zeros(1024, dtype=torch.int16, device="cuda")
    assert L.qgp_probe_scale_decoders(ctypes.c_void_p(f32.data_ptr()), ctypes.c_void_p(ref.data_ptr()),
                                      ctypes.c_void_p(h16.data_ptr())) == 0
    torch.cuda.synchronize()
    table = oracle.e4m3_table()
    hw = f32.cpu().numpy().astype(np.float64).reshape(256, 4)
    want = np.broadcast_to(table[:, None], (256, 4))
    nan = np.isnan(want)
    assert nan.sum() == 8                                   # 0x7F and 0xFF in four positions
    assert np.array_equal(np.isnan(hw), nan)
    assert np.array_equal(hw[~nan], want[~nan])
    assert np.array_equal(np.signbit(hw[~nan]), np.signbit(want[~nan]))
    pos = table[:128]
    assert np.array_equal(ref.cpu().numpy().astype(np.float64).reshape(256, 4)[:127],
                          np.broadcast_to(pos[:127, None], (127, 4)))
    h = h16.cpu().numpy().view(np.float16).astype(np.float64)
    assert np.array_equal(h[:508].reshape(127, 4), np.broadcast_to(pos[:127, None], (127, 4)))
    assert (pos[1:8] < 2.0 ** -6).all()                     # the subnormal codes are among them

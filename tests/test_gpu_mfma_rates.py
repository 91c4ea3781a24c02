"""Matrix-instruction rates on the MI355X (test-only probe,
tests/native/mfma_probe.hip): the K = 16 FP8 instruction that an exact NVFP4
GEMM could issue once per 16-element block (v_mfma_f32_32x32x16_fp8_fp8),
the fp16 instruction the W4A4 kernels run on (v_mfma_f32_32x32x16_f16), and
the K = 64 fp8 and fp4 instructions. Each probe wave runs eight independent
accumulators on all-ones operands; the result must equal iters * K in every
element (checks the instruction's arithmetic), and the time gives the rate,
printed for the design notes (run with -s)."""
import ctypes
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

LIB = os.path.join(os.path.dirname(__file__), "native", "libqgprobe.so")
NAMES = {0: ("fp8 32x32x16", 16), 1: ("f16 32x32x16", 16), 2: ("fp8 32x32x64", 64), 3: ("fp4 32x32x64", 64)}


@pytest.mark.parametrize("waves_per_simd", [1, 4])
@pytest.mark.parametrize("which", [0, 1, 2, 3])
def test_mfma_rate(which, waves_per_simd):
    if not os.path.exists(LIB):
        pytest.fail("tests/native/libqgprobe.so is not built (__graft_entry__.build())")
    L = ctypes.CDLL(LIB)
    L.qgp_mfma_rate.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks, iters = cus * waves_per_simd, 4000 // waves_per_simd
    out = torch.zeros(blocks * 256, dtype=torch.float32, device="cuda")
    ms = ctypes.c_float(0.0)
    assert L.qgp_mfma_rate(which, ctypes.c_void_p(out.data_ptr()), blocks, iters, ctypes.byref(ms)) == 0
    torch.cuda.synchronize()
    name, k = NAMES[which]
    want = 8 * 16 * iters * k                  # 8 accumulators x 16 values, each iters * K
    assert np.all(out.cpu().numpy() == want), (name, out[:4].tolist(), want)
    flops = blocks * 4 * iters * 8 * 2.0 * 32 * 32 * k
    print("mfma rate %s, %d wave(s)/SIMD: %.2f PFLOP/s (%.3f ms)" % (name, waves_per_simd, flops / (ms.value * 1e12),
                                                                    ms.value), flush=True)

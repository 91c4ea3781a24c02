"""The Python binding refuses tensors in host memory before any library
call (the kernels would dereference their addresses on the GPU). Runs on the
CPU: every call below fails in the binding itself."""
import pytest
import torch

import paper_2609_21849_amd as q


def test_host_tensors_are_refused():
    x = torch.zeros((4, 32), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="CUDA"):
        q.quantize(x, q.QG_FMT_FP8_E4M3)
    w = torch.zeros(4096, dtype=torch.uint8)
    with pytest.raises(ValueError, match="CUDA"):
        q.linear(x, w, q.QG_FMT_NVFP4, 16)
    with pytest.raises(ValueError, match="CUDA"):
        q.unpack(w, q.QG_FMT_FP8_E4M3, 16, 128)
    qt = q.QTensor(q.QG_FMT_FP8_E4M3, torch.zeros((4, 32), dtype=torch.uint8), None, torch.ones(1), 4, 32)
    with pytest.raises(ValueError, match="CUDA"):
        q.pack(qt)
    with pytest.raises(ValueError, match="CUDA"):
        q.dequantize(qt)
    # the one-to-one wrappers refuse host tensors too (raw int pointers pass as given)
    with pytest.raises(ValueError, match="CUDA"):
        q.qg_gemm(q.QG_FMT_BF16, x, None, None, 32, q.QG_FMT_NVFP4, w, w.numel(), 4, 16, 32, x, 16,
                  q.QG_OUT_BF16, stream=0)


def test_non_tensor_quantized_operand_is_refused():
    with pytest.raises(ValueError, match="QTensor"):
        q.dequantize(object())

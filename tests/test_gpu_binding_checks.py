"""The allocating helpers check what the C ABI cannot see (element types and
shapes of caller-supplied tensors) and refuse a mismatch before any launch:
an fp32 output into a bf16 buffer would write past its end."""
import pytest
import torch

import paper_2609_21849_amd as q
import synth
from gpu_util import DEV, to_dev_bf16

pytestmark = pytest.mark.gpu


def test_mismatched_tensors_are_refused():
    x = to_dev_bf16(synth.normal_bf16(8, 256, 1.0, 5, 0))
    w = to_dev_bf16(synth.normal_bf16(32, 256, 0.02, 5, 1))
    packed = q.pack(q.quantize(w, q.QG_FMT_FP8_E4M3))
    a = q.quantize(x, q.QG_FMT_FP8_E4M3)
    with pytest.raises(ValueError, match="dtype"):
        q.linear(a, packed, q.QG_FMT_FP8_E4M3, 32, out_dtype=q.QG_OUT_F32,
                 y=torch.empty((8, 32), dtype=torch.bfloat16, device=DEV))
    with pytest.raises(ValueError, match="shape"):
        q.linear(a, packed, q.QG_FMT_FP8_E4M3, 32, y=torch.empty((8, 16), dtype=torch.bfloat16, device=DEV))
    with pytest.raises(ValueError, match="dtype"):
        q.linear(a, packed.view(torch.int32), q.QG_FMT_FP8_E4M3, 32)
    with pytest.raises(ValueError, match="shape"):
        q.dequantize(q.QTensor(a.fmt, a.codes[:, :128], None, a.tensor_scale, 8, 256))
    with pytest.raises(ValueError, match="dtype"):
        q.quantize(x.float(), q.QG_FMT_NVFP4)
    with pytest.raises(ValueError, match="dtype"):
        q.quantize(x, q.QG_FMT_FP8_E4M3, static_scale=torch.ones(1, dtype=torch.float64, device=DEV))
    # a correct call still works
    y = q.linear(a, packed, q.QG_FMT_FP8_E4M3, 32, out_dtype=q.QG_OUT_F32,
                 y=torch.empty((8, 32), dtype=torch.float32, device=DEV))
    torch.cuda.synchronize()
    assert torch.isfinite(y).all()

"""The library's quantizers (dynamic per-tensor FP8 and NVFP4, MXFP4 and
MXFP8) on the seeded workload-shaped tensors of tests/golden/quant_digests.py:
the SHA-256 of every output byte (codes, block scales, tensor-scale bits)
must equal the digest the oracle wrote, i.e. the outputs are bit-identical."""
import numpy as np
import pytest
import torch

import paper_2609_21849_amd as q
from golden import quant_digests as G
from gpu_util import host, log, to_dev_bf16

pytestmark = pytest.mark.gpu

FMT = {"fp8": q.QG_FMT_FP8_E4M3, "nvfp4": q.QG_FMT_NVFP4, "mxfp4": q.QG_FMT_MXFP4, "mxfp8": q.QG_FMT_MXFP8}


@pytest.mark.parametrize("name", list(G.CASES))
def test_library_matches_oracle_digest(name):
    log("golden digest %s" % name)
    fmt = G.CASES[name][0]
    qt = q.quantize(to_dev_bf16(G.make_input(name)), FMT[fmt])
    torch.cuda.synchronize()
    bs = host(qt.block_scales) if qt.block_scales is not None else None
    ts = np.float32(host(qt.tensor_scale)[0]) if qt.tensor_scale is not None else None
    assert G.digest(host(qt.codes), bs, ts) == G.load()["cases"][name]["sha256"]

"""SHA-256 digests of quantized tensors, as regression fixtures.

The cases are seeded synthetic bf16 tensors with the shapes of the paper's
workloads (the small FP8 check, the NVFP4 encoder-sized case, activations of
the denoising transformer with heavy-tailed channels) quantized to FP8 E4M3
(per-tensor scale), NVFP4 (E2M1 elements, E4M3 scale per 16, fp32 tensor
scale) and OCP MXFP4 / MXFP8 (E8M0 scale per 32). The quantization rules are
the format definitions the paper's recipe cites (Sec. 4, quantization
paragraph); the digest covers every output byte: codes, block scales and the
fp32 tensor-scale bits.

Running this file as a script rewrites `quant_digests.json` from the oracle
alone (`python tests/golden/quant_digests.py`). The tests import `CASES`,
`make_input` and `digest` from here: the CPU test recomputes the oracle's
digests, the GPU test digests the library's outputs for the same inputs.
"""
import hashlib
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402

JSON = os.path.join(HERE, "quant_digests.json")

# name: (format, rows, cols, sigma, seed, stream, heavy-tailed channels)
CASES = {
    "fp8_x_128x256": ("fp8", 128, 256, synth.SIGMA_X, 0, 0, False),
    "fp8_w_256x256": ("fp8", 256, 256, synth.SIGMA_W, 0, 1, False),
    "nvfp4_x_512x3072": ("nvfp4", 512, 3072, synth.SIGMA_X, 0, 0, False),
    "nvfp4_w_3072x3072": ("nvfp4", 3072, 3072, synth.SIGMA_W, 0, 1, False),
    "nvfp4_x_heavy_512x3072": ("nvfp4", 512, 3072, synth.SIGMA_X, 0, 0, True),
    "fp8_x_heavy_512x9216": ("fp8", 512, 9216, synth.SIGMA_X, 0, 0, True),
    "mxfp4_x_heavy_512x3072": ("mxfp4", 512, 3072, synth.SIGMA_X, 0, 0, True),
    "mxfp8_x_heavy_512x3072": ("mxfp8", 512, 3072, synth.SIGMA_X, 0, 0, True),
}


def make_input(name: str) -> np.ndarray:
    fmt, rows, cols, sigma, seed, stream, heavy = CASES[name]
    if heavy:
        return synth.normal_bf16(rows, cols, sigma, seed, stream, synth.HEAVY_TAIL_FRAC, synth.HEAVY_TAIL_GAIN)
    return synth.normal_bf16(rows, cols, sigma, seed, stream)


def digest(codes, block_scales, tensor_scale) -> str:
    """SHA-256 over the codes, then the block scales (if any), then the fp32
    tensor-scale bits (if any), each as little-endian bytes in row-major order."""
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(codes, dtype=np.uint8).tobytes())
    if block_scales is not None:
        h.update(np.ascontiguousarray(block_scales, dtype=np.uint8).tobytes())
    if tensor_scale is not None:
        h.update(np.array([tensor_scale], dtype="<f4").tobytes())
    return h.hexdigest()


def oracle_digest(name: str) -> str:
    import oracle
    fmt = CASES[name][0]
    x = make_input(name)
    if fmt == "fp8":
        codes, s = oracle.quantize_fp8(x)
        return digest(codes, None, s)
    if fmt == "nvfp4":
        codes, bs, s = oracle.quantize_nvfp4(x)
        return digest(codes, bs, s)
    codes, sc = oracle.quantize_mx(x, fmt)
    return digest(codes, sc, None)


def load() -> dict:
    with open(JSON) as f:
        return json.load(f)


if __name__ == "__main__":
    out = {"source": "written by tests/golden/quant_digests.py from the CPU oracle (oracle/qg_oracle.c)",
           "cases": {}}
    for name, (fmt, rows, cols, sigma, seed, stream, heavy) in CASES.items():
        out["cases"][name] = {"format": fmt, "rows": rows, "cols": cols, "sigma": sigma, "seed": seed,
                              "stream": stream, "heavy_tail": heavy, "sha256": oracle_digest(name)}
        print(name, out["cases"][name]["sha256"], flush=True)
    with open(JSON, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")

"""The library's E4M3/E2M1 encoders (the __host__ __device__ functions in
csrc/common.hpp that the quantize kernels run) against the CPU oracle's
encoders on every fp32 bit pattern. Host build only, no GPU; about a minute
on 8 cores."""
import os
import shutil
import subprocess

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.slow
def test_device_encoders_match_oracle_on_all_fp32(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    lib = oracle.build(force=False)
    exe = str(tmp_path / "enc_test")
    src = os.path.join(ROOT, "tests", "native", "encoder_exhaustive.cpp")
    subprocess.run([hipcc, "-x", "hip", "--offload-host-only", "-O2", "-fopenmp",
                    "-I" + os.path.join(ROOT, "paper_2609_21849_amd", "csrc"), src,
                    "-L" + os.path.dirname(lib), "-loracle", "-Wl,-rpath," + os.path.dirname(lib),
                    "-o", exe], check=True, capture_output=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=900)
    assert "e4m3_mismatches 0" in r.stdout and "e2m1_mismatches 0" in r.stdout, r.stdout
    assert r.returncode == 0

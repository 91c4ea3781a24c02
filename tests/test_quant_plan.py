"""Host-only check of the two-launch quantizer's launch plan (csrc/quant_plan.hpp,
the header the kernels and the launcher use): regions, slots and limits over
tens of thousands of tensor sizes. No GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_slot_plan_invariants(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "quant_plan_check")
    subprocess.run([hipcc, "-x", "hip", "--offload-host-only", "-O2", "-std=c++20",
                    "-I" + os.path.join(ROOT, "paper_2609_21849_amd", "csrc"),
                    os.path.join(ROOT, "tests", "native", "quant_plan_check.cpp"), "-o", exe],
                   check=True, capture_output=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "violations 0" in r.stdout, r.stdout
    planned = int(r.stdout.split("planned ")[1].split()[0])
    assert planned > 10000, r.stdout

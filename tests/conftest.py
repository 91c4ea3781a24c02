import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_sessionfinish(session, exitstatus):
    """With QG_PARITY_LOG set, write the parity margins the GPU tests
    recorded (max err / sum|a w| per workload case) to that file: a markdown
    table if its name ends in .md, JSON otherwise."""
    path = os.environ.get("QG_PARITY_LOG")
    if not path:
        return
    mod = sys.modules.get("gpu_util")
    if mod is None or not getattr(mod, "MARGINS", None):
        return
    import json
    os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
    with open(path, "w") as f:
        if not path.endswith(".md"):
            json.dump(mod.MARGINS, f, indent=1, sort_keys=True)
            return
        f.write("# GEMM parity margins against the oracle\n\n"
                "Written by the GPU parity tests (`QG_PARITY_LOG=<this file> python -m pytest tests -m gpu`).\n"
                "Bound: |y - y_ref| <= 1e-3 sum_k |a w| over the oracle's exact (fp64) product of the same\n"
                "quantized operands. Last column: outputs where the bf16 rounding of the exact product alone\n"
                "exceeds the bound (those are held to the rounding window instead).\n\n"
                "| case | output | outputs checked | max err / sum abs(a w) | bf16-unreachable outputs |\n"
                "|---|---|---:|---:|---:|\n")
        for name, v in sorted(mod.MARGINS.items()):
            f.write("| %s | %s | %d | %.3e | %d |\n" % (name, v["dtype"], v["outputs_checked"],
                                                    v["max_err_over_sum_abs_aw"],
                                                    v.get("outputs_where_bf16_rounding_alone_exceeds_bound", 0)))

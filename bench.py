"""Benchmark of the quantized-linear hot path on one MI355X.

One step = one pass of the whole path over one batch of seeded synthetic
input shaped like the paper's workloads:
  * denoising-transformer block linears at a 1024^2 image (M = 4608 tokens,
    hidden 3072): QKV 3072->9216, attention-out 3072->3072, MLP-up
    3072->9216, MLP-down 9216->3072, each = run-time activation quantize +
    quantized GEMM, once in FP8 W8A8 and once in NVFP4 W4A4 (the NVFP4 pass
    uses heavy-tailed activations: 0.1 % of input channels x50);
  * the small text encoder's linears 1024->3072 and 3072->1024 with NVFP4
    weights and bf16 activations (W4A16) at M = 1, 16, 256, 512 tokens.
Weights are quantized and packed once before timing (offline PTQ). Inputs
are resident in HBM when the timed region starts.

Prints one JSON line with the aggregate quantized
GEMM throughput of the step, a per-part breakdown, a roofline entry for the
dominant kernel (per-launch HIP events on the launch stream) and the CPU
oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "quantized GEMM TFLOP/s (FP8, NVFP4) at DiT shapes + % MFMA peak; W4A16 HBM GB/s"
PEAK = {"fp8": 5000.0, "f16": 2500.0, "bf16": 2500.0, "fp4": 10100.0, "hbm_gbs": 8000.0}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU work for the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pool-mib", type=int, default=600,
                    help="size of the weight pool for the cold-HBM W4A16 measurement")
    ap.add_argument("--traffic-probe", nargs="?", const="nvfp4", choices=("nvfp4", "fp8", "mxfp4", "mxfp8"),
                    help="only launch the DiT GEMMs of one format (3x per shape) and a calibration copy; "
                         "for rocprofv3 --pmc runs")
    ap.add_argument("--traffic-summary", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "OUT_MD"),
                    help="turn the two counter runs of --traffic-probe into the traffic summary")
    ap.add_argument("--mfma-summary", nargs=2, metavar=("PMC_DIR", "OUT_MD"),
                    help="turn a MfmaUtil counter run of --traffic-probe into the MFMA-utilisation summary")
    ap.add_argument("--stall-summary", nargs=2, metavar=("PMC_DIRS", "OUT_MD"),
                    help="turn the counter passes STALL_PASSES over --traffic-probe (directories comma-separated) "
                         "into the wave-time summary")
    ap.add_argument("--quant-probe", action="store_true",
                    help="only the dynamic activation quantizers (FP8 and NVFP4, 4608 x 3072 and 4608 x 9216, "
                         "3x each) and a calibration copy; for rocprofv3 runs")
    ap.add_argument("--quant-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "TRACE_DIR", "OUT_MD"),
                    help="turn two counter runs and a kernel trace of --quant-probe into the quantizer summary")
    ap.add_argument("--kind", choices=("nvfp4", "fp8", "mxfp4", "mxfp8"), default="nvfp4",
                    help="format of the --traffic-summary / --mfma-summary counter runs")
    ap.add_argument("--w4a16-pool-only", action="store_true",
                    help="only the cold-HBM W4A16 pool measurement (one JSON line); for rocprofv3 runs")
    return ap.parse_args()


# HBM traffic of the dominant kernel, measured with rocprofv3 counters (see
# --traffic-probe / --traffic-summary) and kept as a text summary; reported
# only while the kernel source is the one the counters were taken on.
TRAFFIC_MD = {"nvfp4": os.path.join(ROOT, "profiles", "k_gemm_nvfp4_direct_dit_traffic.md"),
              "fp8": os.path.join(ROOT, "profiles", "k_gemm_fp8_t288_dit_traffic.md")}
KERNEL = {"nvfp4": "k_gemm_nvfp4_direct", "fp8": "k_gemm_fp8_t288", "mxfp4": "k_gemm_mxfp4_direct",
          "mxfp8": "k_gemm_mxfp8_direct"}
# executed-MFMA counter per format (none is known to count the fp4 operand
# instructions, so the MXFP4 summary has MfmaUtil and the clock only)
FLOPS_CTR = {"nvfp4": "MfmaFlopsF16", "fp8": "SQ_INSTS_VALU_MFMA_MOPS_F8", "mxfp8": "SQ_INSTS_VALU_MFMA_MOPS_F8",
             "mxfp4": None}
# counter passes of --stall-summary (each within one pass's per-block counter limits)
STALL_PASSES = (
    "SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_VALU_MFMA_BUSY_CYCLES "
    "SQ_VALU_MFMA_COEXEC_CYCLES SQ_INSTS_VALU SQ_INSTS_MFMA GRBM_GUI_ACTIVE",
    "SQ_ACTIVE_INST_LDS SQ_ACTIVE_INST_VMEM SQ_WAIT_INST_LDS SQ_LDS_BANK_CONFLICT SQ_INSTS_LDS SQ_ACTIVE_INST_SCA "
    "TA_BUSY_avr TA_DATA_STALLED_BY_TC_CYCLES",
    "TCP_TCC_READ_REQ_LATENCY_sum TCP_TCC_READ_REQ_sum TCP_PENDING_STALL_CYCLES_sum TCP_TCR_TCP_STALL_CYCLES_sum "
    "TCC_HIT_sum TCC_MISS_sum")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_21849_amd", "csrc", "gemm.hip")
COPY_BYTES = 512 * 2 ** 20


def source_sha() -> str:
    import hashlib
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def gemm_bytes(kind, m, n, k):
    """Algorithmic bytes of one DiT GEMM: A codes (+ block scales), packed W
    codes (+ scales), bf16 Y."""
    per = {"nvfp4": 0.5 + 1 / 16, "fp8": 1.0, "mxfp4": 0.5 + 1 / 32, "mxfp8": 1.0 + 1 / 32}[kind]
    return m * k * per + n * k * per + 2 * m * n


def traffic_probe(kind):
    import torch
    import paper_2609_21849_amd as q
    import synth
    torch.cuda.set_device(0)
    M = synth.DIT_TOKENS
    fmt = {"nvfp4": q.QG_FMT_NVFP4, "fp8": q.QG_FMT_FP8_E4M3, "mxfp4": q.QG_FMT_MXFP4, "mxfp8": q.QG_FMT_MXFP8}[kind]
    runs = []
    for li, (name, (n, k)) in enumerate(synth.DIT_LINEARS.items()):
        base = 16 * li
        # 4-bit formats: the heavy-tailed activations of the step; 8-bit: N(0, 1)
        x = synth.normal_bf16(M, k, synth.SIGMA_X, 0, base + synth.STREAM_X,
                              outlier_frac=synth.HEAVY_TAIL_FRAC if kind in ("nvfp4", "mxfp4") else 0.0,
                              outlier_gain=synth.HEAVY_TAIL_GAIN, outlier_stream=base + synth.STREAM_OUTLIER)
        w = synth.normal_bf16(n, k, synth.SIGMA_W, 0, base + synth.STREAM_W)
        a = q.quantize(dev_bf16(x), fmt)
        p = q.pack(q.quantize(dev_bf16(w), fmt))
        y = torch.empty((M, n), dtype=torch.bfloat16, device="cuda")
        runs.append((a, p, y, n))
    torch.cuda.synchronize()
    for a, p, y, n in runs:
        for _ in range(3):
            q.linear(a, p, fmt, n, y=y)
    torch.cuda.synchronize()
    src = torch.ones(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print("traffic probe done", flush=True)


QUANT_SHAPES = ((4608, 3072), (4608, 9216))   # the transformer linears' two activation sizes
QUANT_KERNELS = ("k_amax_dense", "k_finalize", "k_quant_dense")


def quant_probe():
    """The dynamic quantizers of the step's activations: FP8 (N(0,1)) and
    NVFP4 (heavy-tailed), each size three times, then the calibration copy."""
    import torch
    import paper_2609_21849_amd as q
    import synth
    torch.cuda.set_device(0)
    for fmt, tail in ((q.QG_FMT_FP8_E4M3, 0.0), (q.QG_FMT_NVFP4, synth.HEAVY_TAIL_FRAC)):
        for (m, k) in QUANT_SHAPES:
            x = dev_bf16(synth.normal_bf16(m, k, synth.SIGMA_X, 0, synth.STREAM_X, outlier_frac=tail,
                                           outlier_gain=synth.HEAVY_TAIL_GAIN, outlier_stream=synth.STREAM_OUTLIER))
            qt = q.quantize(x, fmt)
            torch.cuda.synchronize()
            for _ in range(3):
                q.qg_quantize_act(fmt, x, m, k, k, qt.codes, qt.block_scales, qt.tensor_scale)
            torch.cuda.synchronize()
    src = torch.ones(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print("quant probe done", flush=True)


def quant_summary(fetch_dir, write_dir, trace_dir, out_md):
    """HBM bytes and rates of the three quantizer kernels at the step's
    activation sizes: FETCH_SIZE / WRITE_SIZE per dispatch (copy-calibrated
    as for the GEMMs) and durations from a kernel trace of the same probe;
    the rate is the algorithmic bytes over the kernel's duration."""
    import csv
    import glob
    rows = {}
    for ctr, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rs = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            rs += [r for r in csv.DictReader(open(f)) if r["Counter_Name"] == ctr]
        rs.sort(key=lambda r: int(r.get("Dispatch_Id", 0)))
        rows[ctr] = rs
    tr = []
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        tr += list(csv.DictReader(open(f)))
    tr.sort(key=lambda t: int(t["Start_Timestamp"]))

    def seq(items, name_of):
        out = {kname: [] for kname in QUANT_KERNELS}
        copy = []
        for it in items:
            n = name_of(it)
            for kname in QUANT_KERNELS:
                if kname + "(" in n or kname + "<" in n:
                    out[kname].append(it)
            if "copyBuffer" in n or "copy_kernel" in n:
                copy.append(it)
        return out, copy
    fk, fc = seq(rows["FETCH_SIZE"], lambda r: r["Kernel_Name"])
    wk, wc = seq(rows["WRITE_SIZE"], lambda r: r["Kernel_Name"])
    tk, _ = seq(tr, lambda t: t["Kernel_Name"])
    ncalls = 2 * len(QUANT_SHAPES) * 3
    # q.quantize() before each size's three timed calls adds one call per size
    per_size = 4
    for kname in QUANT_KERNELS:
        assert len(fk[kname]) == len(wk[kname]) == len(tk[kname]) == 2 * len(QUANT_SHAPES) * per_size, \
            (kname, len(fk[kname]), len(wk[kname]), len(tk[kname]), ncalls)
    f_factor = sum(float(r["Counter_Value"]) for r in fc) / len(fc) * 1024 / COPY_BYTES
    w_factor = sum(float(r["Counter_Value"]) for r in wc) / len(wc) * 1024 / COPY_BYTES
    lines = ["# The dynamic activation quantizers at the transformer activation sizes", "",
             "The three kernels of a dynamic per-tensor quantization of a 4608 x 3072 and a 4608 x 9216 bf16 "
             "activation (FP8: N(0,1); NVFP4: heavy-tailed), each call three times after one warm-up call: HBM "
             "bytes per dispatch from FETCH_SIZE and WRITE_SIZE (each scaled by what it reads for a %d MiB "
             "device-to-device copy: fetch factor %.4f, write factor %.4f), kernel durations from a kernel "
             "trace of the same probe (mean of the three timed calls). Algorithmic bytes: amax reads the "
             "activation (2 bytes per element); finalize reads the partial maxima; quantize reads the activation "
             "and writes the codes (FP8 1 byte per element, NVFP4 0.5 plus 1/16 of block scales). The rate is "
             "algorithmic bytes over duration, against the 8 TB/s HBM peak." % (COPY_BYTES >> 20, f_factor, w_factor),
             "", "Commands (repo root, MI355X; $OUT any output directory):", "", "```",
             "cd /tmp && export TMPDIR=/tmp; cd $REPO && timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE "
             "--output-format csv -d $OUT/pmc_fetch_quant -o run -- python3 bench.py --quant-probe",
             "cd /tmp && export TMPDIR=/tmp; cd $REPO && timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE "
             "--output-format csv -d $OUT/pmc_write_quant -o run -- python3 bench.py --quant-probe",
             "cd /tmp && export TMPDIR=/tmp; cd $REPO && timeout -s KILL 120 rocprofv3 --kernel-trace "
             "--output-format csv -d $OUT/trace_quant -o run -- python3 bench.py --quant-probe",
             "python3 bench.py --quant-summary $OUT/pmc_fetch_quant $OUT/pmc_write_quant $OUT/trace_quant <this file>",
             "```", "",
             "| format | activation | kernel | fetch MB | write MB | algorithmic MB | duration us | GB/s | of 8 TB/s |",
             "|---|---|---|---:|---:|---:|---:|---:|---:|"]
    i = 0
    for fname in ("FP8", "NVFP4"):
        for (m, k) in QUANT_SHAPES:
            n = m * k
            alg = {"k_amax_dense": 2.0 * n, "k_finalize": 4096.0,
                   "k_quant_dense": 2.0 * n + (n if fname == "FP8" else n / 2 + n / 16)}
            for kname in QUANT_KERNELS:
                sl = slice(per_size * i + 1, per_size * i + per_size)   # the three timed calls
                fb = sum(float(r["Counter_Value"]) for r in fk[kname][sl]) / 3 * 1024 / f_factor
                wb = sum(float(r["Counter_Value"]) for r in wk[kname][sl]) / 3 * 1024 / w_factor
                us = sum(int(t["End_Timestamp"]) - int(t["Start_Timestamp"]) for t in tk[kname][sl]) / 3 / 1e3
                gbs = alg[kname] / (us * 1e3)
                lines.append("| %s | %d x %d | `%s` | %.1f | %.1f | %.1f | %.2f | %.0f | %.3f |"
                             % (fname, m, k, kname, fb / 1e6, wb / 1e6, alg[kname] / 1e6, us, gbs, gbs / PEAK["hbm_gbs"]))
            i += 1
    lines += ["", "Source: paper_2609_21849_amd/csrc/quantize.hip.", ""]
    with open(out_md, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def read_counter(d, counter, kernel):
    """Per-dispatch values of a counter for `kernel` and for the calibration
    copy, from rocprofv3 --output-format csv runs under directory d."""
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        rows += [r for r in csv.DictReader(open(f)) if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r.get("Dispatch_Id", 0)))
    gemm = [float(r["Counter_Value"]) for r in rows if kernel in r["Kernel_Name"]]
    copy = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]
            or "copy_kernel" in r["Kernel_Name"]]
    return gemm, copy


def mfma_summary(pmc_dir, out_md, kind):
    """MfmaUtil, executed MFMA work and GRBM_GUI_ACTIVE of the DiT GEMMs of
    one format, from one `rocprofv3 --pmc MfmaUtil <flops> GRBM_GUI_ACTIVE`
    run over --traffic-probe."""
    import synth
    kern = KERNEL[kind]
    flops_ctr = FLOPS_CTR[kind]
    util, _ = read_counter(pmc_dir, "MfmaUtil", kern)
    gui, _ = read_counter(pmc_dir, "GRBM_GUI_ACTIVE", kern)
    fl, _ = read_counter(pmc_dir, flops_ctr, kern) if flops_ctr else ([float("nan")] * len(util), None)
    if flops_ctr == "SQ_INSTS_VALU_MFMA_MOPS_F8":
        fl = [v * 512 for v in fl]
    assert len(util) == len(fl) == len(gui) == 12, (len(util), len(fl), len(gui))
    M = synth.DIT_TOKENS
    lines = ["# MFMA utilisation of `%s` at the transformer shapes (M = %d)" % (kern, M), "",
             "rocprofv3 counters over `bench.py --traffic-probe %s` (each of the four DiT-shaped %s GEMMs launched "
             "three times): `MfmaUtil` (SQ_VALU_MFMA_BUSY_CYCLES over the SIMDs / (GRBM_GUI_ACTIVE x SIMD count) x "
             "100), executed MFMA flops (%s) and GRBM_GUI_ACTIVE (summed over the 8 XCDs)."
             % (kind, kind.upper(), (flops_ctr + (" x 512" if flops_ctr == "SQ_INSTS_VALU_MFMA_MOPS_F8" else ""))
                if flops_ctr else "no counter of this rocprofv3 counts the fp4-operand instructions: nan"), "",
             "Command (repo root, MI355X; $OUT any output directory):", "", "```",
             "cd /tmp && export TMPDIR=/tmp; cd $REPO && timeout -s KILL 120 rocprofv3 --pmc MfmaUtil %s"
             "GRBM_GUI_ACTIVE --output-format csv -d $OUT/pmc_mfma_%s -o run -- python3 bench.py "
             "--traffic-probe %s" % (flops_ctr + " " if flops_ctr else "", kind, kind),
             "python3 bench.py --mfma-summary $OUT/pmc_mfma_%s <this file> --kind %s" % (kind, kind), "```", "",
             "| linear (M x N x K) | launch | MfmaUtil % | MFMA flops / 2MNK | GUI-active cycles / 8 |",
             "|---|---:|---:|---:|---:|"]
    for i, (name, (n, k)) in enumerate(synth.DIT_LINEARS.items()):
        for j in range(3):
            t = 3 * i + j
            lines.append("| %s (%dx%dx%d) | %d | %.1f | %.4f | %.0f |" % (name, M, n, k, j + 1, util[t],
                                                                        fl[t] / (2.0 * M * n * k), gui[t] / 8))
    lines += ["", "Source: paper_2609_21849_amd/csrc/gemm.hip, SHA-256 prefix %s." % source_sha(), ""]
    with open(out_md, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def traffic_summary(fetch_dir, write_dir, out_md, kind="nvfp4"):
    import synth

    kern = KERNEL[kind]
    fg, fc = read_counter(fetch_dir, "FETCH_SIZE", kern)
    wg, wc = read_counter(write_dir, "WRITE_SIZE", kern)
    assert len(fg) == len(wg) == 12 and fc and wc, (len(fg), len(wg), len(fc), len(wc))
    f_factor = (sum(fc) / len(fc)) * 1024 / COPY_BYTES   # counter KiB per true byte, x1024
    w_factor = (sum(wc) / len(wc)) * 1024 / COPY_BYTES
    M = synth.DIT_TOKENS
    shapes = list(synth.DIT_LINEARS.items())
    per = []
    for i, (name, (n, k)) in enumerate(shapes):
        fb = sum(fg[3 * i:3 * i + 3]) / 3 * 1024 / f_factor
        wb = sum(wg[3 * i:3 * i + 3]) / 3 * 1024 / w_factor
        per.append({"linear": name, "m": M, "n": n, "k": k, "fetch_bytes": round(fb), "write_bytes": round(wb),
                    "algorithmic_bytes": round(gemm_bytes(kind, M, n, k))})
    t = sum(p["fetch_bytes"] + p["write_bytes"] for p in per) / len(per)
    alg = sum(p["algorithmic_bytes"] for p in per) / len(per)
    data = {"kernel": kern, "source": "paper_2609_21849_amd/csrc/gemm.hip",
            "source_sha": source_sha(), "traffic_bytes_per_launch": round(t),
            "algorithmic_bytes_per_launch": round(alg), "ratio": round(t / alg, 3),
            "copy_calibration": {"bytes": COPY_BYTES, "fetch_kib": sum(fc) / len(fc), "write_kib": sum(wc) / len(wc),
                                 "fetch_factor": round(f_factor, 4), "write_factor": round(w_factor, 4)},
            "per_shape": per}
    lines = ["# HBM traffic of %s at the DiT shapes (M = %d)" % (kern, M), "",
             "Commands (repo root, MI355X; $OUT any output directory):", "",
             "```",
             "rocprofv3 --pmc FETCH_SIZE --output-format csv -d $OUT/pmc_fetch_%s -o run -- python3 bench.py "
             "--traffic-probe %s" % (kind, kind),
             "rocprofv3 --pmc WRITE_SIZE --output-format csv -d $OUT/pmc_write_%s -o run -- python3 bench.py "
             "--traffic-probe %s" % (kind, kind),
             "python3 bench.py --traffic-summary $OUT/pmc_fetch_%s $OUT/pmc_write_%s <this file> --kind %s"
             % (kind, kind, kind),
             "```", "",
             "Each counter is scaled by what it reads for a %d MiB device-to-device copy (%d MiB read, %d MiB "
             "written): fetch factor %.4f, write factor %.4f (counter KiB x 1024 / true bytes)."
             % (COPY_BYTES >> 20, COPY_BYTES >> 20, COPY_BYTES >> 20, f_factor, w_factor), "",
             "| linear | N | K | fetch MB | write MB | algorithmic MB |", "|---|---|---|---|---|---|"]
    for p in per:
        lines.append("| %s | %d | %d | %.1f | %.1f | %.1f |" % (p["linear"], p["n"], p["k"], p["fetch_bytes"] / 1e6,
                                                              p["write_bytes"] / 1e6, p["algorithmic_bytes"] / 1e6))
    lines += ["", "Per launch (mean of the four shapes): %.1f MB measured vs %.1f MB algorithmic (ratio %.3f)."
              % (t / 1e6, alg / 1e6, t / alg), "", "```json", json.dumps(data, indent=1), "```", ""]
    with open(out_md, "w") as f:
        f.write("\n".join(lines))
    print(json.dumps(data))


def stall_summary(pmc_dirs, out_md, kind):
    """Where a DiT GEMM kernel's waves spend their time, from the counter
    passes STALL_PASSES over --traffic-probe (one rocprofv3 run per pass, in
    the directories pmc_dirs, comma-separated): per shape, the mean over the
    second and third launch."""
    import csv
    import glob
    import synth
    kern = KERNEL[kind]
    per = {}   # dispatch -> {counter: value, "ns": duration}
    for d in pmc_dirs.split(","):
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if kern not in r["Kernel_Name"]:
                    continue
                key = (d, int(r["Dispatch_Id"]))
                e = per.setdefault(key, {})
                e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
                e["ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    by_dir = {}
    for (d, disp), e in sorted(per.items()):
        by_dir.setdefault(d, []).append(e)
    shapes = list(synth.DIT_LINEARS.items())
    M = synth.DIT_TOKENS
    rows = []
    for i, (name, (n, k)) in enumerate(shapes):
        v, ns = {}, []
        for d, launches in by_dir.items():
            assert len(launches) == 12, (d, len(launches))
            for e in launches[3 * i + 1:3 * i + 3]:
                ns.append(e["ns"])
                for c, x in e.items():
                    if c != "ns":
                        v.setdefault(c, []).append(x)
        v = {c: sum(x) / len(x) for c, x in v.items()}
        wave = 4.0 * v["SQ_WAVE_CYCLES"]          # wave-cycles (the counter counts quad-cycles)
        rows.append((name, n, k, {
            "clock_ghz": v["GRBM_GUI_ACTIVE"] / 8 / (sum(ns) / len(ns)),
            "mfma_busy_of_wave": v["SQ_VALU_MFMA_BUSY_CYCLES"] / wave,
            "coexec_of_mfma": v["SQ_VALU_MFMA_COEXEC_CYCLES"] / v["SQ_VALU_MFMA_BUSY_CYCLES"],
            "wait_any_of_wave": v["SQ_WAIT_ANY"] / v["SQ_WAVE_CYCLES"],
            "wait_issue_of_wave": v["SQ_WAIT_INST_ANY"] / v["SQ_WAVE_CYCLES"],
            "wait_lds_of_wave": v["SQ_WAIT_INST_LDS"] / v["SQ_WAVE_CYCLES"],
            "valu_per_mfma": (v["SQ_INSTS_VALU"] - v["SQ_INSTS_MFMA"]) / v["SQ_INSTS_MFMA"],
            "lds_conflict_per_lds_inst": v["SQ_LDS_BANK_CONFLICT"] / v["SQ_INSTS_LDS"],
            "l2_hit": v["TCC_HIT_sum"] / (v["TCC_HIT_sum"] + v["TCC_MISS_sum"]),
            "l2_read_latency_cycles": v["TCP_TCC_READ_REQ_LATENCY_sum"] / v["TCP_TCC_READ_REQ_sum"],
            "wave_life_of_kernel": wave / (v["GRBM_GUI_ACTIVE"] / 8) / (4 * 256)}))
    cmds = ["cd /tmp && export TMPDIR=/tmp; cd $REPO && timeout -s KILL 120 rocprofv3 --pmc %s --output-format csv "
            "-d $OUT/pmc_stall_%s_%d -o run -- python3 bench.py --traffic-probe %s" % (p, kind, j + 1, kind)
            for j, p in enumerate(STALL_PASSES)]
    cmds.append("python3 bench.py --stall-summary %s <this file> --kind %s"
                % (",".join("$OUT/pmc_stall_%s_%d" % (kind, j + 1) for j in range(len(STALL_PASSES))), kind))
    cols = [("clock_ghz", "clock (GHz)", "%.2f"), ("wave_life_of_kernel", "wave life / kernel", "%.2f"),
            ("mfma_busy_of_wave", "MFMA busy / wave life", "%.2f"), ("coexec_of_mfma", "VALU co-issue / MFMA busy", "%.2f"),
            ("wait_any_of_wave", "waiting (waitcnt, barrier) / wave life", "%.2f"),
            ("wait_issue_of_wave", "waiting to issue / wave life", "%.2f"),
            ("wait_lds_of_wave", "waiting to issue LDS / wave life", "%.3f"),
            ("valu_per_mfma", "VALU instr. per MFMA", "%.2f"),
            ("lds_conflict_per_lds_inst", "LDS bank-conflict cycles per LDS instr.", "%.2f"),
            ("l2_hit", "L2 hit rate", "%.3f"), ("l2_read_latency_cycles", "L1->L2 read latency (cycles)", "%.0f")]
    lines = ["# Where the waves of `%s` spend their time (transformer shapes, M = %d)" % (kern, M), "",
             "rocprofv3 counters over `bench.py --traffic-probe %s` (each DiT-shaped GEMM launched three times; "
             "the mean of launches 2 and 3 per shape), %d counter passes. Ratios: wave-cycles = 4 x "
             "SQ_WAVE_CYCLES (quad-cycles), matrix-pipe busy = SQ_VALU_MFMA_BUSY_CYCLES (one wave per SIMD, so "
             "per wave), waiting = SQ_WAIT_ANY and SQ_WAIT_INST_ANY (quad-cycles) over SQ_WAVE_CYCLES, VALU "
             "instructions per MFMA = (SQ_INSTS_VALU - SQ_INSTS_MFMA) / SQ_INSTS_MFMA, clock = GRBM_GUI_ACTIVE "
             "per XCD over the dispatch's duration, wave life / kernel = wave-cycles over (1024 waves x "
             "GUI-active cycles per XCD)." % (kind, len(STALL_PASSES)), "",
             "Commands (repo root, MI355X; $OUT any output directory):", "", "```"] + cmds + ["```", "",
             "| linear (M x N x K) | " + " | ".join(c[1] for c in cols) + " |",
             "|---|" + "---:|" * len(cols)]
    for name, n, k, d in rows:
        lines.append("| %s (%dx%dx%d) | " % (name, M, n, k) + " | ".join(f % d[c] for c, _, f in cols) + " |")
    lines += ["", "Source: paper_2609_21849_amd/csrc/gemm.hip, SHA-256 prefix %s." % source_sha(), ""]
    with open(out_md, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def recorded_traffic(kind):
    """(bytes per launch, summary) of the committed traffic summary of the
    `kind` DiT GEMM, or (None, reason) when it is missing or was taken on
    another kernel source."""
    try:
        txt = open(TRAFFIC_MD[kind]).read()
        blob = json.loads(txt.split("```json", 1)[1].split("```", 1)[0])
    except (OSError, IndexError, ValueError):
        return None, "no traffic summary"
    if blob.get("source_sha") != source_sha():
        return None, "kernel source changed since the counters were taken"
    return blob["traffic_bytes_per_launch"], blob


def dev_bf16(bits):
    import torch
    return torch.from_numpy(np.array(bits, dtype=np.uint16, copy=True).view(np.int16)).view(torch.bfloat16).cuda()


def main():
    args = parse()
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary, kind=args.kind)
        return
    if args.mfma_summary:
        mfma_summary(*args.mfma_summary, kind=args.kind)
        return
    if args.stall_summary:
        stall_summary(*args.stall_summary, kind=args.kind)
        return
    if args.quant_summary:
        quant_summary(*args.quant_summary)
        return
    if args.quant_probe:
        quant_probe()
        return
    if args.traffic_probe:
        traffic_probe(args.traffic_probe)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(column/token sharding is a design note only); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_21849_amd as q
    import synth

    q.lib()  # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    if args.w4a16_pool_only:
        print(json.dumps({"w4a16_cold_pool": w4a16_pool(q, synth, args.pool_mib)}), flush=True)
        return
    t_setup = time.time()

    # ------------------------------------------------------------ inputs and offline weights
    M = synth.DIT_TOKENS
    dit = []
    for li, (name, (n, k)) in enumerate(synth.DIT_LINEARS.items()):
        base = 16 * li
        xn = synth.normal_f64(0, base + synth.STREAM_X, M * k).reshape(M, k)
        x_fp8 = synth.f32_to_bf16_bits((xn * synth.SIGMA_X).astype(np.float32))
        ch = synth.outlier_channels(0, base + synth.STREAM_OUTLIER, k, synth.HEAVY_TAIL_FRAC)
        xn[:, ch] *= synth.HEAVY_TAIL_GAIN
        x_nv = synth.f32_to_bf16_bits((xn * synth.SIGMA_X).astype(np.float32))
        del xn
        w = synth.normal_bf16(n, k, synth.SIGMA_W, 0, base + synth.STREAM_W)
        wd = dev_bf16(w)
        ent = {"name": name, "n": n, "k": k, "x": {"fp8": dev_bf16(x_fp8), "nvfp4": dev_bf16(x_nv)}}
        for kind, fmt in (("fp8", q.QG_FMT_FP8_E4M3), ("nvfp4", q.QG_FMT_NVFP4)):
            ent["w_" + kind] = q.pack(q.quantize(wd, fmt))
            # activation code buffers and output, allocated once
            if fmt == q.QG_FMT_FP8_E4M3:
                codes, bs = torch.empty((M, k), dtype=torch.uint8, device="cuda"), None
            else:
                codes = torch.empty((M, k // 2), dtype=torch.uint8, device="cuda")
                bs = torch.empty((M, k // 16), dtype=torch.uint8, device="cuda")
            ent["a_" + kind] = q.QTensor(fmt, codes, bs, torch.empty(1, device="cuda"), M, k)
            ent["y_" + kind] = torch.empty((M, n), dtype=torch.bfloat16, device="cuda")
        ent["w_bf16"] = wd  # for the BF16 baseline of the block chain
        ent["w_mxfp4"] = q.pack(q.quantize(wd, q.QG_FMT_MXFP4))  # the hardware-native block-scaled formats
        ent["w_mxfp8"] = q.pack(q.quantize(wd, q.QG_FMT_MXFP8))
        dit.append(ent)
    enc = []
    for ei, (name, (n, k)) in enumerate(synth.ENCODER_LINEARS.items()):
        base = 64 + 16 * ei
        w = synth.normal_bf16(n, k, synth.SIGMA_W, 0, base + synth.STREAM_W)
        packed = q.pack(q.quantize(dev_bf16(w), q.QG_FMT_NVFP4))
        packed8 = q.pack(q.quantize(dev_bf16(w), q.QG_FMT_FP8_E4M3))
        for m in synth.ENCODER_TOKENS:
            x = dev_bf16(synth.normal_bf16(m, k, synth.SIGMA_X, 0, base + synth.STREAM_X + 100 * m))
            enc.append({"name": name, "n": n, "k": k, "m": m, "x": x, "w": packed, "w8": packed8,
                        "y": torch.empty((m, n), dtype=torch.bfloat16, device="cuda")})
    torch.cuda.synchronize()
    t_setup = time.time() - t_setup

    # ------------------------------------------------------------ the step as a flat launch list
    # (integer pointers keep per-launch host overhead small; the stream handle
    # is appended at launch time, so that the list can also be captured)
    lib = q.lib()
    st = torch.cuda.current_stream().cuda_stream
    plan = []
    for kind, fmt in (("fp8", q.QG_FMT_FP8_E4M3), ("nvfp4", q.QG_FMT_NVFP4)):
        for e in dit:
            a, x, wp, y = e["a_" + kind], e["x"][kind], e["w_" + kind], e["y_" + kind]
            bs = a.block_scales.data_ptr() if a.block_scales is not None else None
            plan.append((("quant", kind, e["name"]), lib.qg_quantize_act,
                         (fmt, x.data_ptr(), M, e["k"], e["k"], a.codes.data_ptr(), bs,
                          a.tensor_scale.data_ptr())))
            plan.append((("gemm", kind, e["name"]), lib.qg_gemm,
                         (fmt, a.codes.data_ptr(), bs, a.tensor_scale.data_ptr(), e["k"], fmt,
                          wp.data_ptr(), wp.numel(), M, e["n"], e["k"], y.data_ptr(), e["n"],
                          q.QG_OUT_BF16)))
    for e in enc:
        plan.append((("gemm", "w4a16", "%s_m%d" % (e["name"], e["m"])), lib.qg_gemm,
                     (q.QG_FMT_BF16, e["x"].data_ptr(), None, None, e["k"], q.QG_FMT_NVFP4,
                      e["w"].data_ptr(), e["w"].numel(), e["m"], e["n"], e["k"], e["y"].data_ptr(),
                      e["n"], q.QG_OUT_BF16)))

    def make_events(n):
        return [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]

    def step(events, stream=st):
        """One pass of the launch list on `stream`; events[i] (or None) brackets launch i."""
        for (key, fn, fargs), ev in zip(plan, events):
            if ev is not None:
                ev[0].record()
            rc = fn(*fargs, stream)
            if ev is not None:
                ev[1].record()
            if rc != 0:
                raise q.QGError(rc, str(key))

    for _ in range(args.warmup):
        step([None] * len(plan))
    torch.cuda.synchronize()
    # Per-launch breakdown (the parts below) from an instrumented pass of its
    # own: an event pair around every launch adds a few microseconds of queue
    # gap per launch, so the timed steps carry events only around the launches
    # of the dominant kernel, whose average duration the roofline needs.
    bd_events = [make_events(len(plan)) for _ in range(args.steps)]
    for i in range(args.steps):
        step(bd_events[i])
    torch.cuda.synchronize()
    durations = {}  # per-launch durations (ms), instrumented pass
    for evs in bd_events:
        for (key, _, _), (s, e) in zip(plan, evs):
            durations.setdefault(key, []).append(s.elapsed_time(e))
    shares = {kind: sum(sum(durations.get(("gemm", kind, e["name"]))) for e in dit) for kind in ("fp8", "nvfp4")}
    dom = max(shares, key=shares.get)
    dom_idx = [i for i, (key, _, _) in enumerate(plan) if key[0] == "gemm" and key[1] == dom]

    # The timed steps: the launch list run --steps times, with events around
    # the launches of the dominant kernel (their durations give the roofline).
    # (ROCm's torch does not allow event-record nodes in captured graphs, so
    # the timed region is the eager launch loop; the graph-replayed step time
    # and the eager step without any event are reported beside it in parts.
    # Graph segments between eager dominant launches were slower than either:
    # each segment replay costs more than the queue gaps it removes.)
    step_events = []
    for _ in range(args.steps):
        ev = [None] * len(plan)
        for i in dom_idx:
            ev[i] = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        step_events.append(ev)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.time()
    t0.record()
    for i in range(args.steps):
        step(step_events[i])
    t1.record()
    torch.cuda.synchronize()
    wall = time.time() - wall0
    step_ms = t0.elapsed_time(t1) / args.steps
    dom_live = {}  # dominant-kernel launch durations (ms) inside the timed steps
    for evs in step_events:
        for i in dom_idx:
            dom_live.setdefault(plan[i][0], []).append(evs[i][0].elapsed_time(evs[i][1]))
    timing_mode = "eager launches (events around the dominant kernel)"
    # the same eager step without any event, for comparison
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(args.steps):
        step([None] * len(plan))
    e1.record()
    torch.cuda.synchronize()
    eager_step_ms = e0.elapsed_time(e1) / args.steps
    # the same step as a graph replay without any inner event (GPU time of the
    # launch list with no host launch latency between launches), for context
    graph_step_us = graph_us(lambda s: step([None] * len(plan), s), reps=args.steps)

    # ------------------------------------------------------------ accounting
    def flops(e, m=M):
        return 2.0 * m * e["n"] * e["k"]

    parts = {}
    total_flops = 0.0
    for kind in ("fp8", "nvfp4"):
        gemm_ms = sum(np.mean(durations.get(("gemm", kind, e["name"]))) for e in dit)
        quant_ms = sum(np.mean(durations.get(("quant", kind, e["name"]))) for e in dit)
        f = sum(flops(e) for e in dit)
        total_flops += f
        # algorithmic bytes of the activation quantizer: read 2 B/elem, write codes (+ scales)
        qbytes = sum(M * e["k"] * (2 + (1.0 if kind == "fp8" else 0.5625)) for e in dit)
        per = {e["name"]: {"gemm_us": round(1e3 * float(np.mean(durations.get(("gemm", kind, e["name"])))), 2),
                           "quant_us": round(1e3 * float(np.mean(durations.get(("quant", kind, e["name"])))), 2),
                           "gemm_tflops": round(flops(e) / (1e9 * float(np.mean(durations.get(("gemm", kind, e["name"]))))), 1)}
               for e in dit}
        parts[kind] = {
            "gemm_tflops": round(f / (gemm_ms * 1e9), 1),
            "linear_tflops_incl_quant": round(f / ((gemm_ms + quant_ms) * 1e9), 1),
            "gemm_frac_of_%s_peak" % kind: round(f / (gemm_ms * 1e9) / PEAK["fp8" if kind == "fp8" else "fp4"], 4),
            "quant_gbs": round(qbytes / (quant_ms * 1e6), 1),
            "per_linear": per,
        }
        if kind == "nvfp4":
            parts[kind]["gemm_frac_of_f16_mfma_peak"] = round(f / (gemm_ms * 1e9) / PEAK["f16"], 4)
    w4 = {}
    for e in enc:
        key = "%s_m%d" % (e["name"], e["m"])
        ms = float(np.mean(durations.get(("gemm", "w4a16", key))))
        byt = e["n"] * e["k"] * 0.5625 + e["m"] * e["k"] * 2 + e["m"] * e["n"] * 2
        total_flops += flops(e, e["m"])
        args_w = next(fa for (k2, _, fa) in plan if k2 == ("gemm", "w4a16", key))
        gus = graph_us(lambda s: lib.qg_gemm(*args_w, s))
        w4[key] = {"us": round(ms * 1e3, 2), "gbs": round(byt / (ms * 1e6), 1),
                   "tflops": round(flops(e, e["m"]) / (ms * 1e9), 2),
                   "graph_us": round(gus, 2) if gus else None,
                   "graph_gbs": round(byt / (gus * 1e3), 1) if gus else None}
    parts["w4a16_single_call"] = w4
    parts["w4a16_single_call_note"] = ("us: HIP events around the call in the instrumented step (host launch "
                                       "latency included); graph_us: GPU time per call from graph replays")
    parts["launch_sum_ms_per_step"] = round(sum(sum(v) for v in durations.values()) / args.steps, 4)
    parts["graph_replay_ms_per_step"] = round(graph_step_us / 1e3, 4) if graph_step_us else None
    parts["eager_no_event_ms_per_step"] = round(eager_step_ms, 4)
    parts["static_scales"] = static_scale_part(q, lib, st, dit, M, flops)
    parts["mx"] = mx_part(q, lib, st, dit, M, flops, parts["nvfp4"], parts["fp8"])
    parts["dit_block_chain"] = block_chain_part(q, dit, M)
    parts["vendor_gemm"] = vendor_gemm_part(q, dit, M, durations)
    parts["weight_streaming"] = weight_streaming_part(q, dit, M)
    parts["w8a8_encoder"] = w8a8_encoder_part(q, enc)
    parts["w4a16_cold_pool"] = w4a16_pool(q, synth, args.pool_mib)
    parts["single_linear"] = single_linear_part(q, synth)

    # dominant kernel: the GEMM kind with the largest share of the step, its
    # launches timed live inside the timed steps
    launches = [(flops(e), d) for e in dit for d in dom_live[("gemm", dom, e["name"])]]
    fl = sum(a for a, _ in launches)
    dur_ms = sum(d for _, d in launches)
    achieved = fl / (dur_ms * 1e9)  # TFLOP/s
    peak = PEAK["fp8"] if dom == "fp8" else PEAK["f16"]
    traffic, tinfo = recorded_traffic(dom)
    roofline = {"bound": "mfma",
                "kernel": "k_gemm_fp8_direct (W8A8, fp8 MFMA)" if dom == "fp8" else "k_gemm_nvfp4_direct (W4A4, fp16 MFMA)",
                "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": traffic,
                "frac_of_fp4_peak": round(achieved / PEAK["fp4"], 4) if dom == "nvfp4" else None,
                "traffic_note": ("HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated), "
                                 "algorithmic %d" % tinfo["algorithmic_bytes_per_launch"]) if traffic else tinfo,
                "avg_launch_us": round(1e3 * dur_ms / len(launches), 2), "launches": len(launches),
                "flops_per_launch_avg": fl / len(launches)}

    # per-format figures: the GEMMs of each format against their own peaks
    # (NVFP4 against the fp4 peak first, and the fp16 matrix rate it runs on)
    pool = parts["w4a16_cold_pool"]
    sl = parts["single_linear"]
    headline = {
        "fp8_w8a8_dit_gemm_tflops": parts["fp8"]["gemm_tflops"],
        "fp8_w8a8_frac_of_fp8_peak": parts["fp8"]["gemm_frac_of_fp8_peak"],
        "nvfp4_w4a4_dit_gemm_tflops": parts["nvfp4"]["gemm_tflops"],
        "nvfp4_w4a4_frac_of_fp4_peak": parts["nvfp4"]["gemm_frac_of_nvfp4_peak"],
        "nvfp4_w4a4_frac_of_f16_mfma_peak": parts["nvfp4"]["gemm_frac_of_f16_mfma_peak"],
        "w4a16_pool_m1_gbs": pool["m1"]["gbs"], "w4a16_pool_m1_frac_of_hbm": pool["m1"]["frac_of_hbm_peak"],
        "w4a16_pool_m16_gbs": pool["m16"]["gbs"], "w4a16_pool_m16_frac_of_hbm": pool["m16"]["frac_of_hbm_peak"],
        "w4a16_pool_m256_frac_of_bf16_peak": pool["m256"]["frac_of_bf16_peak"],
        "w4a16_pool_m512_frac_of_bf16_peak": pool["m512"]["frac_of_bf16_peak"],
        "c1_fp8_128x256x256_linear_us": sl["c1_fp8_128x256x256"]["fused_linear_us"],
        "c1_fp8_128x256x256_quantize_then_gemm_us": sl["c1_fp8_128x256x256"]["linear_us"],
        "c2_nvfp4_512x3072x3072_gemm_us": sl["c2_nvfp4_512x3072x3072"]["gemm_us"],
        "c2_nvfp4_frac_of_roofline_f16_mfma": sl["c2_nvfp4_512x3072x3072"]["frac_of_roofline_f16_mfma"],
    }
    value = total_flops / (step_ms * 1e9)
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "fp8(e4m3)+fp16(nvfp4 exact dequant)+bf16(w4a16)", "data": "synthetic",
        "config": {"workload": "DiT block linears at 1024^2 (M=4608; QKV 3072->9216, attn-out 3072->3072, "
                               "MLP-up 3072->9216, MLP-down 9216->3072) as FP8 W8A8 and NVFP4 W4A4 with "
                               "run-time activation quantization, + W4A16 text-encoder linears "
                               "1024<->3072 at M in {1,16,256,512}",
                   "tokens": M, "seed": 0},
        "roofline": roofline,
        "headline": headline,
        "parts": parts,
        "timing": timing_mode,
        "setup_s": round(t_setup, 1),
        "timed_wall_s": round(wall, 3),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
    print(json.dumps(out), flush=True)


def graph_us(fn, reps=40):
    """GPU time per call of fn(stream) (microseconds): `reps` calls captured in
    a HIP graph, the replay timed with events (no host launch latency between
    the calls); None where the runtime cannot capture them."""
    import torch
    try:
        cs = torch.cuda.Stream()
        with torch.cuda.stream(cs):
            fn(cs.cuda_stream)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cs):
            for _ in range(reps):
                fn(cs.cuda_stream)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (3 * reps) * 1e3
    except Exception as ex:
        print("graph timing unavailable (%s)" % str(ex)[:200], file=sys.stderr)
        return None


def single_linear_part(q, synth, reps=50):
    """The two single-linear configurations: FP8 W8A8 128x256x256 and NVFP4
    W4A4 512x3072x3072 (X ~ N(0,1), W ~ N(0,0.02), seed 0), each call the
    dynamic activation quantize plus the GEMM through the C ABI (the weight
    quantized and packed offline). GPU time per call from graph replays;
    beside it the median of `reps` calls bracketed by HIP events one by one
    (which includes the host's launch latency). The NVFP4 GEMM is placed
    against its roofline:
    max(2MNK / peak, algorithmic bytes / HBM peak) for the fp16 matrix rate
    it runs on, and for the fp4 peak the format nominally targets."""
    import torch
    lib = q.lib()
    st = torch.cuda.current_stream().cuda_stream
    out = {}
    for name, fmt, (m, n, k) in (("c1_fp8_128x256x256", q.QG_FMT_FP8_E4M3, (128, 256, 256)),
                                 ("c2_nvfp4_512x3072x3072", q.QG_FMT_NVFP4, (512, 3072, 3072))):
        x = dev_bf16(synth.normal_bf16(m, k, synth.SIGMA_X, 0, synth.STREAM_X))
        w = dev_bf16(synth.normal_bf16(n, k, synth.SIGMA_W, 0, synth.STREAM_W))
        packed = q.pack(q.quantize(w, fmt))
        nv = fmt == q.QG_FMT_NVFP4
        codes = torch.empty((m, k // 2 if nv else k), dtype=torch.uint8, device="cuda")
        bs = torch.empty((m, k // 16), dtype=torch.uint8, device="cuda") if nv else None
        ts = torch.empty(1, dtype=torch.float32, device="cuda")
        y = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
        bsp = bs.data_ptr() if nv else None
        qargs = (fmt, x.data_ptr(), m, k, k, codes.data_ptr(), bsp, ts.data_ptr(), st)
        gargs = (fmt, codes.data_ptr(), bsp, ts.data_ptr(), k, fmt, packed.data_ptr(), packed.numel(),
                 m, n, k, y.data_ptr(), n, q.QG_OUT_BF16, st)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps + 5)]
        for i in range(reps + 5):
            evs[i][0].record()
            assert lib.qg_quantize_act(*qargs) == 0
            evs[i][1].record()
            assert lib.qg_gemm(*gargs) == 0
            evs[i][2].record()
        torch.cuda.synchronize()
        qus_l = float(np.median([ev[0].elapsed_time(ev[1]) for ev in evs[5:]])) * 1e3
        gus_l = float(np.median([ev[1].elapsed_time(ev[2]) for ev in evs[5:]])) * 1e3
        # GPU time per call from graph replays (the host's launch latency, a
        # few microseconds per call, is part of the event-pair figures above)
        qus = graph_us(lambda s: lib.qg_quantize_act(*qargs[:-1], s)) or qus_l
        gus = graph_us(lambda s: lib.qg_gemm(*gargs[:-1], s)) or gus_l
        flops = 2.0 * m * n * k
        wbytes = n * k * (0.5625 if nv else 1.0)
        abytes = m * k * (0.5625 if nv else 1.0)
        gbytes = wbytes + abytes + m * n * 2
        ent = {"quant_us": round(qus, 2), "gemm_us": round(gus, 2), "linear_us": round(qus + gus, 2),
               "with_host_launch": {"quant_us": round(qus_l, 2), "gemm_us": round(gus_l, 2)},
               "gemm_tflops": round(flops / (gus * 1e6), 1), "gemm_algorithmic_mb": round(gbytes / 1e6, 2)}
        if not nv:
            # the same linear in one launch: qg_linear_fp8 quantizes the bf16
            # activation inside the GEMM (same codes, scale and output bits)
            largs = (x.data_ptr(), k, ts.data_ptr(), packed.data_ptr(), packed.numel(), m, n, k, y.data_ptr(), n,
                     q.QG_OUT_BF16, st)
            fev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(reps + 5)]
            for i in range(reps + 5):
                fev[i][0].record()
                assert lib.qg_linear_fp8(*largs) == 0
                fev[i][1].record()
            torch.cuda.synchronize()
            fus_l = float(np.median([ev[0].elapsed_time(ev[1]) for ev in fev[5:]])) * 1e3
            fus = graph_us(lambda s: lib.qg_linear_fp8(*largs[:-1], s)) or fus_l
            ent["fused_linear_us"] = round(fus, 2)
            ent["with_host_launch"]["fused_linear_us"] = round(fus_l, 2)
        if nv:
            t_f16 = max(flops / (PEAK["f16"] * 1e12), gbytes / (PEAK["hbm_gbs"] * 1e9)) * 1e6
            t_fp4 = max(flops / (PEAK["fp4"] * 1e12), gbytes / (PEAK["hbm_gbs"] * 1e9)) * 1e6
            ent.update({"roofline_us_f16_mfma": round(t_f16, 2), "frac_of_roofline_f16_mfma": round(t_f16 / gus, 4),
                        "roofline_us_fp4": round(t_fp4, 2), "frac_of_roofline_fp4": round(t_fp4 / gus, 4)})
        else:
            ent["note"] = "16.8 MFLOP on 0.16 MB: launch-latency bound, reported in microseconds"
        out[name] = ent
        del packed, codes, bs, ts, y
    return out


def w8a8_encoder_part(q, enc, reps=20):
    """W8A8 at the text-encoder shapes (the FP8 alternative to W4A16 for the
    small encoder): dynamic activation quantize + FP8 GEMM per call, with
    preallocated buffers and raw C-ABI launches: GPU time per call from graph
    replays, and the HIP-event time per launch (host launch latency included)."""
    import torch
    lib = q.lib()
    st = torch.cuda.current_stream().cuda_stream
    out = {}
    for e in enc:
        m, n, k = e["m"], e["n"], e["k"]
        codes = torch.empty((m, k), dtype=torch.uint8, device="cuda")
        ts = torch.empty(1, dtype=torch.float32, device="cuda")
        y = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
        qargs = (q.QG_FMT_FP8_E4M3, e["x"].data_ptr(), m, k, k, codes.data_ptr(), None, ts.data_ptr(), st)
        gargs = (q.QG_FMT_FP8_E4M3, codes.data_ptr(), None, ts.data_ptr(), k, q.QG_FMT_FP8_E4M3,
                 e["w8"].data_ptr(), e["w8"].numel(), m, n, k, y.data_ptr(), n, q.QG_OUT_BF16, st)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps + 3)]
        for i in range(reps + 3):
            evs[i][0].record()
            assert lib.qg_quantize_act(*qargs) == 0
            evs[i][1].record()
            assert lib.qg_gemm(*gargs) == 0
            evs[i][2].record()
        torch.cuda.synchronize()
        qus_l = float(np.mean([ev[0].elapsed_time(ev[1]) for ev in evs[3:]])) * 1e3
        gus_l = float(np.mean([ev[1].elapsed_time(ev[2]) for ev in evs[3:]])) * 1e3
        qus = graph_us(lambda s: lib.qg_quantize_act(*qargs[:-1], s)) or qus_l
        gus = graph_us(lambda s: lib.qg_gemm(*gargs[:-1], s)) or gus_l
        ent = {"quant_us": round(qus, 2), "gemm_us": round(gus, 2),
               "gemm_tflops": round(2 * m * n * k / (gus * 1e6), 2),
               "with_host_launch": {"quant_us": round(qus_l, 2), "gemm_us": round(gus_l, 2)}}
        if m * k <= 65536:
            # quantize + GEMM in one launch (qg_linear_fp8), same output bits
            largs = (e["x"].data_ptr(), k, ts.data_ptr(), e["w8"].data_ptr(), e["w8"].numel(), m, n, k,
                     y.data_ptr(), n, q.QG_OUT_BF16)
            ent["fused_linear_us"] = round(graph_us(lambda s: lib.qg_linear_fp8(*largs, s)) or 0.0, 2)
        out["%s_m%d" % (e["name"], m)] = ent
    return out


def vendor_gemm_part(q, dit, M, durations, reps=20):
    """The vendor GEMM library (hipBLASLt, reached through torch) at the same
    four transformer shapes, for context: BF16 x BF16 (torch.mm) and FP8 E4M3
    x FP8 E4M3 with per-tensor scales (torch._scaled_mm), the same operands
    and output type as this library's W8A8 GEMM. Times are single launches
    bracketed by HIP events (median of `reps`); ratio = vendor time / this
    library's time for the matching GEMM of the step (above 1: this library
    is faster). There is no vendor NVFP4 (E4M3 16-element block scale) GEMM
    on this chip; the W4A4 kernel is compared with the vendor BF16 GEMM."""
    import torch
    out = {}
    one = torch.ones((), device="cuda")
    for e in dit:
        n, k = e["n"], e["k"]
        x = e["x"]["fp8"]
        w = e["w_bf16"]
        a8 = torch.empty((M, k), dtype=torch.uint8, device="cuda")
        ts = torch.empty(1, dtype=torch.float32, device="cuda")
        wq = q.quantize(w, q.QG_FMT_FP8_E4M3)
        st = torch.cuda.current_stream().cuda_stream
        assert q.lib().qg_quantize_act(q.QG_FMT_FP8_E4M3, x.data_ptr(), M, k, k, a8.data_ptr(), None,
                                       ts.data_ptr(), st) == 0
        af8 = a8.view(torch.float8_e4m3fn)
        wf8 = wq.codes.view(torch.float8_e4m3fn)
        y = torch.empty((M, n), dtype=torch.bfloat16, device="cuda")
        fns = {"bf16": lambda: torch.mm(x, w.t(), out=y),
               "fp8": lambda: torch._scaled_mm(af8, wf8.t(), scale_a=ts[0], scale_b=wq.tensor_scale[0],
                                               out_dtype=torch.bfloat16)}
        res = {}
        for kind, f in fns.items():
            try:
                for _ in range(3):
                    f()
                evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
                for s0, s1 in evs:
                    s0.record()
                    f()
                    s1.record()
                torch.cuda.synchronize()
                us = float(np.median([s0.elapsed_time(s1) for s0, s1 in evs])) * 1e3
                res[kind] = {"us": round(us, 2), "tflops": round(2.0 * M * n * k / (us * 1e6), 1)}
            except Exception as ex:  # the vendor path is context only
                res[kind] = {"error": str(ex)[:120]}
        ours_fp8 = 1e3 * float(np.mean(durations[("gemm", "fp8", e["name"])]))
        ours_nv = 1e3 * float(np.mean(durations[("gemm", "nvfp4", e["name"])]))
        if "us" in res.get("fp8", {}):
            res["fp8"]["ratio_vs_w8a8"] = round(res["fp8"]["us"] / ours_fp8, 3)
            # same codes and scales as this library's W8A8 output of the step:
            # the two differ only by accumulation order and bf16 rounding
            yv = fns["fp8"]().float()
            yo = e["y_fp8"].float()
            res["fp8"]["max_diff_vs_w8a8_rel_to_max"] = float((yv - yo).abs().max() / yo.abs().max())
        if "us" in res.get("bf16", {}):
            res["bf16"]["ratio_vs_w4a4"] = round(res["bf16"]["us"] / ours_nv, 3)
        out[e["name"]] = res
        del a8, wq, y
    return out


def block_chain_part(q, dit, M, steps=10):
    """The four linears of one transformer block as a chain, data flowing
    through: QKV -> (attention stubbed: the V third of the QKV output) ->
    attention-out -> MLP-up -> GELU -> MLP-down, in BF16 (hipBLASLt through
    torch.mm: the unquantized baseline), FP8 W8A8 and NVFP4 W4A4 (this
    library: dynamic activation quantization + GEMM per linear). Same
    weights, same input; GELU and the slice are shared glue. Reports the
    chain time per precision and the speed-up over BF16 (the paper's step
    ratio of BF16 -> FP8 -> NVFP4 comes from these linears)."""
    import torch
    import torch.nn.functional as F
    by = {e["name"]: e for e in dit}
    x0 = dit[0]["x"]["fp8"]  # N(0,1) input of the block [M, 3072]

    def chain_bf16():
        h = torch.mm(x0, by["qkv"]["w_bf16"].t())
        v = h[:, 6144:9216]
        a = torch.mm(v, by["attn_out"]["w_bf16"].t())
        u = F.gelu(torch.mm(a, by["mlp_up"]["w_bf16"].t()), approximate="tanh")
        return torch.mm(u, by["mlp_down"]["w_bf16"].t())

    def chain_q(kind, fmt):
        def lin(x, name):
            e = by[name]
            return q.linear(q.quantize(x, fmt), e["w_" + kind], fmt, e["n"])
        h = lin(x0, "qkv")
        v = h[:, 6144:9216]
        a = lin(v, "attn_out")
        u = F.gelu(lin(a, "mlp_up"), approximate="tanh")
        return lin(u, "mlp_down")

    # FP8 with static (calibrated) activation scales and the quantization of
    # QKV's and attention-out's outputs fused into their GEMM epilogues
    # (qg_gemm_quant); the scales are those the dynamic chain derives
    FP8 = q.QG_FMT_FP8_E4M3

    def calibrate():
        sc = {}
        a0 = q.quantize(x0, FP8)
        h = q.linear(a0, by["qkv"]["w_fp8"], FP8, 9216)
        av = q.quantize(h[:, 6144:9216], FP8)
        a = q.linear(av, by["attn_out"]["w_fp8"], FP8, 3072)
        aa = q.quantize(a, FP8)
        u = F.gelu(q.linear(aa, by["mlp_up"]["w_fp8"], FP8, 9216), approximate="tanh")
        au = q.quantize(u, FP8)
        for key, t in (("x0", a0), ("v", av), ("a", aa), ("u", au)):
            sc[key] = t.tensor_scale.clone()
        return sc

    cal = calibrate()
    qkv_codes = torch.empty((M, 9216), dtype=torch.uint8, device="cuda")
    ao_codes = torch.empty((M, 3072), dtype=torch.uint8, device="cuda")

    def chain_fp8_fused():
        a0 = q.quantize(x0, FP8, static_scale=cal["x0"])
        wq, wa = by["qkv"]["w_fp8"], by["attn_out"]["w_fp8"]
        q.qg_gemm_quant(FP8, a0.codes, None, a0.tensor_scale, 3072, FP8, wq, wq.numel(), M, 9216, 3072,
                        qkv_codes, 9216, cal["v"])
        # the V third of the QKV codes is the attention-out operand (row pitch 9216)
        q.qg_gemm_quant(FP8, qkv_codes.data_ptr() + 6144, None, cal["v"], 9216, FP8, wa, wa.numel(), M, 3072,
                        3072, ao_codes, 3072, cal["a"])
        u = F.gelu(q.linear(q.QTensor(FP8, ao_codes, None, cal["a"], M, 3072), by["mlp_up"]["w_fp8"], FP8, 9216),
                   approximate="tanh")
        return q.linear(q.quantize(u, FP8, static_scale=cal["u"]), by["mlp_down"]["w_fp8"], FP8, 3072)

    # the same with NVFP4: calibrated tensor scales, the QKV and attention-out
    # outputs written as NVFP4 codes and block scales by their epilogues
    # (qg_gemm_quant_nvfp4), attention-out reading the V third in place
    NV = q.QG_FMT_NVFP4

    def calibrate_nv():
        sc = {}
        a0 = q.quantize(x0, NV)
        h = q.linear(a0, by["qkv"]["w_nvfp4"], NV, 9216)
        av = q.quantize(h[:, 6144:9216], NV)
        a = q.linear(av, by["attn_out"]["w_nvfp4"], NV, 3072)
        aa = q.quantize(a, NV)
        u = F.gelu(q.linear(aa, by["mlp_up"]["w_nvfp4"], NV, 9216), approximate="tanh")
        au = q.quantize(u, NV)
        for key, t in (("x0", a0), ("v", av), ("a", aa), ("u", au)):
            sc[key] = t.tensor_scale.clone()
        return sc

    cal_nv = calibrate_nv()
    qkv_nv = (torch.empty((M, 9216 // 2), dtype=torch.uint8, device="cuda"),
              torch.empty((M, 9216 // 16), dtype=torch.uint8, device="cuda"))
    ao_nv = (torch.empty((M, 3072 // 2), dtype=torch.uint8, device="cuda"),
             torch.empty((M, 3072 // 16), dtype=torch.uint8, device="cuda"))

    def chain_nvfp4_fused():
        a0 = q.quantize(x0, NV, static_scale=cal_nv["x0"])
        wq, wa = by["qkv"]["w_nvfp4"], by["attn_out"]["w_nvfp4"]
        q.qg_gemm_quant_nvfp4(NV, a0.codes, a0.block_scales, a0.tensor_scale, 3072, NV, wq, wq.numel(), M, 9216,
                              3072, qkv_nv[0], qkv_nv[1], 9216, cal_nv["v"])
        # the V third of the QKV codes and block scales (row pitch 9216 elements)
        q.qg_gemm_quant_nvfp4(NV, qkv_nv[0].data_ptr() + 3072, qkv_nv[1].data_ptr() + 384, cal_nv["v"], 9216, NV,
                              wa, wa.numel(), M, 3072, 3072, ao_nv[0], ao_nv[1], 3072, cal_nv["a"])
        u = F.gelu(q.linear(q.QTensor(NV, ao_nv[0], ao_nv[1], cal_nv["a"], M, 3072), by["mlp_up"]["w_nvfp4"], NV,
                            9216), approximate="tanh")
        return q.linear(q.quantize(u, NV, static_scale=cal_nv["u"]), by["mlp_down"]["w_nvfp4"], NV, 3072)

    runs = {"bf16": chain_bf16, "fp8": lambda: chain_q("fp8", q.QG_FMT_FP8_E4M3),
            "fp8_static_fused": chain_fp8_fused, "nvfp4_static_fused": chain_nvfp4_fused,
            "nvfp4": lambda: chain_q("nvfp4", q.QG_FMT_NVFP4),
            "mxfp4": lambda: chain_q("mxfp4", q.QG_FMT_MXFP4),
            "mxfp8": lambda: chain_q("mxfp8", q.QG_FMT_MXFP8)}
    res = {}
    outs = {}
    for name, fn in runs.items():
        for _ in range(2):
            outs[name] = fn()
        torch.cuda.synchronize()
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        for _ in range(steps):
            fn()
        s1.record()
        torch.cuda.synchronize()
        res[name] = {"ms": round(s0.elapsed_time(s1) / steps, 4)}
    for name in ("fp8", "fp8_static_fused", "nvfp4", "nvfp4_static_fused", "mxfp4", "mxfp8"):
        res[name]["speedup_vs_bf16"] = round(res["bf16"]["ms"] / res[name]["ms"], 3)
        # agreement of the chain output with the BF16 chain (relative Frobenius error)
        d = (outs[name].float() - outs["bf16"].float()).norm() / outs["bf16"].float().norm()
        res[name]["rel_err_vs_bf16"] = round(float(d), 4)
    d = (outs["fp8_static_fused"].float() - outs["fp8"].float()).norm() / outs["fp8"].float().norm()
    res["fp8_static_fused"]["rel_diff_vs_fp8_chain"] = round(float(d), 4)
    d = (outs["nvfp4_static_fused"].float() - outs["nvfp4"].float()).norm() / outs["nvfp4"].float().norm()
    res["nvfp4_static_fused"]["rel_diff_vs_nvfp4_chain"] = round(float(d), 4)
    res["note"] = ("chain time includes the activation quantizers, GELU and the allocating Python "
                   "helpers; attention is stubbed; *_static_fused: calibrated activation scales, the QKV "
                   "and attention-out outputs quantized in their GEMM epilogues (qg_gemm_quant for FP8, "
                   "qg_gemm_quant_nvfp4 for NVFP4), attention-out reading the V third of the codes in place")
    return res


def mx_part(q, lib, st, dit, M, flops, nvfp4, fp8, steps=10):
    """The DiT linears in the OCP MX formats (E2M1 / E4M3 elements, E8M0
    scale per 32, no tensor scale): one quantize kernel + the GEMM on the
    block-scaled matrix instruction per linear, on the same heavy-tailed
    activations as the NVFP4 step. Reports the GEMM rate against the format's
    peak, the speed-up over the exact NVFP4 GEMM (MXFP4) and the per-tensor
    FP8 GEMM (MXFP8), and how far each format's output lies from the
    unquantized product (relative Frobenius error against torch.mm in fp32
    of the bf16 operands, sampled rows)."""
    import torch
    out = {}
    rows = torch.arange(0, M, M // 256, device="cuda")[:256]
    refs = {}
    for e in dit:
        refs[e["name"]] = torch.mm(e["x"]["nvfp4"][rows].float(), e["w_bf16"].float().t())
    for kind, fmt in (("mxfp4", q.QG_FMT_MXFP4), ("mxfp8", q.QG_FMT_MXFP8)):
        plan, bufs = [], {}
        for e in dit:
            k, n = e["k"], e["n"]
            codes = torch.empty((M, k // 2 if kind == "mxfp4" else k), dtype=torch.uint8, device="cuda")
            bs = torch.empty((M, k // 32), dtype=torch.uint8, device="cuda")
            y = torch.empty((M, n), dtype=torch.bfloat16, device="cuda")
            bufs[e["name"]] = (codes, bs, y)
            plan.append((("mxquant", e["name"]), lib.qg_quantize_act,
                         (fmt, e["x"]["nvfp4"].data_ptr(), M, k, k, codes.data_ptr(), bs.data_ptr(), None, st)))
            plan.append((("mxgemm", e["name"]), lib.qg_gemm,
                         (fmt, codes.data_ptr(), bs.data_ptr(), None, k, fmt, e["w_" + kind].data_ptr(),
                          e["w_" + kind].numel(), M, n, k, y.data_ptr(), n, q.QG_OUT_BF16, st)))
        evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in plan]
               for _ in range(steps + 2)]
        for i in range(steps + 2):
            for (key, fn, fargs), (s0, s1) in zip(plan, evs[i]):
                s0.record()
                rc = fn(*fargs)
                s1.record()
                if rc != 0:
                    raise q.QGError(rc, str(key))
        torch.cuda.synchronize()
        dur = {}
        for i in range(2, steps + 2):
            for (key, _, _), (s0, s1) in zip(plan, evs[i]):
                dur.setdefault(key, []).append(s0.elapsed_time(s1))
        gms = {e["name"]: float(np.mean(dur[("mxgemm", e["name"])])) for e in dit}
        qms = {e["name"]: float(np.mean(dur[("mxquant", e["name"])])) for e in dit}
        f = sum(flops(e) for e in dit)
        g_all, q_all = sum(gms.values()), sum(qms.values())
        rate = f / (g_all * 1e9)
        rel = {e["name"]: round(float((bufs[e["name"]][2][rows].float() - refs[e["name"]]).norm()
                                      / refs[e["name"]].norm()), 4) for e in dit}
        out[kind] = {"per_linear": {e["name"]: {"gemm_us": round(1e3 * gms[e["name"]], 2),
                                                "quant_us": round(1e3 * qms[e["name"]], 2),
                                                "gemm_tflops": round(flops(e) / (gms[e["name"]] * 1e9), 1)}
                                    for e in dit},
                     "gemm_tflops": round(rate, 1),
                     "gemm_frac_of_%s_peak" % ("fp4" if kind == "mxfp4" else "fp8"):
                         round(rate / PEAK["fp4" if kind == "mxfp4" else "fp8"], 4),
                     "linear_tflops_incl_quant": round(f / ((g_all + q_all) * 1e9), 1),
                     "rel_err_vs_unquantized": rel}
        if kind == "mxfp4":
            out[kind]["gemm_speedup_vs_nvfp4"] = round(rate / nvfp4["gemm_tflops"], 3)
        else:
            out[kind]["gemm_speedup_vs_fp8"] = round(rate / fp8["gemm_tflops"], 3)
    out["nvfp4_rel_err_vs_unquantized"] = {
        e["name"]: round(float((e["y_nvfp4"][rows].float() - refs[e["name"]]).norm() / refs[e["name"]].norm()), 4)
        for e in dit}
    out["note"] = ("MX formats are the matrix-core-native block scaling (power-of-two scales per 32); their "
                   "outputs differ from NVFP4's / FP8's by design and are checked against their own oracle")
    return out


def weight_streaming_part(q, dit, M, blocks=8, steps=3):
    """Weight streaming (the paper's second memory tool): a transformer of
    `blocks` blocks x the four linears, its packed weights in pinned host
    memory, run through qg_run_layers with the resident subset chosen by
    qg_stream_plan for a range of device budgets. Reports the measured
    host-to-device rate M, the per-linear compute L (quantize + GEMM), the
    reservoir decay factor lambda = L M / W of each linear, T_min, and per
    budget the planned and measured step times. Every block reuses the same
    four weights (one device copy, one pinned host copy each): residency only
    changes where the bytes come from, so this times the schedule, not the
    weights."""
    import ctypes
    import torch
    lib = q.lib()
    comp = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    out = {}
    for kind, fmt in (("fp8", q.QG_FMT_FP8_E4M3), ("nvfp4", q.QG_FMT_NVFP4)):
        host = {}
        for e in dit:
            w = e["w_" + kind]
            h = torch.empty(w.numel(), dtype=torch.uint8, pin_memory=True)
            h.copy_(w)
            host[e["name"]] = h
        # host-to-device rate on the copy stream (largest weight, 5 copies)
        big = max(dit, key=lambda e: e["w_" + kind].numel())
        dst = torch.empty_like(big["w_" + kind])
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        with torch.cuda.stream(copy):
            dst.copy_(host[big["name"]], non_blocking=True)
            ev[0].record()
            for _ in range(5):
                dst.copy_(host[big["name"]], non_blocking=True)
            ev[1].record()
        torch.cuda.synchronize()
        rate = 5 * dst.numel() / (ev[0].elapsed_time(ev[1]) * 1e-3)

        def layer_list(resident):
            L = []
            for b in range(blocks):
                for j, e in enumerate(dit):
                    a = e["a_" + kind]
                    r = int(resident[b * len(dit) + j])
                    w = e["w_" + kind] if r else host[e["name"]]
                    L.append(q.StreamLayer(
                        x=e["x"][kind].data_ptr(), a_fmt=fmt, a_codes=a.codes.data_ptr(),
                        a_block_scales=a.block_scales.data_ptr() if a.block_scales is not None else None,
                        a_tensor_scale=a.tensor_scale.data_ptr(), w_fmt=fmt, w_packed=w.data_ptr(),
                        w_packed_bytes=w.numel(), resident=r, m=M, n=e["n"], k=e["k"],
                        y=e["y_" + kind].data_ptr(), y_dtype=q.QG_OUT_BF16))
            return L

        nl = blocks * len(dit)
        wb = [float(dit[i % len(dit)]["w_" + kind].numel()) for i in range(nl)]
        slot_bytes = (int(max(wb)) + 255) // 256 * 256
        slots = [torch.empty(slot_bytes, dtype=torch.uint8, device="cuda") for _ in range(2)]
        evr, evf = [], []
        for _ in range(2):
            for lst in (evr, evf):
                e_ = torch.cuda.Event()
                e_.record()
                lst.append(e_)
        cursor = ctypes.c_int32(0)

        def run(resident, n_steps):
            layers = layer_list(resident)
            t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            for i in range(n_steps + 1):
                if i == 1:
                    t0.record()
                q.qg_run_layers(layers, slots, slot_bytes, [x.cuda_event for x in evr], [x.cuda_event for x in evf],
                                cursor, compute_stream=comp, copy_stream=copy)
            t1.record()
            torch.cuda.synchronize()
            return t0.elapsed_time(t1) / n_steps * 1e-3

        # per-linear compute time (quantize + GEMM) from a fully resident single block
        lin_s = {}
        for j, e in enumerate(dit):
            one = layer_list([1] * nl)[j:j + 1]
            s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            q.qg_run_layers(one, [], 0, [], [], ctypes.c_int32(0), compute_stream=comp, copy_stream=copy)
            s0.record()
            for _ in range(10):
                q.qg_run_layers(one, [], 0, [], [], ctypes.c_int32(0), compute_stream=comp, copy_stream=copy)
            s1.record()
            torch.cuda.synchronize()
            lin_s[e["name"]] = s0.elapsed_time(s1) / 10 * 1e-3
        cs = [lin_s[dit[i % len(dit)]["name"]] for i in range(nl)]
        a_max = float(max(M * e["k"] * 2 + M * e["n"] * 2 for e in dit))   # bf16 input + output of a linear
        tmin = 2 * max(wb) + a_max
        full = sum(wb) + a_max
        # the two ends first: every weight resident, every weight streamed
        plans = {}
        plans["all_resident"] = {"device_mb": round(full / 1e6, 1), "resident_layers": nl, "streamed_layers": 0,
                                 "predicted_ms": round(sum(cs) * 1e3, 3),
                                 "measured_ms": round(run([1] * nl, steps) * 1e3, 3)}
        _, pred_all = q.qg_stream_simulate(wb, cs, [0] * nl, 2, rate, 3)
        meas_all = run([0] * nl, steps)
        # Calibration: the copy rate the model needs to reproduce the measured
        # all-streamed step (copies share the GPU with the GEMMs there, so the
        # rate is below the idle-GPU one); the model's step time falls
        # monotonically with the rate, so bisection finds it.
        lo_r, hi_r = rate / 20.0, rate * 2.0
        for _ in range(60):
            mid = 0.5 * (lo_r + hi_r)
            if q.qg_stream_simulate(wb, cs, [0] * nl, 2, mid, 3)[1] > meas_all:
                lo_r = mid
            else:
                hi_r = mid
        rate_eff = 0.5 * (lo_r + hi_r)
        plans["all_streamed"] = {"device_mb": round(tmin / 1e6, 1), "resident_layers": 0, "streamed_layers": nl,
                                 "predicted_ms": round(pred_all * 1e3, 3), "measured_ms": round(meas_all * 1e3, 3)}
        # plans under device budgets, chosen with the calibrated rate; the
        # idle-GPU rate's prediction of the same plan is given beside it
        for label, budget in (("resident_100", full), ("resident_75", a_max + 0.75 * sum(wb)),
                              ("resident_50", a_max + 0.5 * sum(wb)), ("resident_25", a_max + 0.25 * sum(wb)),
                              ("t_min", tmin)):
            budget = max(budget, tmin)
            st_, res, pred, dev = q.qg_stream_plan(wb, cs, 2, rate_eff, budget, a_max)
            _, pred_idle = q.qg_stream_simulate(wb, cs, res, 2, rate, 3)
            meas = run(res, steps)
            plans[label] = {"budget_mb": round(budget / 1e6, 1), "device_mb": round(dev / 1e6, 1),
                            "resident_layers": int(sum(res)), "streamed_layers": nl - int(sum(res)),
                            "predicted_ms": round(pred * 1e3, 3), "predicted_idle_rate_ms": round(pred_idle * 1e3, 3),
                            "measured_ms": round(meas * 1e3, 3)}
        lam = {dit[j]["name"]: round(cs[(j - 1) % len(dit)] * rate / wb[j], 3) for j in range(len(dit))}
        out[kind] = {"layers": nl, "h2d_gbs": round(rate / 1e9, 1), "h2d_gbs_calibrated": round(rate_eff / 1e9, 1),
                     "linear_us": {k_: round(v * 1e6, 1) for k_, v in lin_s.items()},
                     "weight_mb": {e["name"]: round(e["w_" + kind].numel() / 1e6, 2) for e in dit},
                     "lambda": lam, "t_min_mb": round(tmin / 1e6, 1), "all_resident_mb": round(full / 1e6, 1),
                     "delta_all_streamed_ms": round(sum(wb) / rate * 1e3, 3),
                     "plans": plans}
    out["note"] = ("lambda = L M / W with L the compute of the preceding linear and M the idle-GPU copy rate; "
                   "delta_all_streamed = N W / M, the paper's overhead bound with no overlapped layer; "
                   "h2d_gbs_calibrated = the rate at which qg_stream_simulate reproduces the measured all-streamed "
                   "step; the budget plans are chosen and predicted with it (predicted_idle_rate_ms: the same plan "
                   "at the idle-GPU rate); all_streamed.predicted_ms uses the idle-GPU rate")
    return out


def static_scale_part(q, lib, st, dit, M, flops, steps=10):
    """The same DiT linears with static (calibrated) activation scales: one
    quantize kernel + the GEMM per linear. The calibrated scale used here is
    the one the dynamic pass derived for the same activations, so the codes
    (and the GEMMs) are those of the dynamic step."""
    import torch
    plan = []
    for kind, fmt in (("fp8", q.QG_FMT_FP8_E4M3), ("nvfp4", q.QG_FMT_NVFP4)):
        for e in dit:
            a, x, wp, y = e["a_" + kind], e["x"][kind], e["w_" + kind], e["y_" + kind]
            s_cal = a.tensor_scale.clone()
            bs = a.block_scales.data_ptr() if a.block_scales is not None else None
            plan.append((("squant", kind, e["name"]), lib.qg_quantize_act_static,
                         (fmt, x.data_ptr(), M, e["k"], e["k"], a.codes.data_ptr(), bs, s_cal.data_ptr(), st)))
            plan.append((("gemm", kind, e["name"]), lib.qg_gemm,
                         (fmt, a.codes.data_ptr(), bs, s_cal.data_ptr(), e["k"], fmt,
                          wp.data_ptr(), wp.numel(), M, e["n"], e["k"], y.data_ptr(), e["n"],
                          q.QG_OUT_BF16, st)))
            e.setdefault("keep", []).append(s_cal)
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in plan]
           for _ in range(steps + 2)]
    for i in range(steps + 2):
        for (key, fn, fargs), (s0, s1) in zip(plan, evs[i]):
            s0.record()
            rc = fn(*fargs)
            s1.record()
            if rc != 0:
                raise q.QGError(rc, str(key))
    torch.cuda.synchronize()
    dur = {}
    for i in range(2, steps + 2):
        for (key, _, _), (s0, s1) in zip(plan, evs[i]):
            dur.setdefault(key, []).append(s0.elapsed_time(s1))
    out = {}
    for kind in ("fp8", "nvfp4"):
        qms = sum(float(np.mean(dur[("squant", kind, e["name"])])) for e in dit)
        gms = sum(float(np.mean(dur[("gemm", kind, e["name"])])) for e in dit)
        f = sum(flops(e) for e in dit)
        out[kind] = {"quant_us": {e["name"]: round(1e3 * float(np.mean(dur[("squant", kind, e["name"])])), 2)
                                  for e in dit},
                     "linear_tflops_incl_quant": round(f / ((gms + qms) * 1e9), 1)}
    return out


def w4a16_pool(q, synth, pool_mib):
    """Cold-HBM W4A16: M in {1, 16} against a pool of distinct encoder weights
    stacked along N (one call streams the whole pool once; pool > 2x the
    256 MB last-level cache): HBM-bound. M in {256, 512} over the same pool
    is past the ridge point and reported against the bf16 matrix peak."""
    import torch
    n1, k1 = synth.ENCODER_LINEARS["down"]            # 1024 x 3072 per weight
    per = n1 * k1 * 0.5625
    layers = max(1, int(pool_mib * 2 ** 20 // per))
    n = layers * n1
    # quantize the pool from one seeded bf16 weight per 64 layers (tiled) to keep setup short
    w = synth.normal_bf16(64 * n1, k1, synth.SIGMA_W, 0, 200)
    wd = torch.from_numpy(w.view(np.int16)).view(torch.bfloat16).cuda()
    reps = (layers + 63) // 64
    wd = wd.repeat(reps, 1)[:n].contiguous()
    packed = q.pack(q.quantize(wd, q.QG_FMT_NVFP4))
    del wd
    res = {"layers": layers, "pool_mb": round(packed.numel() / 1e6, 1),
           "timing": "each call after a read-only pass over 1 GiB of other memory (last-level cache "
                     "evicted, no dirty lines left), HIP events around the call alone"}
    # a plain read of other memory before every timed call: back-to-back calls
    # over one pool can find part of it still in the 256 MB last-level cache
    evict = torch.ones(256 * 2 ** 20, dtype=torch.float32, device="cuda")
    for m in (1, 16, 256, 512):
        x = dev_bf16(synth.normal_bf16(m, k1, synth.SIGMA_X, 0, 300 + m))
        y = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
        fn = lambda: q.qg_gemm(q.QG_FMT_BF16, x, None, None, k1, q.QG_FMT_NVFP4, packed, packed.numel(),
                               m, n, k1, y, n, q.QG_OUT_BF16)
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        reps_t = 10
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(reps_t):
            fn()
        e.record()
        torch.cuda.synchronize()
        ms_b2b = s.elapsed_time(e) / reps_t
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps_t)]
        for a, b in ev:
            evict.sum()
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        ms = sum(a.elapsed_time(b) for a, b in ev) / reps_t
        byt = n * k1 * 0.5625 + m * k1 * 2 + m * n * 2
        res["m%d" % m] = {"us": round(ms * 1e3, 1), "gbs": round(byt / (ms * 1e6), 1),
                          "frac_of_hbm_peak": round(byt / (ms * 1e6) / PEAK["hbm_gbs"], 4),
                          "us_back_to_back": round(ms_b2b * 1e3, 1),
                          "gbs_back_to_back": round(byt / (ms_b2b * 1e6), 1)}
        if m >= 256:
            # past the ridge point (bf16 315 flop/B): bound by the bf16 matrix rate
            tf = 2.0 * m * n * k1 / (ms * 1e9)
            res["m%d" % m].update({"tflops": round(tf, 1), "frac_of_bf16_peak": round(tf / PEAK["bf16"], 4)})
    del packed, evict
    torch.cuda.empty_cache()
    return res


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(target_s: float):
    """The CPU oracle (as it stands) on a bounded sample of the NVFP4 QKV
    linear of the step, on the same inputs as the GPU (heavy-tailed X
    [4608, 3072], W [9216, 3072], seed 0): the activation quantization of the
    whole tensor (one tensor scale over all 4608 rows, the codes the GPU
    computes), its dequantization and the fp64 product for the first R rows.
    The weight is quantized offline (not timed), as on the GPU. Rate =
    2 R N K / (R/4608 of the full-tensor quantize + dequant + product of R
    rows), measured with all host threads and with one thread; R is sized
    so that the all-thread run takes about `target_s` seconds."""
    import oracle
    import synth
    M = synth.DIT_TOKENS
    n, k = synth.DIT_LINEARS["qkv"]
    x = synth.normal_bf16(M, k, synth.SIGMA_X, 0, synth.STREAM_X, synth.HEAVY_TAIL_FRAC, synth.HEAVY_TAIL_GAIN)
    w = synth.normal_bf16(n, k, synth.SIGMA_W, 0, synth.STREAM_W)
    qw, bw, sw = oracle.quantize_nvfp4(w)
    wdeq = oracle.dequant_nvfp4(qw, bw, sw)
    all_threads = oracle.num_threads()

    def run(rows):
        t0 = time.time()
        qa, ba, sa = oracle.quantize_nvfp4(x)
        t_q = time.time() - t0
        t0 = time.time()
        a = oracle.dequant_nvfp4(qa[:rows], ba[:rows], sa)
        oracle.gemm_f64(a, wdeq)
        t_p = time.time() - t0
        return t_q, t_p

    out = {"unit": "TFLOP/s", "kind": "oracle", "cpu_model": cpu_model(), "cores": all_threads}
    # size R from a small probe, then time it with all threads and with one
    oracle.set_num_threads(all_threads)
    t_q, t_p = run(16)
    rows = int(min(M, max(16, 16 * target_s / max(t_p + t_q * 16 / M, 1e-6))))
    for label, threads, r in (("all_threads", all_threads, rows), ("single_thread", 1, max(8, rows // all_threads))):
        oracle.set_num_threads(threads)
        t_q, t_p = run(r)
        t = t_q * r / M + t_p
        out[label] = {"threads": threads, "rows": r, "seconds": round(t_p + t_q, 2),
                      "full_tensor_quantize_s": round(t_q, 3), "product_s": round(t_p, 2),
                      "tflops": round(2.0 * r * n * k / t / 1e12, 6)}
    oracle.set_num_threads(all_threads)
    out["value"] = out["all_threads"]["tflops"]
    out["sample"] = ("NVFP4 W4A4 QKV linear (N=9216, K=3072, heavy-tailed X, seed 0): quantize of the whole "
                     "4608 x 3072 activation (one tensor scale) + dequant + fp64 product of its first %d rows "
                     "(all threads) / %d rows (one thread); weight quantized offline"
                     % (out["all_threads"]["rows"], out["single_thread"]["rows"]))
    return out


if __name__ == "__main__":
    main()

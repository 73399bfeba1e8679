#!/usr/bin/env python3
"""Throughput of one parallel SWA transformer block, forward + backward, on one MI355X.

A step is one pblock_forward + pblock_backward over one batch of seeded
synthetic input already resident in HBM.  The workload is the 175B model's
one-GPU tensor-parallel share (batch 1, seq 2048, hidden 12288, 12 local heads
x 128, local FFN 6144, window 2048 = full causal).  value = model FLOPs of a
step (projection GEMMs plus attention over visible pairs only) / measured time.

Prints one JSON line.  Besides the contract fields it carries:
  roofline      the dominant kernel's achieved rate against MI355X's bf16
                dense MFMA peak, timed with HIP events around that kernel
                inside the timed steps;
  steps         per-step times from a separate pass with events around every
                step;
  ag_in_proj    the in-projection pipelined with the all-gather of its input
                over 8 ranks (one GPU: shards copied from local buffers),
                against the GEMM alone and copies followed by one GEMM;
  rs_out_proj   the out-projection's partial sums pipelined with their
                reduce-scatter over 8 ranks (chunks copied into local
                buffers), against the GEMM alone and one GEMM followed by the
                copies, and the receiving side's sum;
  lamb_step     one fused LAMB optimizer step over the block's parameters
                (fp32 master weights and moments, the step's own gradients,
                bf16 copy), against the HBM peak;
  serial_block  the standard two-LayerNorm block on the same workload and
                kernels (same model FLOPs), and the parallel block's speedup
                over it;
  cpu_baseline  the fp64 CPU oracle timed on this host on whole steps.

Profiling helpers (see the commands recorded in profiles/):
  --copy-calibration   run a plain copy-like kernel of known size, for scaling
                       the FETCH_SIZE / WRITE_SIZE counters;
  --traffic-summary D1 D2 D3 D4
                       turn four rocprofv3 --pmc runs (FETCH_SIZE and WRITE_SIZE
                       of the bench, then of the copy) into the measured HBM
                       traffic per launch of the dominant kernel, written to
                       profiles/ with a fingerprint of the kernel's sources;
                       the bench reports it as roofline.traffic while the
                       sources are unchanged (null otherwise);
  --trace-summary D    markdown table of a rocprofv3 --kernel-trace --stats run,
                       per kernel and launch grid, with the block step each
                       GEMM launch belongs to.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CUs x 2.4 GHz x 4096 dense bf16 FLOP/clk/CU
PEAK_HBM_GBS = 8000.0
METRIC = "parallel-block fwd+bwd TFLOP/s and % of MI355X bf16 MFMA peak"


# GEMM steps of the backward pass that share one launch (the library's
# launch_gemm_pair): dC with dW_out, dh with dW_in; in the serial block each
# weight gradient with the GEMM before it.
GEMM_PAIRS = {"dc": "dw_out", "dh": "dw_in"}
# Workgroups of a persistent shared launch: one per CU.
PERSISTENT_WORKGROUPS = 256
SERIAL_GEMM_PAIRS = {"dg": "dw_down", "dh2": "dw_up", "d_o": "dw_o", "dh1": "dw_qkv"}


def paired_steps(s, block="parallel"):
    """The pairs of GEMM_PAIRS (SERIAL_GEMM_PAIRS) that the library launches
    together for this workload, from its own host query."""
    from paper_2402_15627_amd import pblock as pb
    pairs = GEMM_PAIRS if block == "parallel" else SERIAL_GEMM_PAIRS
    shared = pb.pblock_backward_pairs(pb.config_from_shape(s), block)
    return {a: b for (a, b), on in zip(pairs.items(), shared) if on}


def launch_key(step, s):
    """The launch a step's time is measured on: "dh+dw_in" for a pair."""
    pairs = paired_steps(s)
    return f"{step}+{pairs[step]}" if step in pairs else step


def step_work(s):
    """Algorithmic work of each pb_step: ("mfma", FLOPs) or ("hbm", bytes).
    A GEMM that shares its partner's launch counts there (its own step is
    empty)."""
    work = _step_work(s)
    for a, b in paired_steps(s).items():
        work[a] = ("mfma", work[a][1] + work[b][1])
        work[b] = ("mfma", 0)
    # db_in is then summed inside dW_in's tiles: its step is empty
    if "dh" in paired_steps(s):
        work["db_in"] = ("hbm", 0)
    return work


def _step_work(s):
    from paper_2402_15627_amd.inputs import visible_pairs
    T, H, A, F = s.tokens, s.hidden, s.attn_width, s.ffn
    n_in, k_out = s.n_in, s.k_out
    e = 2 if s.dtype == "bf16" else 4
    P = visible_pairs(s.seq, min(s.window, s.seq))
    return {
        "ln_fwd": ("hbm", 2 * T * H * e + 2 * H * e + 8 * T),
        "in_proj": ("mfma", 2 * T * H * n_in),
        "attn_fwd": ("mfma", 4 * s.batch * A * P),
        "out_proj": ("mfma", 2 * T * k_out * H),
        "dc": ("mfma", 2 * T * H * k_out),
        "dw_out": ("mfma", 2 * H * k_out * T),
        # db_out is summed with dgamma and dbeta in the LN backward's column
        # sums; its step is empty
        "db_out": ("hbm", 0),
        "attn_bwd": ("mfma", 8 * s.batch * A * P),
        "dh": ("mfma", 2 * T * n_in * H),
        "dw_in": ("mfma", 2 * n_in * H * T),
        "db_in": ("hbm", T * n_in * e + 4 * n_in),
        # x, dh and dy read, dx written (dh in the activation type), the row
        # statistics, and the three column-sum partial rows
        "ln_bwd": ("hbm", 4 * T * H * e + 8 * T + 12 * H),
    }


# Sources whose code a step's dominant kernel is built from.
KERNEL_SOURCES = {
    "gemm": ["gemm.hip", "common.h", "kernels.h"],
    "attn": ["attn.hip", "common.h", "kernels.h"],
    "ln": ["ln.hip", "common.h", "kernels.h"],
    "lamb": ["lamb.hip", "common.h", "kernels.h"],
}
STEP_SOURCE = {"in_proj": "gemm", "out_proj": "gemm", "dc": "gemm", "dw_out": "gemm", "dh": "gemm",
               "dw_in": "gemm", "attn_fwd": "attn", "attn_bwd": "attn", "ln_fwd": "ln",
               "ln_bwd": "ln", "db_out": "ln", "db_in": "ln", "lamb": "lamb", "ln": "ln",
               "dc+dw_out": "gemm", "dh+dw_in": "gemm"}
COPY_BYTES = 1 << 30  # read and written once by the calibration copy


def source_fingerprint(step):
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2402_15627_amd", "csrc")
    for f in KERNEL_SOURCES[STEP_SOURCE[step]] + ["../build.py"]:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def gemm_steps(s, block="parallel"):
    """(M, N, K) of each GEMM step as launched."""
    T, H, n_in, k_out = s.tokens, s.hidden, s.n_in, s.k_out
    if block == "serial":
        A, F = s.attn_width, s.ffn
        return {"qkv": (T, 3 * A, H), "o_proj": (T, H, A), "up": (T, F, H), "down": (T, H, F),
                "dg": (T, F, H), "dh2": (T, H, F), "d_o": (T, A, H), "dh1": (T, H, 3 * A),
                "dw_down": (H, F, T), "dw_o": (H, A, T), "dw_up": (F, H, T),
                "dw_qkv": (3 * A, H, T)}
    return {"in_proj": (T, n_in, H), "out_proj": (T, H, k_out), "dc": (T, k_out, H),
            "dw_out": (H, k_out, T), "dh": (T, H, n_in), "dw_in": (n_in, H, T)}


# Template arguments of each GEMM step's kernel as they appear in demangled
# names: A K-contiguous, B K-contiguous, epilogue (pb::Epi value).
GEMM_SIGNATURE = {"in_proj": "<true, true, (pb::Epi)1", "out_proj": "<true, true, (pb::Epi)2",
                  "dc": "<true, false, (pb::Epi)3", "dw_out": "<false, false, (pb::Epi)0",
                  "dh": "<true, false, (pb::Epi)4", "dw_in": "<false, false, (pb::Epi)0",
                  "qkv": "<true, true, (pb::Epi)1", "o_proj": "<true, true, (pb::Epi)2",
                  "up": "<true, true, (pb::Epi)1", "down": "<true, true, (pb::Epi)2",
                  "dg": "<true, false, (pb::Epi)3", "dh2": "<true, false, (pb::Epi)4",
                  "d_o": "<true, false, (pb::Epi)3", "dh1": "<true, false, (pb::Epi)4",
                  "dw_down": "<false, false, (pb::Epi)0", "dw_o": "<false, false, (pb::Epi)0",
                  "dw_up": "<false, false, (pb::Epi)0", "dw_qkv": "<false, false, (pb::Epi)0"}


def demangle(name):
    if not name.startswith("_Z"):
        return name
    try:
        import subprocess
        return subprocess.run(["c++filt", name], capture_output=True, text=True).stdout.strip()
    except OSError:
        return name


def gemm_step_of(name, grid, s, block="parallel"):
    """Block step(s) a GEMM launch belongs to ("" if none; "a/b" when two
    steps launch the same kernel on the same grid)."""
    steps = gemm_steps(s, block)
    if "gemm_bf16_dma_pair" in name:
        tiles = lambda st: gemm_tiles(*steps[st])  # noqa: E731
        # one workgroup per tile of either GEMM, or (persistent) one per CU
        wgs = lambda a, b: (min(PERSISTENT_WORKGROUPS, tiles(a) + tiles(b))  # noqa: E731
                            if "persistent" in name else tiles(a) + tiles(b))
        hits = [f"{a}+{b}" for a, b in paired_steps(s, block).items()
                if GEMM_SIGNATURE[a] in name and wgs(a, b) * 512 == grid]
        return "/".join(hits)
    hits = [st for st, mnk in steps.items()
            if "gemm_bf16" in name and GEMM_SIGNATURE[st] in name
            and gemm_grid_threads(*mnk) == grid]
    return "/".join(hits)


def gemm_tiles(M, N, K):
    """Output tiles of a bf16 GEMM (a shared launch has one workgroup per
    tile of either GEMM)."""
    from paper_2402_15627_amd import pblock as pb
    return pb.pblock_gemm_plan(pb.PB_BF16, M, N, K).tiles


def gemm_grid_threads(M, N, K, dtype="bf16"):
    """Work-items of a GEMM's main launch as the library plans it (its host
    query pblock_gemm_plan): one workgroup per whole tile and one per K-slice
    of each split tile."""
    from paper_2402_15627_amd import pblock as pb
    p = pb.pblock_gemm_plan(pb.PB_BF16 if dtype == "bf16" else pb.PB_F32, M, N, K)
    return p.workgroups * p.threads


def traffic_path(step, workload):
    return os.path.join(ROOT, "profiles", f"{step.replace('+', '_')}_{workload}_traffic.md")


def _counter_rows(d):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    with open(files[0]) as fh:
        return list(csv.DictReader(fh))


def _per_dispatch(rows, counter, pick):
    """Mean over the picked dispatches of a counter (summed over its instances)."""
    per = {}
    for r in rows:
        if r["Counter_Name"] == counter and pick(r):
            per[r["Dispatch_Id"]] = per.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    if not per:
        raise SystemExit(f"no dispatch with {counter} matched")
    return sum(per.values()) / len(per), len(per)


def traffic_summary(dirs, workload, step):
    """FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the step's kernel, scaled
    by what the same counters read for the calibration copy of COPY_BYTES."""
    from paper_2402_15627_amd.inputs import WORKLOADS
    s = WORKLOADS[workload]
    parts = step.split("+")
    if any(p not in gemm_steps(s) for p in parts):
        raise SystemExit(f"traffic summary supports the GEMM steps and pairs, not {step}")
    pick = lambda r: gemm_step_of(r["Kernel_Name"], int(r["Grid_Size"]), s) == step  # noqa: E731
    copy_pick = lambda r: "neg_kernel" in r["Kernel_Name"]  # noqa: E731
    fetch_rows = _counter_rows(dirs[0])
    grid = max(int(r["Grid_Size"]) for r in fetch_rows if pick(r)) if any(
        pick(r) for r in fetch_rows) else 0
    fetch, n1 = _per_dispatch(fetch_rows, "FETCH_SIZE", pick)
    write, n2 = _per_dispatch(_counter_rows(dirs[1]), "WRITE_SIZE", pick)
    cfetch, _ = _per_dispatch(_counter_rows(dirs[2]), "FETCH_SIZE", copy_pick)
    cwrite, _ = _per_dispatch(_counter_rows(dirs[3]), "WRITE_SIZE", copy_pick)
    ff, wf = COPY_BYTES / 1024 / cfetch, COPY_BYTES / 1024 / cwrite
    e = 2 if s.dtype == "bf16" else 4

    def algorithmic(st):  # operands read once, the output written once
        M, N, K = gemm_steps(s)[st]
        return (M * K + N * K) * e + M * N * (4 if st in ("dw_in", "dw_out") else e)
    rec = {
        "step": step, "workload": workload, "grid_threads": grid, "dispatches": [n1, n2],
        "fetch_kib": round(fetch, 1), "write_kib": round(write, 1),
        "copy_bytes": COPY_BYTES, "copy_fetch_kib": round(cfetch, 1),
        "copy_write_kib": round(cwrite, 1), "fetch_scale": round(ff, 4),
        "write_scale": round(wf, 4),
        "traffic_bytes": int(fetch * 1024 * ff + write * 1024 * wf),
        "algorithmic_bytes": sum(algorithmic(p) for p in parts),
        "source_fingerprint": source_fingerprint(step),
    }
    return rec


def lamb_traffic_summary(dirs, workload):
    """FETCH_SIZE / WRITE_SIZE per dispatch of the LAMB step's two streaming
    kernels over the block's parameters, scaled by the calibration copy, next
    to their algorithmic bytes."""
    import numpy as np
    from paper_2402_15627_amd.inputs import WORKLOADS, block_param_shapes
    s = WORKLOADS[workload]
    elements = sum(int(np.prod(sh)) for sh in block_param_shapes(s).values())
    copy_pick = lambda r: "neg_kernel" in r["Kernel_Name"]  # noqa: E731
    cfetch, _ = _per_dispatch(_counter_rows(dirs[2]), "FETCH_SIZE", copy_pick)
    cwrite, _ = _per_dispatch(_counter_rows(dirs[3]), "WRITE_SIZE", copy_pick)
    ff, wf = COPY_BYTES / 1024 / cfetch, COPY_BYTES / 1024 / cwrite
    rec = {"step": "lamb", "workload": workload, "elements": elements, "copy_bytes": COPY_BYTES,
           "copy_fetch_kib": round(cfetch, 1), "copy_write_kib": round(cwrite, 1),
           "fetch_scale": round(ff, 4), "write_scale": round(wf, 4), "kernels": {}}
    total = 0
    for kern, (rd, wr) in {"lamb_moments": (16, 8), "lamb_apply": (12, 6)}.items():
        pick = lambda r, k=kern: k in r["Kernel_Name"]  # noqa: E731
        fetch, n1 = _per_dispatch(_counter_rows(dirs[0]), "FETCH_SIZE", pick)
        write, n2 = _per_dispatch(_counter_rows(dirs[1]), "WRITE_SIZE", pick)
        tb = int(fetch * 1024 * ff + write * 1024 * wf)
        total += tb
        rec["kernels"][kern] = {"dispatches": [n1, n2], "fetch_kib": round(fetch, 1),
                                "write_kib": round(write, 1), "traffic_bytes": tb,
                                "algorithmic_bytes": (rd + wr) * elements}
    rec["traffic_bytes"] = total
    rec["algorithmic_bytes"] = LAMB_BYTES_PER_ELEMENT * elements
    rec["source_fingerprint"] = source_fingerprint("lamb")
    return rec


def ln_traffic_summary(dirs, workload):
    """FETCH_SIZE / WRITE_SIZE per dispatch of the LayerNorm kernels (forward,
    backward apply, and the column sums of its partial rows), scaled by the
    calibration copy, next to each kernel's algorithmic bytes: what it must
    read and write once, its own partial rows included."""
    from paper_2402_15627_amd.inputs import WORKLOADS
    s = WORKLOADS[workload]
    T, H = s.tokens, s.hidden
    e = 2 if s.dtype == "bf16" else 4
    chunks, ng = -(-T // 16), -(-H // 64)
    copy_pick = lambda r: "neg_kernel" in r["Kernel_Name"]  # noqa: E731
    cfetch, _ = _per_dispatch(_counter_rows(dirs[2]), "FETCH_SIZE", copy_pick)
    cwrite, _ = _per_dispatch(_counter_rows(dirs[3]), "WRITE_SIZE", copy_pick)
    ff, wf = COPY_BYTES / 1024 / cfetch, COPY_BYTES / 1024 / cwrite
    kernels = {
        # x read, h written, gamma and beta, the row statistics
        "ln_fwd_wave_bf16": 2 * T * H * e + 2 * H * e + 8 * T,
        # x, dh, dy read, dx written; statistics, the dh GEMM's row terms,
        # gamma, and three fp32 partial rows per 16-row chunk
        "ln_bwd_apply": 4 * T * H * e + 8 * T + 8 * T * ng + H * e + 3 * chunks * H * 4,
        # the partial rows read, dgamma, dbeta, db_out written
        "colsum_rows_f32": 3 * chunks * H * 4 + 3 * H * 4,
    }
    rec = {"step": "ln", "workload": workload, "copy_bytes": COPY_BYTES,
           "copy_fetch_kib": round(cfetch, 1), "copy_write_kib": round(cwrite, 1),
           "fetch_scale": round(ff, 4), "write_scale": round(wf, 4), "kernels": {}}
    total = alg = 0
    for kern, ab in kernels.items():
        pick = lambda r, k=kern: k in r["Kernel_Name"]  # noqa: E731
        fetch, n1 = _per_dispatch(_counter_rows(dirs[0]), "FETCH_SIZE", pick)
        write, n2 = _per_dispatch(_counter_rows(dirs[1]), "WRITE_SIZE", pick)
        tb = int(fetch * 1024 * ff + write * 1024 * wf)
        total += tb
        alg += ab
        rec["kernels"][kern] = {"dispatches": [n1, n2], "fetch_kib": round(fetch, 1),
                                "write_kib": round(write, 1), "traffic_bytes": tb,
                                "algorithmic_bytes": ab, "ratio": round(tb / ab, 3)}
    rec["traffic_bytes"] = total
    rec["algorithmic_bytes"] = alg
    rec["source_fingerprint"] = source_fingerprint("ln")
    return rec


def read_traffic(step, workload):
    """Measured HBM bytes per launch from profiles/, if the sources still match."""
    try:
        with open(traffic_path(step, workload)) as fh:
            text = fh.read()
    except OSError:
        return None
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_fingerprint") != source_fingerprint(step):
        return None
    return rec["traffic_bytes"]


def short_kernel_name(name):
    """Readable kernel name: template arguments spelled out, epilogues named."""
    short = re.sub(r"^void ", "", name).replace("pb::(anonymous namespace)::", "")
    for i, e in enumerate(("StoreF32", "BiasGelu", "BiasResid", "DgeluSplit", "LnGrad")):
        short = short.replace(f"(pb::Epi){i}", e)
    m = re.match(r"_ZN2pb12_GLOBAL__N_1\d+(\w+?)I", short)  # names c++filt leaves
    if m:
        d = re.search(r"Li(\d+)E", short)
        short = m.group(1) + (f"<{d.group(1)}>" if d else "")
    return re.sub(r"\(.*", "", short)[:70]


def trace_summary(d, workload, block="parallel"):
    """Markdown table of a kernel-trace run: one row per (kernel, grid)."""
    from paper_2402_15627_amd.inputs import WORKLOADS
    s = WORKLOADS[workload]
    files = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_trace.csv under {d}")
    groups = {}
    with open(files[0]) as fh:
        for r in csv.DictReader(fh):
            name = demangle(r["Kernel_Name"])
            grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
            dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            groups.setdefault((name, grid), []).append(dur)
    total = sum(sum(v) for v in groups.values())
    rows = []
    for (name, grid), v in groups.items():
        step = gemm_step_of(name, grid, s, block)
        rows.append((sum(v), short_kernel_name(name), grid, step, len(v), sum(v) / len(v), min(v),
                     max(v)))
    rows.sort(reverse=True)
    out = ["| kernel | grid (work-items) | block step | calls | avg us | min us | max us | "
           "% of GPU time |", "|---|---:|---|---:|---:|---:|---:|---:|"]
    for tot, short, grid, step, n, avg, lo, hi in rows:
        out.append(f"| `{short}` | {grid} | {step} | {n} | {avg:.1f} | {lo:.1f} | {hi:.1f} | "
                   f"{100 * tot / total:.1f} |")
    return "\n".join(out)


def cpu_baseline(shape, inputs, min_seconds=10.0, max_steps=6):
    """Time the fp64 oracle (as it stands) on whole forward + backward steps of
    the same workload, repeated until at least min_seconds have elapsed."""
    import numpy as np  # noqa: F401
    from oracle import pblock_oracle as orc
    from paper_2402_15627_amd.inputs import model_flops
    try:
        from threadpoolctl import threadpool_info
        threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:  # threadpoolctl missing: report the host's CPU count
        threads = os.cpu_count()
    cfg = orc.config_from_shape(shape)
    steps, t0 = 0, time.perf_counter()
    while True:
        orc.run_block(cfg, inputs)
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds or steps >= max_steps:
            break
    return {"value": model_flops(shape) * steps / dt / 1e12, "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"{steps} full forward+backward steps of {shape.name} (fp64 numpy, BLAS "
                      f"matmul), same seeded inputs as the GPU run"}


LAMB_BYTES_PER_ELEMENT = 42  # moments pass 16 read + 8 written; update pass 12 read + 4 + 2 written


def device_info():
    """Name, compute units and the driver's maximum shader clock of device 0."""
    import torch
    p = torch.cuda.get_device_properties(0)
    rec = {"name": p.name, "compute_units": p.multi_processor_count,
           "arch": getattr(p, "gcnArchName", None)}
    try:
        import ctypes
        hip = ctypes.CDLL("libamdhip64.so")
        v = ctypes.c_int()
        if hip.hipDeviceGetAttribute(ctypes.byref(v), 5, 0) == 0:  # hipDeviceAttributeClockRate (kHz)
            rec["max_clock_mhz"] = v.value // 1000
    except OSError:
        pass
    return rec


def measured_sclk_mhz(step, seconds=2.0):
    """Median shader clock (MHz) that rocm-smi reports while steps run back to
    back for a few seconds (the chip lowers its clock under sustained matrix
    load); None when rocm-smi is not available."""
    import shutil
    import subprocess
    import threading
    import torch
    exe = shutil.which("rocm-smi") or "/opt/rocm/bin/rocm-smi"
    if not os.path.exists(exe):
        return None
    # Under rocprofv3 every child process loads the profiler's library, which
    # initialises the GPU, so a launcher that re-execs (rocm-smi's
    # "#!/usr/bin/env python3" line) is a forbidden exec: take no samples
    # there.  Elsewhere the script is started by this interpreter directly.
    if any(k.startswith("ROCPROF_") for k in os.environ):
        return None
    with open(exe, "rb") as f:
        head = f.readline()
    cmd = [sys.executable, exe] if head.startswith(b"#!") and b"python" in head else [exe]
    samples = []
    stop = threading.Event()

    def sampler():
        while not stop.is_set():
            try:
                out = subprocess.run(cmd + ["--showclocks", "--json"], capture_output=True,
                                     text=True, timeout=20).stdout
                for card in json.loads(out).values():
                    for k, v in card.items():
                        if k.lower().startswith("sclk"):
                            m = re.search(r"(\d+)\s*mhz", str(v), re.I)
                            if m:
                                samples.append(int(m.group(1)))
            except (OSError, ValueError, subprocess.SubprocessError, AttributeError):
                pass

    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    t0 = time.time()
    while time.time() - t0 < seconds:
        for _ in range(20):
            step()
        torch.cuda.synchronize()
    stop.set()
    th.join(timeout=30)
    return sorted(samples)[len(samples) // 2] if samples else None


def mfma_summary(d, workload):
    """Markdown table of a rocprofv3 --pmc MfmaUtil run: per kernel and grid."""
    from paper_2402_15627_amd.inputs import WORKLOADS
    s = WORKLOADS[workload]
    rows = _counter_rows(d)
    per = {}
    for r in rows:
        if r["Counter_Name"] != "MfmaUtil":
            continue
        key = (demangle(r["Kernel_Name"]), int(r["Grid_Size"]))
        per.setdefault(key, {})[r["Dispatch_Id"]] = float(r["Counter_Value"])
    out = ["| kernel | grid (work-items) | block step | dispatches | MFMA busy % |",
           "|---|---:|---|---:|---:|"]
    for (name, grid), v in sorted(per.items(), key=lambda kv: -sum(kv[1].values()) / len(kv[1])):
        vals = list(v.values())
        out.append(f"| `{short_kernel_name(name)}` | {grid} | {gemm_step_of(name, grid, s)} | {len(vals)} | "
                   f"{sum(vals) / len(vals):.1f} |")
    return "\n".join(out)


def time_lamb(pb, shape, warmup, steps, grads=None):
    """One LAMB step over the parallel block's six parameter tensors (fp32
    master weights, moments and gradients; the bf16 model weights written as
    the copy), timed with events around `steps` consecutive steps."""
    import numpy as np
    import torch
    from paper_2402_15627_amd.inputs import block_param_shapes, make_lamb_state
    shapes = block_param_shapes(shape)
    st = {}
    if grads is None:
        st = make_lamb_state({n: (int(np.prod(sh)),) for n, sh in shapes.items()}, seed=0,
                             w_std=shape.w_std)
    bufs, ts = [], []
    for n, sh in shapes.items():
        numel = int(np.prod(sh))
        if grads is None:
            w, g, m, v = (torch.from_numpy(st[n][k]).cuda() for k in ("w", "g", "m", "v"))
        else:
            w = torch.randn(numel, device="cuda") * shape.w_std
            g = grads[n].reshape(-1)
            m = torch.zeros(numel, device="cuda")
            v = torch.zeros(numel, device="cuda")
        copy = torch.empty(numel, dtype=torch.bfloat16, device="cuda")
        bufs.append((w, g, m, v, copy))
        ts.append(pb.lamb_tensor(w, g, m, v, copy, 0.0 if n.startswith(("b_", "gamma", "beta"))
                                 else 0.01))
    ws = torch.empty(pb.pblock_lamb_workspace_bytes(ts), dtype=torch.uint8, device="cuda")
    elements = sum(int(np.prod(sh)) for sh in shapes.values())

    def step(t):
        pb.pblock_lamb_step(pb.lamb_config(1e-3, step=t), ts, pb.PB_BF16, None, ws)

    for i in range(warmup):
        step(i + 1)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for i in range(steps):
        step(warmup + i + 1)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    nbytes = LAMB_BYTES_PER_ELEMENT * elements
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"ms": round(ms, 4), "elements": elements, "bytes_per_step": nbytes,
            "achieved_gbs": round(gbs, 1), "peak_gbs": PEAK_HBM_GBS,
            "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": read_traffic("lamb", shape.name)}


def time_ag(pb, shape, dev, warmup, steps, tp=8, n_comm=2):
    """The in-projection pipelined with the all-gather of its input over tp
    ranks (shards copied on comm streams, GEMM launches over groups of
    shards as they land), against the GEMM alone and the copies followed by
    one GEMM.  Rank 0's own shard is in place; the other tp - 1 are copied.
    Each variant is timed with events on the compute stream."""
    import torch
    T, H = shape.tokens, shape.hidden
    cfg = pb.config_from_shape(shape)
    act = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    src = (torch.randn(T, H, device="cuda")).to(act)
    h = torch.empty_like(src)
    z = torch.empty(T, shape.n_in, dtype=act, device="cuda")
    c = torch.empty(T, shape.k_out, dtype=act, device="cuda")
    rows = T // tp
    stream = torch.cuda.Stream()
    comm = [torch.cuda.Stream() for _ in range(n_comm)]
    ctx = pb.TpContext(tp)
    out = {}

    def timed(per, in_place):
        nws = pb.pblock_ag_in_proj_workspace_bytes(cfg, tp, per)
        ws = torch.empty(nws, dtype=torch.uint8, device="cuda") if nws else None
        # this rank's own shard is its local LayerNorm output, already in
        # place in h; the others arrive from the peers (all in place: no
        # copies at all)
        h.copy_(src)
        shards = [h[j * rows:(j + 1) * rows] if (in_place or j == 0) else
                  src[j * rows:(j + 1) * rows] for j in range(tp)]
        torch.cuda.synchronize()

        def call():
            pb.pblock_ag_in_proj(cfg, tp, 0, shards, h, dev["w_in"], dev["b_in"], z, c, per, ws,
                                 stream, comm, ctx)
        for _ in range(warmup):
            call()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        return round(e0.elapsed_time(e1) / steps, 4)

    out["gemm_only_ms"] = timed(tp, True)
    out["copies_then_gemm_ms"] = timed(tp, False)
    for per in (1, 2, 4):
        out[f"pipelined_{per}_shards_per_launch_ms"] = timed(per, False)
    ctx.close()
    return {"tp": tp, "n_comm": n_comm, "shard_bytes": rows * H * src.element_size(), **out}


def time_rs(pb, shape, dev, warmup, steps, tp=8, n_comm=2):
    """The out-projection's partial sums pipelined with their reduce-scatter
    over tp ranks (row chunks sent on comm streams as their GEMM launch
    finishes), against the GEMM alone and one GEMM followed by the copies;
    and the receiving side's sum of tp chunks.  Rank 0's own chunk stays in
    place; the other tp - 1 are copied.  Events on the compute stream."""
    import torch
    T, H = shape.tokens, shape.hidden
    cfg = pb.config_from_shape(shape)
    act = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    c = torch.randn(T, shape.k_out, device="cuda").to(act)
    partial = torch.empty(T, H, dtype=act, device="cuda")
    rows = T // tp
    recv = torch.empty(tp, rows, H, dtype=act, device="cuda")
    stream = torch.cuda.Stream()
    comm = [torch.cuda.Stream() for _ in range(n_comm)]
    ctx = pb.TpContext(tp)
    out = {}

    def timed(call):
        for _ in range(warmup):
            call()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        return round(e0.elapsed_time(e1) / steps, 4)

    def send(per, in_place):
        nws = pb.pblock_rs_out_proj_workspace_bytes(cfg, tp, per)
        ws = torch.empty(nws, dtype=torch.uint8, device="cuda") if nws else None
        # this rank's own chunk stays in place (it is reduced locally); the
        # others go to the peers' receive buffers (all in place: no copies)
        dst = [partial[j * rows:(j + 1) * rows] if (in_place or j == 0) else recv[j]
               for j in range(tp)]
        return lambda: pb.pblock_rs_out_proj(cfg, tp, 0, c, dev["w_out"], partial, dst, per, ws,
                                             stream, comm, ctx)

    out["gemm_only_ms"] = timed(send(tp, True))
    out["gemm_then_copies_ms"] = timed(send(tp, False))
    for per in (1, 2, 4):
        out[f"pipelined_{per}_shards_per_launch_ms"] = timed(send(per, False))
    y = torch.empty(rows, H, dtype=act, device="cuda")
    parts = [recv[q] for q in range(tp)]
    ms = timed(lambda: pb.pblock_rs_reduce(cfg, tp, parts, dev["x"].reshape(T, H)[:rows], dev["b_out"], y,
                                           stream))
    nbytes = (tp + 2) * rows * H * partial.element_size()
    out["reduce_ms"] = ms
    out["reduce_gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
    ctx.close()
    return {"tp": tp, "n_comm": n_comm, "chunk_bytes": rows * H * partial.element_size(), **out}


def time_bwd_overlap(pb, shape, dev, warmup, steps, tp=8, n_comm=2):
    """The backward pass's mirror of the two overlaps: the dC GEMM pipelined
    with the all-gather of dy (pblock_ag_dc) and the dh GEMM pipelined with
    the reduce-scatter of its partial sums (pblock_rs_dh), each against the
    GEMM alone and the unpipelined order, timed like time_ag / time_rs."""
    import torch
    T, H = shape.tokens, shape.hidden
    cfg = pb.config_from_shape(shape)
    act = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    rows = T // tp
    src = torch.randn(T, H, device="cuda").to(act)
    dy = torch.empty_like(src)
    z = torch.randn(T, shape.n_in, device="cuda").to(act)
    d_o = torch.empty(T, shape.attn_width, dtype=act, device="cuda")
    dz = torch.randn(T, shape.n_in, device="cuda").to(act)
    w_in_t = dev["w_in"]  # [N_in, H]: dh = dZ W_in
    partial = torch.empty(T, H, dtype=act, device="cuda")
    recv = torch.empty(tp, rows, H, dtype=act, device="cuda")
    stream = torch.cuda.Stream()
    comm = [torch.cuda.Stream() for _ in range(n_comm)]
    ctx = pb.TpContext(tp)

    def timed(call):
        for _ in range(warmup):
            call()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        return round(e0.elapsed_time(e1) / steps, 4)

    def ag(per, in_place):
        nws = pb.pblock_ag_dc_workspace_bytes(cfg, tp, per)
        ws = torch.empty(nws, dtype=torch.uint8, device="cuda") if nws else None
        dy.copy_(src)
        shards = [dy[j * rows:(j + 1) * rows] if (in_place or j == 0) else
                  src[j * rows:(j + 1) * rows] for j in range(tp)]
        torch.cuda.synchronize()
        return lambda: pb.pblock_ag_dc(cfg, tp, 0, shards, dy, dev["w_out"], z, d_o, dz, per, ws,
                                       stream, comm, ctx)

    def rs(per, in_place):
        nws = pb.pblock_rs_dh_workspace_bytes(cfg, tp, per)
        ws = torch.empty(nws, dtype=torch.uint8, device="cuda") if nws else None
        dst = [partial[j * rows:(j + 1) * rows] if (in_place or j == 0) else recv[j]
               for j in range(tp)]
        return lambda: pb.pblock_rs_dh(cfg, tp, 0, dz, w_in_t, partial, dst, per, ws, stream,
                                       comm, ctx)

    out = {"tp": tp, "n_comm": n_comm, "shard_bytes": rows * H * src.element_size()}
    agd = {"gemm_only_ms": timed(ag(tp, True)), "copies_then_gemm_ms": timed(ag(tp, False))}
    rsd = {"gemm_only_ms": timed(rs(tp, True)), "gemm_then_copies_ms": timed(rs(tp, False))}
    for per in (1, 2, 4):
        agd[f"pipelined_{per}_shards_per_launch_ms"] = timed(ag(per, False))
        rsd[f"pipelined_{per}_shards_per_launch_ms"] = timed(rs(per, False))
    ctx.close()
    return {**out, "ag_dc": agd, "rs_dh": rsd}


def time_serial(pb, shape, warmup, steps, parallel_ms, flops):
    """The standard block (two LayerNorms, four projections; the same model
    FLOPs) on the same workload and kernels, timed like the parallel block:
    forward + backward, inputs resident, events around the whole loop."""
    import torch
    from paper_2402_15627_amd.inputs import make_inputs
    act = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    dev = {k: torch.from_numpy(v).to(act).cuda()
           for k, v in make_inputs(shape, seed=0, serial=True).items()}
    blk = pb.SerialBlock(pb.config_from_shape(shape), dev)
    for _ in range(warmup):
        blk.forward()
        blk.backward()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(steps):
        blk.forward()
        blk.backward()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    return {"ms_per_step": round(ms, 4), "value": round(flops / (ms * 1e-3) / 1e12, 2),
            "unit": "TFLOP/s",
            "parallel_speedup": round(ms / parallel_ms, 4) if parallel_ms else None}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="175b_tp8_share")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip timing the CPU oracle")
    ap.add_argument("--block", choices=("parallel", "serial", "lamb"), default="parallel",
                    help="serial: time only the standard two-LayerNorm block; lamb: only the "
                         "LAMB step over the block's parameters (for profiling)")
    ap.add_argument("--no-serial", action="store_true",
                    help="skip timing the serial (two-LayerNorm) block for comparison")
    ap.add_argument("--no-ag", action="store_true",
                    help="skip timing the all-gather and reduce-scatter pipelines")
    ap.add_argument("--no-lamb", action="store_true",
                    help="skip timing the LAMB step over the block's parameters")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run the counter calibration copy and exit")
    ap.add_argument("--traffic-summary", nargs=4, metavar="DIR",
                    help="rocprofv3 --pmc output dirs: FETCH_SIZE and WRITE_SIZE of the bench, "
                         "then of --copy-calibration; writes profiles/<step>_<workload>_traffic.md")
    ap.add_argument("--traffic-step", default="dh+dw_in",
                    help="a GEMM step, or lamb (the LAMB step's two streaming kernels)")
    ap.add_argument("--trace-summary", metavar="DIR",
                    help="print a markdown table of a rocprofv3 --kernel-trace output dir")
    ap.add_argument("--mfma-summary", metavar="DIR",
                    help="print a markdown table of a rocprofv3 --pmc MfmaUtil output dir")
    ap.add_argument("--command", default="", help="command line recorded with a summary")
    args = ap.parse_args()
    if args.trace_summary:
        print(trace_summary(args.trace_summary, args.workload, args.block))
        return
    if args.mfma_summary:
        print(mfma_summary(args.mfma_summary, args.workload))
        return
    if args.traffic_summary:
        if args.traffic_step == "lamb":
            rec = lamb_traffic_summary(args.traffic_summary, args.workload)
            what = "the LAMB step's moments and update kernels"
        elif args.traffic_step == "ln":
            rec = ln_traffic_summary(args.traffic_summary, args.workload)
            what = "the LayerNorm forward, backward and column-sum kernels"
        else:
            rec = traffic_summary(args.traffic_summary, args.workload, args.traffic_step)
            what = f"the {args.traffic_step} GEMM"
        path = traffic_path(args.traffic_step, args.workload)
        with open(path, "w") as fh:
            fh.write(f"# HBM traffic of {what}, {args.workload}\n\n"
                     "FETCH_SIZE and WRITE_SIZE (KiB per dispatch, rocprofv3 --pmc, one counter "
                     "per run) of the matching launches, each scaled by "
                     f"{COPY_BYTES} bytes over what the same counter reads for one dispatch of "
                     "the calibration copy (a read-once, write-once elementwise kernel).\n\n"
                     f"Commands (repository root on the GPU host):\n\n```\n{args.command}\n```\n\n"
                     f"```json\n{json.dumps(rec, indent=1)}\n```\n")
        print(json.dumps(rec))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the block's kernels run on a single MI355X and this "
              "build has no multi-GPU path (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np  # noqa: F401
    import torch

    if args.copy_calibration:
        # a plain elementwise pass: reads COPY_BYTES once and writes them once
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": COPY_BYTES}))
        return

    from paper_2402_15627_amd import pblock as pb
    from paper_2402_15627_amd.inputs import WORKLOADS, make_inputs, model_flops

    shape = WORKLOADS[args.workload]
    pb.load_library()
    if args.block == "lamb":
        rec = time_lamb(pb, shape, args.warmup, args.steps)
        print(json.dumps({"block": "lamb", "workload": shape.name, "steps": args.steps,
                          "warmup": args.warmup, **rec}), flush=True)
        return
    if args.block == "serial":
        flops = model_flops(shape)
        rec = time_serial(pb, shape, args.warmup, args.steps, None, flops)
        print(json.dumps({"block": "serial", "workload": shape.name, "steps": args.steps,
                          "warmup": args.warmup, **rec}), flush=True)
        return
    inputs = make_inputs(shape, seed=0)
    act = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    dev = {k: torch.from_numpy(v).to(act).cuda() for k, v in inputs.items()}
    blk = pb.ParallelBlock(pb.config_from_shape(shape), dev)
    flops = model_flops(shape)
    work = step_work(shape)
    names = pb.STEPS

    def step(ev=None):
        blk.forward(step_ev=ev)
        blk.backward(step_ev=ev)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    def new_event():
        ev = torch.cuda.Event(enable_timing=True)
        ev.record()  # creates the underlying hipEvent_t
        return ev

    # Pass 1: events around every step, to find where the time goes.
    K = args.steps
    evb = [[new_event() for _ in names] for _ in range(K)]
    eve = [[new_event() for _ in names] for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        step(pb.step_events([e.cuda_event for e in evb[i]], [e.cuda_event for e in eve[i]]))
    torch.cuda.synchronize()
    step_ms = {n: sum(evb[i][j].elapsed_time(eve[i][j]) for i in range(K)) / K
               for j, n in enumerate(names)}
    dominant = max(step_ms, key=step_ms.get)
    dj = names.index(dominant)
    # a GEMM the library folded into its partner's launch must take no time
    for a, b in paired_steps(shape).items():
        if step_ms[b] > 0.05 * step_ms[a]:
            raise SystemExit(f"step {b} took {step_ms[b]:.3f} ms: not launched with {a} as "
                             "paired_steps assumes")

    # Pass 2 (the timed region): K steps; events only around the dominant kernel.
    db = [new_event() for _ in range(K)]
    de = [new_event() for _ in range(K)]
    t_start, t_end = new_event(), new_event()
    torch.cuda.synchronize()
    t_start.record()
    dom_ev = []
    for i in range(K):
        hb = [0] * len(names)
        he = [0] * len(names)
        hb[dj] = db[i].cuda_event
        he[dj] = de[i].cuda_event
        dom_ev.append(pb.step_events(hb, he))
    for i in range(K):
        step(dom_ev[i])
    t_end.record()
    torch.cuda.synchronize()
    ms = t_start.elapsed_time(t_end) / K
    dom_ms = sum(db[i].elapsed_time(de[i]) for i in range(K)) / K

    # Per-step spread: a separate pass with events around every whole step.
    sb = [new_event() for _ in range(K)]
    se = [new_event() for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        sb[i].record()
        step()
        se[i].record()
    torch.cuda.synchronize()
    per_step = sorted(sb[i].elapsed_time(se[i]) for i in range(K))
    sclk = measured_sclk_mhz(step)

    value = flops / (ms * 1e-3) / 1e12
    kind, amount = work[dominant]
    if kind == "mfma":
        achieved = amount / (dom_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": read_traffic(launch_key(dominant, shape), shape.name),
                "kernel": launch_key(dominant, shape), "flops_per_launch": amount,
                "avg_ms": round(dom_ms, 4)}
    else:
        achieved = amount / (dom_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                "traffic": read_traffic(dominant, shape.name),
                "kernel": dominant, "bytes_per_launch": amount, "avg_ms": round(dom_ms, 4)}

    steps_out = {}
    for n in names:
        k, a = work[n]
        # a step whose work is done inside another one (db_out: summed with
        # the LN backward's column sums) reports no rate
        rate = a / (step_ms[n] * 1e-3) / (1e12 if k == "mfma" else 1e9) if a else None
        steps_out[n] = {"ms": round(step_ms[n], 4),
                        ("tflops" if k == "mfma" else "gbs"): None if rate is None else round(rate, 1)}

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "pct_of_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if shape.dtype == "bf16" else "f32",
        "data": "synthetic (seeded normal draws, shapes of the paper's Table 1 175B model)",
        "config": {"workload": shape.name, "batch": shape.batch, "seq": shape.seq,
                   "hidden": shape.hidden, "heads": shape.heads, "head_dim": shape.head_dim,
                   "ffn": shape.ffn, "window": shape.window, "flops_per_step": flops,
                   "parallelism": "none: one GPU holding one tensor-parallel rank's share"},
        "roofline": roof,
        "step_ms": {"min": round(per_step[0], 4), "median": round(per_step[K // 2], 4),
                    "max": round(per_step[-1], 4)},
        "device": device_info(),
        "clock": {"sclk_mhz_median": sclk,
                  "pct_of_peak_at_measured_clock":
                      round(100 * value / (PEAK_BF16_TFLOPS * sclk / 2400.0), 2) if sclk else None},
        "steps_breakdown": steps_out,
    }
    if not args.no_serial:
        out["serial_block"] = time_serial(pb, shape, args.warmup, K, ms, flops)
    if not args.no_ag:
        out["ag_in_proj"] = time_ag(pb, shape, dev, 2, 5)
        out["rs_out_proj"] = time_rs(pb, shape, dev, 2, 5)
        out["bwd_overlap"] = time_bwd_overlap(pb, shape, dev, 2, 5)
    if not args.no_lamb:
        names = ("w_in", "b_in", "w_out", "b_out", "gamma", "beta")
        gmap = dict(zip(names, (blk.grads[k] for k in ("dw_in", "db_in", "dw_out", "db_out",
                                                         "dgamma", "dbeta"))))
        out["lamb_step"] = time_lamb(pb, shape, args.warmup, K, gmap)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, inputs)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

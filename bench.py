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
  cpu_baseline  the fp64 CPU oracle timed on this host on one full step.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CUs x 2.4 GHz x 4096 dense bf16 FLOP/clk/CU
PEAK_HBM_GBS = 8000.0
METRIC = "parallel-block fwd+bwd TFLOP/s and % of MI355X bf16 MFMA peak"


def step_work(s):
    """Algorithmic work of each pb_step: ("mfma", FLOPs) or ("hbm", bytes)."""
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
        "db_out": ("hbm", T * H * e + 4 * H),
        "attn_bwd": ("mfma", 8 * s.batch * A * P),
        "dh": ("mfma", 2 * T * n_in * H),
        "dw_in": ("mfma", 2 * n_in * H * T),
        "db_in": ("hbm", T * n_in * e + 4 * n_in),
        "ln_bwd": ("hbm", 3 * T * H * e + 4 * T * H + 8 * T + 8 * H),
    }


def cpu_baseline(shape, inputs):
    """Time the fp64 oracle (as it stands) on one full forward + backward step."""
    import numpy as np  # noqa: F401
    from oracle import pblock_oracle as orc
    from paper_2402_15627_amd.inputs import model_flops
    try:
        from threadpoolctl import threadpool_info
        threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:  # threadpoolctl missing: report the host's CPU count
        threads = os.cpu_count()
    cfg = orc.config_from_shape(shape)
    t0 = time.perf_counter()
    orc.run_block(cfg, inputs)
    dt = time.perf_counter() - t0
    return {"value": model_flops(shape) / dt / 1e12, "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"one full forward+backward step of {shape.name} (fp64 numpy, "
                      f"BLAS matmul), same seeded inputs as the GPU run"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="175b_tp8_share")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip timing the CPU oracle")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the block's kernels run on a single MI355X and this "
              "build has no multi-GPU path (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np  # noqa: F401
    import torch

    from paper_2402_15627_amd import pblock as pb
    from paper_2402_15627_amd.inputs import WORKLOADS, make_inputs, model_flops

    shape = WORKLOADS[args.workload]
    pb.load_library()
    inputs = make_inputs(shape, seed=0)
    act = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    dev = {k: torch.from_numpy(v).to(act).cuda() for k, v in inputs.items()}
    blk = pb.ParallelBlock(pb.config_from_shape(shape), dev)
    flops = model_flops(shape)
    work = step_work(shape)
    names = pb.STEPS

    def step():
        blk.forward()
        blk.backward()

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
        pb.pblock_set_step_events([e.cuda_event for e in evb[i]], [e.cuda_event for e in eve[i]])
        step()
    pb.pblock_set_step_events(None, None)
    torch.cuda.synchronize()
    step_ms = {n: sum(evb[i][j].elapsed_time(eve[i][j]) for i in range(K)) / K
               for j, n in enumerate(names)}
    dominant = max(step_ms, key=step_ms.get)
    dj = names.index(dominant)

    # Pass 2 (the timed region): K steps; events only around the dominant kernel.
    db = [new_event() for _ in range(K)]
    de = [new_event() for _ in range(K)]
    t_start, t_end = new_event(), new_event()
    torch.cuda.synchronize()
    t_start.record()
    for i in range(K):
        hb = [0] * len(names)
        he = [0] * len(names)
        hb[dj] = db[i].cuda_event
        he[dj] = de[i].cuda_event
        pb.pblock_set_step_events(hb, he)
        step()
    t_end.record()
    torch.cuda.synchronize()
    pb.pblock_set_step_events(None, None)
    ms = t_start.elapsed_time(t_end) / K
    dom_ms = sum(db[i].elapsed_time(de[i]) for i in range(K)) / K

    value = flops / (ms * 1e-3) / 1e12
    kind, amount = work[dominant]
    if kind == "mfma":
        achieved = amount / (dom_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": None, "kernel": dominant, "flops_per_launch": amount,
                "avg_ms": round(dom_ms, 4)}
    else:
        achieved = amount / (dom_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
                "kernel": dominant, "bytes_per_launch": amount, "avg_ms": round(dom_ms, 4)}

    steps_out = {}
    for n in names:
        k, a = work[n]
        rate = a / (step_ms[n] * 1e-3) / (1e12 if k == "mfma" else 1e9)
        steps_out[n] = {"ms": round(step_ms[n], 4),
                        ("tflops" if k == "mfma" else "gbs"): round(rate, 1)}

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
        "steps_breakdown": steps_out,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, inputs)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

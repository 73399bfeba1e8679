"""Helpers shared by the GPU parity tests: run the block through the C ABI and
the oracle on the same seeded inputs and compare them normwise."""
from __future__ import annotations

import numpy as np

from oracle import pblock_oracle as orc
from paper_2402_15627_amd.inputs import BlockShape, make_inputs

GRAD_NAMES = ("dx", "dgamma", "dbeta", "dw_in", "db_in", "dw_out", "db_out")
OUT_NAMES = ("y",) + GRAD_NAMES

# Normwise tolerance, max|gpu - ref| / max|ref| per tensor: bf16 storage with
# fp32 accumulation, and the all-fp32 path.
TOL = {"bf16": 2e-2, "f32": 1e-5}


def normwise(a, ref) -> float:
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max()
    return float(np.abs(a - ref).max() / (scale if scale > 0 else 1.0))


def to_device(shape: BlockShape, inp: dict):
    import torch
    act = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(act).cuda() for k, v in inp.items()}


def run_gpu(shape: BlockShape, inp: dict, with_block=False):
    """Forward + backward through the C ABI; returns float64 numpy arrays."""
    import torch
    from paper_2402_15627_amd import pblock as pb
    blk = pb.ParallelBlock(pb.config_from_shape(shape), to_device(shape, inp))
    blk.forward()
    blk.backward()
    torch.cuda.synchronize()
    out = {"y": blk.y.float().cpu().numpy().astype(np.float64)}
    for n in GRAD_NAMES:
        out[n] = blk.grads[n].float().cpu().numpy().astype(np.float64)
    return (out, blk) if with_block else out


def run_oracle(shape: BlockShape, inp: dict, weight_rows=None):
    return orc.run_block(orc.config_from_shape(shape), inp, weight_rows)


def compare(shape: BlockShape, gpu: dict, ref: dict, names=OUT_NAMES):
    errs = {n: normwise(gpu[n], ref[n]) for n in names}
    tol = TOL[shape.dtype]
    bad = {n: e for n, e in errs.items() if not e <= tol}
    return errs, bad


def case(shape: BlockShape, seed=0):
    return make_inputs(shape, seed)

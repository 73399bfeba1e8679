"""GPU checks of the backward's terms that are formed inside GEMM launches
rather than by launches of their own:

  delta = rowsum(dO O) per (batch row, head, token), formed in the dC GEMM's
          epilogue (the attention backward's row terms, Section 3.3 FA-2);
  db_in = sum over tokens of dZ, formed from the A fragments of dW_in's first
          tile column in the dh + dW_in launch.

Each is compared with the same sum over the block's own stored operands (the
stash's O, the workspace's dO and dZ) in fp64: only fp32 summation order
separates them (delta 1e-5 of max |delta|, db_in 1e-4 of max |db_in|).
Shapes take the fused paths (bf16, every GEMM K a multiple of 64, heads of 64
or 128 columns aligned to 128) with several batch rows (the epilogue maps a
token row m to its batch row and position), and db_in is also checked against
the fp64 oracle, as the block parity tests do.  A ragged token count, where
the GEMMs run apart and separate launches form both terms, is checked the same
way.
"""
import sys

import numpy as np
import pytest

from paper_2402_15627_amd.inputs import BlockShape, make_inputs
from tests.parity_util import normwise, run_oracle, to_device

pytestmark = pytest.mark.gpu

SHAPES = [
    BlockShape("fused_d64_b2", 2, 320, 256, 4, 64, 512, 100, "bf16"),
    BlockShape("fused_d128_b3", 3, 128, 384, 2, 128, 640, 64, "bf16"),
    BlockShape("apart_ragged", 1, 333, 256, 2, 128, 512, 50, "bf16"),
]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("s", SHAPES, ids=[s.name for s in SHAPES])
def test_delta_and_db_in_match_their_sums(s):
    import torch
    from paper_2402_15627_amd import pblock as pb
    _say(f"[gpu] fused backward terms {s.name}")
    cfg = pb.config_from_shape(s)
    fused = pb.pblock_backward_pairs(cfg) == (True, True)
    assert fused == (s.name != "apart_ragged")
    inp = make_inputs(s, seed=3)
    blk = pb.ParallelBlock(cfg, to_device(s, inp))
    blk.forward()
    blk.backward()
    torch.cuda.synchronize()
    A, d, S = s.attn_width, s.head_dim, s.seq
    c = blk.saved_view("c").double()[:, :A]
    d_o = blk.workspace_view("d_o").double()
    dz = blk.workspace_view("dz").double()
    delta = blk.workspace_view("delta").double()
    ref = (d_o * c).reshape(s.batch, S, s.heads, d).sum(dim=3).permute(0, 2, 1)
    ed = float((delta - ref).abs().max() / ref.abs().max())
    db_in = blk.grads["db_in"].double()
    eb = float((db_in - dz.sum(dim=0)).abs().max() / dz.sum(dim=0).abs().max())
    eo = normwise(db_in.cpu().numpy(), run_oracle(s, inp)["db_in"])
    _say(f"      delta {ed:.2e}  db_in vs sum(dZ) {eb:.2e}  db_in vs oracle {eo:.2e}")
    assert ed <= 1e-5 and eb <= 1e-4 and eo <= 2e-2

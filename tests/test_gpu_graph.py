"""GPU check that a training step of the block (forward, then backward) can
be captured into a HIP graph and replayed: the calls launch kernels only on
the caller's stream (no allocation, synchronisation or memset; the
backward's queue heads are zeroed by a kernel), so a graph of one step,
replayed, must give the bits of the same step run eagerly.  Each replay
follows eager work on the outputs (they are overwritten with garbage) and a
synchronisation, and every replay is checked; the parallel block and the
serial (standard pre-LN) block alike.
"""
import sys

import pytest

from paper_2402_15627_amd.inputs import BlockShape, make_inputs
from tests.parity_util import to_device

pytestmark = pytest.mark.gpu

SHAPES = [
    BlockShape("graph_1k", 1, 1024, 2048, 16, 128, 4096, 1024, "bf16"),
    BlockShape("graph_edges_f32", 2, 96, 256, 4, 64, 320, 40, "f32"),
]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("block", ["parallel", "serial"])
@pytest.mark.parametrize("s", SHAPES, ids=[s.name for s in SHAPES])
def test_block_step_replays_in_a_graph(s, block):
    import torch
    from paper_2402_15627_amd import pblock as pb
    _say(f"[gpu] graph capture of forward + backward {s.name} {block}")
    cls = pb.ParallelBlock if block == "parallel" else pb.SerialBlock
    inp = make_inputs(s, seed=11, serial=block == "serial")
    blk = cls(pb.config_from_shape(s), to_device(s, inp))
    outs = [blk.y] + list(blk.grads.values())

    def snapshot():
        return [t.clone() for t in outs]

    blk.forward()
    blk.backward()
    torch.cuda.synchronize()
    ref = snapshot()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # a run on the capture stream's kind before capturing
        blk.forward()
        blk.backward()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        blk.forward()
        blk.backward()
    torch.cuda.synchronize()
    for r in range(3):
        for t in outs:
            t.fill_(float("nan") if t.dtype.is_floating_point else 7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        bad = [i for i, (a, b) in enumerate(zip(ref, outs)) if not torch.equal(a, b)]
        assert not bad, f"replay {r}: outputs {bad} differ from the eager step"

"""GPU checks of the persistent shared GEMM launches of the backward passes
(dC + dW_out and dh + dW_in; in the serial block each weight gradient with
the GEMM before it).

Their workgroups take tiles from per-XCD queues whose heads live in the
backward workspace: each call zeroes them before its first shared launch,
and the launches leave them non-zero.  So the results must be the same bits
whatever the workspace held before the call (all-zero or all-ones bytes),
and again when a second backward call reuses the workspace; and since the
order in which workgroups take tiles changes from run to run, bitwise
equality across these runs also shows that no result depends on the
schedule.  Shapes have several hundred tiles per launch (every XCD queue
non-empty, so workgroups take tiles from other XCDs' queues at the end) and
a ragged one with tiles at the matrix edges.  Two blocks whose backward
calls run at the same time on two streams (separate workspaces, so separate
queue heads; the two persistent launches share the CUs) must give the bits
each gives alone.
"""
import sys

import pytest

from paper_2402_15627_amd.inputs import BlockShape, make_inputs
from tests.parity_util import to_device

pytestmark = pytest.mark.gpu

SHAPES = [
    BlockShape("persist_1k", 1, 1024, 2048, 16, 128, 4096, 1024, "bf16"),
    BlockShape("persist_b2_edges", 2, 384, 1280, 10, 64, 2560, 200, "bf16"),
]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _grads(blk):
    return {n: g.clone() for n, g in blk.grads.items()}


def _run(cls, s, inp, fill):
    import torch
    from paper_2402_15627_amd import pblock as pb
    blk = cls(pb.config_from_shape(s), to_device(s, inp))
    blk.ws.fill_(fill)
    blk.forward()
    blk.backward()
    torch.cuda.synchronize()
    first = _grads(blk)
    blk.backward()  # the queue heads are as the first call left them
    torch.cuda.synchronize()
    return first, _grads(blk)


def _same(a, b):
    import torch
    return [n for n in a if not torch.equal(a[n], b[n])]


@pytest.mark.parametrize("s", SHAPES, ids=[s.name for s in SHAPES])
def test_parallel_backward_is_independent_of_queue_state(s):
    import torch  # noqa: F401  (before the library: one HIP runtime)
    from paper_2402_15627_amd import pblock as pb
    _say(f"[gpu] persistent shared launches, parallel block {s.name}")
    cfg = pb.config_from_shape(s)
    assert pb.pblock_backward_pairs(cfg) == (True, True)
    inp = make_inputs(s, seed=5)
    a1, a2 = _run(pb.ParallelBlock, s, inp, 0)
    b1, b2 = _run(pb.ParallelBlock, s, inp, 255)
    bad = _same(a1, a2) + _same(a1, b1) + _same(a1, b2)
    assert not bad, f"gradients differ between runs: {bad}"


@pytest.mark.parametrize("s", SHAPES[:1], ids=[s.name for s in SHAPES[:1]])
def test_serial_backward_is_independent_of_queue_state(s):
    import torch  # noqa: F401  (before the library: one HIP runtime)
    from paper_2402_15627_amd import pblock as pb
    _say(f"[gpu] persistent shared launches, serial block {s.name}")
    cfg = pb.config_from_shape(s)
    assert all(pb.pblock_backward_pairs(cfg, "serial"))
    inp = make_inputs(s, seed=6, serial=True)
    a1, a2 = _run(pb.SerialBlock, s, inp, 0)
    b1, b2 = _run(pb.SerialBlock, s, inp, 255)
    bad = _same(a1, a2) + _same(a1, b1) + _same(a1, b2)
    assert not bad, f"gradients differ between runs: {bad}"


def test_backward_calls_on_two_streams_at_once():
    import torch
    from paper_2402_15627_amd import pblock as pb
    s = SHAPES[0]
    _say(f"[gpu] two concurrent backward calls {s.name}")
    cfg = pb.config_from_shape(s)
    blocks = [pb.ParallelBlock(cfg, to_device(s, make_inputs(s, seed=seed))) for seed in (7, 8)]
    alone = []
    for blk in blocks:
        blk.forward()
        blk.backward()
        torch.cuda.synchronize()
        alone.append(_grads(blk))
    streams = [torch.cuda.Stream() for _ in blocks]
    for st in streams:
        st.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        for blk, st in zip(blocks, streams):
            blk.backward(stream=st)
    torch.cuda.synchronize()
    for i, blk in enumerate(blocks):
        bad = _same(alone[i], _grads(blk))
        assert not bad, f"block {i}: gradients differ when run beside another call: {bad}"

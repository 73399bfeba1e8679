"""GPU parity of the backward pass's dh GEMM pipelined with the
reduce-scatter of its partial sums (pblock_rs_dh on every simulated rank,
then pblock_rs_reduce without residual or bias on every receiving rank), the
mirror of the forward's all-gather (Section 3.2, tensor/sequence-parallel
overlap), against the definition in fp64:

    dh = sum over ranks r of dZ_r W_in,r

(dZ_r [T, N_in_r], W_in,r [N_in_r, H]: rank r's own columns of the
in-projection output gradient and rows of its weight).  The tp ranks run one
after another on the one GPU, each sending its chunks into the receive
buffers of the others.  bf16: the partials travel in bf16, so dh is within
2e-2 normwise; fp32 within 1e-5.  The partials, the placement of every chunk
and independence from the launch grouping and comm streams are checked too.
"""
import sys

import numpy as np
import pytest

from paper_2402_15627_amd.inputs import WORKLOADS, BlockShape, round_to_bf16
from tests.parity_util import normwise

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class Ranks:
    """Seeded inputs of tp ranks: each its own dZ_r [T, N_in] and W_r
    [N_in, H]."""

    def __init__(self, s, tp, seed):
        import torch
        rng = np.random.default_rng(seed)
        T, H, N = s.tokens, s.hidden, s.n_in
        rnd = round_to_bf16 if s.dtype == "bf16" else (lambda a: a)
        self.s, self.tp = s, tp
        self.dz = [rnd(rng.standard_normal((T, N)).astype(np.float32)) for _ in range(tp)]
        self.w = [rnd((s.w_std * rng.standard_normal((N, H))).astype(np.float32))
                  for _ in range(tp)]
        self.act = torch.bfloat16 if s.dtype == "bf16" else torch.float32
        dev = lambda a: torch.from_numpy(a).to(self.act).cuda()  # noqa: E731
        self.d_dz = [dev(a) for a in self.dz]
        self.d_w = [dev(a) for a in self.w]

    def reference(self, rows=None):
        sel = (lambda a: a) if rows is None else (lambda a: a[rows])
        parts = [sel(z).astype(np.float64) @ w.astype(np.float64) for z, w in zip(self.dz, self.w)]
        return sum(parts), parts

    def run(self, per=1, n_comm=2, in_place=()):
        import torch
        from paper_2402_15627_amd import pblock as pb
        s, tp = self.s, self.tp
        T, H = s.tokens, s.hidden
        rows = T // tp
        cfg = pb.config_from_shape(s)
        act = self.act
        recv = [torch.zeros((tp, rows, H), dtype=act, device="cuda") for _ in range(tp)]
        partial = [torch.zeros((T, H), dtype=act, device="cuda") for _ in range(tp)]
        nws = pb.pblock_rs_dh_workspace_bytes(cfg, tp, per)
        ws = torch.empty(nws, dtype=torch.uint8, device="cuda") if nws else None
        stream = torch.cuda.Stream()
        comm = [torch.cuda.Stream() for _ in range(n_comm)]
        stream.wait_stream(torch.cuda.current_stream())
        with pb.TpContext(tp) as ctx:
            for r in range(tp):
                dst = [partial[r][j * rows:(j + 1) * rows] if (r in in_place and j == r)
                       else recv[j][r] for j in range(tp)]
                pb.pblock_rs_dh(cfg, tp, r, self.d_dz[r], self.d_w[r], partial[r], dst, per, ws,
                                stream, comm, ctx)
        dh = torch.empty((T, H), dtype=act, device="cuda")
        for j in range(tp):
            parts = [partial[j][j * rows:(j + 1) * rows] if (j in in_place and q == j)
                     else recv[j][q] for q in range(tp)]
            pb.pblock_rs_reduce(cfg, tp, parts, None, None, dh[j * rows:(j + 1) * rows], stream)
        torch.cuda.synchronize()
        for j in range(tp):
            for q in range(tp):
                if not (q in in_place and q == j):
                    assert torch.equal(recv[j][q], partial[q][j * rows:(j + 1) * rows]), (j, q)
        return dh.float().cpu().numpy(), [p.float().cpu().numpy() for p in partial]


SMALL = BlockShape("rsdh_small", 1, 600, 512, 4, 64, 1000, 64, "bf16", w_std=0.05)
SMALL_F32 = BlockShape("rsdh_small_f32", 2, 48, 128, 2, 64, 96, 16, "f32", w_std=0.05)


@pytest.mark.parametrize("tp,n_comm,in_place,per", [
    (1, 1, (0,), 1), (4, 1, (), 1), (4, 2, (2,), 1), (8, 3, (5,), 1), (8, 8, (), 3),
    (6, 4, (0, 1, 2, 3, 4, 5), 2), (8, 2, (), 8), (5, 2, (), 4),
])
def test_rs_dh_matches_definition(tp, n_comm, in_place, per):
    _say(f"[gpu] rs dh tp={tp} n_comm={n_comm} in_place={in_place} per={per}")
    ranks = Ranks(SMALL, tp, seed=tp)
    dh, parts = ranks.run(per, n_comm, in_place)
    dh_ref, p_ref = ranks.reference()
    e = normwise(dh, dh_ref)
    ep = max(normwise(p, r) for p, r in zip(parts, p_ref))
    _say(f"      dh {e:.2e}  partials {ep:.2e}")
    assert e <= 2e-2 and ep <= 2e-2


def test_rs_dh_fp32_matches_definition():
    _say("[gpu] rs dh fp32")
    ranks = Ranks(SMALL_F32, 4, seed=3)
    dh, _ = ranks.run(2, 2)
    dh_ref, _ = ranks.reference()
    assert normwise(dh, dh_ref) <= 1e-5


def test_rs_dh_does_not_depend_on_the_schedule():
    _say("[gpu] rs dh schedule independence")
    ranks = Ranks(SMALL, 4, seed=9)
    d0, _ = ranks.run(4, 1)
    for per, n_comm in ((1, 2), (2, 4), (3, 1)):
        d, _ = ranks.run(per, n_comm)
        assert normwise(d, d0) <= 1e-2, (per, n_comm)


def test_rs_dh_full_size_175b_share():
    """The 175B share (T = 2048, N_in = 10752, H = 12288) over 8 ranks: sampled
    rows of the reduced dh against the definition."""
    s = WORKLOADS["175b_tp8_share"]
    _say(f"[gpu] rs dh full size {s.name}")
    ranks = Ranks(s, 8, seed=0)
    dh, _ = ranks.run(2, 2)
    rows = np.array([0, 1, 255, 256, 767, 768, 1000, 2047])
    dh_ref, _ = ranks.reference(rows)
    e = normwise(dh[rows], dh_ref)
    _say(f"      dh {e:.2e}")
    assert e <= 2e-2

"""GPU parity of the out-projection pipelined with the reduce-scatter of its
partial sums (pblock_rs_out_proj on every simulated rank, then
pblock_rs_reduce on every receiving rank), against the definition of the
row-parallel out-projection of Eq. 2 in fp64:

    y = x + b_out + sum over ranks r of C_r W_out,r^T

(C_r, W_out,r: rank r's own columns of the out-projection input and weight).
The tp ranks run one after another on the one GPU, each sending its chunks
into the receive buffers of the others.  bf16: the partials travel in bf16,
so y is within 2e-2 normwise (each partial is rounded once, the sum once);
fp32 within 1e-5.  The partial sums themselves, the placement of every chunk,
and independence from the launch grouping, the number of comm streams and
chunks already in place (<= 1e-2 between runs: only the K-split of a few
tiles may differ) are checked too; shapes cover chunks that straddle GEMM
tile rows, groups that wrap past the last rank, and the 175B share.
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
    """Seeded inputs of tp ranks: each its own C_r [T, K_out] and W_r [H,
    K_out]; x [T, H] and b_out [H] are shared."""

    def __init__(self, s, tp, seed):
        import torch
        rng = np.random.default_rng(seed)
        T, H, K = s.tokens, s.hidden, s.k_out
        rnd = round_to_bf16 if s.dtype == "bf16" else (lambda a: a)
        self.s, self.tp = s, tp
        self.x = rnd(rng.standard_normal((T, H)).astype(np.float32))
        self.b = rnd((s.w_std * rng.standard_normal(H)).astype(np.float32))
        self.c = [rnd(rng.standard_normal((T, K)).astype(np.float32)) for _ in range(tp)]
        self.w = [rnd((s.w_std * rng.standard_normal((H, K))).astype(np.float32))
                  for _ in range(tp)]
        self.act = torch.bfloat16 if s.dtype == "bf16" else torch.float32
        dev = lambda a: torch.from_numpy(a).to(self.act).cuda()  # noqa: E731
        self.d_x, self.d_b = dev(self.x), dev(self.b)
        self.d_c = [dev(a) for a in self.c]
        self.d_w = [dev(a) for a in self.w]

    def reference(self, rows=None):
        """fp64 y and the partials P_r (rows: a subset of token rows)."""
        sel = (lambda a: a) if rows is None else (lambda a: a[rows])
        parts = [sel(c).astype(np.float64) @ w.astype(np.float64).T
                 for c, w in zip(self.c, self.w)]
        y = sel(self.x).astype(np.float64) + self.b.astype(np.float64) + sum(parts)
        return y, parts

    def run(self, per=1, n_comm=2, in_place=(), fill=None):
        """Every rank's sending side, then every rank's reduce.  Returns y
        [T, H] and the partials (numpy, fp32)."""
        import torch
        from paper_2402_15627_amd import pblock as pb
        s, tp = self.s, self.tp
        T, H = s.tokens, s.hidden
        rows = T // tp
        cfg = pb.config_from_shape(s)
        act = self.act
        recv = [torch.zeros((tp, rows, H), dtype=act, device="cuda") for _ in range(tp)]
        partial = [torch.zeros((T, H), dtype=act, device="cuda") for _ in range(tp)]
        if fill is not None:
            for t in recv + partial:
                t.fill_(fill)
        nws = pb.pblock_rs_out_proj_workspace_bytes(cfg, tp, per)
        ws = torch.empty(nws, dtype=torch.uint8, device="cuda") if nws else None
        stream = torch.cuda.Stream()
        comm = [torch.cuda.Stream() for _ in range(n_comm)]
        stream.wait_stream(torch.cuda.current_stream())
        ctx = pb.TpContext(tp)
        for r in range(tp):
            dst = [partial[r][j * rows:(j + 1) * rows] if (r in in_place and j == r)
                   else recv[j][r] for j in range(tp)]
            pb.pblock_rs_out_proj(cfg, tp, r, self.d_c[r], self.d_w[r], partial[r], dst, per,
                                  ws, stream, comm, ctx)
        ctx.close()
        y = torch.empty((T, H), dtype=act, device="cuda")
        for j in range(tp):
            parts = [partial[j][j * rows:(j + 1) * rows] if (j in in_place and q == j)
                     else recv[j][q] for q in range(tp)]
            pb.pblock_rs_reduce(cfg, tp, parts, self.d_x[j * rows:(j + 1) * rows], self.d_b,
                                y[j * rows:(j + 1) * rows], stream)
        torch.cuda.synchronize()
        # every chunk landed where it was sent
        for j in range(tp):
            for q in range(tp):
                if not (q in in_place and q == j):
                    assert torch.equal(recv[j][q], partial[q][j * rows:(j + 1) * rows]), (j, q)
        return y.float().cpu().numpy(), [p.float().cpu().numpy() for p in partial]


SMALL = BlockShape("rs_small", 1, 600, 512, 4, 64, 1000, 64, "bf16", w_std=0.05)
SMALL_F32 = BlockShape("rs_small_f32", 2, 48, 128, 2, 64, 96, 16, "f32", w_std=0.05)


@pytest.mark.parametrize("tp,n_comm,in_place,per", [
    (1, 1, (), 1), (1, 1, (0,), 1), (4, 1, (), 1), (4, 2, (2,), 1), (8, 3, (5,), 1),
    (8, 8, (), 3), (6, 4, (0, 1, 2, 3, 4, 5), 2), (8, 2, (), 8), (5, 2, (), 4),
])
def test_rs_out_proj_matches_definition(tp, n_comm, in_place, per):
    _say(f"[gpu] rs out-proj tp={tp} n_comm={n_comm} in_place={in_place} per={per}")
    ranks = Ranks(SMALL, tp, seed=tp)
    y, parts = ranks.run(per, n_comm, in_place)
    y_ref, p_ref = ranks.reference()
    ey = normwise(y, y_ref)
    ep = max(normwise(p, r) for p, r in zip(parts, p_ref))
    _say(f"      y {ey:.2e}  partials {ep:.2e}")
    assert ey <= 2e-2 and ep <= 2e-2


def test_rs_out_proj_fp32_matches_definition():
    _say("[gpu] rs out-proj fp32")
    ranks = Ranks(SMALL_F32, 4, seed=7)
    y, parts = ranks.run(per=2, n_comm=2)
    y_ref, p_ref = ranks.reference()
    assert normwise(y, y_ref) <= 1e-5
    assert max(normwise(p, r) for p, r in zip(parts, p_ref)) <= 1e-5


def test_rs_out_proj_does_not_depend_on_the_schedule():
    _say("[gpu] rs out-proj schedule independence")
    ranks = Ranks(SMALL, 8, seed=2)
    y0, _ = ranks.run(per=8, n_comm=1)
    for per, n_comm, in_place in ((1, 1, ()), (2, 2, (1, 6)), (3, 4, ()), (4, 8, (0,))):
        y, _ = ranks.run(per, n_comm, in_place)
        assert normwise(y, y0) <= 1e-2, (per, n_comm, in_place)


def test_rs_out_proj_overwrites_stale_buffers():
    """Receive and partial buffers hold old values before each run; every
    element of the result must come from this run."""
    _say("[gpu] rs out-proj stale-data check")
    ranks = Ranks(SMALL, 4, seed=3)
    y_ref, _ = ranks.reference()
    for fill in (0.0, 1.0, -2.0):
        y, _ = ranks.run(per=1, n_comm=2, fill=fill)
        assert normwise(y, y_ref) <= 2e-2, fill


def test_rs_reduce_sums_in_rank_order_exactly():
    """The receiving side alone on integer-valued parts (every sum exact in
    fp32 and bf16): y must equal x + b + sum of parts bit for bit."""
    import torch
    from paper_2402_15627_amd import pblock as pb
    _say("[gpu] rs reduce exact sums")
    s = SMALL
    tp, rows, H = 8, SMALL.tokens // 8, SMALL.hidden
    rng = np.random.default_rng(9)
    parts = [rng.integers(-8, 9, (rows, H)).astype(np.float32) for _ in range(tp)]
    x = rng.integers(-8, 9, (rows, H)).astype(np.float32)
    b = rng.integers(-8, 9, H).astype(np.float32)
    want = x + b + sum(parts)
    cuda = lambda a: torch.from_numpy(a).to(torch.bfloat16).cuda()  # noqa: E731
    y = torch.empty((rows, H), dtype=torch.bfloat16, device="cuda")
    pb.pblock_rs_reduce(pb.config_from_shape(s), tp, [cuda(p) for p in parts], cuda(x), cuda(b),
                        y)
    torch.cuda.synchronize()
    assert np.array_equal(y.float().cpu().numpy(), want)


def test_rs_out_proj_full_size_175b_share():
    """One rank of the 175B share (T = 2048, H = 12288, K_out = 7680) over 8
    ranks: its partial on sampled rows against the definition, and the chunks
    it sent in place."""
    import torch
    from paper_2402_15627_amd import pblock as pb
    s = WORKLOADS["175b_tp8_share"]
    _say(f"[gpu] rs out-proj full size {s.name}")
    tp, rank = 8, 3
    rng = np.random.default_rng(0)
    T, H, K = s.tokens, s.hidden, s.k_out
    c = round_to_bf16(rng.standard_normal((T, K)).astype(np.float32))
    w = round_to_bf16((s.w_std * rng.standard_normal((H, K))).astype(np.float32))
    d_c = torch.from_numpy(c).to(torch.bfloat16).cuda()
    d_w = torch.from_numpy(w).to(torch.bfloat16).cuda()
    rows = T // tp
    partial = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
    dst = [torch.empty((rows, H), dtype=torch.bfloat16, device="cuda") for _ in range(tp)]
    cfg = pb.config_from_shape(s)
    nws = pb.pblock_rs_out_proj_workspace_bytes(cfg, tp, 2)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda") if nws else None
    stream = torch.cuda.Stream()
    comm = [torch.cuda.Stream() for _ in range(2)]
    stream.wait_stream(torch.cuda.current_stream())
    with pb.TpContext(tp) as ctx:
        pb.pblock_rs_out_proj(cfg, tp, rank, d_c, d_w, partial, dst, 2, ws, stream, comm, ctx)
    torch.cuda.synchronize()
    sample = np.array([0, 1, 255, 256, 767, 768, 1000, 2047])
    ref = c[sample].astype(np.float64) @ w.astype(np.float64).T
    got = partial.float().cpu().numpy()
    e = normwise(got[sample], ref)
    _say(f"      partial {e:.2e}")
    assert e <= 2e-2
    for j in range(tp):
        assert torch.equal(dst[j], partial[j * rows:(j + 1) * rows]), j

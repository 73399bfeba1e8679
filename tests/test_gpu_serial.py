"""GPU parity of the serial (standard pre-LN) block: the HIP library's serial
entry points, called through the C ABI, against the fp64 serial oracle on the
same seeded inputs, per tensor normwise (bf16 <= 2e-2, fp32 <= 1e-5).

The shapes span several GEMM and attention tiles with ragged tails, a
one-token sequence, both GeLU forms, and a GEMM whose last partial wave of
tiles is split along K.
"""
import sys

import numpy as np
import pytest

from oracle import serial_oracle as so
from oracle.pblock_oracle import config_from_shape
from paper_2402_15627_amd.inputs import WORKLOADS, BlockShape, make_inputs
from tests.parity_util import TOL, normwise, to_device

pytestmark = pytest.mark.gpu

NAMES = ("y", "dx", "dgamma1", "dbeta1", "dgamma2", "dbeta2", "dw_in", "db_in", "dw_out", "db_o",
         "db_down")


def shape(name, **kw):
    base = dict(batch=1, seq=128, hidden=256, heads=4, head_dim=64, ffn=1024, window=64,
                dtype="bf16", w_std=0.02, gamma_std=0.1, beta_std=0.1)
    base.update(kw)
    return BlockShape(name, **base)


CASES = [
    WORKLOADS["tiny_f32"],
    shape("f32_ragged", batch=2, seq=150, hidden=264, heads=2, ffn=136, window=37, dtype="f32"),
    shape("bf16_ragged_d64", batch=2, seq=200, hidden=320, heads=3, ffn=264, window=70),
    shape("bf16_d128_ragged_erf", batch=3, seq=161, hidden=392, heads=3, head_dim=128, ffn=200,
          window=129, gelu_tanh=False),
    shape("bf16_seq1", batch=4, seq=1, hidden=64, heads=1, head_dim=64, ffn=64, window=8),
    # up-projection: 3 x 86 = 258 output tiles, ragged in M and N: 256 whole
    # tiles plus 2 tail tiles split along K; the other GEMMs have small grids
    shape("bf16_split_tail", batch=1, seq=520, hidden=512, heads=4, head_dim=128, ffn=21904,
          window=100),
]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(s, inp):
    import torch
    from paper_2402_15627_amd import pblock as pb
    blk = pb.SerialBlock(pb.config_from_shape(s), to_device(s, inp))
    blk.forward()
    blk.backward()
    torch.cuda.synchronize()
    out = {"y": blk.y.float().cpu().numpy().astype(np.float64)}
    for n, g in blk.grads.items():
        out[n] = g.float().cpu().numpy().astype(np.float64)
    return out, blk


@pytest.mark.parametrize("s", CASES, ids=[c.name for c in CASES])
def test_serial_block_matches_oracle(s):
    _say(f"[gpu] serial parity {s}")
    inp = make_inputs(s, seed=0, serial=True)
    gpu, _ = run_gpu(s, inp)
    ref = so.run_serial(config_from_shape(s), inp)
    errs = {n: normwise(gpu[n], ref[n]) for n in NAMES}
    _say("      normwise errors: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    bad = {n: e for n, e in errs.items() if not e <= TOL[s.dtype]}
    assert not bad, f"{s.name}: over tolerance {TOL[s.dtype]}: {bad}"


@pytest.mark.parametrize("s", [CASES[1], CASES[3]], ids=lambda c: c.name)
def test_serial_stash_matches_oracle(s):
    """Each forward step on its own, as kept in the stash: both LayerNorms,
    the projections, the attention output and its log-sum-exp, and x1."""
    _say(f"[gpu] serial stash parity {s.name}")
    inp = make_inputs(s, seed=1, serial=True)
    _, blk = run_gpu(s, inp)
    cfg = config_from_shape(s)
    f = {k: np.asarray(v, np.float64) for k, v in inp.items()}
    _, c = so.serial_forward(cfg, *[f[n] for n in so.PARAMS])
    T = s.tokens
    ref = {
        "h1": c["h1"].reshape(T, -1),
        "z": np.concatenate([c["qkv"], c["u"]], -1).reshape(T, -1),
        "c": np.concatenate([c["o"], c["g"]], -1).reshape(T, -1),
        "mean1": c["mean1"].reshape(T), "rstd1": c["rstd1"].reshape(T),
        "lse": c["lse"],
        "x1": c["x1"].reshape(T, -1),
        "h2": c["h2"].reshape(T, -1),
        "mean2": c["mean2"].reshape(T), "rstd2": c["rstd2"].reshape(T),
    }
    for name, r in ref.items():
        e = normwise(blk.saved_view(name).float().cpu().numpy(), r)
        _say(f"      {name}: {e:.2e}")
        assert e <= TOL[s.dtype], (name, e)


def test_serial_split_and_unsplit_agree():
    """Without the optional partial-tile workspace every GEMM runs unsplit;
    both runs match the oracle and each other to rounding."""
    import torch
    from paper_2402_15627_amd import pblock as pb
    s = CASES[-1]
    _say(f"[gpu] serial split vs unsplit {s.name}")
    inp = make_inputs(s, seed=4, serial=True)
    blk = pb.SerialBlock(pb.config_from_shape(s), to_device(s, inp))
    assert blk.ws_fwd is not None
    y_split = blk.forward().float().cpu().numpy()
    t = blk.t
    y2 = torch.empty_like(blk.y)
    pb.pblock_serial_forward(blk.cfg, t["x"], t["gamma1"], t["beta1"], t["gamma2"], t["beta2"],
                             t["w_in"], t["b_in"], t["w_out"], t["b_o"], t["b_down"], y2,
                             blk.saved, None)
    torch.cuda.synchronize()
    ref = so.run_serial(config_from_shape(s), inp)["y"].reshape(y_split.shape)
    y_unsplit = y2.float().cpu().numpy()
    assert normwise(y_split, ref) <= 2e-2
    assert normwise(y_unsplit, ref) <= 2e-2
    assert normwise(y_split, y_unsplit) <= 1e-2


def test_serial_forward_without_stash_matches():
    """saved = NULL keeps the stash at the start of the workspace; y is the
    same as with a caller stash, bit for bit."""
    import torch
    from paper_2402_15627_amd import pblock as pb
    s = CASES[2]
    _say(f"[gpu] serial forward without stash {s.name}")
    inp = make_inputs(s, seed=5, serial=True)
    blk = pb.SerialBlock(pb.config_from_shape(s), to_device(s, inp))
    y_ref = blk.forward().clone()
    ws = torch.empty(pb.pblock_serial_workspace_bytes(blk.cfg, pb.WS_FORWARD_WITH_STASH),
                     dtype=torch.uint8, device="cuda")
    y2 = torch.empty_like(blk.y)
    t = blk.t
    pb.pblock_serial_forward(blk.cfg, t["x"], t["gamma1"], t["beta1"], t["gamma2"], t["beta2"],
                             t["w_in"], t["b_in"], t["w_out"], t["b_o"], t["b_down"], y2, None,
                             ws)
    torch.cuda.synchronize()
    assert torch.equal(y_ref, y2)

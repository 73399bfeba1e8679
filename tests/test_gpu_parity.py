"""GPU parity: the HIP library, called through its C ABI, against the fp64
CPU oracle on the same seeded inputs, element by element (normwise per
tensor: bf16 storage with fp32 accumulation <= 2e-2, the fp32 path <= 1e-5).

Sizes here are ones the oracle finishes in seconds but that still span several
GEMM tiles (256 x 256) and attention tiles (128 queries x 64 keys), with
ragged tails in every dimension.
"""
import sys

import numpy as np
import pytest

from paper_2402_15627_amd.inputs import WORKLOADS, BlockShape
from tests.parity_util import TOL, compare, case, normwise, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


def shape(name, **kw):
    base = dict(batch=1, seq=128, hidden=256, heads=4, head_dim=64, ffn=1024, window=64,
                dtype="bf16", w_std=0.02)
    base.update(kw)
    return BlockShape(name, **base)


CASES = [
    WORKLOADS["tiny_f32"],
    WORKLOADS["tiny_f32"].with_(name="tiny_f32_erf", gelu_tanh=False),
    shape("f32_ragged", batch=2, seq=150, hidden=264, heads=2, ffn=136, window=37, dtype="f32"),
    shape("f32_d128_full", batch=1, seq=90, hidden=128, heads=2, head_dim=128, ffn=64,
          window=1000, dtype="f32"),
    shape("bf16_tiny_shape", dtype="bf16"),
    shape("bf16_ragged_d64", batch=2, seq=200, hidden=320, heads=3, ffn=264, window=70),
    shape("bf16_ragged_d64_w1", batch=2, seq=200, hidden=320, heads=3, ffn=264, window=1),
    shape("bf16_ragged_d64_wfull", batch=1, seq=333, hidden=320, heads=3, ffn=264, window=5000),
    shape("bf16_d128", batch=1, seq=384, hidden=512, heads=2, head_dim=128, ffn=512, window=100),
    shape("bf16_d128_ragged_erf", batch=3, seq=161, hidden=392, heads=3, head_dim=128, ffn=200,
          window=129, gelu_tanh=False),
    shape("bf16_seq1", batch=4, seq=1, hidden=64, heads=1, head_dim=64, ffn=64, window=8),
    # head_dim 96 (Table 1's 175B heads): 12-chunk rows, 6 K-steps, 3 output blocks
    shape("bf16_d96_ragged", batch=2, seq=203, hidden=384, heads=3, head_dim=96, ffn=232,
          window=71),
    shape("bf16_d96_full_erf", batch=1, seq=300, hidden=192, heads=2, head_dim=96, ffn=128,
          window=4096, gelu_tanh=False),
    shape("f32_d96", batch=1, seq=77, hidden=96, heads=1, head_dim=96, ffn=64, window=20,
          dtype="f32"),
    shape("bf16_w_edge_tiles", batch=1, seq=512, hidden=256, heads=2, head_dim=128, ffn=256,
          window=64),
    # in-projection: 3 x 86 = 258 output tiles, ragged in M and N: 256 whole
    # tiles plus 2 tail tiles split 8 ways along K
    shape("bf16_split_tail", batch=1, seq=520, hidden=512, heads=4, head_dim=128, ffn=20360,
          window=100),
    # a hidden size that takes the one-wave-per-row LayerNorm forward (2048 =
    # 4 x 512 columns), with 262 rows: the last workgroup holds two rows
    shape("bf16_h2048_wave_ln", batch=2, seq=131, hidden=2048, heads=4, head_dim=128, ffn=512,
          window=90),
]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("s", CASES, ids=[c.name for c in CASES])
def test_block_matches_oracle(s):
    _say(f"[gpu] block parity {s}")
    inp = case(s, seed=0)
    gpu = run_gpu(s, inp)
    ref = run_oracle(s, inp)
    errs, bad = compare(s, gpu, ref)
    _say(f"      normwise errors: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    assert not bad, f"{s.name}: over tolerance {TOL[s.dtype]}: {bad}"


@pytest.mark.parametrize("s", [CASES[0], CASES[5], CASES[9]], ids=lambda c: c.name)
def test_forward_stash_matches_oracle(s):
    """Each forward step on its own: LN output, in-projection (+GeLU),
    attention output and its log-sum-exp, as kept in the stash."""
    _say(f"[gpu] stash parity {s.name}")
    inp = case(s, seed=1)
    _, blk = run_gpu(s, inp, with_block=True)
    from oracle import pblock_oracle as orc
    cfg = orc.config_from_shape(s)
    f = {k: np.asarray(v, np.float64) for k, v in inp.items()}
    _, cache = orc.block_forward(cfg, f["x"], f["gamma"], f["beta"], f["w_in"], f["b_in"],
                                 f["w_out"], f["b_out"])
    T = s.tokens
    ref = {
        "h": cache["h"].reshape(T, -1),
        "z": cache["z"].reshape(T, -1),
        "c": np.concatenate([cache["o"], cache["g"]], -1).reshape(T, -1),
        "mean": cache["mean"].reshape(T),
        "rstd": cache["rstd"].reshape(T),
        "lse": cache["lse"],
    }
    tol = TOL[s.dtype]
    for name, r in ref.items():
        g = blk.saved_view(name).float().cpu().numpy()
        e = normwise(g, r)
        _say(f"      {name}: {e:.2e}")
        assert e <= tol, (name, e)


def test_split_and_unsplit_gemms_agree():
    """Without the optional partial-tile workspace the GEMMs run unsplit; both
    runs must match the oracle, and each other to rounding."""
    import torch
    from paper_2402_15627_amd import pblock as pb
    s = [c for c in CASES if c.name == "bf16_split_tail"][0]
    _say(f"[gpu] split vs unsplit {s.name}")
    inp = case(s, seed=4)
    from tests.parity_util import to_device
    blk = pb.ParallelBlock(pb.config_from_shape(s), to_device(s, inp))
    assert blk.ws_fwd is not None  # this shape does split
    y_split = blk.forward().float().cpu().numpy()
    t = blk.t
    y2 = torch.empty_like(blk.y)
    pb.pblock_forward(blk.cfg, t["x"], t["gamma"], t["beta"], t["w_in"], t["b_in"], t["w_out"],
                      t["b_out"], y2, blk.saved, None)
    torch.cuda.synchronize()
    y_unsplit = y2.float().cpu().numpy()
    ref = run_oracle(s, inp)["y"].reshape(y_split.shape)
    assert normwise(y_split, ref) <= 2e-2
    assert normwise(y_unsplit, ref) <= 2e-2
    assert normwise(y_split, y_unsplit) <= 1e-2


def test_causal_locality_is_bitwise():
    """Changing x at token t may change y only at tokens t .. t+W-1 of the same
    batch row; every other output row must be bitwise identical."""
    import torch
    s = shape("locality", batch=2, seq=300, hidden=256, heads=2, head_dim=128, ffn=256, window=70)
    _say(f"[gpu] locality {s}")
    inp = case(s, seed=2)
    y0 = run_gpu(s, inp)["y"]
    for t in (0, 63, 64, 127, 128, 200, 299):
        inp2 = {k: v.copy() for k, v in inp.items()}
        inp2["x"][1, t, 5] += 0.75
        y1 = run_gpu(s, inp2)["y"]
        assert np.array_equal(y1[0], y0[0]), "other batch row changed"
        changed = np.any(y1[1] != y0[1], axis=-1)
        expect = np.zeros(s.seq, bool)
        expect[t:t + s.window] = True
        assert not np.any(changed & ~expect), (t, np.nonzero(changed & ~expect)[0][:10])
        assert changed[t]


def test_repeat_runs_are_bitwise_identical():
    s = shape("determinism", batch=1, seq=256, hidden=256, heads=2, head_dim=128, ffn=256,
              window=100)
    _say(f"[gpu] determinism {s.name}")
    inp = case(s, seed=3)
    a = run_gpu(s, inp)
    b = run_gpu(s, inp)
    for n in a:
        assert np.array_equal(a[n], b[n]), n


@pytest.mark.parametrize("W", [1, 5, 64, 65, 200, 10000])
@pytest.mark.parametrize("d", [64, 96, 128])
def test_swattn_entry_points_match_oracle(W, d):
    """pblock_swattn_forward / _backward on q, k, v with padded rows, with the
    split workspace (B * heads is small, so long blocks are split) and
    without it; both must match the oracle and agree with each other."""
    import torch
    from oracle import pblock_oracle as orc
    from paper_2402_15627_amd import pblock as pb
    B, S, nh = 2, 1193, 3
    _say(f"[gpu] swattn B={B} S={S} heads={nh} d={d} W={W}")
    rng = np.random.default_rng(W * 7 + d)
    A = nh * d
    ld = A + 8  # padded rows
    q, k, v, do = (rng.standard_normal((B, S, ld)).astype(np.float32) for _ in range(4))
    from paper_2402_15627_amd.inputs import round_to_bf16
    q, k, v, do = (round_to_bf16(a) for a in (q, k, v, do))
    dev = lambda a: torch.from_numpy(a).to(torch.bfloat16).cuda()
    cfg = pb.make_config(B, S, 64, nh, d, 64, W, "bf16")
    u8 = dict(dtype=torch.uint8, device="cuda")
    runs = {}
    for split in (True, False):
        o = torch.zeros((B, S, ld), dtype=torch.bfloat16, device="cuda")
        lse = torch.zeros((B, nh, S), dtype=torch.float32, device="cuda")
        nf = pb.pblock_swattn_workspace_bytes(cfg, pb.ATTN_WS_FORWARD)
        wsf = torch.empty(nf, **u8) if split and nf else None
        pb.pblock_swattn_forward(cfg, dev(q), dev(k), dev(v), ld, o, ld, lse, wsf)
        dq, dk, dv = (torch.zeros((B, S, ld), dtype=torch.bfloat16, device="cuda")
                      for _ in range(3))
        mode = pb.ATTN_WS_BACKWARD if split else pb.ATTN_WS_BACKWARD_MIN
        ws = torch.empty(pb.pblock_swattn_workspace_bytes(cfg, mode), **u8)
        pb.pblock_swattn_backward(cfg, dev(q), dev(k), dev(v), ld, o, ld, dev(do), ld, lse, dq,
                                  dk, dv, ld, ws)
        torch.cuda.synchronize()
        runs[split] = {n: t.float().cpu().numpy()
                       for n, t in (("o", o), ("lse", lse), ("dq", dq), ("dk", dk), ("dv", dv))}
        # padding columns are never written
        assert torch.count_nonzero(o[..., A:]) == 0
        assert torch.count_nonzero(dq[..., A:]) == 0
    got = runs[True]
    for b in range(B):
        for h in range(nh):
            sl = slice(h * d, (h + 1) * d)
            qq, kk, vv, gg = (a[b, :, sl].astype(np.float64) for a in (q, k, v, do))
            o_ref, l_ref = orc.swa_head_forward(qq, kk, vv, W)
            dq_r, dk_r, dv_r = orc.swa_head_backward(qq, kk, vv, gg, W)
            assert normwise(got["o"][b, :, sl], o_ref) <= 2e-2
            np.testing.assert_allclose(got["lse"][b, h], l_ref, rtol=0, atol=2e-2)
            for n, r in (("dq", dq_r), ("dk", dk_r), ("dv", dv_r)):
                e = normwise(got[n][b, :, sl], r)
                assert e <= 2e-2, (b, h, n, e)
    for n in got:
        e = normwise(runs[False][n], got[n])
        assert e <= 1e-2, (n, e)

"""GPU parity of the fused LAMB step: pblock_lamb_step, called through the C
ABI, against the fp64 LAMB oracle on the same seeded optimizer state.

fp32 arithmetic on both moments and the update: m and v within 1e-6
normwise; the updated weights within 1e-5 of the largest change plus the
rounding of the stored fp32 weights (2^-23 of the largest weight: the change
is ~1e-3 of the weight, so rounding w' to fp32 alone moves it by ~1e-4 of the
change); trust ratios within 1e-5 relative; the bf16 and fp32 copies equal
the updated fp32 weights rounded (bit-exact).  Shapes are the parallel block's parameters plus ragged
and empty tensors, and the full parameter set of the 175B share.
"""
import sys

import numpy as np
import pytest

from oracle import lamb_oracle as lo
from paper_2402_15627_amd.inputs import WORKLOADS, block_param_shapes, make_lamb_state
from tests.parity_util import normwise

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def decay_of(name):
    return 0.0 if name.startswith(("b_", "gamma", "beta", "bias")) else 0.01


def run_gpu(state, cfg, copy_dtype="bf16", with_ratio=True):
    """One step on the GPU.  Returns per-tensor numpy w, m, v, copy and the
    ratios."""
    import torch
    from paper_2402_15627_amd import pblock as pb
    names = list(state)
    dev = {n: {k: torch.from_numpy(a.reshape(-1).copy()).cuda() for k, a in st.items()}
           for n, st in state.items()}
    cdt = torch.bfloat16 if copy_dtype == "bf16" else torch.float32
    copies = {n: torch.empty(dev[n]["w"].numel(), dtype=cdt, device="cuda") for n in names}
    ts = [pb.lamb_tensor(dev[n]["w"], dev[n]["g"], dev[n]["m"], dev[n]["v"], copies[n],
                         decay_of(n)) for n in names]
    ws = torch.empty(pb.pblock_lamb_workspace_bytes(ts), dtype=torch.uint8, device="cuda")
    ratio = torch.full((len(names),), -1.0, device="cuda") if with_ratio else None
    pcfg = pb.lamb_config(cfg.lr, cfg.beta1, cfg.beta2, cfg.eps, cfg.step, cfg.bias_correction,
                          cfg.grad_scale)
    pb.pblock_lamb_step(pcfg, ts, pb.PB_BF16 if copy_dtype == "bf16" else pb.PB_F32, ratio, ws)
    torch.cuda.synchronize()
    out = {n: {"w": dev[n]["w"].cpu().numpy(), "m": dev[n]["m"].cpu().numpy(),
               "v": dev[n]["v"].cpu().numpy(), "copy": copies[n].cpu(),
               "w_t": dev[n]["w"].cpu()} for n in names}
    return out, (ratio.cpu().numpy() if with_ratio else None)


def run_oracle(state, cfg):
    names = list(state)
    w, m, v, r = lo.lamb_step(cfg, [state[n]["w"].reshape(-1) for n in names],
                              [state[n]["g"].reshape(-1) for n in names],
                              [state[n]["m"].reshape(-1) for n in names],
                              [state[n]["v"].reshape(-1) for n in names],
                              [decay_of(n) for n in names])
    return {n: {"w": w[i], "m": m[i], "v": v[i]} for i, n in enumerate(names)}, r


def check(state, gpu, ratios, ref, ref_ratios, copy_dtype="bf16"):
    import torch
    for i, n in enumerate(state):
        w0 = state[n]["w"].reshape(-1).astype(np.float64)
        if w0.size == 0:
            continue
        dw = ref[n]["w"] - w0
        err = np.abs(gpu[n]["w"] - ref[n]["w"]).max()
        bound = 1e-5 * np.abs(dw).max() + 2.0 ** -23 * np.abs(ref[n]["w"]).max()
        e_dw = normwise(gpu[n]["w"] - w0, dw)
        e_m = normwise(gpu[n]["m"], ref[n]["m"])
        e_v = normwise(gpu[n]["v"], ref[n]["v"])
        _say(f"      {n} [{w0.size}]: dw={e_dw:.2e} m={e_m:.2e} v={e_v:.2e} "
             f"ratio {ratios[i]:.6g} vs {ref_ratios[i]:.6g}")
        assert err <= bound and e_m <= 1e-6 and e_v <= 1e-6, (n, err, bound)
        assert abs(ratios[i] - ref_ratios[i]) <= 1e-5 * abs(ref_ratios[i]), n
        want = gpu[n]["w_t"].to(torch.bfloat16 if copy_dtype == "bf16" else torch.float32)
        assert torch.equal(gpu[n]["copy"], want), n


SMALL = dict(block_param_shapes(WORKLOADS["tiny_f32"]),
             ragged=(8192 * 2 + 13,), one=(1,), three=(3,), gamma_only=(4,), empty=(0,))


@pytest.mark.parametrize("copy_dtype", ["bf16", "f32"])
@pytest.mark.parametrize("bc,t,gs", [(True, 1, 1.0), (True, 9, 0.25), (False, 3, 1.0)])
def test_lamb_step_matches_oracle(copy_dtype, bc, t, gs):
    _say(f"[gpu] lamb step copy={copy_dtype} bias_correction={bc} step={t} grad_scale={gs}")
    state = make_lamb_state(SMALL, seed=t)
    cfg = lo.LambConfig(lr=2e-3, beta1=0.9, beta2=0.999, eps=1e-6, step=t, bias_correction=bc,
                        grad_scale=gs)
    gpu, ratios = run_gpu(state, cfg, copy_dtype)
    ref, rr = run_oracle(state, cfg)
    check(state, gpu, ratios, ref, rr, copy_dtype)
    # the empty tensor reports ratio 1
    assert ratios[list(SMALL).index("empty")] == 1.0


def test_lamb_three_steps_match_oracle():
    _say("[gpu] lamb three steps")
    state = make_lamb_state(SMALL, seed=11)
    ref_state = {n: {k: a.astype(np.float64) for k, a in st.items()} for n, st in state.items()}
    cur = {n: dict(st) for n, st in state.items()}
    rng = np.random.default_rng(12)
    for t in (1, 2, 3):
        cfg = lo.LambConfig(lr=1e-2, beta1=0.9, beta2=0.99, eps=1e-6, step=t)
        gpu, _ = run_gpu(cur, cfg, with_ratio=False)
        ref, _ = run_oracle(ref_state, cfg)
        for n in state:
            g = (1e-3 * rng.standard_normal(state[n]["w"].shape)).astype(np.float32)
            cur[n] = {"w": gpu[n]["w"].reshape(state[n]["w"].shape),
                      "m": gpu[n]["m"].reshape(state[n]["w"].shape),
                      "v": gpu[n]["v"].reshape(state[n]["w"].shape), "g": g}
            ref_state[n] = {"w": ref[n]["w"].reshape(g.shape), "m": ref[n]["m"].reshape(g.shape),
                            "v": ref[n]["v"].reshape(g.shape), "g": g.astype(np.float64)}
    for n in state:
        w0 = state[n]["w"].astype(np.float64)
        if w0.size == 0:
            continue
        ref_w = ref_state[n]["w"]
        err = np.abs(cur[n]["w"] - ref_w).max()
        bound = 1e-5 * np.abs(ref_w - w0).max() + 3 * 2.0 ** -23 * np.abs(ref_w).max()
        _say(f"      {n}: total change {normwise(cur[n]['w'] - w0, ref_w - w0):.2e}")
        assert err <= bound, (n, err, bound)


def test_lamb_split_calls_and_repeats_are_bitwise_identical():
    """Tensors are independent (one call over all equals one call each), and
    a repeated call gives the same bits."""
    _say("[gpu] lamb split calls / determinism")
    state = make_lamb_state(SMALL, seed=5)
    cfg = lo.LambConfig(lr=1e-3, step=2)
    joint, jr = run_gpu(state, cfg)
    again, ar = run_gpu(state, cfg)
    assert np.array_equal(jr, ar)
    for i, n in enumerate(state):
        one, r1 = run_gpu({n: state[n]}, cfg)
        assert np.array_equal(one[n]["w"], joint[n]["w"]), n
        assert np.array_equal(again[n]["w"], joint[n]["w"]), n
        assert r1[0] == jr[i], n


def test_lamb_full_parameter_set_of_the_175b_share():
    """One step over all six parameter tensors of the 175B model's one-GPU
    share (226.5 M elements), bf16 copy.  At this size the oracle computes
    sampled elements one by one (moments and direction), and two properties
    that hold at any size are checked in full: each tensor's change has norm
    lr ||w|| (the trust ratio's definition), and at the samples it points
    along the oracle's direction, scaled by the reported ratio."""
    import torch
    s = WORKLOADS["175b_tp8_share"]
    _say(f"[gpu] lamb full size {s.name}")
    state = make_lamb_state(block_param_shapes(s), seed=0, w_std=0.006)
    cfg = lo.LambConfig(lr=1e-3, step=100)
    gpu, ratios = run_gpu(state, cfg)
    rng = np.random.default_rng(1)
    for i, n in enumerate(state):
        st = {k: a.reshape(-1) for k, a in state[n].items()}
        size = st["w"].size
        idx = rng.integers(0, size, 2048)
        idx[:2] = (0, size - 1)
        g = cfg.grad_scale * st["g"][idx].astype(np.float64)
        m1, v1 = lo.moments(cfg, g, st["m"][idx].astype(np.float64),
                            st["v"][idx].astype(np.float64))
        w0 = st["w"][idx].astype(np.float64)
        u = lo.direction(cfg, m1, v1, w0, decay_of(n))
        e_m = normwise(gpu[n]["m"][idx], m1)
        e_v = normwise(gpu[n]["v"][idx], v1)
        e_u = normwise((gpu[n]["w"][idx] - w0) / (-cfg.lr * float(ratios[i])), u)
        w_full = torch.from_numpy(st["w"]).cuda().double()
        dw = torch.linalg.vector_norm(gpu[n]["w_t"].cuda().double() - w_full).item()
        wn = torch.linalg.vector_norm(w_full).item()
        _say(f"      {n} [{size}]: m={e_m:.2e} v={e_v:.2e} direction={e_u:.2e} "
             f"|dw|/(lr|w|)={dw / (cfg.lr * wn):.7f} ratio={ratios[i]:.6g}")
        assert e_m <= 1e-6 and e_v <= 1e-6, n
        # w' - w is rounded to fp32 at |w|, so the direction carries
        # ~ulp(|w|) / (lr ratio |u|) of relative error
        assert e_u <= 2e-3, n
        assert abs(dw / (cfg.lr * wn) - 1.0) <= 1e-4, n
        want = gpu[n]["w_t"].to(torch.bfloat16)
        assert torch.equal(gpu[n]["copy"], want), n

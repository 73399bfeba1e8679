"""Pins of the CPU oracle to facts that do not come from the oracle itself.

The paper prints no worked example for one block, so every pin is a closed
form, an invariant, a library routine the definition reduces to, brute force
on tiny inputs or finite differences.  Each is chosen so that a plausible slip
(a dropped term, a wrong sign, an off-by-one window edge, a transposed
operand, a missing scale) fails at least one of them; test_oracle_mutations.py
plants such slips and checks that they are caught.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import pblock_oracle as orc

RNG = np.random.default_rng(1234)


def tiny_cfg(window, batch=2, seq=12, hidden=16, heads=2, head_dim=8, ffn=32, tanh=True):
    return orc.OracleConfig(batch=batch, seq=seq, hidden=hidden, heads=heads,
                            head_dim=head_dim, ffn=ffn, window=window, gelu_tanh=tanh)


def tiny_inputs(cfg, seed=0, w_std=0.3):
    r = np.random.default_rng(seed)
    A, H, F_ = cfg.attn_width, cfg.hidden, cfg.ffn
    return dict(
        x=r.standard_normal((cfg.batch, cfg.seq, H)),
        gamma=1.0 + 0.1 * r.standard_normal(H),
        beta=0.1 * r.standard_normal(H),
        w_in=w_std * r.standard_normal((3 * A + F_, H)),
        b_in=0.1 * r.standard_normal(3 * A + F_),
        w_out=w_std * r.standard_normal((H, A + F_)),
        b_out=0.1 * r.standard_normal(H),
        dy=r.standard_normal((cfg.batch, cfg.seq, H)),
    )


# ------------------------------------------------------------------ LayerNorm
def test_layer_norm_unit_affine_moments():
    x = 3.0 + 2.0 * RNG.standard_normal((5, 64))
    eps = 1e-5
    h, xhat, mean, rstd = orc.layer_norm(x, np.ones(64), np.zeros(64), eps)
    sig2 = np.var(x, axis=-1)  # population variance, numpy's own routine
    np.testing.assert_allclose(h.mean(-1), 0.0, atol=1e-12)
    np.testing.assert_allclose(h.var(-1), sig2 / (sig2 + eps), rtol=1e-12)
    np.testing.assert_allclose(mean, x.mean(-1), rtol=1e-14)


def test_layer_norm_matches_torch():
    x = RNG.standard_normal((3, 7, 48))
    g = 1 + 0.2 * RNG.standard_normal(48)
    b = 0.2 * RNG.standard_normal(48)
    h, *_ = orc.layer_norm(x, g, b, 1e-5)
    ref = F.layer_norm(torch.from_numpy(x), (48,), torch.from_numpy(g), torch.from_numpy(b), 1e-5)
    np.testing.assert_allclose(h, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_layer_norm_backward_matches_torch_autograd():
    x = torch.from_numpy(RNG.standard_normal((4, 32))).requires_grad_()
    g = torch.from_numpy(1 + 0.3 * RNG.standard_normal(32)).requires_grad_()
    b = torch.from_numpy(0.3 * RNG.standard_normal(32)).requires_grad_()
    dh = RNG.standard_normal((4, 32))
    out = F.layer_norm(x, (32,), g, b, 1e-5)
    out.backward(torch.from_numpy(dh))
    _, xhat, _, rstd = orc.layer_norm(x.detach().numpy(), g.detach().numpy(), b.detach().numpy(), 1e-5)
    dx, dg, db = orc.layer_norm_backward(dh, xhat, rstd, g.detach().numpy())
    np.testing.assert_allclose(dx, x.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, g.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(db, b.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_layer_norm_backward_invariances():
    # LN(x + c) = LN(x): the input gradient sums to zero along the row.
    # With eps = 0, LN(a x) = LN(x) for a > 0: the gradient is orthogonal to x - mean.
    x = RNG.standard_normal((6, 40))
    g = 1 + 0.3 * RNG.standard_normal(40)
    dh = RNG.standard_normal((6, 40))
    _, xhat, _, rstd = orc.layer_norm(x, g, np.zeros(40), 0.0)
    dx, _, _ = orc.layer_norm_backward(dh, xhat, rstd, g)
    np.testing.assert_allclose(dx.sum(-1), 0.0, atol=1e-12)
    np.testing.assert_allclose((dx * (x - x.mean(-1, keepdims=True))).sum(-1), 0.0, atol=1e-11)


# ----------------------------------------------------------------------- GeLU
@pytest.mark.parametrize("tanh", [True, False])
def test_gelu_matches_torch(tanh):
    u = np.linspace(-8, 8, 1001)
    ref = F.gelu(torch.from_numpy(u), approximate="tanh" if tanh else "none").numpy()
    np.testing.assert_allclose(orc.gelu(u, tanh), ref, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("tanh", [True, False])
def test_gelu_grad_matches_autograd_and_fixed_points(tanh):
    u = torch.linspace(-8, 8, 1001, dtype=torch.float64, requires_grad=True)
    F.gelu(u, approximate="tanh" if tanh else "none").sum().backward()
    np.testing.assert_allclose(orc.gelu_grad(u.detach().numpy(), tanh), u.grad.numpy(),
                               rtol=1e-11, atol=1e-13)
    assert orc.gelu(np.array(0.0), tanh) == 0.0
    assert abs(orc.gelu_grad(np.array(0.0), tanh) - 0.5) < 1e-15


def test_gelu_forms_differ_measurably():
    # The two forms differ by a few 1e-4: above the fp32 tolerance, so the
    # flag must be the same on both sides of a parity test.
    u = np.linspace(-6, 6, 20001)
    diff = np.abs(orc.gelu(u, True) - orc.gelu(u, False)).max()
    assert 1e-4 < diff < 1e-3


# ---------------------------------------------------------------- attention
def brute_force_head(q, k, v, window):
    """Explicit loops: for each query, the keys j with 0 <= i - j < window."""
    S, d = q.shape
    o = np.zeros_like(v)
    lse = np.zeros(S)
    for i in range(S):
        js = [j for j in range(S) if 0 <= i - j < window]
        sc = [sum(q[i, c] * k[j, c] for c in range(d)) / math.sqrt(d) for j in js]
        mx = max(sc)
        w = [math.exp(s_ - mx) for s_ in sc]
        z = sum(w)
        lse[i] = mx + math.log(z)
        for jj, j in enumerate(js):
            o[i] += (w[jj] / z) * v[j]
    return o, lse


@pytest.mark.parametrize("window", [1, 2, 5, 9, 20])
def test_attention_brute_force(window):
    S, d = 9, 4
    q, k, v = (RNG.standard_normal((S, d)) for _ in range(3))
    o, lse = orc.swa_head_forward(q, k, v, window)
    o_ref, lse_ref = brute_force_head(q, k, v, window)
    np.testing.assert_allclose(o, o_ref, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, lse_ref, rtol=1e-12, atol=1e-13)


def test_attention_window_one_is_identity():
    S, d = 10, 8
    q, k, v, do = (RNG.standard_normal((S, d)) for _ in range(4))
    o, lse = orc.swa_head_forward(q, k, v, 1)
    np.testing.assert_array_equal(o, v)
    np.testing.assert_allclose(lse, (q * k).sum(1) / math.sqrt(d), rtol=1e-14)
    dq, dk, dv = orc.swa_head_backward(q, k, v, do, 1)
    np.testing.assert_array_equal(dq, 0.0)
    np.testing.assert_array_equal(dk, 0.0)
    np.testing.assert_array_equal(dv, do)


@pytest.mark.parametrize("window", [16, 17, 100])
def test_attention_full_window_is_causal_sdpa(window):
    S, d = 16, 8
    q, k, v, do = (RNG.standard_normal((S, d)) for _ in range(4))
    o, _ = orc.swa_head_forward(q, k, v, window)
    qt, kt, vt = (torch.from_numpy(a).requires_grad_() for a in (q, k, v))
    ref = F.scaled_dot_product_attention(qt[None], kt[None], vt[None], is_causal=True)[0]
    np.testing.assert_allclose(o, ref.detach().numpy(), rtol=1e-12, atol=1e-13)
    ref.backward(torch.from_numpy(do))
    dq, dk, dv = orc.swa_head_backward(q, k, v, do, window)
    np.testing.assert_allclose(dq, qt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dk, kt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv, vt.grad.numpy(), rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("window", [1, 3, 7, 30])
def test_attention_zero_query_is_sliding_mean(window):
    S, d = 30, 6
    k, v = RNG.standard_normal((S, d)), RNG.standard_normal((S, d))
    o, lse = orc.swa_head_forward(np.zeros((S, d)), k, v, window)
    c = np.vstack([np.zeros((1, d)), np.cumsum(v, axis=0)])
    i = np.arange(S)
    lo = np.maximum(0, i - window + 1)
    n = (i + 1 - lo)[:, None]
    np.testing.assert_allclose(o, (c[i + 1] - c[lo]) / n, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, np.log(n[:, 0]), rtol=1e-13)


@pytest.mark.parametrize("window", [1, 4, 11])
def test_softmax_rows_sum_to_one(window):
    S, d = 11, 5
    q, k, v = (RNG.standard_normal((S, d)) for _ in range(3))
    _, lse = orc.swa_head_forward(q, k, v, window)
    for i in range(S):
        tot = sum(math.exp(float(q[i] @ k[j]) / math.sqrt(d) - lse[i])
                  for j in range(max(0, i - window + 1), i + 1))
        assert abs(tot - 1.0) < 1e-13


def test_window_edge_is_exactly_w_keys():
    S, d, W = 12, 4, 4
    q, k, v = (RNG.standard_normal((S, d)) for _ in range(3))
    o, _ = orc.swa_head_forward(q, k, v, W)
    i = 9
    v_out = v.copy()
    v_out[i - W] += 5.0  # just outside query i's window
    assert np.array_equal(orc.swa_head_forward(q, k, v_out, W)[0][i], o[i])
    v_in = v.copy()
    v_in[i - W + 1] += 5.0  # the oldest key inside it
    assert not np.allclose(orc.swa_head_forward(q, k, v_in, W)[0][i], o[i])


@pytest.mark.parametrize("window", [1, 3, 12])
def test_attention_backward_finite_differences(window):
    S, d = 7, 3
    q, k, v, do = (RNG.standard_normal((S, d)) for _ in range(4))
    dq, dk, dv = orc.swa_head_backward(q, k, v, do, window)
    eps = 1e-6
    for arr, grad in ((q, dq), (k, dk), (v, dv)):
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            fp = (orc.swa_head_forward(q, k, v, window)[0] * do).sum()
            arr[idx] = old - eps
            fm = (orc.swa_head_forward(q, k, v, window)[0] * do).sum()
            arr[idx] = old
            assert abs((fp - fm) / (2 * eps) - grad[idx]) < 1e-7 * (1 + abs(grad[idx]))


# -------------------------------------------------------------------- block
def torch_block(cfg, t):
    """An independent autograd implementation of Eq. 2, written per head with
    explicit -inf masks (no code shared with the oracle)."""
    A, d = cfg.attn_width, cfg.head_dim
    x = t["x"]
    h = F.layer_norm(x, (cfg.hidden,), t["gamma"], t["beta"], cfg.ln_eps)
    z = F.linear(h, t["w_in"], t["b_in"])
    q, k, v, u = torch.split(z, [A, A, A, cfg.ffn], dim=-1)
    S = cfg.seq
    i = torch.arange(S)[:, None]
    j = torch.arange(S)[None, :]
    keep = (j <= i) & (j > i - cfg.window)
    outs = []
    for hd in range(cfg.heads):
        sl = slice(hd * d, (hd + 1) * d)
        s = q[..., sl] @ k[..., sl].transpose(-1, -2) / math.sqrt(d)
        s = s.masked_fill(~keep, float("-inf"))
        outs.append(torch.softmax(s, dim=-1) @ v[..., sl])
    o = torch.cat(outs, dim=-1)
    g = F.gelu(u, approximate="tanh" if cfg.gelu_tanh else "none")
    attn = F.linear(o, t["w_out"][:, :A])
    mlp = F.linear(g, t["w_out"][:, A:])
    return x + attn + mlp + t["b_out"]


NAMES = ("x", "gamma", "beta", "w_in", "b_in", "w_out", "b_out")


@pytest.mark.parametrize("window,tanh", [(1, True), (3, True), (12, True), (5, False), (40, False)])
def test_block_matches_torch_autograd(window, tanh):
    cfg = tiny_cfg(window, tanh=tanh)
    inp = tiny_inputs(cfg, seed=window)
    res = orc.run_block(cfg, inp)
    t = {n: torch.from_numpy(inp[n].copy()).requires_grad_() for n in NAMES}
    y = torch_block(cfg, t)
    y.backward(torch.from_numpy(inp["dy"]))
    np.testing.assert_allclose(res["y"], y.detach().numpy(), rtol=1e-11, atol=1e-12)
    for n in NAMES:
        np.testing.assert_allclose(res["d" + n], t[n].grad.numpy(), rtol=1e-9, atol=1e-11,
                                   err_msg=n)


@pytest.mark.parametrize("window", [1, 3, 12])
def test_block_finite_differences_every_entry(window):
    cfg = tiny_cfg(window, batch=2, seq=6, hidden=8, heads=2, head_dim=4, ffn=8)
    inp = tiny_inputs(cfg, seed=10 + window)
    res = orc.run_block(cfg, inp)
    dy = inp["dy"]
    eps = 1e-6

    def loss():
        y, _ = orc.block_forward(cfg, *(inp[n] for n in NAMES))
        return float((y * dy).sum())

    for n in NAMES:
        arr = inp[n]
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            lp = loss()
            arr[idx] = old - eps
            lm = loss()
            arr[idx] = old
            fd = (lp - lm) / (2 * eps)
            an = res["d" + n][idx]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (n, idx, fd, an)


def test_zero_out_projection_leaves_residual():
    cfg = tiny_cfg(3)
    inp = tiny_inputs(cfg)
    inp["w_out"][:] = 0.0
    res = orc.run_block(cfg, inp)
    np.testing.assert_array_equal(res["y"], inp["x"] + inp["b_out"])
    np.testing.assert_array_equal(res["dx"], inp["dy"])
    for n in ("dw_in", "db_in", "dgamma", "dbeta"):
        np.testing.assert_array_equal(res[n], 0.0)
    np.testing.assert_allclose(res["db_out"], inp["dy"].sum(axis=(0, 1)), rtol=1e-14)


def test_branches_add():
    cfg = tiny_cfg(4)
    inp = tiny_inputs(cfg)
    A = cfg.attn_width
    full = orc.run_block(cfg, inp)["y"]
    only_attn = dict(inp, w_out=inp["w_out"].copy())
    only_attn["w_out"][:, A:] = 0.0
    only_mlp = dict(inp, w_out=inp["w_out"].copy())
    only_mlp["w_out"][:, :A] = 0.0
    ya = orc.run_block(cfg, only_attn)["y"]
    ym = orc.run_block(cfg, only_mlp)["y"]
    np.testing.assert_allclose(ya + ym - inp["x"] - inp["b_out"], full, rtol=1e-12, atol=1e-12)


def test_without_attention_equals_serial_mlp_block():
    # With W_o = 0, Eq. 1 (serial) and Eq. 2 (parallel) coincide: both are
    # x + MLP(LN(x)).  The serial form is written here with torch's Linear
    # and LayerNorm modules.
    cfg = tiny_cfg(5)
    inp = tiny_inputs(cfg)
    A = cfg.attn_width
    inp["w_out"][:, :A] = 0.0
    y = orc.run_block(cfg, inp)["y"]
    ln = torch.nn.LayerNorm(cfg.hidden, eps=cfg.ln_eps, dtype=torch.float64)
    up = torch.nn.Linear(cfg.hidden, cfg.ffn, dtype=torch.float64)
    down = torch.nn.Linear(cfg.ffn, cfg.hidden, dtype=torch.float64)
    with torch.no_grad():
        ln.weight.copy_(torch.from_numpy(inp["gamma"]))
        ln.bias.copy_(torch.from_numpy(inp["beta"]))
        up.weight.copy_(torch.from_numpy(inp["w_in"][3 * A:]))
        up.bias.copy_(torch.from_numpy(inp["b_in"][3 * A:]))
        down.weight.copy_(torch.from_numpy(inp["w_out"][:, A:]))
        down.bias.copy_(torch.from_numpy(inp["b_out"]))
        x = torch.from_numpy(inp["x"])
        ref = x + down(F.gelu(up(ln(x)), approximate="tanh"))
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_batch_rows_are_independent():
    cfg = tiny_cfg(4, batch=2)
    inp = tiny_inputs(cfg)
    inp["x"][1] = inp["x"][0]
    inp["dy"][1] = inp["dy"][0]
    res = orc.run_block(cfg, inp)
    np.testing.assert_allclose(res["y"][1], res["y"][0], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(res["dx"][1], res["dx"][0], rtol=1e-14, atol=1e-14)
    single = orc.run_block(tiny_cfg(4, batch=1), {n: (v[:1] if v.ndim == 3 else v) for n, v in inp.items()})
    np.testing.assert_allclose(single["y"][0], res["y"][0], rtol=1e-13, atol=1e-13)
    # Parameter gradients of two identical rows are twice those of one.
    np.testing.assert_allclose(res["dw_in"], 2 * single["dw_in"], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("window,t", [(3, 0), (3, 7), (5, 11), (12, 4)])
def test_causal_locality(window, t):
    cfg = tiny_cfg(window, batch=1)
    inp = tiny_inputs(cfg)
    y0 = orc.run_block(cfg, inp)["y"][0]
    inp["x"][0, t, 3] += 0.5  # one feature: a whole-row shift would cancel in LN
    y1 = orc.run_block(cfg, inp)["y"][0]
    changed = np.abs(y1 - y0).max(axis=-1) > 1e-14
    expect = np.zeros(cfg.seq, dtype=bool)
    expect[t:t + window] = True
    np.testing.assert_array_equal(changed, expect)


@pytest.mark.parametrize("window", [1, 4, 12])
def test_head_attention_matches_block_and_autograd(window):
    """head_attention (one head of the block, forward and backward) against
    the block oracle's own cache, and its gradients against torch autograd of
    the independent block: the head's rows of dW_in are sum_b dq_b^T h_b (and
    likewise dk, dv), of db_in sum_b sum_s dq_b."""
    cfg = tiny_cfg(window, batch=2)
    inp = tiny_inputs(cfg, seed=30 + window)
    f = {n: np.asarray(v, np.float64) for n, v in inp.items()}
    _, cache = orc.block_forward(cfg, f["x"], f["gamma"], f["beta"], f["w_in"], f["b_in"],
                                 f["w_out"], f["b_out"])
    t = {n: torch.from_numpy(inp[n].copy()).requires_grad_() for n in NAMES}
    torch_block(cfg, t).backward(torch.from_numpy(inp["dy"]))
    A, d = cfg.attn_width, cfg.head_dim
    for hd in range(cfg.heads):
        cols = slice(hd * d, (hd + 1) * d)
        acc_w = [0.0, 0.0, 0.0]
        acc_b = [0.0, 0.0, 0.0]
        for b in range(cfg.batch):
            r = orc.head_attention(cfg, inp, b, hd)
            np.testing.assert_allclose(r["o"], cache["o"][b, :, cols], rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(r["lse"], cache["lse"][b, hd], rtol=1e-12, atol=1e-13)
            for j, n in enumerate("qkv"):
                zc = slice(j * A + hd * d, j * A + (hd + 1) * d)
                np.testing.assert_allclose(r[n], cache["z"][b, :, zc], rtol=1e-12, atol=1e-13)
            for j, n in enumerate(("dq", "dk", "dv")):
                acc_w[j] = acc_w[j] + r[n].T @ cache["h"][b]
                acc_b[j] = acc_b[j] + r[n].sum(axis=0)
        for j in range(3):
            rows = slice(j * A + hd * d, j * A + (hd + 1) * d)
            np.testing.assert_allclose(acc_w[j], t["w_in"].grad.numpy()[rows], rtol=1e-9,
                                       atol=1e-11)
            np.testing.assert_allclose(acc_b[j], t["b_in"].grad.numpy()[rows], rtol=1e-9,
                                       atol=1e-11)

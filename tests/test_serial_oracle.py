"""Pins for the serial-block oracle, each independent of its chain-rule code:

* special cases where the serial block reduces to the parallel one (checked
  against the separately pinned parallel oracle), which catch a dropped
  residual or a missing bias; each zeroes one branch, so on their own they
  cannot tell which tensor feeds the second LayerNorm;
* fp64 autograd of an independent torch-module implementation with both
  branches active, which fixes the forward composition (the second
  LayerNorm reads x1 = x + attention, not x) and every gradient;
* central finite differences of every gradient on a tiny block.

test_serial_oracle_mutations.py plants slips in the serial oracle and checks
that these pins catch them.
"""
import math

import numpy as np
import pytest
import torch

from oracle import pblock_oracle as po
from oracle import serial_oracle as so

CFG = po.OracleConfig(batch=2, seq=7, hidden=12, heads=2, head_dim=4, ffn=10, window=3,
                      ln_eps=1e-5, gelu_tanh=True)


def draw(cfg, seed):
    rng = np.random.default_rng(seed)
    A, H = cfg.attn_width, cfg.hidden
    n_in, k_out = 3 * A + cfg.ffn, A + cfg.ffn
    r = lambda *s, sc=1.0: sc * rng.standard_normal(s)  # noqa: E731
    return dict(x=r(cfg.batch, cfg.seq, H), gamma1=1 + r(H, sc=0.3), beta1=r(H, sc=0.3),
                gamma2=1 + r(H, sc=0.3), beta2=r(H, sc=0.3), w_in=r(n_in, H, sc=0.4),
                b_in=r(n_in, sc=0.3), w_out=r(H, k_out, sc=0.4), b_o=r(H, sc=0.3),
                b_down=r(H, sc=0.3), dy=r(cfg.batch, cfg.seq, H))


def parallel_of(p, gamma, beta, b_out):
    return dict(x=p["x"], gamma=gamma, beta=beta, w_in=p["w_in"], b_in=p["b_in"],
                w_out=p["w_out"], b_out=b_out, dy=p["dy"])


def test_reduces_to_parallel_without_attention_output():
    """W_o = 0, b_o = 0: x1 = x, so y = x + MLP(LN2(x)) + b_down, which is
    the parallel block with LN2's parameters and b_out = b_down."""
    p = draw(CFG, 1)
    A = CFG.attn_width
    p["w_out"][:, :A] = 0.0
    p["b_o"][:] = 0.0
    s = so.run_serial(CFG, p)
    r = po.run_block(CFG, parallel_of(p, p["gamma2"], p["beta2"], p["b_down"]))
    np.testing.assert_allclose(s["y"], r["y"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(s["dx"], r["dx"], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s["dgamma2"], r["dgamma"], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s["dbeta2"], r["dbeta"], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s["dw_in"][3 * A:], r["dw_in"][3 * A:], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s["dw_out"][:, A:], r["dw_out"][:, A:], rtol=1e-10, atol=1e-12)
    # nothing reaches the attention input projection or LN1
    assert np.abs(s["dw_in"][:3 * A]).max() == 0.0
    assert np.abs(s["dgamma1"]).max() == 0.0


def test_reduces_to_parallel_without_mlp_output():
    """W_down = 0: y = x + Attention(LN1(x)) + b_o + b_down, the parallel
    block with LN1's parameters and b_out = b_o + b_down."""
    p = draw(CFG, 2)
    A = CFG.attn_width
    p["w_out"][:, A:] = 0.0
    s = so.run_serial(CFG, p)
    r = po.run_block(CFG, parallel_of(p, p["gamma1"], p["beta1"], p["b_o"] + p["b_down"]))
    np.testing.assert_allclose(s["y"], r["y"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(s["dx"], r["dx"], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s["dgamma1"], r["dgamma"], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s["dw_in"][:3 * A], r["dw_in"][:3 * A], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s["dw_out"][:, :A], r["dw_out"][:, :A], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(s["db_o"], r["db_out"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(s["db_down"], r["db_out"], rtol=1e-12, atol=1e-12)


def test_attention_reaches_the_output_residual():
    """The attention branch is part of y itself, not only of the MLP's input:
    with the MLP off, y - x - biases is the attention output projection."""
    p = draw(CFG, 3)
    A = CFG.attn_width
    p["w_out"][:, A:] = 0.0
    s = so.run_serial(CFG, p)
    cfg = CFG
    y, cache = so.serial_forward(cfg, *[p[n] for n in so.PARAMS])
    attn = cache["o"] @ p["w_out"][:, :A].T
    np.testing.assert_allclose(y - p["x"] - p["b_o"] - p["b_down"], attn, atol=1e-12)
    assert np.abs(attn).max() > 0.1


@pytest.mark.parametrize("name", ["x", "gamma1", "beta1", "gamma2", "beta2", "w_in", "b_in",
                                  "w_out", "b_o", "b_down"])
def test_gradients_match_finite_differences(name):
    cfg = po.OracleConfig(batch=1, seq=5, hidden=8, heads=2, head_dim=4, ffn=6, window=3)
    p = draw(cfg, 4)
    grads = so.run_serial(cfg, p)
    key = {"x": "dx"}.get(name, "d" + name)
    rng = np.random.default_rng(5)
    direction = rng.standard_normal(p[name].shape)
    eps = 1e-6

    def loss(delta):
        q = dict(p)
        q[name] = p[name] + delta * direction
        y, _ = so.serial_forward(cfg, *[q[n] for n in so.PARAMS])
        return float((y * p["dy"]).sum())

    fd = (loss(eps) - loss(-eps)) / (2 * eps)
    an = float((grads[key] * direction).sum())
    assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (name, fd, an)


# --------------------------------------------------------------------------
# An independent autograd implementation of the standard pre-LN block, with
# both branches active (Section 3.1, Eq. 1 read as the serial block the text
# names).  Written from torch modules and explicit -inf masks; no code is
# shared with the oracle's forward or its chain rule.
def torch_serial_block(cfg, t):
    A, d, S = cfg.attn_width, cfg.head_dim, cfg.seq
    x = t["x"]
    h1 = torch.nn.functional.layer_norm(x, (cfg.hidden,), t["gamma1"], t["beta1"], cfg.ln_eps)
    qkv = torch.nn.functional.linear(h1, t["w_in"][:3 * A], t["b_in"][:3 * A])
    q, k, v = torch.split(qkv, [A, A, A], dim=-1)
    i = torch.arange(S)[:, None]
    j = torch.arange(S)[None, :]
    keep = (j <= i) & (j > i - cfg.window)
    heads = []
    for hd in range(cfg.heads):
        sl = slice(hd * d, (hd + 1) * d)
        s = (q[..., sl] @ k[..., sl].transpose(-1, -2)) / math.sqrt(d)
        heads.append(torch.softmax(s.masked_fill(~keep, float("-inf")), dim=-1) @ v[..., sl])
    x1 = x + torch.nn.functional.linear(torch.cat(heads, dim=-1), t["w_out"][:, :A], t["b_o"])
    h2 = torch.nn.functional.layer_norm(x1, (cfg.hidden,), t["gamma2"], t["beta2"], cfg.ln_eps)
    u = torch.nn.functional.linear(h2, t["w_in"][3 * A:], t["b_in"][3 * A:])
    g = torch.nn.functional.gelu(u, approximate="tanh" if cfg.gelu_tanh else "none")
    return x1 + torch.nn.functional.linear(g, t["w_out"][:, A:], t["b_down"])


@pytest.mark.parametrize("window,tanh", [(1, True), (3, True), (7, False), (20, True)])
def test_matches_torch_autograd_with_both_branches(window, tanh):
    """Both branches on, every gradient: y and all ten gradients equal fp64
    autograd of the block built from torch modules."""
    cfg = po.OracleConfig(batch=2, seq=7, hidden=12, heads=2, head_dim=4, ffn=10, window=window,
                          ln_eps=1e-5, gelu_tanh=tanh)
    p = draw(cfg, 20 + window)
    s = so.run_serial(cfg, p)
    t = {n: torch.from_numpy(p[n].copy()).requires_grad_() for n in so.PARAMS}
    y = torch_serial_block(cfg, t)
    y.backward(torch.from_numpy(p["dy"]))
    # both branches really reach y at these draws
    A = cfg.attn_width
    assert np.abs(p["w_out"][:, :A]).max() > 0 and np.abs(p["w_out"][:, A:]).max() > 0
    np.testing.assert_allclose(s["y"], y.detach().numpy(), rtol=1e-11, atol=1e-12)
    for n in so.PARAMS:
        key = {"x": "dx"}.get(n, "d" + n)
        np.testing.assert_allclose(s[key], t[n].grad.numpy(), rtol=1e-9, atol=1e-11,
                                   err_msg=n)

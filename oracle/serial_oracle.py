"""CPU oracle for the standard (serial) transformer block, forward and
backward, in float64: the block the paper's parallel formulation replaces.

TEST INFRASTRUCTURE ONLY, under the same rules as pblock_oracle: only the
tests, the smoke check and the benchmark's CPU-baseline leg may import it.

What is computed (MegaScale Section 3.1, Eq. 1 read as the standard pre-LN
block the text names; see the readings in the design notes):

    x1 = x + Attention(LN1(x)) + b_o
    y  = x1 + MLP(LN2(x1)) + b_down

with two LayerNorms (gamma1/beta1, gamma2/beta2), the same causal
sliding-window attention as the parallel block, and the parallel block's
packed weights reused as slices:
  w_in  [3A+F, H]  rows Q | K | V (the attention input projection) | MLP-up
  b_in  [3A+F]
  w_out [H, A+F]   columns attention-out | MLP-down
  b_o, b_down [H]  the two output biases (separate here: in the serial block
                   they enter at different points and are both identifiable).

The attention, LayerNorm and GeLU primitives are the ones of pblock_oracle;
the chain rule below is written out step by step from the forward pass.
"""
from __future__ import annotations

import numpy as np

from oracle.pblock_oracle import (OracleConfig, config_from_shape, gelu, gelu_grad,  # noqa: F401
                                  layer_norm, layer_norm_backward, swa_head_backward,
                                  swa_head_forward)

__all__ = ["serial_forward", "serial_backward", "run_serial"]

PARAMS = ("x", "gamma1", "beta1", "gamma2", "beta2", "w_in", "b_in", "w_out", "b_o", "b_down")


def _attention(cfg, q, k, v):
    d = cfg.head_dim
    o = np.zeros(q.shape, dtype=np.float64)
    lse = np.zeros((cfg.batch, cfg.heads, cfg.seq), dtype=np.float64)
    for b in range(cfg.batch):
        for hd in range(cfg.heads):
            sl = slice(hd * d, (hd + 1) * d)
            o[b, :, sl], lse[b, hd] = swa_head_forward(q[b, :, sl], k[b, :, sl], v[b, :, sl],
                                                       cfg.window)
    return o, lse


def serial_forward(cfg: OracleConfig, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o,
                   b_down):
    """The serial block; x is [B, S, H].  Returns (y, cache)."""
    A = cfg.attn_width
    h1, xhat1, mean1, rstd1 = layer_norm(x, gamma1, beta1, cfg.ln_eps)
    qkv = h1 @ w_in[:3 * A].T + b_in[:3 * A]
    q, k, v = qkv[..., :A], qkv[..., A:2 * A], qkv[..., 2 * A:]
    o, lse = _attention(cfg, q, k, v)
    x1 = x + o @ w_out[:, :A].T + b_o
    h2, xhat2, mean2, rstd2 = layer_norm(x1, gamma2, beta2, cfg.ln_eps)
    u = h2 @ w_in[3 * A:].T + b_in[3 * A:]
    g = gelu(u, cfg.gelu_tanh)
    y = x1 + g @ w_out[:, A:].T + b_down
    cache = dict(h1=h1, xhat1=xhat1, mean1=mean1, rstd1=rstd1, qkv=qkv, o=o, lse=lse, x1=x1,
                 h2=h2, xhat2=xhat2, mean2=mean2, rstd2=rstd2, u=u, g=g)
    return y, cache


def serial_backward(cfg: OracleConfig, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o,
                    b_down, cache, dy):
    """Gradients of sum(y * dy) with respect to x and every parameter.

    Returns dx, dgamma1, dbeta1, dgamma2, dbeta2, dw_in, db_in, dw_out, db_o,
    db_down (weight gradients in the packed layouts of w_in and w_out)."""
    A, d = cfg.attn_width, cfg.head_dim
    T = cfg.batch * cfg.seq
    flat = lambda t: t.reshape(T, -1)  # noqa: E731
    # y = x1 + G W_down^T + b_down
    db_down = flat(dy).sum(axis=0)
    dw_down = flat(dy).T @ flat(cache["g"])
    dg = dy @ w_out[:, A:]
    du = dg * gelu_grad(cache["u"], cfg.gelu_tanh)
    # U = h2 W_up^T + b_up
    dw_up = flat(du).T @ flat(cache["h2"])
    db_up = flat(du).sum(axis=0)
    dh2 = du @ w_in[3 * A:]
    # h2 = LN2(x1); x1 also feeds y directly
    dx1_ln, dgamma2, dbeta2 = layer_norm_backward(dh2, cache["xhat2"], cache["rstd2"], gamma2)
    dx1 = dy + dx1_ln
    # x1 = x + O W_o^T + b_o
    db_o = flat(dx1).sum(axis=0)
    dw_o = flat(dx1).T @ flat(cache["o"])
    do = dx1 @ w_out[:, :A]
    qkv = cache["qkv"]
    dqkv = np.zeros_like(qkv)
    for b in range(cfg.batch):
        for hd in range(cfg.heads):
            sl = [slice(j * A + hd * d, j * A + (hd + 1) * d) for j in range(3)]
            dq, dk, dv = swa_head_backward(qkv[b, :, sl[0]], qkv[b, :, sl[1]], qkv[b, :, sl[2]],
                                           do[b, :, hd * d:(hd + 1) * d], cfg.window)
            dqkv[b, :, sl[0]], dqkv[b, :, sl[1]], dqkv[b, :, sl[2]] = dq, dk, dv
    # QKV = h1 W_qkv^T + b_qkv
    dw_qkv = flat(dqkv).T @ flat(cache["h1"])
    db_qkv = flat(dqkv).sum(axis=0)
    dh1 = dqkv @ w_in[:3 * A]
    dx_ln, dgamma1, dbeta1 = layer_norm_backward(dh1, cache["xhat1"], cache["rstd1"], gamma1)
    dx = dx1 + dx_ln
    return dict(dx=dx, dgamma1=dgamma1, dbeta1=dbeta1, dgamma2=dgamma2, dbeta2=dbeta2,
                dw_in=np.concatenate([dw_qkv, dw_up], axis=0),
                db_in=np.concatenate([db_qkv, db_up]),
                dw_out=np.concatenate([dw_o, dw_down], axis=1), db_o=db_o, db_down=db_down)


def run_serial(cfg: OracleConfig, inputs: dict):
    """Forward then backward on a dict of arrays, in float64.  Returns y and
    every gradient."""
    f = {n: np.asarray(inputs[n], dtype=np.float64) for n in PARAMS + ("dy",)}
    args = [f[n] for n in PARAMS]
    y, cache = serial_forward(cfg, *args)
    out = serial_backward(cfg, *args, cache, f["dy"])
    out["y"] = y
    out["lse"] = cache["lse"]
    return out

"""CPU oracle for the parallel transformer block with causal sliding-window
attention, forward and backward, in float64.

TEST INFRASTRUCTURE ONLY.  This module exists to check the HIP library.  Only
the tests, the smoke check and the CPU-baseline leg of the benchmark may import
it; the library and its Python binding never call it, and it shares no code
with them (the seeded input generator is the one common module, and it holds
none of the block's arithmetic).

What is computed (MegaScale, Section 3.1):

* Eq. 2, the parallel block:  y = x + MLP(LN(x)) + Attention(LN(x)), with one
  LayerNorm whose output feeds both branches.
* Sliding-window attention (Section 3.1, "Sliding window attention"): each
  query attends to a fixed window of keys, cost O(s*w) instead of O(s*s).  The
  window is read causally: query i sees key j iff 0 <= i - j < W (W keys, the
  query's own position included), so W >= S is ordinary causal attention.
* Section 3.3 swaps in FlashAttention-2 and fused LayerNorm/GeLU kernels.
  Those change only how the result is evaluated, never the result, so the
  oracle is the plain definition: a dense masked score matrix, an explicit
  softmax, plain matrix products.

The backward pass is the chain rule of the forward pass, written out the
textbook way (softmax Jacobian with the row sum of p*dp, LayerNorm's
closed-form input gradient).  Matrix products use numpy's matmul as the
library primitive; nothing is blocked, fused or reordered.

Parameter layout (the packing is a choice the paper leaves open):
  w_in  [3A+F, H]  rows Q | K | V | MLP-up; head h owns rows h*d..h*d+d-1 of
                   each of Q, K and V.
  b_in  [3A+F]
  w_out [H, A+F]   columns attention-out | MLP-down.
  b_out [H]        the attention and MLP output biases are summed into one
                   vector: in Eq. 2 they always appear added together, so only
                   their sum is identifiable.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np
from scipy.special import erf

__all__ = [
    "OracleConfig",
    "layer_norm",
    "layer_norm_backward",
    "gelu",
    "gelu_grad",
    "window_mask",
    "swa_head_forward",
    "swa_head_backward",
    "block_forward",
    "block_backward",
    "head_attention",
]

SQRT_2_OVER_PI = math.sqrt(2.0 / math.pi)
GELU_TANH_COEF = 0.044715


@dataclass(frozen=True)
class OracleConfig:
    batch: int
    seq: int
    hidden: int
    heads: int
    head_dim: int
    ffn: int
    window: int
    ln_eps: float = 1e-5
    gelu_tanh: bool = True

    @property
    def attn_width(self) -> int:
        return self.heads * self.head_dim


# ---------------------------------------------------------------- LayerNorm
def layer_norm(x, gamma, beta, eps):
    """LN over the last axis with the biased variance and eps inside the root.

    Returns (h, xhat, mean, rstd) with h = gamma * xhat + beta.
    """
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mean) * rstd
    return gamma * xhat + beta, xhat, mean[..., 0], rstd[..., 0]


def layer_norm_backward(dh, xhat, rstd, gamma):
    """Gradient of h = gamma * xhat + beta through LN.

    Returns (dx, dgamma, dbeta); dgamma and dbeta are summed over every
    leading axis.  dx is the closed form
    rstd * (g - mean(g) - xhat * mean(g * xhat)) with g = gamma * dh.
    """
    lead = tuple(range(dh.ndim - 1))
    dgamma = (dh * xhat).sum(axis=lead)
    dbeta = dh.sum(axis=lead)
    g = gamma * dh
    dx = rstd[..., None] * (
        g
        - g.mean(axis=-1, keepdims=True)
        - xhat * (g * xhat).mean(axis=-1, keepdims=True)
    )
    return dx, dgamma, dbeta


# --------------------------------------------------------------------- GeLU
def gelu(u, tanh_form=True):
    """GeLU; tanh_form selects 0.5u(1+tanh(sqrt(2/pi)(u+0.044715u^3))),
    otherwise the exact 0.5u(1+erf(u/sqrt2))."""
    if tanh_form:
        return 0.5 * u * (1.0 + np.tanh(SQRT_2_OVER_PI * (u + GELU_TANH_COEF * u ** 3)))
    return 0.5 * u * (1.0 + erf(u / math.sqrt(2.0)))


def gelu_grad(u, tanh_form=True):
    """Derivative of gelu(u) with respect to u, in the same form."""
    if tanh_form:
        a = SQRT_2_OVER_PI * (u + GELU_TANH_COEF * u ** 3)
        t = np.tanh(a)
        da = SQRT_2_OVER_PI * (1.0 + 3.0 * GELU_TANH_COEF * u ** 2)
        return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * da
    cdf = 0.5 * (1.0 + erf(u / math.sqrt(2.0)))
    pdf = np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)
    return cdf + u * pdf


# ----------------------------------------------- sliding-window attention
def window_mask(seq, window):
    """visible[i, j] is True iff key j lies in query i's causal window."""
    i = np.arange(seq)[:, None]
    j = np.arange(seq)[None, :]
    return (i - j >= 0) & (i - j < window)


def swa_head_forward(q, k, v, window):
    """One (batch row, head): q, k, v are [S, d].

    Returns (o [S, d], lse [S]) where lse is the log of each row's softmax
    denominator in the scaled-score domain (the quantity a flash-style kernel
    keeps for its backward pass).
    """
    S, d = q.shape
    visible = window_mask(S, window)
    s = (q @ k.T) / math.sqrt(d)
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(s - m).sum(axis=1))
    p = np.exp(s - lse[:, None])  # exp(-inf) = 0 outside the window
    return p @ v, lse


def swa_head_backward(q, k, v, do, window):
    """Gradient of one head's attention.  Returns (dq, dk, dv).

    The probabilities are formed again from q and k; the softmax Jacobian is
    ds = p * (dp - rowsum(p * dp)).
    """
    S, d = q.shape
    visible = window_mask(S, window)
    s = np.where(visible, (q @ k.T) / math.sqrt(d), -np.inf)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    p = e / e.sum(axis=1, keepdims=True)
    dv = p.T @ do
    dp = do @ v.T
    ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
    dq = (ds @ k) / math.sqrt(d)
    dk = (ds.T @ q) / math.sqrt(d)
    return dq, dk, dv


# ------------------------------------------------------------------- block
def _split_in(cfg, z):
    A = cfg.attn_width
    return z[..., :A], z[..., A:2 * A], z[..., 2 * A:3 * A], z[..., 3 * A:]


def _heads(t, cfg, b, hd):
    d = cfg.head_dim
    return t[b, :, hd * d:(hd + 1) * d]


def block_forward(cfg: OracleConfig, x, gamma, beta, w_in, b_in, w_out, b_out):
    """Eq. 2 of Section 3.1.  x is [B, S, H]; returns (y, cache).

    The attention branch is O @ W_o^T and the MLP branch is GeLU(U) @ W_down^T,
    with W_o | W_down the two column blocks of w_out; the two branches and the
    residual are added as the equation writes them.
    """
    A = cfg.attn_width
    h, xhat, mean, rstd = layer_norm(x, gamma, beta, cfg.ln_eps)
    z = h @ w_in.T + b_in
    q, k, v, u = _split_in(cfg, z)
    o = np.zeros(q.shape, dtype=np.float64)
    lse = np.zeros((cfg.batch, cfg.heads, cfg.seq), dtype=np.float64)
    d = cfg.head_dim
    for b in range(cfg.batch):
        for hd in range(cfg.heads):
            ob, lb = swa_head_forward(_heads(q, cfg, b, hd), _heads(k, cfg, b, hd),
                                      _heads(v, cfg, b, hd), cfg.window)
            o[b, :, hd * d:(hd + 1) * d] = ob
            lse[b, hd] = lb
    g = gelu(u, cfg.gelu_tanh)
    w_o, w_down = w_out[:, :A], w_out[:, A:]
    attn_branch = o @ w_o.T
    mlp_branch = g @ w_down.T
    y = x + mlp_branch + attn_branch + b_out
    cache = dict(h=h, xhat=xhat, mean=mean, rstd=rstd, z=z, o=o, g=g, lse=lse)
    return y, cache


def block_backward(cfg: OracleConfig, x, gamma, beta, w_in, b_in, w_out, b_out,
                   cache, dy, weight_rows=None):
    """Gradients of sum(y * dy) with respect to x and every parameter.

    Returns a dict with dx, dgamma, dbeta, dw_in, db_in, dw_out, db_out.
    ``weight_rows`` (optional) is a pair (rows_in, rows_out) of index arrays:
    the weight gradients are then returned only for those rows of w_in and
    w_out (each row of a weight gradient is a separate sum over tokens, so the
    selected rows are the same numbers the full product would give).
    """
    A, d = cfg.attn_width, cfg.head_dim
    h, xhat, rstd, z, o, g = (cache[n] for n in ("h", "xhat", "rstd", "z", "o", "g"))
    q, k, v, u = _split_in(cfg, z)
    T = cfg.batch * cfg.seq
    dy2 = dy.reshape(T, -1)
    w_o, w_down = w_out[:, :A], w_out[:, A:]

    # y = x + G W_down^T + O W_o^T + b_out
    db_out = dy2.sum(axis=0)
    c2 = np.concatenate([o, g], axis=-1).reshape(T, -1)
    rows_in, rows_out = (None, None) if weight_rows is None else weight_rows
    if rows_out is None:
        dw_out = dy2.T @ c2
    else:
        dw_out = dy2[:, rows_out].T @ c2
    do = dy @ w_o
    dg = dy @ w_down
    du = dg * gelu_grad(u, cfg.gelu_tanh)

    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(cfg.batch):
        for hd in range(cfg.heads):
            sl = slice(hd * d, (hd + 1) * d)
            dq[b, :, sl], dk[b, :, sl], dv[b, :, sl] = swa_head_backward(
                q[b, :, sl], k[b, :, sl], v[b, :, sl], do[b, :, sl], cfg.window)

    dz = np.concatenate([dq, dk, dv, du], axis=-1)
    dz2 = dz.reshape(T, -1)
    db_in = dz2.sum(axis=0)
    h2 = h.reshape(T, -1)
    if rows_in is None:
        dw_in = dz2.T @ h2
    else:
        dw_in = dz2[:, rows_in].T @ h2
    dh = dz @ w_in
    dx_ln, dgamma, dbeta = layer_norm_backward(dh, xhat, rstd, gamma)
    dx = dy + dx_ln
    return dict(dx=dx, dgamma=dgamma, dbeta=dbeta, dw_in=dw_in, db_in=db_in,
                dw_out=dw_out, db_out=db_out)


def head_attention(cfg: OracleConfig, inputs: dict, b: int, hd: int):
    """One (batch row b, head hd) of the block's attention, forward and
    backward, from the block's inputs (Eq. 2 of Section 3.1 and its
    sliding-window attention; the FlashAttention-2 result of Section 3.3).

    The same definitions as block_forward / block_backward restricted to one
    head: h = LN(x) of row b; q, k, v from that head's rows of w_in and b_in;
    (o, lse) by swa_head_forward; the head's output gradient
    do = dy W_o[:, head columns] (the attention half of dC = dy W_out); and
    (dq, dk, dv) by swa_head_backward.  Only this head's columns are formed,
    so it stays cheap at full size.  Returns a dict of float64 arrays
    q, k, v, o, lse, do, dq, dk, dv ([S, d], lse [S]).
    """
    A, d = cfg.attn_width, cfg.head_dim
    f = {n: np.asarray(inputs[n], dtype=np.float64)
         for n in ("x", "gamma", "beta", "w_in", "b_in", "w_out", "dy")}
    h, _, _, _ = layer_norm(f["x"][b], f["gamma"], f["beta"], cfg.ln_eps)
    cols = slice(hd * d, (hd + 1) * d)
    qkv = []
    for j in range(3):
        rows = slice(j * A + hd * d, j * A + (hd + 1) * d)
        qkv.append(h @ f["w_in"][rows].T + f["b_in"][rows])
    q, k, v = qkv
    o, lse = swa_head_forward(q, k, v, cfg.window)
    do = f["dy"][b] @ f["w_out"][:, cols]
    dq, dk, dv = swa_head_backward(q, k, v, do, cfg.window)
    return dict(q=q, k=k, v=v, o=o, lse=lse, do=do, dq=dq, dk=dk, dv=dv)


def run_block(cfg: OracleConfig, inputs: dict, weight_rows=None):
    """Forward then backward on a dict of arrays (any float dtype), in float64.

    Returns a dict holding y and every gradient.
    """
    f = {n: np.asarray(inputs[n], dtype=np.float64)
         for n in ("x", "gamma", "beta", "w_in", "b_in", "w_out", "b_out", "dy")}
    y, cache = block_forward(cfg, f["x"], f["gamma"], f["beta"], f["w_in"], f["b_in"],
                             f["w_out"], f["b_out"])
    grads = block_backward(cfg, f["x"], f["gamma"], f["beta"], f["w_in"], f["b_in"],
                           f["w_out"], f["b_out"], cache, f["dy"], weight_rows)
    grads["y"] = y
    grads["lse"] = cache["lse"]
    return grads


def config_from_shape(shape) -> OracleConfig:
    """Build an OracleConfig from any object with the block's shape fields."""
    return OracleConfig(batch=shape.batch, seq=shape.seq, hidden=shape.hidden,
                        heads=shape.heads, head_dim=shape.head_dim, ffn=shape.ffn,
                        window=shape.window, ln_eps=shape.ln_eps,
                        gelu_tanh=bool(shape.gelu_tanh))

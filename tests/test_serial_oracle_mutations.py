"""Plant plausible mistakes in the serial-block oracle and check that the pins
of test_serial_oracle.py catch each one.

Every mutation is made consistently in the forward pass and in its chain
rule, so the finite-difference pins (which only compare the backward with the
oracle's own forward) cannot see it; the pins that must catch it are the ones
tied to something outside the oracle.  Everything runs on the CPU.
"""
import numpy as np
import pytest

import tests.test_serial_oracle as pins
from oracle import serial_oracle as so
from oracle.pblock_oracle import layer_norm, layer_norm_backward

ORIGINAL_FORWARD = so.serial_forward
ORIGINAL_BACKWARD = so.serial_backward

PIN_CALLS = [
    lambda: pins.test_reduces_to_parallel_without_attention_output(),
    lambda: pins.test_reduces_to_parallel_without_mlp_output(),
    lambda: pins.test_attention_reaches_the_output_residual(),
    lambda: pins.test_matches_torch_autograd_with_both_branches(3, True),
    lambda: pins.test_matches_torch_autograd_with_both_branches(7, False),
] + [
    (lambda n: (lambda: pins.test_gradients_match_finite_differences(n)))(n) for n in so.PARAMS
]


def count_failures():
    bad = 0
    for call in PIN_CALLS:
        try:
            call()
        except (AssertionError, ValueError, IndexError):
            bad += 1
    return bad


def _ln2_reads_x_forward(cfg, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o, b_down):
    """The second LayerNorm normalises x instead of x1 = x + attention."""
    A = cfg.attn_width
    h1, xhat1, mean1, rstd1 = layer_norm(x, gamma1, beta1, cfg.ln_eps)
    qkv = h1 @ w_in[:3 * A].T + b_in[:3 * A]
    o, lse = so._attention(cfg, qkv[..., :A], qkv[..., A:2 * A], qkv[..., 2 * A:])
    x1 = x + o @ w_out[:, :A].T + b_o
    h2, xhat2, mean2, rstd2 = layer_norm(x, gamma2, beta2, cfg.ln_eps)
    u = h2 @ w_in[3 * A:].T + b_in[3 * A:]
    g = so.gelu(u, cfg.gelu_tanh)
    y = x1 + g @ w_out[:, A:].T + b_down
    cache = dict(h1=h1, xhat1=xhat1, mean1=mean1, rstd1=rstd1, qkv=qkv, o=o, lse=lse, x1=x1,
                 h2=h2, xhat2=xhat2, mean2=mean2, rstd2=rstd2, u=u, g=g)
    return y, cache


def _ln2_reads_x_backward(cfg, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o, b_down,
                          cache, dy):
    """The chain rule of the slip above: LN2's input gradient goes to x, and
    x1 receives only the direct path from y."""
    A = cfg.attn_width
    out = ORIGINAL_BACKWARD(cfg, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o, b_down,
                            cache, dy)
    # The correct chain added LN2's input gradient into dx1, which then
    # reached x directly and also flowed through the attention branch.
    # Recompute with dx1 = dy and add LN2's part to dx at the end.
    du = (dy @ w_out[:, A:]) * so.gelu_grad(cache["u"], cfg.gelu_tanh)
    dh2 = du @ w_in[3 * A:]
    dx_ln2, _, _ = layer_norm_backward(dh2, cache["xhat2"], cache["rstd2"], gamma2)
    T = cfg.batch * cfg.seq
    d = cfg.head_dim
    dx1 = dy
    out["db_o"] = dx1.reshape(T, -1).sum(axis=0)
    dw_o = dx1.reshape(T, -1).T @ cache["o"].reshape(T, -1)
    do = dx1 @ w_out[:, :A]
    qkv = cache["qkv"]
    dqkv = np.zeros_like(qkv)
    for b in range(cfg.batch):
        for hd in range(cfg.heads):
            sl = [slice(j * A + hd * d, j * A + (hd + 1) * d) for j in range(3)]
            dq, dk, dv = so.swa_head_backward(qkv[b, :, sl[0]], qkv[b, :, sl[1]],
                                              qkv[b, :, sl[2]], do[b, :, hd * d:(hd + 1) * d],
                                              cfg.window)
            dqkv[b, :, sl[0]], dqkv[b, :, sl[1]], dqkv[b, :, sl[2]] = dq, dk, dv
    dw_qkv = dqkv.reshape(T, -1).T @ cache["h1"].reshape(T, -1)
    db_qkv = dqkv.reshape(T, -1).sum(axis=0)
    dh1 = dqkv @ w_in[:3 * A]
    dx_ln1, dgamma1, dbeta1 = layer_norm_backward(dh1, cache["xhat1"], cache["rstd1"], gamma1)
    out["dx"] = dx1 + dx_ln1 + dx_ln2
    out["dgamma1"], out["dbeta1"] = dgamma1, dbeta1
    out["dw_in"] = np.concatenate([dw_qkv, out["dw_in"][3 * A:]], axis=0)
    out["db_in"] = np.concatenate([db_qkv, out["db_in"][3 * A:]])
    out["dw_out"] = np.concatenate([dw_o, out["dw_out"][:, A:]], axis=1)
    return out


def _mlp_reads_h1_forward(cfg, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o, b_down):
    """The MLP-up projection reads LN1's output (the parallel block's wiring)
    while LN2's parameters stay in the model: made consistent by moving the
    forward only (the backward then disagrees with finite differences)."""
    y, cache = ORIGINAL_FORWARD(cfg, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o,
                                b_down)
    A = cfg.attn_width
    u = cache["h1"] @ w_in[3 * A:].T + b_in[3 * A:]
    g = so.gelu(u, cfg.gelu_tanh)
    y = cache["x1"] + g @ w_out[:, A:].T + b_down
    cache.update(u=u, g=g)
    return y, cache


def _dropped_attention_residual_forward(cfg, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out,
                                        b_o, b_down):
    """y is built on x instead of x1 (Eq. 1 as printed, read literally)."""
    y, cache = ORIGINAL_FORWARD(cfg, x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o,
                                b_down)
    return y - (cache["x1"] - x), cache


MUTATIONS = {
    "ln2_reads_x": (_ln2_reads_x_forward, _ln2_reads_x_backward),
    "mlp_reads_ln1_output": (_mlp_reads_h1_forward, ORIGINAL_BACKWARD),
    "dropped_attention_residual": (_dropped_attention_residual_forward, ORIGINAL_BACKWARD),
}


def test_ln2_slip_is_self_consistent():
    """The planted LN2 slip really is consistent: its backward matches finite
    differences of its own forward, so only an outside reference can catch it."""
    import oracle.pblock_oracle as po
    cfg = po.OracleConfig(batch=1, seq=5, hidden=8, heads=2, head_dim=4, ffn=6, window=3)
    p = pins.draw(cfg, 4)
    args = [p[n] for n in so.PARAMS]
    y, cache = _ln2_reads_x_forward(cfg, *args)
    grads = _ln2_reads_x_backward(cfg, *args, cache, p["dy"])
    rng = np.random.default_rng(5)
    for name in so.PARAMS:
        key = {"x": "dx"}.get(name, "d" + name)
        direction = rng.standard_normal(p[name].shape)
        eps = 1e-6

        def loss(delta):
            q = dict(p)
            q[name] = p[name] + delta * direction
            yy, _ = _ln2_reads_x_forward(cfg, *[q[n] for n in so.PARAMS])
            return float((yy * p["dy"]).sum())

        fd = (loss(eps) - loss(-eps)) / (2 * eps)
        an = float((grads[key] * direction).sum())
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (name, fd, an)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    fwd, bwd = MUTATIONS[name]
    monkeypatch.setattr(so, "serial_forward", fwd)
    monkeypatch.setattr(so, "serial_backward", bwd)
    assert count_failures() >= 1, f"no pin caught the planted mistake {name}"


def test_unmutated_serial_oracle_passes_every_pin():
    assert count_failures() == 0

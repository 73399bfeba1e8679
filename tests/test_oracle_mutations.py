"""Plant plausible mistakes in the CPU oracle and check that the pins catch them.

Each mutation swaps one oracle function for a subtly wrong copy (an
off-by-one window edge, a dropped term, a wrong sign, a transposed operand, a
missing scale).  The pins of test_oracle_pins.py are then run against the
mutated oracle; at least one of them must fail.  Everything here runs on the
CPU; nothing reaches the GPU path.
"""
import math

import numpy as np
import pytest

import tests.test_oracle_pins as pins
from oracle import pblock_oracle as orc

PIN_CALLS = [
    lambda: pins.test_layer_norm_unit_affine_moments(),
    lambda: pins.test_layer_norm_matches_torch(),
    lambda: pins.test_layer_norm_backward_matches_torch_autograd(),
    lambda: pins.test_gelu_matches_torch(True),
    lambda: pins.test_gelu_grad_matches_autograd_and_fixed_points(True),
    lambda: pins.test_gelu_matches_torch(False),
    lambda: pins.test_gelu_grad_matches_autograd_and_fixed_points(False),
    lambda: pins.test_attention_brute_force(5),
    lambda: pins.test_attention_window_one_is_identity(),
    lambda: pins.test_attention_full_window_is_causal_sdpa(16),
    lambda: pins.test_attention_zero_query_is_sliding_mean(3),
    lambda: pins.test_window_edge_is_exactly_w_keys(),
    lambda: pins.test_zero_out_projection_leaves_residual(),
    lambda: pins.test_branches_add(),
    lambda: pins.test_without_attention_equals_serial_mlp_block(),
    lambda: pins.test_causal_locality(3, 7),
    lambda: pins.test_block_matches_torch_autograd(3, True),
    lambda: pins.test_block_matches_torch_autograd(5, False),
]


def count_failures():
    bad = 0
    for call in PIN_CALLS:
        try:
            call()
        except (AssertionError, ValueError, IndexError):
            bad += 1
    return bad


def _mask_off_by_one(seq, window):
    i = np.arange(seq)[:, None]
    j = np.arange(seq)[None, :]
    return (i - j >= 0) & (i - j <= window)


def _head_forward_no_scale(q, k, v, window):
    S, d = q.shape
    s = np.where(orc.window_mask(S, window), q @ k.T, -np.inf)
    m = s.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(s - m).sum(axis=1))
    return np.exp(s - lse[:, None]) @ v, lse


def _layer_norm_unbiased(x, gamma, beta, eps):
    mean = x.mean(axis=-1, keepdims=True)
    var = x.var(axis=-1, ddof=1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mean) * rstd
    return gamma * xhat + beta, xhat, mean[..., 0], rstd[..., 0]


def _layer_norm_eps_outside(x, gamma, beta, eps):
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / (np.sqrt(var) + eps)
    xhat = (x - mean) * rstd
    return gamma * xhat + beta, xhat, mean[..., 0], rstd[..., 0]


def _ln_backward_dropped_term(dh, xhat, rstd, gamma):
    lead = tuple(range(dh.ndim - 1))
    g = gamma * dh
    dx = rstd[..., None] * (g - g.mean(axis=-1, keepdims=True))
    return dx, (dh * xhat).sum(axis=lead), dh.sum(axis=lead)


def _gelu_no_cubic(u, tanh_form=True):
    if tanh_form:
        return 0.5 * u * (1.0 + np.tanh(orc.SQRT_2_OVER_PI * u))
    return ORIGINAL_GELU(u, False)


def _gelu_grad_sign(u, tanh_form=True):
    if tanh_form:
        a = orc.SQRT_2_OVER_PI * (u + orc.GELU_TANH_COEF * u ** 3)
        t = np.tanh(a)
        da = orc.SQRT_2_OVER_PI * (1.0 + 3.0 * orc.GELU_TANH_COEF * u ** 2)
        return 0.5 * (1.0 + t) - 0.5 * u * (1.0 - t * t) * da
    return ORIGINAL_GELU_GRAD(u, False)


def _head_backward(variant):
    def f(q, k, v, do, window):
        S, d = q.shape
        s = np.where(orc.window_mask(S, window), (q @ k.T) / math.sqrt(d), -np.inf)
        e = np.exp(s - s.max(axis=1, keepdims=True))
        p = e / e.sum(axis=1, keepdims=True)
        dv = p.T @ do
        dp = do @ v.T
        if variant == "no_rowsum":
            ds = p * dp
        else:
            ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
        dq = (ds @ k) / math.sqrt(d)
        dk = ((ds @ q) if variant == "transposed" else (ds.T @ q)) / math.sqrt(d)
        return dq, dk, dv
    return f


def _forward_dropped_attention_residual(cfg, x, gamma, beta, w_in, b_in, w_out, b_out):
    y, cache = ORIGINAL_FORWARD(cfg, x, gamma, beta, w_in, b_in, w_out, b_out)
    A = cfg.attn_width
    return y - cache["o"] @ w_out[:, :A].T, cache


ORIGINAL_FORWARD = orc.block_forward
ORIGINAL_GELU = orc.gelu
ORIGINAL_GELU_GRAD = orc.gelu_grad

MUTATIONS = {
    "window_edge_off_by_one": ("window_mask", _mask_off_by_one),
    "missing_score_scale": ("swa_head_forward", _head_forward_no_scale),
    "unbiased_variance": ("layer_norm", _layer_norm_unbiased),
    "eps_outside_root": ("layer_norm", _layer_norm_eps_outside),
    "ln_backward_dropped_term": ("layer_norm_backward", _ln_backward_dropped_term),
    "gelu_dropped_cubic": ("gelu", _gelu_no_cubic),
    "gelu_grad_wrong_sign": ("gelu_grad", _gelu_grad_sign),
    "softmax_backward_no_rowsum": ("swa_head_backward", _head_backward("no_rowsum")),
    "dk_transposed_operand": ("swa_head_backward", _head_backward("transposed")),
    "dropped_attention_branch": ("block_forward", _forward_dropped_attention_residual),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, bad = MUTATIONS[name]
    monkeypatch.setattr(orc, attr, bad)
    assert count_failures() >= 1, f"no pin caught the planted mistake {name}"


def test_unmutated_oracle_passes_every_pin():
    assert count_failures() == 0

"""Pins for the LAMB-step oracle, each independent of the oracle's code:

* the first step from zero weights is exactly an Adam step, and the moment
  buffers follow torch.optim.Adam's state over several steps (the library's
  implementation of the same recursion);
* the trust ratio's defining property: the update's norm is lr times the
  weight norm;
* closed forms: pure weight decay, a constant gradient under bias correction,
  the first step without bias correction, a zero step;
* scale equivariance in the weights and independence of the tensors.

A second part plants plausible mistakes in the oracle and checks that the
pins catch each one.
"""
import numpy as np
import pytest
import torch

from oracle import lamb_oracle as lo


def rand(seed, n=257, scale=1.0):
    return scale * np.random.default_rng(seed).standard_normal(n)


def test_first_step_from_zero_weights_is_adam():
    """||w|| = 0 gives ratio 1, so LAMB's first step is Adam's (decay acts on
    w = 0 and adds nothing)."""
    cfg = lo.LambConfig(lr=0.01, beta1=0.8, beta2=0.95, eps=1e-3, step=1)
    g = rand(1, scale=1e-3)
    w1, m1, v1, r = lo.lamb_tensor(cfg, np.zeros_like(g), g, np.zeros_like(g),
                                   np.zeros_like(g), weight_decay=0.05)
    p = torch.zeros(g.size, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=0.01, betas=(0.8, 0.95), eps=1e-3)
    p.grad = torch.from_numpy(g.copy())
    opt.step()
    assert r == 1.0
    np.testing.assert_allclose(w1, p.detach().numpy(), rtol=1e-12, atol=1e-15)


def test_moments_follow_torch_adam_state():
    """Five steps with grad_scale = 0.5: m and v match the Adam state kept by
    torch for gradients pre-scaled by 0.5 (its moments do not depend on w
    when weight decay is 0)."""
    n = 100
    w = rand(2, n)
    m = np.zeros(n)
    v = np.zeros(n)
    p = torch.tensor(w.copy(), requires_grad=True)
    opt = torch.optim.Adam([p], lr=1e-3, betas=(0.9, 0.99), eps=1e-8)
    for t in range(1, 6):
        g = rand(10 + t, n)
        cfg = lo.LambConfig(lr=1e-3, beta1=0.9, beta2=0.99, eps=1e-8, step=t, grad_scale=0.5)
        w, m, v, _ = lo.lamb_tensor(cfg, w, g, m, v, 0.01)
        p.grad = torch.from_numpy(0.5 * g)
        opt.step()
    st = opt.state[p]
    np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=1e-16)


@pytest.mark.parametrize("wd,t,bc", [(0.0, 1, True), (0.01, 7, True), (0.3, 3, False)])
def test_update_norm_is_lr_times_weight_norm(wd, t, bc):
    cfg = lo.LambConfig(lr=0.02, step=t, bias_correction=bc)
    w = rand(3)
    g, m, v = rand(4), rand(5, scale=0.1), np.abs(rand(6, scale=0.1))
    w1, _, _, r = lo.lamb_tensor(cfg, w, g, m, v, wd)
    assert np.linalg.norm(w1 - w) == pytest.approx(0.02 * np.linalg.norm(w), rel=1e-12)
    assert r > 0


def test_pure_weight_decay_shrinks_by_lr():
    """g = m = v = 0: u = lambda w, ratio = 1 / lambda, so w' = (1 - lr) w."""
    cfg = lo.LambConfig(lr=0.05, step=4)
    w = rand(7)
    z = np.zeros_like(w)
    w1, m1, v1, r = lo.lamb_tensor(cfg, w, z, z, z, weight_decay=0.1)
    np.testing.assert_allclose(w1, 0.95 * w, rtol=1e-13)
    assert r == pytest.approx(10.0, rel=1e-13)
    assert not m1.any() and not v1.any()


def test_constant_gradient_closed_form():
    """With a constant gradient from zero moments, bias correction gives
    m^ = g and v^ = g^2 at every step, so u = g / (|g| + eps) and each step
    moves w by lr ||w|| along -u / ||u||."""
    eps = 1e-2
    g = rand(8, scale=0.05)
    u = g / (np.abs(g) + eps)
    w = rand(9)
    m = v = np.zeros_like(g)
    for t in range(1, 6):
        cfg = lo.LambConfig(lr=0.1, beta1=0.7, beta2=0.9, eps=eps, step=t)
        expect = w - 0.1 * np.linalg.norm(w) * u / np.linalg.norm(u)
        w, m, v, _ = lo.lamb_tensor(cfg, w, g, m, v, 0.0)
        np.testing.assert_allclose(w, expect, rtol=1e-12, atol=1e-14)


def test_first_step_without_bias_correction():
    eps, b1, b2 = 1e-3, 0.9, 0.99
    cfg = lo.LambConfig(lr=0.01, beta1=b1, beta2=b2, eps=eps, step=1, bias_correction=False)
    g = rand(10, scale=0.01)
    w = rand(11)
    u = (1 - b1) * g / (np.sqrt(1 - b2) * np.abs(g) + eps)
    z = np.zeros_like(g)
    w1, _, _, _ = lo.lamb_tensor(cfg, w, g, z, z, 0.0)
    np.testing.assert_allclose(w1, w - 0.01 * np.linalg.norm(w) / np.linalg.norm(u) * u,
                               rtol=1e-12)


def test_zero_step_leaves_weights():
    cfg = lo.LambConfig(step=2)
    w = rand(12)
    z = np.zeros_like(w)
    w1, _, _, r = lo.lamb_tensor(cfg, w, z, z, z, 0.0)
    assert r == 1.0
    assert np.array_equal(w1, w)


def test_scale_equivariance_in_the_weights():
    """Without weight decay u does not depend on w and the ratio scales with
    ||w||, so scaling w scales w' by the same factor."""
    cfg = lo.LambConfig(lr=0.03, step=5)
    w, g, m, v = rand(13), rand(14), rand(15, scale=0.1), np.abs(rand(16, scale=0.1))
    a, *_ = lo.lamb_tensor(cfg, w, g, m, v, 0.0)
    b, *_ = lo.lamb_tensor(cfg, 3.0 * w, g, m, v, 0.0)
    np.testing.assert_allclose(b, 3.0 * a, rtol=1e-12)


def test_tensors_are_independent():
    """One call over two tensors equals two calls over one: each tensor has
    its own trust ratio."""
    cfg = lo.LambConfig(lr=0.01, step=3)
    ws = [rand(20, 300), 5.0 * rand(21, 40)]
    gs = [rand(22, 300), 0.01 * rand(23, 40)]
    ms = [rand(24, 300, 0.1), rand(25, 40, 0.1)]
    vs = [np.abs(rand(26, 300, 0.1)), np.abs(rand(27, 40, 0.1))]
    wds = [0.01, 0.0]
    jw, jm, jv, jr = lo.lamb_step(cfg, ws, gs, ms, vs, wds)
    for i in range(2):
        w1, m1, v1, r = lo.lamb_tensor(cfg, ws[i], gs[i], ms[i], vs[i], wds[i])
        np.testing.assert_array_equal(jw[i], w1)
        assert jr[i] == r
    # and the two ratios differ (so a shared norm would be visible)
    assert abs(jr[0] - jr[1]) > 1e-3 * max(jr)


# ----------------------------------------------------------- planted mistakes
PINS = [
    test_first_step_from_zero_weights_is_adam,
    test_moments_follow_torch_adam_state,
    lambda: test_update_norm_is_lr_times_weight_norm(0.01, 7, True),
    test_pure_weight_decay_shrinks_by_lr,
    test_constant_gradient_closed_form,
    test_first_step_without_bias_correction,
    test_zero_step_leaves_weights,
    test_scale_equivariance_in_the_weights,
    test_tensors_are_independent,
]


def _failures():
    bad = 0
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            bad += 1
    return bad


def _dir_eps_inside(cfg, m1, v1, w, wd):
    c1 = 1 - cfg.beta1 ** cfg.step if cfg.bias_correction else 1.0
    c2 = 1 - cfg.beta2 ** cfg.step if cfg.bias_correction else 1.0
    return (m1 / c1) / np.sqrt(v1 / c2 + cfg.eps) + wd * w


def _dir_no_bias_correction(cfg, m1, v1, w, wd):
    return m1 / (np.sqrt(v1) + cfg.eps) + wd * w


def _dir_no_sqrt(cfg, m1, v1, w, wd):
    c1 = 1 - cfg.beta1 ** cfg.step if cfg.bias_correction else 1.0
    c2 = 1 - cfg.beta2 ** cfg.step if cfg.bias_correction else 1.0
    return (m1 / c1) / (v1 / c2 + cfg.eps) + wd * w


def _moments_swapped_betas(cfg, g, m, v):
    return cfg.beta2 * m + (1 - cfg.beta2) * g, cfg.beta1 * v + (1 - cfg.beta1) * g * g


def _ratio_inverted(w, u):
    wn, un = np.linalg.norm(w), np.linalg.norm(u)
    return un / wn if wn > 0 and un > 0 else 1.0


def _decay_outside_ratio(cfg, w, grad, m, v, weight_decay=0.0):
    g = cfg.grad_scale * np.asarray(grad, np.float64)
    m1, v1 = lo.moments(cfg, g, m, v)
    r = lo.direction(cfg, m1, v1, w, 0.0)
    ratio = lo.trust_ratio(w, r)
    return w - cfg.lr * (ratio * r + weight_decay * w), m1, v1, ratio


def _global_norm_step(cfg, params, grads, ms, vs, wds):
    g = [cfg.grad_scale * np.asarray(x) for x in grads]
    mv = [lo.moments(cfg, gi, mi, vi) for gi, mi, vi in zip(g, ms, vs)]
    us = [lo.direction(cfg, m1, v1, w, wd) for (m1, v1), w, wd in zip(mv, params, wds)]
    wn = np.sqrt(sum(np.sum(w * w) for w in params))
    un = np.sqrt(sum(np.sum(u * u) for u in us))
    r = wn / un
    return ([w - cfg.lr * r * u for w, u in zip(params, us)], [a for a, _ in mv],
            [b for _, b in mv], [r] * len(params))


MUTATIONS = {
    "eps inside the square root": ("direction", _dir_eps_inside),
    "no bias correction": ("direction", _dir_no_bias_correction),
    "no square root on v": ("direction", _dir_no_sqrt),
    "betas swapped": ("moments", _moments_swapped_betas),
    "trust ratio inverted": ("trust_ratio", _ratio_inverted),
    "decay outside the trust ratio": ("lamb_tensor", _decay_outside_ratio),
    "one norm over all tensors": ("lamb_step", _global_norm_step),
}


def test_pins_pass_on_the_oracle():
    assert _failures() == 0


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(lo, attr, fn)
    assert _failures() >= 1, f"no pin caught: {name}"

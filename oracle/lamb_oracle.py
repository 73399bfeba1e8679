"""CPU oracle for one LAMB optimizer step over a list of tensors, in float64.

TEST INFRASTRUCTURE ONLY, under the same rules as pblock_oracle: only the
tests, the smoke check and the benchmark's CPU-baseline leg may import it.

The paper trains with LAMB (Section 3.1, "LAMB optimizer") to scale the batch
size; it cites You et al. (2020), whose layer-wise algorithm (LAMB, their
Algorithm 2) is what this computes.  Each tensor is one "layer" of the trust
ratio.  For a tensor w with gradient grad, first and second moments m, v and
step number t >= 1:

    g   = grad_scale * grad
    m'  = beta1 m + (1 - beta1) g
    v'  = beta2 v + (1 - beta2) g^2
    m^  = m' / (1 - beta1^t),  v^ = v' / (1 - beta2^t)   (bias correction;
                                                          m^ = m', v^ = v'
                                                          when it is off)
    u   = m^ / (sqrt(v^) + eps) + lambda w
    ratio = ||w|| / ||u||  (Euclidean norms over the whole tensor; 1 when
                            either norm is 0: the scaling function of the
                            algorithm taken as the identity)
    w'  = w - lr * ratio * u

Readings where the cited algorithm leaves a choice: the scaling function is
the identity, eps sits outside the square root (as in Adam), the weight
decay term enters u before the norm is taken, and grad_scale (for example
the inverse of a loss scale or of a micro-batch count) multiplies the
gradient before anything else.
"""
from __future__ import annotations

import numpy as np

__all__ = ["LambConfig", "moments", "direction", "trust_ratio", "lamb_tensor", "lamb_step"]


class LambConfig:
    def __init__(self, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, step=1, bias_correction=True,
                 grad_scale=1.0):
        self.lr, self.beta1, self.beta2, self.eps = lr, beta1, beta2, eps
        self.step, self.bias_correction, self.grad_scale = step, bias_correction, grad_scale


def moments(cfg: LambConfig, g, m, v):
    """Exponential moving averages of g and g^2."""
    m1 = cfg.beta1 * m + (1.0 - cfg.beta1) * g
    v1 = cfg.beta2 * v + (1.0 - cfg.beta2) * g * g
    return m1, v1


def direction(cfg: LambConfig, m1, v1, w, weight_decay):
    """The Adam-style direction with bias correction, plus weight decay."""
    if cfg.bias_correction:
        mh = m1 / (1.0 - cfg.beta1 ** cfg.step)
        vh = v1 / (1.0 - cfg.beta2 ** cfg.step)
    else:
        mh, vh = m1, v1
    return mh / (np.sqrt(vh) + cfg.eps) + weight_decay * w


def trust_ratio(w, u):
    wn = float(np.sqrt(np.sum(w * w)))
    un = float(np.sqrt(np.sum(u * u)))
    return wn / un if wn > 0.0 and un > 0.0 else 1.0


def lamb_tensor(cfg: LambConfig, w, grad, m, v, weight_decay=0.0):
    """One tensor's step.  Returns (w', m', v', ratio)."""
    w = np.asarray(w, np.float64)
    g = cfg.grad_scale * np.asarray(grad, np.float64)
    m1, v1 = moments(cfg, g, np.asarray(m, np.float64), np.asarray(v, np.float64))
    u = direction(cfg, m1, v1, w, weight_decay)
    r = trust_ratio(w, u)
    return w - cfg.lr * r * u, m1, v1, r


def lamb_step(cfg: LambConfig, params, grads, ms, vs, weight_decays):
    """The step over a list of tensors (each with its own trust ratio).
    Returns lists (params', m', v') and the list of ratios."""
    out_w, out_m, out_v, ratios = [], [], [], []
    for w, g, m, v, wd in zip(params, grads, ms, vs, weight_decays):
        w1, m1, v1, r = lamb_tensor(cfg, w, g, m, v, wd)
        out_w.append(w1)
        out_m.append(m1)
        out_v.append(v1)
        ratios.append(r)
    return out_w, out_m, out_v, ratios

"""Seeded synthetic inputs for the parallel transformer block.

This module is shared by the GPU path and by the CPU oracle, and holds none of
the block's arithmetic: it only draws random tensors and rounds them to the
storage type.  The paper's training data is proprietary; the block needs none
of it, so every tensor here is a seeded normal draw with the shapes of the
models in the paper's Table 1 (and the 13B model of its convergence study).

Draw order for one workload is fixed: x, gamma, beta, W_in, b_in, W_out,
b_out, dy, each from ``numpy.random.default_rng(seed)`` as float64, then cast
to float32 and (for bf16 workloads) rounded to bf16 with round-to-nearest-even.
The returned arrays are float32 and, for bf16 workloads, exactly representable
in bf16, so both sides of a parity test start from identical values.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class BlockShape:
    """Shape of one parallel transformer block and its synthetic draw.

    ``window`` counts the keys a query sees, itself included; a window of at
    least ``seq`` is full causal attention.
    """

    name: str
    batch: int
    seq: int
    hidden: int
    heads: int
    head_dim: int
    ffn: int
    window: int
    dtype: str  # "bf16" or "f32"
    w_std: float = 0.02
    gamma_std: float = 0.01
    beta_std: float = 0.01
    x_std: float = 1.0
    dy_std: float = 1.0
    ln_eps: float = 1e-5
    gelu_tanh: bool = True

    @property
    def tokens(self) -> int:
        return self.batch * self.seq

    @property
    def attn_width(self) -> int:
        return self.heads * self.head_dim

    @property
    def n_in(self) -> int:
        """Width of the fused in-projection: Q | K | V | MLP-up."""
        return 3 * self.attn_width + self.ffn

    @property
    def k_out(self) -> int:
        """Width of the fused out-projection input: attention out | GeLU out."""
        return self.attn_width + self.ffn

    def with_(self, **kw) -> "BlockShape":
        return replace(self, **kw)


def visible_pairs(seq: int, window: int) -> int:
    """Number of (query, key) pairs one head attends to under a causal window."""
    if window >= seq:
        return seq * (seq + 1) // 2
    return seq * window - window * (window - 1) // 2


def model_flops(s: BlockShape) -> int:
    """Forward+backward model FLOPs of one block: the six projection GEMMs plus
    the four attention contractions over visible pairs only (no recompute, no
    elementwise work)."""
    T, H = s.tokens, s.hidden
    gemm = 2 * T * H * s.n_in + 2 * T * s.k_out * H
    attn = 4 * s.batch * s.attn_width * visible_pairs(s.seq, s.window)
    return 3 * (gemm + attn)


# Workloads: shapes of the paper's Table 1 models and its 13B study model.
WORKLOADS: dict[str, BlockShape] = {
    s.name: s
    for s in [
        BlockShape("tiny_f32", 1, 128, 256, 4, 64, 1024, 64, "f32",
                   w_std=0.02, gamma_std=0.0, beta_std=0.0),
        BlockShape("13b_shape", 1, 2048, 5120, 40, 128, 20480, 512, "bf16",
                   w_std=0.02),
        BlockShape("175b_tp8_share", 1, 2048, 12288, 12, 128, 6144, 2048, "bf16",
                   w_std=0.006),
        BlockShape("175b_tp8_share_w512", 1, 2048, 12288, 12, 128, 6144, 512, "bf16",
                   w_std=0.006),
        BlockShape("long_seq_8k", 1, 8192, 5120, 40, 128, 20480, 1024, "bf16",
                   w_std=0.02),
        BlockShape("175b_full", 1, 2048, 12288, 96, 128, 49152, 2048, "bf16",
                   w_std=0.006),
        # Table 1's literal 175B heads (128 x 96): one of 8 ranks holds 16
        BlockShape("175b_tp8_share_d96", 1, 2048, 12288, 16, 96, 6144, 2048, "bf16",
                   w_std=0.006),
        BlockShape("175b_full_d96", 1, 2048, 12288, 128, 96, 49152, 2048, "bf16",
                   w_std=0.006),
    ]
}


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32.

    NaN is kept quiet; infinities and values that overflow become infinities,
    as the IEEE rounding rule gives.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    r = r.astype(np.uint32)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = (a.view(np.uint32)[nan] | np.uint32(0x00400000)) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def make_inputs(s: BlockShape, seed: int = 0, serial: bool = False) -> dict[str, np.ndarray]:
    """Draw one block's inputs, parameters and upstream gradient.

    Returns float32 arrays (bf16-exact for bf16 workloads):
    x, dy [batch, seq, hidden]; gamma, beta, b_out [hidden];
    w_in [n_in, hidden] (rows Q | K | V | up, heads contiguous in each);
    b_in [n_in]; w_out [hidden, k_out] (columns attention-out | down).

    serial=True is for the serial block (two LayerNorms, two output biases):
    the same draws, renamed gamma1, beta1 and b_o, followed by gamma2, beta2
    and b_down, so both blocks share x, the weights and dy for a seed.
    """
    rng = np.random.default_rng(seed)
    H = s.hidden

    def draw(shape, std, mean=0.0):
        v = rng.standard_normal(size=shape, dtype=np.float64)
        v = (mean + std * v).astype(np.float32)
        return round_to_bf16(v) if s.dtype == "bf16" else v

    out = {}
    out["x"] = draw((s.batch, s.seq, H), s.x_std)
    out["gamma"] = draw((H,), s.gamma_std, 1.0)
    out["beta"] = draw((H,), s.beta_std)
    out["w_in"] = draw((s.n_in, H), s.w_std)
    out["b_in"] = draw((s.n_in,), s.w_std)
    out["w_out"] = draw((H, s.k_out), s.w_std)
    out["b_out"] = draw((H,), s.w_std)
    out["dy"] = draw((s.batch, s.seq, H), s.dy_std)
    if serial:
        out["gamma1"] = out.pop("gamma")
        out["beta1"] = out.pop("beta")
        out["b_o"] = out.pop("b_out")
        out["gamma2"] = draw((H,), s.gamma_std, 1.0)
        out["beta2"] = draw((H,), s.beta_std)
        out["b_down"] = draw((H,), s.w_std)
    return out


def block_param_shapes(s: BlockShape) -> dict[str, tuple]:
    """Parameter shapes of the parallel block, in the library's packed layout."""
    H = s.hidden
    return {"w_in": (s.n_in, H), "b_in": (s.n_in,), "w_out": (H, s.k_out), "b_out": (H,),
            "gamma": (H,), "beta": (H,)}


def make_lamb_state(shapes: dict, seed: int = 0, w_std: float = 0.02,
                    g_std: float = 1e-3) -> dict[str, dict[str, np.ndarray]]:
    """Seeded optimizer state for a LAMB step: per tensor, fp32 master
    weights w with standard deviation w_std around 0 (around 1 for
    gamma-like tensors, named "gamma*"), gradient g with standard deviation
    g_std, first moment m with g_std / 3, and second moment v = (g_std z)^2
    for a unit-variance z (non-negative, of the size a running average of
    g^2 has).  The draws are uniform with the stated standard deviation
    (uniform draws keep the full-size state, ~10^9 values, quick to make);
    tensors are drawn in the order given, each w, g, m, v in turn, from
    numpy.random.default_rng(seed)."""
    rng = np.random.default_rng(seed)
    half = np.float32(np.sqrt(3.0))  # a uniform draw on [-sqrt 3, sqrt 3] has unit variance
    out = {}
    for name, shape in shapes.items():
        def draw(std, mean=0.0):
            z = rng.random(size=shape, dtype=np.float32)
            z = (2.0 * z - 1.0) * half
            return (np.float32(mean) + np.float32(std) * z).astype(np.float32)
        w = draw(w_std, 1.0 if name.startswith("gamma") else 0.0)
        g = draw(g_std)
        m = draw(g_std / 3)
        v = np.square(draw(g_std))
        out[name] = {"w": w, "g": g, "m": m, "v": v}
    return out

"""Python binding of the C ABI in include/pblock.h (ctypes; argument
marshalling only).

Every entry point has the name of its C function and forwards to it: torch
tensors (or raw integer device addresses) become pointers, the stream defaults
to torch's current stream.  All arithmetic runs in the HIP library; there is no
fallback.  If libpblock.so is missing or cannot be loaded, loading raises
ImportError.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int, c_size_t, c_void_p

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpblock.so")

PB_BF16, PB_F32 = 0, 1
# pblock_workspace_bytes modes
WS_FORWARD_WITH_STASH, WS_BACKWARD, WS_FORWARD = 0, 1, 2
# pblock_swattn_workspace_bytes modes
ATTN_WS_FORWARD, ATTN_WS_BACKWARD_MIN, ATTN_WS_BACKWARD = 0, 1, 2
STATUS = {0: "PB_OK", 1: "PB_ERR_INVALID_ARG", 2: "PB_ERR_UNSUPPORTED", 3: "PB_ERR_WORKSPACE",
          4: "PB_ERR_HIP"}
SAVED_REGIONS = ("h", "z", "c", "mean", "rstd", "lse")
WORKSPACE_REGIONS = ("d_o", "dz", "dh", "delta")
SERIAL_SAVED_REGIONS = ("h1", "z", "c", "mean1", "rstd1", "lse", "x1", "h2", "mean2", "rstd2")

# Every function the header declares (checked by the CPU tests).
EXPORTS = (
    "pblock_validate", "pblock_saved_bytes", "pblock_saved_offsets", "pblock_workspace_bytes",
    "pblock_workspace_offsets",
    "pblock_forward", "pblock_backward", "pblock_swattn_forward",
    "pblock_swattn_workspace_bytes", "pblock_swattn_backward", "pblock_forward_timed",
    "pblock_backward_timed", "pblock_gemm_plan", "pblock_backward_pairs",
    "pblock_tp_context_create", "pblock_tp_context_destroy",
    "pblock_status_string", "pblock_last_error", "pblock_serial_saved_bytes",
    "pblock_serial_saved_offsets", "pblock_serial_workspace_bytes", "pblock_serial_forward",
    "pblock_serial_backward", "pblock_lamb_workspace_bytes", "pblock_lamb_step",
    "pblock_ag_in_proj_workspace_bytes", "pblock_ag_in_proj",
    "pblock_rs_out_proj_workspace_bytes", "pblock_rs_out_proj", "pblock_rs_reduce",
    "pblock_ag_dc_workspace_bytes", "pblock_ag_dc", "pblock_rs_dh_workspace_bytes", "pblock_rs_dh",
    "pblock_swattn_forward_noalloc",
)
NOALLOC_SCRATCH_BYTES = 32 << 20  # PB_NOALLOC_SCRATCH_BYTES
LAMB_MAX_TENSORS = 16

# pb_step order of include/pblock.h
STEPS = ("ln_fwd", "in_proj", "attn_fwd", "out_proj", "dc", "dw_out", "db_out", "attn_bwd", "dh",
         "dw_in", "db_in", "ln_bwd")


class PbConfig(ctypes.Structure):
    _fields_ = [("batch", c_int), ("seq", c_int), ("hidden", c_int), ("heads", c_int),
                ("head_dim", c_int), ("ffn", c_int), ("window", c_int), ("ln_eps", c_float),
                ("gelu_tanh", c_int), ("dtype", c_int)]


class StepEvents(ctypes.Structure):
    """pb_step_events: raw hipEvent_t handles, NULL to skip a step."""
    _fields_ = [("begin", c_void_p * len(STEPS)), ("end", c_void_p * len(STEPS))]


class GemmPlan(ctypes.Structure):
    """pb_gemm_plan."""
    _fields_ = [("tiles", c_int), ("n_full", c_int), ("tail", c_int), ("splits", c_int),
                ("workgroups", c_int), ("threads", c_int)]


class LambConfig(ctypes.Structure):
    """pb_lamb_config."""
    _fields_ = [("lr", c_float), ("beta1", c_float), ("beta2", c_float), ("eps", c_float),
                ("grad_scale", c_float), ("step", c_int), ("bias_correction", c_int)]


class LambTensor(ctypes.Structure):
    """pb_lamb_tensor (device addresses as integers)."""
    _fields_ = [("param", c_void_p), ("grad", c_void_p), ("exp_avg", c_void_p),
                ("exp_avg_sq", c_void_p), ("param_copy", c_void_p), ("numel", c_size_t),
                ("weight_decay", c_float)]


class PblockError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libpblock.so once and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run __graft_entry__.build() "
                          f"(or python -m paper_2402_15627_amd.build)")
    # torch first, when it is installed: the library then binds to the HIP
    # runtime torch has loaded, and both see the same devices and streams (a
    # library loaded before torch brought in a second runtime that reported
    # no device)
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    P = c_void_p
    cfgp = POINTER(PbConfig)
    sig = {
        "pblock_validate": (c_int, [cfgp]),
        "pblock_saved_bytes": (c_size_t, [cfgp]),
        "pblock_saved_offsets": (c_int, [cfgp, POINTER(c_size_t)]),
        "pblock_workspace_bytes": (c_size_t, [cfgp, c_int]),
        "pblock_workspace_offsets": (c_int, [cfgp, POINTER(c_size_t)]),
        "pblock_forward": (c_int, [cfgp, P, P, P, P, P, P, P, P, P, P, c_size_t, P]),
        "pblock_backward": (c_int, [cfgp, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P,
                                    c_size_t, P]),
        "pblock_swattn_forward": (c_int, [cfgp, P, P, P, c_int, P, c_int, P, P, c_size_t, P]),
        "pblock_swattn_workspace_bytes": (c_size_t, [cfgp, c_int]),
        "pblock_swattn_forward_noalloc": (c_int, [cfgp, P, P, P, c_int, P, c_int, P, P]),
        "pblock_swattn_backward": (c_int, [cfgp, P, P, P, c_int, P, c_int, P, c_int, P, P, P, P,
                                           c_int, P, c_size_t, P]),
        "pblock_forward_timed": (c_int, [cfgp, P, P, P, P, P, P, P, P, P, P, c_size_t, P,
                                         POINTER(StepEvents)]),
        "pblock_backward_timed": (c_int, [cfgp, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P,
                                          P, c_size_t, P, POINTER(StepEvents)]),
        "pblock_gemm_plan": (c_int, [c_int, c_int, c_int, c_int, POINTER(GemmPlan)]),
        "pblock_backward_pairs": (c_int, [cfgp, c_int, POINTER(c_int)]),
        "pblock_tp_context_create": (c_int, [c_int, POINTER(c_void_p)]),
        "pblock_tp_context_destroy": (None, [P]),
        "pblock_status_string": (ctypes.c_char_p, [c_int]),
        "pblock_last_error": (ctypes.c_char_p, []),
        "pblock_serial_saved_bytes": (c_size_t, [cfgp]),
        "pblock_serial_saved_offsets": (c_int, [cfgp, POINTER(c_size_t)]),
        "pblock_serial_workspace_bytes": (c_size_t, [cfgp, c_int]),
        "pblock_serial_forward": (c_int, [cfgp] + [P] * 13 + [c_size_t, P]),
        "pblock_serial_backward": (c_int, [cfgp] + [P] * 23 + [c_size_t, P]),
        "pblock_lamb_workspace_bytes": (c_size_t, [c_int, POINTER(LambTensor)]),
        "pblock_ag_in_proj_workspace_bytes": (c_size_t, [cfgp, c_int, c_int]),
        "pblock_ag_in_proj": (c_int, [cfgp, c_int, c_int, POINTER(c_void_p), P, P, P, P, P, c_int,
                                      P, c_size_t, P, c_int, POINTER(c_void_p), P]),
        "pblock_rs_out_proj_workspace_bytes": (c_size_t, [cfgp, c_int, c_int]),
        "pblock_rs_out_proj": (c_int, [cfgp, c_int, c_int, P, P, P, POINTER(c_void_p), c_int, P,
                                       c_size_t, P, c_int, POINTER(c_void_p), P]),
        "pblock_rs_reduce": (c_int, [cfgp, c_int, POINTER(c_void_p), P, P, P, P]),
        "pblock_ag_dc_workspace_bytes": (c_size_t, [cfgp, c_int, c_int]),
        "pblock_ag_dc": (c_int, [cfgp, c_int, c_int, POINTER(c_void_p), P, P, P, P, P, c_int, P,
                                 c_size_t, P, c_int, POINTER(c_void_p), P]),
        "pblock_rs_dh_workspace_bytes": (c_size_t, [cfgp, c_int, c_int]),
        "pblock_rs_dh": (c_int, [cfgp, c_int, c_int, P, P, P, POINTER(c_void_p), c_int, P,
                                 c_size_t, P, c_int, POINTER(c_void_p), P]),
        "pblock_lamb_step": (c_int, [POINTER(LambConfig), c_int, POINTER(LambTensor), c_int, P, P,
                                     c_size_t, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


# ------------------------------------------------------------- marshalling
def _ptr(t):
    """Device address of a tensor, an int address, or None -> NULL."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def _check(status: int):
    if status != 0:
        raise PblockError(status, pblock_last_error())


def make_config(batch, seq, hidden, heads, head_dim, ffn, window, dtype="bf16", ln_eps=1e-5,
                gelu_tanh=True) -> PbConfig:
    return PbConfig(batch, seq, hidden, heads, head_dim, ffn, window, ln_eps, int(bool(gelu_tanh)),
                    PB_BF16 if dtype == "bf16" else PB_F32)


def config_from_shape(s) -> PbConfig:
    """PbConfig from any object with the block's shape fields (e.g. inputs.BlockShape)."""
    return make_config(s.batch, s.seq, s.hidden, s.heads, s.head_dim, s.ffn, s.window, s.dtype,
                       s.ln_eps, s.gelu_tanh)


# ------------------------------------------------------------ entry points
def pblock_validate(cfg: PbConfig) -> int:
    return load_library().pblock_validate(ctypes.byref(cfg))


def pblock_saved_bytes(cfg: PbConfig) -> int:
    return load_library().pblock_saved_bytes(ctypes.byref(cfg))


def pblock_saved_offsets(cfg: PbConfig) -> dict:
    arr = (c_size_t * 6)()
    _check(load_library().pblock_saved_offsets(ctypes.byref(cfg), arr))
    return dict(zip(SAVED_REGIONS, list(arr)))


def pblock_workspace_bytes(cfg: PbConfig, mode: int) -> int:
    """mode: WS_FORWARD, WS_FORWARD_WITH_STASH or WS_BACKWARD."""
    return load_library().pblock_workspace_bytes(ctypes.byref(cfg), int(mode))


def pblock_workspace_offsets(cfg: PbConfig) -> dict:
    """Offsets of d_o, dz, dh and delta in the backward workspace."""
    arr = (c_size_t * len(WORKSPACE_REGIONS))()
    _check(load_library().pblock_workspace_offsets(ctypes.byref(cfg), arr))
    return dict(zip(WORKSPACE_REGIONS, list(arr)))


def step_events(begin, end) -> StepEvents:
    """A pb_step_events from two sequences of len(STEPS) raw hipEvent_t
    handles (ints; 0 or None skips a step)."""
    n = len(STEPS)
    if len(begin) != n or len(end) != n:
        raise ValueError(f"step events need {n} begin and {n} end handles")
    ev = StepEvents()
    for i in range(n):
        ev.begin[i] = begin[i] or None
        ev.end[i] = end[i] or None
    return ev


def pblock_forward(cfg, x, ln_gamma, ln_beta, w_in, b_in, w_out, b_out, y, saved=None, ws=None,
                   stream=None, step_ev=None):
    """step_ev: None, or a StepEvents (see step_events) recorded around each
    step (pblock_forward_timed)."""
    args = (ctypes.byref(cfg), _ptr(x), _ptr(ln_gamma), _ptr(ln_beta), _ptr(w_in), _ptr(b_in),
            _ptr(w_out), _ptr(b_out), _ptr(y), _ptr(saved), _ptr(ws), _nbytes(ws),
            _stream(stream))
    lib = load_library()
    if step_ev is None:
        _check(lib.pblock_forward(*args))
    else:
        _check(lib.pblock_forward_timed(*args, ctypes.byref(step_ev)))


def pblock_backward(cfg, x, ln_gamma, ln_beta, w_in, b_in, w_out, b_out, saved, dy, dx, dgamma,
                    dbeta, dw_in, db_in, dw_out, db_out, ws, stream=None, step_ev=None):
    """step_ev as for pblock_forward (pblock_backward_timed)."""
    args = (ctypes.byref(cfg), _ptr(x), _ptr(ln_gamma), _ptr(ln_beta), _ptr(w_in), _ptr(b_in),
            _ptr(w_out), _ptr(b_out), _ptr(saved), _ptr(dy), _ptr(dx), _ptr(dgamma), _ptr(dbeta),
            _ptr(dw_in), _ptr(db_in), _ptr(dw_out), _ptr(db_out), _ptr(ws), _nbytes(ws),
            _stream(stream))
    lib = load_library()
    if step_ev is None:
        _check(lib.pblock_backward(*args))
    else:
        _check(lib.pblock_backward_timed(*args, ctypes.byref(step_ev)))


def pblock_gemm_plan(dtype: int, M: int, N: int, K: int) -> GemmPlan:
    """The launch of one GEMM as the library makes it (host only)."""
    plan = GemmPlan()
    _check(load_library().pblock_gemm_plan(int(dtype), int(M), int(N), int(K),
                                           ctypes.byref(plan)))
    return plan


def pblock_backward_pairs(cfg: PbConfig, block: str = "parallel") -> tuple:
    """Which backward GEMMs share a launch with the weight gradient after them
    (host only): parallel (dC+dW_out, dh+dW_in); serial (dG+dW_down,
    dh2+dW_up, dO+dW_o, dh1+dW_qkv)."""
    n = 2 if block == "parallel" else 4
    out = (c_int * n)()
    _check(load_library().pblock_backward_pairs(ctypes.byref(cfg), 0 if block == "parallel" else 1,
                                                out))
    return tuple(bool(v) for v in out)


class TpContext:
    """A pb_tp_context: the events of the pipelined all-gather and
    reduce-scatter calls for one tp on the current device."""

    def __init__(self, tp: int):
        h = c_void_p()
        _check(load_library().pblock_tp_context_create(int(tp), ctypes.byref(h)))
        self.tp = int(tp)
        self.handle = h.value

    def close(self):
        if self.handle:
            load_library().pblock_tp_context_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def pblock_swattn_forward(cfg, q, k, v, ld_qkv, o, ld_o, lse, ws=None, stream=None):
    _check(load_library().pblock_swattn_forward(
        ctypes.byref(cfg), _ptr(q), _ptr(k), _ptr(v), ld_qkv, _ptr(o), ld_o, _ptr(lse), _ptr(ws),
        _nbytes(ws), _stream(stream)))


def pblock_swattn_forward_noalloc(cfg, q, k, v, ld_qkv, o, ld_o, lse, stream=None):
    _check(load_library().pblock_swattn_forward_noalloc(
        ctypes.byref(cfg), _ptr(q), _ptr(k), _ptr(v), ld_qkv, _ptr(o), ld_o, _ptr(lse),
        _stream(stream)))


def pblock_swattn_workspace_bytes(cfg, mode: int) -> int:
    """mode: ATTN_WS_FORWARD, ATTN_WS_BACKWARD_MIN or ATTN_WS_BACKWARD."""
    return load_library().pblock_swattn_workspace_bytes(ctypes.byref(cfg), int(mode))


def pblock_swattn_backward(cfg, q, k, v, ld_qkv, o, ld_o, d_o, ld_do, lse, dq, dk, dv, ld_dqkv,
                           ws, stream=None):
    _check(load_library().pblock_swattn_backward(
        ctypes.byref(cfg), _ptr(q), _ptr(k), _ptr(v), ld_qkv, _ptr(o), ld_o, _ptr(d_o), ld_do,
        _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv), ld_dqkv, _ptr(ws), _nbytes(ws),
        _stream(stream)))


def pblock_serial_saved_bytes(cfg: PbConfig) -> int:
    return load_library().pblock_serial_saved_bytes(ctypes.byref(cfg))


def pblock_serial_saved_offsets(cfg: PbConfig) -> dict:
    arr = (c_size_t * len(SERIAL_SAVED_REGIONS))()
    _check(load_library().pblock_serial_saved_offsets(ctypes.byref(cfg), arr))
    return dict(zip(SERIAL_SAVED_REGIONS, list(arr)))


def pblock_serial_workspace_bytes(cfg: PbConfig, mode: int) -> int:
    """mode: WS_FORWARD, WS_FORWARD_WITH_STASH or WS_BACKWARD."""
    return load_library().pblock_serial_workspace_bytes(ctypes.byref(cfg), int(mode))


def pblock_serial_forward(cfg, x, ln1_gamma, ln1_beta, ln2_gamma, ln2_beta, w_in, b_in, w_out,
                          b_o, b_down, y, saved=None, ws=None, stream=None):
    _check(load_library().pblock_serial_forward(
        ctypes.byref(cfg), _ptr(x), _ptr(ln1_gamma), _ptr(ln1_beta), _ptr(ln2_gamma),
        _ptr(ln2_beta), _ptr(w_in), _ptr(b_in), _ptr(w_out), _ptr(b_o), _ptr(b_down), _ptr(y),
        _ptr(saved), _ptr(ws), _nbytes(ws), _stream(stream)))


def pblock_serial_backward(cfg, x, ln1_gamma, ln1_beta, ln2_gamma, ln2_beta, w_in, b_in, w_out,
                           b_o, b_down, saved, dy, dx, dln1_gamma, dln1_beta, dln2_gamma,
                           dln2_beta, dw_in, db_in, dw_out, db_o, db_down, ws, stream=None):
    _check(load_library().pblock_serial_backward(
        ctypes.byref(cfg), _ptr(x), _ptr(ln1_gamma), _ptr(ln1_beta), _ptr(ln2_gamma),
        _ptr(ln2_beta), _ptr(w_in), _ptr(b_in), _ptr(w_out), _ptr(b_o), _ptr(b_down),
        _ptr(saved), _ptr(dy), _ptr(dx), _ptr(dln1_gamma), _ptr(dln1_beta), _ptr(dln2_gamma),
        _ptr(dln2_beta), _ptr(dw_in), _ptr(db_in), _ptr(dw_out), _ptr(db_o), _ptr(db_down),
        _ptr(ws), _nbytes(ws), _stream(stream)))


def lamb_config(lr, beta1=0.9, beta2=0.999, eps=1e-6, step=1, bias_correction=True,
                grad_scale=1.0) -> LambConfig:
    return LambConfig(lr, beta1, beta2, eps, grad_scale, int(step), int(bool(bias_correction)))


def lamb_tensor(param, grad, exp_avg, exp_avg_sq, param_copy=None, weight_decay=0.0):
    """A pb_lamb_tensor from torch tensors (fp32 param, grad and moments of
    equal size; an optional copy of the same size)."""
    return LambTensor(_ptr(param), _ptr(grad), _ptr(exp_avg), _ptr(exp_avg_sq),
                      _ptr(param_copy), param.numel(), weight_decay)


def _lamb_array(tensors):
    arr = (LambTensor * len(tensors))(*tensors)
    return arr


def pblock_lamb_workspace_bytes(tensors) -> int:
    """tensors: a sequence of LambTensor."""
    return load_library().pblock_lamb_workspace_bytes(len(tensors), _lamb_array(tensors))


def pblock_lamb_step(cfg: LambConfig, tensors, copy_dtype=PB_BF16, trust_ratio=None, ws=None,
                     stream=None):
    _check(load_library().pblock_lamb_step(
        ctypes.byref(cfg), len(tensors), _lamb_array(tensors), int(copy_dtype),
        _ptr(trust_ratio), _ptr(ws), _nbytes(ws), _stream(stream)))


def pblock_ag_in_proj_workspace_bytes(cfg: PbConfig, tp: int, shards_per_launch: int) -> int:
    return load_library().pblock_ag_in_proj_workspace_bytes(ctypes.byref(cfg), int(tp),
                                                            int(shards_per_launch))


def pblock_ag_in_proj(cfg, tp, rank, shards, h, w_in, b_in, z, c, shards_per_launch, ws, stream,
                      comm_streams, ctx: TpContext):
    """shards: tp tensors (or addresses), rank j's rows of h; comm_streams: a
    non-empty sequence of streams other than `stream` (torch streams or raw
    handles); ctx: a TpContext for this tp on the current device."""
    if len(shards) != tp:
        raise ValueError(f"{len(shards)} shards for tp={tp}")
    arr = (c_void_p * len(shards))(*[_ptr(t) for t in shards])
    cs = (c_void_p * len(comm_streams))(*[_stream(x) for x in comm_streams])
    _check(load_library().pblock_ag_in_proj(
        ctypes.byref(cfg), int(tp), int(rank), arr, _ptr(h), _ptr(w_in), _ptr(b_in), _ptr(z),
        _ptr(c), int(shards_per_launch), _ptr(ws), _nbytes(ws), _stream(stream),
        len(comm_streams), cs, ctx.handle if ctx is not None else None))


def pblock_rs_out_proj_workspace_bytes(cfg: PbConfig, tp: int, shards_per_launch: int) -> int:
    return load_library().pblock_rs_out_proj_workspace_bytes(ctypes.byref(cfg), int(tp),
                                                             int(shards_per_launch))


def pblock_rs_out_proj(cfg, tp, rank, c, w_out, partial, dst, shards_per_launch, ws, stream,
                       comm_streams, ctx: TpContext):
    """dst: tp tensors (or addresses), where rank j receives this rank's
    chunk j; comm_streams and ctx as for pblock_ag_in_proj."""
    if len(dst) != tp:
        raise ValueError(f"{len(dst)} destinations for tp={tp}")
    arr = (c_void_p * len(dst))(*[_ptr(t) for t in dst])
    cs = (c_void_p * len(comm_streams))(*[_stream(x) for x in comm_streams])
    _check(load_library().pblock_rs_out_proj(
        ctypes.byref(cfg), int(tp), int(rank), _ptr(c), _ptr(w_out), _ptr(partial), arr,
        int(shards_per_launch), _ptr(ws), _nbytes(ws), _stream(stream), len(comm_streams), cs,
        ctx.handle if ctx is not None else None))


def pblock_ag_dc_workspace_bytes(cfg: PbConfig, tp: int, shards_per_launch: int) -> int:
    return load_library().pblock_ag_dc_workspace_bytes(ctypes.byref(cfg), int(tp),
                                                       int(shards_per_launch))


def pblock_ag_dc(cfg, tp, rank, dy_shards, dy, w_out, z, d_o, dz, shards_per_launch, ws, stream,
                 comm_streams, ctx):
    """dy_shards: tp tensors (or addresses), rank j's rows of dy; dy is the
    gathered [T, H]; comm_streams and ctx as for pblock_ag_in_proj."""
    if len(dy_shards) != tp:
        raise ValueError(f"{len(dy_shards)} shards for tp={tp}")
    arr = (c_void_p * tp)(*[_ptr(t) for t in dy_shards])
    cs = (c_void_p * len(comm_streams))(*[_stream(x) for x in comm_streams])
    _check(load_library().pblock_ag_dc(
        ctypes.byref(cfg), int(tp), int(rank), arr, _ptr(dy), _ptr(w_out), _ptr(z), _ptr(d_o),
        _ptr(dz), int(shards_per_launch), _ptr(ws), _nbytes(ws), _stream(stream),
        len(comm_streams), cs, ctx.handle if ctx is not None else None))


def pblock_rs_dh_workspace_bytes(cfg: PbConfig, tp: int, shards_per_launch: int) -> int:
    return load_library().pblock_rs_dh_workspace_bytes(ctypes.byref(cfg), int(tp),
                                                       int(shards_per_launch))


def pblock_rs_dh(cfg, tp, rank, dz, w_in, partial, dst, shards_per_launch, ws, stream,
                 comm_streams, ctx):
    """dst: tp tensors (or addresses), where rank j receives this rank's
    chunk j of the partial dh; comm_streams and ctx as for pblock_ag_in_proj."""
    if len(dst) != tp:
        raise ValueError(f"{len(dst)} destinations for tp={tp}")
    arr = (c_void_p * tp)(*[_ptr(t) for t in dst])
    cs = (c_void_p * len(comm_streams))(*[_stream(x) for x in comm_streams])
    _check(load_library().pblock_rs_dh(
        ctypes.byref(cfg), int(tp), int(rank), _ptr(dz), _ptr(w_in), _ptr(partial), arr,
        int(shards_per_launch), _ptr(ws), _nbytes(ws), _stream(stream), len(comm_streams), cs,
        ctx.handle if ctx is not None else None))


def pblock_rs_reduce(cfg, tp, parts, x_shard, b_out, y_shard, stream=None):
    """parts: tp tensors (or addresses), the chunks this rank received, in
    rank order."""
    if len(parts) != tp:
        raise ValueError(f"{len(parts)} parts for tp={tp}")
    arr = (c_void_p * len(parts))(*[_ptr(t) for t in parts])
    _check(load_library().pblock_rs_reduce(ctypes.byref(cfg), int(tp), arr, _ptr(x_shard),
                                           _ptr(b_out), _ptr(y_shard), _stream(stream)))


def pblock_status_string(status: int) -> str:
    return load_library().pblock_status_string(status).decode()


def pblock_last_error() -> str:
    return load_library().pblock_last_error().decode()


# ------------------------------------------------------- device-side block
class ParallelBlock:
    """One block's device buffers (torch owns the memory) around the C calls.

    ``tensors`` maps x, gamma, beta, w_in, b_in, w_out, b_out, dy to device
    tensors of the activation dtype.  The stash, the workspace and every
    output are allocated once here, so repeated forward()/backward() calls
    allocate nothing.
    """

    def __init__(self, cfg: PbConfig, tensors: dict, device="cuda"):
        import torch
        self.cfg = cfg
        self.t = tensors
        T = cfg.batch * cfg.seq
        H = cfg.hidden
        A = cfg.heads * cfg.head_dim
        n_in, k_out = 3 * A + cfg.ffn, A + cfg.ffn
        act = torch.bfloat16 if cfg.dtype == PB_BF16 else torch.float32
        f32 = torch.float32
        u8 = torch.uint8
        self.y = torch.empty((cfg.batch, cfg.seq, H), dtype=act, device=device)
        self.saved = torch.empty(pblock_saved_bytes(cfg), dtype=u8, device=device)
        self.ws = torch.empty(pblock_workspace_bytes(cfg, WS_BACKWARD), dtype=u8, device=device)
        nf = pblock_workspace_bytes(cfg, WS_FORWARD)
        self.ws_fwd = torch.empty(nf, dtype=u8, device=device) if nf else None
        self.grads = dict(
            dx=torch.empty((cfg.batch, cfg.seq, H), dtype=act, device=device),
            dgamma=torch.empty(H, dtype=f32, device=device),
            dbeta=torch.empty(H, dtype=f32, device=device),
            dw_in=torch.empty((n_in, H), dtype=f32, device=device),
            db_in=torch.empty(n_in, dtype=f32, device=device),
            dw_out=torch.empty((H, k_out), dtype=f32, device=device),
            db_out=torch.empty(H, dtype=f32, device=device),
        )
        self.T = T

    def forward(self, stream=None, step_ev=None):
        t = self.t
        pblock_forward(self.cfg, t["x"], t["gamma"], t["beta"], t["w_in"], t["b_in"], t["w_out"],
                       t["b_out"], self.y, self.saved, self.ws_fwd, stream, step_ev)
        return self.y

    def backward(self, dy=None, stream=None, step_ev=None):
        t, g = self.t, self.grads
        pblock_backward(self.cfg, t["x"], t["gamma"], t["beta"], t["w_in"], t["b_in"], t["w_out"],
                        t["b_out"], self.saved, t["dy"] if dy is None else dy, g["dx"],
                        g["dgamma"], g["dbeta"], g["dw_in"], g["db_in"], g["dw_out"],
                        g["db_out"], self.ws, stream, step_ev)
        return g

    def saved_view(self, name: str):
        """A typed view of one stash region (h, z, c, mean, rstd, lse)."""
        return _stash_view(self.cfg, self.saved, pblock_saved_offsets(self.cfg), name)

    def workspace_view(self, name: str):
        """A typed view of one backward intermediate (d_o, dz, dh, delta) in
        the workspace, valid after backward() until the next call."""
        import torch
        cfg = self.cfg
        T, H, A = cfg.batch * cfg.seq, cfg.hidden, cfg.heads * cfg.head_dim
        act = torch.bfloat16 if cfg.dtype == PB_BF16 else torch.float32
        if name == "delta":
            off = pblock_workspace_offsets(cfg)["delta"]
            n = cfg.batch * cfg.heads * cfg.seq
            return self.ws[off:off + 4 * n].view(torch.float32).view(cfg.batch, cfg.heads,
                                                                     cfg.seq)
        cols = {"d_o": A, "dz": 3 * A + cfg.ffn, "dh": H}[name]
        off = pblock_workspace_offsets(cfg)[name]
        nbytes = T * cols * torch.empty((), dtype=act).element_size()
        return self.ws[off:off + nbytes].view(act).view(T, cols)


def _stash_view(cfg, saved, offsets: dict, name: str):
    import torch
    T, H, A = cfg.batch * cfg.seq, cfg.hidden, cfg.heads * cfg.head_dim
    act = torch.bfloat16 if cfg.dtype == PB_BF16 else torch.float32
    f32 = torch.float32
    shapes = {"z": ((T, 3 * A + cfg.ffn), act), "c": ((T, A + cfg.ffn), act),
              "lse": ((cfg.batch, cfg.heads, cfg.seq), f32)}
    for n in ("h", "h1", "h2", "x1"):
        shapes[n] = ((T, H), act)
    for n in ("mean", "rstd", "mean1", "rstd1", "mean2", "rstd2"):
        shapes[n] = ((T,), f32)
    shape, dt = shapes[name]
    n = 1
    for s_ in shape:
        n *= s_
    off = offsets[name]
    nbytes = n * torch.empty((), dtype=dt).element_size()
    return saved[off:off + nbytes].view(dt).view(shape)


class SerialBlock:
    """The standard pre-LN block's device buffers around the serial C calls.

    ``tensors`` maps x, gamma1, beta1, gamma2, beta2, w_in, b_in, w_out, b_o,
    b_down, dy to device tensors of the activation dtype (w_in and w_out in
    the parallel block's packed layouts).  Buffers are allocated once here.
    """

    def __init__(self, cfg: PbConfig, tensors: dict, device="cuda"):
        import torch
        self.cfg = cfg
        self.t = tensors
        H = cfg.hidden
        A = cfg.heads * cfg.head_dim
        n_in, k_out = 3 * A + cfg.ffn, A + cfg.ffn
        act = torch.bfloat16 if cfg.dtype == PB_BF16 else torch.float32
        f32 = torch.float32
        u8 = torch.uint8
        self.y = torch.empty((cfg.batch, cfg.seq, H), dtype=act, device=device)
        self.saved = torch.empty(pblock_serial_saved_bytes(cfg), dtype=u8, device=device)
        self.ws = torch.empty(pblock_serial_workspace_bytes(cfg, WS_BACKWARD), dtype=u8,
                              device=device)
        nf = pblock_serial_workspace_bytes(cfg, WS_FORWARD)
        self.ws_fwd = torch.empty(nf, dtype=u8, device=device) if nf else None
        self.grads = dict(
            dx=torch.empty((cfg.batch, cfg.seq, H), dtype=act, device=device),
            dgamma1=torch.empty(H, dtype=f32, device=device),
            dbeta1=torch.empty(H, dtype=f32, device=device),
            dgamma2=torch.empty(H, dtype=f32, device=device),
            dbeta2=torch.empty(H, dtype=f32, device=device),
            dw_in=torch.empty((n_in, H), dtype=f32, device=device),
            db_in=torch.empty(n_in, dtype=f32, device=device),
            dw_out=torch.empty((H, k_out), dtype=f32, device=device),
            db_o=torch.empty(H, dtype=f32, device=device),
            db_down=torch.empty(H, dtype=f32, device=device),
        )

    def forward(self, stream=None):
        t = self.t
        pblock_serial_forward(self.cfg, t["x"], t["gamma1"], t["beta1"], t["gamma2"],
                              t["beta2"], t["w_in"], t["b_in"], t["w_out"], t["b_o"],
                              t["b_down"], self.y, self.saved, self.ws_fwd, stream)
        return self.y

    def backward(self, dy=None, stream=None):
        t, g = self.t, self.grads
        pblock_serial_backward(self.cfg, t["x"], t["gamma1"], t["beta1"], t["gamma2"],
                               t["beta2"], t["w_in"], t["b_in"], t["w_out"], t["b_o"],
                               t["b_down"], self.saved, t["dy"] if dy is None else dy, g["dx"],
                               g["dgamma1"], g["dbeta1"], g["dgamma2"], g["dbeta2"], g["dw_in"],
                               g["db_in"], g["dw_out"], g["db_o"], g["db_down"], self.ws,
                               stream)
        return g

    def saved_view(self, name: str):
        """A typed view of one stash region (names in SERIAL_SAVED_REGIONS)."""
        return _stash_view(self.cfg, self.saved, pblock_serial_saved_offsets(self.cfg), name)

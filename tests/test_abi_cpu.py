"""The C ABI on a machine without a GPU: the library loads, exports every
function include/pblock.h declares, and rejects bad arguments on the host
before any HIP call (so these run on the CPU)."""
import ctypes
import os
import re

import pytest

from paper_2402_15627_amd import pblock as pb
from paper_2402_15627_amd.inputs import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pblock.h")

pytestmark = pytest.mark.skipif(not os.path.exists(pb.LIB_PATH), reason="libpblock.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pblock_\w+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(pb.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(pb.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def good_cfg(**kw):
    s = WORKLOADS["13b_shape"]
    c = pb.config_from_shape(s)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("field,value,status", [
    ("hidden", 12, 1), ("hidden", 0, 1), ("ffn", 20, 1), ("batch", 0, 1),
    ("seq", 0, 1), ("heads", 0, 1), ("window", 0, 1), ("head_dim", 80, 2), ("head_dim", 32, 2),
    ("hidden", 40960, 2), ("gelu_tanh", 2, 1), ("dtype", 7, 1), ("ln_eps", 0.0, 1),
    ("ln_eps", float("nan"), 1),
])
def test_validate_rejects(field, value, status):
    c = good_cfg(**{field: value})
    assert pb.pblock_validate(c) == status
    assert pb.pblock_last_error() != ""
    assert pb.pblock_saved_bytes(c) == 0
    assert pb.pblock_workspace_bytes(c, pb.WS_BACKWARD) == 0


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_validate_accepts_every_workload(name):
    assert pb.pblock_validate(pb.config_from_shape(WORKLOADS[name])) == 0


def align(v):
    return (v + 255) // 256 * 256


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_saved_layout(name):
    s = WORKLOADS[name]
    c = pb.config_from_shape(s)
    e = 2 if s.dtype == "bf16" else 4
    T = s.tokens
    sizes = [T * s.hidden * e, T * s.n_in * e, T * s.k_out * e, 4 * T, 4 * T,
             4 * s.batch * s.heads * s.seq]
    off, o = [], 0
    for z in sizes:
        off.append(o)
        o = align(o + z)
    assert pb.pblock_saved_offsets(c) == dict(zip(pb.SAVED_REGIONS, off))
    assert pb.pblock_saved_bytes(c) == o
    split = pb.pblock_workspace_bytes(c, pb.WS_FORWARD)
    assert split % 256 == 0
    assert pb.pblock_workspace_bytes(c, pb.WS_FORWARD_WITH_STASH) == o + split
    # backward workspace holds at least dO, dZ and dh
    assert pb.pblock_workspace_bytes(c, pb.WS_BACKWARD) >= T * s.attn_width * e + T * s.n_in * e + 4 * T * s.hidden
    assert pb.pblock_workspace_bytes(c, 3) == 0


def tail_split(M, N, K, bf16=True):
    """Bytes of fp32 partial tiles of an M x N x K GEMM as the library plans
    it (pblock_gemm_plan): 0 when unsplit."""
    p = pb.pblock_gemm_plan(pb.PB_BF16 if bf16 else pb.PB_F32, M, N, K)
    return p.tail * p.splits * 65536 if p.tail else 0


def test_split_plan_examples():
    """Plans worked out by hand on 256 x 256 tiles and 256 CUs: a partial
    last wave is split along K to fill the chip once; a grid of fewer tiles
    than CUs is split when waves x K-steps per slice, plus a reduction cost of
    3 + 1/16 K-step per partial tile, is lowest.
      2048 x 10752 x 12288: 336 tiles = 256 whole + 80, 80 split 256 // 80 = 3
      2048 x 1536 x 12288: 48 tiles, K-steps 192; cost(s) = ceil(48 s / 256)
        ceil(192 / s) + 3 + 3 s is lowest at s = 5 (1 x 39 + 18 = 57)
      2048 x 4608 x 12288: 144 tiles; s = 3: 2 waves x 64 + 30 = 158 beats
        s = 1 (192) and every other s
      fp32 and a single 4-K-step tile: unsplit."""
    plan = lambda *a: pb.pblock_gemm_plan(*a)  # noqa: E731
    p = plan(pb.PB_BF16, 2048, 10752, 12288)
    assert (p.tiles, p.n_full, p.tail, p.splits) == (336, 256, 80, 3)
    assert (p.workgroups, p.threads) == (256 + 80 * 3, 512)
    p = plan(pb.PB_BF16, 2048, 1536, 12288)
    assert (p.n_full, p.tail, p.splits, p.workgroups) == (0, 48, 5, 240)
    p = plan(pb.PB_BF16, 2048, 4608, 12288)
    assert (p.n_full, p.tail, p.splits) == (0, 144, 3)
    p = plan(pb.PB_F32, 2048, 4608, 12288)
    assert (p.tiles, p.tail, p.splits, p.workgroups, p.threads) == (32 * 72, 0, 1, 32 * 72, 256)
    p = plan(pb.PB_BF16, 128, 256, 256)
    assert (p.tiles, p.tail, p.splits, p.workgroups) == (1, 0, 1, 1)
    # K not a multiple of 64 takes the unsplit path
    p = plan(pb.PB_BF16, 2048, 12288 + 256, 1000)
    assert (p.tiles, p.tail, p.splits, p.workgroups) == (8 * 49, 0, 1, 8 * 49)
    for bad in ((pb.PB_BF16, 0, 1, 1), (pb.PB_BF16, 1, -1, 1), (7, 1, 1, 1)):
        with pytest.raises(pb.PblockError):
            plan(*bad)


def test_backward_pairs_query():
    """bf16 shapes with every K a multiple of 64 share launches; fp32 never."""
    assert pb.pblock_backward_pairs(pb.config_from_shape(WORKLOADS["175b_tp8_share"])) == (True, True)
    assert pb.pblock_backward_pairs(pb.config_from_shape(WORKLOADS["175b_tp8_share"]),
                                    "serial") == (True, True, True, True)
    assert pb.pblock_backward_pairs(pb.config_from_shape(WORKLOADS["tiny_f32"])) == (False, False)
    # 1000 tokens: the weight gradients' K = T is not a multiple of 64
    ragged = pb.make_config(1, 1000, 1024, 8, 128, 2048, 256)
    assert pb.pblock_backward_pairs(ragged) == (False, False)
    assert pb.load_library().pblock_backward_pairs(ctypes.byref(ragged), 2, None) == 1


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_split_workspace_sizes(name):
    s = WORKLOADS[name]
    c = pb.config_from_shape(s)
    bf = s.dtype == "bf16"
    T, H, n_in, k_out = s.tokens, s.hidden, s.n_in, s.k_out
    fwd = max(tail_split(T, n_in, H, bf), tail_split(T, H, k_out, bf)) * 4
    assert pb.pblock_workspace_bytes(c, pb.WS_FORWARD) == align(fwd)


FAKE = 1 << 40  # a 16-byte aligned address; never dereferenced: every call below fails its checks


def fwd_args(**over):
    a = dict(x=FAKE, ln_gamma=FAKE, ln_beta=FAKE, w_in=FAKE, b_in=FAKE, w_out=FAKE, b_out=FAKE,
             y=FAKE, saved=FAKE)
    a.update(over)
    return a


@pytest.mark.parametrize("over,status", [
    (dict(x=None), 1), (dict(w_in=None), 1), (dict(y=FAKE + 8), 1), (dict(b_out=FAKE + 2), 1),
    (dict(saved=None), 1),  # no stash and no workspace
])
def test_forward_rejects_bad_pointers_before_launching(over, status):
    lib = pb.load_library()
    a = fwd_args(**over)
    c = good_cfg()
    st = lib.pblock_forward(ctypes.byref(c), a["x"], a["ln_gamma"], a["ln_beta"], a["w_in"],
                            a["b_in"], a["w_out"], a["b_out"], a["y"], a["saved"], None, 0, None)
    assert st == status, pb.pblock_last_error()


def test_forward_rejects_small_workspace():
    lib = pb.load_library()
    a = fwd_args(saved=None)
    c = good_cfg()
    need = pb.pblock_saved_bytes(c)
    st = lib.pblock_forward(ctypes.byref(c), a["x"], a["ln_gamma"], a["ln_beta"], a["w_in"],
                            a["b_in"], a["w_out"], a["b_out"], a["y"], None, FAKE, need - 1, None)
    assert st == 3
    assert "ws_bytes" in pb.pblock_last_error()


def test_backward_rejects_small_workspace_and_nulls():
    lib = pb.load_library()
    c = good_cfg()
    need = pb.pblock_workspace_bytes(c, pb.WS_BACKWARD)
    args = [FAKE] * 16
    st = lib.pblock_backward(ctypes.byref(c), *args, FAKE, 1024, None)
    assert st == 3
    args[9] = None  # dx
    st = lib.pblock_backward(ctypes.byref(c), *args, FAKE, need, None)
    assert st == 1 and "dx" in pb.pblock_last_error()


def test_swattn_rejects_bad_leading_dimension():
    lib = pb.load_library()
    c = good_cfg()
    A = c.heads * c.head_dim
    st = lib.pblock_swattn_forward(ctypes.byref(c), FAKE, FAKE, FAKE, A - 8, FAKE, A, FAKE, None,
                                   0, None)
    assert st == 1 and "ld_qkv" in pb.pblock_last_error()
    st = lib.pblock_swattn_forward(ctypes.byref(c), FAKE, FAKE, FAKE, A + 4, FAKE, A, FAKE, None,
                                   0, None)
    assert st == 1
    st = lib.pblock_swattn_backward(ctypes.byref(c), FAKE, FAKE, FAKE, A, FAKE, A, FAKE, A, FAKE,
                                    FAKE, FAKE, FAKE, A, FAKE, 0, None)
    assert st == 3


def test_status_strings():
    assert [pb.pblock_status_string(i) for i in range(5)] == [pb.STATUS[i] for i in range(5)]


def test_swattn_workspace_modes():
    """The split workspace is planned only when the blocks are too few to fill
    the GPU: the forward's batch * heads * (seq / 128) blocks, the backward's
    dK/dV and dQ blocks together (they share one launch).  The backward's
    minimum is one fp32 row term per query."""
    lib_ws = pb.pblock_swattn_workspace_bytes
    share = pb.make_config(1, 2048, 1536, 12, 128, 64, 2048, "bf16")  # 576 bwd blocks
    tiny = pb.make_config(1, 2048, 512, 4, 128, 64, 2048, "bf16")     # 192 bwd blocks
    big = pb.make_config(1, 8192, 5120, 40, 128, 64, 1024, "bf16")
    f32 = pb.make_config(1, 2048, 1536, 12, 128, 64, 2048, "f32")
    for c in (share, tiny, big, f32):
        assert lib_ws(c, pb.ATTN_WS_BACKWARD_MIN) == -(-c.batch * c.heads * c.seq * 4 // 256) * 256
        assert lib_ws(c, pb.ATTN_WS_BACKWARD) >= lib_ws(c, pb.ATTN_WS_BACKWARD_MIN)
    assert lib_ws(share, pb.ATTN_WS_FORWARD) > 0  # 192 forward blocks
    assert lib_ws(share, pb.ATTN_WS_BACKWARD) == lib_ws(share, pb.ATTN_WS_BACKWARD_MIN)
    assert lib_ws(tiny, pb.ATTN_WS_BACKWARD) > lib_ws(tiny, pb.ATTN_WS_BACKWARD_MIN)
    for c in (big, f32):
        assert lib_ws(c, pb.ATTN_WS_FORWARD) == 0
        assert lib_ws(c, pb.ATTN_WS_BACKWARD) == lib_ws(c, pb.ATTN_WS_BACKWARD_MIN)
    assert lib_ws(share, 7) == 0


def declared_arities():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    out = {}
    for name, args in re.findall(r"\b(pblock_\w+)\s*\(([^;{]*?)\)\s*;", text):
        a = args.strip()
        out[name] = 0 if a in ("", "void") else a.count(",") + 1
    return out


def test_binding_argument_counts_match_the_header():
    lib = pb.load_library()
    ar = declared_arities()
    assert sorted(ar) == sorted(pb.EXPORTS)
    for name, n in ar.items():
        assert len(getattr(lib, name).argtypes) == n, name


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_serial_saved_layout(name):
    s = WORKLOADS[name]
    c = pb.config_from_shape(s)
    e = 2 if s.dtype == "bf16" else 4
    T, H = s.tokens, s.hidden
    sizes = [T * H * e, T * s.n_in * e, T * s.k_out * e, 4 * T, 4 * T,
             4 * s.batch * s.heads * s.seq, T * H * e, T * H * e, 4 * T, 4 * T]
    off, o = [], 0
    for z in sizes:
        off.append(o)
        o = align(o + z)
    assert pb.pblock_serial_saved_offsets(c) == dict(zip(pb.SERIAL_SAVED_REGIONS, off))
    assert pb.pblock_serial_saved_bytes(c) == o
    split = pb.pblock_serial_workspace_bytes(c, pb.WS_FORWARD)
    assert split % 256 == 0
    assert pb.pblock_serial_workspace_bytes(c, pb.WS_FORWARD_WITH_STASH) == o + split
    # backward: dO, dZ, dh (fp32) and dx1 at least
    assert pb.pblock_serial_workspace_bytes(c, pb.WS_BACKWARD) >= (
        T * s.attn_width * e + T * s.n_in * e + 4 * T * H + T * H * e)
    assert pb.pblock_serial_workspace_bytes(c, 3) == 0


def test_serial_rejects_bad_arguments_before_launching():
    lib = pb.load_library()
    c = good_cfg()
    # forward: no stash and a workspace too small for one
    need = pb.pblock_serial_saved_bytes(c)
    args = [FAKE] * 11  # x .. y
    st = lib.pblock_serial_forward(ctypes.byref(c), *args, None, FAKE, need - 1, None)
    assert st == 3 and "ws_bytes" in pb.pblock_last_error()
    st = lib.pblock_serial_forward(ctypes.byref(c), *args, None, None, 0, None)
    assert st == 1
    bad = list(args)
    bad[3] = FAKE + 4  # ln2_gamma misaligned
    st = lib.pblock_serial_forward(ctypes.byref(c), *bad, FAKE, None, 0, None)
    assert st == 1 and "ln2_gamma" in pb.pblock_last_error()
    # backward: workspace below the required part, then a NULL gradient
    bargs = [FAKE] * 22
    st = lib.pblock_serial_backward(ctypes.byref(c), *bargs, FAKE, 1024, None)
    assert st == 3
    need = pb.pblock_serial_workspace_bytes(c, pb.WS_BACKWARD)
    bargs[21] = None  # db_down
    st = lib.pblock_serial_backward(ctypes.byref(c), *bargs, FAKE, need, None)
    assert st == 1 and "db_down" in pb.pblock_last_error()
    bad_cfg = good_cfg(head_dim=80)
    assert pb.pblock_serial_saved_bytes(bad_cfg) == 0
    assert pb.pblock_serial_workspace_bytes(bad_cfg, pb.WS_BACKWARD) == 0


def test_lamb_workspace_and_validation():
    T = pb.LambTensor
    ts = [T(FAKE, FAKE, FAKE, FAKE, None, 8192 * 3 + 5, 0.01), T(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0.0)]
    # chunks of 1024 elements, each tensor's chunks padded to a group of 256:
    # 256 float2 partials, one double2 group sum, two ratios
    assert pb.pblock_lamb_workspace_bytes(ts) == align(256 * 8) + align(16) + align(2 * 4)
    assert pb.pblock_lamb_workspace_bytes([]) == 0
    assert pb.pblock_lamb_workspace_bytes([ts[0]] * 17) == 0
    lib = pb.load_library()
    good = pb.lamb_config(1e-3, step=1)

    def call(cfg=good, tensors=ts, copy=pb.PB_BF16, ws=FAKE, nbytes=1 << 20):
        arr = (pb.LambTensor * len(tensors))(*tensors)
        return lib.pblock_lamb_step(ctypes.byref(cfg), len(tensors), arr, copy, None, ws, nbytes,
                                    None)

    assert call(nbytes=64) == 3 and "ws_bytes" in pb.pblock_last_error()
    for bad in (pb.lamb_config(1e-3, beta1=1.0), pb.lamb_config(1e-3, eps=0.0),
                pb.lamb_config(1e-3, step=0), pb.lamb_config(float("nan")),
                pb.lamb_config(1e-3, beta2=-0.1)):
        assert call(cfg=bad) == 1
    assert call(copy=5) == 1
    assert call(tensors=[T(FAKE, None, FAKE, FAKE, None, 16, 0.0)]) == 1
    assert "grad" in pb.pblock_last_error()
    assert call(tensors=[T(FAKE, FAKE, FAKE + 8, FAKE, None, 16, 0.0)]) == 1
    assert call(tensors=[T(FAKE, FAKE, FAKE, FAKE, FAKE + 2, 16, 0.0)]) == 1
    assert call(tensors=[T(FAKE, FAKE, FAKE, FAKE, None, 16, -1.0)]) == 1
    # empty tensors need no pointers
    assert pb.pblock_lamb_workspace_bytes([T(None, None, None, None, None, 0, 0.0)]) == align(4)
    assert call(ws=FAKE + 16) == 1


def test_ag_in_proj_rejects_bad_arguments_before_launching():
    lib = pb.load_library()
    c = good_cfg()  # 13B shape: T = 2048, H = 5120

    def call(cfg=c, tp=8, rank=0, per=1, stream=FAKE, comm=(FAKE + 256,), ws=FAKE,
             nbytes=1 << 20):
        shards = (ctypes.c_void_p * tp)(*([FAKE] * tp)) if tp > 0 else None
        cs = (ctypes.c_void_p * max(len(comm), 1))(*comm) if comm else None
        return lib.pblock_ag_in_proj(ctypes.byref(cfg), tp, rank, shards, FAKE, FAKE, FAKE, FAKE,
                                     FAKE, per, ws, nbytes, stream, len(comm), cs, None)

    assert call(tp=3) == 1 and "divisible" in pb.pblock_last_error()
    assert call(tp=65) == 1
    assert call(rank=8) == 1 and call(rank=-1) == 1
    assert call(per=0) == 1 and call(per=9) == 1
    assert call(comm=(FAKE,)) == 1  # comm stream equal to the compute stream
    assert call(comm=(FAKE + 256, FAKE + 256)) == 1  # repeated
    assert call(comm=()) == 1
    assert call(ws=FAKE + 16) == 1
    assert call(cfg=good_cfg(head_dim=80)) == 2
    # every other argument is checked before the context
    assert call() == 1 and "ctx" in pb.pblock_last_error()
    assert pb.pblock_ag_in_proj_workspace_bytes(c, 8, 1) % 256 == 0
    assert pb.pblock_ag_in_proj_workspace_bytes(c, 8, 9) == 0
    assert pb.pblock_ag_in_proj_workspace_bytes(c, 3, 1) == 0


def test_backward_ag_and_rs_reject_bad_arguments_before_launching():
    """pblock_ag_dc and pblock_rs_dh check what their forward counterparts
    check, every other argument before the context."""
    lib = pb.load_library()
    c = good_cfg()  # 13B shape: T = 2048, H = 5120

    def ag(cfg=c, tp=8, rank=0, per=1, stream=FAKE, comm=(FAKE + 256,), ws=FAKE, nbytes=1 << 20,
           shards=None, dy=FAKE):
        sh = (ctypes.c_void_p * tp)(*(shards or [FAKE] * tp)) if tp > 0 else None
        cs = (ctypes.c_void_p * max(len(comm), 1))(*comm) if comm else None
        return lib.pblock_ag_dc(ctypes.byref(cfg), tp, rank, sh, dy, FAKE, FAKE, FAKE, FAKE, per,
                                ws, nbytes, stream, len(comm), cs, None)

    def rs(cfg=c, tp=8, rank=0, per=1, stream=FAKE, comm=(FAKE + 256,), ws=FAKE, nbytes=1 << 20,
           dst=None, dz=FAKE):
        d = (ctypes.c_void_p * tp)(*(dst or [FAKE] * tp)) if tp > 0 else None
        cs = (ctypes.c_void_p * max(len(comm), 1))(*comm) if comm else None
        return lib.pblock_rs_dh(ctypes.byref(cfg), tp, rank, dz, FAKE, FAKE, d, per, ws, nbytes,
                                stream, len(comm), cs, None)

    for call, lst in ((ag, "shards"), (rs, "dst")):
        assert call(tp=3) == 1 and "divisible" in pb.pblock_last_error()
        assert call(tp=65) == 1
        assert call(rank=8) == 1 and call(rank=-1) == 1
        assert call(per=0) == 1 and call(per=9) == 1
        assert call(comm=(FAKE,)) == 1
        assert call(comm=(FAKE + 256, FAKE + 256)) == 1
        assert call(comm=()) == 1
        assert call(ws=FAKE + 16) == 1
        assert call(cfg=good_cfg(head_dim=80)) == 2
        assert call(**{lst: [FAKE] * 7 + [FAKE + 8]}) == 1
        assert "[7]" in pb.pblock_last_error()
        assert call() == 1 and "ctx" in pb.pblock_last_error()
    assert ag(dy=None) == 1 and "dy" in pb.pblock_last_error()
    assert rs(dz=None) == 1 and "dz" in pb.pblock_last_error()
    for f in (pb.pblock_ag_dc_workspace_bytes, pb.pblock_rs_dh_workspace_bytes):
        assert f(c, 8, 1) % 256 == 0 and f(c, 8, 9) == 0 and f(c, 3, 1) == 0
    # dC over 2 shards of 256 rows: 2 x 100 = 200 tiles of K = 5120, fewer
    # than the CUs: split along K (the small-grid plan)
    assert pb.pblock_ag_dc_workspace_bytes(c, 8, 2) > 0
    with pytest.raises(ValueError):
        pb.pblock_ag_dc(c, 8, 0, [FAKE] * 7, FAKE, FAKE, FAKE, FAKE, FAKE, 1, None, FAKE,
                        [FAKE + 256], None)
    with pytest.raises(ValueError):
        pb.pblock_rs_dh(c, 8, 0, FAKE, FAKE, FAKE, [FAKE] * 9, 1, None, FAKE, [FAKE + 256],
                        None)


def test_rs_out_proj_and_reduce_reject_bad_arguments_before_launching():
    lib = pb.load_library()
    c = good_cfg()  # 13B shape: T = 2048, H = 5120

    def call(cfg=c, tp=8, rank=0, per=1, stream=FAKE, comm=(FAKE + 256,), ws=FAKE,
             nbytes=1 << 20, dst=None):
        d = (ctypes.c_void_p * tp)(*(dst or [FAKE] * tp)) if tp > 0 else None
        cs = (ctypes.c_void_p * max(len(comm), 1))(*comm) if comm else None
        return lib.pblock_rs_out_proj(ctypes.byref(cfg), tp, rank, FAKE, FAKE, FAKE, d, per, ws,
                                      nbytes, stream, len(comm), cs, None)

    assert call(tp=3) == 1 and "divisible" in pb.pblock_last_error()
    assert call(tp=65) == 1
    assert call(rank=8) == 1 and call(rank=-1) == 1
    assert call(per=0) == 1 and call(per=9) == 1
    assert call(comm=(FAKE,)) == 1
    assert call(comm=(FAKE + 256, FAKE + 256)) == 1
    assert call(comm=()) == 1
    assert call(ws=FAKE + 16) == 1
    assert call(dst=[FAKE] * 7 + [FAKE + 8]) == 1 and "dst[7]" in pb.pblock_last_error()
    assert call(dst=[FAKE] * 3 + [None] * 5) == 1 and "dst[3]" in pb.pblock_last_error()
    assert call(cfg=good_cfg(head_dim=80)) == 2
    assert call() == 1 and "ctx" in pb.pblock_last_error()
    assert pb.pblock_rs_out_proj_workspace_bytes(c, 8, 1) % 256 == 0
    assert pb.pblock_rs_out_proj_workspace_bytes(c, 8, 9) == 0
    assert pb.pblock_rs_out_proj_workspace_bytes(c, 3, 1) == 0
    # the python wrappers refuse a list of the wrong length
    with pytest.raises(ValueError):
        pb.pblock_rs_out_proj(c, 8, 0, FAKE, FAKE, FAKE, [FAKE] * 7, 1, None, FAKE, [FAKE + 256],
                              None)
    with pytest.raises(ValueError):
        pb.pblock_rs_reduce(c, 8, [FAKE] * 9, FAKE, FAKE, FAKE)

    def reduce(cfg=c, tp=8, parts=None, x=FAKE, b=FAKE, y=FAKE):
        arr = (ctypes.c_void_p * tp)(*(parts or [FAKE] * tp)) if tp > 0 else None
        return lib.pblock_rs_reduce(ctypes.byref(cfg), tp, arr, x, b, y, FAKE)

    assert reduce(tp=3) == 1
    # a context is made for tp in 1..64 (the events need a device)
    h = ctypes.c_void_p(FAKE)
    assert lib.pblock_tp_context_create(0, ctypes.byref(h)) == 1 and h.value is None
    assert lib.pblock_tp_context_create(65, ctypes.byref(h)) == 1
    assert lib.pblock_tp_context_create(8, None) == 1
    lib.pblock_tp_context_destroy(None)
    assert reduce(tp=0) == 1 and reduce(tp=65) == 1
    assert reduce(parts=[FAKE] * 7 + [FAKE + 4]) == 1 and "parts[7]" in pb.pblock_last_error()
    assert reduce(y=None) == 1 and reduce(b=FAKE + 2) == 1


def test_noalloc_attention_rejects_oversized_scratch_on_host():
    """The allocation-free attention forward refuses, before any HIP call, a
    shape whose split plan needs more than PB_NOALLOC_SCRATCH_BYTES of
    scratch (2 heads x 128 over 24000 tokens needs ~47 MB); the pointers are
    never touched."""
    c = pb.make_config(1, 24000, 64, 2, 128, 64, 24000)
    assert pb.pblock_swattn_workspace_bytes(c, pb.ATTN_WS_FORWARD) > pb.NOALLOC_SCRATCH_BYTES
    fake = 1 << 20  # aligned, never dereferenced: the call fails its host check first
    lib = pb.load_library()
    st = lib.pblock_swattn_forward_noalloc(ctypes.byref(c), fake, fake, fake, 256, fake, 256,
                                           fake, None)
    assert st == 2  # PB_ERR_UNSUPPORTED
    assert "scratch" in pb.pblock_last_error()
    # and a bad argument is still an argument error
    st = lib.pblock_swattn_forward_noalloc(ctypes.byref(c), None, fake, fake, 256, fake, 256,
                                           fake, None)
    assert st == 1

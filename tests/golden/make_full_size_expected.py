"""Write sampled oracle outputs for the full-size workloads (tests/golden/*.npz).

Runs the fp64 CPU oracle (oracle/pblock_oracle.py) on the seeded inputs of
each full-size workload and keeps, as float32:
  y, dx        8 token rows (tile edges, first and last rows)
  dw_in        8 rows straddling the Q | K | V | U boundaries
  dw_out       8 rows (output features at tile edges)
  dgamma, dbeta, db_in, db_out in full.
Each weight-gradient row is its own sum over tokens, so computing only the
sampled rows gives exactly the numbers of the full product.
Nothing here calls the HIP library.  Usage:
    python tests/golden/make_full_size_expected.py [workload ...]
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import pblock_oracle as orc  # noqa: E402
from paper_2402_15627_amd.inputs import WORKLOADS, make_inputs  # noqa: E402

FULL_SIZE = ("13b_shape", "175b_tp8_share", "175b_tp8_share_w512", "long_seq_8k", "175b_full",
             "175b_tp8_share_d96", "175b_full_d96")


def sample_rows(s):
    T, H, A, F = s.tokens, s.hidden, s.attn_width, s.ffn
    tok = sorted({0, 1, 255, 256, T // 2 + 37, T - 257, T - 2, T - 1})
    win = sorted({0, A - 1, A, 2 * A + 5, 3 * A - 1, 3 * A, 3 * A + F // 2, 3 * A + F - 1})
    wout = sorted({0, 1, 255, 256, H // 2, H - 257, H - 2, H - 1})
    return np.array(tok), np.array(win), np.array(wout)


def make(name, seed=0):
    s = WORKLOADS[name]
    t0 = time.time()
    inp = make_inputs(s, seed)
    tok, rin, rout = sample_rows(s)
    res = orc.run_block(orc.config_from_shape(s), inp, weight_rows=(rin, rout))
    T = s.tokens
    out = dict(
        tok_rows=tok, w_in_rows=rin, w_out_rows=rout,
        y=res["y"].reshape(T, -1)[tok].astype(np.float32),
        dx=res["dx"].reshape(T, -1)[tok].astype(np.float32),
        dw_in=res["dw_in"].astype(np.float32),
        dw_out=res["dw_out"].astype(np.float32),
        dgamma=res["dgamma"].astype(np.float32), dbeta=res["dbeta"].astype(np.float32),
        db_in=res["db_in"].astype(np.float32), db_out=res["db_out"].astype(np.float32),
        x_checksum=np.float64(np.asarray(inp["x"], np.float64).sum()),
        w_in_checksum=np.float64(np.asarray(inp["w_in"][rin], np.float64).sum()),
        seed=np.int64(seed),
    )
    path = os.path.join(HERE, f"{name}.npz")
    np.savez_compressed(path, **out)
    print(f"{name}: {time.time() - t0:.0f} s -> {path}", flush=True)


if __name__ == "__main__":
    for n in (sys.argv[1:] or FULL_SIZE):
        make(n)

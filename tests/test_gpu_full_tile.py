"""Every row and head of the large forward tiles against the float64 oracle.

The oracle's row function is spread over the host cores, one (head, row
chunk) per worker task: the causal 64K tile (16384 rows x 32 heads) takes
well under a minute on 16 cores, each 1M-token tile (65536 rows x 32 heads)
about a minute and a half."""

import time

import numpy as np
import pytest
import torch

from mesh_inputs import WORKLOADS, make_qkv

from helpers import check_fwd, log, oracle_forward_rows, run_fwd, to_np

pytestmark = pytest.mark.gpu

LARGE = ("mesh1m-nc-gqa", "mesh1m-causal-outlier")


@pytest.mark.parametrize("name", ["causal-64k", *LARGE])
def test_every_row_every_head(gpu, name):
    cfg = WORKLOADS[name]
    q, k, v, _ = make_qkv(cfg)
    qd, kd, vd = (t.to(gpu) for t in (q, k, v))
    o, lse = run_fwd(cfg.problem(), cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    og, lg = to_np(o), to_np(lse)
    del qd, kd, vd, o, lse
    rows = np.arange(cfg.nq * cfg.partition_len)
    worst_o = worst_l = 0.0
    t0 = time.time()
    # Eight heads per oracle batch keeps the float64 results of a batch at a
    # few GB; four on the 1M-token tiles, so that a progress line comes
    # every few seconds.
    per = 4 if name in LARGE else 8
    for h0 in range(0, cfg.num_q_heads, per):
        heads = list(range(h0, min(cfg.num_q_heads, h0 + per)))
        ro, rl = oracle_forward_rows(cfg.problem(), cfg.q_idx, cfg.kv_idx, q,
                                     k, v, rows, heads)
        eo, el = check_fwd(f"{name} heads {heads[0]}..{heads[-1]} "
                           f"(all {rows.size} rows)", og[:, heads],
                           lg[heads], ro, rl)
        worst_o, worst_l = max(worst_o, eo), max(worst_l, el)
        log(f"  heads {heads[0]}..{heads[-1]} done, {time.time() - t0:.0f} s")
    log(f"{name}, every row and head: max|O err| {worst_o:.3e}, "
        f"max|LSE err| {worst_l:.3e}")

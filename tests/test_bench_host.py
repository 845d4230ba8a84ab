"""Host-side checks of bench.py's bookkeeping: the algorithmic FLOP count
(visible pairs of a tile) against brute force over the oracle's positions,
and the single-GPU guard."""

import dataclasses
import os
import subprocess
import sys

import pytest

import bench
import oracle
from mesh_inputs import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("causal", [False, True])
def test_visible_pairs_matches_bruteforce(layout, causal):
    cfg = dataclasses.replace(WORKLOADS["causal-64k"], num_partitions=6, partition_len=16,
                              q_idx=[4, 1, 5], kv_idx=[0, 5, 2, 1],
                              causal=causal, layout=layout)
    qpos = oracle.problem_positions(cfg.problem(), cfg.q_idx)
    kpos = oracle.problem_positions(cfg.problem(), cfg.kv_idx)
    if causal:
        want = int((kpos[None, :] <= qpos[:, None]).sum())
    else:
        want = qpos.size * kpos.size
    assert bench.visible_pairs(cfg) == want


def test_visible_pairs_of_the_tile_configs():
    """causal-64k and striped-causal-64k (same tile, contiguous vs striped)."""
    # causal-64k: 22 full pairs and 4 triangular ones (with their diagonal)
    P = 4096
    assert bench.visible_pairs(WORKLOADS["causal-64k"]) == 22 * P * P + 4 * P * (P + 1) // 2
    # striped: 4 x 8 near-triangular pairs; pairs whose KV partition comes
    # after the Q partition lose their diagonal.
    after = sum(1 for qp in WORKLOADS["striped-causal-64k"].q_idx for kp in WORKLOADS["striped-causal-64k"].kv_idx
                if kp > qp)
    assert bench.visible_pairs(WORKLOADS["striped-causal-64k"]) == 32 * P * (P + 1) // 2 - after * P


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


@pytest.mark.parametrize("layout", [0, 1])
def test_visible_pairs_of_sampled_rows(layout):
    """The CPU baseline's FLOP count over sampled rows follows the layout
    (striped positions interleave the partitions)."""
    cfg = dataclasses.replace(WORKLOADS["causal-64k"], num_partitions=6,
                              partition_len=16, q_idx=[4, 1, 5],
                              kv_idx=[0, 5, 2, 1], causal=True, layout=layout)
    rows = [0, 3, 17, 20, 33, 47]
    qpos = oracle.problem_positions(cfg.problem(), cfg.q_idx)[rows]
    kpos = oracle.problem_positions(cfg.problem(), cfg.kv_idx)
    want = int((kpos[None, :] <= qpos[:, None]).sum())
    assert bench.visible_pairs(cfg, rows) == want

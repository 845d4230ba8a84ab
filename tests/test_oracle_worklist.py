"""Pins of the oracle's block classification and run lists: element-level
brute force, the partition-level statement of Section 3.7, a closed form for a
diagonal partition pair, a hand-derived fixture, and the paper's tile
footprint examples (Sections 3.2 and 3.3)."""

import json
import os

import numpy as np
import pytest

from mesh_inputs import WORKLOADS
from oracle import (EMPTY, FULL, PARTIAL, basic_tile, classify_blocks,
                    classify_blocks_bruteforce, kv_major_run_list, kvr_tile,
                    run_list)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _pair_counts(q_idx, kv_idx):
    """Section 3.7, partition level: (Q_i, KV_j) is fully masked for i < j,
    triangular for i = j, dense for i > j."""
    full = sum(1 for i in q_idx for j in kv_idx if i > j)
    diag = sum(1 for i in q_idx for j in kv_idx if i == j)
    empty = sum(1 for i in q_idx for j in kv_idx if i < j)
    return full, diag, empty


@pytest.mark.parametrize("name,expect", [
    ("tiny-nc", None), ("causal-64k", (22, 4, 6)), ("mesh1m-nc-gqa", None),
    ("mesh1m-causal-outlier", (220, 8, 28))])
def test_partition_pair_classes(name, expect):
    cfg = WORKLOADS[name]
    P, bm, bn = cfg.partition_len, 128, 64
    cls = classify_blocks(cfg.q_idx, cfg.kv_idx, P, bm, bn, cfg.causal)
    nqb, nkb = P // bm, P // bn
    got = [0, 0, 0]
    for a, i in enumerate(cfg.q_idx):
        for b, j in enumerate(cfg.kv_idx):
            blk = cls[a * nqb:(a + 1) * nqb, b * nkb:(b + 1) * nkb]
            if np.all(blk == FULL):
                got[0] += 1
            elif np.all(blk == EMPTY):
                got[2] += 1
            else:
                got[1] += 1
    if cfg.causal:
        assert tuple(got) == _pair_counts(cfg.q_idx, cfg.kv_idx)
        assert tuple(got) == expect
    else:
        assert got == [cfg.nq * cfg.nkv, 0, 0]


@pytest.mark.parametrize("bm,bn", [(128, 64), (64, 64), (128, 128), (64, 128)])
def test_diagonal_pair_closed_form(bm, bn):
    """Same partition on both sides, contiguous positions: Q block qb sees
    every key block entirely before it, straddles the blocks that overlap its
    rows, and is blind to the rest."""
    P = 4096
    cls = classify_blocks([5], [5], P, bm, bn, True)
    for qb in range(P // bm):
        lo, hi = qb * bm, qb * bm + bm - 1
        for kb in range(P // bn):
            klo, khi = kb * bn, kb * bn + bn - 1
            want = FULL if khi <= lo else (EMPTY if klo > hi else PARTIAL)
            assert cls[qb, kb] == want
    if bm == 128 and bn == 64:
        counts = np.bincount(cls.ravel(), minlength=3)
        assert counts[FULL] == 992 and counts[PARTIAL] == 64
        assert counts[EMPTY] == 992
        rho = bm // bn
        for qb in range(P // bm):
            row = cls[qb]
            assert np.all(row[:rho * qb] == FULL)
            assert np.all(row[rho * qb:rho * qb + rho] == PARTIAL)
            assert np.all(row[rho * qb + rho:] == EMPTY)


@pytest.mark.parametrize("name", ["tiny-nc", "causal-64k", "bwd-causal-64k"])
def test_block_classes_match_bruteforce_on_workloads(name):
    cfg = WORKLOADS[name]
    args = (cfg.q_idx, cfg.kv_idx, cfg.partition_len, 128, 64, cfg.causal)
    np.testing.assert_array_equal(classify_blocks(*args),
                                  classify_blocks_bruteforce(*args))


def test_block_classes_match_bruteforce_random():
    rng = np.random.default_rng(7)
    for _ in range(40):
        n = int(rng.integers(2, 9))
        bm = int(rng.choice([4, 8, 16]))
        bn = int(rng.choice([4, 8, 16]))
        P = int(np.lcm(bm, bn) * rng.integers(1, 4))
        q_idx = list(rng.choice(n, size=int(rng.integers(1, n + 1)),
                                replace=False))
        kv_idx = list(rng.choice(n, size=int(rng.integers(1, n + 1)),
                                 replace=False))
        causal = bool(rng.integers(0, 2))
        args = (q_idx, kv_idx, P, bm, bn, causal)
        np.testing.assert_array_equal(classify_blocks(*args),
                                      classify_blocks_bruteforce(*args))


def test_run_list_hand_fixture():
    g = json.load(open(os.path.join(GOLDEN, "runlist_small.json")))
    cls = classify_blocks(g["q_idx"], g["kv_idx"], g["partition_len"],
                          g["bm"], g["bn"], g["causal"])
    np.testing.assert_array_equal(cls, np.array(g["cls"]))
    nkb = g["partition_len"] // g["bn"]
    nqb = g["partition_len"] // g["bm"]
    ptr, runs = run_list(cls, len(g["kv_idx"]), nkb)
    assert ptr.tolist() == g["qblk_ptr"]
    assert runs.tolist() == g["runs"]
    kptr, kruns = kv_major_run_list(cls, len(g["q_idx"]), nqb)
    assert kptr.tolist() == g["kv_major_ptr"]
    assert kruns.tolist() == g["kv_major_runs"]


def test_run_list_covers_exactly_the_non_empty_blocks():
    cfg = WORKLOADS["mesh1m-causal-outlier"]
    P, bm, bn = cfg.partition_len, 128, 64
    cls = classify_blocks(cfg.q_idx, cfg.kv_idx, P, bm, bn, True)
    nkb = P // bn
    ptr, runs = run_list(cls, cfg.nkv, nkb)
    rebuilt = np.zeros_like(cls)
    for qblk, b, s, e, c in runs:
        rebuilt[qblk, b * nkb + s:b * nkb + e] = c
    np.testing.assert_array_equal(rebuilt, cls)
    for q in range(cls.shape[0]):
        seg = runs[ptr[q]:ptr[q + 1]]
        assert np.all(seg[:, 0] == q)


def test_paper_footprint_examples():
    g = json.load(open(os.path.join(GOLDEN, "footprints.json")))
    for ex in g["basic"]:
        assert basic_tile(ex["g"], ex["a"], ex["b"]) == (ex["q"], ex["kv"])
    for ex in g["kvr"]:
        assert kvr_tile(ex["g"], ex["a"], ex["b"]) == (ex["q"], ex["kv"])


def test_config_tiles_are_mesh_tiles():
    """The 1M-token non-causal tile is GPU 18 of a 16x16 basic tiling."""
    cfg = WORKLOADS["mesh1m-nc-gqa"]
    assert basic_tile(18, 16, 16) == (cfg.q_idx, cfg.kv_idx)

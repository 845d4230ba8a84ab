"""Pins of the oracle under the striped sequence layout of Section 3.7 (token r
of partition p at position r*n + p): the position map itself, a library
routine (torch scaled_dot_product_attention / autograd in float64 on the
position-ordered sequence), the block-class closed form of a striped pair,
brute force, and the merge invariant across a split of the KV footprint."""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import STRIPED, lse_merge, tile_backward, tile_forward
from oracle.worklist import (EMPTY, FULL, PARTIAL, classify_blocks,
                             classify_blocks_bruteforce)


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _prob(n, P, hq, hkv, d, causal=True):
    return dict(num_partitions=n, partition_len=P, num_q_heads=hq,
                num_kv_heads=hkv, head_dim=d, causal=int(causal),
                softmax_scale=1.0 / math.sqrt(d), layout=STRIPED)


def test_striped_positions_deal_round_robin():
    pos = oracle.token_positions([0, 1, 2, 3], 3, STRIPED, 4).reshape(4, 3)
    np.testing.assert_array_equal(pos, [[0, 4, 8], [1, 5, 9], [2, 6, 10],
                                        [3, 7, 11]])
    # Every partition list that names all partitions covers the sequence once.
    pos = oracle.token_positions([2, 0, 3, 1], 5, STRIPED, 4)
    np.testing.assert_array_equal(np.sort(pos), np.arange(20))
    # Positions grow with the row inside a partition (block extremes sit at the
    # block's first and last rows).
    assert np.all(np.diff(pos.reshape(4, 5), axis=1) == 4)


def _position_order(prob, idx):
    pos = oracle.problem_positions(prob, idx)
    return np.argsort(pos), pos


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2)])
def test_full_striped_tile_is_causal_attention_of_the_sequence(hq, hkv):
    """A tile whose Q and KV lists name every partition (any order) computes
    causal attention of the whole sequence: after sorting rows by position it
    equals the library's causal SDPA."""
    n, P, d = 4, 12, 16
    prob = _prob(n, P, hq, hkv, d)
    q_idx, kv_idx = [2, 0, 3, 1], [1, 3, 0, 2]
    q = _rand((n * P, hq, d), 1)
    k, v = _rand((n * P, hkv, d), 2), _rand((n * P, hkv, d), 3)
    o, lse = tile_forward(prob, q_idx, kv_idx, q, k, v)
    qo, qpos = _position_order(prob, q_idx)
    ko, kpos = _position_order(prob, kv_idx)
    np.testing.assert_array_equal(qpos[qo], np.arange(n * P))
    np.testing.assert_array_equal(kpos[ko], np.arange(n * P))
    tq = torch.from_numpy(q[qo]).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k[ko]).permute(1, 0, 2)[None]
    tv = torch.from_numpy(v[ko]).permute(1, 0, 2)[None]
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True,
                                         scale=prob["softmax_scale"],
                                         enable_gqa=hq != hkv)
    np.testing.assert_allclose(o[qo], ref[0].permute(1, 0, 2).numpy(),
                               rtol=0, atol=1e-12)
    # LSE: library log-sum-exp of the causally masked scores.
    g = hq // hkv
    for h in range(hq):
        x = torch.from_numpy(prob["softmax_scale"] * q[qo, h] @ k[ko, h // g].T)
        x = x.masked_fill(torch.ones(n * P, n * P, dtype=torch.bool).triu(1),
                          float("-inf"))
        np.testing.assert_allclose(lse[h, qo], torch.logsumexp(x, 1).numpy(),
                                   rtol=0, atol=1e-12)


def test_striped_first_token_closed_form():
    """Position 0 is token 0 of partition 0: it sees only itself, so O = v_0
    and LSE = s q_0 . k_0; the token at position 1 (token 0 of partition 1)
    sees positions 0 and 1 only."""
    n, P, d = 3, 4, 8
    prob = _prob(n, P, 1, 1, d)
    q = _rand((n * P, 1, d), 4)
    k, v = _rand((n * P, 1, d), 5), _rand((n * P, 1, d), 6)
    o, lse = tile_forward(prob, [0, 1, 2], [0, 1, 2], q, k, v)
    s = prob["softmax_scale"]
    np.testing.assert_allclose(o[0, 0], v[0, 0], atol=1e-12)
    assert abs(lse[0, 0] - s * q[0, 0] @ k[0, 0]) < 1e-12
    r1 = P  # buffer row of token 0 of partition 1
    x = np.array([s * q[r1, 0] @ k[0, 0], s * q[r1, 0] @ k[r1, 0]])
    w = np.exp(x - x.max())
    np.testing.assert_allclose(o[r1, 0], (w[0] * v[0, 0] + w[1] * v[r1, 0])
                               / w.sum(), atol=1e-12)


@pytest.mark.parametrize("bm,bn", [(16, 8), (8, 8), (32, 8)])
def test_striped_pair_block_closed_form(bm, bn):
    """Under the striped layout every partition pair is near-triangular: key
    row r' is visible to query row r iff r' < r, or r' = r and the key's
    partition is not after the query's.  With bm = rho * bn, Q block qb of any
    pair therefore has rho*qb FULL blocks, then rho PARTIAL, then EMPTY ones,
    whichever of the two partitions comes first."""
    n, P = 4, 64
    rho = bm // bn
    idx = [0, 1, 2, 3]
    cls = classify_blocks(idx, idx, P, bm, bn, True, STRIPED, n)
    nqb, nkb = P // bm, P // bn
    for a in range(n):
        for b in range(n):
            sub = cls[a * nqb:(a + 1) * nqb, b * nkb:(b + 1) * nkb]
            for qb in range(nqb):
                want = np.full(nkb, EMPTY)
                want[:rho * qb] = FULL
                want[rho * qb:rho * (qb + 1)] = PARTIAL
                np.testing.assert_array_equal(sub[qb], want)
    np.testing.assert_array_equal(
        cls, classify_blocks_bruteforce(idx, idx, P, bm, bn, True, STRIPED, n))


def test_striped_element_rule_on_the_diagonal():
    """Blocks of one row: the class of (query row r, key row r') is FULL iff
    r' < r or (r' = r and kv partition <= q partition)."""
    n, P = 3, 5
    for qp in range(n):
        for kp in range(n):
            cls = classify_blocks([qp], [kp], P, 1, 1, True, STRIPED, n)
            r = np.arange(P)
            want = (r[None, :] < r[:, None]) | (
                (r[None, :] == r[:, None]) & (kp <= qp))
            np.testing.assert_array_equal(cls == FULL, want)
            np.testing.assert_array_equal(cls == EMPTY, ~want)


def test_striped_classes_match_bruteforce_random_tiles():
    rng = np.random.default_rng(7)
    for _ in range(20):
        n = int(rng.integers(2, 9))
        P = int(rng.choice([8, 16, 32]))
        bm = int(rng.choice([b for b in (4, 8, 16) if P % b == 0]))
        bn = int(rng.choice([b for b in (4, 8) if P % b == 0]))
        q_idx = list(rng.choice(n, int(rng.integers(1, n + 1)), replace=False))
        kv_idx = list(rng.choice(n, int(rng.integers(1, n + 1)), replace=False))
        np.testing.assert_array_equal(
            classify_blocks(q_idx, kv_idx, P, bm, bn, True, STRIPED, n),
            classify_blocks_bruteforce(q_idx, kv_idx, P, bm, bn, True,
                                       STRIPED, n))


def test_striped_merge_over_kv_split_equals_whole_footprint():
    """Merging the partials of a KV footprint split over several tiles (the
    RS-Q reduction of Algorithm 2) gives the tile over the whole footprint."""
    n, P, d = 6, 8, 16
    prob = _prob(n, P, 2, 2, d)
    q_idx = [5, 1, 3]
    parts = [[0, 4], [2], [5, 3, 1]]
    q = _rand((len(q_idx) * P, 2, d), 8)
    kv_all = [p for part in parts for p in part]
    k = _rand((n * P, 2, d), 9)
    v = _rand((n * P, 2, d), 10)

    def rows_of(idx):
        return np.concatenate([np.arange(P) + kv_all.index(p) * P for p in idx])

    o_full, lse_full = tile_forward(prob, q_idx, kv_all, q, k, v)
    os_, ls_ = [], []
    for part in parts:
        r = rows_of(part)
        o_p, l_p = tile_forward(prob, q_idx, part, q, k[r], v[r])
        os_.append(o_p)
        ls_.append(l_p)
    for h in range(2):
        o_m, lse_m = lse_merge(np.stack([o_p[:, h] for o_p in os_]),
                               np.stack([l_p[h] for l_p in ls_]))
        np.testing.assert_allclose(o_m, o_full[:, h], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse_m, lse_full[h], rtol=0, atol=1e-12)


def test_full_striped_tile_backward_matches_autograd():
    """Gradients of the whole-sequence striped tile equal torch autograd of
    causal SDPA on the position-ordered sequence (float64)."""
    n, P, d, hq, hkv = 3, 8, 16, 4, 2
    prob = _prob(n, P, hq, hkv, d)
    q_idx, kv_idx = [1, 2, 0], [2, 0, 1]
    q = _rand((n * P, hq, d), 11)
    k, v = _rand((n * P, hkv, d), 12), _rand((n * P, hkv, d), 13)
    do = _rand((n * P, hq, d), 14)
    dq, dk, dv, q_heads, _ = tile_backward(prob, q_idx, kv_idx, q, k, v, do)
    assert q_heads == list(range(hq))
    qo, _ = _position_order(prob, q_idx)
    ko, _ = _position_order(prob, kv_idx)
    tq = torch.from_numpy(q[qo]).permute(1, 0, 2)[None].requires_grad_()
    tk = torch.from_numpy(k[ko]).permute(1, 0, 2)[None].requires_grad_()
    tv = torch.from_numpy(v[ko]).permute(1, 0, 2)[None].requires_grad_()
    out = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True,
                                         scale=prob["softmax_scale"],
                                         enable_gqa=True)
    out.backward(torch.from_numpy(do[qo]).permute(1, 0, 2)[None])
    np.testing.assert_allclose(dq[qo], tq.grad[0].permute(1, 0, 2).numpy(),
                               rtol=0, atol=1e-10)
    np.testing.assert_allclose(dk[ko], tk.grad[0].permute(1, 0, 2).numpy(),
                               rtol=0, atol=1e-10)
    np.testing.assert_allclose(dv[ko], tv.grad[0].permute(1, 0, 2).numpy(),
                               rtol=0, atol=1e-10)

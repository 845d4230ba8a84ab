"""Pins of the oracle's forward and merge against things other than itself:
a library routine (torch scaled_dot_product_attention and logsumexp in float64
on the CPU), closed forms, invariants and brute force on tiny inputs."""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import attention_rows, lse_merge, tile_forward, token_positions


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _sdpa(q, k, v, causal, scale, gqa=False):
    """torch SDPA in float64 on [rows, heads, d] numpy arrays."""
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2)[None]
    out = F.scaled_dot_product_attention(tq, tk, tv, is_causal=causal,
                                         scale=scale, enable_gqa=gqa)
    return out[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("d", [16, 64])
def test_rows_match_torch_sdpa(causal, d):
    S = 48
    q, k, v = (_rand((S, d), s) for s in (1, 2, 3))
    scale = 1.0 / math.sqrt(d)
    pos = np.arange(S)
    o, lse = attention_rows(q, k, v, pos, pos, causal, scale)
    ref = _sdpa(q[:, None], k[:, None], v[:, None], causal, scale)[:, 0]
    np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)
    # LSE against the library log-sum-exp of the masked scores.
    x = torch.from_numpy(scale * q @ k.T)
    if causal:
        x = x.masked_fill(torch.ones(S, S, dtype=torch.bool).triu(1),
                          float("-inf"))
    np.testing.assert_allclose(lse, torch.logsumexp(x, dim=1).numpy(),
                               rtol=0, atol=1e-12)


def test_rows_match_bruteforce_loops():
    """Pure-Python loops with math.exp on a tiny case."""
    S, d = 6, 3
    q, k, v = _rand((S, d), 4), _rand((S, d), 5), _rand((S, d), 6)
    scale = 0.7
    pos = np.array([3, 9, 10, 11, 20, 21])
    o, lse = attention_rows(q, k, v, pos, pos, True, scale)
    for i in range(S):
        xs = [scale * sum(q[i, c] * k[j, c] for c in range(d))
              if pos[j] <= pos[i] else None for j in range(S)]
        z = sum(math.exp(x) for x in xs if x is not None)
        assert abs(lse[i] - math.log(z)) < 1e-12
        for c in range(d):
            want = sum(math.exp(x) / z * v[j, c]
                       for j, x in enumerate(xs) if x is not None)
            assert abs(o[i, c] - want) < 1e-12


def test_closed_form_zero_keys_uniform():
    """K = 0: every allowed key has score 0, so O is the mean of the allowed V
    rows and LSE = ln |J|."""
    S, d = 40, 8
    q, v = _rand((S, d), 7), _rand((S, d), 8)
    k = np.zeros((S, d))
    pos = np.arange(S)
    o, lse = attention_rows(q, k, v, pos, pos, True, 0.3)
    for i in range(S):
        np.testing.assert_allclose(o[i], v[:i + 1].mean(axis=0), atol=1e-13)
        assert abs(lse[i] - math.log(i + 1)) < 1e-13


def test_closed_form_first_token_and_constant_v():
    S, d = 32, 8
    q, k = _rand((S, d), 9), _rand((S, d), 10)
    pos = np.arange(S)
    v = _rand((S, d), 11)
    o, lse = attention_rows(q, k, v, pos, pos, True, 0.25)
    # causal row 0 sees only key 0: O = v_0, LSE = x_00.
    np.testing.assert_allclose(o[0], v[0], atol=1e-15)
    assert abs(lse[0] - 0.25 * float(q[0] @ k[0])) < 1e-13
    # V constant along keys: O equals that constant for every row.
    vc = np.tile(_rand((1, d), 12), (S, 1))
    o2, _ = attention_rows(q, k, vc, pos, pos, False, 0.25)
    np.testing.assert_allclose(o2, vc, atol=1e-13)


def test_no_visible_key_gives_zero_and_neg_inf():
    q, k, v = _rand((4, 8), 1), _rand((5, 8), 2), _rand((5, 8), 3)
    o, lse = attention_rows(q, k, v, np.arange(4), np.arange(10, 15), True, 1.0)
    assert np.all(o == 0.0) and np.all(np.isneginf(lse))


def test_convex_combination():
    """Weights exp(x_j - LSE) are >= 0 and sum to 1; so per channel O lies in
    [min_J v_j, max_J v_j]."""
    S, d = 64, 16
    q, k, v = (_rand((S, d), s) * 3 for s in (13, 14, 15))
    pos = np.arange(S)
    o, lse = attention_rows(q, k, v, pos, pos, True, 0.5)
    x = 0.5 * q @ k.T
    for i in range(S):
        w = np.exp(x[i, :i + 1] - lse[i])
        assert np.all(w >= 0) and abs(w.sum() - 1) < 1e-12
        assert np.all(o[i] >= v[:i + 1].min(axis=0) - 1e-12)
        assert np.all(o[i] <= v[:i + 1].max(axis=0) + 1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_merge_over_any_split_equals_full(causal):
    """The online-softmax reducer merges partials over disjoint key sets
    exactly (Section 2.2): any split of the keys, merged, equals attention over
    all of them -- including splits with parts that are invisible to a row."""
    rng = np.random.default_rng(21)
    S, d = 96, 16
    q, k, v = (rng.standard_normal((S, d)) for _ in range(3))
    pos = np.arange(S)
    full_o, full_lse = attention_rows(q, k, v, pos, pos, causal, 0.4)
    for trial in range(5):
        cuts = np.sort(rng.choice(np.arange(1, S), size=trial + 2,
                                  replace=False))
        bounds = np.concatenate(([0], cuts, [S, S]))  # last part is empty
        perm = rng.permutation(S) if trial % 2 else np.arange(S)
        parts_o, parts_l = [], []
        for a, b in zip(bounds[:-1], bounds[1:]):
            sel = perm[a:b]
            po, pl = attention_rows(q, k[sel], v[sel], pos, pos[sel], causal,
                                    0.4)
            parts_o.append(po)
            parts_l.append(pl)
        mo, ml = lse_merge(np.stack(parts_o), np.stack(parts_l))
        np.testing.assert_allclose(mo, full_o, rtol=0, atol=1e-12)
        np.testing.assert_allclose(ml, full_lse, rtol=0, atol=1e-12)


def test_merge_lse_is_library_logsumexp_and_all_empty():
    rng = np.random.default_rng(3)
    lse = rng.standard_normal((5, 7)) * 5
    lse[1, 2] = -np.inf
    lse[:, 6] = -np.inf
    o = rng.standard_normal((5, 7, 4))
    mo, ml = lse_merge(o, lse)
    ref = torch.logsumexp(torch.from_numpy(lse), dim=0).numpy()
    np.testing.assert_allclose(ml[:6], ref[:6], atol=1e-12)
    assert np.isneginf(ml[6]) and np.all(mo[6] == 0)
    w = np.exp(lse[:, 0] - ref[0])
    np.testing.assert_allclose(mo[0], (w[:, None] * o[:, 0]).sum(0),
                               atol=1e-12)


def test_single_part_merge_is_identity():
    rng = np.random.default_rng(5)
    o = rng.standard_normal((1, 9, 3))
    lse = rng.standard_normal((1, 9))
    mo, ml = lse_merge(o, lse)
    np.testing.assert_allclose(mo, o[0], atol=1e-15)
    np.testing.assert_allclose(ml, lse[0], atol=1e-15)


@pytest.mark.parametrize("causal", [False, True])
def test_tile_covering_whole_sequence_is_full_attention(causal):
    """A tile whose Q and KV lists both cover every partition is plain
    attention over the whole sequence (library routine), whatever the list
    order."""
    n, P, H, d = 4, 16, 2, 8
    rng = np.random.default_rng(31)
    q, k, v = (rng.standard_normal((n * P, H, d)) for _ in range(3))
    prob = dict(partition_len=P, num_q_heads=H, num_kv_heads=H,
                causal=causal, softmax_scale=0.35)
    o, lse = tile_forward(prob, list(range(n)), list(range(n)), q, k, v)
    np.testing.assert_allclose(o, _sdpa(q, k, v, causal, 0.35), atol=1e-12)
    # Permuted KV list: the KV buffer is stacked in list order.
    order = [2, 0, 3, 1]
    kp = np.concatenate([k[p * P:(p + 1) * P] for p in order])
    vp = np.concatenate([v[p * P:(p + 1) * P] for p in order])
    o2, lse2 = tile_forward(prob, list(range(n)), order, q, kp, vp)
    np.testing.assert_allclose(o2, o, atol=1e-12)
    np.testing.assert_allclose(lse2, lse, atol=1e-12)


def test_causal_tile_with_all_past_keys_is_full_causal_rows():
    """Shape of the causal 64K workload, scaled down: Q partitions {4..7} over
    KV partitions {0..7} of a 16-partition sequence.  The KV list holds every
    key at or before the Q rows, so the tile equals rows 4P..8P-1 of causal
    attention over the first 8P tokens (library routine)."""
    P, H, d = 8, 2, 16
    rng = np.random.default_rng(41)
    q_all, k_all, v_all = (rng.standard_normal((8 * P, H, d)) for _ in range(3))
    prob = dict(partition_len=P, num_q_heads=H, num_kv_heads=H, causal=True,
                softmax_scale=0.25)
    o, _ = tile_forward(prob, [4, 5, 6, 7], list(range(8)),
                        q_all[4 * P:], k_all, v_all)
    ref = _sdpa(q_all, k_all, v_all, True, 0.25)[4 * P:]
    np.testing.assert_allclose(o, ref, atol=1e-12)


def test_gqa_head_map_matches_library():
    """Consecutive query heads share a KV head (Section 4.8); torch's
    enable_gqa uses the same grouping."""
    P, hq, hkv, d = 16, 8, 2, 8
    rng = np.random.default_rng(51)
    q = rng.standard_normal((2 * P, hq, d))
    k, v = (rng.standard_normal((2 * P, hkv, d)) for _ in range(2))
    prob = dict(partition_len=P, num_q_heads=hq, num_kv_heads=hkv,
                causal=True, softmax_scale=0.3)
    o, _ = tile_forward(prob, [0, 1], [0, 1], q, k, v)
    np.testing.assert_allclose(o, _sdpa(q, k, v, True, 0.3, gqa=True),
                               atol=1e-12)
    assert [oracle.q_head_to_kv_head(h, hq, hkv) for h in range(hq)] == \
        [0, 0, 0, 0, 1, 1, 1, 1]


def test_tile_row_and_head_selection():
    P, H, d = 16, 3, 8
    rng = np.random.default_rng(61)
    q = rng.standard_normal((2 * P, H, d))
    k, v = (rng.standard_normal((3 * P, H, d)) for _ in range(2))
    prob = dict(partition_len=P, num_q_heads=H, num_kv_heads=H, causal=True,
                softmax_scale=0.3)
    o, lse = tile_forward(prob, [2, 5], [1, 2, 3], q, k, v)
    rows = [0, 5, 17, 31]
    o2, lse2 = tile_forward(prob, [2, 5], [1, 2, 3], q, k, v, rows=rows,
                            heads=[2, 0])
    np.testing.assert_allclose(o2, o[rows][:, [2, 0]], atol=0)
    np.testing.assert_allclose(lse2, lse[[2, 0]][:, rows], atol=0)


def test_positions_are_contiguous_partitions():
    pos = token_positions([3, 1], 4)
    assert pos.tolist() == [12, 13, 14, 15, 4, 5, 6, 7]

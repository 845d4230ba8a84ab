"""Pins of the oracle's gradients: torch autograd through float64 SDPA
(library routine), central finite differences, and the identities that hold
when O and LSE are consistent over the full key set."""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import attention_rows, attention_rows_bwd, tile_backward


def _autograd(q, k, v, do, causal, scale, gqa=False):
    tq, tk, tv = (torch.from_numpy(a).permute(1, 0, 2)[None].requires_grad_()
                  for a in (q, k, v))
    out = F.scaled_dot_product_attention(tq, tk, tv, is_causal=causal,
                                         scale=scale, enable_gqa=gqa)
    out.backward(torch.from_numpy(do).permute(1, 0, 2)[None])
    return tuple(t.grad[0].permute(1, 0, 2).numpy() for t in (tq, tk, tv))


@pytest.mark.parametrize("causal", [False, True])
def test_rows_bwd_matches_autograd(causal):
    S, d, scale = 40, 16, 0.3
    rng = np.random.default_rng(1)
    q, k, v, do = (rng.standard_normal((S, d)) for _ in range(4))
    pos = np.arange(S)
    o, lse = attention_rows(q, k, v, pos, pos, causal, scale)
    D = (do * o).sum(1)
    dq, dk, dv = attention_rows_bwd(q, k, v, do, lse, D, pos, pos, causal,
                                    scale)
    rq, rk, rv = _autograd(q[:, None], k[:, None], v[:, None], do[:, None],
                           causal, scale)
    for a, b in ((dq, rq[:, 0]), (dk, rk[:, 0]), (dv, rv[:, 0])):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-11)


def test_rows_bwd_finite_differences():
    """Central differences of f = <dO, O(q, k, v)> in float64."""
    S, d, scale, h = 6, 4, 0.5, 1e-6
    rng = np.random.default_rng(2)
    q, k, v, do = (rng.standard_normal((S, d)) for _ in range(4))
    pos = np.arange(S) * 2

    def f(q_, k_, v_):
        return float((attention_rows(q_, k_, v_, pos, pos, True, scale)[0]
                      * do).sum())

    o, lse = attention_rows(q, k, v, pos, pos, True, scale)
    dq, dk, dv = attention_rows_bwd(q, k, v, do, lse, (do * o).sum(1), pos,
                                    pos, True, scale)
    for which, grad in ((0, dq), (1, dk), (2, dv)):
        num = np.zeros_like(grad)
        for idx in np.ndindex(*grad.shape):
            args_p = [q.copy(), k.copy(), v.copy()]
            args_m = [q.copy(), k.copy(), v.copy()]
            args_p[which][idx] += h
            args_m[which][idx] -= h
            num[idx] = (f(*args_p) - f(*args_m)) / (2 * h)
        err = np.abs(num - grad).max() / max(np.abs(grad).max(), 1e-30)
        assert err < 1e-6, (which, err)


def test_tile_backward_gqa_matches_autograd_and_identities():
    """Tile backward with GQA (dK, dV summed over the query heads of a group)
    against autograd; when the tile holds every visible key, sum_j dK_j = 0 and
    sum_j dV_j = sum_i dO_i per head group."""
    P, hq, hkv, d, scale = 8, 4, 2, 8, 0.4
    rng = np.random.default_rng(3)
    q, do = (rng.standard_normal((4 * P, hq, d)) for _ in range(2))
    k, v = (rng.standard_normal((4 * P, hkv, d)) for _ in range(2))
    prob = dict(partition_len=P, num_q_heads=hq, num_kv_heads=hkv,
                causal=True, softmax_scale=scale)
    idx = [0, 1, 2, 3]
    dq, dk, dv, q_heads, _ = tile_backward(prob, idx, idx, q, k, v, do,
                                           row_chunk=7)
    rq, rk, rv = _autograd(q, k, v, do, True, scale, gqa=True)
    assert q_heads == [0, 1, 2, 3]
    np.testing.assert_allclose(dq, rq, atol=1e-11)
    np.testing.assert_allclose(dk, rk, atol=1e-11)
    np.testing.assert_allclose(dv, rv, atol=1e-11)
    np.testing.assert_allclose(dk.sum(0), 0.0, atol=1e-10)
    grp = do.reshape(4 * P, hkv, hq // hkv, d).sum(axis=(0, 2))
    np.testing.assert_allclose(dv.sum(0), grp, atol=1e-10)


def test_tile_backward_row_selection():
    P, H, d, scale = 8, 2, 8, 0.4
    rng = np.random.default_rng(4)
    q, do = (rng.standard_normal((2 * P, H, d)) for _ in range(2))
    k, v = (rng.standard_normal((3 * P, H, d)) for _ in range(2))
    prob = dict(partition_len=P, num_q_heads=H, num_kv_heads=H, causal=True,
                softmax_scale=scale)
    full = tile_backward(prob, [1, 2], [0, 1, 2], q, k, v, do)
    part = tile_backward(prob, [1, 2], [0, 1, 2], q, k, v, do, kv_heads=[1],
                         q_rows=[0, 9], kv_rows=[3, 20])
    np.testing.assert_allclose(part[0], full[0][[0, 9]][:, [1]], atol=1e-13)
    np.testing.assert_allclose(part[1], full[1][[3, 20]][:, [1]], atol=1e-13)
    np.testing.assert_allclose(part[2], full[2][[3, 20]][:, [1]], atol=1e-13)

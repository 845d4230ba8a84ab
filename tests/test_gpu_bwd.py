"""GPU parity of mesh_attn_tile_bwd against the float64 oracle, through the C
ABI.  The GPU backward consumes the GPU forward's O (bf16) and LSE, as a
caller would; the oracle recomputes its own float64 forward."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2512_20968_amd as ma
from mesh_inputs import WORKLOADS, make_grad, make_qkv, sample_rows

from helpers import check_grad, log, run_fwd, to_np

pytestmark = pytest.mark.gpu


def _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse, accumulate=0, init=None):
    P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads, cfg.num_kv_heads,
                     cfg.head_dim)
    dev = qd.device
    if init is None:
        dq = torch.empty((cfg.nq * P, hq, d), dtype=torch.float32, device=dev)
        dk = torch.empty((cfg.nkv * P, hkv, d), dtype=torch.float32,
                         device=dev)
        dv = torch.empty_like(dk)
    else:
        dq, dk, dv = (t.clone() for t in init)
    ma.mesh_attn_tile_bwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o, dod, lse,
                          dq, dk, dv, accumulate=accumulate)
    return dq, dk, dv


def _setup(cfg, gpu):
    q, k, v, _ = make_qkv(cfg)
    do = make_grad(cfg)
    qd, kd, vd, dod = (t.to(gpu) for t in (q, k, v, do))
    prob = cfg.problem()
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    return prob, (q, k, v, do), (qd, kd, vd, dod), o, lse


SMALL = [
    # (q_idx, kv_idx, hq, hkv, d, causal)
    ([0, 1], [0, 1], 4, 4, 64, False),
    ([0, 1], [0, 1], 4, 4, 64, True),
    ([2, 3], [0, 1, 2, 3], 4, 2, 128, True),
    ([3, 1], [1, 0, 3], 6, 3, 128, True),
    ([1, 2], [0, 3], 2, 1, 128, False),
]

# Several blocks per partition (P = 1024: 8 dQ Q blocks and 8 dK/dV KV
# blocks per partition) at both head dims.
MULTI = [
    # (q_idx, kv_idx, hq, hkv, d)
    ([2, 1], [0, 2, 1], 4, 2, 64),
    ([2, 1], [0, 2, 1], 2, 1, 128),
]


@pytest.mark.parametrize("q_idx,kv_idx,hq,hkv,d,causal", SMALL)
def test_small_tiles_every_row(gpu, q_idx, kv_idx, hq, hkv, d, causal):
    """Small tiles (GQA, both head dims, causal and not, permuted lists):
    every row of dQ, dK, dV checked."""
    cfg = dataclasses.replace(WORKLOADS["tiny-nc"], num_partitions=4, partition_len=256,
                              q_idx=q_idx, kv_idx=kv_idx, num_q_heads=hq,
                              num_kv_heads=hkv, head_dim=d, causal=causal,
                              seed=21, grad_seed=22)
    prob, (q, k, v, do), (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    dq, dk, dv = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    torch.cuda.synchronize()
    rdq, rdk, rdv, q_heads, _ = oracle.tile_backward(
        prob, q_idx, kv_idx, to_np(q), to_np(k), to_np(v), to_np(do))
    tag = f"tile {q_idx}x{kv_idx} hq={hq} hkv={hkv} d={d} c={causal}"
    check_grad(f"{tag} dq", to_np(dq), rdq)
    check_grad(f"{tag} dk", to_np(dk), rdk)
    check_grad(f"{tag} dv", to_np(dv), rdv)


@pytest.mark.parametrize("q_idx,kv_idx,hq,hkv,d", MULTI)
def test_multi_block_partitions_every_row(gpu, q_idx, kv_idx, hq, hkv, d):
    """Causal GQA tile with 1024-token partitions (diagonal pairs spanning
    several blocks, a permuted KV list): every row of dQ, dK, dV."""
    cfg = dataclasses.replace(WORKLOADS["tiny-nc"], num_partitions=3,
                              partition_len=1024, q_idx=q_idx, kv_idx=kv_idx,
                              num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                              causal=True, seed=41, grad_seed=42)
    prob, (q, k, v, do), (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    dq, dk, dv = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    torch.cuda.synchronize()
    rdq, rdk, rdv, _, _ = oracle.tile_backward(
        prob, q_idx, kv_idx, to_np(q), to_np(k), to_np(v), to_np(do))
    tag = f"P=1024 tile {q_idx}x{kv_idx} hq={hq} hkv={hkv} d={d}"
    check_grad(f"{tag} dq", to_np(dq), rdq)
    check_grad(f"{tag} dk", to_np(dk), rdk)
    check_grad(f"{tag} dv", to_np(dv), rdv)


def test_rows_and_keys_nobody_sees(gpu):
    """Causal tile {0, 2} x {1, 3}: the rows of Q partition 0 see no key and
    the keys of KV partition 3 are seen by no row.  Their gradient rows must
    be exactly zero (written into uninitialised outputs), every other row
    within tolerance of the oracle."""
    cfg = dataclasses.replace(WORKLOADS["tiny-nc"], num_partitions=4, partition_len=256,
                              q_idx=[0, 2], kv_idx=[1, 3], num_q_heads=4,
                              num_kv_heads=2, head_dim=128, causal=True,
                              seed=21, grad_seed=22)
    P = cfg.partition_len
    prob, (q, k, v, do), (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    assert torch.all(torch.isneginf(lse[:, :P]))
    dq, dk, dv = (torch.full_like(t, float("nan"))
                  for t in _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse))
    ma.mesh_attn_tile_bwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o, dod,
                          lse, dq, dk, dv)
    torch.cuda.synchronize()
    assert torch.all(dq[:P] == 0), "dQ of rows without a visible key"
    assert torch.all(dk[P:] == 0) and torch.all(dv[P:] == 0), \
        "dK, dV of keys no row sees"
    rdq, rdk, rdv, _, _ = oracle.tile_backward(
        prob, cfg.q_idx, cfg.kv_idx, to_np(q), to_np(k), to_np(v), to_np(do))
    check_grad("unseen rows/keys dq", to_np(dq), rdq)
    check_grad("unseen rows/keys dk", to_np(dk), rdk)
    check_grad("unseen rows/keys dv", to_np(dv), rdv)


def test_accumulate_adds_into_outputs(gpu):
    cfg = dataclasses.replace(WORKLOADS["tiny-nc"], causal=True, seed=31, grad_seed=32)
    prob, _, (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    g1 = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    init = tuple(torch.randn_like(t) for t in g1)
    g2 = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse, accumulate=1, init=init)
    torch.cuda.synchronize()
    for a, b, c in zip(g1, g2, init):
        torch.testing.assert_close(b, a + c, rtol=0, atol=1e-5)


def test_backward_is_deterministic(gpu):
    cfg = dataclasses.replace(WORKLOADS["causal-64k"], q_idx=[6, 7], kv_idx=[0, 5, 6, 7],
                              partition_len=1024, num_q_heads=8,
                              num_kv_heads=8, grad_seed=4)
    prob, _, (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    a = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    b = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_causal64k_backward_sampled_rows(gpu):
    """Full-size backward of the causal 64K tile.  The oracle runs its own
    float64 forward for every row of three heads, then checks dQ on the
    sampled Q rows and dK, dV on sampled KV rows of those heads.  On all
    heads, two identities that hold because the tile holds every key the Q
    rows can see: sum_j dK_j = 0 and sum_j dV_j = sum_i dO_i."""
    cfg = WORKLOADS["bwd-causal-64k"]
    prob, (q, k, v, do), (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    log("causal-64k backward: GPU")
    dq, dk, dv = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    torch.cuda.synchronize()
    # Identities, all heads.  P and dS are rounded to bf16 before the MFMAs
    # (relative error 2^-9 per term, random-walking over ~10^4 terms), so the
    # sums are compared with the L1 mass of the terms they add up.
    sdk = dk.sum(0)
    sdv = dv.sum(0)
    sdo = dod.float().sum(0)
    mass_k = dk.abs().sum(0)
    mass_v = dv.abs().sum(0)
    rk = float((sdk.abs() / mass_k).max())
    rv = float(((sdv - sdo).abs() / mass_v).max())
    log(f"causal-64k backward: max |sum dK| / sum|dK| = {rk:.3e}, "
        f"max |sum dV - sum dO| / sum|dV| = {rv:.3e}")
    assert rk <= 1e-2 and rv <= 1e-2
    heads = [0, 17, 31]
    q_rows = sample_rows(cfg, cfg.nq)
    kv_rows = sample_rows(cfg, cfg.nkv, seed_offset=2000)
    log(f"causal-64k backward: oracle on heads {heads}, {len(q_rows)} dQ rows, "
        f"{len(kv_rows)} dK/dV rows")
    rdq, rdk, rdv, q_heads, _ = oracle.tile_backward(
        prob, cfg.q_idx, cfg.kv_idx, to_np(q), to_np(k), to_np(v), to_np(do),
        kv_heads=heads, q_rows=q_rows, kv_rows=kv_rows)
    qr = torch.tensor(q_rows, device=gpu)
    kr = torch.tensor(kv_rows, device=gpu)
    check_grad("causal-64k dq", to_np(dq[qr][:, q_heads]), rdq)
    check_grad("causal-64k dk", to_np(dk[kr][:, heads]), rdk)
    check_grad("causal-64k dv", to_np(dv[kr][:, heads]), rdv)


def test_mesh1m_gqa_backward_full_size(gpu):
    """Backward at the 1M-token non-causal GQA tile's full size (65536 rows,
    32 query heads on 8 KV heads).  dQ of sampled rows of two query heads (in
    different KV groups) against the float64 definition on those rows; on
    every KV head, the identities that hold because each row's softmax runs
    over exactly the tile's keys: sum_j dK_j = 0 and sum_j dV_j = sum of dO
    over the rows and the query heads of the group."""
    from oracle.attention import (attention_rows, attention_rows_bwd,
                                  problem_positions)
    cfg = dataclasses.replace(WORKLOADS["mesh1m-nc-gqa"], grad_seed=8)
    prob, (q, k, v, do), (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    log("mesh1m-nc-gqa backward: GPU")
    dq, dk, dv = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    torch.cuda.synchronize()
    g = cfg.num_q_heads // cfg.num_kv_heads
    sdk = dk.sum(0)
    sdv = dv.sum(0)
    sdo = dod.float().sum(0).view(cfg.num_kv_heads, g, -1).sum(1)
    rk = float((sdk.abs() / dk.abs().sum(0)).max())
    rv = float(((sdv - sdo).abs() / dv.abs().sum(0)).max())
    log(f"mesh1m-nc-gqa backward: max |sum dK| / sum|dK| = {rk:.3e}, "
        f"max |sum dV - sum dO| / sum|dV| = {rv:.3e}")
    assert rk <= 1e-2 and rv <= 1e-2
    rows = np.asarray(sample_rows(cfg, cfg.nq, n_random=16))
    qpos = problem_positions(prob, cfg.q_idx)
    kpos = problem_positions(prob, cfg.kv_idx)
    scale = float(prob["softmax_scale"])
    for h in (0, 29):
        hk = h // g
        f64 = lambda t: t.double().numpy()
        qh, doh = f64(q[rows, h]), f64(do[rows, h])
        kh, vh = f64(k[:, hk]), f64(v[:, hk])
        oh, lh = attention_rows(qh, kh, vh, qpos[rows], kpos, False, scale)
        D = np.sum(doh * oh, axis=1)
        rdq, _, _ = attention_rows_bwd(qh, kh, vh, doh, lh, D, qpos[rows],
                                       kpos, False, scale)
        got = to_np(dq[torch.as_tensor(rows, device=gpu), h])
        check_grad(f"mesh1m-nc-gqa dq head {h} ({len(rows)} rows)", got, rdq)

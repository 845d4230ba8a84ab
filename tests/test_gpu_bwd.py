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

from helpers import (check_grad, log, oracle_backward_rows, queued_tail_config,
                     run_fwd, to_np)

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


def _gpu_backward_cpu(cfg, gpu):
    """GPU forward and backward of a full-size workload; inputs and gradients
    returned as CPU tensors (the device copies are freed)."""
    prob, (q, k, v, do), (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    log(f"{cfg.name}: GPU backward")
    dq, dk, dv = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    torch.cuda.synchronize()
    out = dict(prob=prob, q=q, k=k, v=v, do=do, dq=dq.cpu(), dk=dk.cpu(),
               dv=dv.cpu())
    del qd, kd, vd, dod, o, lse, dq, dk, dv
    torch.cuda.empty_cache()
    return out


@pytest.fixture(scope="module")
def bwd64k(gpu):
    return _gpu_backward_cpu(WORKLOADS["bwd-causal-64k"], gpu)


@pytest.fixture(scope="module")
def bwd1m(gpu):
    return _gpu_backward_cpu(
        dataclasses.replace(WORKLOADS["mesh1m-nc-gqa"], grad_seed=8), gpu)


def test_causal64k_backward_identities(bwd64k):
    """Full-size backward of the causal 64K tile, all heads: the tile holds
    every key its Q rows can see, so sum_j dK_j = 0 and sum_j dV_j = sum_i
    dO_i.  P and dS are rounded to bf16 before the MFMAs (relative error 2^-9
    per term, random-walking over ~10^4 terms), so the sums are compared with
    the L1 mass of the terms they add up."""
    dk, dv, do = bwd64k["dk"], bwd64k["dv"], bwd64k["do"]
    rk = float((dk.sum(0).abs() / dk.abs().sum(0)).max())
    rv = float(((dv.sum(0) - do.float().sum(0)).abs() / dv.abs().sum(0)).max())
    log(f"causal-64k backward: max |sum dK| / sum|dK| = {rk:.3e}, "
        f"max |sum dV - sum dO| / sum|dV| = {rv:.3e}")
    assert rk <= 1e-2 and rv <= 1e-2


@pytest.mark.parametrize("heads", [range(0, 16), range(16, 32)],
                         ids=["heads0-15", "heads16-31"])
def test_causal64k_backward_sampled_rows(bwd64k, heads):
    """Full-size backward of the causal 64K tile against the float64 oracle,
    on every head (half of them per test): dQ on the sampled Q rows and dK,
    dV on the sampled KV rows.  The oracle's forward covers every row of
    each head (its LSE and D enter every dK, dV row)."""
    cfg = WORKLOADS["bwd-causal-64k"]
    b = bwd64k
    heads = list(heads)
    q_rows = sample_rows(cfg, cfg.nq)
    kv_rows = sample_rows(cfg, cfg.nkv, seed_offset=2000)
    log(f"causal-64k backward: oracle on heads {heads[0]}..{heads[-1]}, "
        f"{len(q_rows)} dQ rows, {len(kv_rows)} dK/dV rows")
    rdq, rdk, rdv, q_heads = oracle_backward_rows(
        b["prob"], cfg.q_idx, cfg.kv_idx, b["q"], b["k"], b["v"], b["do"],
        heads, q_rows, kv_rows)
    assert q_heads == heads
    for i, h in enumerate(heads):
        check_grad(f"causal-64k dq h{h}", to_np(b["dq"][q_rows][:, h]),
                   rdq[:, i])
        check_grad(f"causal-64k dk h{h}", to_np(b["dk"][kv_rows][:, h]),
                   rdk[:, i])
        check_grad(f"causal-64k dv h{h}", to_np(b["dv"][kv_rows][:, h]),
                   rdv[:, i])


def test_queued_items_ragged_tail_backward(gpu):
    """Both backward kernels on the work-queue path with ragged tails and
    the plain item order (queued_tail_config: 8274 dQ items, 197 x 2 Q
    blocks of 128 rows x 21 query heads on 7 KV heads).  dQ, dK and dV start
    as NaN, so an item no workgroup took would show; dQ on sampled rows and
    dK, dV on sampled KV rows of every head against the oracle."""
    cfg = dataclasses.replace(queued_tail_config(), grad_seed=64)
    assert cfg.nq * (cfg.partition_len // 128) * cfg.num_q_heads >= 4096
    prob, (q, k, v, do), (qd, kd, vd, dod), o, lse = _setup(cfg, gpu)
    P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads, cfg.num_kv_heads,
                     cfg.head_dim)
    nan = float("nan")
    init = (torch.full((cfg.nq * P, hq, d), nan, device=gpu),
            torch.full((cfg.nkv * P, hkv, d), nan, device=gpu),
            torch.full((cfg.nkv * P, hkv, d), nan, device=gpu))
    log(f"{cfg.name}: GPU backward")
    dq, dk, dv = _run_bwd(prob, cfg, qd, kd, vd, o, dod, lse, init=init)
    torch.cuda.synchronize()
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        assert not torch.isnan(t).any(), f"{name} has unwritten items"
    q_rows = sample_rows(cfg, cfg.nq, n_random=2)
    kv_rows = sample_rows(cfg, cfg.nkv, seed_offset=2000, n_random=4)
    heads = list(range(hkv))
    log(f"{cfg.name}: oracle on {len(q_rows)} dQ rows, {len(kv_rows)} dK/dV "
        f"rows, every head")
    rdq, rdk, rdv, q_heads = oracle_backward_rows(
        prob, cfg.q_idx, cfg.kv_idx, q, k, v, do, heads, q_rows, kv_rows)
    dqc, dkc, dvc = dq.cpu(), dk.cpu(), dv.cpu()
    for i, h in enumerate(q_heads):
        check_grad(f"queued-tail dq h{h}", to_np(dqc[q_rows][:, h]), rdq[:, i])
    for i, hk in enumerate(heads):
        check_grad(f"queued-tail dk h{hk}", to_np(dkc[kv_rows][:, hk]),
                   rdk[:, i])
        check_grad(f"queued-tail dv h{hk}", to_np(dvc[kv_rows][:, hk]),
                   rdv[:, i])


def test_causal64k_head_dim64_backward_sampled(gpu):
    """The head_dim 64 backward kernels on the full-size causal 64K tile:
    dQ on the sampled Q rows and dK, dV on the sampled KV rows of every head
    against the float64 oracle."""
    cfg = dataclasses.replace(WORKLOADS["bwd-causal-64k"], head_dim=64,
                              name="bwd-causal-64k-d64")
    b = _gpu_backward_cpu(cfg, gpu)
    heads = list(range(cfg.num_q_heads))
    q_rows = sample_rows(cfg, cfg.nq)
    kv_rows = sample_rows(cfg, cfg.nkv, seed_offset=2000)
    log(f"causal-64k d64 backward: oracle on all {len(heads)} heads")
    rdq, rdk, rdv, q_heads = oracle_backward_rows(
        b["prob"], cfg.q_idx, cfg.kv_idx, b["q"], b["k"], b["v"], b["do"],
        heads, q_rows, kv_rows)
    assert q_heads == heads
    for i, h in enumerate(heads):
        check_grad(f"causal-64k d64 dq h{h}", to_np(b["dq"][q_rows][:, h]),
                   rdq[:, i])
        check_grad(f"causal-64k d64 dk h{h}", to_np(b["dk"][kv_rows][:, h]),
                   rdk[:, i])
        check_grad(f"causal-64k d64 dv h{h}", to_np(b["dv"][kv_rows][:, h]),
                   rdv[:, i])


def test_mesh1m_gqa_backward_identities_and_dq(bwd1m):
    """Backward at the 1M-token non-causal GQA tile's full size (65536 rows,
    32 query heads on 8 KV heads).  On every KV head, the identities that
    hold because each row's softmax runs over exactly the tile's keys: sum_j
    dK_j = 0 and sum_j dV_j = sum of dO over the rows and the query heads of
    the group.  dQ of sampled rows of two query heads (in different KV
    groups) against the float64 definition on those rows."""
    from oracle.attention import (attention_rows, attention_rows_bwd,
                                  problem_positions)
    cfg = dataclasses.replace(WORKLOADS["mesh1m-nc-gqa"], grad_seed=8)
    b = bwd1m
    prob = b["prob"]
    q, k, v, do, dq, dk, dv = (b[x] for x in
                               ("q", "k", "v", "do", "dq", "dk", "dv"))
    g = cfg.num_q_heads // cfg.num_kv_heads
    sdo = do.float().sum(0).view(cfg.num_kv_heads, g, -1).sum(1)
    rk = float((dk.sum(0).abs() / dk.abs().sum(0)).max())
    rv = float(((dv.sum(0) - sdo).abs() / dv.abs().sum(0)).max())
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
        check_grad(f"mesh1m-nc-gqa dq head {h} ({len(rows)} rows)",
                   to_np(dq[rows, h]), rdq)


@pytest.mark.parametrize("kv_head", [0, 7])
def test_mesh1m_gqa_backward_dkdv_sampled(bwd1m, kv_head):
    """dK and dV of one KV head at the 1M-token GQA tile's full size, element
    by element on sampled KV rows, summed over the group's four query heads,
    against the float64 oracle (whose forward covers all 65536 rows of each
    of those heads); dQ of those heads on sampled rows as well."""
    cfg = dataclasses.replace(WORKLOADS["mesh1m-nc-gqa"], grad_seed=8)
    b = bwd1m
    q_rows = sample_rows(cfg, cfg.nq, n_random=4)
    kv_rows = sample_rows(cfg, cfg.nkv, seed_offset=2000, n_random=16)
    log(f"mesh1m-nc-gqa backward: oracle on KV head {kv_head}, "
        f"{len(kv_rows)} dK/dV rows, {len(q_rows)} dQ rows")
    rdq, rdk, rdv, q_heads = oracle_backward_rows(
        b["prob"], cfg.q_idx, cfg.kv_idx, b["q"], b["k"], b["v"], b["do"],
        [kv_head], q_rows, kv_rows)
    check_grad(f"mesh1m-nc-gqa dk kv head {kv_head}",
               to_np(b["dk"][kv_rows][:, kv_head]), rdk[:, 0])
    check_grad(f"mesh1m-nc-gqa dv kv head {kv_head}",
               to_np(b["dv"][kv_rows][:, kv_head]), rdv[:, 0])
    for i, h in enumerate(q_heads):
        check_grad(f"mesh1m-nc-gqa dq head {h}", to_np(b["dq"][q_rows][:, h]),
                   rdq[:, i])

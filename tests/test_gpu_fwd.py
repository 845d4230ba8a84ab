"""GPU parity of mesh_attn_tile_fwd and mesh_attn_lse_merge against the
float64 oracle, through the C ABI, on the same seeded inputs."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2512_20968_amd as ma
from mesh_inputs import WORKLOADS, make_merge_parts, make_qkv, sample_rows

from helpers import (check_fwd, log, oracle_forward_rows, queued_tail_config,
                     run_fwd, to_np)

pytestmark = pytest.mark.gpu


def _inputs(cfg, dev):
    q, k, v, extra = make_qkv(cfg)
    return (q, k, v), tuple(t.to(dev) for t in (q, k, v)), extra


def _problem(cfg, **kw):
    p = cfg.problem()
    p.update(kw)
    return p


@pytest.mark.parametrize("causal", [0, 1])
def test_tiny_tile_fused_and_split_merge(gpu, causal):
    """Tiny tile {0,1} x {0,1}: every row checked, by the fused call and by one
    call per KV partition (float32 partials) folded by the merge kernel."""
    cfg = WORKLOADS["tiny-nc"]
    prob = _problem(cfg, causal=causal)
    (q, k, v), (qd, kd, vd), _ = _inputs(cfg, gpu)
    P = cfg.partition_len
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    ro, rl = oracle.tile_forward(prob, cfg.q_idx, cfg.kv_idx, to_np(q),
                                 to_np(k), to_np(v))
    check_fwd(f"cfg1 causal={causal} fused", to_np(o), to_np(lse), ro, rl)
    parts = [run_fwd(prob, cfg.q_idx, [cfg.kv_idx[b]],
                     qd, kd[b * P:(b + 1) * P].contiguous(),
                     vd[b * P:(b + 1) * P].contiguous(), torch.float32)
             for b in range(cfg.nkv)]
    po = torch.stack([p[0] for p in parts])
    pl = torch.stack([p[1] for p in parts])
    mo = torch.empty_like(o)
    ml = torch.empty_like(lse)
    ma.mesh_attn_lse_merge(po, pl, mo, ml)
    torch.cuda.synchronize()
    check_fwd(f"cfg1 causal={causal} split+merge", to_np(mo), to_np(ml), ro, rl)
    # Each float32 partial is itself a tile result over one KV partition.
    for b in range(cfg.nkv):
        rpo, rpl = oracle.tile_forward(prob, cfg.q_idx, [cfg.kv_idx[b]],
                                       to_np(q), to_np(k[b * P:(b + 1) * P]),
                                       to_np(v[b * P:(b + 1) * P]))
        check_fwd(f"cfg1 causal={causal} partial {b}", to_np(po[b]),
                  to_np(pl[b]), rpo, rpl)


def test_tiny_tile_convex_combination(gpu):
    """Every output row is a convex combination of V rows: per channel it lies
    within [min_j v_j, max_j v_j] over the visible keys (up to bf16 rounding of
    the output)."""
    cfg = WORKLOADS["tiny-nc"]
    prob = _problem(cfg, causal=1)
    (q, k, v), (qd, kd, vd), _ = _inputs(cfg, gpu)
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, torch.float32)
    torch.cuda.synchronize()
    og = to_np(o)
    vn = to_np(v)
    P = cfg.partition_len
    qpos = oracle.token_positions(cfg.q_idx, P)
    kpos = oracle.token_positions(cfg.kv_idx, P)
    for h in range(cfg.num_q_heads):
        for i in range(0, og.shape[0], 7):
            vis = kpos <= qpos[i]
            lo = vn[vis, h].min(axis=0)
            hi = vn[vis, h].max(axis=0)
            assert np.all(og[i, h] >= lo - 1e-5) and np.all(og[i, h] <= hi + 1e-5)


def _sampled_parity(cfg, gpu, rows_extra=None, heads=None):
    (q, k, v), (qd, kd, vd), extra = _inputs(cfg, gpu)
    prob = cfg.problem()
    log(f"{cfg.name}: launching forward")
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    extra_local = extra.get("q_outlier_rows", ())
    rows = sample_rows(cfg, cfg.nq, extra_local=extra_local)
    heads = list(range(cfg.num_q_heads)) if heads is None else heads
    log(f"{cfg.name}: oracle on {len(rows)} rows x {len(heads)} heads")
    ro, rl = oracle_forward_rows(prob, cfg.q_idx, cfg.kv_idx, q, k, v, rows,
                                 heads)
    og = o[torch.tensor(rows, device=gpu)][:, heads].float().cpu().numpy()
    lg = lse[heads][:, torch.tensor(rows, device=gpu)].cpu().numpy()
    check_fwd(f"{cfg.name} sampled", og, lg, ro, rl)
    return o, lse


def test_causal64k_sampled(gpu):
    _sampled_parity(WORKLOADS["causal-64k"], gpu)


def test_causal64k_head_dim64_sampled(gpu):
    """The head_dim 64 kernel (its own swizzles and load shapes) on the
    full-size causal 64K tile, sampled rows of every head."""
    _sampled_parity(dataclasses.replace(WORKLOADS["causal-64k"], head_dim=64,
                                        name="causal-64k-d64"), gpu)


def test_mesh1m_nc_gqa_sampled(gpu):
    _sampled_parity(WORKLOADS["mesh1m-nc-gqa"], gpu)


def test_queued_items_ragged_tail_plain_order(gpu):
    """The work-queue path with a ragged tail (queued_tail_config): O and LSE
    start as NaN, so an item that no workgroup took would stay NaN; sampled
    rows of every head against the oracle."""
    cfg = queued_tail_config()
    assert cfg.nq * cfg.num_q_heads >= 4096
    assert (cfg.nq * cfg.num_q_heads) % 8 != 0 and cfg.num_kv_heads % 8 != 0
    (q, k, v), (qd, kd, vd), _ = _inputs(cfg, gpu)
    prob = cfg.problem()
    P, hq, d = cfg.partition_len, cfg.num_q_heads, cfg.head_dim
    o = torch.full((cfg.nq * P, hq, d), float("nan"), dtype=torch.bfloat16,
                   device=gpu)
    lse = torch.full((hq, cfg.nq * P), float("nan"), dtype=torch.float32,
                     device=gpu)
    log(f"{cfg.name}: launching forward ({cfg.nq * hq} items)")
    ma.mesh_attn_tile_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o, lse)
    torch.cuda.synchronize()
    assert not torch.isnan(o).any() and not torch.isnan(lse).any()
    rows = sample_rows(cfg, cfg.nq, n_random=2)
    heads = list(range(hq))
    ro, rl = oracle_forward_rows(prob, cfg.q_idx, cfg.kv_idx, q, k, v, rows,
                                 heads)
    idx = torch.tensor(rows, device=gpu)
    check_fwd(f"{cfg.name} sampled", o[idx].float().cpu().numpy(),
              lse[:, idx].cpu().numpy(), ro, rl)


def test_mesh1m_causal_outlier_sampled(gpu):
    _sampled_parity(WORKLOADS["mesh1m-causal-outlier"], gpu)


def test_tile_above_diagonal_has_no_visible_key(gpu):
    """Causal tile whose KV partitions all lie after its Q partitions: every
    row sees nothing, O = 0 and LSE = -inf.  A mixed tile keeps both kinds."""
    cfg = dataclasses.replace(WORKLOADS["tiny-nc"], q_idx=[0, 1], kv_idx=[2, 3], seed=5)
    (q, k, v), (qd, kd, vd), _ = _inputs(cfg, gpu)
    prob = _problem(cfg, causal=1)
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    assert torch.all(o == 0) and torch.all(torch.isneginf(lse))
    cfg2 = dataclasses.replace(WORKLOADS["tiny-nc"], q_idx=[0, 3], kv_idx=[2, 1], seed=6)
    (q, k, v), (qd, kd, vd), _ = _inputs(cfg2, gpu)
    o, lse = run_fwd(prob, cfg2.q_idx, cfg2.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    ro, rl = oracle.tile_forward(prob, cfg2.q_idx, cfg2.kv_idx, to_np(q),
                                 to_np(k), to_np(v))
    assert np.isneginf(rl).any() and np.isfinite(rl).any()
    check_fwd("mixed empty rows", to_np(o), to_np(lse), ro, rl)


@pytest.mark.parametrize("d,hq,hkv", [(128, 8, 2), (64, 6, 3), (128, 4, 4)])
def test_kvr_strided_list_gqa_causal(gpu, d, hq, hkv):
    """Strided, non-contiguous KV footprint as KV Partition Rotation produces
    (c + t*a), several Q partitions spanning the diagonal, GQA, both head dims;
    every row checked."""
    cfg = dataclasses.replace(WORKLOADS["tiny-nc"], num_partitions=9, partition_len=256,
                              q_idx=[3, 4, 5], kv_idx=[1, 4, 7],
                              num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                              causal=True, seed=9)
    (q, k, v), (qd, kd, vd), _ = _inputs(cfg, gpu)
    prob = cfg.problem()
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    ro, rl = oracle.tile_forward(prob, cfg.q_idx, cfg.kv_idx, to_np(q),
                                 to_np(k), to_np(v))
    check_fwd(f"kvr d={d} hq={hq} hkv={hkv}", to_np(o), to_np(lse), ro, rl)


def test_forward_is_deterministic(gpu):
    cfg = dataclasses.replace(WORKLOADS["causal-64k"], q_idx=[6, 7], kv_idx=[0, 5, 6, 7],
                              partition_len=1024, num_q_heads=8,
                              num_kv_heads=8)
    (q, k, v), (qd, kd, vd), _ = _inputs(cfg, gpu)
    prob = cfg.problem()
    o1, l1 = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    o2, l2 = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.parametrize("d,hq,hkv", [(64, 8, 2), (128, 4, 1)])
def test_multi_block_partitions_every_row(gpu, d, hq, hkv):
    """1024-token partitions (four 256-row Q blocks and sixteen 64-key blocks
    per partition, so diagonal pairs mix FULL, PARTIAL and EMPTY blocks),
    causal GQA, permuted lists, both head dims: every row checked."""
    cfg = dataclasses.replace(WORKLOADS["tiny-nc"], num_partitions=3,
                              partition_len=1024, q_idx=[2, 1],
                              kv_idx=[0, 2, 1], num_q_heads=hq,
                              num_kv_heads=hkv, head_dim=d, causal=True,
                              seed=43)
    (q, k, v), (qd, kd, vd), _ = _inputs(cfg, gpu)
    prob = cfg.problem()
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    ro, rl = oracle.tile_forward(prob, cfg.q_idx, cfg.kv_idx, to_np(q),
                                 to_np(k), to_np(v))
    check_fwd(f"P=1024 causal GQA d={d} hq={hq} hkv={hkv}", to_np(o),
              to_np(lse), ro, rl)


@pytest.mark.parametrize("kparts,rows,heads,d,in_dt,out_dt,ninf", [
    (1, 37, 3, 64, torch.float32, torch.float32, 0.0),
    (2, 1000, 4, 64, torch.float32, torch.bfloat16, 0.1),
    (5, 777, 2, 128, torch.bfloat16, torch.bfloat16, 0.3),
    (16, 4096, 4, 128, torch.bfloat16, torch.float32, 0.0),
    (9, 333, 1, 8, torch.float32, torch.float32, 0.5),
    # more partials than one load batch (16 bf16 / 8 float32 per batch): the
    # running reducer across batches and a ragged last batch
    (17, 200, 2, 128, torch.bfloat16, torch.bfloat16, 0.2),
    (33, 100, 2, 64, torch.float32, torch.float32, 0.3),
])
def test_merge_parity(gpu, kparts, rows, heads, d, in_dt, out_dt, ninf):
    o, lse = make_merge_parts(kparts, rows, heads, d, seed=kparts + rows,
                              dtype=in_dt, neg_inf_frac=ninf)
    if ninf > 0:
        lse[:, 0, :3] = float("-inf")   # rows with every part empty
    od, ld = o.to(gpu), lse.to(gpu)
    mo = torch.empty((rows, heads, d), dtype=out_dt, device=gpu)
    ml = torch.empty((heads, rows), dtype=torch.float32, device=gpu)
    ma.mesh_attn_lse_merge(od, ld, mo, ml)
    torch.cuda.synchronize()
    on = o.float().numpy()
    ln = lse.numpy()
    for h in range(heads):
        ro, rl = oracle.lse_merge(on[:, :, h], ln[:, h])
        og = to_np(mo[:, h])
        if out_dt == torch.bfloat16:
            # A bf16 output is compared with the oracle's result rounded to
            # bf16 (round to nearest even), at the plain bar.
            ro = to_np(torch.from_numpy(ro).to(torch.bfloat16))
        check_fwd(f"merge k={kparts} h={h}", og[:, None],
                  to_np(ml[h])[None], ro[:, None], rl[None])


def test_merge_zero_rows_is_noop(gpu):
    o = torch.empty((3, 0, 2, 64), dtype=torch.bfloat16, device=gpu)
    lse = torch.empty((3, 2, 0), dtype=torch.float32, device=gpu)
    mo = torch.empty((0, 2, 64), dtype=torch.bfloat16, device=gpu)
    ml = torch.empty((2, 0), dtype=torch.float32, device=gpu)
    ma.mesh_attn_lse_merge(o, lse, mo, ml)
    torch.cuda.synchronize()

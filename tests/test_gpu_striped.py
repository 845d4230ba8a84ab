"""GPU parity under the striped sequence layout (Section 3.7: token r of
partition p at position r*n + p), forward and backward, against the float64
oracle through the C ABI.  Under this layout every partition pair is
near-triangular, so every Q block has PARTIAL runs whose mask offset depends
on the order of the two partitions."""

import dataclasses

import pytest
import torch

import oracle
import paper_2512_20968_amd as ma
from mesh_inputs import WORKLOADS, make_grad, make_qkv, sample_rows

from helpers import (check_fwd, check_grad, log, oracle_backward_rows,
                     oracle_forward_rows, run_fwd, to_np)

pytestmark = pytest.mark.gpu


def _cfg(**kw):
    base = dict(num_partitions=4, partition_len=256, q_idx=[2, 0, 3, 1],
                kv_idx=[1, 3, 0, 2], num_q_heads=4, num_kv_heads=2,
                head_dim=64, causal=True, seed=41, grad_seed=42, layout=1)
    base.update(kw)
    return dataclasses.replace(WORKLOADS["tiny-nc"], **base)


def _inputs(cfg, dev):
    q, k, v, _ = make_qkv(cfg)
    return (q, k, v), tuple(t.to(dev) for t in (q, k, v))


@pytest.mark.parametrize("d,hq,hkv", [(64, 4, 2), (128, 4, 4)])
def test_striped_whole_sequence_tile_every_row(gpu, d, hq, hkv):
    """Q and KV lists name every partition (permuted): causal attention of
    the whole sequence.  Fused call, then one float32 partial per KV
    partition folded by the merge kernel."""
    cfg = _cfg(head_dim=d, num_q_heads=hq, num_kv_heads=hkv)
    prob = cfg.problem()
    (q, k, v), (qd, kd, vd) = _inputs(cfg, gpu)
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    ro, rl = oracle.tile_forward(prob, cfg.q_idx, cfg.kv_idx, to_np(q),
                                 to_np(k), to_np(v))
    check_fwd(f"striped whole d={d}", to_np(o), to_np(lse), ro, rl)
    P = cfg.partition_len
    parts = [run_fwd(prob, cfg.q_idx, [cfg.kv_idx[b]], qd,
                     kd[b * P:(b + 1) * P].contiguous(),
                     vd[b * P:(b + 1) * P].contiguous(), torch.float32)
             for b in range(cfg.nkv)]
    mo, ml = torch.empty_like(o), torch.empty_like(lse)
    ma.mesh_attn_lse_merge(torch.stack([p[0] for p in parts]),
                           torch.stack([p[1] for p in parts]), mo, ml)
    torch.cuda.synchronize()
    check_fwd(f"striped whole d={d} split+merge", to_np(mo), to_np(ml), ro, rl)


@pytest.mark.parametrize("q_idx,kv_idx", [([1, 6], [0, 3, 7]),
                                          ([7], [6, 7]),
                                          ([0], [5, 2])])
def test_striped_mesh_tiles_every_row(gpu, q_idx, kv_idx):
    """Tiles of a larger mesh with KV partitions before, equal to and after
    the Q partitions (mask offset 0 or -1 on the diagonal of each pair)."""
    cfg = _cfg(num_partitions=8, partition_len=512, q_idx=q_idx,
               kv_idx=kv_idx, head_dim=128, num_q_heads=2, num_kv_heads=1)
    prob = cfg.problem()
    (q, k, v), (qd, kd, vd) = _inputs(cfg, gpu)
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    ro, rl = oracle.tile_forward(prob, cfg.q_idx, cfg.kv_idx, to_np(q),
                                 to_np(k), to_np(v))
    check_fwd(f"striped tile {q_idx}x{kv_idx}", to_np(o), to_np(lse), ro, rl)


@pytest.mark.parametrize("name", ["striped-causal-64k", "striped-mesh1m-causal"])
def test_striped_workloads_sampled(gpu, name):
    cfg = WORKLOADS[name]
    prob = cfg.problem()
    (q, k, v), (qd, kd, vd) = _inputs(cfg, gpu)
    log(f"{cfg.name}: launching forward")
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    torch.cuda.synchronize()
    rows = sample_rows(cfg, cfg.nq)
    heads = list(range(cfg.num_q_heads))
    log(f"{cfg.name}: oracle on {len(rows)} rows x {len(heads)} heads")
    ro, rl = oracle_forward_rows(prob, cfg.q_idx, cfg.kv_idx, q, k, v, rows,
                                 heads)
    r = torch.tensor(rows, device=gpu)
    check_fwd(f"{cfg.name} sampled", to_np(o[r][:, heads]),
              to_np(lse[heads][:, r]), ro, rl)


def _bwd(prob, cfg, qd, kd, vd, o, dod, lse):
    P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads, cfg.num_kv_heads,
                     cfg.head_dim)
    dq = torch.empty((cfg.nq * P, hq, d), dtype=torch.float32, device=qd.device)
    dk = torch.empty((cfg.nkv * P, hkv, d), dtype=torch.float32,
                     device=qd.device)
    dv = torch.empty_like(dk)
    ma.mesh_attn_tile_bwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o, dod, lse,
                          dq, dk, dv)
    return dq, dk, dv


@pytest.mark.parametrize("q_idx,kv_idx,d,hq,hkv", [
    ([2, 0, 3, 1], [1, 3, 0, 2], 64, 4, 2),
    ([1, 3], [3, 0, 2], 128, 2, 2),
])
def test_striped_backward_every_row(gpu, q_idx, kv_idx, d, hq, hkv):
    cfg = _cfg(q_idx=q_idx, kv_idx=kv_idx, head_dim=d, num_q_heads=hq,
               num_kv_heads=hkv)
    prob = cfg.problem()
    (q, k, v), (qd, kd, vd) = _inputs(cfg, gpu)
    do = make_grad(cfg)
    dod = do.to(gpu)
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    dq, dk, dv = _bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    torch.cuda.synchronize()
    rdq, rdk, rdv, _, _ = oracle.tile_backward(
        prob, cfg.q_idx, cfg.kv_idx, to_np(q), to_np(k), to_np(v), to_np(do))
    tag = f"striped bwd {q_idx}x{kv_idx} d={d}"
    check_grad(f"{tag} dq", to_np(dq), rdq)
    check_grad(f"{tag} dk", to_np(dk), rdk)
    check_grad(f"{tag} dv", to_np(dv), rdv)


def test_striped_causal64k_backward_sampled(gpu):
    """Full-size backward of the striped 64K tile against the float64
    oracle on every head: dQ on sampled Q rows, dK and dV on sampled KV rows
    (the oracle's forward covers every row of each head)."""
    cfg = WORKLOADS["striped-causal-64k"]
    prob = cfg.problem()
    (q, k, v), (qd, kd, vd) = _inputs(cfg, gpu)
    do = make_grad(cfg)
    dod = do.to(gpu)
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    log("striped-causal-64k: GPU backward")
    dq, dk, dv = _bwd(prob, cfg, qd, kd, vd, o, dod, lse)
    torch.cuda.synchronize()
    heads = list(range(cfg.num_q_heads))
    q_rows = sample_rows(cfg, cfg.nq, n_random=16)
    kv_rows = sample_rows(cfg, cfg.nkv, seed_offset=2000, n_random=16)
    log(f"striped-causal-64k: oracle on {len(heads)} heads, {len(q_rows)} dQ "
        f"rows, {len(kv_rows)} dK/dV rows")
    rdq, rdk, rdv, q_heads = oracle_backward_rows(
        prob, cfg.q_idx, cfg.kv_idx, q, k, v, do, heads, q_rows, kv_rows)
    qr = torch.tensor(q_rows, device=gpu)
    kr = torch.tensor(kv_rows, device=gpu)
    check_grad("striped-causal-64k dq", to_np(dq[qr][:, q_heads]), rdq)
    check_grad("striped-causal-64k dk", to_np(dk[kr][:, heads]), rdk)
    check_grad("striped-causal-64k dv", to_np(dv[kr][:, heads]), rdv)

"""Forty-eight seeded random tiles, forward and backward, every row and head
against the float64 oracle: partition counts and lengths (256 to 2048),
Q and KV index lists (subsets in any order, overlapping or not), GQA ratios,
both head dims, causal or not, both layouts, with and without the x8
outlier rows.  Each case is small enough for the oracle to take every row;
together they cover shapes the named workloads do not."""

import random

import pytest
import torch

import oracle
import paper_2512_20968_amd as ma
from mesh_inputs import TileConfig, make_grad, make_qkv

from helpers import check_fwd, check_grad, log, run_fwd, to_np

pytestmark = pytest.mark.gpu

HEADS = [(4, 4), (6, 3), (8, 2), (2, 1), (4, 1)]


def _random_case(i):
    r = random.Random(7000 + i)
    n = r.randint(3, 10)
    P = r.choice([256, 512, 1024, 2048])
    nq = r.randint(1, min(3 if P < 2048 else 2, n))
    nkv = r.randint(1, min(4 if P < 2048 else 2, n))
    q_idx = r.sample(range(n), nq)
    kv_idx = r.sample(range(n), nkv)
    hq, hkv = r.choice(HEADS)
    return TileConfig(f"random-{i}", n, P, q_idx, kv_idx, hq, hkv,
                      r.choice([64, 128]), r.random() < 0.7, seed=7100 + i,
                      outliers=r.random() < 0.3, grad_seed=7200 + i,
                      layout=int(r.random() < 0.4))


CASES = [_random_case(i) for i in range(48)]


@pytest.mark.parametrize("cfg", CASES, ids=[c.name for c in CASES])
def test_random_tile_forward_and_backward(gpu, cfg):
    q, k, v, _ = make_qkv(cfg)
    do = make_grad(cfg)
    qd, kd, vd, dod = (t.to(gpu) for t in (q, k, v, do))
    prob = cfg.problem()
    log(f"{cfg.name}: n={cfg.num_partitions} P={cfg.partition_len} "
        f"q={cfg.q_idx} kv={cfg.kv_idx} heads={cfg.num_q_heads}/"
        f"{cfg.num_kv_heads} d={cfg.head_dim} causal={int(cfg.causal)} "
        f"layout={cfg.layout} outliers={int(cfg.outliers)}")
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    o32, lse32 = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd,
                         torch.float32)
    P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads, cfg.num_kv_heads,
                     cfg.head_dim)
    dq = torch.empty((cfg.nq * P, hq, d), dtype=torch.float32, device=gpu)
    dk = torch.empty((cfg.nkv * P, hkv, d), dtype=torch.float32, device=gpu)
    dv = torch.empty_like(dk)
    ma.mesh_attn_tile_bwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o, dod, lse,
                          dq, dk, dv)
    torch.cuda.synchronize()
    qn, kn, vn, don = (to_np(t) for t in (q, k, v, do))
    ro, rl = oracle.tile_forward(prob, cfg.q_idx, cfg.kv_idx, qn, kn, vn)
    check_fwd(f"{cfg.name} bf16 out", to_np(o), to_np(lse), ro, rl)
    check_fwd(f"{cfg.name} f32 out", to_np(o32), to_np(lse32), ro, rl)
    rdq, rdk, rdv, q_heads, _ = oracle.tile_backward(prob, cfg.q_idx, cfg.kv_idx,
                                                     qn, kn, vn, don)
    assert list(q_heads) == list(range(hq))
    check_grad(f"{cfg.name} dq", to_np(dq), rdq)
    check_grad(f"{cfg.name} dk", to_np(dk), rdk)
    check_grad(f"{cfg.name} dv", to_np(dv), rdv)

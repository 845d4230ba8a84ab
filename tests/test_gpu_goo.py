"""GPU parity of the GOO compute tasks (Section 3.4) through the C ABI: each
chunk call C-i-j against the oracle's chunk task, and the running
accumulation of C-i-0 .. C-i-(k_KV-1) against the oracle's (and the fused
kernel's) whole tile on the rows of Q chunk i, in the planner's order."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2512_20968_amd as ma
from mesh_inputs import WORKLOADS, make_qkv, sample_rows
from oracle import goo

from helpers import check_fwd, check_grad, log, run_fwd, to_np

pytestmark = pytest.mark.gpu


def _rows(P, n_parts, k, i, dev=None):
    r = goo.chunk_buffer_rows(P, n_parts, k, i)
    return torch.tensor(r, device=dev) if dev is not None else r


def _run_chunks(cfg, qd, kd, vd, kq, kkv, order):
    """Run every C-i-j in ``order`` (a list of (i, j)); the first task of each
    Q chunk writes, the others accumulate.  Returns {i: (o, lse)}."""
    P, hq, d = cfg.partition_len, cfg.num_q_heads, cfg.head_dim
    prob = cfg.problem()
    out = {}
    qbuf = {i: qd[_rows(P, cfg.nq, kq, i, qd.device)].contiguous()
            for i in range(kq)}
    kbuf = {j: (kd[_rows(P, cfg.nkv, kkv, j, qd.device)].contiguous(),
                vd[_rows(P, cfg.nkv, kkv, j, qd.device)].contiguous())
            for j in range(kkv)}
    for i, j in order:
        first = i not in out
        if first:
            rq = cfg.nq * P // kq
            out[i] = (torch.empty((rq, hq, d), dtype=torch.float32,
                                  device=qd.device),
                      torch.empty((hq, rq), dtype=torch.float32,
                                  device=qd.device))
        ma.mesh_attn_chunk_fwd(prob, cfg.q_idx, cfg.kv_idx, (i, kq, j, kkv),
                               qbuf[i], kbuf[j][0], kbuf[j][1], out[i][0],
                               out[i][1], accumulate=0 if first else 1)
    return out


def _small(layout, **kw):
    base = dict(num_partitions=4, partition_len=1024, q_idx=[2, 3],
                kv_idx=[0, 1, 2, 3], num_q_heads=4, num_kv_heads=2,
                head_dim=128, causal=True, seed=51, layout=layout)
    base.update(kw)
    return dataclasses.replace(WORKLOADS["tiny-nc"], **base)


@pytest.mark.parametrize("layout", [0, 1])
def test_single_chunk_task_matches_oracle(gpu, layout):
    cfg = _small(layout)
    q, k, v, _ = make_qkv(cfg)
    P = cfg.partition_len
    kq, kkv, i, j = 2, 4, 1, 2
    qr, kr = _rows(P, cfg.nq, kq, i), _rows(P, cfg.nkv, kkv, j)
    qd, kd, vd = (t.to(gpu) for t in (q[qr], k[kr], v[kr]))
    o = torch.empty((len(qr), cfg.num_q_heads, cfg.head_dim),
                    dtype=torch.float32, device=gpu)
    lse = torch.empty((cfg.num_q_heads, len(qr)), dtype=torch.float32,
                      device=gpu)
    ma.mesh_attn_chunk_fwd(cfg.problem(), cfg.q_idx, cfg.kv_idx,
                           (i, kq, j, kkv), qd, kd, vd, o, lse)
    torch.cuda.synchronize()
    ro, rl = goo.chunk_forward(cfg.problem(), cfg.q_idx, cfg.kv_idx, kq, i,
                               kkv, j, to_np(q[qr]), to_np(k[kr]),
                               to_np(v[kr]))
    check_fwd(f"C-{i}-{j} layout={layout}", to_np(o), to_np(lse), ro, rl)


@pytest.mark.parametrize("layout,kq,kkv", [(0, 2, 4), (1, 4, 2), (0, 1, 16),
                                           (1, 4, 4)])
def test_accumulated_chunks_equal_the_tile(gpu, layout, kq, kkv):
    """All chunk tasks, in the GOO planner's order, accumulate to the tile:
    every row against the oracle, and against the fused kernel."""
    cfg = _small(layout)
    q, k, v, _ = make_qkv(cfg)
    qd, kd, vd = (t.to(gpu) for t in (q, k, v))
    steps = ma.mesh_attn_goo_plan(kq, kkv, 0.5, 1.0, 0.5,
                                  np.full((kq, kkv), 0.5), 1.05)
    order = [t for _, tasks in steps for t in tasks]
    assert sorted(order) == [(i, j) for i in range(kq) for j in range(kkv)]
    out = _run_chunks(cfg, qd, kd, vd, kq, kkv, order)
    fo, fl = run_fwd(cfg.problem(), cfg.q_idx, cfg.kv_idx, qd, kd, vd,
                     torch.float32)
    torch.cuda.synchronize()
    ro, rl = oracle.tile_forward(cfg.problem(), cfg.q_idx, cfg.kv_idx,
                                 to_np(q), to_np(k), to_np(v))
    P = cfg.partition_len
    for i in range(kq):
        r = _rows(P, cfg.nq, kq, i)
        tag = f"chunks {kq}x{kkv} layout={layout} Q chunk {i}"
        check_fwd(tag, to_np(out[i][0]), to_np(out[i][1]), ro[r], rl[:, r])
        # The fused kernel rounds P to bf16 against other running maxima, so
        # the two agree to the forward tolerance, not bit for bit.
        check_fwd(tag + " vs fused", to_np(out[i][0]), to_np(out[i][1]),
                  to_np(fo)[r], to_np(fl)[:, r])


def test_causal64k_in_4x4_chunk_tasks(gpu):
    """The causal 64K tile as 16 chunk tasks: sampled rows against the
    oracle, all rows against the fused kernel."""
    cfg = WORKLOADS["causal-64k"]
    kq = kkv = 4
    q, k, v, _ = make_qkv(cfg)
    qd, kd, vd = (t.to(gpu) for t in (q, k, v))
    order = [(i, j) for i in range(kq) for j in range(kkv)]
    log("causal-64k: 16 chunk tasks")
    out = _run_chunks(cfg, qd, kd, vd, kq, kkv, order)
    fo, fl = run_fwd(cfg.problem(), cfg.q_idx, cfg.kv_idx, qd, kd, vd,
                     torch.float32)
    torch.cuda.synchronize()
    P = cfg.partition_len
    o_all = torch.empty_like(fo)
    l_all = torch.empty_like(fl)
    for i in range(kq):
        r = _rows(P, cfg.nq, kq, i, gpu)
        o_all[r] = out[i][0]
        l_all[:, r] = out[i][1]
    check_fwd("causal-64k as 4x4 chunks vs fused (all rows)", to_np(o_all),
              to_np(l_all), to_np(fo).astype(np.float64),
              to_np(fl).astype(np.float64))
    rows = sample_rows(cfg, cfg.nq, n_random=16)
    heads = [0, 9, 31]
    ro, rl = oracle.tile_forward(cfg.problem(), cfg.q_idx, cfg.kv_idx,
                                 to_np(q), to_np(k), to_np(v), rows=rows,
                                 heads=heads)
    rr = torch.tensor(rows, device=gpu)
    check_fwd("causal-64k as 4x4 chunks", to_np(o_all[rr][:, heads]),
              to_np(l_all[heads][:, rr]), ro, rl)


@pytest.mark.parametrize("layout,kq,kkv", [(0, 2, 2), (1, 1, 4), (1, 4, 1)])
def test_chunk_backward_sums_to_the_tile(gpu, layout, kq, kkv):
    """Every C-i-j backward, accumulated into zeroed gradients, against the
    oracle's tile gradients (every row), and one chunk task alone against the
    oracle's chunk backward."""
    from mesh_inputs import make_grad
    cfg = _small(layout, grad_seed=52)
    q, k, v, _ = make_qkv(cfg)
    do = make_grad(cfg)
    qd, kd, vd, dod = (t.to(gpu) for t in (q, k, v, do))
    prob = cfg.problem()
    P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads, cfg.num_kv_heads,
                     cfg.head_dim)
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    dq = torch.zeros((cfg.nq * P, hq, d), dtype=torch.float32, device=gpu)
    dk = torch.zeros((cfg.nkv * P, hkv, d), dtype=torch.float32, device=gpu)
    dv = torch.zeros_like(dk)
    single = None
    for i in range(kq):
        qr = _rows(P, cfg.nq, kq, i, gpu)
        qc, oc, doc = (t[qr].contiguous() for t in (qd, o, dod))
        lc = lse[:, qr].contiguous()
        for j in range(kkv):
            kr = _rows(P, cfg.nkv, kkv, j, gpu)
            kc, vc = kd[kr].contiguous(), vd[kr].contiguous()
            gq = torch.zeros((qc.shape[0], hq, d), dtype=torch.float32,
                             device=gpu)
            gk = torch.zeros((kc.shape[0], hkv, d), dtype=torch.float32,
                             device=gpu)
            gv = torch.zeros_like(gk)
            ma.mesh_attn_chunk_bwd(prob, cfg.q_idx, cfg.kv_idx,
                                   (i, kq, j, kkv), qc, kc, vc, oc, doc, lc,
                                   gq, gk, gv, accumulate=1)
            dq[qr] += gq
            dk[kr] += gk
            dv[kr] += gv
            if single is None:
                single = (i, j, gq, gk, gv)
    torch.cuda.synchronize()
    rdq, rdk, rdv, _, _ = oracle.tile_backward(
        prob, cfg.q_idx, cfg.kv_idx, to_np(q), to_np(k), to_np(v), to_np(do))
    tag = f"chunk bwd {kq}x{kkv} layout={layout}"
    check_grad(f"{tag} dq", to_np(dq), rdq)
    check_grad(f"{tag} dk", to_np(dk), rdk)
    check_grad(f"{tag} dv", to_np(dv), rdv)
    i, j, gq, gk, gv = single
    cq, ck, cv = goo.chunk_backward(prob, cfg.q_idx, cfg.kv_idx, kq, i, kkv, j,
                                    to_np(q), to_np(k), to_np(v), to_np(do))
    check_grad(f"{tag} C-{i}-{j} dq", to_np(gq), cq)
    check_grad(f"{tag} C-{i}-{j} dk", to_np(gk), ck)
    check_grad(f"{tag} C-{i}-{j} dv", to_np(gv), cv)


def test_causal64k_backward_as_2x2_chunk_tasks(gpu):
    """The full-size causal 64K backward as 2 x 2 chunk tasks accumulated into
    zeroed gradients: every row against the fused tile backward (itself
    checked against the oracle in test_gpu_bwd), within the summation-order
    tolerance of the gradients."""
    from mesh_inputs import make_grad
    cfg = WORKLOADS["bwd-causal-64k"]
    q, k, v, _ = make_qkv(cfg)
    do = make_grad(cfg)
    qd, kd, vd, dod = (t.to(gpu) for t in (q, k, v, do))
    prob = cfg.problem()
    P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads, cfg.num_kv_heads,
                     cfg.head_dim)
    o, lse = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd)
    fdq = torch.empty((cfg.nq * P, hq, d), dtype=torch.float32, device=gpu)
    fdk = torch.empty((cfg.nkv * P, hkv, d), dtype=torch.float32, device=gpu)
    fdv = torch.empty_like(fdk)
    ma.mesh_attn_tile_bwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o, dod,
                          lse, fdq, fdk, fdv)
    kq = kkv = 2
    dq = torch.zeros_like(fdq)
    dk = torch.zeros_like(fdk)
    dv = torch.zeros_like(fdk)
    log("causal-64k backward as 2x2 chunk tasks")
    for i in range(kq):
        qr = _rows(P, cfg.nq, kq, i, gpu)
        qc, oc, doc = (t[qr].contiguous() for t in (qd, o, dod))
        lc = lse[:, qr].contiguous()
        gq = torch.zeros((qc.shape[0], hq, d), dtype=torch.float32,
                         device=gpu)
        for j in range(kkv):
            kr = _rows(P, cfg.nkv, kkv, j, gpu)
            kc, vc = kd[kr].contiguous(), vd[kr].contiguous()
            gk = dk[kr].contiguous()
            gv = dv[kr].contiguous()
            # accumulate: dQ over the KV chunks, dK/dV over the Q chunks
            ma.mesh_attn_chunk_bwd(prob, cfg.q_idx, cfg.kv_idx,
                                   (i, kq, j, kkv), qc, kc, vc, oc, doc, lc,
                                   gq, gk, gv, accumulate=1)
            dk[kr] = gk
            dv[kr] = gv
        dq[qr] = gq
    torch.cuda.synchronize()
    for name, got, ref in (("dq", dq, fdq), ("dk", dk, fdk), ("dv", dv, fdv)):
        err = float((got - ref).abs().max())
        scale = float(ref.abs().max())
        log(f"causal-64k chunks vs fused {name}: max err {err:.3e}, "
            f"max |{name}| {scale:.3e}")
        # same products, different fp32 summation order across the chunks
        assert err <= 1e-3 * scale, name

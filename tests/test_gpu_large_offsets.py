"""Buffers past 2^31 elements: forward and backward of 130 Q partitions of
4096 rows x 32 query heads x 128 (Q, O, dO: 2.18e9 elements each, dQ 8.7 GB)
against one KV partition (8 KV heads), so every row, head and output offset
beyond the 2^31-th element has to be formed in 64 bits.

Q and dO are drawn on the device from a seeded generator (the host-side
generators would need ~30 GB of host memory); K and V on the host.  The
oracle gets host copies of the sampled rows only: rows at the start, on both
sides of the 2^31-element boundary and at the end, on every head.  dK and dV
are checked through the identities of a tile whose rows see exactly its
keys: sum_j dK_j = 0 and sum_j dV_j = sum of dO over the group's rows and
heads."""

import math

import numpy as np
import pytest
import torch

import paper_2512_20968_amd as ma
from oracle.attention import attention_rows, attention_rows_bwd

from helpers import check_fwd, check_grad, log, to_np

pytestmark = pytest.mark.gpu

P, NQ, HQ, HKV, D = 4096, 130, 32, 8, 128


@pytest.fixture(scope="module")
def big(gpu):
    rows = NQ * P
    assert rows * HQ * D > 2 ** 31
    prob = dict(num_partitions=NQ + 1, partition_len=P, num_q_heads=HQ,
                num_kv_heads=HKV, head_dim=D, causal=0, layout=0,
                softmax_scale=float(np.float32(1.0 / math.sqrt(D))))
    q_idx, kv_idx = list(range(NQ)), [NQ]
    g = torch.Generator(device=gpu).manual_seed(51)
    q = torch.randn((rows, HQ, D), generator=g, device=gpu,
                    dtype=torch.bfloat16)
    do = torch.randn((rows, HQ, D), generator=g, device=gpu,
                     dtype=torch.bfloat16)
    gc = torch.Generator().manual_seed(52)
    k = torch.randn((P, HKV, D), generator=gc).to(torch.bfloat16)
    v = torch.randn((P, HKV, D), generator=gc).to(torch.bfloat16)
    kd, vd = k.to(gpu), v.to(gpu)
    o = torch.empty((rows, HQ, D), dtype=torch.bfloat16, device=gpu)
    lse = torch.empty((HQ, rows), dtype=torch.float32, device=gpu)
    log(f"large offsets: forward of {rows} rows x {HQ} heads")
    ma.mesh_attn_tile_fwd(prob, q_idx, kv_idx, q, kd, vd, o, lse)
    dq = torch.empty((rows, HQ, D), dtype=torch.float32, device=gpu)
    dk = torch.empty((P, HKV, D), dtype=torch.float32, device=gpu)
    dv = torch.empty_like(dk)
    log("large offsets: backward")
    ma.mesh_attn_tile_bwd(prob, q_idx, kv_idx, q, kd, vd, o, do, lse, dq, dk,
                          dv)
    torch.cuda.synchronize()
    # First row whose Q/O elements start at or past 2^31.
    edge = 2 ** 31 // (HQ * D)
    sel = sorted({0, 1, P - 1, edge - 2, edge - 1, edge, edge + 1,
                  rows - 2, rows - 1,
                  *np.random.default_rng(53).integers(edge, rows, 24).tolist()})
    idx = torch.tensor(sel, device=gpu)
    out = dict(prob=prob, k=k, v=v, rows=sel,
               q=q[idx].cpu(), do=do[idx].cpu(), o=o[idx].cpu(),
               lse=lse[:, idx].cpu(), dq=dq[idx].cpu(), dk=dk.cpu(),
               dv=dv.cpu(),
               sum_do=do.float().sum(0).view(HKV, HQ // HKV, D).sum(1).cpu())
    del q, do, o, lse, dq, kd, vd
    torch.cuda.empty_cache()
    return out


def _oracle_rows(b):
    """Forward (O, LSE) and dQ of the sampled rows, every head, in float64."""
    n = len(b["rows"])
    kpos = np.arange(P, dtype=np.int64)
    qpos = np.zeros(n, dtype=np.int64)
    scale = b["prob"]["softmax_scale"]
    ro = np.zeros((n, HQ, D))
    rl = np.zeros((HQ, n))
    rdq = np.zeros((n, HQ, D))
    for h in range(HQ):
        hk = h // (HQ // HKV)
        qh = to_np(b["q"][:, h]).astype(np.float64)
        kh = to_np(b["k"][:, hk]).astype(np.float64)
        vh = to_np(b["v"][:, hk]).astype(np.float64)
        doh = to_np(b["do"][:, h]).astype(np.float64)
        o, lse = attention_rows(qh, kh, vh, qpos, kpos, False, scale)
        dlt = np.sum(doh * o, axis=1)
        dq, _, _ = attention_rows_bwd(qh, kh, vh, doh, lse, dlt, qpos, kpos,
                                      False, scale)
        ro[:, h], rl[h], rdq[:, h] = o, lse, dq
    return ro, rl, rdq


def test_forward_and_dq_past_int32_offsets(big):
    ro, rl, rdq = _oracle_rows(big)
    check_fwd(f"large offsets, {len(big['rows'])} rows x {HQ} heads",
              to_np(big["o"]), to_np(big["lse"]), ro, rl)
    check_grad("large offsets dq", to_np(big["dq"]), rdq)


def test_dkdv_identities_past_int32_offsets(big):
    dk, dv, sdo = big["dk"], big["dv"], big["sum_do"]
    rk = float((dk.sum(0).abs() / dk.abs().sum(0)).max())
    rv = float(((dv.sum(0) - sdo).abs() / dv.abs().sum(0)).max())
    log(f"large offsets: max |sum dK| / sum|dK| = {rk:.3e}, "
        f"max |sum dV - sum dO| / sum|dV| = {rv:.3e}")
    assert rk <= 1e-2 and rv <= 1e-2


def test_merge_past_int32_offsets(gpu):
    """LSE merge of 16 bf16 partials of 33000 rows x 32 heads x 128 (2.16e9
    elements): rows whose last-partial elements lie past 2^31 (and a few
    before) against the oracle's reducer, O compared with the oracle's result
    rounded to bf16."""
    from oracle.attention import lse_merge
    k, rows, h, d = 16, 33000, 32, 128
    assert k * rows * h * d > 2 ** 31
    g = torch.Generator(device=gpu).manual_seed(54)
    o_parts = torch.randn((k, rows, h, d), generator=g, device=gpu,
                          dtype=torch.bfloat16)
    lse_parts = (torch.randn((k, h, rows), generator=g, device=gpu) * 4
                 + 10).float()
    o = torch.empty((rows, h, d), dtype=torch.bfloat16, device=gpu)
    lse = torch.empty((h, rows), dtype=torch.float32, device=gpu)
    ma.mesh_attn_lse_merge(o_parts, lse_parts, o, lse)
    torch.cuda.synchronize()
    # First row of the last partial whose elements start past 2^31.
    edge = (2 ** 31 - (k - 1) * rows * h * d) // (h * d)
    sel = sorted({0, edge - 1, edge, edge + 1, rows - 1,
                  *np.random.default_rng(55).integers(edge, rows, 16).tolist()})
    idx = torch.tensor(sel, device=gpu)
    op = to_np(o_parts[:, idx]).astype(np.float64)     # [k, n, h, d]
    lp = to_np(lse_parts[:, :, idx]).astype(np.float64)  # [k, h, n]
    ro = np.zeros((len(sel), h, d))
    rl = np.zeros((h, len(sel)))
    for hh in range(h):
        ro[:, hh], rl[hh] = lse_merge(op[:, :, hh], lp[:, hh])
    ro_bf16 = to_np(torch.from_numpy(ro).to(torch.bfloat16))
    check_fwd(f"large-offset merge, {len(sel)} rows x {h} heads",
              to_np(o[idx]), to_np(lse[:, idx]), ro_bf16, rl)

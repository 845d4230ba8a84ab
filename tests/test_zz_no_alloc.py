"""The allocation-free forward (mesh_attn_tile_fwd_noalloc) against the
forward with a caller workspace (mesh_attn_tile_fwd), through the C ABI.

Both launch the same tile kernel; the allocation-free call builds the work
list on the device into the library's scratch array instead of uploading the
host-built list, so O and LSE must agree bit for bit.  Consecutive calls on a
GPU share the scratch array: the checks run two calls in a row, the second on
a smaller tile, and tiles of both workgroup-order paths (KV heads a multiple
of 8 or not), both layouts and both output dtypes."""

import ctypes
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2512_20968_amd as ma
from mesh_inputs import WORKLOADS, make_qkv

from helpers import check_fwd, log, queued_tail_config, run_fwd, to_np


def _noalloc(prob, cfg, qd, kd, vd, out_dtype):
    P, hq, d = cfg.partition_len, cfg.num_q_heads, cfg.head_dim
    o = torch.full((cfg.nq * P, hq, d), float("nan"), dtype=out_dtype,
                   device=qd.device)
    lse = torch.full((hq, cfg.nq * P), float("nan"), dtype=torch.float32,
                     device=qd.device)
    ma.mesh_attn_tile_fwd_noalloc(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o,
                                  lse)
    return o, lse


def _case(cfg, gpu, out_dtype, check_oracle=False):
    q, k, v, _ = make_qkv(cfg)
    qd, kd, vd = (t.to(gpu) for t in (q, k, v))
    prob = cfg.problem()
    o1, l1 = _noalloc(prob, cfg, qd, kd, vd, out_dtype)
    o2, l2 = run_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, out_dtype)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2), f"{cfg.name}: O differs"
    assert torch.equal(l1, l2), f"{cfg.name}: LSE differs"
    log(f"{cfg.name}: noalloc forward equals the workspace forward bit for "
        f"bit")
    if check_oracle:
        ro, rl = oracle.tile_forward(prob, cfg.q_idx, cfg.kv_idx, to_np(q),
                                     to_np(k), to_np(v))
        check_fwd(f"{cfg.name} noalloc", to_np(o1), to_np(l1), ro, rl)


@pytest.mark.gpu
def test_noalloc_matches_workspace_forward(gpu):
    # 1. The causal 64K tile (32 KV heads: KV-head-per-XCD order), bf16 out.
    _case(WORKLOADS["causal-64k"], gpu, torch.bfloat16)
    # 2. Right after, a smaller tile: 4 KV heads (round-robin order), causal,
    #    float32 partials, every row against the oracle too.
    small = dataclasses.replace(WORKLOADS["tiny-nc"], causal=True, seed=61)
    _case(small, gpu, torch.float32, check_oracle=True)
    # 3. Striped layout, GQA, several blocks per partition, permuted lists.
    striped = dataclasses.replace(
        WORKLOADS["tiny-nc"], num_partitions=4, partition_len=1024,
        q_idx=[3, 0, 2], kv_idx=[1, 3, 0], num_q_heads=8, num_kv_heads=2,
        head_dim=128, causal=True, layout=1, seed=62)
    _case(striped, gpu, torch.bfloat16, check_oracle=True)
    # 4. Past 4096 items with a ragged tail and the plain item order.
    _case(queued_tail_config(), gpu, torch.bfloat16)
    # 5. The 1M-token GQA tile at full size (8 KV heads), then the tiny one.
    _case(WORKLOADS["mesh1m-nc-gqa"], gpu, torch.bfloat16)
    _case(WORKLOADS["tiny-nc"], gpu, torch.bfloat16, check_oracle=True)


def test_noalloc_rejects_tiles_beyond_its_scratch():
    """Checked on the host before anything is launched (the fake device
    addresses are never used)."""
    lib = ma.load_library()
    I32P = ctypes.POINTER(ctypes.c_int32)
    fake = [ctypes.c_void_p(0x10000 * (i + 1)) for i in range(5)]

    def call(prob, nq, nkv):
        pr = ma.Problem.make(prob)
        qa = np.arange(nq, dtype=np.int32)
        ka = np.arange(nkv, dtype=np.int32)
        return lib.mesh_attn_tile_fwd_noalloc(
            ctypes.byref(pr), qa.ctypes.data_as(I32P), nq,
            ka.ctypes.data_as(I32P), nkv, *fake[:4], 0, fake[4], None)

    base = dict(num_partitions=512, partition_len=256, num_q_heads=4,
                num_kv_heads=4, head_dim=64, causal=1, layout=0,
                softmax_scale=0.125)
    # more partitions in a list than the kernel arguments carry
    assert call(base, 257, 1) == ma._binding.MA_ERR_UNSUPPORTED
    assert "256" in ma.mesh_attn_last_error()
    # a work list larger than the scratch array: 256 x 256 partitions of
    # 4096 rows
    big = dict(base, partition_len=4096, num_q_heads=32, num_kv_heads=32,
               head_dim=128)
    assert call(big, 256, 256) == ma._binding.MA_ERR_UNSUPPORTED
    assert "scratch" in ma.mesh_attn_last_error()
    # the usual argument checks still apply
    assert call(dict(base, head_dim=96), 1, 1) == \
        ma._binding.MA_ERR_UNSUPPORTED


@pytest.mark.gpu
def test_noalloc_forward_in_a_captured_graph(gpu):
    """The allocation-free forward captured into a HIP graph (two kernel
    launches and nothing else) and replayed three times.  Before each replay
    the outputs are overwritten and an eager allocation-free forward of
    another tile rewrites the shared scratch array, so the replay has to
    rebuild its own work list; every replay must reproduce the eager forward
    bit for bit."""
    cfg = dataclasses.replace(WORKLOADS["tiny-nc"], causal=True, seed=63,
                              partition_len=1024, num_partitions=4,
                              q_idx=[3, 1], kv_idx=[0, 1, 3])
    other = dataclasses.replace(cfg, q_idx=[2], kv_idx=[2, 0], seed=64)
    q, k, v, _ = make_qkv(cfg)
    qd, kd, vd = (t.to(gpu) for t in (q, k, v))
    q2, k2, v2, _ = make_qkv(other)
    q2d, k2d, v2d = (t.to(gpu) for t in (q2, k2, v2))
    prob = cfg.problem()
    P, hq, d = cfg.partition_len, cfg.num_q_heads, cfg.head_dim
    ref_o, ref_l = _noalloc(prob, cfg, qd, kd, vd, torch.bfloat16)  # eager
    torch.cuda.synchronize()
    o = torch.empty((cfg.nq * P, hq, d), dtype=torch.bfloat16, device=gpu)
    lse = torch.empty((hq, cfg.nq * P), dtype=torch.float32, device=gpu)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ma.mesh_attn_tile_fwd_noalloc(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd,
                                      o, lse)
    for rep in range(3):
        o.fill_(float("nan"))
        lse.fill_(float("nan"))
        _noalloc(other.problem(), other, q2d, k2d, v2d, torch.float32)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, ref_o), f"replay {rep}: O differs"
        assert torch.equal(lse, ref_l), f"replay {rep}: LSE differs"
    log("noalloc forward: three graph replays equal the eager forward")

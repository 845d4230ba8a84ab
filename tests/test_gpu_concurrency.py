"""Concurrent calls from several host threads, each on its own stream.

ctypes releases the GIL, so the library's host code (validation, the plan
cache and its pinned upload buffers and events) runs in parallel in four
threads while their kernels overlap on the GPU.  Each thread alternates
between two tiles of its own (so the shared plan cache keeps changing) and
two of them also run the backward; every result must equal the
single-threaded result of the same call bit for bit (both passes are
deterministic)."""

import dataclasses
import threading

import pytest
import torch

import paper_2512_20968_amd as ma
from mesh_inputs import WORKLOADS, make_grad, make_qkv

from helpers import log

pytestmark = pytest.mark.gpu


def _tiles():
    base = dataclasses.replace(WORKLOADS["tiny-nc"], num_partitions=6,
                               partition_len=1024, causal=True)
    lists = [([5, 2], [0, 2, 4, 5]), ([3], [3, 1]), ([4, 0, 1], [1, 4]),
             ([2, 5], [5]), ([1], [0, 1, 2, 3, 4, 5]), ([0, 3], [3, 0]),
             ([4], [4, 2, 0]), ([5, 1], [1, 5, 3])]
    return [dataclasses.replace(base, q_idx=q, kv_idx=kv, seed=70 + i,
                                grad_seed=90 + i, layout=i % 2)
            for i, (q, kv) in enumerate(lists)]


class _Case:
    def __init__(self, cfg, gpu, with_bwd):
        self.cfg = cfg
        q, k, v, _ = make_qkv(cfg)
        self.q, self.k, self.v = (t.to(gpu) for t in (q, k, v))
        P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads, cfg.num_kv_heads,
                         cfg.head_dim)
        self.o = torch.empty((cfg.nq * P, hq, d), dtype=torch.bfloat16,
                             device=gpu)
        self.lse = torch.empty((hq, cfg.nq * P), dtype=torch.float32,
                               device=gpu)
        self.with_bwd = with_bwd
        if with_bwd:
            self.do = make_grad(cfg).to(gpu)
            self.dq = torch.empty((cfg.nq * P, hq, d), dtype=torch.float32,
                                  device=gpu)
            self.dk = torch.empty((cfg.nkv * P, hkv, d), dtype=torch.float32,
                                  device=gpu)
            self.dv = torch.empty_like(self.dk)

    def run(self):
        c = self.cfg
        ma.mesh_attn_tile_fwd(c.problem(), c.q_idx, c.kv_idx, self.q, self.k,
                              self.v, self.o, self.lse)
        if self.with_bwd:
            ma.mesh_attn_tile_bwd(c.problem(), c.q_idx, c.kv_idx, self.q,
                                  self.k, self.v, self.o, self.do, self.lse,
                                  self.dq, self.dk, self.dv)

    def outputs(self):
        outs = [self.o, self.lse]
        if self.with_bwd:
            outs += [self.dq, self.dk, self.dv]
        return [t.clone() for t in outs]


def test_threads_on_separate_streams_match_serial_results(gpu):
    tiles = _tiles()
    # Thread t owns tiles 2t and 2t+1; threads 0 and 2 also run the backward.
    cases = [[_Case(tiles[2 * t + j], gpu, with_bwd=(t % 2 == 0))
              for j in range(2)] for t in range(4)]
    refs = []
    for per in cases:
        refs.append([])
        for c in per:
            c.run()
            torch.cuda.synchronize()
            refs[-1].append(c.outputs())
    failures = []
    start = threading.Barrier(4)

    def work(t):
        try:
            stream = torch.cuda.Stream(device=gpu)
            start.wait()
            with torch.cuda.stream(stream):
                for it in range(24):
                    j = it % 2
                    c = cases[t][j]
                    c.o.fill_(float("nan"))
                    c.lse.fill_(float("nan"))
                    c.run()
                    stream.synchronize()
                    for got, want in zip(c.outputs(), refs[t][j]):
                        if not torch.equal(got, want):
                            failures.append(f"thread {t} iteration {it} tile "
                                            f"{c.cfg.q_idx}x{c.cfg.kv_idx}")
                            return
        except Exception as e:  # collected and re-raised in the main thread
            failures.append(f"thread {t}: {e!r}")

    threads = [threading.Thread(target=work, args=(t,)) for t in range(4)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not failures, failures
    log("four threads on four streams: every result equals the serial one")

"""Seeded synthetic inputs for the tile-attention workloads.

This package is shared by the tests, the benchmark, the HIP path and the oracle
path.  It holds shapes, seeds and random draws only -- none of the method's
arithmetic.  All draws use a CPU ``torch.Generator`` so that both sides see
bit-identical bfloat16 tensors.

The workloads stand in for one GPU's share of the paper's runs (BF16, head dim
128, contiguous or striped partitions of a long sequence; Sections 3.7, 4.1).  The paper uses no
dataset: its inputs are random activations of the attention operator, so i.i.d.
N(0, 1) tensors cast to bfloat16 have the paper's shapes and value range.
"""

from dataclasses import dataclass, field
from typing import List, Optional

import torch


@dataclass(frozen=True)
class TileConfig:
    name: str
    num_partitions: int       # n: partitions of the whole sequence
    partition_len: int        # P: tokens per partition
    q_idx: List[int]          # the tile's Q partitions, in buffer order
    kv_idx: List[int]         # the tile's KV partitions, in buffer order
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    causal: bool
    seed: int
    outliers: bool = False    # one Q row and one K row per partition scaled x8
    grad_seed: Optional[int] = None   # seed of dO for a backward workload
    layout: int = 0           # 0: contiguous partitions, 1: striped positions
    note: str = field(default="", compare=False)

    @property
    def softmax_scale(self) -> float:
        # 1/sqrt(d) rounded to float32: the value the library receives.
        return float(torch.tensor(self.head_dim, dtype=torch.float64).rsqrt()
                     .to(torch.float32))

    @property
    def nq(self) -> int:
        return len(self.q_idx)

    @property
    def nkv(self) -> int:
        return len(self.kv_idx)

    def problem(self) -> dict:
        return dict(num_partitions=self.num_partitions,
                    partition_len=self.partition_len,
                    num_q_heads=self.num_q_heads,
                    num_kv_heads=self.num_kv_heads,
                    head_dim=self.head_dim,
                    causal=int(self.causal),
                    softmax_scale=self.softmax_scale,
                    layout=self.layout)


# Seeded synthetic workloads, by name.
WORKLOADS = {
    "tiny-nc": TileConfig(
        "tiny-nc", 4, 256, [0, 1], [0, 1], 4, 4, 64, False, seed=0,
        note="1024 tokens, 4 partitions of 256, tile {0,1}x{0,1}"),
    "causal-64k": TileConfig(
        "causal-64k", 16, 4096, [4, 5, 6, 7], list(range(8)),
        32, 32, 128, True, seed=1,
        note="65536 tokens, 16 partitions of 4096, tile {4..7}x{0..7}"),
    "mesh1m-nc-gqa": TileConfig(
        "mesh1m-nc-gqa", 256, 4096, list(range(16, 32)),
        list(range(32, 48)), 32, 8, 128, False, seed=2,
        note="1M tokens, 256 partitions, 16x16 tile Q16..31 x KV32..47"),
    "mesh1m-causal-outlier": TileConfig(
        "mesh1m-causal-outlier", 256, 4096, list(range(24, 40)),
        list(range(16, 32)), 32, 32, 128, True, seed=3, outliers=True,
        note="1M tokens, 16x16 tile Q24..39 x KV16..31, x8 outlier rows"),
    "bwd-causal-64k": TileConfig(
        "bwd-causal-64k", 16, 4096, [4, 5, 6, 7], list(range(8)),
        32, 32, 128, True, seed=1, grad_seed=4,
        note="backward of the causal-64k tile; dO from seed 4"),
    # Striped layout (token r of partition p at position r*n + p): every
    # partition pair is near-triangular, so every tile of a mesh carries about
    # the same causal work.
    "striped-causal-64k": TileConfig(
        "striped-causal-64k", 16, 4096, [4, 5, 6, 7], list(range(8)),
        32, 32, 128, True, seed=5, grad_seed=6, layout=1,
        note="65536 tokens striped over 16 partitions of 4096, "
             "tile {4..7}x{0..7}; dO from seed 6"),
    "striped-mesh1m-causal": TileConfig(
        "striped-mesh1m-causal", 256, 4096, list(range(24, 40)),
        list(range(16, 32)), 32, 32, 128, True, seed=7, layout=1,
        note="1M tokens striped over 256 partitions, 16x16 tile "
             "Q24..39 x KV16..31"),
}
# Forward launches of equal-length items: one Q partition of 4096 rows
# against 16 KV partitions, non-causal, Hq query heads on Hq/4 KV heads, so
# 16 Q blocks x Hq heads = 64, 128, 256 or 512 workgroups of 1024 KV blocks
# each keep a quarter, half, all or twice all of the 256 compute units busy.
for _hq in (4, 8, 16, 32):
    _name = f"items-{16 * _hq}"
    WORKLOADS[_name] = TileConfig(
        _name, 64, 4096, [0], list(range(16, 32)), _hq, _hq // 4, 128, False,
        seed=11, note=f"{16 * _hq} equal items: Q partition 0 x KV 16..31, "
                      f"{_hq} q heads / {_hq // 4} kv heads, non-causal")
# Backward launches of equal-length dK/dV items: 16 Q partitions of 4096
# rows against 2, 4 or 8 KV partitions, non-causal, 4 query heads on one KV
# head, so 64, 128 or 256 dK/dV workgroups of 128 keys, each over all 65536
# query rows of the group's 4 heads.
for _nkv in (2, 4, 8):
    _name = f"bwd-items-{32 * _nkv}"
    WORKLOADS[_name] = TileConfig(
        _name, 64, 4096, list(range(16)), list(range(32, 32 + _nkv)), 4, 1,
        128, False, seed=12, grad_seed=13,
        note=f"{32 * _nkv} equal dK/dV items: Q 0..15 x KV 32..{31 + _nkv}, "
             f"4 q heads / 1 kv head, non-causal; dO from seed 13")
del _hq, _nkv, _name


def make_qkv(cfg: TileConfig):
    """Q [nq*P, Hq, d], K and V [nkv*P, Hkv, d] as bfloat16 CPU tensors.

    Draw order: Q, K, V from ``Generator(seed)``, all N(0,1) in float32.  With
    ``outliers``, the same generator then draws one row index per Q partition
    and one per K partition; those rows (every head and dim) are multiplied by
    8 in float32 (exact) before the cast.  Returns ``(q, k, v, extra)`` with
    ``extra['q_outlier_rows']`` / ``['k_outlier_rows']`` as local row indices.
    """
    g = torch.Generator(device="cpu").manual_seed(cfg.seed)
    P, d = cfg.partition_len, cfg.head_dim
    q = torch.randn((cfg.nq * P, cfg.num_q_heads, d), generator=g)
    k = torch.randn((cfg.nkv * P, cfg.num_kv_heads, d), generator=g)
    v = torch.randn((cfg.nkv * P, cfg.num_kv_heads, d), generator=g)
    extra = {}
    if cfg.outliers:
        qo = torch.randint(0, P, (cfg.nq,), generator=g)
        ko = torch.randint(0, P, (cfg.nkv,), generator=g)
        for a in range(cfg.nq):
            q[a * P + int(qo[a])] *= 8.0
        for b in range(cfg.nkv):
            k[b * P + int(ko[b])] *= 8.0
        extra["q_outlier_rows"] = [int(x) for x in qo]
        extra["k_outlier_rows"] = [int(x) for x in ko]
    return (q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16),
            extra)


def make_grad(cfg: TileConfig):
    """dO [nq*P, Hq, d] bfloat16, N(0,1) from ``Generator(grad_seed)``."""
    g = torch.Generator(device="cpu").manual_seed(cfg.grad_seed)
    return torch.randn((cfg.nq * cfg.partition_len, cfg.num_q_heads,
                        cfg.head_dim), generator=g).to(torch.bfloat16)


def sample_rows(cfg: TileConfig, n_list: int, seed_offset: int = 1000,
                extra_local=(), n_random: int = 64):
    """Deterministic sample of tile rows for parity checks on large tiles.

    For every partition of a list of ``n_list`` partitions: local rows
    {0, 1, 63, 64, 127, 128, P/2, P-2, P-1} (block edges), the rows in
    ``extra_local`` (e.g. that partition's outlier row), and ``n_random`` rows
    from ``Generator(seed_offset + seed)``.  Returns sorted unique tile-buffer
    row indices.
    """
    P = cfg.partition_len
    g = torch.Generator(device="cpu").manual_seed(seed_offset + cfg.seed)
    fixed = [0, 1, 63, 64, 127, 128, P // 2, P - 2, P - 1]
    rows = set()
    for a in range(n_list):
        loc = set(r for r in fixed if 0 <= r < P)
        if extra_local:
            loc.add(int(extra_local[a]))
        loc.update(int(x) for x in torch.randint(0, P, (n_random,),
                                                  generator=g))
        rows.update(a * P + r for r in loc)
    return sorted(rows)


def make_merge_parts(k_parts: int, rows: int, heads: int, head_dim: int,
                     seed: int, dtype=torch.bfloat16, neg_inf_frac: float = 0.0):
    """Synthetic partial results for a merge: O parts [k][rows][H][d] ~ N(0,1)
    in ``dtype`` and LSE parts [k][H][rows] ~ 4*N(0,1) + 10 (float32).  With
    ``neg_inf_frac`` > 0 that fraction of LSE entries is set to -inf (a part
    with no visible key), chosen by the same generator."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    o = torch.randn((k_parts, rows, heads, head_dim), generator=g).to(dtype)
    lse = torch.randn((k_parts, heads, rows), generator=g) * 4.0 + 10.0
    if neg_inf_frac > 0:
        mask = torch.rand((k_parts, heads, rows), generator=g) < neg_inf_frac
        lse[mask] = float("-inf")
    return o, lse

"""Block classification of a tile and its canonical run list.

Test infrastructure only (see the package docstring).

The tile's Q buffer is cut into Q blocks of ``bm`` rows and its KV buffer into
KV blocks of ``bn`` rows; both sizes divide the partition length P, so a block
never straddles two partitions.  Q block ``a*(P/bm) + qb`` is block ``qb`` of
list entry ``a`` (buffer order); likewise for KV blocks.

Under the causal rule of Section 3.7 (a key is visible to a query iff its global
position is not larger) a (Q block, KV block) pair is

* EMPTY   (0) when no (query, key) pair in it is visible,
* FULL    (2) when every pair is visible (always, without a mask),
* PARTIAL (1) otherwise.

Section 3.7 states the partition-level version: a partition pair (Q_i, KV_j) is
fully masked for i < j, triangular for i = j and dense for i > j.

Canonical run list (the layout the library must reproduce byte for byte): for
every Q block in buffer order, for every KV list entry ``b`` in list order, the
maximal runs of consecutive KV blocks ``kb`` (ascending) of equal class, with
EMPTY runs dropped.  A run is ``(qblk, b, kb_begin, kb_end, cls)`` with
``kb_end`` exclusive; ``qblk_ptr[q]`` is the index of the first run of Q block
``q`` and ``qblk_ptr[-1]`` the number of runs.  The KV-major mirror swaps the
roles of the two sides (runs of Q blocks per KV block).
"""

import numpy as np

from .attention import CONTIGUOUS, token_positions

EMPTY, PARTIAL, FULL = 0, 1, 2


def classify_blocks(q_idx, kv_idx, part_len, bm, bn, causal,
                    layout=CONTIGUOUS, num_partitions=None):
    """Class of every (Q block, KV block) pair from the extreme positions of
    the two blocks: EMPTY if the first key comes after the last query, FULL if
    the last key comes no later than the first query, PARTIAL otherwise.
    Positions grow with the row inside a partition under both layouts, so a
    block's first and last rows hold its extreme positions.
    Returns ``uint8 [nq*P/bm, nkv*P/bn]``."""
    P = int(part_len)
    assert P % bm == 0 and P % bn == 0
    qpos = token_positions(q_idx, P, layout, num_partitions)
    kpos = token_positions(kv_idx, P, layout, num_partitions)
    q_first, q_last = qpos[::bm], qpos[bm - 1::bm]
    k_first, k_last = kpos[::bn], kpos[bn - 1::bn]
    if not causal:
        return np.full((q_first.size, k_first.size), FULL, dtype=np.uint8)
    cls = np.full((q_first.size, k_first.size), PARTIAL, dtype=np.uint8)
    cls[k_first[None, :] > q_last[:, None]] = EMPTY
    cls[k_last[None, :] <= q_first[:, None]] = FULL
    return cls


def classify_blocks_bruteforce(q_idx, kv_idx, part_len, bm, bn, causal,
                               layout=CONTIGUOUS, num_partitions=None):
    """Same classes from every single (query, key) pair of every block: FULL if
    all pairs are visible, EMPTY if none is, PARTIAL otherwise.  Cost grows with
    the number of token pairs; meant for small tiles."""
    P = int(part_len)
    qpos = token_positions(q_idx, P, layout, num_partitions)
    kpos = token_positions(kv_idx, P, layout, num_partitions)
    nqb, nkb = qpos.size // bm, kpos.size // bn
    cls = np.empty((nqb, nkb), dtype=np.uint8)
    for qb in range(nqb):
        qs = qpos[qb * bm:(qb + 1) * bm]
        if causal:
            vis = kpos[None, :] <= qs[:, None]            # [bm, keys]
        else:
            vis = np.ones((bm, kpos.size), dtype=bool)
        vis = vis.reshape(bm, nkb, bn)
        every = vis.all(axis=(0, 2))
        some = vis.any(axis=(0, 2))
        cls[qb] = np.where(every, FULL, np.where(some, PARTIAL, EMPTY))
    return cls


def run_list(cls, n_lists, blocks_per_part):
    """Canonical runs of a class matrix ``cls [rows, n_lists*blocks_per_part]``.

    For every row (a Q block), for every list entry ``b``, maximal runs of equal
    class among the entry's ``blocks_per_part`` blocks, EMPTY dropped.  Returns
    ``(ptr int32 [rows+1], runs int32 [n_runs, 5])`` with run rows
    ``(row, b, begin, end, cls)``.
    """
    cls = np.asarray(cls)
    rows = cls.shape[0]
    ptr = np.zeros(rows + 1, dtype=np.int32)
    out = []
    for r in range(rows):
        for b in range(n_lists):
            seg = cls[r, b * blocks_per_part:(b + 1) * blocks_per_part]
            cuts = np.flatnonzero(np.diff(seg)) + 1
            starts = np.concatenate(([0], cuts))
            ends = np.concatenate((cuts, [blocks_per_part]))
            for s, e in zip(starts, ends):
                c = int(seg[s])
                if c != EMPTY:
                    out.append((r, b, int(s), int(e), c))
        ptr[r + 1] = len(out)
    runs = np.array(out, dtype=np.int32).reshape(-1, 5)
    return ptr, runs


def kv_major_run_list(cls, n_q_lists, q_blocks_per_part):
    """The same rule applied to the transposed class matrix: for every KV block,
    runs of Q blocks per Q list entry (the orientation a backward pass that owns
    KV blocks iterates in)."""
    return run_list(np.asarray(cls).T, n_q_lists, q_blocks_per_part)

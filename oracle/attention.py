"""Float64 definition of the tile attention, its merge and its gradients.

Test infrastructure only (see the package docstring).

Notation follows the paper.  A sequence of N tokens is split evenly into n
partitions of P = N / n tokens (Section 2.2, Section 3.1); a GPU's tile is the
product of a list of Q partitions and a list of KV partitions (the footprints
I_g^Q and I_g^KV of Section 3.1).  A tile buffer stacks its partitions in the
order of the index list, so row ``a*P + r`` of the Q buffer is token ``r`` of
partition ``q_idx[a]``.  Tensors are ``[rows][heads][head_dim]``; LSE is
``[heads][rows]``, natural log.
"""

import numpy as np

NEG_INF = -np.inf


CONTIGUOUS, STRIPED = 0, 1


def token_positions(part_ids, part_len, layout=CONTIGUOUS, num_partitions=None):
    """Global token position of every row of a stacked partition buffer.

    ``layout = CONTIGUOUS``: the sequence is split evenly and contiguously
    (Section 2.2: Q, K and V are split evenly along the sequence dimension),
    so token ``r`` of partition ``p`` sits at position ``p * P + r``.

    ``layout = STRIPED``: for causal attention Section 3.7 interleaves token
    positions across the partitions (the striped layout of Striped Attention)
    so that every tile holds a similar share of visible pairs.  The paper
    gives no formula; the reading used here deals the positions round robin:
    token ``r`` of partition ``p`` sits at position ``r * n + p``, with ``n``
    = ``num_partitions``.
    """
    part_ids = np.asarray(part_ids, dtype=np.int64)
    r = np.arange(int(part_len), dtype=np.int64)
    if layout == CONTIGUOUS:
        pos = part_ids[:, None] * int(part_len) + r[None, :]
    elif layout == STRIPED:
        n = int(num_partitions)
        assert n >= 1 and np.all((part_ids >= 0) & (part_ids < n))
        pos = r[None, :] * n + part_ids[:, None]
    else:
        raise ValueError(f"unknown layout {layout}")
    return pos.reshape(-1)


def problem_positions(prob, part_ids):
    """``token_positions`` of a partition list under a problem description
    (``partition_len``, ``num_partitions`` and optional ``layout``)."""
    return token_positions(part_ids, prob["partition_len"],
                           int(prob.get("layout", CONTIGUOUS)),
                           prob.get("num_partitions"))


def q_head_to_kv_head(h, num_q_heads, num_kv_heads):
    """GQA: each group of g = Hq / Hkv consecutive query heads shares one KV
    head (Section 4.8), so query head h reads KV head h // g."""
    g = num_q_heads // num_kv_heads
    return h // g


def _allowed(qpos, kpos, causal):
    """Causal rule of Section 3.7: a token attends to itself and to the tokens
    before it, i.e. key position <= query position.  Without a mask every pair
    is allowed."""
    if not causal:
        return np.ones((qpos.shape[0], kpos.shape[0]), dtype=bool)
    return kpos[None, :] <= qpos[:, None]


def attention_rows(q, k, v, qpos, kpos, causal, scale):
    """Attention of query rows ``q [m,d]`` over keys ``k, v [n,d]``.

    The definition of Section 2.1, ``O = softmax(s Q K^T) V``, restricted to the
    allowed keys J of each row, and the LSE statistic of the partial results of
    Section 2.2 (one scalar per query row and head):

        x_j = s * <q, k_j>,  M = max_J x_j,  L = sum_J exp(x_j - M),
        LSE = M + ln L,      O = sum_J exp(x_j - LSE) v_j.

    Two passes (max, then exponentials), not an online softmax.  A row with no
    allowed key gets O = 0 and LSE = -inf.  Returns ``(o [m,d], lse [m])``.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    x = float(scale) * (q @ k.T)
    allowed = _allowed(np.asarray(qpos), np.asarray(kpos), causal)
    x = np.where(allowed, x, NEG_INF)
    m = x.max(axis=1) if x.shape[1] else np.full(x.shape[0], NEG_INF)
    empty = ~np.isfinite(m)
    m_safe = np.where(empty, 0.0, m)
    w = np.exp(x - m_safe[:, None])          # masked entries: exp(-inf) = 0
    l = w.sum(axis=1)
    l_safe = np.where(empty, 1.0, l)
    lse = np.where(empty, NEG_INF, m_safe + np.log(l_safe))
    o = (w @ v) / l_safe[:, None]
    o[empty] = 0.0
    return o, lse


def lse_merge(o_parts, lse_parts):
    """Online-softmax reducer (Section 2.2, Algorithm 2's reduce-scatter).

    Folds partial results ``(O_k [m,d], lse_k [m])`` of the same query rows over
    disjoint key sets into the result over the union of the key sets.  The paper
    cites the reducer without printing it; this is the standard max-shifted
    log-sum-exp combine:

        M = max_k lse_k,  lse = M + ln sum_k exp(lse_k - M),
        O = sum_k exp(lse_k - lse) O_k.

    Parts with lse = -inf carry zero weight; if every part is -inf the result is
    O = 0, lse = -inf.  ``o_parts [k,m,d]``, ``lse_parts [k,m]``.
    """
    o_parts = np.asarray(o_parts, dtype=np.float64)
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    M = lse_parts.max(axis=0)
    empty = ~np.isfinite(M)
    M_safe = np.where(empty, 0.0, M)
    w = np.exp(lse_parts - M_safe[None, :])  # [k, m]
    s = w.sum(axis=0)
    s_safe = np.where(empty, 1.0, s)
    lse = np.where(empty, NEG_INF, M_safe + np.log(s_safe))
    o = np.einsum("km,kmd->md", w / s_safe[None, :], o_parts)
    o[empty] = 0.0
    return o, lse


def attention_rows_bwd(q, k, v, do, lse, D, qpos, kpos, causal, scale):
    """Contribution of query rows ``q [m,d]`` to the attention gradients.

    The paper's backward (Section 3.5, Algorithm 3) computes partial dQ and dKV
    from (Q_u, KV_v, O_u, dO_u) and sums them; it does not print the kernel's
    equations.  These are the gradients of <dO, O(Q, K, V)> for the definition
    in ``attention_rows``, written with the final LSE and with
    D_i = sum_c dO_ic O_ic taken from the final output O:

        P_ij  = exp(x_ij - LSE_i)      (0 where the pair is masked)
        dV_j  = sum_i P_ij dO_i
        dP_ij = <dO_i, v_j>
        dS_ij = P_ij (dP_ij - D_i)
        dQ_i  = s sum_j dS_ij k_j
        dK_j  = s sum_i dS_ij q_i

    Returns ``(dq [m,d], dk [n,d], dv [n,d])``; dk and dv hold only the
    contribution of these m rows.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    lse = np.asarray(lse, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    x = float(scale) * (q @ k.T)
    allowed = _allowed(np.asarray(qpos), np.asarray(kpos), causal)
    live = np.isfinite(lse)
    lse_safe = np.where(live, lse, 0.0)
    p = np.where(allowed & live[:, None], np.exp(x - lse_safe[:, None]), 0.0)
    dv = p.T @ do
    dp = do @ v.T
    ds = p * (dp - D[:, None])
    dq = float(scale) * (ds @ k)
    dk = float(scale) * (ds.T @ q)
    return dq, dk, dv


def _as_f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def tile_forward(prob, q_idx, kv_idx, q, k, v, rows=None, heads=None,
                 row_chunk=256):
    """Attention of every (Q partition, KV partition) pair of a tile, merged
    over the tile's KV footprint (the loop of Algorithm 1 / Algorithm 2).

    ``prob`` holds ``partition_len, num_q_heads, num_kv_heads, causal,
    softmax_scale`` and, for the striped layout, ``layout`` and
    ``num_partitions`` (see ``token_positions``).  ``q [nq*P, Hq, d]``,
    ``k, v [nkv*P, Hkv, d]`` (any float dtype; widened exactly to float64).
    ``rows`` selects tile rows of the Q buffer (default all), ``heads``
    selects query heads (default all).

    The result equals attention over the concatenation of the tile's KV
    partitions, so it is computed in one pass per row here.  Returns
    ``o [len(rows), len(heads), d]`` and ``lse [len(heads), len(rows)]``.
    """
    return forward_at_positions(prob, problem_positions(prob, q_idx),
                                problem_positions(prob, kv_idx), q, k, v,
                                rows, heads, row_chunk)


def forward_at_positions(prob, qpos, kpos, q, k, v, rows=None, heads=None,
                         row_chunk=256):
    """``tile_forward`` for buffers whose rows sit at the given global
    positions (``qpos [rows_q]``, ``kpos [rows_kv]``), e.g. the chunk buffers
    of Section 3.4."""
    hq, hkv = int(prob["num_q_heads"]), int(prob["num_kv_heads"])
    causal = bool(prob["causal"])
    scale = float(prob["softmax_scale"])
    qpos, kpos = np.asarray(qpos), np.asarray(kpos)
    rows = np.arange(qpos.shape[0]) if rows is None else np.asarray(rows)
    heads = list(range(hq)) if heads is None else list(heads)
    d = q.shape[2]
    o = np.zeros((rows.shape[0], len(heads), d))
    lse = np.zeros((len(heads), rows.shape[0]))
    kv_cache = {}
    for hi, h in enumerate(heads):
        hk = q_head_to_kv_head(h, hq, hkv)
        if hk not in kv_cache:
            kv_cache.clear()
            kv_cache[hk] = (_as_f64(k[:, hk, :]), _as_f64(v[:, hk, :]))
        kh, vh = kv_cache[hk]
        for s in range(0, rows.shape[0], row_chunk):
            r = rows[s:s + row_chunk]
            oh, lh = attention_rows(_as_f64(q[r, h, :]), kh, vh, qpos[r], kpos,
                                    causal, scale)
            o[s:s + row_chunk, hi, :] = oh
            lse[hi, s:s + row_chunk] = lh
    return o, lse


def tile_backward(prob, q_idx, kv_idx, q, k, v, do, kv_heads=None,
                  q_rows=None, kv_rows=None, row_chunk=512):
    """Tile gradients (the per-pair loop of Algorithm 3, summed over the tile).

    For each selected KV head the oracle first runs its own float64 forward
    over every query row of the query heads that share it (Section 4.8) to get
    the final O and LSE, then forms D = rowsum(dO * O) and the gradients of
    ``attention_rows_bwd``.  dK and dV of a KV head are summed over its query
    heads.  ``q_rows`` / ``kv_rows`` select which rows of dQ / dK, dV are
    returned (default all).

    Returns ``dq [len(q_rows), len(q_heads), d]``, ``dk, dv [len(kv_rows),
    len(kv_heads), d]``, the list of query heads (in the order of dq's second
    axis), and the forward ``(o, lse)`` of those heads over all rows.
    """
    P = int(prob["partition_len"])
    hq, hkv = int(prob["num_q_heads"]), int(prob["num_kv_heads"])
    causal = bool(prob["causal"])
    scale = float(prob["softmax_scale"])
    g = hq // hkv
    qpos = problem_positions(prob, q_idx)
    kpos = problem_positions(prob, kv_idx)
    nrq, nrk = qpos.shape[0], kpos.shape[0]
    kv_heads = list(range(hkv)) if kv_heads is None else list(kv_heads)
    q_rows = np.arange(nrq) if q_rows is None else np.asarray(q_rows)
    kv_rows = np.arange(nrk) if kv_rows is None else np.asarray(kv_rows)
    q_heads = [hk * g + j for hk in kv_heads for j in range(g)]
    d = q.shape[2]
    dq = np.zeros((q_rows.shape[0], len(q_heads), d))
    dk = np.zeros((kv_rows.shape[0], len(kv_heads), d))
    dv = np.zeros_like(dk)
    o_all = np.zeros((nrq, len(q_heads), d))
    lse_all = np.zeros((len(q_heads), nrq))
    for ki, hk in enumerate(kv_heads):
        kh, vh = _as_f64(k[:, hk, :]), _as_f64(v[:, hk, :])
        ks, vs = kh[kv_rows], vh[kv_rows]
        for j in range(g):
            h = hk * g + j
            hi = ki * g + j
            qh, doh = _as_f64(q[:, h, :]), _as_f64(do[:, h, :])
            for s in range(0, nrq, row_chunk):
                sl = slice(s, s + row_chunk)
                o_all[sl, hi], lse_all[hi, sl] = attention_rows(
                    qh[sl], kh, vh, qpos[sl], kpos, causal, scale)
            D = np.sum(doh * o_all[:, hi], axis=1)
            # dQ of the selected rows: every key of the tile contributes.
            r = q_rows
            dq[:, hi], _, _ = attention_rows_bwd(
                qh[r], kh, vh, doh[r], lse_all[hi, r], D[r], qpos[r], kpos,
                causal, scale)
            # dK, dV of the selected keys: every query row contributes.
            for s in range(0, nrq, row_chunk):
                sl = slice(s, s + row_chunk)
                _, dks, dvs = attention_rows_bwd(
                    qh[sl], ks, vs, doh[sl], lse_all[hi, sl], D[sl],
                    qpos[sl], kpos[kv_rows], causal, scale)
                dk[:, ki] += dks
                dv[:, ki] += dvs
    return dq, dk, dv, q_heads, (o_all, lse_all)

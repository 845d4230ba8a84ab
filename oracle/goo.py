"""Greedy Overlapping Optimization (GOO, Section 3.4): the chunk tasks of a
tile and the step-based greedy planner that orders them.

Test infrastructure only (see the package docstring).

Decomposition.  Each local Q partition is cut into ``k_q`` chunks along the
sequence and each local KV partition into ``k_kv`` chunks.  The Q all-gather
and the output reduce-scatter become ``k_q`` chunk collectives (AG-Q-i,
RS-Q-i), the KV all-gather ``k_kv`` of them (AG-KV-j), and the tile's
attention becomes ``k_q * k_kv`` compute tasks C-i-j (Q chunk i of every
partition of the Q footprint against KV chunk j of every partition of the KV
footprint).  Dependencies: C-i-j needs AG-Q-i and AG-KV-j; RS-Q-i needs every
C-i-j.

Planner.  One step per chunk collective (plus compute-only steps when needed);
each step runs exactly one collective and zero or more compute tasks, all of
which must be ready when the step starts.  The collective of a step is the
candidate with the highest profit = (time of the compute tasks it would make
ready) / (its own time); the step is then filled with already-ready compute
tasks, earliest Q chunk first, until their time reaches gamma * (collective
time).  When no collective can run but compute is ready, a compute-only step
runs one task.  Candidates are every chunk collective that can run: each
AG-Q-i and AG-KV-j not yet scheduled, and each RS-Q-i not yet scheduled whose
compute tasks are all done.  (The paper's worked example looks only at the
lowest-index chunk of each type, a simplification it states for that example;
with equal task costs the general rule picks the same chunks.)

Readings where the paper leaves a choice (the same in the library):
* ties in profit go to the candidate that makes more compute ready, then to
  the order AG-KV, AG-Q, RS-Q (the choices of the worked example), then to
  the lower chunk index;
* among ready compute tasks the order is (Q chunk, KV chunk) ascending;
* a step's fill stops at the first task that brings the total to the target
  or above (the worked example's steps 3, 4 and 6);
* sums of task times run in ascending chunk order (profits) or in fill order
  (step totals), so that the decisions are reproducible bit for bit.
"""

import numpy as np

from .attention import forward_at_positions, lse_merge, problem_positions

AG_Q, AG_KV, RS_Q = "AG-Q", "AG-KV", "RS-Q"
_KIND_ORDER = {AG_KV: 0, AG_Q: 1, RS_Q: 2}


def chunk_rows(part_len, k, i):
    """Local rows ``[i*P/k, (i+1)*P/k)`` of chunk ``i`` of a partition cut into
    ``k`` equal chunks (Section 3.4: chunks along the sequence dimension)."""
    P = int(part_len)
    assert P % k == 0 and 0 <= i < k
    c = P // k
    return range(i * c, (i + 1) * c)


def chunk_buffer_rows(part_len, n_parts, k, i):
    """Rows of a stacked tile buffer (``n_parts`` partitions of ``part_len``
    rows) that make up the output of the chunk collective ``i``: chunk ``i``
    of every partition, in partition order (the concatenation AG-Q-i or
    AG-KV-j produces)."""
    P = int(part_len)
    rows = []
    for a in range(n_parts):
        rows.extend(a * P + r for r in chunk_rows(P, k, i))
    return rows


def goo_plan(k_q, k_kv, t_ag_q, t_ag_kv, t_rs_q, t_c, gamma=1.05):
    """Step-based greedy schedule of the chunk tasks of one tile.

    ``t_c[i][j]`` is the estimated time of compute task C-i-j; the collective
    times are per type (all chunks of a type move the same number of bytes).
    Returns a list of steps ``(comm, tasks)`` with ``comm`` either ``None``
    (compute-only step) or ``(kind, chunk)`` and ``tasks`` a list of
    ``(i, j)``.
    """
    t_comm = {AG_Q: float(t_ag_q), AG_KV: float(t_ag_kv), RS_Q: float(t_rs_q)}
    ag_q, ag_kv, rs_q = set(), set(), set()
    done = set()
    steps = []

    def ready_tasks():
        return sorted((i, j) for i in ag_q for j in ag_kv if (i, j) not in done)

    def unlock(kind, idx):
        # summed in ascending chunk order, so that every implementation of the
        # planner adds the same floating-point numbers in the same order
        if kind == AG_Q:
            return sum(float(t_c[idx][j]) for j in range(k_kv) if j in ag_kv)
        if kind == AG_KV:
            return sum(float(t_c[i][idx]) for i in range(k_q) if i in ag_q)
        return 0.0

    while len(ag_q) < k_q or len(ag_kv) < k_kv or len(rs_q) < k_q:
        cands = [(AG_Q, i) for i in range(k_q) if i not in ag_q]
        cands += [(AG_KV, j) for j in range(k_kv) if j not in ag_kv]
        cands += [(RS_Q, i) for i in range(k_q) if i not in rs_q
                  and all((i, j) in done for j in range(k_kv))]
        ready = ready_tasks()
        if not cands:
            # No collective can run: one ready task advances the dependencies.
            assert ready, "planner stuck"
            steps.append((None, [ready[0]]))
            done.add(ready[0])
            continue
        best = None
        for kind, idx in cands:
            u = unlock(kind, idx)
            key = (u / t_comm[kind], u, -_KIND_ORDER[kind], -idx)
            if best is None or key > best[0]:
                best = (key, kind, idx)
        _, kind, idx = best
        target = float(gamma) * t_comm[kind]
        tasks, total = [], 0.0
        for t in ready:
            if total >= target:
                break
            tasks.append(t)
            total += float(t_c[t[0]][t[1]])
        steps.append(((kind, idx), tasks))
        done.update(tasks)
        {AG_Q: ag_q, AG_KV: ag_kv, RS_Q: rs_q}[kind].add(idx)
    return steps


def plan_makespan(steps, t_ag_q, t_ag_kv, t_rs_q, t_c):
    """Estimated time of a schedule: steps run back to back, and inside a step
    the collective and the compute tasks run concurrently."""
    t_comm = {AG_Q: t_ag_q, AG_KV: t_ag_kv, RS_Q: t_rs_q}
    total = 0.0
    for comm, tasks in steps:
        tc = t_comm[comm[0]] if comm else 0.0
        total += max(tc, sum(t_c[i][j] for i, j in tasks))
    return total


def chunk_forward(prob, q_idx, kv_idx, k_q, i, k_kv, j, q, k, v, heads=None):
    """Compute task C-i-j: attention of the AG-Q-i buffer (chunk ``i`` of
    every partition of ``q_idx``) over the AG-KV-j buffer (chunk ``j`` of
    every partition of ``kv_idx``), with the causal rule on the rows' global
    positions.  ``q [nq*P/k_q, Hq, d]``, ``k, v [nkv*P/k_kv, Hkv, d]``.
    Returns the partial ``(o, lse)`` of the chunk pair."""
    P = int(prob["partition_len"])
    qpos = problem_positions(prob, q_idx)[
        chunk_buffer_rows(P, len(q_idx), k_q, i)]
    kpos = problem_positions(prob, kv_idx)[
        chunk_buffer_rows(P, len(kv_idx), k_kv, j)]
    return forward_at_positions(prob, qpos, kpos, q, k, v, heads=heads)


def accumulate_partial(o_run, lse_run, o_new, lse_new):
    """Running accumulation of chunk partials (the reducer of Section 2.2 on
    two parts): fold ``(o_new [rows, H, d], lse_new [H, rows])`` into the
    running ``(o_run, lse_run)``; returns the new running pair."""
    o = np.empty_like(np.asarray(o_run, dtype=np.float64))
    lse = np.empty_like(np.asarray(lse_run, dtype=np.float64))
    for h in range(o.shape[1]):
        o[:, h], lse[h] = lse_merge(np.stack([o_run[:, h], o_new[:, h]]),
                                    np.stack([lse_run[h], lse_new[h]]))
    return o, lse


def chunk_backward(prob, q_idx, kv_idx, k_q, i, k_kv, j, q, k, v, do):
    """Backward of compute task C-i-j (Algorithm 3's per-pair loop on one
    chunk pair).  ``q, do [nq*P, Hq, d]`` and ``k, v [nkv*P, Hkv, d]`` are the
    whole tile's buffers: the final O and LSE of the Q chunk's rows are those
    over every key of the tile (computed here), while the gradient terms run
    over the rows of Q chunk i and the keys of KV chunk j only.  Returns
    ``dq [rows of Q chunk i, Hq, d]`` and ``dk, dv [rows of KV chunk j, Hkv,
    d]`` (dK, dV summed over the query heads of each KV head)."""
    from .attention import attention_rows, attention_rows_bwd, q_head_to_kv_head
    P = int(prob["partition_len"])
    hq, hkv = int(prob["num_q_heads"]), int(prob["num_kv_heads"])
    causal = bool(prob["causal"])
    scale = float(prob["softmax_scale"])
    qpos = problem_positions(prob, q_idx)
    kpos = problem_positions(prob, kv_idx)
    qr = np.asarray(chunk_buffer_rows(P, len(q_idx), k_q, i))
    kr = np.asarray(chunk_buffer_rows(P, len(kv_idx), k_kv, j))
    d = q.shape[2]
    dq = np.zeros((qr.size, hq, d))
    dk = np.zeros((kr.size, hkv, d))
    dv = np.zeros((kr.size, hkv, d))
    for h in range(hq):
        hk = q_head_to_kv_head(h, hq, hkv)
        qh = np.asarray(q[qr, h, :], dtype=np.float64)
        doh = np.asarray(do[qr, h, :], dtype=np.float64)
        kh = np.asarray(k[:, hk, :], dtype=np.float64)
        vh = np.asarray(v[:, hk, :], dtype=np.float64)
        o, lse = attention_rows(qh, kh, vh, qpos[qr], kpos, causal, scale)
        D = np.sum(doh * o, axis=1)
        gq, gk, gv = attention_rows_bwd(qh, kh[kr], vh[kr], doh, lse, D,
                                        qpos[qr], kpos[kr], causal, scale)
        dq[:, h] = gq
        dk[:, hk] += gk
        dv[:, hk] += gv
    return dq, dk, dv

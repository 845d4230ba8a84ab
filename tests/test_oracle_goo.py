"""Pins of the GOO oracle (Section 3.4): the paper's worked example (chunk
token ranges and the planner's steps, tests/golden/goo_worked_example.json),
schedule invariants on random instances, and the chunk compute tasks, whose
running accumulation over the KV chunks must equal the unchunked tile."""

import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import goo

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "goo_worked_example.json")
GOLDEN_NU = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                         "goo_nonuniform.json")


def _golden():
    return json.load(open(GOLDEN))


def test_worked_example_chunk_tokens():
    g = _golden()
    P = g["tokens_per_gpu"]
    pos = oracle.token_positions(g["q_group"], P)
    rows = goo.chunk_buffer_rows(P, len(g["q_group"]), g["k_q"], 0)
    assert [int(x) for x in pos[rows]] == g["ag_q0_tokens"]
    own = oracle.token_positions([4], P)
    for i, want in enumerate(g["gpu4_q_chunks"]):
        assert [int(own[r]) for r in goo.chunk_rows(P, g["k_q"], i)] == want


def test_worked_example_schedule():
    g = _golden()
    c = g["costs"]
    kq, kkv = g["k_q"], g["k_kv"]
    t_c = [[c["c"]] * kkv for _ in range(kq)]
    steps = goo.goo_plan(kq, kkv, c["ag_q"], c["ag_kv"], c["rs_q"], t_c,
                         gamma=c["gamma"])
    # 2 k_Q + k_KV collective steps plus the two compute-only steps
    assert len(steps) == 2 * kq + kkv + len(g["compute_only_steps"])
    for s, (kind, idx) in g["comm_of_step"].items():
        assert steps[int(s) - 1][0] == (kind, idx), s
    for s, tasks in g["tasks_of_step"].items():
        assert sorted(steps[int(s) - 1][1]) == sorted(map(tuple, tasks)), s
    only = [n + 1 for n, (comm, _) in enumerate(steps) if comm is None]
    assert only == g["compute_only_steps"]
    for n in only:
        assert len(steps[n - 1][1]) == 1


def _golden_steps(case):
    return [((tuple(c) if c else None), [tuple(t) for t in tasks])
            for c, tasks in case["steps"]]


@pytest.mark.parametrize("case", json.load(open(GOLDEN_NU))["cases"],
                         ids=lambda c: c["name"])
def test_nonuniform_costs_higher_index_chunk_wins(case):
    """Hand-derived schedules with unequal task times (Section 3.4's rule
    over every schedulable chunk): a higher-index AG-Q or AG-KV chunk that
    unlocks more compute goes before the lowest-index one."""
    steps = goo.goo_plan(case["k_q"], case["k_kv"], case["t_ag_q"],
                         case["t_ag_kv"], case["t_rs_q"], case["t_c"],
                         case["gamma"])
    assert steps == _golden_steps(case)


@pytest.mark.parametrize("case", json.load(open(GOLDEN_NU))["cases"],
                         ids=lambda c: c["name"])
def test_nonuniform_makespan(case):
    """plan_makespan of the hand-derived schedules equals their makespan
    worked out by hand (steps back to back, each as long as the longer of
    its collective and its tasks)."""
    steps = _golden_steps(case)
    assert goo.plan_makespan(steps, case["t_ag_q"], case["t_ag_kv"],
                             case["t_rs_q"], case["t_c"]) == case["makespan"]


def test_every_chunk_is_a_candidate():
    """On random unequal costs the chosen collective always has the highest
    profit among all schedulable chunks (not only the lowest-index ones)."""
    rng = np.random.default_rng(77)
    higher = 0
    for _ in range(50):
        kq, kkv = int(rng.integers(2, 5)), int(rng.integers(2, 5))
        tq, tkv, trs = (float(x) for x in rng.uniform(0.2, 2.0, 3))
        t_c = rng.uniform(0.1, 2.0, (kq, kkv)).tolist()
        steps = goo.goo_plan(kq, kkv, tq, tkv, trs, t_c, 1.05)
        ag_q, ag_kv = set(), set()
        t_comm = {goo.AG_Q: tq, goo.AG_KV: tkv, goo.RS_Q: trs}
        for comm, _tasks in steps:
            if comm is None:
                continue
            kind, idx = comm
            if kind != goo.RS_Q:
                def unlock(kd, x):
                    if kd == goo.AG_Q:
                        return sum(t_c[x][j] for j in sorted(ag_kv))
                    return sum(t_c[i][x] for i in sorted(ag_q))
                best = max([unlock(goo.AG_Q, i) / tq for i in range(kq)
                            if i not in ag_q] +
                           [unlock(goo.AG_KV, j) / tkv for j in range(kkv)
                            if j not in ag_kv])
                assert unlock(kind, idx) / t_comm[kind] >= best - 1e-12
                pending = ag_q if kind == goo.AG_Q else ag_kv
                n = kq if kind == goo.AG_Q else kkv
                if idx != min(x for x in range(n) if x not in pending):
                    higher += 1
            (ag_q if kind == goo.AG_Q else ag_kv
             if kind == goo.AG_KV else set()).add(idx)
    assert higher > 0


def _check_invariants(kq, kkv, tq, tkv, trs, t_c, gamma, steps):
    seen_comm = {}
    seen_task = {}
    for n, (comm, tasks) in enumerate(steps):
        if comm is None:
            assert len(tasks) == 1
        else:
            assert comm not in seen_comm
            seen_comm[comm] = n
        for t in tasks:
            assert t not in seen_task
            seen_task[t] = n
    assert set(seen_comm) == ({(goo.AG_Q, i) for i in range(kq)}
                              | {(goo.AG_KV, j) for j in range(kkv)}
                              | {(goo.RS_Q, i) for i in range(kq)})
    assert set(seen_task) == {(i, j) for i in range(kq) for j in range(kkv)}
    t_comm = {goo.AG_Q: tq, goo.AG_KV: tkv, goo.RS_Q: trs}
    for (i, j), n in seen_task.items():
        # ready when the step starts: both gathers in strictly earlier steps
        assert seen_comm[(goo.AG_Q, i)] < n and seen_comm[(goo.AG_KV, j)] < n
    for i in range(kq):
        assert all(seen_task[(i, j)] < seen_comm[(goo.RS_Q, i)]
                   for j in range(kkv))
    for comm, tasks in steps:
        if comm is None or not tasks:
            continue
        # just enough: without its last task the step was below its target
        target = gamma * t_comm[comm[0]]
        assert sum(t_c[i][j] for i, j in tasks[:-1]) < target


@pytest.mark.parametrize("seed", range(12))
def test_schedule_invariants_random(seed):
    rng = np.random.default_rng(seed)
    kq = int(rng.integers(1, 5))
    kkv = int(rng.integers(1, max(2, 16 // kq) + 1))
    kkv = min(kkv, 16 // kq)
    tq, tkv, trs = (float(x) for x in rng.uniform(0.1, 2.0, 3))
    t_c = rng.uniform(0.05, 1.5, (kq, kkv)).tolist()
    gamma = float(rng.choice([1.0, 1.05, 1.2]))
    steps = goo.goo_plan(kq, kkv, tq, tkv, trs, t_c, gamma)
    _check_invariants(kq, kkv, tq, tkv, trs, t_c, gamma, steps)
    # a serial schedule (every collective, then every task) is never faster
    serial = kq * (tq + trs) + kkv * tkv + float(np.sum(t_c))
    assert goo.plan_makespan(steps, tq, tkv, trs, t_c) <= serial + 1e-12


def test_first_step_cannot_overlap_and_profit_rule():
    """Nothing is ready before the first gather, so step 1 runs alone; when
    one gather is cheaper per unlocked compute it goes first."""
    steps = goo.goo_plan(2, 2, 1.0, 0.25, 0.5, [[1.0, 1.0], [1.0, 1.0]], 1.0)
    assert steps[0][1] == []
    # after AG-KV-0 (tie at zero profit, AG-KV first), AG-Q-0 unlocks 1.0
    # for 1.0 (profit 1) and AG-KV-1 unlocks nothing: AG-Q-0 next.
    assert steps[0][0] == (goo.AG_KV, 0) and steps[1][0] == (goo.AG_Q, 0)


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("kq,kkv", [(2, 3), (4, 1), (1, 4)])
def test_chunk_tasks_accumulate_to_the_tile(layout, kq, kkv):
    """Running accumulation of C-i-0 .. C-i-(k_KV-1) equals the unchunked
    tile on the rows of Q chunk i, for every i."""
    n, P, d, hq, hkv = 4, 24, 8, 2, 1
    prob = dict(num_partitions=n, partition_len=P, num_q_heads=hq,
                num_kv_heads=hkv, head_dim=d, causal=1,
                softmax_scale=1.0 / math.sqrt(d), layout=layout)
    q_idx, kv_idx = [3, 1], [0, 2, 1]
    rng = np.random.default_rng(5)
    q = rng.standard_normal((len(q_idx) * P, hq, d))
    k = rng.standard_normal((len(kv_idx) * P, hkv, d))
    v = rng.standard_normal((len(kv_idx) * P, hkv, d))
    o_tile, lse_tile = oracle.tile_forward(prob, q_idx, kv_idx, q, k, v)
    for i in range(kq):
        qr = goo.chunk_buffer_rows(P, len(q_idx), kq, i)
        o_run = np.zeros((len(qr), hq, d))
        lse_run = np.full((hq, len(qr)), -np.inf)
        for j in range(kkv):
            kr = goo.chunk_buffer_rows(P, len(kv_idx), kkv, j)
            o_c, lse_c = goo.chunk_forward(prob, q_idx, kv_idx, kq, i, kkv, j,
                                           q[qr], k[kr], v[kr])
            o_run, lse_run = goo.accumulate_partial(o_run, lse_run, o_c, lse_c)
        np.testing.assert_allclose(o_run, o_tile[qr], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse_run, lse_tile[:, qr], rtol=0,
                                   atol=1e-12)


@pytest.mark.parametrize("kq,kkv", [(2, 3), (3, 1)])
def test_chunk_backward_sums_to_the_tile(kq, kkv):
    """dQ of Q chunk i summed over the KV chunks, and dK, dV of KV chunk j
    summed over the Q chunks, equal the tile's gradients (GQA, causal)."""
    n, P, d, hq, hkv = 4, 12, 8, 4, 2
    prob = dict(num_partitions=n, partition_len=P, num_q_heads=hq,
                num_kv_heads=hkv, head_dim=d, causal=1,
                softmax_scale=1.0 / math.sqrt(d), layout=1)
    q_idx, kv_idx = [3, 0], [1, 2, 3]
    rng = np.random.default_rng(9)
    q = rng.standard_normal((len(q_idx) * P, hq, d))
    k = rng.standard_normal((len(kv_idx) * P, hkv, d))
    v = rng.standard_normal((len(kv_idx) * P, hkv, d))
    do = rng.standard_normal((len(q_idx) * P, hq, d))
    tdq, tdk, tdv, heads, _ = oracle.tile_backward(prob, q_idx, kv_idx, q, k,
                                                   v, do)
    assert heads == list(range(hq))
    sdq = np.zeros_like(tdq)
    sdk = np.zeros_like(tdk)
    sdv = np.zeros_like(tdv)
    for i in range(kq):
        qr = goo.chunk_buffer_rows(P, len(q_idx), kq, i)
        for j in range(kkv):
            kr = goo.chunk_buffer_rows(P, len(kv_idx), kkv, j)
            gq, gk, gv = goo.chunk_backward(prob, q_idx, kv_idx, kq, i, kkv, j,
                                            q, k, v, do)
            sdq[qr] += gq
            sdk[kr] += gk
            sdv[kr] += gv
    np.testing.assert_allclose(sdq, tdq, rtol=0, atol=1e-12)
    np.testing.assert_allclose(sdk, tdk, rtol=0, atol=1e-12)
    np.testing.assert_allclose(sdv, tdv, rtol=0, atol=1e-12)

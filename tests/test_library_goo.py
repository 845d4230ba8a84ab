"""Host-side checks of the library's GOO planner (Section 3.4): the paper's
worked example, identical schedules to the oracle's planner on random
instances (the schedule is integer data, compared exactly), and argument
errors.  Chunk-call argument checks that fail before any launch."""

import json
import os

import numpy as np
import pytest

import paper_2512_20968_amd as ma
from oracle import goo

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "goo_worked_example.json")
GOLDEN_NU = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                         "goo_nonuniform.json")


def test_worked_example():
    g = json.load(open(GOLDEN))
    c = g["costs"]
    kq, kkv = g["k_q"], g["k_kv"]
    steps = ma.mesh_attn_goo_plan(kq, kkv, c["ag_q"], c["ag_kv"], c["rs_q"],
                                  [[c["c"]] * kkv] * kq, c["gamma"])
    assert len(steps) == 2 * kq + kkv + len(g["compute_only_steps"])
    for s, (kind, idx) in g["comm_of_step"].items():
        assert steps[int(s) - 1][0] == (kind, idx)
    for s, tasks in g["tasks_of_step"].items():
        assert sorted(steps[int(s) - 1][1]) == sorted(map(tuple, tasks))
    assert [n + 1 for n, (cm, _) in enumerate(steps) if cm is None] == \
        g["compute_only_steps"]


@pytest.mark.parametrize("case", json.load(open(GOLDEN_NU))["cases"],
                         ids=lambda c: c["name"])
def test_nonuniform_golden(case):
    """Hand-derived schedules with unequal task times: a higher-index chunk
    that unlocks more compute is chosen (Section 3.4's rule over every
    schedulable chunk)."""
    got = ma.mesh_attn_goo_plan(case["k_q"], case["k_kv"], case["t_ag_q"],
                                case["t_ag_kv"], case["t_rs_q"],
                                case["t_c"], case["gamma"])
    want = [((tuple(c) if c else None), [tuple(t) for t in tasks])
            for c, tasks in case["steps"]]
    assert got == want


@pytest.mark.parametrize("seed", range(40))
def test_same_schedule_as_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    kq = int(rng.integers(1, 7))
    kkv = int(rng.integers(1, 7))
    if seed % 4 == 0:
        # equal costs: many exact ties, decided by the tie rules
        tq, tkv, trs = 0.5, 1.0, 0.5
        t_c = np.full((kq, kkv), 0.5)
    else:
        tq, tkv, trs = (float(x) for x in rng.uniform(0.05, 3.0, 3))
        t_c = rng.uniform(0.0, 2.0, (kq, kkv))
        if seed % 4 == 1:
            t_c = np.round(t_c * 4) / 4   # coarse values: ties in profit
    gamma = float(rng.choice([1.0, 1.05, 1.5]))
    want = goo.goo_plan(kq, kkv, tq, tkv, trs, t_c.tolist(), gamma)
    got = ma.mesh_attn_goo_plan(kq, kkv, tq, tkv, trs, t_c, gamma)
    assert got == want


@pytest.mark.parametrize("args", [
    (0, 2, 1.0, 1.0, 1.0, 1.05),
    (2, 0, 1.0, 1.0, 1.0, 1.05),
    (2, 2, 0.0, 1.0, 1.0, 1.05),
    (2, 2, 1.0, float("inf"), 1.0, 1.05),
    (2, 2, 1.0, 1.0, float("nan"), 1.05),
    (2, 2, 1.0, 1.0, 1.0, 0.0),
    (65, 64, 1.0, 1.0, 1.0, 1.05),
])
def test_planner_rejects_invalid(args):
    kq, kkv, a, b, c, gamma = args
    t_c = np.ones((max(kq, 1), max(kkv, 1)))
    lib = ma.load_library()
    import ctypes
    steps = (ma.GooStep * 8)()
    tasks = np.zeros((max(kq * kkv, 1), 2), dtype=np.int32)
    n = ctypes.c_int32(0)
    st = lib.mesh_attn_goo_plan(
        kq, kkv, a, b, c,
        t_c.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), gamma, steps, 8,
        tasks.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), ctypes.byref(n))
    assert st == ma._binding.MA_ERR_INVALID_ARG


def test_planner_negative_task_time_and_capacity():
    with pytest.raises(ma.MeshAttnError):
        ma.mesh_attn_goo_plan(2, 2, 1.0, 1.0, 1.0, [[1.0, -1.0], [1.0, 1.0]])
    import ctypes
    lib = ma.load_library()
    t_c = np.ones((3, 3))
    steps = (ma.GooStep * 4)()
    tasks = np.zeros((9, 2), dtype=np.int32)
    n = ctypes.c_int32(0)
    st = lib.mesh_attn_goo_plan(
        3, 3, 0.5, 1.0, 0.5, t_c.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
        1.0, steps, 4, tasks.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
        ctypes.byref(n))
    assert st == ma._binding.MA_ERR_CAPACITY


@pytest.mark.parametrize("chunk", [(0, 3, 0, 1), (1, 1, 0, 1), (0, 1, 2, 2),
                                   (0, 32, 0, 1), (0, 1, 0, 128)])
def test_chunk_fwd_rejects_bad_chunks(chunk):
    """Chunk index out of range or chunks that are not whole blocks (4096
    rows: 3 does not divide, 4096/32 = 128 < 256 Q rows per block, 4096/128 =
    32 < 64 KV rows per block).  The C entry point checks before touching any
    pointer, so dummy device addresses never reach a kernel."""
    import ctypes
    lib = ma.load_library()
    prob = ma.Problem.make(dict(num_partitions=16, partition_len=4096,
                                num_q_heads=32, num_kv_heads=32, head_dim=128,
                                causal=1, layout=0, softmax_scale=0.0884))
    q_idx = (ctypes.c_int32 * 1)(4)
    kv_idx = (ctypes.c_int32 * 1)(0)
    ch = ma.Chunk(*chunk)
    st = lib.mesh_attn_chunk_fwd(ctypes.byref(prob), q_idx, 1, kv_idx, 1,
                                 ctypes.byref(ch), None, None, None, None,
                                 None, 0, None, 0, None)
    assert st == ma._binding.MA_ERR_INVALID_ARG
    assert "chunk" in ma.mesh_attn_last_error()

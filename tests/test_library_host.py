"""Host-side checks of the C-ABI library that need no GPU: every symbol the
header declares is exported, the work list is bit-exact against the oracle's
classifier, and invalid arguments are rejected before anything is launched."""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2512_20968_amd as ma
from mesh_inputs import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "mesh_attn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mesh_attn_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = ma.load_library()
    declared = _declared()
    assert len(declared) >= 10
    for name in declared:
        assert hasattr(lib, name), name
    assert declared == ma.exported_symbols()


@pytest.mark.parametrize("pass_", [0, 1])
def test_block_shape(pass_):
    for d in (64, 128):
        bm, bn = ma.mesh_attn_block_shape(d, pass_)
        assert bm > 0 and bn > 0 and 4096 % bm == 0 and 4096 % bn == 0
    assert ma.mesh_attn_block_shape(96, pass_) == (0, 0)
    assert ma.mesh_attn_block_shape(128, 2) == (0, 0)


def _check_bitexact(prob, q_idx, kv_idx, bm, bn):
    P = prob["partition_len"]
    want_cls = oracle.classify_blocks(q_idx, kv_idx, P, bm, bn, prob["causal"],
                                      prob.get("layout", 0),
                                      prob["num_partitions"])
    got_cls = ma.mesh_attn_classify(prob, q_idx, kv_idx, bm, bn)
    assert got_cls.dtype == np.uint8
    np.testing.assert_array_equal(got_cls, want_cls)
    want_ptr, want_runs = oracle.run_list(want_cls, len(kv_idx), P // bn)
    ptr, runs = ma.mesh_attn_worklist(prob, q_idx, kv_idx, bm, bn)
    np.testing.assert_array_equal(ptr, want_ptr)
    np.testing.assert_array_equal(runs, want_runs)
    want_ptr, want_runs = oracle.kv_major_run_list(want_cls, len(q_idx),
                                                   P // bm)
    ptr, runs = ma.mesh_attn_worklist_kv_major(prob, q_idx, kv_idx, bm, bn)
    np.testing.assert_array_equal(ptr, want_ptr)
    np.testing.assert_array_equal(runs, want_runs)


@pytest.mark.parametrize("name", list(WORKLOADS))
@pytest.mark.parametrize("pass_", [0, 1])
def test_worklist_bitexact_on_workloads(name, pass_):
    cfg = WORKLOADS[name]
    bm, bn = ma.mesh_attn_block_shape(cfg.head_dim, pass_)
    _check_bitexact(cfg.problem(), cfg.q_idx, cfg.kv_idx, bm, bn)


def test_worklist_bitexact_random_tiles():
    rng = np.random.default_rng(11)
    for _ in range(60):
        n = int(rng.integers(1, 12))
        bm = int(rng.choice([1, 2, 4, 8, 16]))
        bn = int(rng.choice([1, 2, 4, 8, 16]))
        P = int(np.lcm(bm, bn) * rng.integers(1, 5))
        q_idx = [int(x) for x in rng.choice(n, size=int(rng.integers(1, n + 1)),
                                            replace=False)]
        kv_idx = [int(x) for x in rng.choice(n,
                                             size=int(rng.integers(1, n + 1)),
                                             replace=False)]
        prob = dict(num_partitions=n, partition_len=P, num_q_heads=2,
                    num_kv_heads=1, head_dim=64,
                    causal=int(rng.integers(0, 2)), softmax_scale=0.125,
                    layout=int(rng.integers(0, 2)))
        _check_bitexact(prob, q_idx, kv_idx, bm, bn)


def test_worklist_small_hand_fixture():
    import json
    g = json.load(open(os.path.join(ROOT, "tests", "golden",
                                    "runlist_small.json")))
    prob = dict(num_partitions=3, partition_len=g["partition_len"],
                num_q_heads=1, num_kv_heads=1, head_dim=64, causal=1,
                softmax_scale=1.0)
    ptr, runs = ma.mesh_attn_worklist(prob, g["q_idx"], g["kv_idx"], g["bm"],
                                      g["bn"])
    assert ptr.tolist() == g["qblk_ptr"] and runs.tolist() == g["runs"]
    ptr, runs = ma.mesh_attn_worklist_kv_major(prob, g["q_idx"], g["kv_idx"],
                                               g["bm"], g["bn"])
    assert ptr.tolist() == g["kv_major_ptr"]
    assert runs.tolist() == g["kv_major_runs"]


def _prob(**kw):
    p = dict(num_partitions=4, partition_len=256, num_q_heads=4,
             num_kv_heads=4, head_dim=64, causal=1, softmax_scale=0.125)
    p.update(kw)
    return p


@pytest.mark.parametrize("kw,q_idx,kv_idx,status", [
    (dict(num_q_heads=6, num_kv_heads=4), [0], [0], ma._binding.MA_ERR_INVALID_ARG),
    (dict(causal=2), [0], [0], ma._binding.MA_ERR_INVALID_ARG),
    (dict(layout=2), [0], [0], ma._binding.MA_ERR_INVALID_ARG),
    (dict(layout=-1), [0], [0], ma._binding.MA_ERR_INVALID_ARG),
    (dict(softmax_scale=0.0), [0], [0], ma._binding.MA_ERR_INVALID_ARG),
    (dict(softmax_scale=float("nan")), [0], [0], ma._binding.MA_ERR_INVALID_ARG),
    ({}, [0, 4], [0], ma._binding.MA_ERR_INVALID_ARG),
    ({}, [0, 0], [0], ma._binding.MA_ERR_INVALID_ARG),
    ({}, [0], [-1], ma._binding.MA_ERR_INVALID_ARG),
    (dict(partition_len=100), [0], [0], ma._binding.MA_ERR_INVALID_ARG),
])
def test_worklist_rejects_invalid(kw, q_idx, kv_idx, status):
    with pytest.raises(ma.MeshAttnError) as ei:
        ma.mesh_attn_worklist(_prob(**kw), q_idx, kv_idx, 128, 64)
    assert ei.value.status == status
    assert ma.mesh_attn_last_error() != ""


def _raw_fwd(prob, q_idx, kv_idx, ptrs, ws_bytes, o_dtype=0):
    lib = ma.load_library()
    pr = ma.Problem.make(prob)
    qa = np.asarray(q_idx, np.int32)
    ka = np.asarray(kv_idx, np.int32)
    I32P = ctypes.POINTER(ctypes.c_int32)
    return lib.mesh_attn_tile_fwd(
        ctypes.byref(pr), qa.ctypes.data_as(I32P), len(qa),
        ka.ctypes.data_as(I32P), len(ka), *[ctypes.c_void_p(p) for p in ptrs[:4]],
        o_dtype, ctypes.c_void_p(ptrs[4]), ctypes.c_void_p(ptrs[5]), ws_bytes,
        None)


def test_fwd_validation_before_launch():
    """Every rejection happens on the host: these calls pass fake device
    addresses, which are never dereferenced because validation fails first."""
    good = [0x10000 * (i + 1) for i in range(6)]
    need = ma.mesh_attn_fwd_workspace_size(_prob(), 2, 2)
    assert need > 0
    cases = [
        (_prob(head_dim=96), good, need, 0, ma._binding.MA_ERR_UNSUPPORTED),
        (_prob(), good[:5] + [0], need, 0, ma._binding.MA_ERR_INVALID_ARG),
        (_prob(), [good[0] + 8] + good[1:], need, 0,
         ma._binding.MA_ERR_INVALID_ARG),
        (_prob(), good, need - 1, 0, ma._binding.MA_ERR_WORKSPACE_TOO_SMALL),
        (_prob(), good, need, 7, ma._binding.MA_ERR_INVALID_ARG),
        (_prob(partition_len=192), good, need, 0,
         ma._binding.MA_ERR_INVALID_ARG),
    ]
    for prob, ptrs, wsb, odt, status in cases:
        assert _raw_fwd(prob, [0, 1], [0, 1], ptrs, wsb, odt) == status, prob
        assert ma.mesh_attn_last_error()


def test_merge_validation_before_launch():
    lib = ma.load_library()
    v = ctypes.c_void_p(0x10000)
    for kparts, rows, heads, d, status in [
            (0, 4, 1, 64, ma._binding.MA_ERR_INVALID_ARG),
            (2, -1, 1, 64, ma._binding.MA_ERR_INVALID_ARG),
            (2, 4, 0, 64, ma._binding.MA_ERR_INVALID_ARG),
            (2, 4, 1, 60, ma._binding.MA_ERR_UNSUPPORTED),
            (2, 4, 1, 512, ma._binding.MA_ERR_UNSUPPORTED)]:
        st = lib.mesh_attn_lse_merge(kparts, rows, heads, d, v, 0, v, v, 0, v,
                                     None)
        assert st == status
    # rows == 0 is a valid no-op that touches nothing.
    assert lib.mesh_attn_lse_merge(2, 0, 1, 64, None, 0, None, None, 0, None,
                                   None) == 0


def test_bwd_validation_before_launch():
    lib = ma.load_library()
    pr = ma.Problem.make(_prob())
    qa = np.asarray([0, 1], np.int32)
    I32P = ctypes.POINTER(ctypes.c_int32)
    ptrs = [ctypes.c_void_p(0x10000 * (i + 1)) for i in range(9)]
    need = ma.mesh_attn_bwd_workspace_size(pr, 2, 2)
    ws = ctypes.c_void_p(0x100000)
    st = lib.mesh_attn_tile_bwd(ctypes.byref(pr), qa.ctypes.data_as(I32P), 2,
                                qa.ctypes.data_as(I32P), 2, *ptrs, 2, ws, need,
                                None)
    assert st == ma._binding.MA_ERR_INVALID_ARG
    st = lib.mesh_attn_tile_bwd(ctypes.byref(pr), qa.ctypes.data_as(I32P), 2,
                                qa.ctypes.data_as(I32P), 2, *ptrs, 0, ws,
                                need - 1, None)
    assert st == ma._binding.MA_ERR_WORKSPACE_TOO_SMALL


def test_product_has_no_cpu_fallback_and_no_oracle_import():
    """The binding and the library sources never reach the oracle."""
    pkg = os.path.join(ROOT, "paper_2512_20968_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text, f


def test_struct_layouts_match_the_header(tmp_path):
    """The binding's ctypes structs have the header's field offsets and sizes
    (a C program built from include/mesh_attn.h prints them)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    structs = {"ma_problem_t": ma.Problem, "ma_run_t": ma._binding.Run,
               "ma_chunk_t": ma.Chunk, "ma_goo_step_t": ma.GooStep}
    lines = ["#include <stddef.h>", "#include <stdio.h>",
             '#include "mesh_attn.h"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", '
                         f'offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([gcc, "-D__HIP_PLATFORM_AMD__", "-I",
                    os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True,
                         text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l}
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, \
                (cname, fname)
    # the problem's field order is the one of the boundary's definition
    assert [f for f, _ in ma.Problem._fields_] == [
        "num_partitions", "partition_len", "num_q_heads", "num_kv_heads",
        "head_dim", "causal", "layout", "softmax_scale"]


def test_concurrent_host_calls_and_thread_local_errors():
    """Eight threads call the work-list builders at once (ctypes releases the
    GIL, so the library runs them concurrently) and each provokes its own
    error: every list equals the single-threaded one, and every thread reads
    its own last-error text (the text is per thread)."""
    import threading
    prob = _prob(num_partitions=16, partition_len=512)
    q_idx, kv_idx = [9, 3, 12], [0, 5, 9, 12, 15]
    ref = ma.mesh_attn_worklist(prob, q_idx, kv_idx, 128, 64)
    ref_kv = ma.mesh_attn_worklist_kv_major(prob, q_idx, kv_idx, 128, 64)
    failures = []
    start = threading.Barrier(8)

    def work(t):
        try:
            start.wait()
            for it in range(40):
                ptr, runs = ma.mesh_attn_worklist(prob, q_idx, kv_idx, 128, 64)
                assert np.array_equal(ptr, ref[0])
                assert np.array_equal(runs, ref[1])
                ptr, runs = ma.mesh_attn_worklist_kv_major(prob, q_idx, kv_idx,
                                                           128, 64)
                assert np.array_equal(ptr, ref_kv[0])
                assert np.array_equal(runs, ref_kv[1])
                bad = 100 + 8 * it + t
                with pytest.raises(ma.MeshAttnError) as ei:
                    ma.mesh_attn_worklist(prob, [bad], kv_idx, 128, 64)
                want = f"= {bad} outside [0, 16)"
                assert want in ei.value.args[0], ei.value.args[0]
                assert want in ma.mesh_attn_last_error()
        except Exception as e:  # collected and re-raised in the main thread
            failures.append(f"thread {t}: {e!r}")

    threads = [threading.Thread(target=work, args=(t,)) for t in range(8)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not failures, failures

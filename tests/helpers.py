"""Shared helpers of the GPU parity tests (inputs to device, oracle on
sampled rows, tolerance checks).  The tolerances are the parity bar: forward
max |O err| <= 2e-2 and max |LSE err| <= 1e-3 (absolute) for bf16 inputs with
float32 accumulation; backward max |dX err| <= 5e-2 * max |dX|."""

import sys
import time

import numpy as np
import torch

import oracle
import paper_2512_20968_amd as ma

O_TOL = 2e-2
LSE_TOL = 1e-3
GRAD_REL_TOL = 5e-2


def queued_tail_config():
    """A causal tile of 4137 forward items (197 Q blocks of 256 rows x 21
    query heads): more than the 4096 items from which the forward takes the
    last quarter of every XCD lane from per-lane counters, an item count that
    is not a multiple of 8, and 7 KV heads (so the plain item order rather
    than the KV-head-per-XCD one).  Q partitions 3..199 against KV partitions
    0, 100 and 199 of 256 tokens: FULL, PARTIAL and EMPTY block pairs."""
    import dataclasses
    from mesh_inputs import WORKLOADS
    return dataclasses.replace(
        WORKLOADS["tiny-nc"], name="queued-tail", num_partitions=200,
        partition_len=256, q_idx=list(range(3, 200)), kv_idx=[0, 100, 199],
        num_q_heads=21, num_kv_heads=7, head_dim=64, causal=True, seed=63)


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def to_np(t):
    """bf16/float tensor -> float32 numpy (exact widening)."""
    return t.detach().float().cpu().numpy()


def run_fwd(prob, q_idx, kv_idx, q, k, v, out_dtype=torch.bfloat16):
    dev = q.device
    P = prob["partition_len"]
    hq, d = prob["num_q_heads"], prob["head_dim"]
    rows = len(q_idx) * P
    o = torch.empty((rows, hq, d), dtype=out_dtype, device=dev)
    lse = torch.empty((hq, rows), dtype=torch.float32, device=dev)
    ma.mesh_attn_tile_fwd(prob, q_idx, kv_idx, q, k, v, o, lse)
    return o, lse


def check_fwd(tag, o_gpu, lse_gpu, o_ref, lse_ref):
    """o_* [rows, H, d], lse_* [H, rows]; -inf pattern must match exactly."""
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    lse_gpu = np.asarray(lse_gpu, dtype=np.float64)
    assert np.all(np.isfinite(o_gpu)), f"{tag}: non-finite O"
    ninf_g, ninf_r = np.isneginf(lse_gpu), np.isneginf(lse_ref)
    assert np.array_equal(ninf_g, ninf_r), \
        f"{tag}: -inf LSE pattern differs ({ninf_g.sum()} vs {ninf_r.sum()})"
    eo = float(np.abs(o_gpu - o_ref).max()) if o_ref.size else 0.0
    fin = ~ninf_r
    el = float(np.abs(lse_gpu[fin] - lse_ref[fin]).max()) if fin.any() else 0.0
    log(f"{tag}: max|O err| {eo:.3e}  max|LSE err| {el:.3e}")
    assert eo <= O_TOL, f"{tag}: max|O err| {eo} > {O_TOL}"
    assert el <= LSE_TOL, f"{tag}: max|LSE err| {el} > {LSE_TOL}"
    return eo, el


def check_grad(tag, g, r):
    g = np.asarray(g, dtype=np.float64)
    assert np.all(np.isfinite(g)), f"{tag}: non-finite gradient"
    scale = float(np.abs(r).max())
    err = float(np.abs(g - r).max())
    log(f"{tag}: max|err| {err:.3e}  max|ref| {scale:.3e}  "
        f"ratio {err / max(scale, 1e-30):.3e}")
    assert err <= GRAD_REL_TOL * scale, f"{tag}: {err} > 5e-2 * {scale}"
    return err / max(scale, 1e-30)


# ---------------------------------------------------------------------------
# The float64 oracle on many rows and heads, spread over host processes.
#
# A full-size backward check needs the oracle's forward over every query row
# of the checked heads (the final LSE and D of every row enter dK and dV).
# The oracle's row functions are called here unchanged, one (query head, row
# chunk) per task, and the partial dK, dV of the chunks are summed -- the
# same decomposition the oracle's own tile loop uses.  Workers are started
# from a fresh interpreter (forkserver), never touch the GPU, run one BLAS
# thread each, and read the inputs through read-only memory maps.
# ---------------------------------------------------------------------------

_W = {}


def oracle_workers():
    import os
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _worker_init(files):
    from threadpoolctl import threadpool_limits
    _W["limit"] = threadpool_limits(1)
    for name, (path, shape) in files.items():
        _W[name] = np.memmap(path, dtype=np.float32, mode="r", shape=shape)


def _bwd_task(args):
    """One (query head, row chunk): forward of the chunk's rows over every key
    (final O, LSE), D = rowsum(dO * O), then dQ of the checked rows in the
    chunk and the chunk's contribution to dK, dV of the checked keys."""
    from oracle.attention import attention_rows, attention_rows_bwd
    (hi, hk_i, lo, hi_row, qsel, kv_rows, qpos, kpos, causal, scale) = args
    qh = np.asarray(_W["q"][hi, lo:hi_row], dtype=np.float64)
    doh = np.asarray(_W["do"][hi, lo:hi_row], dtype=np.float64)
    kh = np.asarray(_W["k"][hk_i], dtype=np.float64)
    vh = np.asarray(_W["v"][hk_i], dtype=np.float64)
    qp = qpos[lo:hi_row]
    o, lse = attention_rows(qh, kh, vh, qp, kpos, causal, scale)
    D = np.sum(doh * o, axis=1)
    dq = None
    if len(qsel):
        r = np.asarray(qsel) - lo
        dq, _, _ = attention_rows_bwd(qh[r], kh, vh, doh[r], lse[r], D[r],
                                      qp[r], kpos, causal, scale)
    dk = dv = None
    if len(kv_rows):
        _, dk, dv = attention_rows_bwd(qh, kh[kv_rows], vh[kv_rows], doh, lse,
                                       D, qp, kpos[kv_rows], causal, scale)
    return hi, hk_i, qsel, dq, dk, dv


def _fwd_task(args):
    """Forward of one (query head, chunk of selected rows) over every key."""
    from oracle.attention import attention_rows
    (hi, hk_i, rsel, qpos, kpos, causal, scale) = args
    qh = np.asarray(_W["q"][hi, rsel], dtype=np.float64)
    kh = np.asarray(_W["k"][hk_i], dtype=np.float64)
    vh = np.asarray(_W["v"][hk_i], dtype=np.float64)
    o, lse = attention_rows(qh, kh, vh, qpos[rsel], kpos, causal, scale)
    return hi, rsel, o, lse


def _pool_map(arrays, fn, tasks):
    """Runs ``fn`` over ``tasks`` in worker processes that see ``arrays``
    (name -> CPU tensor [rows][heads][d]) as float32 memory maps laid out
    [heads][rows][d].  Yields the results in task order."""
    import os
    import shutil
    import tempfile
    from concurrent.futures import ProcessPoolExecutor
    import multiprocessing as mp

    shm = "/dev/shm" if os.path.isdir("/dev/shm") else None
    tmpdir = tempfile.mkdtemp(prefix="oracle_", dir=shm)
    try:
        files = {}
        for name, t in arrays.items():
            a = np.ascontiguousarray(t.float().permute(1, 0, 2).numpy())
            path = os.path.join(tmpdir, name)
            mm = np.memmap(path, dtype=np.float32, mode="w+", shape=a.shape)
            mm[:] = a
            mm.flush()
            del mm, a
            files[name] = (path, tuple(t.shape[i] for i in (1, 0, 2)))
        ctx = mp.get_context("forkserver")
        with ProcessPoolExecutor(max_workers=oracle_workers(), mp_context=ctx,
                                 initializer=_worker_init,
                                 initargs=(files,)) as ex:
            for r in ex.map(fn, tasks):
                yield r
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)


def oracle_forward_rows(prob, q_idx, kv_idx, q, k, v, rows, heads,
                        row_chunk=512):
    """The oracle's forward (O, LSE) of the selected tile rows and query
    heads, as ``oracle.tile_forward(..., rows=rows, heads=heads)`` returns
    them, computed row chunk by row chunk in worker processes."""
    hq, hkv = int(prob["num_q_heads"]), int(prob["num_kv_heads"])
    g = hq // hkv
    heads = list(heads)
    kv_heads = sorted({h // g for h in heads})
    rows = np.asarray(rows, dtype=np.int64)
    qpos = oracle.problem_positions(prob, q_idx)
    kpos = oracle.problem_positions(prob, kv_idx)
    tasks = [(hi, kv_heads.index(h // g), rows[s:s + row_chunk], qpos, kpos,
              bool(prob["causal"]), float(prob["softmax_scale"]))
             for hi, h in enumerate(heads)
             for s in range(0, rows.shape[0], row_chunk)]
    d = q.shape[2]
    o = np.zeros((rows.shape[0], len(heads), d))
    lse = np.zeros((len(heads), rows.shape[0]))
    pos = {int(r): i for i, r in enumerate(rows)}
    arrays = {"q": q[:, heads], "k": k[:, kv_heads], "v": v[:, kv_heads]}
    for hi, rsel, oc, lc in _pool_map(arrays, _fwd_task, tasks):
        idx = [pos[int(r)] for r in rsel]
        o[idx, hi] = oc
        lse[hi, idx] = lc
    return o, lse


def oracle_backward_rows(prob, q_idx, kv_idx, q, k, v, do, kv_heads, q_rows,
                         kv_rows, row_chunk=512):
    """dQ of ``q_rows`` and dK, dV of ``kv_rows`` for the query heads of
    ``kv_heads`` (all query heads of each KV head), from the oracle's float64
    row functions.  ``q, do [rows_q, Hq, d]`` and ``k, v [rows_kv, Hkv, d]``
    are CPU tensors.  Returns ``dq [len(q_rows), len(q_heads), d]``, ``dk, dv
    [len(kv_rows), len(kv_heads), d]`` and the list of query heads."""
    hq, hkv = int(prob["num_q_heads"]), int(prob["num_kv_heads"])
    g = hq // hkv
    causal = bool(prob["causal"])
    scale = float(prob["softmax_scale"])
    kv_heads = list(kv_heads)
    q_heads = [hk * g + j for hk in kv_heads for j in range(g)]
    q_rows = np.asarray(sorted(q_rows), dtype=np.int64)
    kv_rows = np.asarray(kv_rows, dtype=np.int64)
    qpos = oracle.problem_positions(prob, q_idx)
    kpos = oracle.problem_positions(prob, kv_idx)
    nrq = qpos.shape[0]
    d = q.shape[2]
    tasks = []
    for ki in range(len(kv_heads)):
        for j in range(g):
            hi = ki * g + j
            for lo in range(0, nrq, row_chunk):
                hi_row = min(nrq, lo + row_chunk)
                qsel = q_rows[(q_rows >= lo) & (q_rows < hi_row)]
                tasks.append((hi, ki, lo, hi_row, qsel, kv_rows, qpos, kpos,
                              causal, scale))
    dq = np.zeros((len(q_rows), len(q_heads), d))
    dk = np.zeros((len(kv_rows), len(kv_heads), d))
    dv = np.zeros_like(dk)
    where = {int(r): i for i, r in enumerate(q_rows)}
    arrays = {"q": q[:, q_heads], "do": do[:, q_heads], "k": k[:, kv_heads],
              "v": v[:, kv_heads]}
    # Partial sums are added in task order, so the result does not depend on
    # which worker finishes first.
    for hi, ki, qsel, gq, gk, gv in _pool_map(arrays, _bwd_task, tasks):
        if gq is not None:
            for t, r in enumerate(qsel):
                dq[where[int(r)], hi] = gq[t]
        if gk is not None:
            dk[:, ki] += gk
            dv[:, ki] += gv
    return dq, dk, dv, q_heads

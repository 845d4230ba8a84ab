"""ctypes binding of the mesh_attn C ABI.

torch is used for device memory and the current stream only.
"""

import ctypes
import os
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libmesh_attn.so"

MA_OK, MA_ERR_INVALID_ARG, MA_ERR_UNSUPPORTED = 0, 1, 2
MA_ERR_WORKSPACE_TOO_SMALL, MA_ERR_HIP, MA_ERR_CAPACITY = 3, 4, 5
MA_BF16, MA_FP32 = 0, 1
MA_CLS_EMPTY, MA_CLS_PARTIAL, MA_CLS_FULL = 0, 1, 2

_STATUS = {0: "MA_OK", 1: "MA_ERR_INVALID_ARG", 2: "MA_ERR_UNSUPPORTED",
           3: "MA_ERR_WORKSPACE_TOO_SMALL", 4: "MA_ERR_HIP",
           5: "MA_ERR_CAPACITY"}


class MeshAttnError(RuntimeError):
    def __init__(self, fn, status, text):
        self.status = status
        super().__init__(f"{fn}: {_STATUS.get(status, status)}: {text}")


MA_LAYOUT_CONTIGUOUS, MA_LAYOUT_STRIPED = 0, 1


class Problem(ctypes.Structure):
    """ma_problem_t."""
    _fields_ = [("num_partitions", ctypes.c_int32),
                ("partition_len", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32),
                ("causal", ctypes.c_int32),
                ("layout", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float)]

    @classmethod
    def make(cls, prob):
        if isinstance(prob, Problem):
            return prob
        return cls(num_partitions=int(prob["num_partitions"]),
                   partition_len=int(prob["partition_len"]),
                   num_q_heads=int(prob["num_q_heads"]),
                   num_kv_heads=int(prob["num_kv_heads"]),
                   head_dim=int(prob["head_dim"]),
                   causal=int(prob["causal"]),
                   layout=int(prob.get("layout", MA_LAYOUT_CONTIGUOUS)),
                   softmax_scale=float(prob["softmax_scale"]))


class Run(ctypes.Structure):
    """ma_run_t: one run of the work list."""
    _fields_ = [("qblk", ctypes.c_int32),
                ("kv_list_pos", ctypes.c_int32),
                ("kb_begin", ctypes.c_int32),
                ("kb_end", ctypes.c_int32),
                ("cls", ctypes.c_int32)]


_lock = threading.Lock()
_lib = None

class Chunk(ctypes.Structure):
    """ma_chunk_t: compute task C-i-j of a tile cut into k_Q x k_KV chunks."""
    _fields_ = [("q_chunk", ctypes.c_int32),
                ("num_q_chunks", ctypes.c_int32),
                ("kv_chunk", ctypes.c_int32),
                ("num_kv_chunks", ctypes.c_int32)]


class GooStep(ctypes.Structure):
    """ma_goo_step_t."""
    _fields_ = [("comm_kind", ctypes.c_int32),
                ("comm_chunk", ctypes.c_int32),
                ("first_task", ctypes.c_int32),
                ("num_tasks", ctypes.c_int32)]


MA_GOO_NONE, MA_GOO_AG_Q, MA_GOO_AG_KV, MA_GOO_RS_Q = 0, 1, 2, 3
GOO_KIND_NAMES = {MA_GOO_AG_Q: "AG-Q", MA_GOO_AG_KV: "AG-KV",
                  MA_GOO_RS_Q: "RS-Q"}

_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_p = ctypes.c_void_p
_sz = ctypes.c_size_t
_PROB = ctypes.POINTER(Problem)
_I32P = ctypes.POINTER(ctypes.c_int32)

_SIGNATURES = {
    "mesh_attn_block_shape": (None, [_i32, _i32, _I32P, _I32P]),
    "mesh_attn_classify": (_i32, [_PROB, _I32P, _i32, _I32P, _i32, _i32, _i32,
                                  _p]),
    "mesh_attn_worklist": (_i32, [_PROB, _I32P, _i32, _I32P, _i32, _i32, _i32,
                                  _I32P, ctypes.POINTER(Run), _i64,
                                  ctypes.POINTER(ctypes.c_int64)]),
    "mesh_attn_worklist_kv_major": (_i32, [_PROB, _I32P, _i32, _I32P, _i32,
                                           _i32, _i32, _I32P,
                                           ctypes.POINTER(Run), _i64,
                                           ctypes.POINTER(ctypes.c_int64)]),
    "mesh_attn_fwd_workspace_size": (_sz, [_PROB, _i32, _i32]),
    "mesh_attn_bwd_workspace_size": (_sz, [_PROB, _i32, _i32]),
    "mesh_attn_tile_fwd": (_i32, [_PROB, _I32P, _i32, _I32P, _i32, _p, _p, _p,
                                  _p, _i32, _p, _p, _sz, _p]),
    "mesh_attn_tile_fwd_noalloc": (_i32, [_PROB, _I32P, _i32, _I32P, _i32, _p,
                                          _p, _p, _p, _i32, _p, _p]),
    "mesh_attn_lse_merge": (_i32, [_i32, _i64, _i32, _i32, _p, _i32, _p, _p,
                                   _i32, _p, _p]),
    "mesh_attn_tile_bwd": (_i32, [_PROB, _I32P, _i32, _I32P, _i32, _p, _p, _p,
                                  _p, _p, _p, _p, _p, _p, _i32, _p, _sz, _p]),
    "mesh_attn_chunk_fwd_workspace_size": (_sz, [_PROB, _i32, _i32]),
    "mesh_attn_chunk_fwd": (_i32, [_PROB, _I32P, _i32, _I32P, _i32,
                                   ctypes.POINTER(Chunk), _p, _p, _p, _p, _p,
                                   _i32, _p, _sz, _p]),
    "mesh_attn_chunk_bwd_workspace_size": (_sz, [_PROB, _i32, _i32]),
    "mesh_attn_chunk_bwd": (_i32, [_PROB, _I32P, _i32, _I32P, _i32,
                                   ctypes.POINTER(Chunk), _p, _p, _p, _p, _p,
                                   _p, _p, _p, _p, _i32, _p, _sz, _p]),
    "mesh_attn_goo_plan": (_i32, [_i32, _i32, ctypes.c_double, ctypes.c_double,
                                  ctypes.c_double,
                                  ctypes.POINTER(ctypes.c_double),
                                  ctypes.c_double, ctypes.POINTER(GooStep),
                                  _i32, _I32P, _I32P]),
    "mesh_attn_last_error": (ctypes.c_char_p, []),
}


def library_path():
    return os.path.join(_HERE, _LIB_NAME)


def load_library():
    """Load libmesh_attn.so from the package directory (built by
    ``__graft_entry__.build()``).  Raises if it is missing."""
    global _lib
    with _lock:
        if _lib is None:
            path = library_path()
            if not os.path.exists(path):
                raise MeshAttnError("load_library", -1,
                                    f"{path} not built; run the build first")
            lib = ctypes.CDLL(path)
            for name, (res, args) in _SIGNATURES.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
    return _lib


def exported_symbols():
    return sorted(_SIGNATURES)


def mesh_attn_last_error():
    return load_library().mesh_attn_last_error().decode()


def _check(fn, status):
    if status != MA_OK:
        raise MeshAttnError(fn, status, mesh_attn_last_error())


def _idx(lst):
    arr = np.ascontiguousarray(np.asarray(list(lst), dtype=np.int32))
    return arr, arr.ctypes.data_as(_I32P), int(arr.size)


# ---------------------------------------------------------------------------
# Host-only work-list calls
# ---------------------------------------------------------------------------

def mesh_attn_block_shape(head_dim, pass_=0):
    bm, bn = ctypes.c_int32(0), ctypes.c_int32(0)
    load_library().mesh_attn_block_shape(int(head_dim), int(pass_),
                                         ctypes.byref(bm), ctypes.byref(bn))
    return bm.value, bn.value


def mesh_attn_classify(prob, q_idx, kv_idx, bm, bn):
    pr = Problem.make(prob)
    qa, qp, nq = _idx(q_idx)
    ka, kp, nkv = _idx(kv_idx)
    P = pr.partition_len
    nqb = nq * P // bm if bm > 0 else 0
    nkb = nkv * P // bn if bn > 0 else 0
    out = np.zeros((max(nqb, 1), max(nkb, 1)), dtype=np.uint8)
    st = load_library().mesh_attn_classify(
        ctypes.byref(pr), qp, nq, kp, nkv, int(bm), int(bn),
        out.ctypes.data_as(_p))
    _check("mesh_attn_classify", st)
    return out[:nqb, :nkb]


def _worklist(name, prob, q_idx, kv_idx, bm, bn, kv_major):
    lib = load_library()
    pr = Problem.make(prob)
    qa, qp, nq = _idx(q_idx)
    ka, kp, nkv = _idx(kv_idx)
    P = pr.partition_len
    nrows = (nkv * P // bn) if kv_major else (nq * P // bm)
    fn = getattr(lib, name)
    ptr = np.zeros(max(nrows, 0) + 1, dtype=np.int32)
    n = ctypes.c_int64(0)
    st = fn(ctypes.byref(pr), qp, nq, kp, nkv, int(bm), int(bn),
            ptr.ctypes.data_as(_I32P), None, 0, ctypes.byref(n))
    if st not in (MA_OK, MA_ERR_CAPACITY):
        _check(name, st)
    # ma_run_t is five int32 without padding: an [n, 5] int32 array has its
    # layout.
    assert ctypes.sizeof(Run) == 5 * 4
    runs = np.zeros((n.value, 5), dtype=np.int32)
    st = fn(ctypes.byref(pr), qp, nq, kp, nkv, int(bm), int(bn),
            ptr.ctypes.data_as(_I32P),
            runs.ctypes.data_as(ctypes.POINTER(Run)) if n.value else None,
            n.value, ctypes.byref(n))
    _check(name, st)
    return ptr, runs


def mesh_attn_worklist(prob, q_idx, kv_idx, bm, bn):
    """Canonical Q-major run list: ``(qblk_ptr, runs[n, 5])``."""
    return _worklist("mesh_attn_worklist", prob, q_idx, kv_idx, bm, bn, False)


def mesh_attn_worklist_kv_major(prob, q_idx, kv_idx, bm, bn):
    """KV-major mirror: ``(kvblk_ptr, runs[n, 5])``."""
    return _worklist("mesh_attn_worklist_kv_major", prob, q_idx, kv_idx, bm,
                     bn, True)


def mesh_attn_fwd_workspace_size(prob, nq, nkv):
    return int(load_library().mesh_attn_fwd_workspace_size(
        ctypes.byref(Problem.make(prob)), int(nq), int(nkv)))


def mesh_attn_bwd_workspace_size(prob, nq, nkv):
    return int(load_library().mesh_attn_bwd_workspace_size(
        ctypes.byref(Problem.make(prob)), int(nq), int(nkv)))


# ---------------------------------------------------------------------------
# Device calls (torch tensors)
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _stream_ptr(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, name, shape, dtypes):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} dtype {t.dtype} not in {dtypes}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} shape {tuple(t.shape)} != {tuple(shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _dtype_code(t):
    torch = _torch()
    return MA_FP32 if t.dtype == torch.float32 else MA_BF16


def _workspace(nbytes, device, ws, stream=None):
    torch = _torch()
    if ws is None:
        ws = torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)
        if stream is not None:
            ws.record_stream(stream)
    if ws.device.type != "cuda" or not ws.is_contiguous():
        raise ValueError("workspace must be a contiguous GPU tensor")
    return ws, ws.numel() * ws.element_size()


def mesh_attn_tile_fwd(prob, q_idx, kv_idx, q, k, v, o, lse, ws=None,
                       stream=None):
    """O and LSE of the tile.  ``o`` bf16 (final) or float32 (partial)."""
    torch = _torch()
    pr = Problem.make(prob)
    qa, qp, nq = _idx(q_idx)
    ka, kp, nkv = _idx(kv_idx)
    P, hq, hkv, d = (pr.partition_len, pr.num_q_heads, pr.num_kv_heads,
                     pr.head_dim)
    args = [
        _dev(q, "q", (nq * P, hq, d), (torch.bfloat16,)),
        _dev(k, "k", (nkv * P, hkv, d), (torch.bfloat16,)),
        _dev(v, "v", (nkv * P, hkv, d), (torch.bfloat16,)),
        _dev(o, "o", (nq * P, hq, d), (torch.bfloat16, torch.float32)),
    ]
    lp = _dev(lse, "lse", (hq, nq * P), (torch.float32,))
    need = mesh_attn_fwd_workspace_size(pr, nq, nkv)
    ws, wsb = _workspace(need, q.device, ws, stream)
    st = load_library().mesh_attn_tile_fwd(
        ctypes.byref(pr), qp, nq, kp, nkv, *args[:3], args[3], _dtype_code(o),
        lp, ctypes.c_void_p(ws.data_ptr()), wsb, _stream_ptr(stream))
    _check("mesh_attn_tile_fwd", st)
    return o, lse


def mesh_attn_tile_fwd_noalloc(prob, q_idx, kv_idx, q, k, v, o, lse,
                               stream=None):
    """``mesh_attn_tile_fwd`` without a workspace: the library builds the work
    list on the device in its own fixed scratch array and allocates
    nothing."""
    torch = _torch()
    pr = Problem.make(prob)
    qa, qp, nq = _idx(q_idx)
    ka, kp, nkv = _idx(kv_idx)
    P, hq, hkv, d = (pr.partition_len, pr.num_q_heads, pr.num_kv_heads,
                     pr.head_dim)
    args = [
        _dev(q, "q", (nq * P, hq, d), (torch.bfloat16,)),
        _dev(k, "k", (nkv * P, hkv, d), (torch.bfloat16,)),
        _dev(v, "v", (nkv * P, hkv, d), (torch.bfloat16,)),
        _dev(o, "o", (nq * P, hq, d), (torch.bfloat16, torch.float32)),
    ]
    lp = _dev(lse, "lse", (hq, nq * P), (torch.float32,))
    st = load_library().mesh_attn_tile_fwd_noalloc(
        ctypes.byref(pr), qp, nq, kp, nkv, *args[:3], args[3], _dtype_code(o),
        lp, _stream_ptr(stream))
    _check("mesh_attn_tile_fwd_noalloc", st)
    return o, lse


def mesh_attn_lse_merge(o_parts, lse_parts, o_out, lse_out, stream=None):
    """Fold ``o_parts [k, rows, H, d]``, ``lse_parts [k, H, rows]``."""
    torch = _torch()
    if o_parts.dim() != 4:
        raise ValueError("o_parts must be [k, rows, heads, head_dim]")
    kparts, rows, heads, d = (int(x) for x in o_parts.shape)
    a = _dev(o_parts, "o_parts", (kparts, rows, heads, d),
             (torch.bfloat16, torch.float32))
    b = _dev(lse_parts, "lse_parts", (kparts, heads, rows), (torch.float32,))
    c = _dev(o_out, "o_out", (rows, heads, d), (torch.bfloat16, torch.float32))
    e = _dev(lse_out, "lse_out", (heads, rows), (torch.float32,))
    st = load_library().mesh_attn_lse_merge(
        kparts, rows, heads, d, a, _dtype_code(o_parts), b, c,
        _dtype_code(o_out), e, _stream_ptr(stream))
    _check("mesh_attn_lse_merge", st)
    return o_out, lse_out


def mesh_attn_tile_bwd(prob, q_idx, kv_idx, q, k, v, o, d_o, lse, dq, dk, dv,
                       accumulate=0, ws=None, stream=None):
    """dQ, dK, dV (float32) of the tile from the final O and LSE."""
    torch = _torch()
    pr = Problem.make(prob)
    qa, qp, nq = _idx(q_idx)
    ka, kp, nkv = _idx(kv_idx)
    P, hq, hkv, d = (pr.partition_len, pr.num_q_heads, pr.num_kv_heads,
                     pr.head_dim)
    bf, f32 = (torch.bfloat16,), (torch.float32,)
    args = [
        _dev(q, "q", (nq * P, hq, d), bf),
        _dev(k, "k", (nkv * P, hkv, d), bf),
        _dev(v, "v", (nkv * P, hkv, d), bf),
        _dev(o, "o", (nq * P, hq, d), bf),
        _dev(d_o, "d_o", (nq * P, hq, d), bf),
        _dev(lse, "lse", (hq, nq * P), f32),
        _dev(dq, "dq", (nq * P, hq, d), f32),
        _dev(dk, "dk", (nkv * P, hkv, d), f32),
        _dev(dv, "dv", (nkv * P, hkv, d), f32),
    ]
    need = mesh_attn_bwd_workspace_size(pr, nq, nkv)
    ws, wsb = _workspace(need, q.device, ws, stream)
    st = load_library().mesh_attn_tile_bwd(
        ctypes.byref(pr), qp, nq, kp, nkv, *args, int(accumulate),
        ctypes.c_void_p(ws.data_ptr()), wsb, _stream_ptr(stream))
    _check("mesh_attn_tile_bwd", st)
    return dq, dk, dv


# ---------------------------------------------------------------------------
# GOO (Section 3.4): chunk compute tasks and the step planner
# ---------------------------------------------------------------------------

def mesh_attn_chunk_fwd_workspace_size(prob, nq, nkv):
    return int(load_library().mesh_attn_chunk_fwd_workspace_size(
        ctypes.byref(Problem.make(prob)), int(nq), int(nkv)))


def mesh_attn_chunk_fwd(prob, q_idx, kv_idx, chunk, q, k, v, o, lse,
                        accumulate=0, ws=None, stream=None):
    """Compute task C-i-j, ``chunk = (i, k_q, j, k_kv)``: ``q`` holds chunk i
    of every Q partition, ``k, v`` chunk j of every KV partition; ``o``
    (float32) and ``lse`` receive, or with ``accumulate=1`` fold in, the
    chunk pair's partial."""
    torch = _torch()
    pr = Problem.make(prob)
    qa, qp, nq = _idx(q_idx)
    ka, kp, nkv = _idx(kv_idx)
    ch = Chunk(*(int(x) for x in chunk))
    P, hq, hkv, d = (pr.partition_len, pr.num_q_heads, pr.num_kv_heads,
                     pr.head_dim)
    if ch.num_q_chunks < 1 or ch.num_kv_chunks < 1:
        raise ValueError("chunk counts must be >= 1")
    rq, rk = nq * (P // ch.num_q_chunks), nkv * (P // ch.num_kv_chunks)
    bf, f32 = (torch.bfloat16,), (torch.float32,)
    args = [
        _dev(q, "q", (rq, hq, d), bf),
        _dev(k, "k", (rk, hkv, d), bf),
        _dev(v, "v", (rk, hkv, d), bf),
        _dev(o, "o", (rq, hq, d), f32),
        _dev(lse, "lse", (hq, rq), f32),
    ]
    need = mesh_attn_chunk_fwd_workspace_size(pr, nq, nkv)
    ws, wsb = _workspace(need, q.device, ws, stream)
    st = load_library().mesh_attn_chunk_fwd(
        ctypes.byref(pr), qp, nq, kp, nkv, ctypes.byref(ch), *args,
        int(accumulate), ctypes.c_void_p(ws.data_ptr()), wsb,
        _stream_ptr(stream))
    _check("mesh_attn_chunk_fwd", st)
    return o, lse


def mesh_attn_chunk_bwd_workspace_size(prob, nq, nkv):
    return int(load_library().mesh_attn_chunk_bwd_workspace_size(
        ctypes.byref(Problem.make(prob)), int(nq), int(nkv)))


def mesh_attn_chunk_bwd(prob, q_idx, kv_idx, chunk, q, k, v, o, d_o, lse, dq,
                        dk, dv, accumulate=0, ws=None, stream=None):
    """Backward of compute task C-i-j, ``chunk = (i, k_q, j, k_kv)``: chunk
    buffers as in ``mesh_attn_chunk_fwd``, with the final O and LSE of the
    chunk's Q rows; float32 ``dq`` (Q chunk) and ``dk, dv`` (KV chunk)."""
    torch = _torch()
    pr = Problem.make(prob)
    qa, qp, nq = _idx(q_idx)
    ka, kp, nkv = _idx(kv_idx)
    ch = Chunk(*(int(x) for x in chunk))
    P, hq, hkv, d = (pr.partition_len, pr.num_q_heads, pr.num_kv_heads,
                     pr.head_dim)
    if ch.num_q_chunks < 1 or ch.num_kv_chunks < 1:
        raise ValueError("chunk counts must be >= 1")
    rq, rk = nq * (P // ch.num_q_chunks), nkv * (P // ch.num_kv_chunks)
    bf, f32 = (torch.bfloat16,), (torch.float32,)
    args = [
        _dev(q, "q", (rq, hq, d), bf),
        _dev(k, "k", (rk, hkv, d), bf),
        _dev(v, "v", (rk, hkv, d), bf),
        _dev(o, "o", (rq, hq, d), bf),
        _dev(d_o, "d_o", (rq, hq, d), bf),
        _dev(lse, "lse", (hq, rq), f32),
        _dev(dq, "dq", (rq, hq, d), f32),
        _dev(dk, "dk", (rk, hkv, d), f32),
        _dev(dv, "dv", (rk, hkv, d), f32),
    ]
    need = mesh_attn_chunk_bwd_workspace_size(pr, nq, nkv)
    ws, wsb = _workspace(need, q.device, ws, stream)
    st = load_library().mesh_attn_chunk_bwd(
        ctypes.byref(pr), qp, nq, kp, nkv, ctypes.byref(ch), *args,
        int(accumulate), ctypes.c_void_p(ws.data_ptr()), wsb,
        _stream_ptr(stream))
    _check("mesh_attn_chunk_bwd", st)
    return dq, dk, dv


def mesh_attn_goo_plan(k_q, k_kv, t_ag_q, t_ag_kv, t_rs_q, t_c, gamma=1.05):
    """Greedy step schedule of a tile's chunk tasks.  Returns a list of steps
    ``(comm, tasks)``: ``comm`` is ``None`` for a compute-only step, else
    ``(kind, chunk)`` with kind "AG-Q", "AG-KV" or "RS-Q"; ``tasks`` is a list
    of ``(i, j)``."""
    k_q, k_kv = int(k_q), int(k_kv)
    tc = np.ascontiguousarray(np.asarray(t_c, dtype=np.float64))
    if tc.shape != (k_q, k_kv):
        raise ValueError(f"t_c shape {tc.shape} != ({k_q}, {k_kv})")
    max_steps = 2 * k_q + k_kv + k_q * k_kv
    steps = (GooStep * max_steps)()
    tasks = np.zeros((k_q * k_kv, 2), dtype=np.int32)
    n = ctypes.c_int32(0)
    st = load_library().mesh_attn_goo_plan(
        k_q, k_kv, float(t_ag_q), float(t_ag_kv), float(t_rs_q),
        tc.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), float(gamma),
        steps, max_steps, tasks.ctypes.data_as(_I32P), ctypes.byref(n))
    _check("mesh_attn_goo_plan", st)
    out = []
    for s_ in steps[:n.value]:
        comm = (None if s_.comm_kind == MA_GOO_NONE
                else (GOO_KIND_NAMES[s_.comm_kind], int(s_.comm_chunk)))
        out.append((comm, [tuple(int(x) for x in tasks[t])
                           for t in range(s_.first_task,
                                          s_.first_task + s_.num_tasks)]))
    return out

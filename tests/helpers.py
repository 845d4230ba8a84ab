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

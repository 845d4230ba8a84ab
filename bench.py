#!/usr/bin/env python3
"""Benchmark of the single-GPU tile compute of Mesh-Attention on MI355X.

One step runs every stage of the hot path once, on one stream, with inputs
resident in HBM:

  fwd    mesh_attn_tile_fwd on the causal 64K-token tile (16 partitions of
         4096 tokens; Q partitions 4..7 x KV partitions 0..7; 32 heads,
         head_dim 128, bf16): work list, scores, causal mask, online softmax,
         PV, epilogue.
  merge  mesh_attn_lse_merge folding 16 bf16 partials of 4096 rows x 32
         heads x 128 (the reduce-scatter fold of a 16x16 mesh); two copies of
         the partials alternate between steps, so the reads come from HBM.
  bwd    mesh_attn_tile_bwd of the same causal tile (dO from seed 4), using
         the forward's O and LSE.

`value` is the forward tile TFLOP/s: algorithmic FLOPs of the tile
(4 * d * Hq * visible (query, key) pairs) divided by the forward call's mean
duration over the timed steps, measured with HIP events on the launch stream.
`ms_per_step` is the whole step.  Per-stage figures are under `legs` (mean
and median over the timed steps; the forward's also gives the host time of
building the tile's work list, which the library caches and which is outside
the timed steps).
Prints one JSON line on stdout; progress goes to stderr.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr,
          flush=True)


def visible_pairs(cfg):
    """Number of visible (query, key) pairs of a tile (per head)."""
    import numpy as np
    P = cfg.partition_len
    total = 0
    for qp in cfg.q_idx:
        qpos = qp * P + np.arange(P, dtype=np.int64)
        for kp in cfg.kv_idx:
            if not cfg.causal:
                total += P * P
            elif cfg.layout == 1:
                # striped: key row r' visible to query row r iff
                # r' * n + kp <= r * n + qp, i.e. r' <= r (kp <= qp) or
                # r' < r (kp > qp)
                total += P * (P + 1) // 2 - (P if kp > qp else 0)
            else:
                k0 = kp * P
                # keys k0..k0+P-1 visible to query at position x: clamp(x-k0+1)
                total += int(np.clip(qpos - k0 + 1, 0, P).sum())
    return total


def source_digest(names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2512_20968_amd", "csrc", n),
                  "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel, digest):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    ent = data.get(kernel)
    if not ent or ent.get("source_digest") != digest:
        return None
    return ent.get("bytes_per_launch")


def cpu_baseline(cfg, budget_s):
    """Time the float64 oracle on a bounded sample of the forward tile."""
    import numpy as np
    import oracle
    from mesh_inputs import make_qkv, sample_rows
    from threadpoolctl import threadpool_info, threadpool_limits
    cores = len(os.sched_getaffinity(0))
    cores = min(cores, 16)
    q, k, v, _ = make_qkv(cfg)
    qf, kf, vf = (t.float().numpy() for t in (q, k, v))
    rows = sample_rows(cfg, cfg.nq, n_random=448)
    P = cfg.partition_len
    qpos = np.array([cfg.q_idx[r // P] * P + r % P for r in rows])
    # visible keys per sampled row (contiguous partitions, causal)
    kpos = np.concatenate([kp * P + np.arange(P) for kp in cfg.kv_idx])
    vis = np.array([(kpos <= x).sum() if cfg.causal else kpos.size
                    for x in qpos])
    done_heads = 0
    used = cores
    t0 = time.perf_counter()
    with threadpool_limits(limits=cores):
        for h in range(cfg.num_q_heads):
            oracle.tile_forward(cfg.problem(), cfg.q_idx, cfg.kv_idx, qf, kf,
                                vf, rows=rows, heads=[h])
            done_heads += 1
            if time.perf_counter() - t0 > budget_s:
                break
        infos = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if infos:
            used = max(int(i["num_threads"]) for i in infos)
    dt = time.perf_counter() - t0
    flops = 4.0 * cfg.head_dim * done_heads * float(vis.sum())
    rate = flops / dt
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    cpu_model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    full = 4.0 * cfg.head_dim * cfg.num_q_heads * visible_pairs(cfg)
    return {"value": rate / 1e12, "unit": "TFLOP/s", "cores": used,
            "kind": "oracle", "cpu_model": cpu_model,
            "projected_full_tile_s": round(full / rate, 1),
            "sample": (f"float64 oracle forward of {len(rows)} sampled query "
                       f"rows x {done_heads} heads of the {cfg.name} tile "
                       f"({flops / 1e9:.1f} GFLOP algorithmic, {dt:.1f} s)")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--legs", default="fwd,merge,bwd",
                    help="comma list of fwd, merge, bwd, chunks (chunks: the "
                         "forward of the same tile as k_Q x k_KV GOO chunk "
                         "tasks, see --chunks)")
    ap.add_argument("--chunks", default="4x4",
                    help="k_Q x k_KV of the chunks leg")
    ap.add_argument("--workload", default="causal-64k",
                    choices=("causal-64k", "mesh1m-nc-gqa",
                             "mesh1m-causal-outlier", "striped-causal-64k",
                             "striped-mesh1m-causal"),
                    help="forward tile: causal-64k (default), mesh1m-nc-gqa "
                         "(1M-token non-causal GQA 16x16 tile), "
                         "mesh1m-causal-outlier (1M-token causal 16x16 tile "
                         "with outliers), striped-causal-64k, "
                         "striped-mesh1m-causal; the backward leg runs on "
                         "the two 64K tiles only")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle time for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one 1 GiB device-to-device copy (HBM "
                         "counter calibration under rocprofv3 --pmc)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU (asked for "
              f"--gpus {args.gpus}); the multi-GPU mesh is not implemented.",
              file=sys.stderr)
        sys.exit(2)
    legs = [x for x in args.legs.split(",") if x]

    import torch
    import paper_2512_20968_amd as ma
    from mesh_inputs import WORKLOADS, make_grad, make_merge_parts, make_qkv

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = WORKLOADS[args.workload]
    if "bwd" in legs and args.workload not in ("causal-64k",
                                               "striped-causal-64k"):
        legs.remove("bwd")
    prob = cfg.problem()
    P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads, cfg.num_kv_heads,
                     cfg.head_dim)
    rq, rkv = cfg.nq * P, cfg.nkv * P
    log(f"generating inputs ({cfg.name})")
    q, k, v, _ = make_qkv(cfg)
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    del q, k, v
    o = torch.empty((rq, hq, d), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((hq, rq), dtype=torch.float32, device=dev)
    ws_f = torch.empty(ma.mesh_attn_fwd_workspace_size(prob, cfg.nq, cfg.nkv),
                       dtype=torch.uint8, device=dev)
    if "bwd" in legs:
        # dO of the backward workload of this tile (bwd-causal-64k is the
        # backward of causal-64k; the striped tile carries its own seed).
        do = make_grad(WORKLOADS["bwd-causal-64k"]
                       if args.workload == "causal-64k" else cfg).to(dev)
        dq = torch.empty((rq, hq, d), dtype=torch.float32, device=dev)
        dk = torch.empty((rkv, hkv, d), dtype=torch.float32, device=dev)
        dv = torch.empty_like(dk)
        ws_b = torch.empty(ma.mesh_attn_bwd_workspace_size(prob, cfg.nq,
                                                           cfg.nkv),
                           dtype=torch.uint8, device=dev)
    if "chunks" in legs:
        # The buffers the chunk all-gathers would produce (chunk i of every
        # Q partition, chunk j of every KV partition), built before timing.
        kq, kkv = (int(x) for x in args.chunks.lower().split("x"))
        cq, ckv = P // kq, P // kkv
        def gather(t, n_parts, c, i):
            return torch.cat([t[a * P + i * c:a * P + (i + 1) * c]
                              for a in range(n_parts)]).contiguous()
        cqd = [gather(qd, cfg.nq, cq, i) for i in range(kq)]
        ckd = [gather(kd, cfg.nkv, ckv, j) for j in range(kkv)]
        cvd = [gather(vd, cfg.nkv, ckv, j) for j in range(kkv)]
        co = [torch.empty((cfg.nq * cq, hq, d), dtype=torch.float32,
                          device=dev) for _ in range(kq)]
        cl = [torch.empty((hq, cfg.nq * cq), dtype=torch.float32, device=dev)
              for _ in range(kq)]
        ws_c = torch.empty(ma.mesh_attn_chunk_fwd_workspace_size(
            prob, cfg.nq, cfg.nkv), dtype=torch.uint8, device=dev)
    if "merge" in legs:
        mk, mrows, mh, md = 16, 4096, 32, 128
        mo_parts, ml_parts = make_merge_parts(mk, mrows, mh, md, seed=7)
        mo_parts, ml_parts = mo_parts.to(dev), ml_parts.to(dev)
        # Two copies of the partials, used in turn: 545 MB each, more than
        # the 256 MB last-level cache, so every merge reads from HBM even when
        # it runs alone (--legs merge).
        msets = [(mo_parts, ml_parts), (mo_parts.clone(), ml_parts.clone())]
        mo = torch.empty((mrows, mh, md), dtype=torch.bfloat16, device=dev)
        ml = torch.empty((mh, mrows), dtype=torch.float32, device=dev)

    stream = torch.cuda.current_stream()
    step_no = [0]

    def run_step(ev=None):
        if "fwd" in legs:
            if ev: ev["fwd"][0].record(stream)
            ma.mesh_attn_tile_fwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o,
                                  lse, ws=ws_f)
            if ev: ev["fwd"][1].record(stream)
        if "chunks" in legs:
            if ev: ev["chunks"][0].record(stream)
            for i in range(kq):
                for j in range(kkv):
                    ma.mesh_attn_chunk_fwd(prob, cfg.q_idx, cfg.kv_idx,
                                           (i, kq, j, kkv), cqd[i], ckd[j],
                                           cvd[j], co[i], cl[i],
                                           accumulate=int(j > 0), ws=ws_c)
            if ev: ev["chunks"][1].record(stream)
        if "merge" in legs:
            if ev: ev["merge"][0].record(stream)
            ma.mesh_attn_lse_merge(*msets[step_no[0] % 2], mo, ml)
            if ev: ev["merge"][1].record(stream)
        if "bwd" in legs:
            if ev: ev["bwd"][0].record(stream)
            ma.mesh_attn_tile_bwd(prob, cfg.q_idx, cfg.kv_idx, qd, kd, vd, o,
                                  do, lse, dq, dk, dv, ws=ws_b)
            if ev: ev["bwd"][1].record(stream)
        step_no[0] += 1

    if args.calib_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        src.fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration copy: 1073741824 bytes read, 1073741824 written")
        del src, dst

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()
    events = [{n: (torch.cuda.Event(enable_timing=True),
                   torch.cuda.Event(enable_timing=True)) for n in legs}
              for _ in range(args.steps)]
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run_step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    leg_times = {n: sorted(e[n][0].elapsed_time(e[n][1]) for e in events)
                 for n in legs}
    leg_ms = {n: sum(t) / args.steps for n, t in leg_times.items()}
    leg_med = {n: (t[(len(t) - 1) // 2] + t[len(t) // 2]) / 2
               for n, t in leg_times.items()}
    log(f"step {ms_step:.3f} ms; " +
        ", ".join(f"{n} {leg_ms[n]:.3f} ms" for n in legs))

    # Host time of the canonical work list (built once per tile and cached by
    # the library, so it is outside the timed steps).
    bm, bn = ma.mesh_attn_block_shape(d, 0)
    t_wl = time.perf_counter()
    _, wl_runs = ma.mesh_attn_worklist(prob, cfg.q_idx, cfg.kv_idx, bm, bn)
    wl_ms = (time.perf_counter() - t_wl) * 1e3

    pairs = visible_pairs(cfg)
    fwd_flop = 4.0 * d * hq * pairs
    bwd_flop = 10.0 * d * hq * pairs
    out_legs = {}
    roofline = None
    value = None
    if "fwd" in legs:
        tf = fwd_flop / (leg_ms["fwd"] * 1e-3) / 1e12
        value = tf
        dig = source_digest(["tile_fwd.hip", "tile_common.h", "internal.h"])
        roofline = {"bound": "mfma", "achieved": round(tf, 2),
                    "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(tf / PEAK_BF16_TFLOPS, 4),
                    "traffic": load_traffic("tile_fwd", dig),
                    "kernel": "tile_fwd_kernel<128,bf16 out>",
                    "flop_per_launch": fwd_flop}
        out_legs["fwd"] = {"ms": round(leg_ms["fwd"], 4),
                           "ms_median": round(leg_med["fwd"], 4),
                           "tflops": round(tf, 2),
                           "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                           "flop": fwd_flop,
                           "worklist_host_ms": round(wl_ms, 3),
                           "worklist_runs": int(len(wl_runs))}
    if "chunks" in legs:
        tc = fwd_flop / (leg_ms["chunks"] * 1e-3) / 1e12
        out_legs["chunks"] = {"ms": round(leg_ms["chunks"], 4),
                              "ms_median": round(leg_med["chunks"], 4),
                              "tflops": round(tc, 2),
                              "frac_bf16_peak": round(tc / PEAK_BF16_TFLOPS,
                                                      4),
                              "chunks": f"{kq}x{kkv}",
                              "launches": kq * kkv, "flop": fwd_flop}
    if "merge" in legs:
        mbytes = (mk * mrows * mh * (md * 2 + 4) + mrows * mh * (md * 2 + 4))
        gbs = mbytes / (leg_ms["merge"] * 1e-3) / 1e9
        mdig = source_digest(["lse_merge.hip", "internal.h"])
        out_legs["merge"] = {"ms": round(leg_ms["merge"], 4),
                             "ms_median": round(leg_med["merge"], 4),
                             "traffic": load_traffic("lse_merge", mdig),
                             "GB/s": round(gbs, 1),
                             "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4),
                             "bytes": mbytes,
                             "shape": f"k={mk} x {mrows} rows x {mh} heads x "
                                      f"{md}, bf16 in/out"}
    if "bwd" in legs:
        tb = bwd_flop / (leg_ms["bwd"] * 1e-3) / 1e12
        out_legs["bwd"] = {"ms": round(leg_ms["bwd"], 4),
                           "ms_median": round(leg_med["bwd"], 4),
                           "tflops": round(tb, 2),
                           "frac_bf16_peak": round(tb / PEAK_BF16_TFLOPS, 4),
                           "flop": bwd_flop}

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the float64 oracle on host cores (bounded sample)")
        cpu = cpu_baseline(cfg, args.cpu_budget)
        log(f"oracle: {cpu['value'] * 1e3:.3f} GFLOP/s on {cpu['cores']} "
            f"threads")

    line = {
        "metric": "tile attention fwd TFLOP/s on 1 MI355X + % of bf16 MFMA "
                  "peak; merge GB/s",
        "value": round(value, 2) if value is not None else None,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 Q/K/V/dO)",
        "config": {"workload": f"{cfg.name} tile: {cfg.note}; "
                               f"{hq} q heads / {hkv} kv heads, head_dim {d}"
                               f"; step = " + " + ".join(
                                   {"fwd": "tile_fwd", "merge":
                                    "lse_merge(16x4096x32x128)",
                                    "bwd": "tile_bwd",
                                    "chunks": f"{args.chunks} chunk_fwd"}[x]
                                   for x in legs),
                   "legs": legs},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "legs": out_legs,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark of the single-GPU tile compute of Mesh-Attention on MI355X.

One step runs every stage of the hot path, on one stream, with inputs
resident in HBM (all bf16, head_dim 128):

  fwd              mesh_attn_tile_fwd on the headline tile, by default
                   mesh1m-nc-gqa: one GPU's share of a 1M-token, 256-GPU mesh
                   (256 partitions of 4096 tokens, Q partitions 16..31 x KV
                   partitions 32..47, non-causal, 32 query heads on 8 KV
                   heads) -- the largest single-GPU workload.  Work list,
                   scores, online softmax, PV, epilogue.
  fwd_causal64k    the same call on the causal 64K-token tile (16 partitions
                   of 4096, Q 4..7 x KV 0..7, 32 heads): causal mask, skipped
                   blocks, diagonal blocks.
  fwd_mesh1m_causal  the same call on the 1M-token causal tile that straddles
                   the diagonal (Q 24..39 x KV 16..31, x8 outlier rows).
  merge            mesh_attn_lse_merge folding 16 bf16 partials of 4096 rows
                   x 32 heads x 128 (the reduce-scatter fold of a 16x16
                   mesh); two copies of the partials alternate between steps,
                   so the reads come from HBM.
  bwd              mesh_attn_tile_bwd of the causal 64K tile (dO from seed 4)
                   with that tile's forward O and LSE.
  chunks           the headline tile's forward as 4x4 GOO chunk tasks
                   (mesh_attn_chunk_fwd, float32 running partials).
  bwd_striped      (not in the default step) the backward of the striped
                   64K tile (dO from seed 6).
  bwd_gqa          (not in the default step) the backward of the 1M-token
                   non-causal GQA tile (32 query heads on 8 KV heads, dO
                   from seed 8).
  fwd_items64 .. fwd_items512  (not in the default step) the forward on 64,
                   128, 256 or 512 items of equal length (1024 KV blocks
                   each), i.e. a quarter, half, all or twice all of the 256
                   compute units busy: the same work per compute unit at
                   different chip load, which separates the kernel's
                   efficiency in clock cycles from the clock the chip holds.
  bwd_items64 .. bwd_items256  (not in the default step) the backward on
                   64, 128 or 256 dK/dV items of equal length (a quarter,
                   half or all of the compute units for the dK/dV kernel),
                   for the same comparison.

`value` is the headline tile's forward TFLOP/s: algorithmic FLOPs
(4 * d * Hq * visible (query, key) pairs) divided by the forward call's mean
duration over the timed steps, measured with HIP events on the launch stream.
`roofline` is that kernel against the bf16 dense MFMA peak.  `ms_per_step`
is the whole step; every stage's figures are under `legs` (mean and median
over the timed steps).  Prints one JSON line on stdout; progress goes to
stderr.
"""

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

DEFAULT_LEGS = ("fwd", "fwd_causal64k", "fwd_mesh1m_causal", "merge", "bwd",
                "chunks")
ITEM_LEGS = ("fwd_items64", "fwd_items128", "fwd_items256", "fwd_items512")
BWD_ITEM_LEGS = ("bwd_items64", "bwd_items128", "bwd_items256")
FWD_LEGS = ("fwd", "fwd_causal64k", "fwd_mesh1m_causal") + ITEM_LEGS
BWD_LEGS = ("bwd", "bwd_striped", "bwd_gqa") + BWD_ITEM_LEGS
ALL_LEGS = (DEFAULT_LEGS + ("bwd_striped", "bwd_gqa") + ITEM_LEGS +
            BWD_ITEM_LEGS)


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr,
          flush=True)


def positions(cfg, part_ids):
    """Global token positions of a stacked partition buffer (contiguous:
    p * P + r; striped: r * n + p)."""
    import numpy as np
    P = cfg.partition_len
    r = np.arange(P, dtype=np.int64)
    p = np.asarray(part_ids, dtype=np.int64)[:, None]
    pos = r[None, :] * cfg.num_partitions + p if cfg.layout == 1 \
        else p * P + r[None, :]
    return pos.reshape(-1)


def visible_pairs(cfg, q_rows=None):
    """Visible (query, key) pairs of a tile per head, over every query row or
    over the buffer rows ``q_rows``."""
    import numpy as np
    qpos = positions(cfg, cfg.q_idx)
    if q_rows is not None:
        qpos = qpos[np.asarray(q_rows)]
    nk = cfg.nkv * cfg.partition_len
    if not cfg.causal:
        return int(qpos.size) * nk
    kpos = np.sort(positions(cfg, cfg.kv_idx))
    return int(np.searchsorted(kpos, qpos, side="right").sum())


def source_digest(names):
    """Digest of the named kernel sources and of the build script, whose
    compile flags shape the kernels too."""
    h = hashlib.sha256()
    paths = [os.path.join(ROOT, "paper_2512_20968_amd", "csrc", n)
             for n in names]
    paths.append(os.path.join(ROOT, "paper_2512_20968_amd", "build.py"))
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(key, digest):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    ent = data.get(key)
    if not ent or ent.get("source_digest") != digest:
        return None
    return ent.get("bytes_per_launch")


def cpu_baseline(cfg, budget_s):
    """Time the float64 oracle, as it stands, on a bounded sample of the
    headline tile: sampled query rows, one head after another until the
    budget is spent, every core of the affinity set for its BLAS."""
    import oracle
    from mesh_inputs import make_qkv, sample_rows
    from threadpoolctl import threadpool_info, threadpool_limits
    cores = len(os.sched_getaffinity(0))
    q, k, v, _ = make_qkv(cfg)
    qf, kf, vf = (t.float().numpy() for t in (q, k, v))
    rows = sample_rows(cfg, cfg.nq, n_random=64)
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
    flops = 4.0 * cfg.head_dim * done_heads * visible_pairs(cfg, rows)
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
            "affinity_cores": cores,
            "projected_full_tile_s": round(full / rate, 1),
            "sample": (f"float64 oracle forward of {len(rows)} sampled query "
                       f"rows x {done_heads} of {cfg.num_q_heads} heads of "
                       f"the {cfg.name} tile ({flops / 1e9:.1f} GFLOP "
                       f"algorithmic, {dt:.1f} s)")}


class Tile:
    """Device buffers of one forward (and optionally backward) workload."""

    def __init__(self, ma, cfg, dev, with_bwd=False, grad_cfg=None):
        import torch
        from mesh_inputs import make_grad, make_qkv
        self.cfg = cfg
        self.prob = cfg.problem()
        P, hq, hkv, d = (cfg.partition_len, cfg.num_q_heads,
                         cfg.num_kv_heads, cfg.head_dim)
        rq, rkv = cfg.nq * P, cfg.nkv * P
        log(f"generating inputs ({cfg.name})")
        q, k, v, _ = make_qkv(cfg)
        self.q, self.k, self.v = (t.to(dev) for t in (q, k, v))
        del q, k, v
        self.o = torch.empty((rq, hq, d), dtype=torch.bfloat16, device=dev)
        self.lse = torch.empty((hq, rq), dtype=torch.float32, device=dev)
        self.ws = torch.empty(ma.mesh_attn_fwd_workspace_size(
            self.prob, cfg.nq, cfg.nkv), dtype=torch.uint8, device=dev)
        self.flop = 4.0 * d * hq * visible_pairs(cfg)
        if with_bwd:
            self.do = make_grad(grad_cfg or cfg).to(dev)
            self.dq = torch.empty((rq, hq, d), dtype=torch.float32,
                                  device=dev)
            self.dk = torch.empty((rkv, hkv, d), dtype=torch.float32,
                                  device=dev)
            self.dv = torch.empty_like(self.dk)
            self.ws_b = torch.empty(ma.mesh_attn_bwd_workspace_size(
                self.prob, cfg.nq, cfg.nkv), dtype=torch.uint8, device=dev)
            self.bwd_flop = 10.0 * d * hq * visible_pairs(cfg)

    def fwd(self, ma):
        c = self.cfg
        ma.mesh_attn_tile_fwd(self.prob, c.q_idx, c.kv_idx, self.q, self.k,
                              self.v, self.o, self.lse, ws=self.ws)

    def bwd(self, ma):
        c = self.cfg
        ma.mesh_attn_tile_bwd(self.prob, c.q_idx, c.kv_idx, self.q, self.k,
                              self.v, self.o, self.do, self.lse, self.dq,
                              self.dk, self.dv, ws=self.ws_b)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--legs", default=",".join(DEFAULT_LEGS),
                    help="comma list of " + ", ".join(ALL_LEGS))
    ap.add_argument("--chunks", default="4x4",
                    help="k_Q x k_KV of the chunks leg")
    ap.add_argument("--workload", default="mesh1m-nc-gqa",
                    choices=("mesh1m-nc-gqa", "causal-64k",
                             "mesh1m-causal-outlier", "striped-causal-64k",
                             "striped-mesh1m-causal"),
                    help="tile of the headline fwd leg and of the chunks "
                         "leg (default mesh1m-nc-gqa, the largest "
                         "single-GPU tile)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle time for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one 1 GiB device-to-device copy (HBM "
                         "counter calibration under rocprofv3 --pmc)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU (asked for "
              f"--gpus {args.gpus}); it has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    legs = [x for x in args.legs.split(",") if x]
    for x in legs:
        if x not in ALL_LEGS:
            ap.error(f"unknown leg {x}")

    import torch
    import paper_2512_20968_amd as ma
    from mesh_inputs import WORKLOADS, make_merge_parts

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    head_cfg = WORKLOADS[args.workload]
    tiles = {}
    if "fwd" in legs or "chunks" in legs:
        tiles["fwd"] = Tile(ma, head_cfg, dev)
    if "fwd_causal64k" in legs:
        tiles["fwd_causal64k"] = Tile(ma, WORKLOADS["causal-64k"], dev)
    if "fwd_mesh1m_causal" in legs:
        tiles["fwd_mesh1m_causal"] = Tile(
            ma, WORKLOADS["mesh1m-causal-outlier"], dev)
    for name in ITEM_LEGS:
        if name in legs:
            tiles[name] = Tile(ma, WORKLOADS[f"items-{name[9:]}"], dev)
    for name in BWD_ITEM_LEGS:
        if name in legs:
            t = Tile(ma, WORKLOADS[f"bwd-items-{name[9:]}"], dev,
                     with_bwd=True)
            t.fwd(ma)
            tiles[name] = t
    if "bwd" in legs:
        # The backward workload is the backward of the causal 64K tile: same
        # inputs (seed 1), dO from seed 4, O and LSE from its forward, which
        # runs once here, before timing (the fwd_causal64k leg rewrites the
        # same values in its own buffers).
        t = Tile(ma, WORKLOADS["causal-64k"], dev, with_bwd=True,
                 grad_cfg=WORKLOADS["bwd-causal-64k"])
        t.fwd(ma)
        tiles["bwd"] = t
    if "bwd_striped" in legs:
        t = Tile(ma, WORKLOADS["striped-causal-64k"], dev, with_bwd=True)
        t.fwd(ma)
        tiles["bwd_striped"] = t
    if "bwd_gqa" in legs:
        gcfg = dataclasses.replace(WORKLOADS["mesh1m-nc-gqa"], grad_seed=8)
        t = Tile(ma, gcfg, dev, with_bwd=True)
        t.fwd(ma)
        tiles["bwd_gqa"] = t
    if "chunks" in legs:
        # The buffers the chunk all-gathers would produce (chunk i of every
        # Q partition, chunk j of every KV partition), built before timing.
        ht = tiles["fwd"]
        cfg = head_cfg
        P, hq, d = cfg.partition_len, cfg.num_q_heads, cfg.head_dim
        kq, kkv = (int(x) for x in args.chunks.lower().split("x"))
        cq, ckv = P // kq, P // kkv

        def gather(t, n_parts, c, i):
            return torch.cat([t[a * P + i * c:a * P + (i + 1) * c]
                              for a in range(n_parts)]).contiguous()
        cqd = [gather(ht.q, cfg.nq, cq, i) for i in range(kq)]
        ckd = [gather(ht.k, cfg.nkv, ckv, j) for j in range(kkv)]
        cvd = [gather(ht.v, cfg.nkv, ckv, j) for j in range(kkv)]
        co = [torch.empty((cfg.nq * cq, hq, d), dtype=torch.float32,
                          device=dev) for _ in range(kq)]
        cl = [torch.empty((hq, cfg.nq * cq), dtype=torch.float32, device=dev)
              for _ in range(kq)]
        ws_c = torch.empty(ma.mesh_attn_chunk_fwd_workspace_size(
            cfg.problem(), cfg.nq, cfg.nkv), dtype=torch.uint8, device=dev)
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

    def leg(name, ev, fn):
        if ev:
            ev[name][0].record(stream)
        fn()
        if ev:
            ev[name][1].record(stream)

    def run_step(ev=None):
        for name in legs:
            if name in FWD_LEGS:
                leg(name, ev, lambda: tiles[name].fwd(ma))
            elif name in BWD_LEGS:
                leg(name, ev, lambda: tiles[name].bwd(ma))
            elif name == "merge":
                leg(name, ev, lambda: ma.mesh_attn_lse_merge(
                    *msets[step_no[0] % 2], mo, ml))
            elif name == "chunks":
                def chunks():
                    c = head_cfg
                    for i in range(kq):
                        for j in range(kkv):
                            ma.mesh_attn_chunk_fwd(
                                c.problem(), c.q_idx, c.kv_idx,
                                (i, kq, j, kkv), cqd[i], ckd[j], cvd[j],
                                co[i], cl[i], accumulate=int(j > 0), ws=ws_c)
                leg(name, ev, chunks)
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

    fwd_dig = source_digest(["tile_fwd.hip", "tile_common.h", "internal.h"])
    out_legs = {}
    roofline = None
    value = None
    for name in FWD_LEGS:
        if name not in legs:
            continue
        t = tiles[name]
        tf = t.flop / (leg_ms[name] * 1e-3) / 1e12
        # Host time of the tile's canonical work list (built once per tile
        # and cached by the library, so outside the timed steps).
        bm, bn = ma.mesh_attn_block_shape(t.cfg.head_dim, 0)
        t_wl = time.perf_counter()
        _, wl_runs = ma.mesh_attn_worklist(t.prob, t.cfg.q_idx, t.cfg.kv_idx,
                                           bm, bn)
        wl_ms = (time.perf_counter() - t_wl) * 1e3
        out_legs[name] = {"workload": t.cfg.name,
                          "ms": round(leg_ms[name], 4),
                          "ms_median": round(leg_med[name], 4),
                          "tflops": round(tf, 2),
                          "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                          "flop": t.flop,
                          "traffic": load_traffic(f"tile_fwd@{t.cfg.name}",
                                                  fwd_dig),
                          "worklist_host_ms": round(wl_ms, 3),
                          "worklist_runs": int(len(wl_runs))}
        if name in ITEM_LEGS:
            items = int(name[9:])
            busy = min(items, 256)
            out_legs[name]["busy_cus"] = busy
            out_legs[name]["tflops_per_256_busy_cus"] = round(
                tf * 256 / busy, 2)
        if name == "fwd":
            value = tf
            roofline = {"bound": "mfma", "achieved": round(tf, 2),
                        "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(tf / PEAK_BF16_TFLOPS, 4),
                        "traffic": out_legs[name]["traffic"],
                        "kernel": "tile_fwd_kernel<128, bf16 out>",
                        "workload": t.cfg.name,
                        "flop_per_launch": t.flop}
    if "chunks" in legs:
        t = tiles["fwd"]
        tc = t.flop / (leg_ms["chunks"] * 1e-3) / 1e12
        out_legs["chunks"] = {"workload": t.cfg.name,
                              "ms": round(leg_ms["chunks"], 4),
                              "ms_median": round(leg_med["chunks"], 4),
                              "tflops": round(tc, 2),
                              "frac_bf16_peak": round(tc / PEAK_BF16_TFLOPS,
                                                      4),
                              "chunks": f"{kq}x{kkv}",
                              "launches": kq * kkv, "flop": t.flop}
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
    for name in BWD_LEGS:
        if name not in legs:
            continue
        t = tiles[name]
        tb = t.bwd_flop / (leg_ms[name] * 1e-3) / 1e12
        wl = {"bwd": "bwd-causal-64k", "bwd_gqa": "bwd-mesh1m-nc-gqa"}
        out_legs[name] = {"workload": wl.get(name, t.cfg.name),
                          "ms": round(leg_ms[name], 4),
                          "ms_median": round(leg_med[name], 4),
                          "tflops": round(tb, 2),
                          "frac_bf16_peak": round(tb / PEAK_BF16_TFLOPS, 4),
                          "flop": t.bwd_flop}

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the float64 oracle on host cores (bounded sample)")
        cpu = cpu_baseline(head_cfg, args.cpu_budget)
        log(f"oracle: {cpu['value'] * 1e3:.3f} GFLOP/s on {cpu['cores']} "
            f"threads")

    step_desc = {"fwd": f"tile_fwd({head_cfg.name})",
                 "fwd_causal64k": "tile_fwd(causal-64k)",
                 "fwd_mesh1m_causal": "tile_fwd(mesh1m-causal-outlier)",
                 "merge": "lse_merge(16x4096x32x128)",
                 "bwd": "tile_bwd(causal-64k)",
                 "bwd_striped": "tile_bwd(striped-causal-64k)",
                 "bwd_gqa": "tile_bwd(mesh1m-nc-gqa)",
                 "chunks": f"{args.chunks} chunk_fwd({head_cfg.name})"}
    step_desc.update({n: f"tile_fwd(items-{n[9:]})" for n in ITEM_LEGS})
    step_desc.update({n: f"tile_bwd(bwd-items-{n[9:]})"
                      for n in BWD_ITEM_LEGS})
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
        "config": {"workload": f"{head_cfg.name} tile: {head_cfg.note}; "
                               f"{head_cfg.num_q_heads} q heads / "
                               f"{head_cfg.num_kv_heads} kv heads, head_dim "
                               f"{head_cfg.head_dim}",
                   "step": " + ".join(step_desc[x] for x in legs),
                   "legs": legs},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "legs": out_legs,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

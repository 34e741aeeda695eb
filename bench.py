#!/usr/bin/env python3
"""Benchmark of CoverPrune's hot path on one MI355X.

One step = one pass of the hot path over one synthetic scene resident in
HBM: the FST cost and the greedy selection of K tokens over it in one call
(coverprune_prune, whose cost epilogue also writes the greedy's first gains):
CoverPrune's prune latency.  The same two parts as separate calls
(coverprune_fst_cost, then coverprune_sgs_select) are timed beside the step,
with the same result.  The default workload is the 16384-token, 3584-wide bfloat16
scene whose 1 GiB float32 cost matrix stays in HBM (K = 1638).
CoverPrune-Lite (coverprune_lite_select), the alternative method of Sec. 4,
is timed on its own beside the step, on this scene and on its 32768-token
workload.

Prints one JSON line: prune latency in ms per scene, the dominant kernel's
roofline fraction, the dense greedy sweep's HBM fraction, and the CPU oracle
timed on the host for comparison.  Timed beside the step (never inside it):
the local greedy on 64-nearest tables, the device capacity from 16
neighbours, the literal greedy (entropic transport per step), and four
6272-token scenes greedied one by one and in one batched launch.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 matrix peak, TFLOP/s
F32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix peak, TFLOP/s
METRIC = "prune latency ms/scene; FST-cost MFMA % peak; SGS sweep HBM GB/s % peak"


def _args():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="n16384_d3584")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lite-workload", default="lite_n32768_d3584",
                    help="also time CoverPrune-Lite alone on this workload ('' to skip)")
    ap.add_argument("--sgs", choices=("incremental", "dense"), default="incremental",
                    help="form of the greedy inside the timed step (the same greedy; picks can differ "
                         "only between gains within rounding of each other); dense times the two calls "
                         "as the step")
    ap.add_argument("--literal-rounds", type=int, default=50,
                    help="scaling rounds per step of the literal greedy timed beside the step (0 to skip)")
    ap.add_argument("--literal-eps", type=float, default=0.05,
                    help="entropic regularisation of the literal greedy, in cost units")
    ap.add_argument("--batch-scenes", type=int, default=4,
                    help="scenes of the paper's 6272-token shape whose greedies are timed one by one and "
                         "batched (0 to skip)")
    ap.add_argument("--dump-maps", default="",
                    help="write this process's memory map (/proc/self/maps) to this file just before exit, so "
                         "that addresses in a crash report from process teardown name their libraries")
    ap.add_argument("--ceilings", action="store_true",
                    help="only measure the achievable ceilings: a 1 GiB device-to-device copy (also the "
                         "calibration kernel for the HBM byte counters) and a 16384 x 3584 x 16384 bf16 "
                         "torch.matmul")
    return ap.parse_args()


def ceilings():
    """Plain copy and library GEMM on the same device, for the achievable
    fractions of HBM and MFMA peak."""
    import torch

    dev = torch.device("cuda:0")
    src = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)   # 1 GiB
    dst = torch.empty_like(src)
    a = torch.randn(16384, 3584, device=dev, dtype=torch.bfloat16)
    b = torch.randn(3584, 16384, device=dev, dtype=torch.bfloat16)
    out = {}
    for name, fn, work in (("copy_1GiB", lambda: dst.copy_(src), 2.0 * src.numel() * 4),
                           ("matmul_bf16_16384x3584x16384", lambda: a @ b, 2.0 * 16384 * 16384 * 3584)):
        fn()
        torch.cuda.synchronize()
        e0 = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        e1 = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        for i in range(5):
            e0[i].record()
            fn()
            e1[i].record()
        torch.cuda.synchronize()
        ms = min(x.elapsed_time(y) for x, y in zip(e0, e1))
        if name.startswith("copy"):
            out[name] = {"ms": round(ms, 4), "GB/s": round(work / ms / 1e6, 1),
                         "frac_of_peak": round(work / ms / 1e6 / HBM_PEAK_GBS, 4)}
        else:
            out[name] = {"ms": round(ms, 4), "TFLOP/s": round(work / ms / 1e9, 1),
                         "frac_of_peak": round(work / ms / 1e9 / BF16_PEAK_TFLOPS, 4)}
    print(json.dumps({"ceilings": out, "device": torch.cuda.get_device_name(0)}), flush=True)


def traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    rocprofv3 counter summary (FETCH_SIZE + WRITE_SIZE, calibrated against a
    plain copy), or None when there is none or the kernel's source has changed
    since the counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                key, val = line.split(":", 1)
                rec[key.strip()] = val.strip()
    # One source file, or several separated by commas (hashed in that order).
    h = hashlib.sha256()
    for name in rec.get("source", "").split(","):
        src = os.path.join(ROOT, name.strip())
        if not name.strip() or not os.path.isfile(src):
            return None
        with open(src, "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != rec.get("source_sha256"):
        return None
    return float(rec["traffic_bytes_per_launch"])


def _timed(fn, starts, ends, i):
    starts[i].record()
    out = fn()
    ends[i].record()
    return out


def cpu_baseline(scene, lite_h):
    """The oracle, untouched, on the host cores, on a bounded sample of the
    workload, scaled to one scene:
      cost    discrepancies + maxima + FST cost for 256 source rows against all
              targets, scaled by N / 256;
      greedy  2 greedy steps at full N (an N x N float64 cost; the step's work
              does not depend on the values), scaled by K / 2;
      lite    CoverPrune-Lite on the whole scene (not scaled)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import fst, lite, sgs

    n, k = scene.n, scene.k
    F = fst.widen_features(scene.feats, scene.dtype)
    rows = np.arange(min(256, n))
    t0 = time.perf_counter()
    m = (float(fst.feature_discrepancy(F, rows).max()), float(fst.spatial_discrepancy(scene.pos, rows).max()),
         float(fst.temporal_discrepancy(scene.frame, rows).max()))
    fst.fst_cost_ref(F, scene.pos, scene.frame, rows=rows, maxima=m)
    t_cost = (time.perf_counter() - t0) * n / rows.size

    C = np.random.default_rng(0).random((n, n))
    steps = 2
    t0 = time.perf_counter()
    sgs.sgs_ref(C, scene.capacity.astype(np.float64), steps, 3.0)
    t_sgs = (time.perf_counter() - t0) * k / steps
    del C

    t0 = time.perf_counter()
    lite.lite_ref(F, scene.pos, scene.frame, scene.capacity, k, h=lite_h)
    t_lite = time.perf_counter() - t0

    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {
        "value": round((t_cost + t_sgs) * 1e3, 1),
        "unit": "ms/scene",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"FST cost for {rows.size} of {n} source rows (x{n / rows.size:.0f}), "
                   f"{steps} of {k} greedy steps at full N (x{k / steps:.0f}); Lite on the whole scene "
                   f"reported apart in parts_ms; "
                   f"numpy float64, {threads} BLAS threads on {os.cpu_count()} host cpus "
                   f"({platform.processor() or platform.machine()})"),
        "parts_ms": {"fst_cost": round(t_cost * 1e3, 1), "sgs_select": round(t_sgs * 1e3, 1),
                     "lite_select": round(t_lite * 1e3, 1)},
    }


def time_lite(name, seed, reps, dev):
    """CoverPrune-Lite alone on its own workload: HIP-event time per call and
    the feature stream's share of HBM peak (features are read once).  Timed
    with the workload's own capacities (the FST capacity of Eq. 9-10 from
    coverprune_fst_capacity, computed before the timed calls, where the
    workload names it) and with the generator's uniform capacities."""
    import numpy as np
    import torch

    import paper_2608_13226_amd as cp
    from scenes import CONFIGS, make_scene, to_device

    cfg = CONFIGS[name]
    scene = make_scene(cfg, seed)
    t = to_device(scene, dev)
    lib = cp.library()
    dt = cp.CP_BF16 if scene.dtype == "bf16" else cp.CP_F32
    ws = torch.empty(lib.coverprune_lite_workspace(scene.n, scene.dim, scene.k, dt), dtype=torch.uint8, device=dev)
    caps = {cfg.capacity: t["capacity"]}
    cap_ms = None
    if cfg.fst_capacity_nn:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        v, _ = cp.fst_capacity(t["feats"], t["pos"], t["frame"], cfg.fst_capacity_nn)
        e1.record()
        torch.cuda.synchronize()
        cap_ms = e0.elapsed_time(e1)
        caps = {f"fst{cfg.fst_capacity_nn}": v, **caps}
    feat_bytes = float(scene.n) * scene.dim * (2 if scene.dtype == "bf16" else 4)
    runs = {}
    for key, cap in caps.items():
        run = lambda: cp.lite_select(t["feats"], t["pos"], t["frame"], cap, scene.k,
                                     voxel_size=cfg.voxel or 0.25, workspace=ws)
        r = run()
        torch.cuda.synchronize()
        sizes = torch.bincount(r.group.long()).cpu().numpy()
        e0 = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
        e1 = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
        for i in range(reps):
            e0[i].record()
            run()
            e1[i].record()
        torch.cuda.synchronize()
        ms = float(np.mean([a.elapsed_time(b) for a, b in zip(e0, e1)]))
        runs[key] = {"ms_per_scene": round(ms, 4), "group_sizes": [int(sizes.min()), int(sizes.max())],
                     "hbm": {"achieved": round(feat_bytes / (ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                             "unit": "GB/s", "bytes": feat_bytes,
                             "note": "features read once; whole call timed"}}
    first = next(iter(runs))
    return {"workload": name, "n": scene.n, "d": scene.dim, "k": scene.k, "voxel_m": cfg.voxel,
            "capacity": first, "ms_per_scene": runs[first]["ms_per_scene"], "hbm": runs[first]["hbm"],
            "by_capacity": runs, "fst_capacity_ms": None if cap_ms is None else round(cap_ms, 3)}


def main():
    args = _args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the hot path is a single-GPU library "
              "(multi-GPU scaling is one scene per GPU with no communication).", file=sys.stderr)
        sys.exit(2)
    if args.ceilings:
        ceilings()
        return

    import numpy as np
    import torch

    import paper_2608_13226_amd as cp
    from scenes import CONFIGS, make_scene, to_device

    cfg = CONFIGS[args.workload]
    lite_h = cfg.voxel or 0.25
    scene = make_scene(cfg, args.seed)
    n, d, k = scene.n, scene.dim, scene.k
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t = to_device(scene, dev)
    lib = cp.library()
    dt = cp.CP_BF16 if scene.dtype == "bf16" else cp.CP_F32

    # Every buffer is allocated before timing.
    cost = torch.empty((n, n), dtype=torch.float32, device=dev)
    maxima = torch.empty(3, dtype=torch.float32, device=dev)
    ws_f = torch.empty(lib.coverprune_fst_cost_workspace(n, d, dt), dtype=torch.uint8, device=dev)
    ws_p = torch.empty(lib.coverprune_prune_workspace(n, d, k, dt), dtype=torch.uint8, device=dev)
    ws_s = torch.empty(max(lib.coverprune_sgs_workspace(n, k, f) for f in
                           (cp.CP_SGS_DENSE, cp.CP_SGS_INCREMENTAL, cp.CP_SGS_INCREMENTAL | cp.CP_SGS_COMPACT)),
                       dtype=torch.uint8, device=dev)
    ws_l = torch.empty(lib.coverprune_lite_workspace(n, d, k, dt), dtype=torch.uint8, device=dev)

    run_f = lambda: cp.fst_cost(t["feats"], t["pos"], t["frame"], out=cost, maxima=maxima, workspace=ws_f)
    run_s = lambda: cp.sgs_select(cost, t["capacity"], k, workspace=ws_s, incremental=args.sgs == "incremental")
    fused = args.sgs == "incremental"

    def step(i=None, ev=None):
        if fused:
            run = lambda: cp.prune(t["feats"], t["pos"], t["frame"], t["capacity"], k, out=cost, maxima=maxima,
                                   workspace=ws_p)[2]
            return run() if ev is None else _timed(run, ev["p0"], ev["p1"], i)
        if ev is None:
            run_f()
            return run_s()
        _timed(run_f, ev["f0"], ev["f1"], i)
        return _timed(run_s, ev["s0"], ev["s1"], i)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    K = args.steps
    ev = {key: [torch.cuda.Event(enable_timing=True) for _ in range(K)]
          for key in ("p0", "p1", "f0", "f1", "s0", "s1")}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        r = step(i, ev)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / K

    def avg(a, b):
        return float(np.mean([ev[a][i].elapsed_time(ev[b][i]) for i in range(K)]))

    # The step's two parts as separate calls, timed beside the step (the
    # cost's epilogue and the greedy's own first pass instead of the fused
    # epilogue): the same cost and picks.
    p_ms = avg("p0", "p1") if fused else None
    if fused:
        sel_step = r.selected.clone()
        for i in range(K):
            _timed(run_f, ev["f0"], ev["f1"], i)
            rs = _timed(run_s, ev["s0"], ev["s1"], i)
        torch.cuda.synchronize()
        assert torch.equal(rs.selected, sel_step), "coverprune_prune and the two calls picked differently"
    f_ms, s_ms = avg("f0", "f1"), avg("s0", "s1")

    # CoverPrune-Lite on the same scene, outside the step (an alternative to
    # the cost and greedy, not a part of them).
    run_l = lambda: cp.lite_select(t["feats"], t["pos"], t["frame"], t["capacity"], k,
                                   voxel_size=lite_h, workspace=ws_l)
    run_l()
    torch.cuda.synchronize()
    l0 = [torch.cuda.Event(enable_timing=True) for _ in range(max(K, 5))]
    l1 = [torch.cuda.Event(enable_timing=True) for _ in range(max(K, 5))]
    for i in range(len(l0)):
        _timed(run_l, l0, l1, i)
    torch.cuda.synchronize()
    l_ms = float(np.mean([a.elapsed_time(b) for a, b in zip(l0, l1)]))

    sel = r.selected.cpu().numpy()
    assert len(set(sel.tolist())) == k, "greedy returned repeated tokens"

    # The dense sweep, timed on its own outside the step: its HBM fraction is
    # the greedy's streaming figure.  Algorithmic bytes per launch: the N x N
    # float32 cost read once per step, plus the per-target vectors (capacity
    # and best cost read, best cost written).
    def time_sgs(incremental, reps, compact=False):
        e0 = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
        e1 = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
        out = None
        for i in range(reps):
            e0[i].record()
            out = cp.sgs_select(cost, t["capacity"], k, workspace=ws_s, incremental=incremental, compact=compact)
            e1[i].record()
        torch.cuda.synchronize()
        return float(np.mean([x.elapsed_time(y) for x, y in zip(e0, e1)])), out

    dense_bytes = k * (4.0 * n * n + 12.0 * n)
    if args.sgs == "dense":
        dense_ms, rd = s_ms, r
    else:
        dense_ms, rd = time_sgs(False, 1)
    dense_gbs = dense_bytes / (dense_ms * 1e-3) / 1e9
    dense = {"kernel": "sgs_dense_kernel", "ms": round(dense_ms, 3), "bound": "hbm",
             "achieved": round(dense_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
             "frac": round(dense_gbs / HBM_PEAK_GBS, 4), "bytes": dense_bytes,
             "traffic": traffic("sgs_dense_kernel", cfg.name)}
    dsel = rd.selected.cpu().numpy()
    same = bool(np.array_equal(dsel, sel))
    diverge = np.nonzero(dsel != sel)[0]
    first_diff = int(diverge[0]) if diverge.size else None

    # Incremental form: algorithmic bytes are the step-0 pass over the whole
    # cost, one cost element per target per step (the pick's column), and one
    # row of N costs per target whose best cost the pick lowers.  The number of
    # such (step, target) pairs is replayed on the host from the cost and the
    # picks, outside the timed region.  The transposed copy that the rows
    # schedule writes in its step-0 pass and the candidate lists of its later
    # steps are not counted.  The unit is the whole sgs_select call (its
    # kernels run back to back on one stream: slot clearing, scale, first
    # pass, the early kernel while steps lower many targets, the rows kernel
    # to step 128, list build, list kernel), so one pair of events brackets
    # it; inside coverprune_prune the same kernels run without the first
    # pass.  The compact schedule (changes exchanged
    # between blocks, no copy) is timed beside it.
    compact = None
    if args.sgs == "incremental":
        c_ms, rc = time_sgs(True, 1, compact=True)
        compact = {"ms": round(c_ms, 3), "us_per_greedy_step": round(c_ms * 1e3 / k, 2),
                   "same_picks": bool(np.array_equal(rc.selected.cpu().numpy(), sel))}
        C = cost.cpu().numpy()                     # target-major: C[j, s]
        b = np.full(n, np.float32(3.0), np.float32)       # c0: sgs_select's default, the sum of the unit weights
        changed = 0
        for tt in sel:
            col = C[:, int(tt)]
            hit = col < b
            changed += int(hit.sum())
            b = np.where(hit, col, b)
        del C
        sgs_bytes = 4.0 * n * n + 4.0 * n * k + 4.0 * n * changed
        sgs_gbs = sgs_bytes / (s_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(sgs_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(sgs_gbs / HBM_PEAK_GBS, 4), "traffic": traffic("sgs_select", cfg.name),
                    "kernel": "sgs_select (inc_first_pass_kernel, sgs_early_kernel, sgs_rows_kernel, "
                              "list_build_kernel, sgs_list_kernel)",
                    "bytes_per_launch": sgs_bytes, "ms_per_launch": round(s_ms, 3),
                    "changed_targets": changed, "us_per_greedy_step": round(s_ms * 1e3 / k, 2)}
    else:
        roofline = {key: dense[key] for key in ("bound", "achieved", "peak", "unit", "frac", "traffic", "kernel")}
        roofline.update({"bytes_per_launch": dense_bytes, "ms_per_launch": round(dense_ms, 3)})

    # The latency floor of a greedy step on this device: the candidate
    # exchange alone, and followed by the dependent read of the row the
    # winner names (coverprune_step_floor: the greedy's launch shape, slots,
    # waits and loads, nothing else), over the cost's rows.  A step of the
    # rows schedule does both (or only the read, when its winner was
    # predicted), then applies the targets the pick improves.
    ws_floor = torch.empty(lib.coverprune_step_floor_workspace(), dtype=torch.uint8, device=dev)
    floor_rounds = 4096

    def floor_us(read_rows):
        cp.step_floor(cost, 64, read_rows=read_rows, workspace=ws_floor)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        cp.step_floor(cost, floor_rounds, read_rows=read_rows, workspace=ws_floor)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / floor_rounds

    exch_us, step_floor_us = floor_us(False), floor_us(True)
    roofline["latency_floor"] = {
        "exchange_us": round(exch_us, 3), "exchange_and_row_read_us": round(step_floor_us, 3),
        "greedy_us_per_step": round(s_ms * 1e3 / k, 3),
        "greedy_over_floor": round(s_ms * 1e3 / k / step_floor_us, 3), "rounds": floor_rounds,
        "note": "coverprune_step_floor: rounds of the greedy's candidate exchange (+ the dependent read of the "
                "winner's 64 KB row); greedy_us_per_step is the whole sgs_select call over K, whose steps "
                "after the 128th skip the exchange when the winner is predicted"}

    # Local greedy (Eq. 13) on the same cost: the g-nearest tables, then the
    # greedy with gains over each candidate's table row.  The paper leaves g
    # open; 64 neighbours per token is the setting timed here.
    local = None
    if n <= 16384:
        g_loc = 64
        nbr = torch.empty((n, g_loc), dtype=torch.int32, device=dev)
        ws_loc = torch.empty(lib.coverprune_sgs_local_workspace(n, k), dtype=torch.uint8, device=dev)
        reps = 3
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3 * reps)]
        for i in range(reps):
            e[3 * i].record()
            cp.knn(t["pos"], g_loc, out=nbr)
            e[3 * i + 1].record()
            rl = cp.sgs_local_select(cost, t["capacity"], nbr, k, workspace=ws_loc)
            e[3 * i + 2].record()
        torch.cuda.synchronize()
        knn_ms = float(np.mean([e[3 * i].elapsed_time(e[3 * i + 1]) for i in range(reps)]))
        loc_ms = float(np.mean([e[3 * i + 1].elapsed_time(e[3 * i + 2]) for i in range(reps)]))
        lsel = rl.selected.cpu().numpy()
        assert len(set(lsel.tolist())) == k, "local greedy returned repeated tokens"
        local = {"g": g_loc, "knn_ms": round(knn_ms, 3), "sgs_local_ms": round(loc_ms, 3),
                 "us_per_greedy_step": round(loc_ms * 1e3 / k, 2),
                 "objective": float(rl.objective[-1].item()),
                 "dense_objective": float(r.objective[-1].item()),
                 "picks_shared_with_dense": int(len(set(lsel.tolist()) & set(sel.tolist())))}

    # FST capacity (Eq. 9-10) from 16 neighbours per token, timed on its own:
    # the workload's capacities are an input of the step.
    cap = None
    if n <= 16384:
        n_nb = 16
        ws_c = torch.empty(lib.coverprune_fst_capacity_workspace(n, n_nb), dtype=torch.uint8, device=dev)
        v_out = torch.empty(n, dtype=torch.float32, device=dev)
        r_out = torch.empty(n, dtype=torch.float64, device=dev)
        reps = 3
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
        for i in range(reps):
            e[2 * i].record()
            cp.fst_capacity(t["feats"], t["pos"], t["frame"], n_nb, out=v_out, score=r_out, workspace=ws_c)
            e[2 * i + 1].record()
        torch.cuda.synchronize()
        cap_ms = float(np.mean([e[2 * i].elapsed_time(e[2 * i + 1]) for i in range(reps)]))
        # Gathered feature rows: one neighbour row per scored pair.
        gather = float(n) * n_nb * d * (2 if scene.dtype == "bf16" else 4)
        cap = {"n_nb": n_nb, "ms": round(cap_ms, 3), "gathered_row_bytes": gather,
               "gathered_gbs": round(gather / (cap_ms * 1e-3) / 1e9, 1)}

    # The greedy with each step's transport solved as written (Eq. 11-15),
    # timed once on the same cost: its picks against the timed greedy's, and
    # both sets priced by the same final transport solve.  Algorithmic bytes:
    # per step l, every scaling round reads the n x l float64 matrix once and
    # the score reads the cost once.
    lit = None
    if args.literal_rounds > 0 and k <= 4096:
        rounds, eps = args.literal_rounds, args.literal_eps
        ws_lit = torch.empty(lib.coverprune_sgs_literal_workspace(n, k), dtype=torch.uint8, device=dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        rl = cp.sgs_literal_select(cost, t["capacity"], k, epsilon=eps, rounds=rounds, workspace=ws_lit)
        e1.record()
        torch.cuda.synchronize()
        lit_ms = e0.elapsed_time(e1)
        hot = cp.sgs_literal_select(cost, t["capacity"], k, epsilon=eps, rounds=rounds, follow=r.selected,
                                    steps=False, workspace=ws_lit)
        torch.cuda.synchronize()
        lsel = rl.selected.cpu().numpy()
        lit_bytes = sum(rounds * 8.0 * n * l + 4.0 * n * n for l in range(k)) + rounds * 8.0 * n * k
        lit = {"eps": eps, "rounds": rounds, "ms": round(lit_ms, 1),
               "us_per_greedy_step": round(lit_ms * 1e3 / k, 1),
               "achieved_gbs": round(lit_bytes / (lit_ms * 1e-3) / 1e9, 1), "bytes": lit_bytes,
               "picks_shared_with_step": int(len(set(lsel.tolist()) & set(sel.tolist()))),
               "transport_cost_literal": float(rl.objective[0].item()),
               "transport_cost_step_picks": float(hot.objective[0].item())}
        del ws_lit

    # Serving shape: several scenes of the paper's 32 x 196 = 6272 tokens,
    # K = 628, pruned before their prefills.  The greedies one after another
    # against one batched launch (costs from the FST kernel, made beforehand).
    batch = None
    if args.batch_scenes > 0:
        bcfg = CONFIGS["paper_n6272_d3584"]
        bcosts, bcaps, bks = [], [], []
        for i in range(args.batch_scenes):
            bs = make_scene(bcfg, args.seed + 1 + i)
            bt = to_device(bs, dev)
            c, _ = cp.fst_cost(bt["feats"], bt["pos"], bt["frame"])
            bcosts.append(c)
            bcaps.append(bt["capacity"])
            bks.append(bs.k)
            del bt
        ws_b = torch.empty(max(lib.coverprune_sgs_workspace(int(c.shape[0]), kk, cp.CP_SGS_INCREMENTAL)
                               for c, kk in zip(bcosts, bks)), dtype=torch.uint8, device=dev)
        ws_bb = torch.empty(lib.coverprune_sgs_batch_workspace(
            (cp._SgsScene * len(bks))(*[cp._SgsScene(0, 0, int(c.shape[0]), kk, 3.0, 0, 0, 0, 0)
                                        for c, kk in zip(bcosts, bks)]), len(bks), cp.CP_SGS_INCREMENTAL),
                            dtype=torch.uint8, device=dev)
        for _ in range(2):                      # warm-up of both forms
            one = [cp.sgs_select(c, v, kk, workspace=ws_b, incremental=True).selected
                   for c, v, kk in zip(bcosts, bcaps, bks)]
            many = cp.sgs_select_batch(bcosts, bcaps, bks, workspace=ws_bb)
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record()
        one = [cp.sgs_select(c, v, kk, workspace=ws_b, incremental=True).selected.clone()
               for c, v, kk in zip(bcosts, bcaps, bks)]
        e[1].record()
        many = cp.sgs_select_batch(bcosts, bcaps, bks, workspace=ws_bb)
        e[2].record()
        torch.cuda.synchronize()
        seq_ms, bat_ms = e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2])
        same_b = all(bool(torch.equal(a, b.selected)) for a, b in zip(one, many))
        batch = {"workload": bcfg.name, "scenes": len(bks), "n": int(bcosts[0].shape[0]), "k": bks[0],
                 "sequential_ms": round(seq_ms, 3), "batched_ms": round(bat_ms, 3),
                 "scenes_per_s_sequential": round(len(bks) / (seq_ms * 1e-3), 1),
                 "scenes_per_s_batched": round(len(bks) / (bat_ms * 1e-3), 1), "same_picks": same_b}
        del bcosts, bcaps, ws_b, ws_bb

    # FST cost: symmetric Gram needs N (N + 1) D flops; the whole call (prep,
    # Gram, epilogue) is timed, so this fraction is a lower bound for the Gram.
    gram_flops = float(n) * (n + 1) * d
    peak = BF16_PEAK_TFLOPS if scene.dtype == "bf16" else F32_MFMA_PEAK_TFLOPS
    f_tflops = gram_flops / (f_ms * 1e-3) / 1e12
    lite_bytes = float(n) * d * (2 if scene.dtype == "bf16" else 4) + 64.0 * n
    out = {
        "metric": METRIC,
        "value": round(ms_per_step, 3),
        "unit": "ms/scene",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": scene.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "n": n, "d": d, "k": k, "features": scene.dtype,
                   "lite_voxel_m": lite_h, "seed": args.seed, "sgs": args.sgs},
        "roofline": roofline,
        "breakdown": {
            "prune_ms": round(p_ms, 3) if fused else None,
            "fst_cost_ms": round(f_ms, 3),
            "sgs_select_ms": round(s_ms, 3),
            "sgs_dense_sweep": dense,
            "sgs_dense_same_picks": same,
            "sgs_dense_first_different_step": first_diff,
            "sgs_compact_schedule": compact,
            "sgs_local": local,
            "fst_capacity": cap,
            "sgs_literal": lit,
            "sgs_batch": batch,
            "two_calls_ms_per_scene": round(f_ms + s_ms, 3),
            "lite_select_ms_same_scene": round(l_ms, 3),
            "fst_cost_mfma": {"bound": "mfma", "achieved": round(f_tflops, 1), "peak": peak,
                              "unit": "TFLOP/s", "frac": round(f_tflops / peak, 4),
                              "flops": gram_flops, "note": "whole fst_cost call timed"},
            "lite_hbm": {"achieved": round(lite_bytes / (l_ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "bytes": lite_bytes},
        },
        "device": torch.cuda.get_device_name(0),
    }
    if args.lite_workload:
        out["lite_workload"] = time_lite(args.lite_workload, args.seed, max(K, 5), dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(scene, lite_h)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    _a = _args()
    if _a.dump_maps:
        import atexit

        def _dump_maps(path=_a.dump_maps):
            with open("/proc/self/maps") as src, open(path, "w") as dst:
                dst.write(src.read())

        atexit.register(_dump_maps)
    main()
    # Leave no device work or memory of ours to process teardown (the HIP
    # runtime's and a profiler's exit handlers): every tensor of main() is
    # gone once it returns, and torch's cache goes back to the runtime.
    if "torch" in sys.modules:
        import gc

        import torch
        if torch.cuda.is_initialized():
            torch.cuda.synchronize()
            gc.collect()
            torch.cuda.empty_cache()
            torch.cuda.synchronize()
    sys.stdout.flush()
    sys.stderr.flush()

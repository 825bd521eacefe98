#!/usr/bin/env python3
"""Benchmark of the generalized-sparse-convolution hot path on one MI355X.

One step = one pass of the whole hot path over a workload, inputs already
resident in HBM: coordinate hash table, output coordinates (strided layers),
kernel maps, block plans (where they pay: a pass with and one without are
timed first, ``--plan auto``), convolution forward, input gradient and weight
gradient.

    python bench.py [--steps K] [--warmup W]            # all five workloads
    python bench.py --workload N [...]                  # one workload

By default every workload (0..4) is timed in turn and the JSON line's headline
(``value``, ``roofline``) is workload 4, the indoor scenes at 2 cm with 256
channels in bfloat16, the largest of them by arithmetic; the others are
reported under ``configs`` with their stage times, their forward+backward time
against its roofline target and the roofline fraction of their forward
kernel.  ``value`` is voxels (input rows) per second of whole steps; the
conv-only rate, the effective GFLOP/s and the kernel-map build time are
reported beside it.  ``roofline`` covers the dominant kernel (the forward
gather-MFMA-scatter), timed with HIP events on the stream it runs on.
``cpu_baseline`` times the CPU oracle (test infrastructure, never tuned) on a
bounded sample of the headline workload, stage by stage, on this host's cores.
"""
from __future__ import annotations

import argparse
import contextlib
import gc
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
MFMA_FP32_PEAK_TFLOPS = 157.3
METRIC = "sparse-conv fwd+bwd voxels/s & effective GFLOP/s; kernel-map build ms"


@contextlib.contextmanager
def no_gc():
    """No garbage-collection pass inside a timed region: one over the
    process's objects stalls the host for tens of ms, and the GPU then idles
    between the kernels it was to be given."""
    gc.collect()
    gc.disable()
    try:
        yield
    finally:
        gc.enable()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def fwd_bytes(n_pairs, n_out, ci, co, K, s):
    """Gather model: one input row and one index pair per kernel-map pair,
    every output row written once, the weights read once."""
    return n_pairs * (s * ci + 8) + n_out * s * co + K * ci * co * s


def measured_peaks(torch):
    """The box's own ceilings, for context beside the published ones: a device
    to device copy of 1 GiB (read + write bytes per second) and a 8192^3 bf16
    matrix product (hipBLASLt through torch), each the best of a few runs."""
    src = torch.empty(2**28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    a = torch.randn(8192, 8192, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(8192, 8192, device="cuda", dtype=torch.bfloat16)
    best_copy, best_mm = float("inf"), float("inf")
    for _ in range(5):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.mm(a, b)
        e2.record()
        torch.cuda.synchronize()
        best_copy = min(best_copy, e0.elapsed_time(e1))
        best_mm = min(best_mm, e1.elapsed_time(e2))
    del src, dst, a, b
    return {"copy_GBs": round(2 * 2**30 / (best_copy * 1e-3) / 1e9, 1),
            "bf16_gemm_TFLOPs": round(2 * 8192**3 / (best_mm * 1e-3) / 1e12, 1)}


def stage_stats(samples):
    """Median, 10th and 90th percentiles of per-step stage times (ms)."""
    import numpy as np
    return {q: {k: round(float(np.percentile(v, pct)), 4) for k, v in samples.items()}
            for q, pct in (("median", 50), ("p10", 10), ("p90", 90))}


def forward_kernel(gsc, dtype: str, ci: int, co: int, K: int, planned: bool, epilogue: bool = False) -> str:
    """Name of the kernel gsc_sparse_conv_fwd launches for this layer (the
    library's dispatch: block engine on a plan, else the map's row form)."""
    dt = gsc.GSC_BF16 if dtype == "bf16" else gsc.GSC_F32
    ep = "true" if epilogue else "false"
    if planned and gsc.gsc_conv_block_engine(dt, ci, co, K):
        if dtype == "bf16":
            if K <= 29:   # the tile engine (16 blocks by all output columns per workgroup)
                return f"k_conv_tile_bf16<{ci}, {co}, gsc::WIdentity, {ep}>"
            return f"k_conv_blk_bf16<{ci}, {128 if co == 256 else co}, gsc::WIdentity, {ep}>"
        return f"k_conv_blk_f32<{ci}, {co}, false, {ep}, false>"
    if dtype == "bf16":
        if ci in (128, 256) and co in (128, 256):
            return f"k_conv_bf16_dma<{ci}, {co}, gsc::WIdentity>"
        return "k_conv_bf16"
    return f"k_conv_f32<{ci}, {co}, false, gsc::WIdentity>"


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of ``kernel`` on ``workload`` from the committed
    counter summary (profiles/hbm_traffic_*), or None when there is none or
    the kernel's source has changed since the counters were taken."""
    import glob
    import hashlib
    for f in glob.glob(os.path.join(ROOT, "profiles", "hbm_traffic_*.md")):
        text = open(f).read()
        fields = dict(re.findall(r"^(kernel|source|source_sha256|traffic_bytes_per_launch): (.+)$", text, re.M))
        if fields.get("kernel") != kernel or workload not in os.path.basename(f).replace("_cube3", ""):
            continue
        src = os.path.join(ROOT, fields["source"])
        if not os.path.exists(src) or hashlib.sha256(open(src, "rb").read()).hexdigest() != fields["source_sha256"]:
            return None
        return int(fields["traffic_bytes_per_launch"])
    return None


def _blas_threads():
    """Cores this process may run on and the BLAS thread pools numpy uses
    (limited to those cores)."""
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threadpool_limits(cores)
        blas = [(i.get("internal_api"), i.get("num_threads")) for i in threadpool_info()]
    except Exception:
        blas = []
    threads = max([t for _, t in blas if t] or [1])
    return cores, min(threads, cores), blas


def _oracle_pass(O, coords, layers, D, X, dY):
    """One pass of the oracle over a sparse tensor, stage by stage (seconds):
    coordinate map, output coordinates (strided layers), kernel maps, forward,
    backward (the same stages the GPU pass times)."""
    import numpy as np
    t = {}
    t0 = time.perf_counter()
    O.coordinate_map(coords)
    t["coords"] = time.perf_counter() - t0
    X = X.astype(np.float64)
    dY = dY.astype(np.float64)
    kinds = [L.kind for L in layers]
    if kinds == ["subm"]:
        L = layers[0]
        t0 = time.perf_counter()
        m = O.kernel_map(coords, coords, O.region(L.region, L.ksize, D))
        t["map"] = time.perf_counter() - t0
        t0 = time.perf_counter()
        O.conv_forward(X, L.W, m, len(coords))
        t["fwd"] = time.perf_counter() - t0
        t0 = time.perf_counter()
        O.conv_backward(X, L.W, dY, m)
        t["bwd"] = time.perf_counter() - t0
        return t
    L0, L1 = layers
    t0 = time.perf_counter()
    out = O.output_coordinates(coords, L0.stride)
    t["out_coords"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    kd = O.kernel_map(coords, out, O.region(L0.region, L0.ksize, D))
    td = O.transposed_map(kd)
    t["map"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    Y1 = O.conv_forward(X, L0.W, kd, len(out))
    O.conv_forward(Y1, L1.W, td, len(coords))
    t["fwd"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    dY1, _ = O.conv_backward(Y1, L1.W, dY, td)
    O.conv_backward(X, L0.W, dY1, kd)
    t["bwd"] = time.perf_counter() - t0
    return t


def cpu_baseline(wl, max_rows: int = 400000, reps: int = 1):
    """Time the CPU oracle on this host: one pass over the first ``max_rows``
    coordinate rows of the workload in (b, x, y, z[, t]) order (a slab of the
    first scene, taken as a sparse tensor of its own), or over all of it when
    it is smaller; the median of ``reps`` passes.  Per-stage milliseconds and
    voxels per second of the whole pass."""
    import numpy as np
    import oracle.gsc_oracle as O
    cores, threads, blas = _blas_threads()
    n = min(wl.n, max_rows)
    order = np.lexsort(wl.coords.T[::-1])[:n]
    order.sort()   # rows keep their relative order
    coords = wl.coords[order]
    X, dY = wl.X[order], wl.dY[order]
    runs = [_oracle_pass(O, coords, wl.layers, wl.D, X, dY) for _ in range(reps)]
    import statistics
    stages = {k: statistics.median(r[k] for r in runs) for k in runs[0]}
    total = statistics.median(sum(r.values()) for r in runs)
    if n == wl.n:
        sample = f"all {n} voxels of {wl.name}"
    else:
        sample = (f"the first {n} of the {wl.n} voxels of {wl.name} in (b, x, y, z) order (a slab of the first "
                  f"scene, x <= {int(coords[:, 1].max())}), as a sparse tensor of its own")
    return {"value": n / total, "unit": "voxels/s", "cores": threads, "kind": "oracle",
            "sample": f"{sample}; {'median of ' + str(reps) + ' passes' if reps > 1 else 'one pass'}: "
                      f"dict coordinate and kernel maps (single-threaded Python) + float64 numpy matmuls "
                      f"({threads} BLAS threads on {cores} cores); {total:.1f} s",
            "stage_ms": {k: round(v * 1e3, 1) for k, v in stages.items()},
            "seconds": round(total, 3), "voxels": n, "affinity_cores": cores, "blas": blas}


def pool_bytes(n_pairs, n_out, C, K, mode):
    """Forward pooling pass: each output's K neighbour entries, one input row
    per pair, the output row, its argmax row (max) and its count."""
    return n_out * K * 4 + n_pairs * C * 4 + n_out * C * 4 * (2 if mode == "max" else 1) + n_out * 4


def pool_cpu_baseline(mode: str):
    """The oracle's pooling pass (map, forward, backward) over the same scene
    (about 12 s of single-threaded Python)."""
    import numpy as np
    import oracle.gsc_oracle as O
    from paper_1904_08755_amd import workloads as WL
    wl = WL.make_workload(1)
    t0 = time.perf_counter()
    out = O.output_coordinates(wl.coords, 2)
    maps = O.kernel_map(wl.coords, out, O.region("cube", 2, wl.D))
    X = wl.X.astype(np.float64)
    Y, arg, N = O.pool_forward(X, maps, len(out), mode)
    O.pool_backward(np.ones_like(Y), maps, wl.n, mode, arg, N)
    t = time.perf_counter() - t0
    return {"value": wl.n / t, "unit": "voxels/s", "cores": 1, "kind": "oracle",
            "sample": f"one full pooling pass (map, forward, backward) of the scene ({wl.n} voxels), "
                      f"single-threaded Python; {t:.1f} s", "seconds": t}


def run_pool(args):
    """Pooling pass over workload 1's scene: table, stride-2 output coordinates,
    the 2^3 window's map and its role-reversed map (dense forms), pooling
    forward and backward.  One JSON line, like the convolution pass."""
    import numpy as np
    import torch

    from paper_1904_08755_amd import gsc, regions
    from paper_1904_08755_amd import workloads as WL

    wl = WL.make_workload(1)
    coords = torch.from_numpy(wl.coords).cuda()
    X = torch.from_numpy(wl.X).cuda()
    offs = regions.hypercube(2, wl.D)
    C, K = X.shape[1], len(offs)
    n = wl.n
    # every buffer allocated once (output rows <= input rows)
    table = torch.empty(gsc.gsc_table_bytes(n), dtype=torch.uint8, device="cuda")
    out_table = torch.empty(gsc.gsc_table_bytes(n), dtype=torch.uint8, device="cuda")
    fb = gsc.MapBuffers(n, K, wl.D, "cuda", dense=True)
    tb = gsc.MapBuffers(n, K, wl.D, "cuda", dense=True)
    host_offs, host_neg = gsc._host_i32(offs), gsc._host_i32(-offs)
    pooled = gsc.Pooled(torch.empty((n, C), dtype=torch.float32, device="cuda"),
                        torch.empty((n, C), dtype=torch.int32, device="cuda"),
                        torch.empty((n,), dtype=torch.int32, device="cuda"))
    dX = torch.empty((n, C), dtype=torch.float32, device="cuda")
    unpooled = gsc.Pooled(torch.empty((n, C), dtype=torch.float32, device="cuda"), None,
                          torch.empty((n,), dtype=torch.int32, device="cuda"))
    dXc = torch.empty((n, C), dtype=torch.float32, device="cuda")
    stride_result = torch.empty(2, dtype=torch.int64, pin_memory=True)

    def one(mark):
        gsc.gsc_coords_build(coords, table, sync=False)
        # the count of the output rows is read once the map onto the input
        # rows (which needs only the output table) is enqueued behind them
        pending = gsc.gsc_coords_stride(coords, 2, out_table=out_table, defer=True, result=stride_result)
        tmap = gsc.gsc_kernel_map(out_table, coords, -offs, sync=False, bufs=tb, host_offsets=host_neg, dense=True)
        out, _ = pending.finish()
        fmap = gsc.gsc_kernel_map(table, out, offs, sync=False, bufs=fb, host_offsets=host_offs, dense=True)
        mark("map")
        p = gsc.gsc_sparse_pool_fwd(X, fmap, args.pool, out=pooled)
        mark("fwd")
        g = gsc.gsc_sparse_pool_bwd(p.Y, tmap, args.pool, p, dX=dX)
        mark("bwd")
        if args.unpool:   # back to the fine rows (the transposed pooling) and its gradient
            u = gsc.gsc_sparse_pool_fwd(p.Y, tmap, args.pool, out=unpooled)
            mark("unpool_fwd")
            gsc.gsc_sparse_pool_bwd(u.Y, fmap, args.pool, u, dX=dXc[:p.Y.shape[0]])
            mark("unpool_bwd")
        return fmap, p, g

    for _ in range(args.warmup):
        one(lambda name: None)
    torch.cuda.synchronize()
    evs = []
    with no_gc():
        t0 = time.perf_counter()
        for _ in range(args.steps):
            ev = []

            def mark(name, ev=ev):
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                ev.append((name, e))

            mark("start")
            fmap, p, dX = one(mark)
            evs.append(ev)
        torch.cuda.synchronize()
        sec = (time.perf_counter() - t0) / args.steps
    stages = ["map", "fwd", "bwd"] + (["unpool_fwd", "unpool_bwd"] if args.unpool else [])
    ms = {k: [] for k in stages}
    for ev in evs:
        d = dict(ev)
        prev = "start"
        for k in stages:
            ms[k].append(d[prev].elapsed_time(d[k]))
            prev = k
    ms = {k: float(np.mean(v)) for k, v in ms.items()}
    n_pairs, n_out = fmap.count(), fmap.n_out
    nbytes = pool_bytes(n_pairs, n_out, C, K, args.pool)
    ach = nbytes / (ms["fwd"] * 1e-3) / 1e9
    roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_pool_fwd",
            "bytes_per_launch": int(nbytes), "avg_launch_us": round(ms["fwd"] * 1e3, 2)}
    cpu = None if args.no_cpu_baseline else pool_cpu_baseline(args.pool)
    out = {
        "metric": f"sparse {args.pool}-pool fwd+bwd{' and unpool fwd+bwd' if args.unpool else ''} voxels/s", "value": round(wl.n / sec, 1), "unit": "voxels/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(sec * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{wl.name}_{args.pool}pool2_s2{'_unpool' if args.unpool else ''}", "voxels": wl.n,
                   "pooled_rows": n_out,
                   "map_pairs": n_pairs, "channels": C, "parallelism": "single GPU"},
        "pool_fwd_bwd_voxels_per_s": round(wl.n / ((ms["fwd"] + ms["bwd"]) * 1e-3), 1),
        "stage_ms": {k: round(v, 4) for k, v in ms.items()},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def scene_points(scale: float = 1.0):
    """The float points of workload 1's two scenes (before voxelisation),
    their batch indices and per-point labels (the surface each point lies on
    is not tracked, so the labels are a seeded random class per point)."""
    import numpy as np
    from paper_1904_08755_amd import workloads as WL
    pts, bs = [], []
    n = int(round(WL.SCENE_POINTS_2CM * scale * scale))
    for b in range(2):
        geom = WL.draw_scene(WL.rng_for(1, WL.S_GEOM, b), scale=scale)
        p = WL.sample_points(geom, WL.rng_for(1, WL.S_GEOM, b, 1), n)
        pts.append(np.asarray(p, np.float32))
        bs.append(np.full(len(p), b, np.int32))
    P, B = np.concatenate(pts), np.concatenate(bs)
    L = np.random.default_rng(np.random.SeedSequence(WL.ROOT_SEED, spawn_key=(2000,))).integers(0, 20, len(P))
    return P, B, L.astype(np.int32)


def run_quantize(args):
    """Quantization of the scenes' points at 2 cm (the step before the
    hash table): voxel rows, representatives, labels, inverse map.  The call
    synchronises once (it returns the voxel count)."""
    import numpy as np
    import torch

    from paper_1904_08755_amd import gsc
    P, B, L = scene_points()
    tp, tb, tl = torch.from_numpy(P).cuda(), torch.from_numpy(B).cuda(), torch.from_numpy(L).cuda()
    for _ in range(args.warmup):
        q = gsc.gsc_quantize(tp, 0.02, batch=tb, labels=tl)
    torch.cuda.synchronize()
    with no_gc():
        t0 = time.perf_counter()
        for _ in range(args.steps):
            q = gsc.gsc_quantize(tp, 0.02, batch=tb, labels=tl)
        torch.cuda.synchronize()
        sec = (time.perf_counter() - t0) / args.steps
    n, n_out = len(P), int(q.coords.shape[0])
    cpu = None
    if not args.no_cpu_baseline:
        import oracle.gsc_oracle as O
        t1 = time.perf_counter()
        O.quantize(P, B, 0.02, L)
        tc = time.perf_counter() - t1
        cpu = {"value": n / tc, "unit": "points/s", "cores": 1, "kind": "oracle",
               "sample": f"all {n} points, single-threaded Python; {tc:.1f} s", "seconds": tc}
    out = {
        "metric": "sparse tensor quantization points/s", "value": round(n / sec, 1), "unit": "points/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(sec * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "scene2cm_b2_points_quantize", "points": n, "voxels": n_out, "voxel_m": 0.02,
                   "parallelism": "single GPU"},
        "roofline": None, "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


# forward+backward targets (microseconds) of the workloads: 50 % of the HBM
# roofline for the fp32 layers (C <= 64), 40 % of the bf16 MFMA peak for the
# 256-channel layer; workload 0 is bound by launch latency (no target)
TARGET_US = {0: None, 1: 140.0, 2: 338.0, 3: 90.0, 4: 352.0}


def conv_pass_bytes(pairs, layers, n_ins, n_outs, s):
    """Gather-model bytes of forward + input gradient + weight gradient of
    every layer: one gathered row and one index pair per kernel-map pair and
    pass, every output row written once, the weights read once (dW written
    once in fp32)."""
    tot = 0.0
    for m, L, n_in, n_out in zip(pairs, layers, n_ins, n_outs):
        K = L.W.shape[0]
        tot += fwd_bytes(m, n_out, L.c_in, L.c_out, K, s)
        tot += m * (s * L.c_out + 8) + n_in * s * L.c_in + K * L.c_in * L.c_out * s
        tot += m * (s * (L.c_in + L.c_out) + 8) + 4 * K * L.c_in * L.c_out
    return tot


def bench_conv(args, wid: int, region=None, affine: bool = False, plan_mode: str = "auto",
               steps: int = None, warmup: int = None) -> dict:
    """Time ``steps`` whole passes of workload ``wid`` (after ``warmup``
    untimed ones) and return its results: per-step time, voxels/s, stage
    times (mean, median, p10, p90) from HIP events on the stream, the
    forward+backward time against its target, and the roofline of the
    forward kernel of the first layer."""
    import numpy as np
    import torch

    from paper_1904_08755_amd import gsc, pipeline
    from paper_1904_08755_amd import workloads as WL

    steps = args.steps if steps is None else steps
    warmup = args.warmup if warmup is None else warmup
    t = time.perf_counter()
    wl = WL.make_workload(wid, region=region)
    log(f"workload {wl.name}: n={wl.n} ({time.perf_counter() - t:.1f} s to generate)")
    dw = pipeline.to_device(wl, "cuda")
    epi = None
    if affine:
        rng = np.random.default_rng(np.random.SeedSequence(WL.ROOT_SEED, spawn_key=(wl.config_id, 9)))
        co = wl.layers[0].c_out
        epi = (torch.from_numpy(rng.uniform(0.5, 2.0, co).astype(np.float32)).cuda(),
               torch.from_numpy(rng.uniform(-0.5, 0.5, co).astype(np.float32)).cuda())
    torch.cuda.synchronize()

    # block plans or the row form: the faster of the two on this workload
    use_plan = plan_mode == "yes" or (plan_mode == "auto" and pipeline.choose_block_plans(dw, epi))
    log(f"  block plans: {'yes' if use_plan else 'no'}" + (" (measured choice)" if plan_mode == "auto" else ""))
    plan0 = pipeline.StepPlan(dw, use_plan=use_plan, epilogue=epi)
    for _ in range(warmup):
        plan0.run()
    gsc.gsc_table_status(plan0.table)   # the build of the warm-up passes succeeded
    del plan0
    torch.cuda.synchronize()
    log(f"  warmup done ({warmup} steps)")

    steps_events = []
    plan = pipeline.StepPlan(dw, use_plan=use_plan, epilogue=epi)
    torch.cuda.synchronize()
    with no_gc():
        t0 = time.perf_counter()
        for _ in range(steps):
            ev = []

            def mark(name, ev=ev):
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                ev.append((name, e))

            mark("start")
            last = plan.run(mark)
            steps_events.append(ev)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
    sec = (t1 - t0) / steps
    log(f"  timed {steps} steps: {sec * 1e3:.3f} ms/step")

    stage = {"map": [], "plan": [], "fwd": [], "bwd": []}
    for ev in steps_events:
        d = dict(ev)
        stage["map"].append(d["start"].elapsed_time(d["map"]))
        stage["plan"].append(d["map"].elapsed_time(d["plan"]))
        stage["fwd"].append(d["plan"].elapsed_time(d["fwd"]))
        stage["bwd"].append(d["fwd"].elapsed_time(d["bwd"]))
    ms = {k: float(np.mean(v)) for k, v in stage.items()}
    stats = stage_stats(stage)

    L0 = wl.layers[0]
    s = 2 if wl.dtype == "bf16" else 4
    pairs = [km.count() for km in last.kmaps]
    n_outs = [km.n_out for km in last.kmaps]
    n_ins = [wl.n] + n_outs[:-1]
    flops = sum(6.0 * m * L.c_in * L.c_out for m, L in zip(pairs, wl.layers))
    conv_s = (ms["fwd"] + ms["bwd"]) * 1e-3
    fb_med_us = (stats["median"]["fwd"] + stats["median"]["bwd"]) * 1e3
    km0 = last.kmaps[0]
    # dominant kernel: the forward convolution of layer 0
    planned = bool(plan.plans)
    kernel = forward_kernel(gsc, wl.dtype, L0.c_in, L0.c_out, km0.K, planned, epilogue=epi is not None)
    wname = wl.name.replace("_cube3", "")
    traffic = measured_traffic(kernel, wname)
    dom_bytes = fwd_bytes(pairs[0], n_outs[0], L0.c_in, L0.c_out, km0.K, s)
    if len(wl.layers) == 1:
        dom_ms = ms["fwd"]
    else:   # the first layer's forward launch, timed on its own
        dom_ms = float(np.mean([dict(ev)["plan"].elapsed_time(dict(ev)["fwd0"]) for ev in steps_events]))
    pass_bytes = conv_pass_bytes(pairs, wl.layers, n_ins, n_outs, s)
    roof = None
    if dom_ms and wl.dtype == "bf16":
        # wide bf16 layer: the per-offset contractions on the MFMA units
        dom_flops = 2.0 * pairs[0] * L0.c_in * L0.c_out
        ach = dom_flops / (dom_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": traffic,
                "kernel": kernel, "flops_per_launch": int(dom_flops),
                "bytes_per_launch": int(dom_bytes), "avg_launch_us": round(dom_ms * 1e3, 2)}
        fb = {"bound": "mfma", "unit": "TFLOP/s", "achieved": round(flops / conv_s / 1e12, 2),
              "frac": round(flops / conv_s / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)}
    elif dom_ms:
        ach = dom_bytes / (dom_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": kernel, "bytes_per_launch": int(dom_bytes),
                "avg_launch_us": round(dom_ms * 1e3, 2)}
        fb = {"bound": "hbm", "unit": "GB/s", "achieved": round(pass_bytes / conv_s / 1e9, 1),
              "frac": round(pass_bytes / conv_s / 1e9 / HBM_PEAK_GBS, 4)}
    fb.update({"us": round(conv_s * 1e6, 2), "us_median": round(fb_med_us, 2),
               "target_us": TARGET_US.get(wid) if region in (None, "hybrid") else None,
               "flops": flops, "gather_model_bytes": int(pass_bytes)})
    out = {
        "workload": wl.name, "dtype": wl.dtype, "voxels": wl.n, "D": wl.D,
        "layers": [f"{L.kind}:{L.region}{L.ksize}/s{L.stride}:{L.c_in}->{L.c_out}" for L in wl.layers],
        "kernel_map_pairs": pairs, "block_plan": planned,
        "ms_per_step": round(sec * 1e3, 4), "voxels_per_s": round(wl.n / sec, 1),
        "conv_fwd_bwd_voxels_per_s": round(wl.n / conv_s, 1),
        "effective_gflops": round(flops / conv_s / 1e9, 1),
        "kernel_map_build_ms": round(ms["map"], 4),
        "block_plan_ms": round(ms["plan"], 4),
        "stage_ms": {k: round(v, 4) for k, v in ms.items()},
        "stage_ms_median": stats["median"], "stage_ms_p10": stats["p10"], "stage_ms_p90": stats["p90"],
        "fwd_bwd": fb,
        "roofline": roof,
        "_wl": wl,
    }
    if epi is not None:
        out["epilogue"] = "batchnorm_affine+relu"
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=None,
                    help="0..4: time this workload only (default: all five, headline workload 4, the indoor "
                         "scenes at 2 cm with 256 channels in bf16)")
    ap.add_argument("--region", choices=["hybrid", "cube", "spatial", "cross"], default=None,
                    help="region of workload 3 (3D video): hybrid (default, 29 offsets), cube (tesseract, 81), "
                         "spatial (3^3 at zero time offset, 27: each frame on its own), cross (9)")
    ap.add_argument("--affine", action="store_true",
                    help="forward with batch normalisation (per-channel affine form) and ReLU fused into the "
                         "convolution's output write (Sec. 4.5); single-layer workloads")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--plan", choices=["auto", "yes", "no"], default="auto",
                    help="block plans: the faster of plans and row form timed on the workload (auto), or always/never "
                         "(a profiler's per-launch overhead can change what auto measures)")
    ap.add_argument("--no-plan", action="store_true", help="the same as --plan no")
    ap.add_argument("--pool", choices=["max", "avg", "sum"], default=None,
                    help="time pooling instead (Sec. 4.3, 4.4): the 2^3 stride-2 window over the scene of workload 1")
    ap.add_argument("--unpool", action="store_true",
                    help="with --pool avg|sum: also unpool (the transposed pooling, Sec. 4.4) back to the input rows, "
                         "forward and backward")
    ap.add_argument("--quantize", action="store_true",
                    help="time sparse tensor quantization (Alg. 1) of the two indoor scenes' points at 2 cm instead")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, copy 256 MiB once (a copy of known size for scaling the "
                         "FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print("bench.py runs on one GPU only: the sparse-convolution path here is a single-GPU build "
              "(no collectives); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_1904_08755_amd import gsc

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    gsc.lib()
    if args.unpool and args.pool not in ("avg", "sum"):
        print("--unpool needs --pool avg or --pool sum", file=sys.stderr)
        sys.exit(2)
    if args.pool:
        return run_pool(args)
    if args.quantize:
        return run_quantize(args)
    if args.region is not None and args.workload != 3:
        print("--region applies to workload 3 (the 3D video) only", file=sys.stderr)
        sys.exit(2)
    if args.affine and args.workload not in (0, 1, 3, 4):
        print("--affine applies to one of the single-layer workloads (--workload 0, 1, 3 or 4)", file=sys.stderr)
        sys.exit(2)

    plan_mode = "no" if args.no_plan else args.plan
    others = {}
    if args.workload is None:   # every workload; the headline is workload 4
        for wid in (0, 1, 2, 3):
            r = bench_conv(args, wid, plan_mode=plan_mode)
            r.pop("_wl")
            others[r.pop("workload")] = r
        head_id = 4
    else:
        head_id = args.workload
    head = bench_conv(args, head_id, region=args.region, affine=args.affine, plan_mode=plan_mode)
    wl = head.pop("_wl")
    roof = head.pop("roofline")

    if args.copy_calibration:
        src = torch.empty(64 * 2**20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: 268435456 bytes read, 268435456 bytes written")

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        cpu = cpu_baseline(wl)
        log(f"cpu baseline: {cpu['seconds']:.1f} s")
        if args.workload is None:   # the small workload 0 whole, median of 5
            from paper_1904_08755_amd import workloads as WL
            cpu["random64_c3to16_cube3"] = cpu_baseline(WL.make_workload(0), reps=5)

    config = {"workload": head.pop("workload"), "voxels": head.pop("voxels"), "D": head.pop("D"),
              "layers": head.pop("layers"), "kernel_map_pairs": head.pop("kernel_map_pairs"),
              "block_plan": head.pop("block_plan"), "parallelism": "single GPU"}
    if "epilogue" in head:
        config["epilogue"] = head.pop("epilogue")
    dtype = head.pop("dtype")
    ms_step = head.pop("ms_per_step")
    head.pop("voxels_per_s")
    out = {
        "metric": METRIC,
        "value": round(wl.n / (ms_step * 1e-3), 1),
        "unit": "voxels/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": config,
        **head,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    if others:
        out["configs"] = others
    if roof is not None and not args.copy_calibration:   # (a counter run's only copy is the calibration)
        peaks = measured_peaks(torch)
        ref = peaks["bf16_gemm_TFLOPs"] if roof["bound"] == "mfma" else peaks["copy_GBs"]
        roof["measured_peak"] = ref
        roof["frac_of_measured_peak"] = round(roof["achieved"] / ref, 4)
        out["measured_peaks"] = peaks
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark: frames/s of the per-frame clustering + density hot path on one GPU.

One step = cluster_frames + density_frames over one batch of synthetic frames
(default: 64 frames x 2000 birds, 1920x1080 px, eps 40 px, minPts 4, density
grid 128x72, sigma 30 px).  The two calls are independent analytics of the
same batch, so a step issues them on two streams (default priority) and joins.
Inputs are resident in device memory before any timed region.

Timed regions (each bracketed by device synchronisation):
  1. K steps replayed from HIP graphs captured from the step (graphs of up
     to 10 steps; host launch cost out of the loop), once with the two calls
     on two streams and once on one stream.  Step k reads and writes copy
     k mod R of the batch (inputs and outputs), with R copies together larger
     than twice the 256 MB memory-side cache (at most 1000 copies), so each
     step finds its data in HBM, not in a cache.  Every copy's outputs are
     checked against the eager outputs first.  `value` is the faster of the
     two modes (`config.streams` says which): on large batches the two
     kernels compete for compute units and one stream wins.
  2. the same replays on one copy of the batch (`warm_value`: inputs and
     outputs stay in L2 and the memory-side cache where they fit).
  3. per-kernel durations for the roofline: K steps issued eagerly on one
     stream (each kernel alone on the GPU), each after a write of flush_mb
     MiB that evicts the caches, with HIP events recorded on that stream.

Prints one JSON line on stdout; progress goes to stderr.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HEADLINE = "batch64x2000_1080p"
METRIC = "frames/sec (cluster+density) at 2000 birds/frame"

# MI355X published peaks
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0

# the sources each entry point's kernels are built from (a counter summary
# holds for the traffic of the current kernels only if all of them match)
KERNEL_SOURCES = {
    "cluster": ["paper_2512_07009_amd/csrc/cluster.hip", "paper_2512_07009_amd/csrc/cluster_big.hip",
                "paper_2512_07009_amd/csrc/cluster_common.h"],
    "density": ["paper_2512_07009_amd/csrc/density.hip"],
    "heatmap": ["paper_2512_07009_amd/csrc/heatmap.hip", "paper_2512_07009_amd/csrc/cluster_common.h"],
    "roi": ["paper_2512_07009_amd/csrc/roi.hip"],
    "drinker": ["paper_2512_07009_amd/csrc/roi.hip"],
    "mask": ["paper_2512_07009_amd/csrc/mask.hip", "paper_2512_07009_amd/csrc/cluster_common.h"],
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_hash(rels) -> str:
    """sha256[:16] of the named source files, concatenated in order."""
    h = hashlib.sha256()
    for rel in rels:
        with open(os.path.join(ROOT, rel), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    that summary was taken from the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"source sha256\[:16\]:\s*`?([0-9a-f]{16})", text)
    m_bytes = re.search(r"HBM bytes per launch \(scaled\):\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != source_hash(KERNEL_SOURCES[kernel]):
        return None
    return float(m_bytes.group(1))


def cpu_baseline(xy, off, w, budget_s: float, one_thread_s: float):
    """The CPU oracle on the host cores: whole frames, as many as fit about
    budget_s; then on one thread, the whole batch if it fits one_thread_s,
    else the first 8 frames."""
    import oracle
    threads = oracle.default_threads()
    F = len(off) - 1

    def run(n, n_threads):
        sxy, soff = xy[: off[n]], off[: n + 1]
        t0 = time.perf_counter()
        oracle.cluster_frames(sxy, soff, w.eps_q, w.min_pts, n_threads=n_threads)
        oracle.density_frames(sxy, soff, w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px,
                              n_threads=n_threads)
        return time.perf_counter() - t0

    def rate(n, n_threads, probe):
        """Frames/s over the first n frames (the probe is that run when n is
        1); a batch that runs in under a second is repeated until about 1 s."""
        dt = probe if n == 1 else run(n, n_threads)
        reps = 1
        while dt < 1.0:
            dt += run(n, n_threads)
            reps += 1
        return reps * n / dt, reps, dt

    # probe one frame, then size the sample (clustering threads over frames,
    # density over grid rows)
    per_frame = max(run(1, threads), 1e-6)
    n = int(max(1, min(F, budget_s / per_frame)))
    v, reps, dt = rate(n, threads, per_frame)
    per_frame1 = max(run(1, 1), 1e-6)
    n1 = F if per_frame1 * F <= one_thread_s else int(min(F, 8))
    v1, reps1, dt1 = rate(n1, 1, per_frame1)

    def what(k, r, t):
        return (f"all {F} frames" if k == F else f"first {k} of {F} frames") + \
            (f" x{r}" if r > 1 else "") + f", {t:.1f} s wall"
    model = ""
    try:
        with open("/proc/cpuinfo") as fh:
            model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": v, "unit": "frames/s", "cores": threads, "kind": "oracle",
            "sample": f"{w.name} (clustering + density): " + what(n, reps, dt),
            "one_thread_value": v1, "one_thread_sample": what(n1, reps1, dt1),
            "cpu_model": model}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--mask-workload", default="masks8x2000_720p",
                    help="segmentation batch for the detection post-processing entry")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=10.0,
                    help="target wall seconds for the oracle sample (all host cores)")
    ap.add_argument("--cpu-one-thread-s", type=float, default=30.0,
                    help="the one-thread oracle leg takes the whole batch if it fits this many seconds, "
                         "else the first 8 frames")
    ap.add_argument("--rotate-mb", type=float, default=512,
                    help="MiB of batch copies that `value` rotates over (0: one copy, warm caches)")
    ap.add_argument("--no-graph", action="store_true", help="time `value` from eager launches")
    ap.add_argument("--streams", choices=("auto", "1", "2"), default="auto",
                    help="step modes timed for `value`: both (the faster is reported), one stream, or two")
    ap.add_argument("--flush-mb", type=float, default=512,
                    help="MiB written before each launch timed for the roofline (0: warm back-to-back launches only)")
    ap.add_argument("--calibrate-copy-mb", type=float, default=0,
                    help="also run one plain device copy of this many MiB (counter scaling)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(frames would shard across GPUs by contiguous ranges, with no collective)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2512_07009_amd as flock
    from paper_2512_07009_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    xy, off, _ = wl.generate(args.workload)
    F, T = len(off) - 1, xy.shape[0]
    max_fp = int(np.diff(off).max())
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dxy = torch.from_numpy(xy).to(dev)
    doff = torch.from_numpy(off).to(dev)
    labels = torch.empty(T, dtype=torch.int32, device=dev)
    kind = torch.empty(T, dtype=torch.uint8, device=dev)
    ncl = torch.empty(F, dtype=torch.int32, device=dev)
    dens = torch.empty((F, w.grid_h, w.grid_w), dtype=torch.float32, device=dev)
    stream = main_stream = torch.cuda.current_stream(dev)
    cells = w.grid_w * w.grid_h
    log(f"workload {w.name}: {F} frames, {T} birds, max {max_fp}/frame; {flock.version()}")

    side = torch.cuda.Stream(dev)  # default priority

    def buffers(src_xy, src_off):
        return {"xy": src_xy, "off": src_off,
                "labels": torch.empty(T, dtype=torch.int32, device=dev),
                "kind": torch.empty(T, dtype=torch.uint8, device=dev),
                "ncl": torch.empty(F, dtype=torch.int32, device=dev),
                "dens": torch.empty((F, w.grid_h, w.grid_w), dtype=torch.float32, device=dev)}

    home = {"xy": dxy, "off": doff, "labels": labels, "kind": kind, "ncl": ncl, "dens": dens}

    def run_pair(k, concurrent, evs=None, launch_stream=None, buf=None):
        """cluster_frames on `stream` (or `launch_stream`), density_frames on
        `side` (or also on the first stream when not concurrent), with the join
        back on the first stream; on the batch copy `buf` (default: the first)."""
        stream = launch_stream if launch_stream is not None else main_stream
        b = buf if buf is not None else home
        sd = side
        ds = sd if concurrent else stream
        if concurrent:
            fork = torch.cuda.Event()
            fork.record(stream)
            sd.wait_event(fork)
        if evs is not None:
            evs[0].record(stream)
        flock.cluster_frames(b["xy"], b["off"], w.eps_px, w.min_pts, max_fp, out=(b["labels"], b["kind"], b["ncl"]),
                             stream=stream)
        if evs is not None:
            evs[1].record(stream)
            evs[2].record(ds)
        flock.density_frames(b["xy"], b["off"], w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px,
                             max_fp, out=b["dens"], stream=ds)
        if evs is not None:
            evs[3].record(ds)
        if concurrent:
            join = torch.cuda.Event()
            join.record(sd)
            stream.wait_event(join)

    # a buffer larger than L2 and the 256 MB memory-side cache together:
    # writing it before a timed launch makes that launch read its inputs from HBM
    flush = torch.empty(int(args.flush_mb) << 20, dtype=torch.uint8, device=dev) if args.flush_mb > 0 else None

    def evict(k):
        if flush is not None:
            flush.fill_(k & 0xff)

    def timed(concurrent, K, cold=False):
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
        torch.cuda.synchronize(dev)
        t0 = time.perf_counter()
        for k in range(K):
            if cold:
                evict(k)
            run_pair(k, concurrent, evs[k])
        torch.cuda.synchronize(dev)
        wall = time.perf_counter() - t0
        t_c = sum(e[0].elapsed_time(e[1]) for e in evs) / K * 1e-3   # s per launch
        t_d = sum(e[2].elapsed_time(e[3]) for e in evs) / K * 1e-3
        return wall, t_c, t_d

    def per_launch(fn, K):
        """Average duration of fn() on the main stream: back to back (warm
        caches), and each launch after the flush (cold, inputs from HBM)."""
        for _ in range(3):
            fn()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize(dev)
        e[0].record(stream)
        for _ in range(K):
            fn()
        e[1].record(stream)
        torch.cuda.synchronize(dev)
        warm = e[0].elapsed_time(e[1]) / K * 1e-3
        if flush is None:
            return warm, warm
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
        for k in range(K):
            evict(k)
            evs[k][0].record(stream)
            fn()
            evs[k][1].record(stream)
        torch.cuda.synchronize(dev)
        return sum(a.elapsed_time(b) for a, b in evs) / K * 1e-3, warm

    if args.calibrate_copy_mb > 0:
        # a plain device copy of known size, for scaling HBM byte counters
        nbytes = int(args.calibrate_copy_mb) << 20
        src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize(dev)
        log(f"calibration copy: {nbytes} bytes read and written")
        del src, dst

    log("warmup")
    for k in range(args.warmup):
        run_pair(k, True)
        run_pair(k, False)
    torch.cuda.synchronize(dev)
    K = args.steps

    # 1-2. graph replays: the two-stream step and the one-stream step, over
    #      rotated copies of the batch and on one copy
    ref = (labels.clone(), kind.clone(), ncl.clone(), dens.clone())
    gsteps = min(K, 10)
    step_bytes = xy.nbytes + off.nbytes + 5 * T + 4 * F + 4 * F * cells
    n_copies = 1
    if args.rotate_mb > 0:
        n_copies = min(1000, max(2, -(-int(args.rotate_mb * (1 << 20)) // step_bytes)))
        n_copies = -(-n_copies // gsteps) * gsteps
    copies = [home] + [buffers(dxy.clone(), doff.clone()) for _ in range(n_copies - 1)]
    rotation = {"copies": n_copies, "bytes_per_copy": step_bytes, "total_mb": n_copies * step_bytes / 2**20}
    log(f"graph replays over {n_copies} copies of the batch ({rotation['total_mb']:.0f} MiB), then on one copy")

    def same_as_ref(b):
        return (torch.equal(b["labels"], ref[0]) and torch.equal(b["kind"], ref[1]) and torch.equal(b["ncl"], ref[2])
                and torch.equal(b["dens"], ref[3]))

    def capture_steps(grp, concurrent, joined, cap):
        """The steps of one graph: one stream; or two streams joined after
        every step; or two streams, the clustering launches of the steps in
        order on one and the density launches on the other, joined once at
        the graph's end (each step still runs both over its own batch copy;
        a step's density launch may start before the previous step's
        clustering has ended)."""
        if concurrent and not joined:
            fork = torch.cuda.Event()
            fork.record(cap)
            side.wait_event(fork)
            for b in grp:
                flock.cluster_frames(b["xy"], b["off"], w.eps_px, w.min_pts, max_fp,
                                     out=(b["labels"], b["kind"], b["ncl"]), stream=cap)
                flock.density_frames(b["xy"], b["off"], w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px,
                                     max_fp, out=b["dens"], stream=side)
            join = torch.cuda.Event()
            join.record(side)
            cap.wait_event(join)
        else:
            for k, b in enumerate(grp):
                run_pair(k, concurrent, launch_stream=cap, buf=b)

    def replay_wall(concurrent, bufs, joined=False):
        """Capture graphs of `gsteps` steps cycling over `bufs`, check one pass
        over every copy against the eager outputs, then time K steps."""
        cap = torch.cuda.Stream(dev)
        cap.wait_stream(main_stream)
        groups = [bufs[i:i + gsteps] for i in range(0, len(bufs), gsteps)] if len(bufs) > 1 else [bufs * gsteps]
        graphs = []
        for grp in groups:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cap):
                capture_steps(grp, concurrent, joined, cap)
            graphs.append(g)
        rem = None
        if K % gsteps:
            grp = groups[(K // gsteps) % len(groups)][:K % gsteps]
            rem = torch.cuda.CUDAGraph()
            with torch.cuda.graph(rem, stream=cap):
                capture_steps(grp, concurrent, joined, cap)
        torch.cuda.synchronize(dev)
        for b in bufs:
            b["labels"].fill_(-7)
            b["dens"].fill_(-1.0)
        for g in graphs:
            g.replay()
        torch.cuda.synchronize(dev)
        if not all(same_as_ref(b) for b in bufs):
            raise RuntimeError("graph replay differs from the eager outputs")
        plan = [graphs[i % len(graphs)] for i in range(K // gsteps)] + ([rem] if rem is not None else [])
        torch.cuda.synchronize(dev)
        t0 = time.perf_counter()
        for g in plan:
            g.replay()
        torch.cuda.synchronize(dev)
        return time.perf_counter() - t0

    graph_note = None
    modes = {"auto": (True, False), "1": (False,), "2": (True,)}[args.streams]
    walls, warm_walls = {}, {}
    joined_wall = None
    if not args.no_graph:
        try:
            for concurrent in modes:
                walls[concurrent] = replay_wall(concurrent, copies)
                warm_walls[concurrent] = replay_wall(concurrent, [home]) if n_copies > 1 else walls[concurrent]
            if True in modes:
                joined_wall = replay_wall(True, copies, joined=True)
        except RuntimeError as ex:
            graph_note = f"graph replay unavailable ({ex}); value timed eagerly on one copy"
            log(graph_note)
            walls, warm_walls = {}, {}

    # 3. eager steps with per-kernel events in each mode; the roofline's
    #    durations come from one-stream steps (each kernel alone on the GPU),
    #    each step after the flush
    log("eager steps with events")
    eager = {c: timed(c, K) for c in modes}
    if not walls:
        walls = warm_walls = {c: eager[c][0] for c in modes}
    concurrent = min(modes, key=lambda c: walls[c])
    wall = walls[concurrent]
    warm_wall = min(warm_walls.values())
    _, w_cluster, w_density = eager[False] if False in modes else timed(False, K)
    if flush is not None:
        log("one-stream eager steps with events after a cache flush")
        _, t_cluster, t_density = timed(False, K, cold=True)
    else:
        t_cluster, t_density = w_cluster, w_density
    ms_per_step = wall / K * 1e3
    value = F / (wall / K)

    log("heatmap, roi, drinker and mask entries")
    # 4. heatmap analytics of the step's density grids (its own entry point,
    #    not part of `value`): hot cells at twice the frame-average density
    area = (w.width_px / w.grid_w) * (w.height_px / w.grid_h)
    heat_thr = 2.0 * T / (F * w.width_px * w.height_px)
    hout = {"labels": torch.empty((F, w.grid_h, w.grid_w), dtype=torch.int32, device=dev),
            "n_components": torch.empty(F, dtype=torch.int32, device=dev),
            "entropy": torch.empty(F, dtype=torch.float64, device=dev),
            "degree": torch.empty(F, dtype=torch.float64, device=dev),
            "comp_cells": torch.empty((F, w.grid_h, w.grid_w), dtype=torch.int32, device=dev),
            "comp_mass": torch.empty((F, w.grid_h, w.grid_w), dtype=torch.float64, device=dev)}
    t_heat, t_heat_warm = per_launch(lambda: flock.heatmap_frames(dens, area, heat_thr, 8, out=hout, stream=stream), K)

    # 5. region-of-interest filter and counts (its own entry point, not part of
    #    `value`): a strip along the left wall, a five-vertex polygon
    Wq, Hq = 16 * w.width_px, 16 * w.height_px
    roi_poly = [[0, 0], [Wq // 8, 0], [Wq // 6, Hq // 2], [Wq // 8, Hq], [0, Hq]]
    rout = {"counts": torch.empty(F, dtype=torch.int32, device=dev),
            "xy": torch.empty((T, 2), dtype=torch.int32, device=dev),
            "offsets": torch.empty(F + 1, dtype=torch.int32, device=dev),
            "index": torch.empty(T, dtype=torch.int32, device=dev)}
    t_roi, t_roi_warm = per_launch(lambda: flock.roi_filter_frames(dxy, doff, roi_poly, out=rout, stream=stream), K)
    kept = int(rout["offsets"][-1].item())

    # 6. drinker-line proximity (its own entry point, not part of `value`): two
    #    drinker lines across the frame, 20 px
    dlines = [[Wq // 10, Hq // 4, 9 * Wq // 10, Hq // 4], [Wq // 10, 3 * Hq // 4, 9 * Wq // 10, 3 * Hq // 4]]
    dthr = 16 * 20
    dout = {"drinking": torch.empty(T, dtype=torch.uint8, device=dev),
            "line": torch.empty(T, dtype=torch.int32, device=dev),
            "counts": torch.empty(F, dtype=torch.int32, device=dev)}
    t_drink, t_drink_warm = per_launch(
        lambda: flock.drinker_proximity_frames(dxy, doff, dlines, dthr, out=dout, stream=stream), K)

    # 7. detection post-processing (its own entry point, not part of `value`):
    #    a batch of segmentation outputs, its own synthetic input
    prob_np, mw = wl.mask_batch(args.mask_workload)
    prob = torch.from_numpy(prob_np).to(dev)
    MF, MH, MW = prob_np.shape
    mcap = flock.mask_capacity(MF, MH, MW, mw.connectivity)
    mout = {"labels": torch.empty((MF, MH, MW), dtype=torch.int32, device=dev),
            "n_components": torch.empty(MF, dtype=torch.int32, device=dev),
            "offsets": torch.empty(MF + 1, dtype=torch.int32, device=dev),
            "label": torch.empty(mcap, dtype=torch.int32, device=dev),
            "area": torch.empty(mcap, dtype=torch.int32, device=dev),
            "box": torch.empty((mcap, 4), dtype=torch.int32, device=dev),
            "centroid": torch.empty((mcap, 2), dtype=torch.float64, device=dev),
            "xy": torch.empty((mcap, 2), dtype=torch.int32, device=dev),
            "score": torch.empty(mcap, dtype=torch.float32, device=dev)}
    t_mask, t_mask_warm = per_launch(lambda: flock.mask_components_frames(prob, mw.threshold, mw.connectivity, capacity=mcap,
                                                                   out=mout, stream=stream), K)
    n_det = int(mout["offsets"][-1].item())
    del prob, mout

    # algorithmic work per launch
    cluster_bytes = 13 * T + 8 * F + 4          # xy 8 + labels 4 + kind 1 per bird; offsets, n_clusters
    density_flops = 2.0 * w.grid_w * w.grid_h * T
    cl = {"bound": "hbm", "achieved": cluster_bytes / t_cluster / 1e9, "peak": HBM_PEAK_GBS,
          "unit": "GB/s", "per_launch_us": t_cluster * 1e6, "warm_per_launch_us": w_cluster * 1e6,
          "two_stream_per_launch_us": eager[True][1] * 1e6 if True in eager else None,
          "algorithmic_bytes": cluster_bytes}
    cl["frac"] = cl["achieved"] / cl["peak"]
    cl["traffic"] = committed_traffic("cluster", w.name)
    de = {"bound": "mfma", "achieved": density_flops / t_density / 1e12, "peak": MFMA_F16_PEAK_TFLOPS,
          "unit": "TFLOP/s", "per_launch_us": t_density * 1e6, "warm_per_launch_us": w_density * 1e6,
          "two_stream_per_launch_us": eager[True][2] * 1e6 if True in eager else None,
          "algorithmic_flops": density_flops}
    de["frac"] = de["achieved"] / de["peak"]
    de["traffic"] = committed_traffic("density", w.name)
    heat_bytes = 20 * F * cells + 20 * F  # density 4 + labels 4 + cells 4 + mass 8 per cell; 20 B per frame
    he = {"bound": "hbm", "achieved": heat_bytes / t_heat / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
          "per_launch_us": t_heat * 1e6, "warm_per_launch_us": t_heat_warm * 1e6, "algorithmic_bytes": heat_bytes,
          "threshold": heat_thr, "connectivity": 8, "in_value": False}
    he["frac"] = he["achieved"] / he["peak"]
    he["traffic"] = committed_traffic("heatmap", w.name)
    roi_bytes = 8 * T + 12 * kept + 12 * F + 8  # xy in; kept xy + index out; offsets in, counts + offsets out
    ro = {"bound": "hbm", "achieved": roi_bytes / t_roi / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
          "per_launch_us": t_roi * 1e6, "warm_per_launch_us": t_roi_warm * 1e6, "algorithmic_bytes": roi_bytes,
          "kept_birds": kept,
          "roi_vertices": len(roi_poly), "in_value": False}
    ro["frac"] = ro["achieved"] / ro["peak"]
    ro["traffic"] = committed_traffic("roi", w.name)
    drink_bytes = 13 * T + 8 * F + 4  # xy in, flag and line out per bird; offsets in, counts out
    dr = {"bound": "hbm", "achieved": drink_bytes / t_drink / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
          "per_launch_us": t_drink * 1e6, "warm_per_launch_us": t_drink_warm * 1e6, "algorithmic_bytes": drink_bytes,
          "lines": len(dlines),
          "threshold_px": dthr / 16, "in_value": False}
    dr["frac"] = dr["achieved"] / dr["peak"]
    dr["traffic"] = committed_traffic("drinker", w.name)
    mpx = MF * MH * MW
    # prob in and labels out per pixel; 52 B per component (label, area, box,
    # centroid, 1/16-px centroid, score); counts and offsets per frame
    mask_bytes = 8 * mpx + 52 * n_det + 8 * MF + 4
    ma = {"bound": "hbm", "achieved": mask_bytes / t_mask / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
          "per_launch_us": t_mask * 1e6, "warm_per_launch_us": t_mask_warm * 1e6, "algorithmic_bytes": mask_bytes,
          "workload": mw.name,
          "frames": MF, "frame_px": [MW, MH], "components": n_det, "threshold": mw.threshold,
          "connectivity": mw.connectivity, "frames_per_s": MF / t_mask, "in_value": False}
    ma["frac"] = ma["achieved"] / ma["peak"]
    ma["traffic"] = committed_traffic("mask", mw.name)
    if not args.no_cpu_baseline:
        import oracle
        log("timing the CPU oracle beside the heatmap, roi, drinker and mask entries")
        t0 = time.perf_counter()
        oracle.mask_components(prob_np, mw.threshold, mw.connectivity)
        ma["oracle_frames_per_s"] = MF / (time.perf_counter() - t0)
        ma["oracle_threads"] = 1
        # bounded samples: the first frames, up to 4M grid cells / 2M birds
        nh = int(max(1, min(F, (1 << 22) // cells)))
        dens_np = dens[:nh].float().cpu().numpy()
        t0 = time.perf_counter()
        oracle.heatmap_frames(dens_np, area, heat_thr, 8)
        he["oracle_frames_per_s"] = nh / (time.perf_counter() - t0)
        he["oracle_threads"] = oracle.default_threads()
        he["oracle_sample_frames"] = nh
        nb = int(max(1, np.searchsorted(off, 1 << 21, side="right") - 1))
        sxy, soff = xy[: off[nb]], off[: nb + 1]
        t0 = time.perf_counter()
        oracle.roi_filter(sxy, soff, roi_poly)
        ro["oracle_frames_per_s"] = nb / (time.perf_counter() - t0)
        t0 = time.perf_counter()
        oracle.drinkers(sxy, soff, dlines, dthr)
        dr["oracle_frames_per_s"] = nb / (time.perf_counter() - t0)
        ro["oracle_threads"] = dr["oracle_threads"] = 1
        ro["oracle_sample_frames"] = dr["oracle_sample_frames"] = nb
    dominant = ("cluster_frames", cl) if t_cluster >= t_density else ("density_frames", de)
    roof = {k: dominant[1][k] for k in ("bound", "achieved", "peak", "unit", "frac", "traffic")}
    roof["kernel"] = dominant[0]

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i32+f16",
        "data": "synthetic",
        "config": {"workload": w.name, "frames": F, "birds": T, "birds_per_frame_max": max_fp,
                   "frame_px": [w.width_px, w.height_px], "eps_px": w.eps_px, "min_pts": w.min_pts,
                   "grid": [w.grid_w, w.grid_h], "sigma_px": w.sigma_px, "parallelism": "single-gpu",
                   "streams": 2 if concurrent else 1},
        "birds_per_s": T / (wall / K),
        "warm_value": F / (warm_wall / K),
        "rotation": rotation,
        "two_stream_frames_per_s": F / (walls[True] / K) if True in walls else None,
        "two_stream_joined_frames_per_s": F / (joined_wall / K) if joined_wall else None,
        "one_stream_frames_per_s": F / (walls[False] / K) if False in walls else None,
        "eager_two_stream_frames_per_s": F / (eager[True][0] / K) if True in eager else None,
        "eager_one_stream_frames_per_s": F / (eager[False][0] / K) if False in eager else None,
        "timing": graph_note or ("value: HIP graph replay of the faster of the two-stream and one-stream steps, "
                                 "step k on copy k mod rotation.copies of the batch (inputs and outputs), so its "
                                 "data comes from HBM where the copies exceed the caches; two streams: the "
                                 "clustering launches of a graph's steps in order on one stream, the density "
                                 "launches on the other, joined once per graph of up to 10 steps "
                                 "(two_stream_joined_frames_per_s: joined after every step instead); warm_value: "
                                 "the same replays on one copy; two/one_stream_frames_per_s: rotated, per mode; kernel "
                                 "durations (per_launch_us, roofline): HIP events around each launch in an eager "
                                 "one-stream run, each launch after a write of flush_mb MiB that evicts L2 and "
                                 "the memory-side cache (warm_per_launch_us: back to back; "
                                 "two_stream_per_launch_us: back to back, the two kernels on two streams)"),
        "flush_mb": args.flush_mb,
        "roofline": roof,
        "kernels": {"cluster_frames": cl, "density_frames": de, "heatmap_frames": he, "roi_filter_frames": ro,
                    "drinker_proximity_frames": dr, "mask_components_frames": ma},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        out["cpu_baseline"] = cpu_baseline(xy, off, w, args.cpu_budget_s, args.cpu_one_thread_s)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

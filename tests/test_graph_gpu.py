"""Both entry points captured in one HIP graph (two streams), replayed several
times with eager work in between; every replay must equal the eager outputs
bit for bit (both paths are deterministic)."""

import numpy as np
import pytest
import torch

import paper_2512_07009_amd as flock
from paper_2512_07009_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _batches():
    xy, off, w = wl.generate("batch64x2000_1080p", n_frames=16)
    yield "headline frames", xy, off, w, int(np.diff(off).max())
    rng = np.random.default_rng(3)
    big = np.stack([rng.integers(0, 16 * 3840, 24000), rng.integers(0, 16 * 2160, 24000)], 1).astype(np.int32)
    small = rng.integers(0, 16 * 1000, (500, 2)).astype(np.int32)
    xy2, off2 = wl.pack([small, big, small[:70]])
    # max_frame_points 0: the large frame takes the multi-workgroup path; one
    # frame of few birds splits density into bird slices with a workspace
    yield "large frame", xy2, off2, wl.WORKLOADS["house30000_4k"], 0


@pytest.mark.parametrize("case", range(2))
def test_graph_replays_match_eager(case):
    name, xy, off, w, mfp = list(_batches())[case]
    dev = torch.device("cuda")
    F, T = len(off) - 1, xy.shape[0]
    dxy, doff = torch.from_numpy(xy).to(dev), torch.from_numpy(off).to(dev)
    labels = torch.empty(T, dtype=torch.int32, device=dev)
    kind = torch.empty(T, dtype=torch.uint8, device=dev)
    ncl = torch.empty(F, dtype=torch.int32, device=dev)
    dens = torch.empty((F, w.grid_h, w.grid_w), dtype=torch.float32, device=dev)
    main, side = torch.cuda.Stream(dev), torch.cuda.Stream(dev)

    def step():
        fork = torch.cuda.Event()
        fork.record(main)
        side.wait_event(fork)
        flock.cluster_frames(dxy, doff, w.eps_px, w.min_pts, mfp, out=(labels, kind, ncl), stream=main)
        flock.density_frames(dxy, doff, w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px, mfp, out=dens,
                             stream=side)
        join = torch.cuda.Event()
        join.record(side)
        main.wait_event(join)

    with torch.cuda.stream(main):
        step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (labels, kind, ncl, dens)]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=main):
        step()
    torch.cuda.synchronize()

    other_xy, other_off = wl.random_batch(9, 5, 300)
    oxy, ooff = torch.from_numpy(other_xy).to(dev), torch.from_numpy(other_off).to(dev)
    for rep in range(4):
        for t, v in ((labels, -7), (kind, 9), (ncl, -3), (dens, -1.0)):
            t.fill_(v)
        # eager work of the program between replays
        flock.cluster_frames(oxy, ooff, 40.0, 4, 300)
        flock.density_frames(oxy, ooff, 1920, 1080, 128, 72, 30.0, 300)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, want, what in zip((labels, kind, ncl, dens), ref, ("labels", "kind", "n_clusters", "density")):
            assert torch.equal(got, want), f"{name}: replay {rep} {what} differs from eager"


@pytest.mark.parametrize("case", range(2))
def test_graph_pipelined_steps_match_eager(case):
    """Several steps in one graph on two streams joined once at its end (the
    clustering launches of the steps in order on one stream, the density
    launches on the other), each step on its own copy of the batch; every
    replay, with eager work in between, equals the eager outputs of every
    copy bit for bit."""
    name, xy, off, w, mfp = list(_batches())[case]
    dev = torch.device("cuda")
    F, T = len(off) - 1, xy.shape[0]
    steps = 3
    bufs = []
    for k in range(steps):
        bufs.append({"xy": torch.from_numpy(xy).to(dev), "off": torch.from_numpy(off).to(dev),
                     "labels": torch.empty(T, dtype=torch.int32, device=dev),
                     "kind": torch.empty(T, dtype=torch.uint8, device=dev),
                     "ncl": torch.empty(F, dtype=torch.int32, device=dev),
                     "dens": torch.empty((F, w.grid_h, w.grid_w), dtype=torch.float32, device=dev)})
    outs = ("labels", "kind", "ncl", "dens")
    main, side = torch.cuda.Stream(dev), torch.cuda.Stream(dev)
    with torch.cuda.stream(main):
        b = bufs[0]
        flock.cluster_frames(b["xy"], b["off"], w.eps_px, w.min_pts, mfp, out=(b["labels"], b["kind"], b["ncl"]),
                             stream=main)
        flock.density_frames(b["xy"], b["off"], w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px, mfp,
                             out=b["dens"], stream=main)
    torch.cuda.synchronize()
    ref = [bufs[0][o].clone() for o in outs]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=main):
        fork = torch.cuda.Event()
        fork.record(main)
        side.wait_event(fork)
        for b in bufs:
            flock.cluster_frames(b["xy"], b["off"], w.eps_px, w.min_pts, mfp,
                                 out=(b["labels"], b["kind"], b["ncl"]), stream=main)
            flock.density_frames(b["xy"], b["off"], w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px, mfp,
                                 out=b["dens"], stream=side)
        join = torch.cuda.Event()
        join.record(side)
        main.wait_event(join)
    torch.cuda.synchronize()

    other_xy, other_off = wl.random_batch(9, 5, 300)
    oxy, ooff = torch.from_numpy(other_xy).to(dev), torch.from_numpy(other_off).to(dev)
    for rep in range(4):
        for b in bufs:
            for o, v in zip(outs, (-7, 9, -3, -1.0)):
                b[o].fill_(v)
        flock.cluster_frames(oxy, ooff, 40.0, 4, 300)
        flock.density_frames(oxy, ooff, 1920, 1080, 128, 72, 30.0, 300)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, b in enumerate(bufs):
            for o, want in zip(outs, ref):
                assert torch.equal(b[o], want), f"{name}: replay {rep} step {k} {o} differs from eager"


def test_graph_replays_match_eager_analytics():
    """heatmap_frames, roi_filter_frames, drinker_proximity_frames and
    mask_components_frames captured in one graph, replayed several times with
    eager work in between; every replay equals the eager outputs bit for bit."""
    dev = torch.device("cuda")
    xy, off, w = wl.generate("batch64x2000_1080p", n_frames=8)
    F, T = len(off) - 1, xy.shape[0]
    dxy, doff = torch.from_numpy(xy).to(dev), torch.from_numpy(off).to(dev)
    grids = torch.from_numpy(wl.heat_grids(21, 6, 72, 128)).to(dev)
    prob = torch.from_numpy(wl.bird_masks(22, 3, 200, 300, n_birds=150)).to(dev)
    Wq, Hq = 16 * w.width_px, 16 * w.height_px
    poly = [[0, 0], [Wq // 8, 0], [Wq // 6, Hq // 2], [Wq // 8, Hq], [0, Hq]]
    lines = [[Wq // 10, Hq // 4, 9 * Wq // 10, Hq // 4], [Wq // 10, 3 * Hq // 4, 9 * Wq // 10, 3 * Hq // 4]]
    cap = flock.mask_capacity(3, 200, 300, 8)
    e = lambda *shape, dt=torch.int32: torch.empty(*shape, dtype=dt, device=dev)
    hout = {"labels": e((6, 72, 128)), "n_components": e(6), "entropy": e(6, dt=torch.float64),
            "degree": e(6, dt=torch.float64), "comp_cells": e((6, 72, 128)),
            "comp_mass": e((6, 72, 128), dt=torch.float64)}
    rout = {"counts": e(F), "xy": e((T, 2)), "offsets": e(F + 1), "index": e(T)}
    dout = {"drinking": e(T, dt=torch.uint8), "line": e(T), "counts": e(F)}
    mout = {"labels": e((3, 200, 300)), "n_components": e(3), "offsets": e(4), "label": e(cap), "area": e(cap),
            "box": e((cap, 4)), "centroid": e((cap, 2), dt=torch.float64), "xy": e((cap, 2)),
            "score": e(cap, dt=torch.float32)}
    main = torch.cuda.Stream(dev)

    def step():
        flock.heatmap_frames(grids, 225.0, 2e-4, 8, out=hout, stream=main)
        flock.roi_filter_frames(dxy, doff, poly, out=rout, stream=main)
        flock.drinker_proximity_frames(dxy, doff, lines, 320, out=dout, stream=main)
        flock.mask_components_frames(prob, 0.5, 8, capacity=cap, out=mout, stream=main)

    outs = [t for d in (hout, rout, dout, mout) for t in d.values()]
    with torch.cuda.stream(main):
        step()
    torch.cuda.synchronize()
    # rows past the written counts of the capacity-sized outputs are not outputs
    kept, ndet = int(rout["offsets"][-1]), int(mout["offsets"][-1])
    valid = {id(rout["xy"]): kept, id(rout["index"]): kept}
    for k in ("label", "area", "box", "centroid", "xy", "score"):
        valid[id(mout[k])] = ndet
    outs = [t[:valid[id(t)]] if id(t) in valid else t for t in outs]
    ref = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=main):
        step()
    torch.cuda.synchronize()
    other = torch.from_numpy(wl.bird_masks(23, 2, 90, 130, n_birds=40)).to(dev)
    for rep in range(4):
        for t in outs:
            t.fill_(7)
        # eager work of the program between replays
        flock.mask_components_frames(other, 0.4, 4)
        flock.heatmap_frames(grids[:2].contiguous(), 100.0, 1e-4, 4)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (got, want) in enumerate(zip(outs, ref)):
            assert torch.equal(got, want), f"replay {rep}: output {i} differs from eager"

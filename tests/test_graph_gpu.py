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

"""GPU parity of roi_filter_frames (through the C ABI) against the CPU oracle.

Bar: bit-exact counts, CSR offsets, kept coordinates and input indices.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2512_07009_amd as flock
from paper_2512_07009_amd import workloads as wl

pytestmark = pytest.mark.gpu


def run(xy, off, poly, with_index=True):
    dxy = torch.from_numpy(np.ascontiguousarray(xy)).cuda()
    doff = torch.from_numpy(np.ascontiguousarray(off)).cuda()
    out = flock.roi_filter_frames(dxy, doff, poly, with_index=with_index)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}


def check(xy, off, poly, tag="", with_index=True):
    got = run(xy, off, poly, with_index)
    ref = oracle.roi_filter(xy, off, poly)
    k = int(ref["offsets"][-1])
    assert np.array_equal(got["counts"], ref["counts"]), f"{tag} counts"
    assert np.array_equal(got["offsets"], ref["offsets"]), f"{tag} offsets"
    assert np.array_equal(got["xy"][:k], ref["xy"]), f"{tag} xy"
    if with_index:
        assert np.array_equal(got["index"][:k], ref["index"]), f"{tag} index"
    return got, ref


W, H = 1920 * 16, 1080 * 16


def polygons():
    rng = np.random.default_rng(4)
    rect = [[W // 10, H // 5], [W // 2, H // 5], [W // 2, 4 * H // 5], [W // 10, 4 * H // 5]]
    wall = [[0, 0], [W // 8, 0], [W // 6, H // 2], [W // 8, H], [0, H]]            # strip near a wall
    t = np.linspace(0, 2 * np.pi, 21)[:-1]
    r = np.where(np.arange(20) % 2 == 0, 0.45, 0.2) * H
    star = np.stack([W / 2 + r * np.cos(t), H / 2 + r * np.sin(t)], 1).astype(np.int64).tolist()
    t64 = np.linspace(0, 2 * np.pi, 65)[:-1]
    circle64 = np.stack([W / 3 + 0.3 * H * np.cos(t64), H / 2 + 0.3 * H * np.sin(t64)], 1).astype(np.int64).tolist()
    tri = rng.integers(0, H, (3, 2)).tolist()
    return {"rect": rect, "wall": wall, "star": star, "circle64": circle64, "triangle": tri,
            "rect_reversed": rect[::-1]}


@pytest.mark.parametrize("name", ["rect", "wall", "star", "circle64", "triangle", "rect_reversed"])
def test_random_batches_gpu(name):
    poly = polygons()[name]
    for seed in range(3):
        xy, off = wl.random_batch(900 + seed, 20, 800)
        check(xy, off, poly, tag=f"{name} seed {seed}")


def test_points_on_edges_and_vertices_gpu():
    """Birds and vertices on one lattice: many birds sit exactly on edges,
    vertices and the test ray through a vertex."""
    step = 64
    gx, gy = np.meshgrid(np.arange(0, 40 * step, step), np.arange(0, 30 * step, step))
    pts = np.stack([gx.ravel(), gy.ravel()], 1).astype(np.int32)
    xy, off = wl.pack([pts, pts[::3], pts[:0], pts[5:9]])
    polys = [[[0, 0], [20 * step, 0], [20 * step, 10 * step], [10 * step, 10 * step], [10 * step, 20 * step],
              [0, 20 * step]],
             [[5 * step, 5 * step], [25 * step, 10 * step], [5 * step, 15 * step]],
             [[0, 0], [10 * step, 0], [10 * step, 4 * step], [6 * step, 4 * step], [4 * step, 8 * step],
              [0, 8 * step]]]
    for i, p in enumerate(polys):
        check(xy, off, p, tag=f"lattice poly {i}")
        check(xy, off, p, tag=f"lattice poly {i} no index", with_index=False)


def test_all_in_all_out_and_empty_gpu():
    xy, off = wl.random_batch(77, 10, 500)
    everything = [[-16, -16], [W + 16, -16], [W + 16, H + 16], [-16, H + 16]]
    got, _ = check(xy, off, everything, tag="all in")
    assert int(got["offsets"][-1]) == xy.shape[0]
    got, _ = check(xy, off, [[-100, -100], [-50, -100], [-50, -50]], tag="all out")
    assert int(got["offsets"][-1]) == 0
    e_xy, e_off = wl.pack([np.zeros((0, 2), np.int32)] * 3)
    check(e_xy, e_off, everything, tag="empty frames")


@pytest.mark.parametrize("name", ["batch64x2000_1080p", "batch256xpoisson8000_4k", "house30000_4k",
                                  "stream1800x5000_1080p"])
def test_workloads_gpu(name):
    xy, off, w = wl.generate(name)
    Wq, Hq = 16 * w.width_px, 16 * w.height_px
    wall = [[0, 0], [Wq // 8, 0], [Wq // 6, Hq // 2], [Wq // 8, Hq], [0, Hq]]
    check(xy, off, wall, tag=name)


def test_deterministic_gpu():
    xy, off = wl.random_batch(31, 12, 900)
    poly = polygons()["star"]
    a = run(xy, off, poly)
    b = run(xy, off, poly)
    k = int(a["offsets"][-1])
    for key in ("counts", "offsets"):
        assert np.array_equal(a[key], b[key])
    assert np.array_equal(a["xy"][:k], b["xy"][:k]) and np.array_equal(a["index"][:k], b["index"][:k])

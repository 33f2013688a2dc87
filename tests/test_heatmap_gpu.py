"""GPU parity of heatmap_frames (through the C ABI) against the CPU oracle.

Bars: labels, n_components and comp_cells bit-exact (the hot test is the same
float32 comparison on both sides); entropy within 1e-9 absolute; degree
within 1e-12 relative; comp_mass within 1e-9 relative (fixed-point sums on
the device, fp64 sums in the oracle).
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2512_07009_amd as flock
from paper_2512_07009_amd import workloads as wl

pytestmark = pytest.mark.gpu


def run(grids, area, thr, conn):
    d = torch.from_numpy(np.ascontiguousarray(grids, dtype=np.float32)).cuda()
    out = flock.heatmap_frames(d, area, thr, conn)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def check(grids, area, thr, conn, tag=""):
    got = run(grids, area, thr, conn)
    ref = oracle.heatmap_frames(grids, area, thr, conn)
    for k in ("labels", "n_components", "comp_cells"):
        if not np.array_equal(got[k], ref[k]):
            bad = np.argwhere(got[k] != ref[k])[:5]
            raise AssertionError(f"{tag} {k} differs at {bad.tolist()}")
    np.testing.assert_allclose(got["entropy"], ref["entropy"], rtol=0, atol=1e-9, err_msg=f"{tag} entropy")
    np.testing.assert_allclose(got["degree"], ref["degree"], rtol=1e-12, atol=0, err_msg=f"{tag} degree")
    np.testing.assert_allclose(got["comp_mass"], ref["comp_mass"], rtol=1e-9, atol=0, err_msg=f"{tag} mass")
    return got


SHAPES = [(1, 1, 1), (2, 3, 5), (3, 33, 31), (2, 64, 64), (4, 45, 70), (3, 72, 128), (1, 131, 257)]


@pytest.fixture(params=["auto", "tiled"])
def path(request, monkeypatch):
    """auto: grids that fit in LDS take the one-workgroup-per-frame kernel;
    tiled: FLOCK_HEATMAP_PATH=tiled forces the tiled kernels for every grid."""
    if request.param == "tiled":
        monkeypatch.setenv("FLOCK_HEATMAP_PATH", "tiled")
    return request.param


@pytest.mark.parametrize("conn", [4, 8])
@pytest.mark.parametrize("F,h,w", SHAPES)
def test_random_grids_gpu(F, h, w, conn, path):
    g = wl.heat_grids(100 * h + w + conn, F, h, w)
    pos = g[g > 0]
    for q in (0.3, 0.7, 0.95):
        thr = float(np.quantile(pos, q)) if pos.size else 1e-4
        check(g, 3.5, thr, conn, tag=f"{F}x{h}x{w} q{q}")


@pytest.mark.parametrize("conn", [4, 8])
def test_tile_boundaries_gpu(conn, path):
    """Checkerboards and stripes put components across every tile edge and
    corner; one all-hot frame is a single component spanning all tiles."""
    h, w = 70, 100
    yy, xx = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    frames = [((xx + yy) % 2 == 0), (xx % 32 == 31) | (yy % 32 == 0), np.ones((h, w), bool),
              ((xx // 2 + yy // 2) % 2 == 0), (xx == yy) | (xx == w - 1 - yy)]
    g = np.stack([np.where(m, 1.0, 0.25) for m in frames]).astype(np.float32)
    check(g, 1.0, 0.5, conn, tag="patterns")


def test_edge_cases_gpu(path):
    g = np.zeros((3, 40, 50), np.float32)
    g[1] = 0.01
    g[2, 5, 7] = 0.02
    check(g, 2.0, 0.015, 8, tag="zero/flat/point")
    got = check(g, 2.0, 1.0, 8, tag="above max")
    assert (got["labels"] == -1).all() and (got["n_components"] == 0).all()
    one = np.full((1, 1, 1), 0.5, np.float32)
    got = check(one, 4.0, 0.5, 4, tag="1x1")
    assert got["labels"][0, 0, 0] == 0 and got["comp_mass"][0, 0, 0] == 2.0


@pytest.mark.parametrize("name", ["batch64x2000_1080p", "batch256xpoisson8000_4k", "house30000_4k",
                                  "stream1800x5000_1080p"])
def test_workload_grid_shapes_gpu(name):
    """Full batch shapes of the workloads (frames x grid), synthetic grids."""
    w = wl.WORKLOADS[name]
    F = min(w.n_frames, 400)
    g = wl.heat_grids(w.seed, F, w.grid_h, w.grid_w, n_blobs=12, empty_frac=0.0 if F == 1 else 0.1)
    pos = g[g > 0]
    area = (w.width_px / w.grid_w) * (w.height_px / w.grid_h)
    check(g, area, float(np.quantile(pos, 0.8)), 8, tag=name)


def test_deterministic_gpu(path):
    g = wl.heat_grids(7, 6, 90, 140)
    thr = float(np.quantile(g[g > 0], 0.6))
    a = run(g, 1.0, thr, 8)
    b = run(g, 1.0, thr, 8)
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k

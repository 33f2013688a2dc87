"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: labels, kinds and n_clusters bit-exact; density within a relative L-inf
error of 1e-3 of each frame's maximum (exact zeros for empty frames).
"""

import os

import numpy as np
import pytest
import torch

import oracle
import paper_2512_07009_amd as flock
from paper_2512_07009_amd import workloads as wl

pytestmark = pytest.mark.gpu

DENSITY_RTOL_OF_MAX = 1e-3


def dev_batch(xy, off):
    return (torch.from_numpy(np.ascontiguousarray(xy)).to("cuda"),
            torch.from_numpy(np.ascontiguousarray(off)).to("cuda"))


def max_count(off):
    return int(np.diff(off).max()) if len(off) > 1 else 0


def run_cluster(xy, off, eps_q, min_pts, max_fp=None):
    dxy, doff = dev_batch(xy, off)
    labels, kind, ncl = flock.cluster_frames(dxy, doff, eps_q / 16.0, min_pts,
                                             max_count(off) if max_fp is None else max_fp)
    torch.cuda.synchronize()
    return labels.cpu().numpy(), kind.cpu().numpy(), ncl.cpu().numpy()


def run_density(xy, off, w, h, gx, gy, sigma, max_fp=None):
    dxy, doff = dev_batch(xy, off)
    d = flock.density_frames(dxy, doff, w, h, gx, gy, sigma,
                             max_count(off) if max_fp is None else max_fp)
    torch.cuda.synchronize()
    return d.cpu().numpy()


def sub_batch(xy, off, frames):
    parts = [xy[off[f]:off[f + 1]] for f in frames]
    return wl.pack(parts)


def assert_cluster_equal(got, xy, off, eps_q, min_pts, frames=None, tag=""):
    labels, kind, ncl = got
    if frames is None:
        frames = list(range(len(off) - 1))
    sxy, soff = sub_batch(xy, off, frames)
    rl, rk, rn = oracle.cluster_frames(sxy, soff, eps_q, min_pts)
    for j, f in enumerate(frames):
        b, e = off[f], off[f + 1]
        sb, se = soff[j], soff[j + 1]
        if not np.array_equal(kind[b:e], rk[sb:se]):
            bad = np.nonzero(kind[b:e] != rk[sb:se])[0][:5]
            raise AssertionError(f"{tag} frame {f}: kind differs at {bad.tolist()}")
        if not np.array_equal(labels[b:e], rl[sb:se]):
            bad = np.nonzero(labels[b:e] != rl[sb:se])[0][:5]
            raise AssertionError(f"{tag} frame {f}: labels differ at {bad.tolist()} "
                                 f"got {labels[b:e][bad].tolist()} want {rl[sb:se][bad].tolist()}")
        assert ncl[f] == rn[j], f"{tag} frame {f}: n_clusters {ncl[f]} != {rn[j]}"


def assert_density_close(got, ref, counts=None, sigma=None, tag=""):
    """max |got - ref| <= 1e-3 * max(ref) per frame.

    With counts and sigma given, an absolute floor of n_f * c * 2^-24 is added
    (c = 1 / (2 pi sigma^2)): fp16 factors carry an absolute error of up to
    2^-25 each in their subnormal range, so a frame whose whole density lies
    below that range (every bird > 5.9 sigma from every cell centre) is only
    resolved to that floor.  The five workloads are checked without it.
    """
    worst = 0.0
    for f in range(ref.shape[0]):
        m = ref[f].max()
        if m == 0.0:
            assert (got[f] == 0).all(), f"{tag} frame {f}: empty frame not exactly zero"
            continue
        floor = 0.0
        if counts is not None:
            floor = counts[f] * 2.0 ** -24 / (2.0 * np.pi * sigma * sigma)
        diff = np.abs(got[f].astype(np.float64) - ref[f]).max()
        err = diff / m
        worst = max(worst, err if diff > floor else 0.0)
        assert diff <= DENSITY_RTOL_OF_MAX * m + floor, f"{tag} frame {f}: rel L-inf error {err:.3e}"
    return worst


# ---------------------------------------------------------------------------
# clustering
# ---------------------------------------------------------------------------

def test_handbuilt_gpu(handbuilt):
    for case in handbuilt:
        xy, off = wl.pack([np.asarray(f, np.int32).reshape(-1, 2) for f in case["frames"]])
        labels, kind, ncl = run_cluster(xy, off, case["eps_q"], case["min_pts"])
        for f in range(len(case["frames"])):
            assert labels[off[f]:off[f + 1]].tolist() == case["labels"][f], case["name"]
            assert kind[off[f]:off[f + 1]].tolist() == case["kind"][f], case["name"]
        assert ncl.tolist() == case["n_clusters"], case["name"]


RANDOM_PARAMS = [(640, 4), (640, 1), (400, 6), (960, 5), (1, 2), (0, 2), (32766, 3), (100, 3)]


@pytest.mark.parametrize("eps_q,min_pts", RANDOM_PARAMS)
def test_random_batches_gpu(eps_q, min_pts):
    for seed in range(3):
        xy, off = wl.random_batch(1000 * eps_q + 10 * min_pts + seed, 24, 700)
        got = run_cluster(xy, off, eps_q, min_pts)
        assert_cluster_equal(got, xy, off, eps_q, min_pts, tag=f"seed {seed}")


@pytest.mark.parametrize("max_fp", [8, 100])
def test_inplace_path_gpu(max_fp):
    """Frames above max_frame_points take the in-place path; results are identical."""
    xy, off = wl.random_batch(77 + max_fp, 16, 600)
    got = run_cluster(xy, off, 640, 4, max_fp=max_fp)
    assert_cluster_equal(got, xy, off, 640, 4, tag=f"max_fp {max_fp}")


def test_frame_above_lds_capacity_gpu():
    rng = np.random.default_rng(5)
    big = np.stack([rng.integers(0, 16 * 800, 12000), rng.integers(0, 16 * 600, 12000)], 1).astype(np.int32)
    small = rng.integers(0, 16 * 500, (300, 2)).astype(np.int32)
    xy, off = wl.pack([small, big, small[:50]])
    got = run_cluster(xy, off, 160, 5, max_fp=0)
    assert_cluster_equal(got, xy, off, 160, 5, tag="big frame")


def _lattice_frame(seed, nx, ny, eps_q):
    """One point per cell of side floor(E / sqrt 2) on an nx x ny lattice,
    jittered inside its cell: every point is a core cell of its own."""
    side = int(np.floor(np.sqrt(eps_q * eps_q / 2.0)))
    while 2 * (side + 1) ** 2 <= eps_q * eps_q:
        side += 1
    rng = np.random.default_rng(seed)
    gx, gy = np.meshgrid(np.arange(nx), np.arange(ny))
    pts = np.stack([gx.ravel() * side, gy.ravel() * side], 1)
    jit = rng.integers(0, max(side // 4, 1), pts.shape)
    jit[0] = 0  # the bounding-box corner stays on a cell corner
    return (pts + jit).astype(np.int32)


def test_union_many_core_cells_gpu():
    """A frame with more core cells than the register-held union stage takes
    (one point per cell, 4500 cells) goes through the general stage."""
    big = _lattice_frame(3, 75, 60, 640)
    small = _lattice_frame(4, 20, 10, 640)
    xy, off = wl.pack([small, big, small[:50]])
    got = run_cluster(xy, off, 640, 4)
    assert_cluster_equal(got, xy, off, 640, 4, tag="lattice")


def test_compact_plan_gpu(monkeypatch):
    """More frames than compute units, none above 5120 points: two clustering
    workgroups share a compute unit, with half its LDS each.  The batch mixes
    random frames (ties, duplicates, empty frames), 4K-wide frames of 5000
    points whose cell grid exceeds the compact cell table (coarsened grid),
    and a lattice frame with 2660 core cells.  Results equal the oracle and
    the one-workgroup-per-compute-unit plan (FLOCK_CLUSTER_COMPACT=0)."""
    n_cus = torch.cuda.get_device_properties(0).multi_processor_count
    rng = np.random.default_rng(11)
    xy_r, off_r = wl.random_batch(4242, n_cus + 40, 400)
    frames = [xy_r[off_r[f]:off_r[f + 1]] for f in range(len(off_r) - 1)]
    wide = [np.stack([rng.integers(0, 16 * 3840, 5000), rng.integers(0, 16 * 2160, 5000)], 1).astype(np.int32)
            for _ in range(3)]
    frames = frames[:100] + wide + [_lattice_frame(7, 70, 38, 640)] + frames[100:]
    xy, off = wl.pack(frames)
    assert len(off) - 1 > n_cus and max_count(off) <= 5120
    got = run_cluster(xy, off, 640, 4)
    assert_cluster_equal(got, xy, off, 640, 4, tag="compact")
    monkeypatch.setenv("FLOCK_CLUSTER_COMPACT", "0")
    ref = run_cluster(xy, off, 640, 4)
    for a, b in zip(got, ref):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("eps_q,min_pts", [(640, 4), (960, 5), (400, 6)])
def test_union_lds_stage_gpu(eps_q, min_pts, monkeypatch):
    """FLOCK_CLUSTER_UNION=lds forces the general union stage for every frame."""
    monkeypatch.setenv("FLOCK_CLUSTER_UNION", "lds")
    for seed in range(2):
        xy, off = wl.random_batch(31 * eps_q + seed, 24, 900)
        got = run_cluster(xy, off, eps_q, min_pts)
        assert_cluster_equal(got, xy, off, eps_q, min_pts, tag=f"seed {seed}")
    xy, off, w = wl.generate("batch64x2000_1080p")
    frames = [0, 1, 2, 3]
    sxy, soff = sub_batch(xy, off, frames)
    got = run_cluster(sxy, soff, w.eps_q, w.min_pts)
    assert_cluster_equal(got, sxy, soff, w.eps_q, w.min_pts, tag="batch64x2000_1080p")


@pytest.mark.parametrize("max_fp", [0, 20000])
def test_large_frame_path_gpu(max_fp):
    """Frames above the on-chip capacity use the multi-workgroup path: dense
    frames, a frame whose cell grid is coarsened (huge spread, small eps),
    and small frames around them."""
    rng = np.random.default_rng(11)
    dense = np.stack([rng.normal(20000, 3000, 15000), rng.normal(15000, 2500, 15000)], 1)
    dense = np.clip(np.round(dense), 0, 60000).astype(np.int32)
    spread = rng.integers(0, 1 << 20, (12000, 2)).astype(np.int32)
    spread[:3000] = spread[3000:6000] + rng.integers(-8, 9, (3000, 2)).astype(np.int32)
    spread = np.clip(spread, 0, None)
    small = rng.integers(0, 16 * 300, (500, 2)).astype(np.int32)
    xy, off = wl.pack([small, dense, np.zeros((0, 2), np.int32), spread, small[:40]])
    for eps_q, min_pts in ((160, 5), (16, 2)):
        got = run_cluster(xy, off, eps_q, min_pts, max_fp=max_fp)
        assert_cluster_equal(got, xy, off, eps_q, min_pts, tag=f"large eps {eps_q} max_fp {max_fp}")


def test_workspace_too_small_gpu():
    xy, off = wl.random_batch(1, 3, 50)
    dxy, doff = dev_batch(xy, off)
    lib = flock.lib()
    need = lib.cluster_frames_workspace(3, xy.shape[0], 0)
    assert need > 0
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    labels = torch.empty(xy.shape[0], dtype=torch.int32, device="cuda")
    kind = torch.empty(xy.shape[0], dtype=torch.uint8, device="cuda")
    import ctypes
    st = lib.cluster_frames(ctypes.c_void_p(dxy.data_ptr()), ctypes.c_void_p(doff.data_ptr()), 3,
                            xy.shape[0], 0, 640, 4, ctypes.c_void_p(labels.data_ptr()),
                            ctypes.c_void_p(kind.data_ptr()), None, ctypes.c_void_p(ws.data_ptr()),
                            need - 1, None)
    assert st == flock.binding.FLOCK_ENOMEM
    # and with NULL workspace the library allocates stream-ordered scratch itself
    st = lib.cluster_frames(ctypes.c_void_p(dxy.data_ptr()), ctypes.c_void_p(doff.data_ptr()), 3,
                            xy.shape[0], 0, 640, 4, ctypes.c_void_p(labels.data_ptr()),
                            ctypes.c_void_p(kind.data_ptr()), None, None, 0, None)
    assert st == 0
    torch.cuda.synchronize()
    rl, rk, _ = oracle.cluster_frames(xy, off, 640, 4)
    assert np.array_equal(labels.cpu().numpy(), rl) and np.array_equal(kind.cpu().numpy(), rk)


def test_lattice_ties_gpu():
    frames = [wl.lattice_frame(30, 20, 640), wl.lattice_frame(25, 25, 452, 1000, 2000),
              wl.lattice_frame(10, 10, 641), np.concatenate([wl.lattice_frame(12, 12, 384),
                                                             wl.lattice_frame(12, 12, 512, 384, 0)])]
    xy, off = wl.pack(frames)
    for min_pts in (2, 3, 5, 6):
        got = run_cluster(xy, off, 640, min_pts)
        assert_cluster_equal(got, xy, off, 640, min_pts, tag=f"lattice minPts {min_pts}")


def test_single_large_frame_gpu():
    """A batch of one frame above the on-chip capacity runs the
    multi-workgroup path alone (no on-chip launch).  With offsets that break
    the contract, a frame past total gets n_clusters -1 and a frame shorter
    than total is still clustered."""
    rng = np.random.default_rng(21)
    big = np.stack([rng.integers(0, 16 * 900, 12000), rng.integers(0, 16 * 700, 12000)], 1).astype(np.int32)
    xy, off = wl.pack([big])
    got = run_cluster(xy, off, 160, 5, max_fp=0)
    assert_cluster_equal(got, xy, off, 160, 5, tag="one large frame")
    _, _, ncl = run_cluster(xy, np.array([0, 13000], np.int32), 160, 5, max_fp=0)
    assert ncl[0] == -1
    short = np.array([0, 500], np.int32)
    got = run_cluster(xy, short, 160, 5, max_fp=0)
    assert_cluster_equal(got, xy, short, 160, 5, tag="frame shorter than total")


def test_large_frame_one_component_gpu():
    """Frames above the on-chip capacity whose cores form one component
    spanning the whole frame (a jittered lattice, every cell of the grid
    holding cores): many concurrent hooks meet in one tree of the global
    forest, and the farther cell pairs all find their cells joined.  Beside
    them, one frame of many small components (a sparse lattice of tight
    groups)."""
    rng = np.random.default_rng(33)
    g = np.stack(np.meshgrid(np.arange(150), np.arange(100)), -1).reshape(-1, 2) * 96
    one = (g + rng.integers(0, 48, g.shape)).astype(np.int32)           # 15000 points, spacing 6 px
    c = np.stack(np.meshgrid(np.arange(40), np.arange(30)), -1).reshape(-1, 2) * 16 * 40
    groups = (np.repeat(c, 10, 0) + rng.integers(0, 16 * 6, (c.shape[0] * 10, 2))).astype(np.int32)  # 12000
    xy, off = wl.pack([one, groups])
    for eps_q, min_pts in ((160, 4), (200, 6)):
        got = run_cluster(xy, off, eps_q, min_pts, max_fp=0)
        assert_cluster_equal(got, xy, off, eps_q, min_pts, tag=f"one component eps {eps_q}")
        ncl = got[2]
        assert ncl[0] == 1, ncl


def test_large_frame_thin_grids_gpu():
    """Frames above the on-chip capacity whose cell grids are thinner than
    the 16 x 8-cell blocks of the tiled unions: one row of cells, three
    columns of cells, and a grid whose width and height leave partial
    blocks on both edges."""
    rng = np.random.default_rng(44)
    eps_q, min_pts = 200, 4  # cells of 141 quanta
    row = np.stack([rng.integers(0, 2_000_000, 12000), rng.integers(0, 120, 12000)], 1).astype(np.int32)
    col = np.stack([rng.integers(0, 400, 12000), rng.integers(0, 1_000_000, 12000)], 1).astype(np.int32)
    odd = np.stack([rng.integers(0, 141 * 137, 12000), rng.integers(0, 141 * 73, 12000)], 1).astype(np.int32)
    xy, off = wl.pack([row, col, odd])
    got = run_cluster(xy, off, eps_q, min_pts, max_fp=0)
    assert_cluster_equal(got, xy, off, eps_q, min_pts, tag="thin grids")


def test_bad_offsets_do_not_fault_gpu():
    xy = np.zeros((10, 2), np.int32)
    off = np.array([0, 5, 3, 10, 12], np.int32)   # frame 1 negative, frame 3 past total
    labels, kind, ncl = run_cluster(xy, off, 640, 2, max_fp=10)
    assert ncl[1] == -1 and ncl[3] == -1
    assert ncl[0] == 1


def test_validate_mode_rejects_bad_offsets_gpu():
    xy = np.zeros((10, 2), np.int32)
    off = np.array([0, 5, 3, 10], np.int32)
    os.environ["FLOCK_VALIDATE"] = "1"
    try:
        with pytest.raises(ValueError, match="decrease"):
            run_cluster(xy, off, 640, 2)
        xy2, off2 = wl.random_batch(3, 4, 50)
        got = run_cluster(xy2, off2, 640, 3)
        assert_cluster_equal(got, xy2, off2, 640, 3)
    finally:
        del os.environ["FLOCK_VALIDATE"]


def test_determinism_and_batch_independence_gpu():
    xy, off, w = wl.generate("batch64x2000_1080p", n_frames=8)
    a = run_cluster(xy, off, w.eps_q, w.min_pts)
    b = run_cluster(xy, off, w.eps_q, w.min_pts)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    # frame 3 alone gives the same labels as inside the batch
    sxy, soff = sub_batch(xy, off, [3])
    alone = run_cluster(sxy, soff, w.eps_q, w.min_pts)
    assert np.array_equal(alone[0], a[0][off[3]:off[4]])
    assert np.array_equal(alone[1], a[1][off[3]:off[4]])


def test_permutation_invariance_gpu():
    xy, off, w = wl.generate("batch64x2000_1080p", n_frames=1)
    base_l, base_k, base_n = run_cluster(xy, off, w.eps_q, w.min_pts)
    perm = np.random.default_rng(1).permutation(xy.shape[0])
    pl, pk, pn = run_cluster(xy[perm], off, w.eps_q, w.min_pts)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(len(perm))
    assert np.array_equal(pk[inv], base_k) and pn[0] == base_n[0]
    mapped = np.where(pl[inv] >= 0, perm[np.maximum(pl[inv], 0)], -1)
    canon = {}
    for i in np.nonzero(base_k == 2)[0]:
        canon.setdefault(mapped[i], i)
    assert np.array_equal(np.array([canon[m] if m >= 0 else -1 for m in mapped]), base_l)


# ---------------------------------------------------------------------------
# density
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("w,h,gx,gy,sigma", [
    (1920, 1080, 64, 36, 30.0), (1920, 1080, 128, 72, 30.0), (3840, 2160, 256, 144, 45.0),
    (1920, 1080, 1, 1, 30.0), (640, 480, 17, 5, 12.5), (1000, 700, 100, 37, 3.0),
    (1920, 1080, 128, 72, 0.7), (1920, 1080, 33, 19, 2000.0),
])
def test_density_random_gpu(w, h, gx, gy, sigma):
    xy, off = wl.random_batch(gx * 1000 + gy, 12, 400, width_px=w, height_px=h)
    got = run_density(xy, off, w, h, gx, gy, sigma)
    ref = oracle.density_frames(xy, off, w, h, gx, gy, sigma)
    worst = assert_density_close(got, ref, np.diff(off), sigma, tag=f"{gx}x{gy} sigma {sigma}")
    print(f"density {gx}x{gy} sigma {sigma}: worst rel err {worst:.2e}")


@pytest.mark.parametrize("max_fp", [0, 50])
def test_density_input_order_path_gpu(max_fp):
    """Frames above max_frame_points (all of them for 0) keep their input order."""
    xy, off = wl.random_batch(4242 + max_fp, 10, 300)
    got = run_density(xy, off, 1920, 1080, 128, 72, 30.0, max_fp=max_fp)
    ref = oracle.density_frames(xy, off, 1920, 1080, 128, 72, 30.0)
    assert_density_close(got, ref, np.diff(off), 30.0, tag=f"max_fp {max_fp}")


@pytest.mark.parametrize("path", ["table", "recur"])
@pytest.mark.parametrize("w,h,gx,gy,sigma,frames", [
    (1920, 1080, 128, 72, 30.0, 20), (3840, 2160, 512, 288, 20.0, 3), (3840, 2160, 256, 144, 45.0, 6),
])
def test_density_paths_gpu(path, w, h, gx, gy, sigma, frames, monkeypatch):
    """Both ways of making the factor tiles (exact tables / recurrence) agree with the oracle."""
    monkeypatch.setenv("FLOCK_DENSITY_PATH", path)
    xy, off = wl.random_batch(gx + frames, frames, 1500, width_px=w, height_px=h)
    got = run_density(xy, off, w, h, gx, gy, sigma)
    ref = oracle.density_frames(xy, off, w, h, gx, gy, sigma)
    worst = assert_density_close(got, ref, np.diff(off), sigma, tag=f"{path} {gx}x{gy}")
    print(f"density {path} {gx}x{gy}: worst rel err {worst:.2e}")


@pytest.mark.parametrize("split", ["3", "16"])
def test_density_bird_slices_gpu(split, monkeypatch):
    """Frames split into bird slices whose partial grids are added afterwards,
    including frames with fewer birds than slices and an empty frame."""
    monkeypatch.setenv("FLOCK_DENSITY_SPLIT", split)
    rng = np.random.default_rng(77)
    frames = [np.stack([rng.integers(0, 16 * 1920, n), rng.integers(0, 16 * 1080, n)], 1).astype(np.int32)
              for n in (6000, 3, 0, 700)]
    xy, off = wl.pack(frames)
    assert flock.lib().density_frames_workspace(len(frames), xy.shape[0], 128, 72) > 0
    got = run_density(xy, off, 1920, 1080, 128, 72, 30.0)
    ref = oracle.density_frames(xy, off, 1920, 1080, 128, 72, 30.0)
    assert_density_close(got, ref, np.diff(off), 30.0, tag="slices")
    assert not got[2].any()


def test_density_workspace_gpu(monkeypatch):
    """A launch split into three bird slices: a workspace one byte short is
    refused; the caller's workspace and the library's own give the grid."""
    import ctypes
    monkeypatch.setenv("FLOCK_DENSITY_SPLIT", "3")
    rng = np.random.default_rng(5)
    xy, off = wl.pack([np.stack([rng.integers(0, 16 * 1920, 4000), rng.integers(0, 16 * 1080, 4000)],
                                1).astype(np.int32)])
    dxy, doff = dev_batch(xy, off)
    lib = flock.lib()
    need = lib.density_frames_workspace(1, xy.shape[0], 128, 72)
    assert need > 0
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    out = torch.empty((1, 72, 128), dtype=torch.float32, device="cuda")
    args = (ctypes.c_void_p(dxy.data_ptr()), ctypes.c_void_p(doff.data_ptr()), 1, xy.shape[0], 0, 1920, 1080,
            128, 72, ctypes.c_float(30.0), ctypes.c_void_p(out.data_ptr()))
    assert lib.density_frames(*args, ctypes.c_void_p(ws.data_ptr()), need - 1, None) == flock.binding.FLOCK_ENOMEM
    ref = oracle.density_frames(xy, off, 1920, 1080, 128, 72, 30.0)
    for w, nbytes in ((ctypes.c_void_p(ws.data_ptr()), need), (None, 0)):  # caller's, then the library's
        out.fill_(-1.0)
        assert lib.density_frames(*args, w, nbytes, None) == 0
        torch.cuda.synchronize()
        assert_density_close(out.cpu().numpy(), ref, np.diff(off), 30.0, tag="workspace")


def test_density_single_bird_peak_gpu():
    sigma = 30.0
    # bird exactly at the centre of cell (40, 30) of a 128 x 72 grid on 1920 x 1080
    xy, off = wl.pack([np.array([[16 * 607 + 8, 16 * 457 + 8]], np.int32)])
    got = run_density(xy, off, 1920, 1080, 128, 72, sigma)[0]
    peak = 1.0 / (2.0 * np.pi * sigma * sigma)
    assert np.unravel_index(np.argmax(got), got.shape) == (30, 40)
    assert abs(got[30, 40] - peak) <= 1e-3 * peak


def test_density_determinism_gpu():
    xy, off, w = wl.generate("batch64x2000_1080p", n_frames=4)
    a = run_density(xy, off, w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px)
    b = run_density(xy, off, w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px)
    assert np.array_equal(a, b)


# ---------------------------------------------------------------------------
# the five workloads at full size, in the launch configuration the bench uses
# ---------------------------------------------------------------------------

# Every frame's labels, kinds and n_clusters are compared with the oracle.
# Density: whole grids where the oracle's direct sum over every cell finishes
# in seconds; on the two large batches whole grids of a few frames, and in
# every frame 64 random cells plus the GPU's largest cell, whose oracle value
# (<= the frame's true maximum) stands in for the maximum in the tolerance.
DENSITY_FULL_FRAMES = {"single500_1080p": None, "batch64x2000_1080p": None,
                       "batch256xpoisson8000_4k": [0, 1, 100, 255], "house30000_4k": None,
                       "stream1800x5000_1080p": [0, 1, 900, 1799]}
DENSITY_SAMPLED_CELLS = 64


def assert_density_sampled(dens, xy, off, w, n_cells, seed, tag=""):
    """Every frame: n_cells random cells and the GPU's argmax cell against the
    oracle's direct sum at those cells; |err| <= 1e-3 * oracle(argmax cell)."""
    F = len(off) - 1
    rng = np.random.default_rng(seed)
    flat = dens.reshape(F, -1)
    amax = flat.argmax(axis=1)
    fr = np.repeat(np.arange(F, dtype=np.int32), n_cells + 1)
    cell = rng.integers(0, w.grid_w * w.grid_h, (F, n_cells + 1))
    cell[:, 0] = amax
    cell = cell.ravel()
    gy, gx = cell // w.grid_w, cell % w.grid_w
    ref = oracle.density_cells(xy, off, w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px,
                               fr, gx, gy).reshape(F, n_cells + 1)
    got = flat[np.arange(F)[:, None], cell.reshape(F, n_cells + 1)].astype(np.float64)
    worst = 0.0
    for f in range(F):
        m = ref[f, 0]
        if m == 0.0:
            assert (flat[f] == 0).all(), f"{tag} frame {f}: empty frame not exactly zero"
            continue
        err = np.abs(got[f] - ref[f]).max() / m
        assert err <= DENSITY_RTOL_OF_MAX, f"{tag} frame {f}: sampled rel error {err:.3e}"
        worst = max(worst, err)
    return worst


@pytest.mark.parametrize("name", wl.WORKLOAD_ORDER)
def test_workload_parity_gpu(name):
    xy, off, w = wl.generate(name)
    print(f"{name}: {len(off) - 1} frames, {xy.shape[0]} birds", flush=True)
    got = run_cluster(xy, off, w.eps_q, w.min_pts)
    print(f"{name}: clustering done on the GPU; oracle on every frame", flush=True)
    assert_cluster_equal(got, xy, off, w.eps_q, w.min_pts, tag=name)
    print(f"{name}: clustering exact on all {len(off) - 1} frames", flush=True)
    dens = run_density(xy, off, w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px)
    frames = DENSITY_FULL_FRAMES[name] or list(range(len(off) - 1))
    sxy, soff = sub_batch(xy, off, frames)
    ref = oracle.density_frames(sxy, soff, w.width_px, w.height_px, w.grid_w, w.grid_h, w.sigma_px)
    worst = assert_density_close(dens[frames], ref, tag=name)
    if DENSITY_FULL_FRAMES[name] is not None:
        ws = assert_density_sampled(dens, xy, off, w, DENSITY_SAMPLED_CELLS, seed=len(off), tag=name)
        print(f"{name}: density sampled cells of every frame, worst rel err {ws:.2e}", flush=True)
    print(f"{name}: density worst rel err {worst:.2e} on {len(frames)} whole grids", flush=True)


def test_density_birds_outside_frame_gpu():
    """Birds anywhere in the coordinate range 0 <= x, y < 2^24 quanta: just
    outside the frame (their tails reach the grid), far outside (no
    contribution) and at the largest coordinate, beside birds inside."""
    rng = np.random.default_rng(2024)
    W, H = 1920, 1080
    inside = np.stack([rng.integers(0, 16 * W, 300), rng.integers(0, 16 * H, 300)], 1)
    near = np.stack([rng.integers(16 * W, 16 * (W + 200), 200), rng.integers(0, 16 * (H + 200), 200)], 1)
    below = np.stack([rng.integers(0, 16 * W, 100), rng.integers(16 * H, 16 * (H + 150), 100)], 1)
    far = rng.integers(16 * 4 * W, 1 << 24, (200, 2))
    edge = np.array([[(1 << 24) - 1, (1 << 24) - 1], [(1 << 24) - 1, 0], [0, (1 << 24) - 1],
                     [16 * W, 16 * H], [16 * W - 1, 16 * H - 1]])
    frames = [np.concatenate([inside, near, below, far, edge]).astype(np.int32),
              far.astype(np.int32), np.concatenate([near, edge]).astype(np.int32)]
    xy, off = wl.pack(frames)
    for gx, gy, sigma in ((128, 72, 30.0), (256, 144, 45.0), (100, 37, 20.0)):
        got = run_density(xy, off, W, H, gx, gy, sigma)
        ref = oracle.density_frames(xy, off, W, H, gx, gy, sigma)
        assert_density_close(got, ref, np.diff(off), sigma, tag=f"outside {gx}x{gy}")
        assert not got[1].any(), "birds far outside the frame must leave the grid at zero"


def test_wide_frame_inplace_route_gpu():
    """A frame within the on-chip capacity (max_frame_points covers it) but
    wider than 65535 quanta (4096 px) cannot use 16-bit packed coordinates:
    the on-chip kernel clusters it in place, beside frames that take the
    packed path."""
    rng = np.random.default_rng(99)
    centres = np.stack([rng.integers(0, 16 * 8000, 12), rng.integers(0, 16 * 2000, 12)], 1)
    wide = np.concatenate([c + rng.normal(0, 16 * 60, (250, 2)) for c in centres])
    wide = np.concatenate([wide, [[0, 0], [16 * 8000, 16 * 2000]]])
    wide = np.clip(np.round(wide), 0, (1 << 24) - 1).astype(np.int32)
    small = rng.integers(0, 16 * 1000, (400, 2)).astype(np.int32)
    xy, off = wl.pack([small, wide, small[:30]])
    assert np.ptp(wide[:, 0]) > 0xffff
    got = run_cluster(xy, off, 640, 4)
    assert_cluster_equal(got, xy, off, 640, 4, tag="wide frame")
    assert (got[1][off[1]:off[2]] == 2).sum() > 1000

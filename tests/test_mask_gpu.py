"""GPU parity of mask_components_frames (through the C ABI) against the CPU oracle.

Bar: bit-exact labels image, per-frame counts and offsets, and per
component label, area, box, 1/16-px centroid and score; the fp64 centroid
is the correctly rounded quotient of the same exact integer sums on both
sides, so it is compared bit for bit too.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2512_07009_amd as flock
from paper_2512_07009_amd import workloads as wl

pytestmark = pytest.mark.gpu

FIELDS = ["label", "area", "box", "centroid", "xy", "score"]


def run(prob, threshold, conn, with_labels=True, capacity=None):
    d = torch.from_numpy(np.ascontiguousarray(prob, dtype=np.float32)).cuda()
    out = flock.mask_components_frames(d, threshold, conn, with_labels=with_labels, capacity=capacity)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}


def check(prob, threshold, conn, tag="", with_labels=True, capacity=None):
    print(f"mask parity {tag} shape {tuple(prob.shape)} conn {conn}", flush=True)
    got = run(prob, threshold, conn, with_labels, capacity)
    ref = oracle.mask_components(prob, threshold, conn)
    k = int(ref["offsets"][-1])
    assert np.array_equal(got["offsets"], ref["offsets"]), f"{tag} offsets"
    assert np.array_equal(got["n_components"], ref["n_components"]), f"{tag} n_components"
    if with_labels:
        assert np.array_equal(got["labels"], ref["labels"]), f"{tag} labels"
    n = k if capacity is None else min(k, capacity)
    for f in FIELDS:
        assert np.array_equal(got[f][:n], ref[f][:n]), f"{tag} {f}"
    return got, ref


SHAPES = [(3, 37, 53), (2, 130, 200), (2, 64, 64), (1, 129, 65), (2, 65, 129), (1, 1, 1), (1, 1, 300),
          (1, 300, 1), (4, 97, 191)]


@pytest.mark.parametrize("conn", [4, 8])
@pytest.mark.parametrize("shape", SHAPES, ids=["x".join(map(str, s)) for s in SHAPES])
def test_bird_masks_gpu(shape, conn):
    F, H, W = shape
    for seed in range(3):
        prob = wl.bird_masks(300 + seed, F, H, W, n_birds=max(1, H * W // 250), major_px=(2.0, 9.0),
                             minor_px=(1.0, 4.0), speckle_frac=0.02, empty_frac=0.2)
        check(prob, 0.5, conn, tag=f"seed {seed}")


@pytest.mark.parametrize("conn", [4, 8])
def test_checkerboard_full_tiles_gpu(conn):
    # the most pieces a tile can hold (4 neighbours: a checkerboard; 8: every
    # other row and column), several accumulation passes per tile
    yy, xx = np.mgrid[0:150, 0:140]
    cb = ((xx + yy) % 2 == 0).astype(np.float32)
    grid = ((xx % 2 == 0) & (yy % 2 == 0)).astype(np.float32)
    check(np.stack([cb, grid, 1.0 - cb]), 0.5, conn, tag="checkerboards")


@pytest.mark.parametrize("conn", [4, 8])
def test_serpentine_gpu(conn):
    # one component winding through every tile: long union chains, and every
    # piece but the first relabelled
    H, W = 300, 260
    sp = np.zeros((H, W), np.float32)
    sp[::2, :] = 1.0
    for r in range(1, H, 2):
        sp[r, W - 1 if (r // 2) % 2 == 0 else 0] = 1.0
    spiral = np.zeros((H, W), np.float32)
    t, b, l, r = 0, H - 1, 0, W - 1
    while t <= b and l <= r:
        spiral[t, l:r + 1] = 1
        spiral[t:b + 1, r] = 1
        spiral[b, l:r + 1] = 1
        spiral[t + 2:b + 1, l] = 1
        if t + 2 <= b:
            spiral[t + 2, l:r - 1] = 1
        t, b, l, r = t + 4, b - 2, l + 2, r - 4
    check(np.stack([sp, spiral, sp[::-1, ::-1].copy()]), 0.5, conn, tag="serpentine")


@pytest.mark.parametrize("conn", [4, 8])
def test_combs_merged_above_gpu(conn):
    # teeth in the lower band of tiles joined by a bar in the upper band:
    # every tooth is a piece of its tile whose component starts in the tile
    # above (32 such pieces per tile, and 4 with sparser teeth)
    H, W = 150, 200
    dense = np.zeros((H, W), np.float32)
    dense[63, :] = 1.0
    dense[64:140, ::2] = 1.0
    sparse = np.zeros((H, W), np.float32)
    sparse[60:64, 5:190] = 1.0
    sparse[64:150, ::16] = 1.0
    check(np.stack([dense, sparse, dense[:, ::-1].copy()]), 0.5, conn, tag="combs")


@pytest.mark.parametrize("conn", [4, 8])
def test_full_and_empty_frames_gpu(conn):
    prob = np.zeros((4, 200, 333), np.float32)
    prob[1] = 1.0
    prob[3, 100:, :] = 0.75
    got, ref = check(prob, 0.5, conn, tag="full/empty")
    assert got["n_components"].tolist() == [0, 1, 0, 1]


@pytest.mark.parametrize("shape", [(1, 1, 32768), (1, 32768, 1), (2000, 8, 8), (3, 2, 5000)],
                         ids=["row32768", "col32768", "2000x8x8", "3x2x5000"])
def test_extreme_shapes_gpu(shape):
    # the widest and tallest frames the entry point takes, many tiny frames,
    # and two-row strips (tiles of one partial band)
    rng = np.random.default_rng(sum(shape))
    prob = (rng.random(shape) < 0.45).astype(np.float32) * rng.uniform(0.51, 1.0, shape).astype(np.float32)
    for conn in (4, 8):
        check(prob, 0.5, conn, tag="extreme")


def test_batch_above_local_rank_limit_gpu():
    # more than 2^26 pixels: the component ranks take the separate scan launch
    rng = np.random.default_rng(44)
    prob = rng.random((3, 4096, 6000), dtype=np.float32)
    check(prob, 0.7, 8, tag="large batch")


def test_threshold_ties_nan_inf_gpu():
    rng = np.random.default_rng(5)
    prob = rng.choice(np.array([0.5, np.nextafter(np.float32(0.5), np.float32(1)), 0.25, np.nan, np.inf, 0.9],
                               np.float32), size=(2, 90, 140))
    for conn in (4, 8):
        check(prob, 0.5, conn, tag="ties")
    check(rng.random((2, 70, 70), dtype=np.float32), 0.0, 8, tag="threshold 0")


@pytest.mark.parametrize("name", list(wl.MASK_WORKLOADS))
def test_workload_batches_gpu(name):
    prob, w = wl.mask_batch(name)
    check(prob, w.threshold, w.connectivity, tag=name)
    check(prob[:2], w.threshold, 4, tag=name + " 4-neighbour")


def test_optional_outputs_and_capacity_gpu():
    prob = wl.bird_masks(77, 3, 150, 230, n_birds=120, speckle_frac=0.01)
    ref = oracle.mask_components(prob, 0.5, 8)
    k = int(ref["offsets"][-1])
    check(prob, 0.5, 8, tag="no labels", with_labels=False)
    check(prob, 0.5, 8, tag="capacity", capacity=k // 2)
    check(prob, 0.5, 8, tag="capacity 0", capacity=0)
    d = torch.from_numpy(prob).cuda()
    out = flock.mask_components_frames(d, 0.5, 8)
    out2 = {"labels": None, "n_components": torch.empty(3, dtype=torch.int32, device="cuda"),
            "offsets": torch.empty(4, dtype=torch.int32, device="cuda"),
            "xy": torch.empty((k, 2), dtype=torch.int32, device="cuda")}
    flock.mask_components_frames(d, 0.5, 8, capacity=k, out=out2)
    torch.cuda.synchronize()
    assert torch.equal(out2["xy"], out["xy"][:k])
    assert torch.equal(out2["offsets"], out["offsets"])


def test_back_to_back_shapes_gpu():
    # workspace and outputs of one call do not leak into the next
    a = wl.bird_masks(81, 2, 200, 300, n_birds=300)
    b = wl.bird_masks(82, 3, 70, 90, n_birds=40)
    for prob in (a, b, a):
        check(prob, 0.5, 8, tag="back to back")


def test_feeds_cluster_input_gpu():
    # xy and offsets form a valid batch for the clustering entry points
    prob = wl.bird_masks(90, 3, 180, 320, n_birds=200)
    d = torch.from_numpy(prob).cuda()
    out = flock.mask_components_frames(d, 0.5, 8)
    k = int(out["offsets"][-1].item())
    xy = out["xy"][:k].contiguous()
    labels, kind, ncl = flock.cluster_frames(xy, out["offsets"], 4.0, 3)
    torch.cuda.synchronize()
    ref = oracle.mask_components(prob, 0.5, 8)
    cl = oracle.cluster_frames(ref["xy"], ref["offsets"].astype(np.int32), flock.eps_to_quanta(4.0), 3)
    assert np.array_equal(labels.cpu().numpy(), cl[0])


def test_rejects_gpu():
    d = torch.zeros((1, 4, 4), dtype=torch.float32, device="cuda")
    for t, c in [(-1.0, 8), (float("nan"), 8), (float("inf"), 8), (0.5, 6)]:
        with pytest.raises(ValueError):
            flock.mask_components_frames(d, t, c)

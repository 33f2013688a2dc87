"""Pins for the CPU oracle's region-of-interest filter (no GPU).

Checks that do not restate the oracle's crossing test:
  * hand-built polygons with hand-derived answers, including vertices and
    edges on the test ray (tests/golden/roi_handbuilt.json);
  * rectangles against the closed-form interval test, an L shape against
    the union of two rectangles;
  * convex polygons (scipy.spatial.ConvexHull) against the half-plane test
    (every edge's cross product >= 0 for a counter-clockwise hull);
  * invariance under reversed vertex order, rotated start vertex and
    translation; the batch CSR (order, counts, indices) against a loop.
"""

import json
import os

import numpy as np
import pytest
from scipy.spatial import ConvexHull

import oracle
from paper_2512_07009_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "roi_handbuilt.json")


def inside_all(poly, pts):
    return np.array([oracle.point_in_polygon(poly, int(x), int(y)) for x, y in pts], np.int32)


def test_handbuilt():
    for case in json.load(open(GOLDEN))["cases"]:
        got = inside_all(case["polygon"], case["points"])
        assert got.tolist() == case["inside"], case["name"]


def test_rectangles_closed_form():
    rng = np.random.default_rng(1)
    for _ in range(30):
        x0, x1 = sorted(rng.integers(-50, 50, 2))
        y0, y1 = sorted(rng.integers(-50, 50, 2))
        if x0 == x1 or y0 == y1:
            continue
        poly = [[x0, y0], [x1, y0], [x1, y1], [x0, y1]]
        pts = rng.integers(-60, 60, (200, 2))
        want = ((pts[:, 0] >= x0) & (pts[:, 0] <= x1) & (pts[:, 1] >= y0) & (pts[:, 1] <= y1)).astype(np.int32)
        assert np.array_equal(inside_all(poly, pts), want)


def test_l_shape_is_union_of_rectangles():
    poly = [[0, 0], [40, 0], [40, 15], [15, 15], [15, 30], [0, 30]]
    yy, xx = np.meshgrid(np.arange(-3, 44), np.arange(-3, 44), indexing="ij")
    pts = np.stack([xx.ravel(), yy.ravel()], 1)
    r1 = (pts[:, 0] >= 0) & (pts[:, 0] <= 40) & (pts[:, 1] >= 0) & (pts[:, 1] <= 15)
    r2 = (pts[:, 0] >= 0) & (pts[:, 0] <= 15) & (pts[:, 1] >= 0) & (pts[:, 1] <= 30)
    assert np.array_equal(inside_all(poly, pts), (r1 | r2).astype(np.int32))


def test_convex_polygons_half_planes():
    rng = np.random.default_rng(2)
    for _ in range(10):
        cloud = rng.integers(0, 1000, (12, 2))
        hull = ConvexHull(cloud)
        poly = cloud[hull.vertices]          # counter-clockwise
        pts = rng.integers(-50, 1050, (400, 2))
        a = poly.astype(np.int64)
        b = np.roll(a, -1, axis=0)
        cross = ((b[:, 0] - a[:, 0])[None, :] * (pts[:, 1, None] - a[None, :, 1])
                 - (b[:, 1] - a[:, 1])[None, :] * (pts[:, 0, None] - a[None, :, 0]))
        want = (cross >= 0).all(axis=1).astype(np.int32)
        assert np.array_equal(inside_all(poly, pts), want)


def test_invariances():
    rng = np.random.default_rng(3)
    poly = np.array([[0, 0], [30, 5], [25, 25], [12, 14], [3, 28]], np.int64)
    pts = rng.integers(-5, 35, (500, 2))
    base = inside_all(poly, pts)
    assert np.array_equal(inside_all(poly[::-1], pts), base)
    assert np.array_equal(inside_all(np.roll(poly, 2, axis=0), pts), base)
    t = np.array([1000, -700])
    assert np.array_equal(inside_all(poly + t, pts + t), base)
    assert 0 < base.sum() < len(base)


def test_batch_csr():
    xy, off = wl.random_batch(5, 7, 300)
    poly = [[100 * 16, 100 * 16], [1500 * 16, 200 * 16], [1200 * 16, 900 * 16], [300 * 16, 700 * 16]]
    r = oracle.roi_filter(xy, off, poly)
    keep = inside_all(poly, xy).astype(bool)
    idx = np.nonzero(keep)[0]
    assert np.array_equal(r["index"], idx)
    assert np.array_equal(r["xy"], xy[idx])
    for f in range(len(off) - 1):
        n = int(keep[off[f]:off[f + 1]].sum())
        assert r["counts"][f] == n
        assert r["offsets"][f + 1] - r["offsets"][f] == n
    assert r["offsets"][0] == 0 and r["offsets"][-1] == len(idx)


def test_rejects_bad_polygons():
    xy, off = wl.random_batch(6, 2, 10)
    with pytest.raises(ValueError):
        oracle.roi_filter(xy, off, [[0, 0], [1, 1]])

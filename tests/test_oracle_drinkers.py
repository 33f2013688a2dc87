"""Pins for the CPU oracle's drinker-line proximity (no GPU).

Checks that do not restate the oracle's exact integer test:
  * hand-built segments and points with hand-derived answers, including
    distances exactly at the threshold and degenerate segments
    (tests/golden/drinkers_handbuilt.json);
  * a float64 clamped-projection distance (numpy) on random points whose
    distance is not within 1e-6 of the threshold;
  * invariance under swapped segment ends, translation and a quarter turn;
  * per-frame counts and first indices over a batch.
"""

import json
import os

import numpy as np
import pytest

import oracle
from paper_2512_07009_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "drinkers_handbuilt.json")


def first_line(lines, pts, t):
    xy, off = wl.pack([np.asarray(pts, np.int32).reshape(-1, 2)])
    return oracle.drinkers(xy, off, lines, t)["line"]


def test_handbuilt():
    for case in json.load(open(GOLDEN))["cases"]:
        assert first_line(case["lines"], case["points"], case["t"]).tolist() == case["line"], case["name"]


def seg_dist(p, seg):
    a = np.array(seg[:2], np.float64)
    b = np.array(seg[2:], np.float64)
    u = b - a
    L = u @ u
    w = p - a
    s = np.clip((w @ u) / L, 0.0, 1.0) if L > 0 else np.zeros(len(p))
    near = a + s[:, None] * u
    return np.hypot(*(p - near).T)


def test_float_distance_away_from_threshold():
    rng = np.random.default_rng(7)
    for trial in range(20):
        seg = rng.integers(-2000, 2000, 4).tolist()
        t = int(rng.integers(1, 600))
        pts = rng.integers(-2600, 2600, (400, 2))
        d = seg_dist(pts.astype(np.float64), seg)
        ok = np.abs(d - t) > 1e-6
        got = first_line([seg], pts, t)
        assert np.array_equal((got[ok] == 0), d[ok] < t), f"trial {trial}"


def test_invariances():
    rng = np.random.default_rng(8)
    segs = rng.integers(-500, 500, (5, 4))
    pts = rng.integers(-700, 700, (600, 2))
    base = first_line(segs, pts, 120)
    swapped = segs[:, [2, 3, 0, 1]]
    assert np.array_equal(first_line(swapped, pts, 120), base)
    d = np.array([3333, -1234])
    assert np.array_equal(first_line(segs + np.tile(d, 2), pts + d, 120), base)
    rot = np.stack([-segs[:, 1], segs[:, 0], -segs[:, 3], segs[:, 2]], 1)
    assert np.array_equal(first_line(rot, np.stack([-pts[:, 1], pts[:, 0]], 1), 120), base)
    assert 0 < (base >= 0).sum() < len(base)


def test_batch_counts():
    xy, off = wl.random_batch(12, 9, 400)
    lines = [[0, 5000, 30000, 5000], [8000, 0, 8000, 17000]]
    r = oracle.drinkers(xy, off, lines, 640)
    for f in range(len(off) - 1):
        assert r["counts"][f] == int(r["drinking"][off[f]:off[f + 1]].sum())
    assert np.array_equal(r["drinking"].astype(bool), r["line"] >= 0)


def test_rejects_bad_arguments():
    xy, off = wl.random_batch(13, 2, 10)
    with pytest.raises(ValueError):
        oracle.drinkers(xy, off, np.zeros((0, 4), np.int32), 10)
    with pytest.raises(ValueError):
        oracle.drinkers(xy, off, [[0, 0, 1, 1]], -1)

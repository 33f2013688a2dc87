"""Seeded synthetic workloads: reproducibility, shapes and ranges (no GPU)."""

import numpy as np
import pytest

from paper_2512_07009_amd import workloads as wl


@pytest.mark.parametrize("name", ["single500_1080p", "batch64x2000_1080p", "house30000_4k"])
def test_reproducible_and_in_range(name):
    a = wl.generate(name)
    b = wl.generate(name)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    xy, off, w = a
    assert xy.dtype == np.int32 and off.dtype == np.int32
    assert off[0] == 0 and off[-1] == xy.shape[0] and (np.diff(off) >= 0).all()
    assert len(off) == w.n_frames + 1
    assert (xy[:, 0] >= 0).all() and (xy[:, 0] < 16 * w.width_px).all()
    assert (xy[:, 1] >= 0).all() and (xy[:, 1] < 16 * w.height_px).all()


def test_counts():
    assert wl.generate("single500_1080p")[0].shape[0] == 500
    xy, off, _ = wl.generate("batch64x2000_1080p")
    assert (np.diff(off) == 2000).all()
    xy, off, _ = wl.generate("house30000_4k")
    assert xy.shape[0] == 30000


def test_prefix_property():
    full = wl.generate("batch256xpoisson8000_4k", n_frames=6)
    part = wl.generate("batch256xpoisson8000_4k", n_frames=3)
    n = part[1][-1]
    assert np.array_equal(full[0][:n], part[0])
    assert np.array_equal(full[1][:4], part[1])
    counts = np.diff(full[1])
    assert (counts > 7000).all() and (counts < 9000).all()


def test_stream_is_jittered_copy():
    xy, off, w = wl.generate("stream1800x5000_1080p", n_frames=3)
    assert (np.diff(off) == 5000).all()
    f0 = xy[off[0]:off[1]].astype(np.int64)
    f1 = xy[off[1]:off[2]].astype(np.int64)
    d = np.hypot(*(f1 - f0).T) / 16.0
    # 99% of birds move by N(0, 2 px) per axis, 1% are re-spawned anywhere
    assert np.mean(d < 12.0) > 0.985
    assert np.mean(d < 12.0) < 1.0


def test_random_batch_has_empty_frames_and_duplicates():
    xy, off = wl.random_batch(5, 40, 50)
    counts = np.diff(off)
    assert (counts == 0).any()
    assert counts.max() <= 50
    assert xy.shape[0] == off[-1]

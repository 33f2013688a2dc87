"""Pins for the CPU oracle's heatmap analytics (no GPU).

Checks that do not restate the oracle's code:
  * hand-built grids with hand-derived labels, counts, masses, entropy and
    degree (tests/golden/heatmap_handbuilt.json);
  * scipy.ndimage.label as an independent connected-component labelling
    (partition equality on random grids, both neighbourhoods);
  * closed forms of the entropy (uniform grids: ln N; scale and permutation
    invariance) and of the degree (threshold below every positive cell: 1,
    above every cell: 0);
  * conservation: component cells add up to the hot cells, component masses
    to cell_area times the hot density; batch and thread independence.
"""

import json
import math
import os

import numpy as np
import pytest
from scipy import ndimage

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "heatmap_handbuilt.json")
BELOW_HALF = float(np.nextafter(np.float32(0.5), np.float32(0.0)))


def _grid(rows):
    return np.array([[BELOW_HALF if v == "below_half" else v for v in r] for r in rows], np.float32)


@pytest.mark.parametrize("conn", [4, 8])
def test_handbuilt(conn):
    for case in json.load(open(GOLDEN))["cases"]:
        g = _grid(case["grid"])[None]
        r = oracle.heatmap_frames(g, case["cell_area"], case["threshold"], conn)
        k = str(conn)
        assert r["labels"][0].tolist() == case["labels"][k], case["name"]
        assert int(r["n_components"][0]) == case["n_components"][k], case["name"]
        cells = {str(c): int(v) for c, v in enumerate(r["comp_cells"][0].ravel()) if v}
        assert cells == case["comp_cells"][k], case["name"]
        if "comp_mass" in case:
            mass = {str(c): float(v) for c, v in enumerate(r["comp_mass"][0].ravel()) if v}
            assert mass.keys() == case["comp_mass"].keys(), case["name"]
            for c, v in case["comp_mass"].items():
                assert mass[c] == pytest.approx(v, rel=1e-15), case["name"]
        if "degree" in case:
            assert float(r["degree"][0]) == pytest.approx(case["degree"], rel=1e-15), case["name"]
        if "entropy_terms" in case:
            h = -sum(n * p * math.log(p) for n, p in case["entropy_terms"])
            assert float(r["entropy"][0]) == pytest.approx(h, rel=1e-14, abs=1e-15), case["name"]


def _min_index_relabel(lab):
    """scipy labels (0 background, 1..n components) -> smallest cell index, -1."""
    flat = lab.ravel()
    out = np.full(flat.shape, -1, np.int64)
    for c in range(1, int(flat.max()) + 1):
        idx = np.nonzero(flat == c)[0]
        out[idx] = idx.min()
    return out.reshape(lab.shape)


@pytest.mark.parametrize("conn", [4, 8])
def test_components_match_scipy(conn):
    rng = np.random.default_rng(11 + conn)
    structure = ndimage.generate_binary_structure(2, 1 if conn == 4 else 2)
    for trial in range(20):
        h, w = rng.integers(1, 40, 2)
        g = rng.random((h, w)).astype(np.float32)
        thr = float(rng.uniform(0.3, 0.8))
        r = oracle.heatmap_frames(g[None], 1.0, thr, conn)
        lab, n = ndimage.label(g >= np.float32(thr), structure=structure)
        assert int(r["n_components"][0]) == n
        assert np.array_equal(r["labels"][0], _min_index_relabel(lab)), f"trial {trial}"


def test_entropy_closed_forms():
    for n in (1, 2, 7, 100):
        g = np.zeros((1, 10, 10), np.float32)
        g.reshape(-1)[:n] = 0.3
        r = oracle.heatmap_frames(g, 1.0, 0.1)
        assert float(r["entropy"][0]) == pytest.approx(math.log(n), abs=1e-12)
    rng = np.random.default_rng(3)
    g = rng.random((1, 17, 23)).astype(np.float32)
    base = float(oracle.heatmap_frames(g, 1.0, 0.5)["entropy"][0])
    scaled = float(oracle.heatmap_frames(g * np.float32(4.0), 1.0, 2.0)["entropy"][0])
    perm = rng.permutation(g.size)
    shuffled = float(oracle.heatmap_frames(g.reshape(-1)[perm].reshape(g.shape), 1.0, 0.5)["entropy"][0])
    assert scaled == pytest.approx(base, rel=1e-12)
    assert shuffled == pytest.approx(base, rel=1e-12)
    assert 0.0 < base < math.log(g.size)


def test_degree_limits_and_conservation():
    rng = np.random.default_rng(5)
    g = (rng.random((3, 20, 30)) + 0.01).astype(np.float32)
    lo = oracle.heatmap_frames(g, 1.5, float(g.min()))
    assert np.allclose(lo["degree"], 1.0, rtol=0, atol=1e-15)
    assert (lo["n_components"] == 1).all()
    hi = oracle.heatmap_frames(g, 1.5, float(g.max()) * 1.01)
    assert (hi["degree"] == 0.0).all() and (hi["n_components"] == 0).all()
    assert (hi["labels"] == -1).all()
    mid = oracle.heatmap_frames(g, 1.5, 0.6)
    for f in range(3):
        hot = g[f] >= np.float32(0.6)
        assert int(mid["comp_cells"][f].sum()) == int(hot.sum())
        assert float(mid["comp_mass"][f].sum()) == pytest.approx(1.5 * float(g[f][hot].astype(np.float64).sum()),
                                                                 rel=1e-12)
        assert float(mid["degree"][f]) == pytest.approx(
            float(g[f][hot].astype(np.float64).sum()) / float(g[f].astype(np.float64).sum()), rel=1e-12)


def test_batch_and_threads_independent():
    rng = np.random.default_rng(9)
    g = rng.random((5, 13, 19)).astype(np.float32)
    g[2] = 0.0
    whole = oracle.heatmap_frames(g, 2.0, 0.7, 8, n_threads=4)
    for f in range(5):
        one = oracle.heatmap_frames(g[f:f + 1], 2.0, 0.7, 8, n_threads=1)
        for k in whole:
            assert np.array_equal(whole[k][f:f + 1], one[k]), (k, f)


def test_rejects_bad_arguments():
    g = np.ones((1, 2, 2), np.float32)
    for thr, conn in ((0.0, 8), (-1.0, 8), (0.5, 6)):
        with pytest.raises(ValueError):
            oracle.heatmap_frames(g, 1.0, thr, conn)

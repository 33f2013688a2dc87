"""Pins for the CPU oracle's clustering (no GPU).

The oracle is checked against things other than itself:
  * hand-built point sets whose labels were derived by hand from the DBSCAN
    definition (tests/golden/dbscan_handbuilt.json);
  * scikit-learn's DBSCAN (core set, core partition, noise set) and, for
    min_pts = 1, scipy's radius-pair search plus graph connected components;
  * scipy's radius-neighbour counts;
  * invariants that the definition fixes: permutation, translation, scaling,
    batch independence and monotonicity in eps and min_pts.
"""

import numpy as np
import pytest
from scipy.sparse import coo_matrix
from scipy.sparse.csgraph import connected_components
from scipy.spatial import cKDTree
from sklearn.cluster import DBSCAN

import oracle
from paper_2512_07009_amd import workloads as wl


def _frames_to_batch(frames):
    return wl.pack([np.asarray(f, dtype=np.int32).reshape(-1, 2) for f in frames])


def test_handbuilt_cases(handbuilt):
    for case in handbuilt:
        xy, off = _frames_to_batch(case["frames"])
        labels, kind, ncl = oracle.cluster_frames(xy, off, case["eps_q"], case["min_pts"], n_threads=2)
        for f in range(len(case["frames"])):
            b, e = off[f], off[f + 1]
            assert labels[b:e].tolist() == case["labels"][f], case["name"]
            assert kind[b:e].tolist() == case["kind"][f], case["name"]
        assert ncl.tolist() == case["n_clusters"], case["name"]


def _random_frame(seed, n, spread=4000, clusters=4, std=300):
    rng = np.random.default_rng(seed)
    centres = rng.integers(0, spread, (clusters, 2))
    pick = rng.integers(0, clusters, n)
    pts = np.round(centres[pick] + rng.normal(0, std, (n, 2)))
    pts = np.clip(pts, 0, 2 ** 20).astype(np.int32)
    # some exact duplicates and some points exactly eps apart along an axis
    if n > 10:
        pts[: n // 20] = pts[n // 20: 2 * (n // 20)]
    return pts


def _canon_partition(labels):
    """Map labels to first-occurrence order so two labelings compare as partitions."""
    seen = {}
    out = []
    for lab in labels:
        if lab < 0:
            out.append(-1)
            continue
        if lab not in seen:
            seen[lab] = len(seen)
        out.append(seen[lab])
    return out


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("eps_q,min_pts", [(640, 4), (400, 6), (960, 5), (200, 2)])
def test_against_sklearn(seed, eps_q, min_pts):
    xy = _random_frame(seed, 400)
    labels, kind, ncl = oracle.dbscan_frame(xy, eps_q, min_pts)
    db = DBSCAN(eps=float(eps_q), min_samples=min_pts, algorithm="kd_tree").fit(xy.astype(np.float64))
    core_sk = np.zeros(len(xy), bool)
    core_sk[db.core_sample_indices_] = True
    # the core set is unique
    assert np.array_equal(kind == 2, core_sk)
    # the partition of the core points is unique
    assert _canon_partition(labels[core_sk]) == _canon_partition(db.labels_[core_sk])
    assert ncl == len(set(db.labels_[core_sk].tolist()))
    # noise (no core neighbour) is unique
    assert np.array_equal(kind == 0, db.labels_ == -1)
    # a border point's cluster is the cluster of one of its core neighbours
    tree = cKDTree(xy.astype(np.float64))
    for i in np.nonzero(kind == 1)[0]:
        nb = [j for j in tree.query_ball_point(xy[i].astype(np.float64), float(eps_q)) if core_sk[j]]
        assert labels[i] in {labels[j] for j in nb}


@pytest.mark.parametrize("seed", range(4))
def test_min_pts_one_is_connected_components(seed):
    xy = _random_frame(100 + seed, 500)
    eps_q = 500
    labels, kind, ncl = oracle.dbscan_frame(xy, eps_q, 1)
    assert (kind == 2).all()
    pairs = cKDTree(xy.astype(np.float64)).query_pairs(float(eps_q), output_type="ndarray")
    n = len(xy)
    g = coo_matrix((np.ones(len(pairs)), (pairs[:, 0], pairs[:, 1])), shape=(n, n))
    nc, comp = connected_components(g, directed=False)
    # canonical label: smallest index in the component
    first = {}
    for i, c in enumerate(comp):
        first.setdefault(c, i)
    expect = np.array([first[c] for c in comp], np.int32)
    assert np.array_equal(labels, expect)
    assert ncl == nc


@pytest.mark.parametrize("seed", range(4))
def test_counts_against_scipy(seed):
    xy = _random_frame(200 + seed, 600)
    for eps_q in (0, 1, 300, 640):
        cnt = oracle.neighbour_counts(xy, eps_q)
        tree = cKDTree(xy.astype(np.float64))
        ref = np.array([len(tree.query_ball_point(p, float(eps_q))) for p in xy.astype(np.float64)])
        assert np.array_equal(cnt, ref)


@pytest.mark.parametrize("seed", range(5))
def test_permutation_invariance(seed):
    xy = _random_frame(300 + seed, 350, std=200)
    eps_q, min_pts = 640, 4
    labels, kind, _ = oracle.dbscan_frame(xy, eps_q, min_pts)
    perm = np.random.default_rng(seed).permutation(len(xy))
    l2, k2, _ = oracle.dbscan_frame(xy[perm], eps_q, min_pts)
    # back to original order
    inv = np.empty_like(perm)
    inv[perm] = np.arange(len(perm))
    k_back = k2[inv]
    assert np.array_equal(k_back, kind)
    # label values refer to permuted indices: map them to original indices,
    # then canonicalise each cluster by its smallest original core index.
    l_back = l2[inv]
    mapped = np.where(l_back >= 0, perm[np.maximum(l_back, 0)], -1)
    canon = {}
    for i in np.nonzero(kind == 2)[0]:
        canon.setdefault(mapped[i], i)
    relab = np.array([canon[m] if m >= 0 else -1 for m in mapped], np.int32)
    assert np.array_equal(relab, labels)


@pytest.mark.parametrize("seed", range(3))
def test_translation_and_scaling(seed):
    xy = _random_frame(400 + seed, 300)
    eps_q, min_pts = 640, 4
    base = oracle.dbscan_frame(xy, eps_q, min_pts)
    moved = oracle.dbscan_frame(xy + np.array([12345, 777], np.int32), eps_q, min_pts)
    scaled = oracle.dbscan_frame(xy * 2, eps_q * 2, min_pts)
    for other in (moved, scaled):
        assert np.array_equal(other[0], base[0])
        assert np.array_equal(other[1], base[1])
        assert other[2] == base[2]


def test_batch_independence():
    frames = [_random_frame(500 + s, 100 + 50 * s) for s in range(5)]
    frames.insert(2, np.zeros((0, 2), np.int32))
    xy, off = wl.pack(frames)
    labels, kind, ncl = oracle.cluster_frames(xy, off, 640, 4, n_threads=3)
    for f, fr in enumerate(frames):
        l1, k1, n1 = oracle.dbscan_frame(fr, 640, 4)
        assert np.array_equal(labels[off[f]:off[f + 1]], l1)
        assert np.array_equal(kind[off[f]:off[f + 1]], k1)
        assert ncl[f] == n1


@pytest.mark.parametrize("seed", range(3))
def test_monotonicity(seed):
    xy = _random_frame(600 + seed, 300)
    core = {}
    for eps_q in (300, 640, 900):
        for mp in (2, 4, 8):
            core[eps_q, mp] = oracle.dbscan_frame(xy, eps_q, mp)[1] == 2
    for eps_q in (300, 640, 900):
        assert (core[eps_q, 8] <= core[eps_q, 4]).all() and (core[eps_q, 4] <= core[eps_q, 2]).all()
    for mp in (2, 4, 8):
        assert (core[300, mp] <= core[640, mp]).all() and (core[640, mp] <= core[900, mp]).all()


def test_invalid_arguments():
    with pytest.raises(ValueError):
        oracle.dbscan_frame([[0, 0]], 640, 0)
    with pytest.raises(ValueError):
        oracle.cluster_frames(np.zeros((2, 2), np.int32), np.array([0, 3], np.int32), 640, 4)

"""Pins for the CPU oracle's detection post-processing (no GPU).

Checks that do not restate the oracle's code:
  * hand-built masks with hand-derived labels, areas, boxes, centroids,
    1/16-px centroids and scores (tests/golden/mask_components_handbuilt.json);
  * scipy.ndimage as an independent implementation: label (partition of the
    foreground), find_objects (boxes), center_of_mass (centroids), sum and
    maximum by label (areas, scores), on random masks of bird-like blobs in
    both neighbourhoods;
  * exact rationals (fractions.Fraction) for floor(16 * mean);
  * invariants: 8-neighbour components are unions of 4-neighbour ones, a
    higher threshold only splits or shrinks components, transposing the mask
    permutes the components, every pixel of a component has an index no
    smaller than its label, areas add up to the foreground count;
  * special cases: checkerboards, single rows and columns, one pixel, empty
    batches, NaN and infinite probabilities, and the rejected arguments.
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy import ndimage

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mask_components_handbuilt.json")
STRUCT = {4: ndimage.generate_binary_structure(2, 1), 8: ndimage.generate_binary_structure(2, 2)}


def _value(v, threshold):
    if v == "threshold":
        return np.float32(threshold)
    if v == "above_threshold":
        return np.nextafter(np.float32(threshold), np.float32(np.inf))
    return np.float32(v)


def _golden_cases():
    for case in json.load(open(GOLDEN))["cases"]:
        conns = case["connectivity"] if isinstance(case["connectivity"], list) else [case["connectivity"]]
        for c in conns:
            yield case, c


def test_handbuilt():
    n = 0
    for case, conn in _golden_cases():
        t = case["threshold"]
        prob = np.array([[[_value(v, t) for v in row] for row in fr] for fr in case["frames"]], np.float32)
        r = oracle.mask_components(prob, t, conn)
        name = f'{case["name"]}/{conn}'
        assert r["labels"].tolist() == case["labels"], name
        comps = case["components"]
        assert int(r["offsets"][-1]) == len(comps), name
        frames = np.repeat(np.arange(prob.shape[0]), np.diff(r["offsets"]))
        for k, c in enumerate(comps):
            assert int(frames[k]) == c["frame"], name
            assert int(r["label"][k]) == c["label"], name
            assert int(r["area"][k]) == c["area"], name
            assert r["box"][k].tolist() == c["box"], name
            sx, sy = c["centroid_sum"]
            assert r["centroid"][k].tolist() == [sx / c["area"], sy / c["area"]], name
            assert r["xy"][k].tolist() == c["xy"], name
            assert r["score"][k] == _value(c["score"], t), name
        n += 1
    assert n >= 10


def blob_masks(seed, n_frames, h, w, n_blobs=12, noise=0.01):
    """Probability maps with elliptical blobs and isolated speckles."""
    rng = np.random.default_rng(seed)
    yy, xx = np.mgrid[0:h, 0:w].astype(np.float64)
    out = rng.uniform(0.0, 0.45, (n_frames, h, w))
    for f in range(n_frames):
        for _ in range(int(rng.integers(0, n_blobs + 1))):
            cx, cy = rng.uniform(0, w), rng.uniform(0, h)
            a, b, th = rng.uniform(1.0, 6.0), rng.uniform(0.7, 3.5), rng.uniform(0, np.pi)
            u = (xx - cx) * np.cos(th) + (yy - cy) * np.sin(th)
            v = -(xx - cx) * np.sin(th) + (yy - cy) * np.cos(th)
            r2 = (u / a) ** 2 + (v / b) ** 2
            out[f] = np.maximum(out[f], np.where(r2 <= 1.0, 1.0 - 0.4 * r2, 0.0))
        speck = rng.random((h, w)) < noise
        out[f][speck] = rng.uniform(0.5, 1.0, int(speck.sum()))
    return out.astype(np.float32)


def _scipy_components(fg2d, prob2d, conn):
    lab, n = ndimage.label(fg2d, structure=STRUCT[conn])
    flat = lab.ravel()
    idx = np.arange(1, n + 1)
    first = ndimage.minimum(np.arange(flat.size).reshape(lab.shape), lab, idx) if n else []
    order = np.argsort(first, kind="stable")
    objs = ndimage.find_objects(lab)
    com = ndimage.center_of_mass(fg2d.astype(np.float64), lab, idx) if n else []
    area = ndimage.sum(np.ones_like(lab), lab, idx) if n else []
    score = ndimage.maximum(prob2d, lab, idx) if n else []
    out = []
    for o in order:
        sl = objs[o]
        ys, xs = np.nonzero(lab == o + 1)
        out.append({"label": int(first[o]), "area": int(area[o]),
                    "box": [sl[1].start, sl[0].start, sl[1].stop - sl[1].start, sl[0].stop - sl[0].start],
                    "centroid": (float(com[o][1]), float(com[o][0])), "score": np.float32(score[o]),
                    "sums": (int(xs.sum()), int(ys.sum())), "lab": lab == o + 1})
    return out


@pytest.mark.parametrize("conn", [4, 8])
@pytest.mark.parametrize("seed,shape", [(1, (3, 37, 53)), (2, (2, 64, 64)), (3, (4, 19, 130))])
def test_against_scipy(conn, seed, shape):
    prob = blob_masks(seed, *shape)
    t = 0.5
    r = oracle.mask_components(prob, t, conn)
    for f in range(shape[0]):
        ref = _scipy_components(prob[f] > t, prob[f], conn)
        k0, k1 = int(r["offsets"][f]), int(r["offsets"][f + 1])
        assert k1 - k0 == len(ref) == int(r["n_components"][f])
        for k, c in zip(range(k0, k1), ref):
            assert int(r["label"][k]) == c["label"]
            assert int(r["area"][k]) == c["area"]
            assert r["box"][k].tolist() == c["box"]
            assert r["centroid"][k] == pytest.approx(c["centroid"], rel=1e-13, abs=1e-13)
            assert r["score"][k] == c["score"]
            sx, sy = c["sums"]
            assert r["xy"][k].tolist() == [int(Fraction(16 * sx, c["area"])), int(Fraction(16 * sy, c["area"]))]
            assert np.array_equal(r["labels"][f] == c["label"], c["lab"])
        assert ((r["labels"][f] >= 0) == (prob[f] > t)).all()


def test_label_is_first_pixel_and_areas_add_up():
    prob = blob_masks(7, 3, 48, 80, n_blobs=20)
    r = oracle.mask_components(prob, 0.5, 8)
    for f in range(3):
        lab = r["labels"][f].ravel()
        idx = np.arange(lab.size)
        fg = lab >= 0
        assert (lab[fg] <= idx[fg]).all()
        assert (lab[lab[fg]] == lab[fg]).all()
        assert int(r["area"][r["offsets"][f]:r["offsets"][f + 1]].sum()) == int(fg.sum())
        labs = r["label"][r["offsets"][f]:r["offsets"][f + 1]]
        assert (np.diff(labs) > 0).all()


def test_eight_unions_of_four():
    prob = blob_masks(8, 2, 40, 40, n_blobs=25, noise=0.05)
    r4 = oracle.mask_components(prob, 0.5, 4)["labels"]
    r8 = oracle.mask_components(prob, 0.5, 8)["labels"]
    for l4 in np.unique(r4[r4 >= 0]):
        sel = r4 == l4
        assert len(np.unique(r8[sel])) == 1
    assert len(np.unique(r8[r8 >= 0])) <= len(np.unique(r4[r4 >= 0]))


def test_higher_threshold_refines():
    prob = blob_masks(9, 2, 50, 70)
    lo = oracle.mask_components(prob, 0.5, 8)["labels"]
    hi = oracle.mask_components(prob, 0.8, 8)["labels"]
    assert ((hi >= 0) <= (lo >= 0)).all()
    for lab in np.unique(hi[hi >= 0]):
        assert len(np.unique(lo[hi == lab])) == 1


@pytest.mark.parametrize("conn", [4, 8])
def test_transpose_permutes_components(conn):
    prob = blob_masks(10, 2, 33, 45)
    a = oracle.mask_components(prob, 0.5, conn)
    b = oracle.mask_components(np.ascontiguousarray(prob.transpose(0, 2, 1)), 0.5, conn)
    assert a["n_components"].tolist() == b["n_components"].tolist()
    for f in range(2):
        sa = sorted(zip(a["area"][a["offsets"][f]:a["offsets"][f + 1]].tolist(),
                        map(tuple, a["box"][a["offsets"][f]:a["offsets"][f + 1]].tolist())))
        sb = sorted(zip(b["area"][b["offsets"][f]:b["offsets"][f + 1]].tolist(),
                        [(bx[1], bx[0], bx[3], bx[2]) for bx in b["box"][b["offsets"][f]:b["offsets"][f + 1]].tolist()]))
        assert sa == sb


def test_checkerboard():
    yy, xx = np.mgrid[0:9, 0:12]
    prob = ((xx + yy) % 2 == 0).astype(np.float32)[None]
    r4 = oracle.mask_components(prob, 0.5, 4)
    assert int(r4["n_components"][0]) == int((prob > 0.5).sum())
    assert (r4["area"] == 1).all()
    r8 = oracle.mask_components(prob, 0.5, 8)
    assert int(r8["n_components"][0]) == 1
    assert r8["box"][0].tolist() == [0, 0, 12, 9]


@pytest.mark.parametrize("shape", [(1, 1, 1), (1, 1, 17), (1, 23, 1), (2, 1, 5)])
def test_thin_shapes(shape):
    rng = np.random.default_rng(sum(shape))
    prob = rng.random(shape).astype(np.float32)
    for conn in (4, 8):
        r = oracle.mask_components(prob, 0.5, conn)
        for f in range(shape[0]):
            ref = _scipy_components(prob[f] > 0.5, prob[f], conn)
            assert int(r["n_components"][f]) == len(ref)
            k0 = int(r["offsets"][f])
            for k, c in enumerate(ref):
                assert int(r["label"][k0 + k]) == c["label"] and int(r["area"][k0 + k]) == c["area"]


def test_nan_inf_and_empty():
    prob = np.array([[[np.nan, np.inf, 0.2]]], np.float32)
    r = oracle.mask_components(prob, 0.1, 4)
    assert r["labels"].tolist() == [[[-1, 1, 1]]]
    assert r["area"].tolist() == [2] and r["box"].tolist() == [[1, 0, 2, 1]]
    assert r["centroid"].tolist() == [[1.5, 0.0]] and r["xy"].tolist() == [[24, 0]]
    assert np.isinf(r["score"][0])
    e = oracle.mask_components(np.zeros((0, 4, 4), np.float32), 0.5, 8)
    assert e["offsets"].tolist() == [0] and e["label"].size == 0


@pytest.mark.parametrize("t,conn", [(-0.5, 8), (float("nan"), 8), (float("inf"), 8), (0.5, 6)])
def test_rejects(t, conn):
    with pytest.raises(Exception):
        oracle.mask_components(np.zeros((1, 2, 2), np.float32), t, conn)

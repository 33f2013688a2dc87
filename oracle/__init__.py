"""CPU oracle for the per-frame clustering and density path.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library or its binding.

The arithmetic lives in ``oracle.c`` (plain C, fp64 for the density, int64 for
distances); this module only compiles it with gcc and marshals numpy arrays.
The definitions it follows are stated at the top of ``oracle.c``:
standard DBSCAN (Ester et al., 1996) as the point-level reading of the
paper's connected-component clustering (Section 2.3), the direct-sum
Gaussian density grid of Algorithm 1 (Section 3.6), and the heatmap
analytics of Section 2.3 and Algorithm 1 (threshold, connected components of
grid cells, entropy, clustering degree), region-of-interest filtering with
per-frame region counts (Section 2.2, Algorithm 1), drinker-line proximity
(Section 2.3), and the detection post-processing of Section 3.2 (mask
components with area, box and centroid).
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# A test-only hook: load a differently built oracle (the mutation tests build
# copies of oracle.c with one planted mistake each and point this at them).
_LIB_OVERRIDE = os.environ.get("ORACLE_LIB_OVERRIDE")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc -O2, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            lib = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            lib = ctypes.CDLL(_LIB)
        p = ctypes.c_void_p
        i32 = ctypes.c_int32
        lib.oracle_dbscan_frame.argtypes = [p, i32, i32, i32, p, p]
        lib.oracle_dbscan_frame.restype = i32
        lib.oracle_neighbour_counts.argtypes = [p, i32, i32, p]
        lib.oracle_neighbour_counts.restype = i32
        lib.oracle_density_cell.argtypes = [p, i32, i32, i32, i32, i32, ctypes.c_double, i32, i32]
        lib.oracle_density_cell.restype = ctypes.c_double
        lib.oracle_cluster_frames.argtypes = [p, p, i32, i32, i32, p, p, p, i32]
        lib.oracle_cluster_frames.restype = i32
        lib.oracle_density_frames.argtypes = [p, p, i32, i32, i32, i32, i32, ctypes.c_double, p, i32]
        lib.oracle_density_frames.restype = i32
        lib.oracle_density_cells.argtypes = [p, p, i32, i32, i32, i32, i32, ctypes.c_double,
                                             p, p, p, ctypes.c_int64, p, i32]
        lib.oracle_density_cells.restype = i32
        lib.oracle_heatmap_frames.argtypes = [p, i32, i32, i32, ctypes.c_double, ctypes.c_float, i32,
                                              p, p, p, p, p, p, i32]
        lib.oracle_heatmap_frames.restype = i32
        lib.oracle_point_in_polygon.argtypes = [p, i32, i32, i32]
        lib.oracle_point_in_polygon.restype = i32
        lib.oracle_roi_filter.argtypes = [p, p, i32, p, i32, p, p, p, p]
        lib.oracle_roi_filter.restype = i32
        lib.oracle_near_segment.argtypes = [i32] * 7
        lib.oracle_near_segment.restype = i32
        lib.oracle_drinkers.argtypes = [p, p, i32, p, i32, i32, p, p, p]
        lib.oracle_drinkers.restype = i32
        lib.oracle_mask_components.argtypes = [p, i32, i32, i32, ctypes.c_float, i32, p, p, p, ctypes.c_int64,
                                               p, p, p, p, p, p]
        lib.oracle_mask_components.restype = ctypes.c_int64
        _lib = lib
    return _lib


def default_threads() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _xy(xy) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(xy, dtype=np.int32).reshape(-1, 2))
    return a


def _check(rc: int, what: str):
    if rc < 0:
        raise ValueError(f"oracle {what}: error {rc}")


def neighbour_counts(xy, eps_q: int) -> np.ndarray:
    """Per-point count of points within eps (self included), one frame."""
    a = _xy(xy)
    out = np.zeros(a.shape[0], np.int32)
    _check(_load().oracle_neighbour_counts(_ptr(a), a.shape[0], int(eps_q), _ptr(out)), "counts")
    return out


def dbscan_frame(xy, eps_q: int, min_pts: int):
    """One frame: returns (labels int32[n], kind uint8[n], n_clusters)."""
    a = _xy(xy)
    n = a.shape[0]
    labels = np.zeros(n, np.int32)
    kind = np.zeros(n, np.uint8)
    r = _load().oracle_dbscan_frame(_ptr(a), n, int(eps_q), int(min_pts), _ptr(labels), _ptr(kind))
    _check(r, "dbscan_frame")
    return labels, kind, int(r)


def cluster_frames(xy, offsets, eps_q: int, min_pts: int, n_threads: int | None = None):
    """Batch: returns (labels int32[T], kind uint8[T], n_clusters int32[F])."""
    a = _xy(xy)
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32))
    F = off.shape[0] - 1
    T = a.shape[0]
    if F < 0 or (F >= 0 and int(off[-1]) != T):
        raise ValueError("offsets do not describe xy")
    labels = np.zeros(T, np.int32)
    kind = np.zeros(T, np.uint8)
    ncl = np.zeros(max(F, 0), np.int32)
    r = _load().oracle_cluster_frames(_ptr(a), _ptr(off), F, int(eps_q), int(min_pts),
                                      _ptr(labels), _ptr(kind), _ptr(ncl),
                                      n_threads or default_threads())
    _check(r, "cluster_frames")
    return labels, kind, ncl


def density_frames(xy, offsets, width_px: int, height_px: int, grid_w: int, grid_h: int,
                   sigma_px: float, n_threads: int | None = None) -> np.ndarray:
    """Batch: returns float64[F, grid_h, grid_w] in birds per px^2."""
    a = _xy(xy)
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32))
    F = off.shape[0] - 1
    if int(off[-1]) != a.shape[0]:
        raise ValueError("offsets do not describe xy")
    out = np.zeros((F, grid_h, grid_w), np.float64)
    r = _load().oracle_density_frames(_ptr(a), _ptr(off), F, int(width_px), int(height_px),
                                      int(grid_w), int(grid_h), float(sigma_px), _ptr(out),
                                      n_threads or default_threads())
    _check(r, "density_frames")
    return out


def density_cells(xy, offsets, width_px: int, height_px: int, grid_w: int, grid_h: int,
                  sigma_px: float, frame, gx, gy, n_threads: int | None = None) -> np.ndarray:
    """Density at sampled cells (frame[k], gy[k], gx[k]); float64[m]."""
    a = _xy(xy)
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32))
    F = off.shape[0] - 1
    fr = np.ascontiguousarray(np.asarray(frame, dtype=np.int32))
    cx = np.ascontiguousarray(np.asarray(gx, dtype=np.int32))
    cy = np.ascontiguousarray(np.asarray(gy, dtype=np.int32))
    m = fr.shape[0]
    out = np.zeros(m, np.float64)
    r = _load().oracle_density_cells(_ptr(a), _ptr(off), F, int(width_px), int(height_px),
                                     int(grid_w), int(grid_h), float(sigma_px), _ptr(fr),
                                     _ptr(cx), _ptr(cy), m, _ptr(out),
                                     n_threads or default_threads())
    _check(r, "density_cells")
    return out


def heatmap_frames(density, cell_area: float, threshold: float, connectivity: int = 8,
                   n_threads: int | None = None):
    """Heatmap analytics of float32 density grids [F, grid_h, grid_w].

    Returns a dict: labels int32[F, h, w] (smallest cell index of the
    component, -1 cold), n_components int32[F], entropy float64[F],
    degree float64[F], comp_cells int32[F, h, w] and comp_mass float64[F, h, w]
    (at label cells, 0 elsewhere).
    """
    d = np.ascontiguousarray(np.asarray(density, dtype=np.float32))
    if d.ndim != 3:
        raise ValueError("density must be [F, grid_h, grid_w]")
    F, gh, gw = d.shape
    labels = np.zeros(d.shape, np.int32)
    comp_cells = np.zeros(d.shape, np.int32)
    comp_mass = np.zeros(d.shape, np.float64)
    ncomp = np.zeros(F, np.int32)
    ent = np.zeros(F, np.float64)
    deg = np.zeros(F, np.float64)
    r = _load().oracle_heatmap_frames(_ptr(d), F, gw, gh, float(cell_area), float(threshold),
                                      int(connectivity), _ptr(labels), _ptr(ncomp), _ptr(ent),
                                      _ptr(deg), _ptr(comp_cells), _ptr(comp_mass),
                                      n_threads or default_threads())
    _check(r, "heatmap_frames")
    return {"labels": labels, "n_components": ncomp, "entropy": ent, "degree": deg,
            "comp_cells": comp_cells, "comp_mass": comp_mass}


def point_in_polygon(poly, x: int, y: int) -> bool:
    """Closed polygon (even-odd rule) test of one point, exact integers."""
    pg = np.ascontiguousarray(np.asarray(poly, dtype=np.int32).reshape(-1, 2))
    return bool(_load().oracle_point_in_polygon(_ptr(pg), pg.shape[0], int(x), int(y)))


def roi_filter(xy, offsets, poly):
    """Birds inside the ROI polygon (closed, even-odd), in input order.

    Returns a dict: counts int32[F], xy int32[K, 2], offsets int32[F + 1]
    (CSR of the kept birds), index int32[K] (their input indices).
    """
    a = _xy(xy)
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32))
    pg = np.ascontiguousarray(np.asarray(poly, dtype=np.int32).reshape(-1, 2))
    F = off.shape[0] - 1
    if int(off[-1]) != a.shape[0]:
        raise ValueError("offsets do not describe xy")
    counts = np.zeros(max(F, 0), np.int32)
    oxy = np.zeros_like(a)
    ooff = np.zeros(F + 1, np.int32)
    oidx = np.zeros(a.shape[0], np.int32)
    k = _load().oracle_roi_filter(_ptr(a), _ptr(off), F, _ptr(pg), pg.shape[0], _ptr(counts), _ptr(oxy),
                                  _ptr(ooff), _ptr(oidx))
    _check(k, "roi_filter")
    return {"counts": counts, "xy": oxy[:k].copy(), "offsets": ooff, "index": oidx[:k].copy()}


def near_segment(x: int, y: int, seg, t: int) -> bool:
    """Is point (x, y) strictly closer than t to the closed segment (ax, ay, bx, by)?"""
    ax, ay, bx, by = (int(v) for v in seg)
    return bool(_load().oracle_near_segment(int(x), int(y), ax, ay, bx, by, int(t)))


def drinkers(xy, offsets, lines, t: int):
    """Birds strictly closer than t quanta to some drinker-line segment.

    Returns a dict: drinking uint8[T], line int32[T] (smallest index of such a
    segment, -1 if none), counts int32[F].
    """
    a = _xy(xy)
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32))
    ln = np.ascontiguousarray(np.asarray(lines, dtype=np.int32).reshape(-1, 4))
    F = off.shape[0] - 1
    if int(off[-1]) != a.shape[0]:
        raise ValueError("offsets do not describe xy")
    drinking = np.zeros(a.shape[0], np.uint8)
    line = np.zeros(a.shape[0], np.int32)
    counts = np.zeros(max(F, 0), np.int32)
    r = _load().oracle_drinkers(_ptr(a), _ptr(off), F, _ptr(ln), ln.shape[0], int(t), _ptr(drinking),
                                _ptr(line), _ptr(counts))
    _check(r, "drinkers")
    return {"drinking": drinking, "line": line, "counts": counts}


def mask_components(prob, threshold: float, connectivity: int = 8):
    """Connected components of prob > threshold in float32 masks [F, H, W].

    Returns a dict: labels int32[F, H, W] (first pixel of the component in
    raster order, -1 background), n_components int32[F], offsets int64[F + 1]
    (CSR of the component list), label int32[K], area int32[K],
    box int32[K, 4] (x, y, width, height), centroid float64[K, 2],
    xy int32[K, 2] (centroid in 1/16 px, floor(16 * sum / area)),
    score float32[K] (largest probability in the component).
    """
    p = np.ascontiguousarray(np.asarray(prob, dtype=np.float32))
    if p.ndim != 3:
        raise ValueError("prob must be [F, H, W]")
    F, h, w = p.shape
    labels = np.zeros(p.shape, np.int32)
    ncomp = np.zeros(F, np.int32)
    offs = np.zeros(F + 1, np.int64)

    def run(cap):
        lab = np.zeros(cap, np.int32)
        area = np.zeros(cap, np.int32)
        box = np.zeros((cap, 4), np.int32)
        cen = np.zeros((cap, 2), np.float64)
        qxy = np.zeros((cap, 2), np.int32)
        score = np.zeros(cap, np.float32)
        k = _load().oracle_mask_components(_ptr(p), F, w, h, float(threshold), int(connectivity), _ptr(labels),
                                           _ptr(ncomp), _ptr(offs), cap, _ptr(lab), _ptr(area), _ptr(box),
                                           _ptr(cen), _ptr(qxy), _ptr(score))
        _check(int(k), "mask_components")
        return int(k), lab, area, box, cen, qxy, score

    # small batches in one pass; large ones count first, then fill
    k, lab, area, box, cen, qxy, score = run(int(p.size) if p.size <= (1 << 22) else 0)
    if k > lab.shape[0]:
        k, lab, area, box, cen, qxy, score = run(k)
    return {"labels": labels, "n_components": ncomp, "offsets": offs, "label": lab[:k].copy(),
            "area": area[:k].copy(), "box": box[:k].copy(), "centroid": cen[:k].copy(),
            "xy": qxy[:k].copy(), "score": score[:k].copy()}

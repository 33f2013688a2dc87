"""Seeded synthetic workloads: ragged batches of bird centroids.

The paper's farm footage is private, so every input here is synthetic, shaped
after what the paper states about it: overhead 1080p cameras (Section 2.1),
10k-30k birds per house (Section 1), five-minute 30 fps videos and tracked
per-frame positions feeding the clustering module (Sections 2.3, 3.6, 4).

This module draws random numbers only.  It holds none of the arithmetic of
the clustering or density method, and it is the one piece of code shared by
the HIP path's callers and the CPU oracle's callers.

Layout of a batch (the CSR form the library consumes):
  xy      int32 [T, 2]   (x, y) in 1/16 px, 0 <= x < 16*W, 0 <= y < 16*H
  offsets int32 [F + 1]  offsets[0] = 0, non-decreasing, offsets[F] = T;
                          frame f is xy[offsets[f]:offsets[f+1]]

Quantisation: a position p px becomes floor(16 p) quanta.
"""

from __future__ import annotations

from dataclasses import dataclass, asdict

import numpy as np

QUANTA_PER_PX = 16


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: batch shape plus the method's parameters."""

    name: str
    seed: int
    n_frames: int
    width_px: int
    height_px: int
    eps_px: float
    min_pts: int
    grid_w: int
    grid_h: int
    sigma_px: float
    recipe: str

    @property
    def eps_q(self) -> int:
        return int(round(self.eps_px * QUANTA_PER_PX))

    def as_dict(self) -> dict:
        return asdict(self)


WORKLOADS: dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("single500_1080p", 1001, 1, 1920, 1080, 40.0, 4, 64, 36, 30.0,
                 "1 frame, 500 birds uniform over the frame"),
        Workload("batch64x2000_1080p", 1002, 64, 1920, 1080, 40.0, 4, 128, 72, 30.0,
                 "64 frames x 2000 birds: 6-component Gaussian mixture "
                 "(std 80-200 px) + 10% uniform noise"),
        Workload("batch256xpoisson8000_4k", 1003, 256, 3840, 2160, 60.0, 5, 256, 144, 45.0,
                 "256 frames, Poisson(8000) birds each: 12-component mixture "
                 "(std 60-300 px)"),
        Workload("house30000_4k", 1004, 1, 3840, 2160, 25.0, 6, 512, 288, 20.0,
                 "1 frame, 30000 birds: 70% uniform + 20 tight clusters (std 40 px)"),
        Workload("stream1800x5000_1080p", 1005, 1800, 1920, 1080, 40.0, 4, 128, 72, 30.0,
                 "1800-frame stream of 5000 birds: N(0,2 px) jitter per frame, "
                 "1% re-spawned uniformly"),
    ]
}

# Order used by tests and the bench: smallest case first, headline second.
WORKLOAD_ORDER = list(WORKLOADS)


def _quantise(p: np.ndarray, extent_px: int) -> np.ndarray:
    q = np.floor(p * QUANTA_PER_PX).astype(np.int64)
    return np.clip(q, 0, QUANTA_PER_PX * extent_px - 1).astype(np.int32)


def _uniform(rng, n, w, h):
    return rng.uniform(0.0, w, n), rng.uniform(0.0, h, n)


def _mixture(rng, n, w, h, n_comp, std_lo, std_hi):
    """n draws from an equal-weight isotropic Gaussian mixture; draws that
    fall outside [0, w) x [0, h) are drawn again from the same component."""
    mx = rng.uniform(0.0, w, n_comp)
    my = rng.uniform(0.0, h, n_comp)
    sd = rng.uniform(std_lo, std_hi, n_comp)
    comp = rng.integers(0, n_comp, n)
    x = np.empty(n)
    y = np.empty(n)
    todo = np.arange(n)
    while todo.size:
        c = comp[todo]
        xs = rng.normal(mx[c], sd[c])
        ys = rng.normal(my[c], sd[c])
        ok = (xs >= 0) & (xs < w) & (ys >= 0) & (ys < h)
        x[todo[ok]] = xs[ok]
        y[todo[ok]] = ys[ok]
        todo = todo[~ok]
    return x, y


def _frame_to_q(x, y, w, h):
    return np.stack([_quantise(x, w), _quantise(y, h)], axis=1)


def generate(name: str, n_frames: int | None = None):
    """Return (xy int32[T,2], offsets int32[F+1], Workload) for a named workload.

    Frames are drawn in order from one generator, so the first k frames of a
    workload are identical whatever n_frames asks for (a prefix is a valid
    bounded sample of the full batch).
    """
    wl = WORKLOADS[name]
    F = wl.n_frames if n_frames is None else min(int(n_frames), wl.n_frames)
    rng = np.random.default_rng(wl.seed)
    W, H = wl.width_px, wl.height_px
    frames: list[np.ndarray] = []

    if name == "single500_1080p":
        for _ in range(F):
            x = rng.integers(0, QUANTA_PER_PX * W, 500)
            y = rng.integers(0, QUANTA_PER_PX * H, 500)
            frames.append(np.stack([x, y], axis=1).astype(np.int32))
    elif name == "batch64x2000_1080p":
        for _ in range(F):
            x1, y1 = _mixture(rng, 1800, W, H, 6, 80.0, 200.0)
            x2, y2 = _uniform(rng, 200, W, H)
            q = _frame_to_q(np.concatenate([x1, x2]), np.concatenate([y1, y2]), W, H)
            frames.append(q[rng.permutation(q.shape[0])])
    elif name == "batch256xpoisson8000_4k":
        for _ in range(F):
            n = int(rng.poisson(8000))
            x, y = _mixture(rng, n, W, H, 12, 60.0, 300.0)
            q = _frame_to_q(x, y, W, H)
            frames.append(q[rng.permutation(n)])
    elif name == "house30000_4k":
        for _ in range(F):
            x1, y1 = _uniform(rng, 21000, W, H)
            xs, ys = [x1], [y1]
            for _c in range(20):
                xc, yc = _mixture(rng, 450, W, H, 1, 40.0, 40.0)
                xs.append(xc)
                ys.append(yc)
            q = _frame_to_q(np.concatenate(xs), np.concatenate(ys), W, H)
            frames.append(q[rng.permutation(q.shape[0])])
    elif name == "stream1800x5000_1080p":
        n = 5000
        x1, y1 = _mixture(rng, 4500, W, H, 6, 80.0, 200.0)
        x2, y2 = _uniform(rng, 500, W, H)
        perm = rng.permutation(n)
        x = np.concatenate([x1, x2])[perm]
        y = np.concatenate([y1, y2])[perm]
        top_x = np.nextafter(float(W), 0.0)
        top_y = np.nextafter(float(H), 0.0)
        for t in range(F):
            if t > 0:
                x = np.clip(x + rng.normal(0.0, 2.0, n), 0.0, top_x)
                y = np.clip(y + rng.normal(0.0, 2.0, n), 0.0, top_y)
                re = rng.choice(n, 50, replace=False)
                x[re] = rng.uniform(0.0, W, 50)
                y[re] = rng.uniform(0.0, H, 50)
            frames.append(_frame_to_q(x, y, W, H))
    else:  # pragma: no cover - WORKLOADS and this switch list the same names
        raise KeyError(name)

    return pack(frames) + (wl,)


def pack(frames: list[np.ndarray]):
    """Concatenate per-frame int32[n_f, 2] arrays into (xy, offsets)."""
    counts = np.array([f.shape[0] for f in frames], dtype=np.int64)
    offsets = np.zeros(len(frames) + 1, dtype=np.int64)
    np.cumsum(counts, out=offsets[1:])
    if frames and offsets[-1] > 0:
        xy = np.ascontiguousarray(np.concatenate(frames, axis=0), dtype=np.int32)
    else:
        xy = np.zeros((0, 2), dtype=np.int32)
    return xy, offsets.astype(np.int32)


def random_batch(seed: int, n_frames: int, max_points: int, width_px: int = 1920,
                 height_px: int = 1080, clustered: bool = True,
                 dup_frac: float = 0.05, empty_frac: float = 0.1):
    """Small ragged batch for parity tests: empty frames, duplicate points,
    clustered and uniform frames, and counts drawn uniformly in [0, max_points]."""
    rng = np.random.default_rng(seed)
    frames = []
    for _ in range(n_frames):
        if rng.random() < empty_frac:
            frames.append(np.zeros((0, 2), np.int32))
            continue
        n = int(rng.integers(0, max_points + 1))
        if clustered and n > 0 and rng.random() < 0.7:
            k = int(rng.integers(1, 6))
            x, y = _mixture(rng, n, width_px, height_px, k, 10.0, 120.0)
        else:
            x, y = _uniform(rng, n, width_px, height_px)
        q = _frame_to_q(x, y, width_px, height_px)
        nd = int(dup_frac * n)
        if nd and n > 1:
            src = rng.integers(0, n, nd)
            dst = rng.integers(0, n, nd)
            q[dst] = q[src]
        frames.append(q)
    return pack(frames)


def lattice_frame(nx: int, ny: int, step_q: int, x0: int = 0, y0: int = 0):
    """Points on a square lattice with spacing step_q quanta (exact-distance
    ties for the radius test when step_q equals the radius)."""
    gx, gy = np.meshgrid(np.arange(nx), np.arange(ny))
    return np.stack([x0 + step_q * gx.ravel(), y0 + step_q * gy.ravel()], axis=1).astype(np.int32)


def heat_grids(seed: int, n_frames: int, grid_h: int, grid_w: int, n_blobs: int = 6,
               peak: float = 1e-3, empty_frac: float = 0.1) -> np.ndarray:
    """Seeded density-like grids float32[F, grid_h, grid_w] for the heatmap
    analytics: per frame a few cone-shaped blobs (value peak * max(0, 1 - r/R),
    random centre, radius R and height) over a faint random floor, some cells
    exactly zero, and some frames all zero.  Not a kernel density estimate:
    only grids of the right shape and value range."""
    rng = np.random.default_rng(seed)
    gy, gx = np.meshgrid(np.arange(grid_h, dtype=np.float64), np.arange(grid_w, dtype=np.float64), indexing="ij")
    out = np.zeros((n_frames, grid_h, grid_w), np.float32)
    for f in range(n_frames):
        if rng.random() < empty_frac:
            continue
        g = rng.random((grid_h, grid_w)) * peak * 0.05
        g[rng.random((grid_h, grid_w)) < 0.2] = 0.0
        for _ in range(int(rng.integers(1, n_blobs + 1))):
            cx, cy = rng.uniform(0, grid_w), rng.uniform(0, grid_h)
            rad = rng.uniform(1.5, max(2.0, 0.3 * max(grid_w, grid_h)))
            amp = peak * rng.uniform(0.2, 1.0)
            g += amp * np.maximum(0.0, 1.0 - np.hypot(gx - cx, gy - cy) / rad)
        out[f] = g.astype(np.float32)
    return out


@dataclass(frozen=True)
class MaskWorkload:
    """One synthetic batch of segmentation outputs for the detection
    post-processing: per-pixel bird probabilities, float32 [F, H, W]."""

    name: str
    seed: int
    n_frames: int
    width_px: int
    height_px: int
    n_birds: int
    threshold: float
    connectivity: int
    recipe: str

    def as_dict(self) -> dict:
        return asdict(self)


MASK_WORKLOADS: dict[str, MaskWorkload] = {
    w.name: w
    for w in [
        MaskWorkload("masks8x2000_720p", 2001, 8, 1280, 720, 2000, 0.5, 8,
                     "batch of 8 frames at 1280x720, 2000 elliptical birds per frame "
                     "(6-component mixture + 10% uniform), speckle false positives"),
        MaskWorkload("masks8x2000_1080p", 2002, 8, 1920, 1080, 2000, 0.5, 8,
                     "batch of 8 frames at 1920x1080, 2000 elliptical birds per frame "
                     "(6-component mixture + 10% uniform), speckle false positives"),
    ]
}


def bird_masks(seed: int, n_frames: int, height_px: int, width_px: int, n_birds: int,
               major_px: tuple = (7.0, 10.0), minor_px: tuple = (4.0, 6.0),
               speckle_frac: float = 2e-4, empty_frac: float = 0.0) -> np.ndarray:
    """Seeded probability maps float32[F, H, W] shaped like a segmentation
    network's bird output: a faint background in [0, 0.1), one soft ellipse
    per bird (random orientation, semi-axes drawn from major_px and minor_px,
    value 1 at the centre falling below 0.5 a little outside the nominal
    ellipse; overlapping birds keep the larger value), birds placed by a
    6-component Gaussian mixture (std 80-200 px at 1920 px width, scaled with
    the width) plus 10% uniform, and isolated speckle pixels in [0.5, 1)
    (single-pixel false positives).  Frames drawn empty (background only)
    with probability empty_frac."""
    rng = np.random.default_rng(seed)
    H, W = int(height_px), int(width_px)
    out = np.empty((n_frames, H, W), np.float32)
    scale = W / 1920.0
    for f in range(n_frames):
        g = rng.random((H, W), dtype=np.float32) * np.float32(0.1)
        if rng.random() < empty_frac or n_birds <= 0:
            out[f] = g
            continue
        n_mix = int(round(0.9 * n_birds))
        x1, y1 = _mixture(rng, n_mix, W, H, 6, 80.0 * scale, 200.0 * scale)
        x2, y2 = _uniform(rng, n_birds - n_mix, W, H)
        xs, ys = np.concatenate([x1, x2]), np.concatenate([y1, y2])
        maj = rng.uniform(*major_px, n_birds)
        mnr = rng.uniform(*minor_px, n_birds)
        th = rng.uniform(0.0, np.pi, n_birds)
        for cx, cy, a, b, t in zip(xs, ys, maj, mnr, th):
            r = int(np.ceil(1.1 * a)) + 1
            xa, xb = max(0, int(cx) - r), min(W, int(cx) + r + 1)
            ya, yb = max(0, int(cy) - r), min(H, int(cy) + r + 1)
            if xa >= xb or ya >= yb:
                continue
            yy, xx = np.mgrid[ya:yb, xa:xb]
            dx, dy = xx + 0.5 - cx, yy + 0.5 - cy
            u = dx * np.cos(t) + dy * np.sin(t)
            v = -dx * np.sin(t) + dy * np.cos(t)
            p = np.clip(1.15 - 0.6 * ((u / a) ** 2 + (v / b) ** 2), 0.0, 1.0).astype(np.float32)
            np.maximum(g[ya:yb, xa:xb], p, out=g[ya:yb, xa:xb])
        k = int(rng.binomial(H * W, speckle_frac))
        if k:
            idx = rng.integers(0, H * W, k)
            g.ravel()[idx] = rng.uniform(0.5, 1.0, k).astype(np.float32)
        out[f] = g
    return out


def mask_batch(name: str, n_frames: int | None = None):
    """(prob float32[F, H, W], MaskWorkload) for a named mask workload; the
    first k frames are the same whatever n_frames asks for."""
    wl = MASK_WORKLOADS[name]
    F = wl.n_frames if n_frames is None else min(int(n_frames), wl.n_frames)
    s = wl.width_px / 1280.0
    prob = bird_masks(wl.seed, F, wl.height_px, wl.width_px, wl.n_birds,
                      major_px=(7.0 * s, 10.0 * s), minor_px=(4.0 * s, 6.0 * s))
    return prob, wl

"""The C ABI library loads, exports what include/flock.h declares, and rejects
bad arguments on the host before touching any device (no GPU needed)."""

import ctypes
import math
import os
import re

import pytest

from paper_2512_07009_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flock.h")

FAKE = ctypes.c_void_p(0x100000)       # never dereferenced on the EINVAL paths
FAKE4 = ctypes.c_void_p(0x100004)      # 4-byte aligned, not 8


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, re.M)))


def test_library_exports_every_declared_function():
    lib = binding.lib()
    names = declared_functions()
    assert {"cluster_frames", "density_frames", "cluster_frames_workspace",
            "density_frames_workspace", "flock_last_error", "flock_version"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name
    assert binding.version().startswith("flock ")


def _cluster(n_frames=1, total=4, max_fp=0, eps_q=640, min_pts=4, xy=FAKE, offsets=FAKE,
             labels=FAKE, kind=FAKE, ncl=FAKE):
    return binding.lib().cluster_frames(xy, offsets, n_frames, total, max_fp, eps_q, min_pts,
                                        labels, kind, ncl, None, 0, None)


def _density(n_frames=1, total=4, max_fp=0, w=1920, h=1080, gx=128, gy=72, sigma=30.0, xy=FAKE,
             offsets=FAKE, out=FAKE):
    return binding.lib().density_frames(xy, offsets, n_frames, total, max_fp, w, h, gx, gy, sigma,
                                        out, None, 0, None)


@pytest.mark.parametrize("kwargs,needle", [
    (dict(n_frames=-1), "n_frames"),
    (dict(total=-5), "total"),
    (dict(max_fp=-1), "max_frame_points"),
    (dict(eps_q=-1), "eps_q"),
    (dict(eps_q=32767), "eps_q"),
    (dict(min_pts=0), "min_pts"),
    (dict(offsets=None), "offsets"),
    (dict(xy=None), "non-NULL"),
    (dict(labels=None), "non-NULL"),
    (dict(xy=FAKE4), "aligned"),
])
def test_cluster_rejects_bad_arguments(kwargs, needle):
    assert _cluster(**kwargs) == binding.FLOCK_EINVAL
    assert needle in binding.lib().flock_last_error().decode()


@pytest.mark.parametrize("kwargs,needle", [
    (dict(n_frames=-1), "n_frames"),
    (dict(max_fp=-2), "max_frame_points"),
    (dict(w=0), "extent"),
    (dict(h=-3), "extent"),
    (dict(gx=0), "grid"),
    (dict(gy=5000), "grid"),
    (dict(sigma=0.0), "sigma"),
    (dict(sigma=-1.0), "sigma"),
    (dict(sigma=math.nan), "sigma"),
    (dict(sigma=math.inf), "sigma"),
    (dict(out=None), "non-NULL"),
    (dict(xy=FAKE4), "aligned"),
])
def test_density_rejects_bad_arguments(kwargs, needle):
    assert _density(**kwargs) == binding.FLOCK_EINVAL
    assert needle in binding.lib().flock_last_error().decode()


def _density_noalloc(n_frames=1, total=4, max_fp=0, w=1920, h=1080, gx=128, gy=72, sigma=30.0, xy=FAKE,
                     offsets=FAKE, out=FAKE):
    return binding.lib().density_frames_noalloc(xy, offsets, n_frames, total, max_fp, w, h, gx, gy, sigma,
                                                out, None)


@pytest.mark.parametrize("kwargs,needle", [
    (dict(n_frames=-1), "n_frames"),
    (dict(gy=5000), "grid"),
    (dict(sigma=math.nan), "sigma"),
    (dict(out=None), "non-NULL"),
    (dict(xy=FAKE4), "aligned"),
])
def test_density_noalloc_rejects_bad_arguments(kwargs, needle):
    assert _density_noalloc(**kwargs) == binding.FLOCK_EINVAL
    assert needle in binding.lib().flock_last_error().decode()
    assert _density_noalloc(n_frames=0, total=0, xy=None, offsets=None, out=None) == 0


def _heatmap(n_frames=1, gw=128, gh=72, area=225.0, thr=1e-4, conn=8, dens=FAKE, labels=FAKE, ncomp=FAKE,
             ent=FAKE, deg=FAKE, cells=FAKE, mass=FAKE):
    return binding.lib().heatmap_frames(dens, n_frames, gw, gh, area, thr, conn, labels, ncomp, ent, deg,
                                        cells, mass, None, 0, None)


@pytest.mark.parametrize("kwargs,needle", [
    (dict(n_frames=-1), "n_frames"),
    (dict(gw=0), "grid"),
    (dict(gh=4097), "grid"),
    (dict(area=-1.0), "cell_area"),
    (dict(area=math.inf), "cell_area"),
    (dict(thr=0.0), "threshold"),
    (dict(thr=-1.0), "threshold"),
    (dict(thr=math.nan), "threshold"),
    (dict(conn=6), "connectivity"),
    (dict(dens=None), "non-NULL"),
    (dict(mass=None), "non-NULL"),
    (dict(mass=FAKE4), "aligned"),
    (dict(ent=FAKE4), "aligned"),
])
def test_heatmap_rejects_bad_arguments(kwargs, needle):
    assert _heatmap(**kwargs) == binding.FLOCK_EINVAL
    assert needle in binding.lib().flock_last_error().decode()


SQUARE = (ctypes.c_int32 * 8)(0, 0, 160, 0, 160, 160, 0, 160)
FAR = (ctypes.c_int32 * 8)(0, 0, 1 << 25, 0, 160, 160, 0, 160)


def _roi(n_frames=1, total=4, poly=SQUARE, nv=4, xy=FAKE, offsets=FAKE, counts=FAKE, oxy=FAKE, ooff=FAKE,
         oidx=FAKE):
    return binding.lib().roi_filter_frames(xy, offsets, n_frames, total, poly, nv, counts, oxy, ooff, oidx,
                                           None, 0, None)


@pytest.mark.parametrize("kwargs,needle", [
    (dict(n_frames=-1), "n_frames"),
    (dict(total=-1), "total"),
    (dict(nv=2), "n_vertices"),
    (dict(nv=65), "n_vertices"),
    (dict(poly=None), "roi_xy"),
    (dict(poly=FAR), "2^24"),
    (dict(offsets=None), "non-NULL"),
    (dict(ooff=None), "non-NULL"),
    (dict(oxy=None), "non-NULL"),
    (dict(xy=FAKE4), "aligned"),
])
def test_roi_rejects_bad_arguments(kwargs, needle):
    assert _roi(**kwargs) == binding.FLOCK_EINVAL
    assert needle in binding.lib().flock_last_error().decode()


LINES = (ctypes.c_int32 * 8)(0, 0, 160, 0, 0, 0, 0, 160)
FAR_LINE = (ctypes.c_int32 * 4)(0, 0, -(1 << 25), 0)


def _drink(n_frames=1, total=4, lines=LINES, nl=2, thr=64, xy=FAKE, offsets=FAKE, drinking=FAKE, line=FAKE,
           counts=FAKE):
    return binding.lib().drinker_proximity_frames(xy, offsets, n_frames, total, lines, nl, thr, drinking, line,
                                                  counts, None, 0, None)


@pytest.mark.parametrize("kwargs,needle", [
    (dict(n_frames=-1), "n_frames"),
    (dict(total=-1), "total"),
    (dict(nl=0), "n_lines"),
    (dict(nl=65), "n_lines"),
    (dict(lines=None), "lines"),
    (dict(lines=FAR_LINE, nl=1), "2^24"),
    (dict(thr=-1), "threshold_q"),
    (dict(thr=(1 << 24) + 1), "threshold_q"),
    (dict(offsets=None), "non-NULL"),
    (dict(drinking=None), "non-NULL"),
    (dict(drinking=FAKE4), "16-byte"),
    (dict(xy=FAKE4), "aligned"),
])
def test_drinkers_rejects_bad_arguments(kwargs, needle):
    assert _drink(**kwargs) == binding.FLOCK_EINVAL
    assert needle in binding.lib().flock_last_error().decode()


def _mask(n_frames=1, w=64, h=48, thr=0.5, conn=8, cap=16, prob=FAKE, labels=FAKE, ncomp=FAKE, offs=FAKE,
          lab=FAKE, area=FAKE, box=FAKE, cen=FAKE, xy=FAKE, score=FAKE):
    return binding.lib().mask_components_frames(prob, n_frames, w, h, thr, conn, labels, ncomp, offs, cap, lab, area,
                                                box, cen, xy, score, None, 0, None)


@pytest.mark.parametrize("kwargs,needle", [
    (dict(n_frames=-1), "n_frames"),
    (dict(w=0), "frame"),
    (dict(h=32769), "frame"),
    (dict(thr=-0.5), "threshold"),
    (dict(thr=math.nan), "threshold"),
    (dict(thr=math.inf), "threshold"),
    (dict(conn=6), "connectivity"),
    (dict(cap=-1), "capacity"),
    (dict(prob=None), "non-NULL"),
    (dict(offs=None), "non-NULL"),
    (dict(ncomp=None), "non-NULL"),
    (dict(prob=ctypes.c_void_p(0x100002)), "aligned"),
    (dict(box=FAKE4), "16-byte"),
    (dict(cen=FAKE4), "16-byte"),
    (dict(xy=FAKE4), "8-byte"),
])
def test_mask_rejects_bad_arguments(kwargs, needle):
    assert _mask(**kwargs) == binding.FLOCK_EINVAL
    assert needle in binding.lib().flock_last_error().decode()


def test_mask_rejects_batches_beyond_int32_pixels():
    assert _mask(n_frames=1024, w=32768, h=32768) == binding.FLOCK_EUNSUPPORTED


def test_empty_batches_are_noops_without_a_device():
    assert _mask(n_frames=0, prob=None, labels=None, ncomp=None, offs=None, lab=None, area=None, box=None, cen=None,
                 xy=None, score=None) == 0
    assert _drink(n_frames=0, total=0, xy=None, offsets=None, drinking=None, line=None, counts=None) == 0
    assert _roi(n_frames=0, total=0, xy=None, offsets=None, counts=None, oxy=None, ooff=None, oidx=None) == 0
    assert _heatmap(n_frames=0, dens=None, labels=None, ncomp=None, ent=None, deg=None, cells=None,
                    mass=None) == 0
    assert _cluster(n_frames=0, total=0, xy=None, offsets=None, labels=None, kind=None, ncl=None) == 0
    assert _density(n_frames=0, total=0, xy=None, offsets=None, out=None) == 0
    assert binding.lib().flock_last_error().decode() == ""


def test_workspace_queries():
    lib = binding.lib()
    assert lib.cluster_frames_workspace(64, 128000, 2000) >= 0
    assert lib.density_frames_workspace(64, 128000, 128, 72) >= 0
    assert lib.heatmap_frames_workspace(64, 128, 72) > 0
    assert lib.heatmap_frames_workspace(0, 128, 72) == 0
    assert lib.roi_filter_frames_workspace(64, 128000) >= 128000
    assert lib.roi_filter_frames_workspace(0, 0) == 0
    assert lib.drinker_proximity_frames_workspace(64, 128000) > 0
    assert lib.drinker_proximity_frames_workspace(0, 0) == 0
    # 8 neighbours: a record and a key (56 bytes) per 2 x 2 block of pixels
    assert lib.mask_components_frames_workspace(8, 1280, 720, 8) >= 56 * 8 * 640 * 360
    assert lib.mask_components_frames_workspace(8, 1280, 720, 4) >= 56 * 8 * 1280 * 720 // 2
    assert lib.mask_components_frames_workspace(0, 1280, 720, 8) == 0


def test_eps_to_quanta():
    assert binding.eps_to_quanta(40.0) == 640
    assert binding.eps_to_quanta(25.0) == 400
    assert binding.eps_to_quanta(0.0625) == 1
    with pytest.raises(ValueError):
        binding.eps_to_quanta(0.01)

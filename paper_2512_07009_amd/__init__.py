"""MI355X (gfx950) per-frame bird clustering and Gaussian density grids.

The hot path of the clustering module of "Optimizing Video Analytics
Inference Pipelines: A Case Study" (arXiv 2512.07009, Section 2.3 and
Section 3.6 / Algorithm 1, and its heatmap thresholding, grid components,
entropy and clustering degree, and the region-of-interest filter with
per-frame region counts, and drinker-line proximity), and the detection
post-processing of Section 3.2 (mask components with statistics), as hand-written HIP
kernels behind a C ABI (include/flock.h, libflock.so).  This package is the thin Python binding:

    labels, kind, n_clusters = cluster_frames(xy, offsets, eps_px, min_pts)
    density = density_frames(xy, offsets, width_px, height_px, grid_w, grid_h, sigma_px)
    stats = heatmap_frames(density, cell_area_px2, threshold, connectivity)
    kept = roi_filter_frames(xy, offsets, roi_polygon_quanta)
    near = drinker_proximity_frames(xy, offsets, drinker_segments_quanta, threshold_quanta)
    det = mask_components_frames(prob, threshold, connectivity)

``workloads`` holds the seeded synthetic input generators.
"""

from .binding import (FlockError, cluster_frames, density_frames, drinker_proximity_frames,  # noqa: F401
                      eps_to_quanta, heatmap_frames, lib, mask_capacity, mask_components_frames,
                      roi_filter_frames, version)

__all__ = ["cluster_frames", "density_frames", "heatmap_frames", "roi_filter_frames", "drinker_proximity_frames",
           "mask_components_frames", "mask_capacity", "eps_to_quanta", "lib", "version", "FlockError"]

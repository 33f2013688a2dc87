/*
 * flock.h - C ABI of the MI355X (gfx950) per-frame bird clustering and
 * density library (libflock.so).
 *
 * The library computes, for a batch of video frames that each hold a ragged
 * set of detected bird centroids, the two per-frame analytics of the paper's
 * clustering module (Section 2.3; Section 3.6 and Algorithm 1):
 *   - radius-neighbour clustering of the birds (core / border / noise kinds
 *     and connected-component cluster labels), and
 *   - a Gaussian kernel density grid.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  Batch layout (CSR over frames; the paper's "frames" of tracked positions,
 *  Algorithm 1):
 *    xy       device, int32[total][2]: (x, y) of each bird in 1/16 px,
 *             0 <= x, y < 2^24.  Frame f is rows offsets[f] .. offsets[f+1]-1.
 *    offsets  device, int32[n_frames + 1]: offsets[0] = 0, non-decreasing,
 *             offsets[n_frames] = total.
 *    n_frames, total: host copies of the batch sizes.
 *  Every pointer argument is device memory owned by the caller; the library
 *  neither frees nor keeps it after the call returns.
 *  stream: a hipStream_t (NULL = the null stream).  Calls only enqueue work:
 *  outputs are valid once the stream reaches the call's point.  No host-device
 *  copy and no synchronisation happens, except when the environment variable
 *  FLOCK_VALIDATE=1 asks for a synchronous device-side check of offsets.
 *  Errors: a negative status; flock_last_error() then describes it.  On
 *  FLOCK_EINVAL nothing is enqueued and the outputs are untouched.  A frame
 *  whose offsets are inconsistent (negative count, past total) is never read;
 *  its outputs are left untouched and its n_clusters entry is set to -1.
 *  Thread safety: calls on different streams may run concurrently; the only
 *  global state is a per-thread error string and a once-initialised cache of
 *  device properties.
 *  Graph capture: a call enqueues only kernel launches when it is given the
 *  workspace its *_workspace() query asks for (or when that query returns 0),
 *  so it can be captured into a HIP graph.  With a NULL workspace where one
 *  is needed the library allocates and frees its scratch stream-ordered
 *  (hipMallocAsync / hipFreeAsync), which a capture records as memory nodes;
 *  pass a workspace (or use density_frames_noalloc) under capture.
 */
#ifndef FLOCK_H
#define FLOCK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t flock_status;

#define FLOCK_OK 0
#define FLOCK_EINVAL (-1)      /* bad argument: nothing enqueued, outputs untouched */
#define FLOCK_ENOMEM (-2)      /* workspace too small, or allocation failed */
#define FLOCK_EDEVICE (-3)     /* a HIP runtime call failed (message has its text) */
#define FLOCK_EUNSUPPORTED (-4) /* device is not gfx950, or a size beyond the limits */

/*
 * cluster_frames - radius-neighbour (DBSCAN-style) clustering of every frame.
 *
 * The paper's clustering module groups nearby birds by connected-component
 * analysis (Section 2.3) and names the per-frame distance loops as the
 * bottleneck (Section 3.6).  The point-level definition computed here is
 * standard DBSCAN (Ester et al., 1996) with these exact conventions:
 *   neighbours   (x_i - x_j)^2 + (y_i - y_j)^2 <= eps_q^2, in exact integer
 *                arithmetic on the 1/16-px coordinates; a bird is its own
 *                neighbour and coincident birds count;
 *   core         a bird with >= min_pts neighbours;
 *   cluster      a connected component of core birds under the neighbour
 *                relation; its label is the smallest frame-local index of a
 *                core bird in it (global index = label + offsets[f]);
 *   border       a non-core bird with a core neighbour: it joins the cluster
 *                of its nearest core neighbour, ties broken by the smaller
 *                (y, x) of that core;
 *   noise        every other bird: label -1.
 *
 * Arguments:
 *   max_frame_points  host: an upper bound on the birds in any one frame
 *                     (used to size on-chip storage), or 0 if unknown.  A
 *                     frame above the bound is still clustered correctly, on a
 *                     slower path.
 *   eps_q             radius in 1/16 px, 0 <= eps_q <= 32766 (eps px = eps_q/16).
 *   min_pts           >= 1; the count includes the bird itself.
 *   labels            device out, int32[total]: frame-local cluster label or -1.
 *   kind              device out, uint8[total]: 0 noise, 1 border, 2 core.
 *   n_clusters        device out, int32[n_frames] (or NULL): clusters per frame.
 *   workspace         device scratch of workspace_bytes bytes, at least
 *                     cluster_frames_workspace(...) of them, 256-byte aligned;
 *                     or NULL, in which case the library allocates and frees
 *                     its scratch stream-ordered (hipMallocAsync/hipFreeAsync).
 * Labels, kinds and n_clusters are a deterministic function of the input:
 * they do not depend on the order of birds within a frame beyond the labels'
 * index convention, nor on thread scheduling.
 */
flock_status cluster_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames,
                            int32_t total, int32_t max_frame_points, int32_t eps_q,
                            int32_t min_pts, int32_t *labels, uint8_t *kind,
                            int32_t *n_clusters, void *workspace, size_t workspace_bytes,
                            void *stream);

/* Bytes of workspace cluster_frames needs for this batch shape (may be 0). */
size_t cluster_frames_workspace(int32_t n_frames, int32_t total, int32_t max_frame_points);

/*
 * density_frames - Gaussian kernel density grid of every frame.
 *
 * Algorithm 1 (Section 3.6) computes, for every grid cell and every bird, a
 * distance-based contribution to the cell's density; the paper vectorises
 * the grid-to-bird distances.  The grid here has grid_w x grid_h cells tiling
 * the frame [0, width_px) x [0, height_px), evaluated at the cell centres
 *     cx = (gx + 1/2) width_px / grid_w,   cy = (gy + 1/2) height_px / grid_h,
 * and each bird (x, y) = (x_q/16, y_q/16) px adds an isotropic Gaussian of
 * bandwidth sigma_px with unit mass:
 *     density[f][gy][gx] = sum_i exp(-((cx-x_i)^2 + (cy-y_i)^2) / (2 sigma^2))
 *                          / (2 pi sigma^2)                    [birds / px^2]
 * The sum factorises as density = c * Fy . Fx^T with Fx[gx][i] and Fy[gy][i]
 * the per-axis Gaussian factors; it is evaluated as that contraction over
 * the birds on the matrix cores, fp16 factors with fp32 accumulation.
 * Accuracy: relative to the frame's maximum, |error| <= 1e-3 (the fp16
 * rounding of the two factors bounds each term's relative error by about
 * 2^-10); an empty frame gives exact zeros.
 *
 * Arguments:
 *   max_frame_points      host: an upper bound on the birds in any one frame,
 *                         or 0 if unknown (a planning hint; every value >= 0
 *                         gives the same result).
 *   width_px, height_px   frame extent, >= 1.
 *   grid_w, grid_h        grid size, 1 .. 4096 each.
 *   sigma_px              bandwidth, finite, > 0.
 *   density               device out, float[n_frames][grid_h][grid_w].
 *   workspace             as for cluster_frames, sized by
 *                         density_frames_workspace(...).  Batches with few
 *                         frames are split into bird slices whose partial
 *                         grids are kept there and added in slice order.
 * The result is deterministic (fixed summation order).  Frames whose offsets
 * are invalid (checked only with FLOCK_VALIDATE) leave their grid unspecified.
 */
flock_status density_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames,
                            int32_t total, int32_t max_frame_points, int32_t width_px,
                            int32_t height_px, int32_t grid_w, int32_t grid_h, float sigma_px,
                            float *density, void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of workspace density_frames needs for this batch shape and grid
 * (0 when no split is needed); the same value bounds every call with these
 * four arguments, whatever the frame extent and sigma. */
size_t density_frames_workspace(int32_t n_frames, int32_t total, int32_t grid_w, int32_t grid_h);

/*
 * density_frames_noalloc - density_frames for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid allocation.
 *
 * Arguments, result and accuracy are those of density_frames (the same plan
 * and kernels, so the same bits), without the workspace: a launch split into
 * bird slices keeps its partial grids in a static scratch array of the
 * library, 16 MiB per device (n_frames * slices * grid_w * grid_h * 4 bytes;
 * density_frames_workspace() gives that size for a batch shape).  The call
 * allocates nothing and makes no host-device copy or synchronisation
 * (FLOCK_VALIDATE is ignored here).
 * Errors: FLOCK_ENOMEM, with nothing enqueued, when the batch needs more
 * partial-grid bytes than the scratch holds; otherwise as density_frames.
 * Every call on one device shares that device's scratch: calls that overlap
 * in time on one device (concurrent streams, or threads) race and must be
 * serialised by the caller.  Every byte a call reads from the scratch it has
 * written first, so nothing needs clearing between calls.
 */
flock_status density_frames_noalloc(const int32_t *xy, const int32_t *offsets, int32_t n_frames,
                                    int32_t total, int32_t max_frame_points, int32_t width_px,
                                    int32_t height_px, int32_t grid_w, int32_t grid_h, float sigma_px,
                                    float *density, void *stream);

/*
 * heatmap_frames - heatmap analytics of every frame's density grid.
 *
 * The clustering module of Section 2.3 thresholds the density heatmaps and
 * applies connected component analysis; Algorithm 1 computes the heatmap,
 * its entropy and a clustering degree per frame.  The paper fixes none of
 * the details; this entry point computes, per frame f and cell
 * c = gy * grid_w + gx:
 *   hot          density[f][c] >= threshold;
 *   labels       connected hot cells under the 4-neighbourhood (shared edge)
 *                or the 8-neighbourhood (shared edge or corner) form a
 *                component, labelled by its smallest cell index; cold cells
 *                get -1;
 *   comp_cells, comp_mass   at each component's label cell, its number of
 *                cells and cell_area_px2 * (sum of its density) (expected
 *                birds); 0 at every other cell;
 *   n_components number of components;
 *   entropy      -sum p ln p over the cells with density > 0,
 *                p = density / S, S the sum of those cells (0 if S = 0);
 *   degree       (sum of density over hot cells) / S (0 if S = 0): the share
 *                of the frame's density mass that lies in components.
 *
 * Arguments:
 *   density          device in, float[n_frames][grid_h][grid_w], finite and
 *                    >= 0 (the output of density_frames).
 *   grid_w, grid_h   1 .. 4096 each.
 *   cell_area_px2    area of one cell in px^2 (W H / (grid_w grid_h)), >= 0.
 *   threshold        birds / px^2, finite and > 0.
 *   connectivity     4 or 8.
 *   labels, comp_cells   device out, int32[n_frames][grid_h][grid_w].
 *   comp_mass        device out, double[n_frames][grid_h][grid_w], 8-byte
 *                    aligned.
 *   n_components     device out, int32[n_frames].
 *   entropy, degree  device out, double[n_frames].
 *   workspace        as for cluster_frames, sized by heatmap_frames_workspace.
 * Every output is deterministic: sums are taken in a fixed order, and the
 * component masses are summed as 64-bit integers of a per-frame fixed-point
 * scale (each cell rounded to within 2^(lg - 62) of the frame's largest cell,
 * lg = ceil(log2(grid_w grid_h))).
 */
flock_status heatmap_frames(const float *density, int32_t n_frames, int32_t grid_w, int32_t grid_h,
                            double cell_area_px2, float threshold, int32_t connectivity,
                            int32_t *labels, int32_t *n_components, double *entropy, double *degree,
                            int32_t *comp_cells, double *comp_mass, void *workspace,
                            size_t workspace_bytes, void *stream);

/* Bytes of workspace heatmap_frames needs for this batch shape. */
size_t heatmap_frames_workspace(int32_t n_frames, int32_t grid_w, int32_t grid_h);

/*
 * roi_filter_frames - birds inside a region of interest, and per-frame counts.
 *
 * The wall pipeline counts the birds in a region near the wall (Section
 * 2.2), and Algorithm 1 filters the birds to the region of interest before
 * the density.  A bird is kept when its point (x_q, y_q) lies in the closed
 * polygon roi_xy (edges and vertices included; even-odd rule, which for a
 * simple polygon is its interior plus its boundary), tested exactly in
 * integers.  Kept birds keep their input order.
 *
 * Arguments:
 *   xy, offsets, n_frames, total   the batch, as for cluster_frames.
 *   roi_xy        host in, int32[n_vertices][2], vertices in 1/16 px with
 *                 |coordinate| <= 2^24, in either orientation; the last
 *                 vertex joins the first.  Copied during the call.
 *   n_vertices    3 .. 64.
 *   counts        device out, int32[n_frames]: kept birds per frame.
 *   out_xy        device out, int32[total][2] capacity: the kept birds, frame
 *                 after frame (the first out_offsets[n_frames] rows written).
 *   out_offsets   device out, int32[n_frames + 1]: CSR offsets of out_xy.
 *   out_index     device out, int32[total] capacity, or NULL: the input index
 *                 of each kept bird.
 *   workspace     as for cluster_frames, sized by roi_filter_frames_workspace.
 * Offsets must describe the batch (checked only with FLOCK_VALIDATE); with
 * invalid offsets the outputs are unspecified but every access stays in
 * bounds.
 */
flock_status roi_filter_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t total,
                               const int32_t *roi_xy, int32_t n_vertices, int32_t *counts, int32_t *out_xy,
                               int32_t *out_offsets, int32_t *out_index, void *workspace,
                               size_t workspace_bytes, void *stream);

/* Bytes of workspace roi_filter_frames needs for this batch (a flag per bird,
 * a count and a base per block of 2048 birds, and 12 bytes per bird, rounded
 * up to whole blocks, where each block stages its kept birds). */
size_t roi_filter_frames_workspace(int32_t n_frames, int32_t total);

/*
 * drinker_proximity_frames - birds near drinker lines, and per-frame counts.
 *
 * The drinker pipeline computes each bird's distance to the nearest drinker
 * line and classifies the bird as drinking when the distance falls below a
 * threshold (Section 2.3).  Drinker lines are closed segments; the distance
 * is from the bird's point to the nearest point of a segment (end points
 * included); a bird drinks when that distance is strictly below
 * threshold_q for some segment.  The test is exact in integers.
 *
 * Arguments:
 *   xy, offsets, n_frames, total   the batch, as for cluster_frames
 *                    (coordinates 0 <= x, y < 2^24).
 *   lines            host in, int32[n_lines][4] = (ax, ay, bx, by) in 1/16 px,
 *                    |coordinate| <= 2^24.  Copied during the call.
 *   n_lines          1 .. 64.
 *   threshold_q      distance threshold in 1/16 px, 0 .. 2^24.
 *   drinking         device out, uint8[total] (16-byte aligned): 1 if drinking.
 *   line             device out, int32[total], or NULL: the smallest index of
 *                    a segment strictly within the threshold, -1 if none.
 *   counts           device out, int32[n_frames]: drinking birds per frame.
 *   workspace        as for cluster_frames, sized by
 *                    drinker_proximity_frames_workspace.
 */
flock_status drinker_proximity_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames,
                                      int32_t total, const int32_t *lines, int32_t n_lines,
                                      int32_t threshold_q, uint8_t *drinking, int32_t *line,
                                      int32_t *counts, void *workspace, size_t workspace_bytes,
                                      void *stream);

/* Bytes of workspace drinker_proximity_frames needs for this batch. */
size_t drinker_proximity_frames_workspace(int32_t n_frames, int32_t total);

/*
 * mask_components_frames - detection post-processing of a batch of
 * segmentation outputs.
 *
 * Section 3.2 turns the segmentation network's output into detections with
 * a connected-components-with-statistics routine (threshold, connected
 * components, bounding boxes; Section 2.3 gives each box a confidence
 * score).  Per frame f and pixel p = y * width + x:
 *   foreground   prob[f][p] > threshold (NaN is background);
 *   labels       connected foreground pixels under the 4-neighbourhood
 *                (shared edge) or the 8-neighbourhood (shared edge or corner)
 *                form a component, labelled by its first pixel in raster
 *                order (smallest p); background gets -1;
 *   components   listed frame after frame, in label order within a frame:
 *                label, area (pixels), box (x, y, width, height), centroid
 *                (mean x, mean y of the pixel indices, correctly rounded
 *                quotient of exact integer sums), xy = floor(16 sum / area)
 *                per axis (the centroid in the 1/16-px layout of
 *                cluster_frames, with comp_offsets as its offsets), and score
 *                (largest probability among the component's pixels).
 *
 * Arguments:
 *   prob            device in, float[n_frames][height][width].
 *   width, height   1 .. 32768 each; n_frames * width * height < 2^31.
 *   threshold       finite and >= 0.
 *   connectivity    4 or 8.
 *   labels          device out, int32[n_frames][height][width], or NULL.
 *   n_components    device out, int32[n_frames].
 *   comp_offsets    device out, int32[n_frames + 1]: CSR offsets of the
 *                   component list; comp_offsets[n_frames] is the count K.
 *   capacity        rows of the component outputs; components with rank
 *                   >= capacity are counted but not written.
 *   comp_label, comp_area   device out, int32[capacity], or NULL.
 *   comp_box        device out, int32[capacity][4], 16-byte aligned, or NULL.
 *   comp_centroid   device out, double[capacity][2], 16-byte aligned, or NULL.
 *   comp_xy         device out, int32[capacity][2], 8-byte aligned, or NULL.
 *   comp_score      device out, float[capacity], or NULL.
 *   workspace       as for cluster_frames, sized by
 *                   mask_components_frames_workspace.
 * Every output is deterministic: statistics are integer sums, minima and
 * maxima, so their order of accumulation does not matter.
 */
flock_status mask_components_frames(const float *prob, int32_t n_frames, int32_t width, int32_t height,
                                    float threshold, int32_t connectivity, int32_t *labels,
                                    int32_t *n_components, int32_t *comp_offsets, int32_t capacity,
                                    int32_t *comp_label, int32_t *comp_area, int32_t *comp_box,
                                    double *comp_centroid, int32_t *comp_xy, float *comp_score,
                                    void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of workspace mask_components_frames needs for this batch shape: 56
 * bytes per possible piece of a component inside a 64 x 64 tile (a quarter
 * of the pixels with 8 neighbours, half with 4), plus the tile seams and a
 * bit per pixel. */
size_t mask_components_frames_workspace(int32_t n_frames, int32_t width, int32_t height, int32_t connectivity);

/* Text of the last error on this thread ("" if none); valid until the next
 * library call on this thread. */
const char *flock_last_error(void);

/* Library version string, e.g. "flock 0.1.0 gfx950". */
const char *flock_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FLOCK_H */

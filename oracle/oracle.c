/*
 * oracle.c - plain, slow, obviously correct CPU oracle for the per-frame
 * clustering and density-grid path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  The GPU library shares no
 * code, header, table or constant with it.
 *
 * What it computes (the paper's clustering module, Section 2.3, and its
 * per-frame density computation, Section 3.6 / Algorithm 1):
 *
 *  1. Radius-neighbour clustering of the birds of each frame.  The paper's
 *     clustering module finds groups of nearby birds by connected-component
 *     analysis (Section 2.3); the point-level reading used here is standard
 *     DBSCAN (Ester, Kriegel, Sander and Xu, KDD 1996):
 *       - two birds are neighbours when their Euclidean distance is <= eps
 *         (closed ball; a bird is its own neighbour, duplicates count);
 *       - a bird is a core point when it has >= min_pts neighbours;
 *       - clusters are the connected components of the core points under the
 *         neighbour relation, found by breadth-first expansion from each
 *         unvisited core point in ascending index order, so a cluster's label
 *         is the smallest frame-local index among its core points;
 *       - a non-core bird with at least one core neighbour is a border point
 *         and joins the cluster of its nearest core neighbour, ties broken by
 *         the smaller (y, x) of that core; any other bird is noise (-1).
 *     Coordinates are integers in 1/16 px and eps_q = 16 * eps, so the
 *     neighbour test is the exact integer comparison dx^2 + dy^2 <= eps_q^2
 *     (done in int64).
 *
 *  2. The Gaussian density grid of each frame (Algorithm 1, DefaultClustering:
 *     for every grid cell, for every bird, accumulate a distance-based
 *     contribution).  The grid has grid_w x grid_h cells tiling the frame
 *     [0, W) x [0, H) px, evaluated at cell centres
 *         cx = (gx + 1/2) W / grid_w,   cy = (gy + 1/2) H / grid_h,
 *     and each bird at (x, y) = (x_q / 16, y_q / 16) px contributes the
 *     isotropic 2-D Gaussian with bandwidth sigma px, normalised to unit mass:
 *         density[gy][gx] = sum_i exp(-((cx - x)^2 + (cy - y)^2) / (2 sigma^2))
 *                           / (2 pi sigma^2)            [birds per px^2]
 *     This is the direct double sum in fp64 with libm exp, one grid cell at a
 *     time; it makes no use of the sum's separability.
 *
 *  3. Heatmap analytics of each frame's density grid (the clustering module
 *     of Section 2.3 thresholds the density heatmaps and applies connected
 *     component analysis; Algorithm 1 then computes the heatmap, its entropy
 *     and a clustering degree).  Readings, since the paper fixes none of the
 *     details:
 *       - the heatmap is the density grid D itself, normalised to
 *         p = D / S with S = sum of the positive cells (cells with D <= 0
 *         carry no mass);
 *       - a cell is hot when D >= threshold (threshold > 0, in birds/px^2);
 *       - clusters are the connected components of the hot cells under
 *         4-neighbourhood (shared edge) or 8-neighbourhood (shared edge or
 *         corner), found by breadth-first expansion from each unvisited hot
 *         cell in ascending row-major index, so a component's label is its
 *         smallest frame-local index gy * grid_w + gx; cold cells get -1;
 *       - per component: its cell count and its mass, cell_area times the sum
 *         of D over its cells (expected birds), stored at the label cell;
 *       - entropy H = -sum over positive cells of p ln p (natural log), 0 for
 *         a frame with S = 0;
 *       - clustering degree = (sum of D over hot cells) / S, the share of the
 *         frame's density mass that lies in clusters (0 when S = 0).
 *     All sums are fp64 in row-major order.
 *
 *  4. Region-of-interest filtering and per-frame region counts (the wall
 *     pipeline counts the birds in a region near the wall, Section 2.2;
 *     Algorithm 1 filters the birds to the ROI).  Reading: the ROI is a
 *     polygon with integer vertices in quanta; a bird is inside when its
 *     point lies in the closed polygon, boundary included, under the
 *     even-odd rule (for a simple polygon: its interior plus its edges).
 *     Kept birds keep their input order; per frame the count of kept birds.
 *     The test is exact integer arithmetic (int64 products of coordinates
 *     below 2^24).
 *
 *  5. Drinker-line proximity (the drinker pipeline measures each bird's
 *     distance to the nearest drinker line and classifies the bird as
 *     drinking when that distance falls below a threshold, Section 2.3).
 *     Reading: drinker lines are segments with integer end points in quanta;
 *     the distance is the Euclidean distance from the bird's point to the
 *     closed segment (its nearest point, end points included); a bird drinks
 *     when the distance to some segment is strictly below the threshold T
 *     (quanta).  Per bird: the flag and the smallest index of such a segment
 *     (-1 if none); per frame: the number of drinking birds.  The comparison
 *     is exact: squared distances to end points in int64, and for a point
 *     projecting inside the segment cross^2 < T^2 |b - a|^2 in 128 bits.
 *
 *  6. Detection post-processing (Section 3.2: the segmentation output is
 *     thresholded and grouped into connected regions with their statistics,
 *     replacing skimage.regionprops by OpenCV's connectedComponentsWithStats).
 *     Reading: a pixel is foreground when its probability is strictly above
 *     the threshold; components are connected foreground pixels under the
 *     4- or 8-neighbourhood, labelled by their first pixel in raster order
 *     (smallest index y * W + x), background -1; components are listed per
 *     frame in label order with area (pixels), bounding box (x, y, width,
 *     height) and centroid (mean x, mean y of the pixel indices, as the
 *     OpenCV routine reports it), the centroid in 1/16 px rounded down (the
 *     position layout of the clustering input), and a confidence score, the
 *     largest probability among the component's pixels (Section 2.3 gives
 *     boxes confidence scores without saying how; this is a reading).  The
 *     threshold is finite and >= 0 (the output is a probability).
 *
 * Threads only split independent work items (whole frames for clustering
 * and heatmaps, whole grid rows for density); each item is computed exactly
 * as above.
 */

#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ENOMEM (-2)

/* ------------------------------------------------------------------------ */
/* Clustering of one frame                                                  */
/* ------------------------------------------------------------------------ */

static int64_t sq_dist(const int32_t *xy, int32_t i, int32_t j)
{
    int64_t dx = (int64_t)xy[2 * i] - (int64_t)xy[2 * j];
    int64_t dy = (int64_t)xy[2 * i + 1] - (int64_t)xy[2 * j + 1];
    return dx * dx + dy * dy;
}

/* Returns the number of clusters (>= 0), or a negative error code.
 * labels[i]: frame-local label (smallest core index of the cluster) or -1.
 * kind[i]:   0 noise, 1 border, 2 core. */
int32_t oracle_dbscan_frame(const int32_t *xy, int32_t n, int32_t eps_q, int32_t min_pts,
                            int32_t *labels, uint8_t *kind)
{
    if (n < 0 || eps_q < 0 || min_pts < 1) return ORACLE_EINVAL;
    if (n == 0) return 0;
    const int64_t e2 = (int64_t)eps_q * (int64_t)eps_q;

    int64_t *count = (int64_t *)calloc((size_t)n, sizeof(int64_t));
    uint8_t *core = (uint8_t *)calloc((size_t)n, 1);
    int32_t *comp = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    int32_t *queue = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    if (!count || !core || !comp || !queue) {
        free(count); free(core); free(comp); free(queue);
        return ORACLE_ENOMEM;
    }

    /* Neighbour counts (self and duplicates included) and core flags. */
    for (int32_t i = 0; i < n; ++i) {
        int64_t c = 0;
        for (int32_t j = 0; j < n; ++j)
            if (sq_dist(xy, i, j) <= e2) ++c;
        count[i] = c;
        core[i] = (uint8_t)(c >= (int64_t)min_pts);
    }

    /* Clusters: breadth-first expansion over core points, seeds ascending. */
    for (int32_t i = 0; i < n; ++i) comp[i] = -1;
    int32_t n_clusters = 0;
    for (int32_t s = 0; s < n; ++s) {
        if (!core[s] || comp[s] >= 0) continue;
        ++n_clusters;
        int32_t head = 0, tail = 0;
        comp[s] = s;
        queue[tail++] = s;
        while (head < tail) {
            int32_t p = queue[head++];
            for (int32_t j = 0; j < n; ++j) {
                if (core[j] && comp[j] < 0 && sq_dist(xy, p, j) <= e2) {
                    comp[j] = s;
                    queue[tail++] = j;
                }
            }
        }
    }

    /* Cores keep their component; non-cores take the nearest core neighbour's
     * component (key: squared distance, then y, then x of the core). */
    for (int32_t i = 0; i < n; ++i) {
        if (core[i]) {
            labels[i] = comp[i];
            kind[i] = 2;
            continue;
        }
        int32_t best = -1;
        int64_t best_d2 = 0;
        for (int32_t j = 0; j < n; ++j) {
            if (!core[j]) continue;
            int64_t d2 = sq_dist(xy, i, j);
            if (d2 > e2) continue;
            int better = 0;
            if (best < 0) better = 1;
            else if (d2 != best_d2) better = d2 < best_d2;
            else if (xy[2 * j + 1] != xy[2 * best + 1]) better = xy[2 * j + 1] < xy[2 * best + 1];
            else better = xy[2 * j] < xy[2 * best];
            if (better) { best = j; best_d2 = d2; }
        }
        if (best >= 0) {
            labels[i] = comp[best];
            kind[i] = 1;
        } else {
            labels[i] = -1;
            kind[i] = 0;
        }
    }

    free(count); free(core); free(comp); free(queue);
    return n_clusters;
}

/* Neighbour counts alone (self included), for tests of the count step. */
int32_t oracle_neighbour_counts(const int32_t *xy, int32_t n, int32_t eps_q, int32_t *count)
{
    if (n < 0 || eps_q < 0) return ORACLE_EINVAL;
    const int64_t e2 = (int64_t)eps_q * (int64_t)eps_q;
    for (int32_t i = 0; i < n; ++i) {
        int32_t c = 0;
        for (int32_t j = 0; j < n; ++j)
            if (sq_dist(xy, i, j) <= e2) ++c;
        count[i] = c;
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Density of one grid cell / one frame                                     */
/* ------------------------------------------------------------------------ */

static const double kPi = 3.14159265358979323846;

double oracle_density_cell(const int32_t *xy, int32_t n, int32_t width_px, int32_t height_px,
                           int32_t grid_w, int32_t grid_h, double sigma_px, int32_t gx, int32_t gy)
{
    const double cx = ((double)gx + 0.5) * (double)width_px / (double)grid_w;
    const double cy = ((double)gy + 0.5) * (double)height_px / (double)grid_h;
    const double two_s2 = 2.0 * sigma_px * sigma_px;
    double acc = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        const double x = (double)xy[2 * i] / 16.0;
        const double y = (double)xy[2 * i + 1] / 16.0;
        const double dx = cx - x, dy = cy - y;
        acc += exp(-(dx * dx + dy * dy) / two_s2);
    }
    return acc / (kPi * two_s2);
}

static int density_args_ok(int32_t width_px, int32_t height_px, int32_t grid_w, int32_t grid_h,
                           double sigma_px)
{
    return width_px >= 1 && height_px >= 1 && grid_w >= 1 && grid_h >= 1 &&
           isfinite(sigma_px) && sigma_px > 0.0;
}

/* ------------------------------------------------------------------------ */
/* Batches: a thread pool over independent work items                       */
/* ------------------------------------------------------------------------ */

typedef struct {
    /* batch */
    const int32_t *xy;
    const int32_t *offsets;
    int32_t n_frames;
    /* clustering */
    int32_t eps_q, min_pts;
    int32_t *labels;
    uint8_t *kind;
    int32_t *n_clusters;
    /* density */
    int32_t width_px, height_px, grid_w, grid_h;
    double sigma_px;
    double *density;
    const int32_t *cell_frame, *cell_gx, *cell_gy;
    /* work distribution */
    int64_t n_items;
    int64_t next;          /* shared counter */
    int32_t status;        /* first error seen */
    int mode;              /* 0 cluster, 1 density grid, 2 density cells */
} job_t;

static void run_item(job_t *job, int64_t item)
{
    if (job->mode == 0) {
        int32_t f = (int32_t)item;
        int32_t b = job->offsets[f], e = job->offsets[f + 1];
        int32_t r = oracle_dbscan_frame(job->xy + 2 * (int64_t)b, e - b, job->eps_q, job->min_pts,
                                        job->labels + b, job->kind + b);
        if (r < 0) __atomic_store_n(&job->status, r, __ATOMIC_RELAXED);
        else if (job->n_clusters) job->n_clusters[f] = r;
    } else if (job->mode == 1) {
        int32_t f = (int32_t)(item / job->grid_h);
        int32_t gy = (int32_t)(item % job->grid_h);
        int32_t b = job->offsets[f], e = job->offsets[f + 1];
        double *row = job->density + ((int64_t)f * job->grid_h + gy) * job->grid_w;
        for (int32_t gx = 0; gx < job->grid_w; ++gx)
            row[gx] = oracle_density_cell(job->xy + 2 * (int64_t)b, e - b, job->width_px,
                                          job->height_px, job->grid_w, job->grid_h, job->sigma_px,
                                          gx, gy);
    } else {
        int32_t f = job->cell_frame[item];
        int32_t b = job->offsets[f], e = job->offsets[f + 1];
        job->density[item] = oracle_density_cell(job->xy + 2 * (int64_t)b, e - b, job->width_px,
                                                  job->height_px, job->grid_w, job->grid_h,
                                                  job->sigma_px, job->cell_gx[item],
                                                  job->cell_gy[item]);
    }
}

static void *worker(void *arg)
{
    job_t *job = (job_t *)arg;
    for (;;) {
        int64_t item = __atomic_fetch_add(&job->next, 1, __ATOMIC_RELAXED);
        if (item >= job->n_items) break;
        run_item(job, item);
    }
    return NULL;
}

static int32_t run_job(job_t *job, int32_t n_threads)
{
    if (n_threads < 1) n_threads = 1;
    if ((int64_t)n_threads > job->n_items) n_threads = (int32_t)(job->n_items > 0 ? job->n_items : 1);
    job->next = 0;
    job->status = ORACLE_OK;
    if (n_threads == 1) {
        worker(job);
        return job->status;
    }
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)n_threads);
    if (!th) return ORACLE_ENOMEM;
    int32_t started = 0;
    for (; started < n_threads; ++started)
        if (pthread_create(&th[started], NULL, worker, job) != 0) break;
    if (started == 0) worker(job);
    for (int32_t t = 0; t < started; ++t) pthread_join(th[t], NULL);
    free(th);
    return job->status;
}

static int offsets_ok(const int32_t *offsets, int32_t n_frames)
{
    if (n_frames < 0 || (n_frames > 0 && !offsets)) return 0;
    if (n_frames > 0 && offsets[0] != 0) return 0;
    for (int32_t f = 0; f < n_frames; ++f)
        if (offsets[f + 1] < offsets[f]) return 0;
    return 1;
}

int32_t oracle_cluster_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames,
                              int32_t eps_q, int32_t min_pts, int32_t *labels, uint8_t *kind,
                              int32_t *n_clusters, int32_t n_threads)
{
    if (!offsets_ok(offsets, n_frames) || eps_q < 0 || min_pts < 1) return ORACLE_EINVAL;
    job_t job;
    memset(&job, 0, sizeof job);
    job.xy = xy; job.offsets = offsets; job.n_frames = n_frames;
    job.eps_q = eps_q; job.min_pts = min_pts;
    job.labels = labels; job.kind = kind; job.n_clusters = n_clusters;
    job.n_items = n_frames;
    job.mode = 0;
    return run_job(&job, n_threads);
}

/* density: [n_frames][grid_h][grid_w] fp64 */
int32_t oracle_density_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames,
                              int32_t width_px, int32_t height_px, int32_t grid_w, int32_t grid_h,
                              double sigma_px, double *density, int32_t n_threads)
{
    if (!offsets_ok(offsets, n_frames) ||
        !density_args_ok(width_px, height_px, grid_w, grid_h, sigma_px))
        return ORACLE_EINVAL;
    job_t job;
    memset(&job, 0, sizeof job);
    job.xy = xy; job.offsets = offsets; job.n_frames = n_frames;
    job.width_px = width_px; job.height_px = height_px;
    job.grid_w = grid_w; job.grid_h = grid_h; job.sigma_px = sigma_px;
    job.density = density;
    job.n_items = (int64_t)n_frames * grid_h;
    job.mode = 1;
    return run_job(&job, n_threads);
}

/* Density at m sampled cells: cell k is (frame[k], gx[k], gy[k]); out[k] fp64. */
int32_t oracle_density_cells(const int32_t *xy, const int32_t *offsets, int32_t n_frames,
                             int32_t width_px, int32_t height_px, int32_t grid_w, int32_t grid_h,
                             double sigma_px, const int32_t *cell_frame, const int32_t *cell_gx,
                             const int32_t *cell_gy, int64_t m, double *out, int32_t n_threads)
{
    if (!offsets_ok(offsets, n_frames) ||
        !density_args_ok(width_px, height_px, grid_w, grid_h, sigma_px) || m < 0)
        return ORACLE_EINVAL;
    for (int64_t k = 0; k < m; ++k)
        if (cell_frame[k] < 0 || cell_frame[k] >= n_frames || cell_gx[k] < 0 ||
            cell_gx[k] >= grid_w || cell_gy[k] < 0 || cell_gy[k] >= grid_h)
            return ORACLE_EINVAL;
    job_t job;
    memset(&job, 0, sizeof job);
    job.xy = xy; job.offsets = offsets; job.n_frames = n_frames;
    job.width_px = width_px; job.height_px = height_px;
    job.grid_w = grid_w; job.grid_h = grid_h; job.sigma_px = sigma_px;
    job.density = out;
    job.cell_frame = cell_frame; job.cell_gx = cell_gx; job.cell_gy = cell_gy;
    job.n_items = m;
    job.mode = 2;
    return run_job(&job, n_threads);
}

/* ------------------------------------------------------------------------ */
/* Heatmap analytics of one frame                                           */
/* ------------------------------------------------------------------------ */

/* density: [grid_h][grid_w] fp32; labels, comp_cells: [grid_h][grid_w];
 * comp_mass: [grid_h][grid_w] fp64; returns the number of components. */
int32_t oracle_heatmap_frame(const float *density, int32_t grid_w, int32_t grid_h, double cell_area,
                             float threshold, int32_t connectivity, int32_t *labels,
                             int32_t *comp_cells, double *comp_mass, double *entropy,
                             double *degree)
{
    if (grid_w < 1 || grid_h < 1 || !(threshold > 0.0f) || (connectivity != 4 && connectivity != 8))
        return ORACLE_EINVAL;
    const int64_t cells = (int64_t)grid_w * grid_h;
    int64_t *queue = (int64_t *)malloc((size_t)cells * sizeof(int64_t));
    if (!queue) return ORACLE_ENOMEM;
    for (int64_t c = 0; c < cells; ++c) {
        labels[c] = -1;
        comp_cells[c] = 0;
        comp_mass[c] = 0.0;
    }
    int32_t n_comp = 0;
    for (int64_t seed = 0; seed < cells; ++seed) {
        if (!(density[seed] >= threshold) || labels[seed] >= 0) continue;
        /* breadth-first expansion over hot neighbours */
        int64_t head = 0, tail = 0;
        queue[tail++] = seed;
        labels[seed] = (int32_t)seed;
        while (head < tail) {
            const int64_t c = queue[head++];
            const int32_t gx = (int32_t)(c % grid_w), gy = (int32_t)(c / grid_w);
            for (int32_t dy = -1; dy <= 1; ++dy)
                for (int32_t dx = -1; dx <= 1; ++dx) {
                    if (dx == 0 && dy == 0) continue;
                    if (connectivity == 4 && dx != 0 && dy != 0) continue;
                    const int32_t nx = gx + dx, ny = gy + dy;
                    if (nx < 0 || nx >= grid_w || ny < 0 || ny >= grid_h) continue;
                    const int64_t nc = (int64_t)ny * grid_w + nx;
                    if (density[nc] >= threshold && labels[nc] < 0) {
                        labels[nc] = (int32_t)seed;
                        queue[tail++] = nc;
                    }
                }
        }
        ++n_comp;
    }
    free(queue);
    /* per-component cells and mass, at the label cell */
    for (int64_t c = 0; c < cells; ++c) {
        if (labels[c] < 0) continue;
        comp_cells[labels[c]] += 1;
        comp_mass[labels[c]] += (double)density[c];
    }
    for (int64_t c = 0; c < cells; ++c) comp_mass[c] *= cell_area;
    /* entropy of p = D / S and the hot share of S */
    double S = 0.0, hot = 0.0;
    for (int64_t c = 0; c < cells; ++c) {
        if (density[c] > 0.0f) S += (double)density[c];
        if (labels[c] >= 0) hot += (double)density[c];
    }
    double H = 0.0;
    if (S > 0.0) {
        for (int64_t c = 0; c < cells; ++c) {
            if (!(density[c] > 0.0f)) continue;
            const double pc = (double)density[c] / S;
            H -= pc * log(pc);
        }
    }
    *entropy = H;
    *degree = S > 0.0 ? hot / S : 0.0;
    return n_comp;
}

/* Batch of n_frames grids, frames split over threads. */
typedef struct {
    const float *density;
    int32_t n_frames, grid_w, grid_h, connectivity;
    double cell_area;
    float threshold;
    int32_t *labels, *n_components, *comp_cells;
    double *comp_mass, *entropy, *degree;
    int32_t next, rc;
    pthread_mutex_t mu;
} heat_job_t;

static void *heat_worker(void *arg)
{
    heat_job_t *job = (heat_job_t *)arg;
    const int64_t cells = (int64_t)job->grid_w * job->grid_h;
    for (;;) {
        pthread_mutex_lock(&job->mu);
        const int32_t f = job->next++;
        pthread_mutex_unlock(&job->mu);
        if (f >= job->n_frames) break;
        const int32_t r = oracle_heatmap_frame(job->density + f * cells, job->grid_w, job->grid_h,
                                               job->cell_area, job->threshold, job->connectivity,
                                               job->labels + f * cells, job->comp_cells + f * cells,
                                               job->comp_mass + f * cells, job->entropy + f,
                                               job->degree + f);
        pthread_mutex_lock(&job->mu);
        if (r < 0) job->rc = r;
        else job->n_components[f] = r;
        pthread_mutex_unlock(&job->mu);
    }
    return NULL;
}

int32_t oracle_heatmap_frames(const float *density, int32_t n_frames, int32_t grid_w, int32_t grid_h,
                              double cell_area, float threshold, int32_t connectivity,
                              int32_t *labels, int32_t *n_components, double *entropy,
                              double *degree, int32_t *comp_cells, double *comp_mass,
                              int32_t n_threads)
{
    if (n_frames < 0 || grid_w < 1 || grid_h < 1 || !(threshold > 0.0f) ||
        (connectivity != 4 && connectivity != 8))
        return ORACLE_EINVAL;
    heat_job_t job;
    memset(&job, 0, sizeof job);
    job.density = density; job.n_frames = n_frames; job.grid_w = grid_w; job.grid_h = grid_h;
    job.connectivity = connectivity; job.cell_area = cell_area; job.threshold = threshold;
    job.labels = labels; job.n_components = n_components; job.comp_cells = comp_cells;
    job.comp_mass = comp_mass; job.entropy = entropy; job.degree = degree;
    pthread_mutex_init(&job.mu, NULL);
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 64) n_threads = 64;
    pthread_t th[64];
    int32_t started = 0;
    for (int32_t t = 0; t < n_threads; ++t)
        if (pthread_create(&th[t], NULL, heat_worker, &job) == 0) ++started;
    if (started == 0) heat_worker(&job);
    for (int32_t t = 0; t < started; ++t) pthread_join(th[t], NULL);
    pthread_mutex_destroy(&job.mu);
    return job.rc;
}

/* ------------------------------------------------------------------------ */
/* Region of interest                                                       */
/* ------------------------------------------------------------------------ */

/* Point (px, py) on the closed segment from (ax, ay) to (bx, by). */
static int on_segment(int64_t px, int64_t py, int64_t ax, int64_t ay, int64_t bx, int64_t by)
{
    const int64_t cross = (bx - ax) * (py - ay) - (by - ay) * (px - ax);
    if (cross != 0) return 0;
    const int64_t lo_x = ax < bx ? ax : bx, hi_x = ax < bx ? bx : ax;
    const int64_t lo_y = ay < by ? ay : by, hi_y = ay < by ? by : ay;
    return px >= lo_x && px <= hi_x && py >= lo_y && py <= hi_y;
}

/* 1 if (px, py) lies in the closed polygon (even-odd rule), else 0.
 * poly: n vertices (x, y); the last vertex joins the first. */
int32_t oracle_point_in_polygon(const int32_t *poly, int32_t n, int32_t px, int32_t py)
{
    int inside = 0;
    for (int32_t i = 0; i < n; ++i) {
        const int32_t j = (i + 1) % n;
        const int64_t ax = poly[2 * i], ay = poly[2 * i + 1];
        const int64_t bx = poly[2 * j], by = poly[2 * j + 1];
        if (on_segment(px, py, ax, ay, bx, by)) return 1;
        /* does the edge cross the ray from (px, py) towards +x?  An edge
         * counts when exactly one end lies strictly above the ray's line
         * (so a vertex on the line is counted once), and the crossing point
         * lies to the right of px:
         *     px < ax + (py - ay) (bx - ax) / (by - ay)                     */
        if ((ay > py) != (by > py)) {
            const int64_t lhs = (int64_t)(px - ax) * (by - ay);
            const int64_t rhs = (int64_t)(py - ay) * (bx - ax);
            const int right = (by > ay) ? (lhs < rhs) : (lhs > rhs);
            if (right) inside = !inside;
        }
    }
    return inside;
}

/* Batch: keep[i] = 1 for birds inside the ROI; counts[f] = kept birds of
 * frame f; kept birds are also written in order to out_xy / out_index with
 * CSR out_offsets[F + 1]. */
int32_t oracle_roi_filter(const int32_t *xy, const int32_t *offsets, int32_t n_frames,
                          const int32_t *poly, int32_t n_vertices, int32_t *counts,
                          int32_t *out_xy, int32_t *out_offsets, int32_t *out_index)
{
    if (!offsets_ok(offsets, n_frames) || n_vertices < 3 || !poly) return ORACLE_EINVAL;
    int32_t k = 0;
    if (n_frames >= 0) out_offsets[0] = 0;
    for (int32_t f = 0; f < n_frames; ++f) {
        int32_t c = 0;
        for (int32_t i = offsets[f]; i < offsets[f + 1]; ++i) {
            if (!oracle_point_in_polygon(poly, n_vertices, xy[2 * i], xy[2 * i + 1])) continue;
            out_xy[2 * k] = xy[2 * i];
            out_xy[2 * k + 1] = xy[2 * i + 1];
            out_index[k] = i;
            ++k;
            ++c;
        }
        counts[f] = c;
        out_offsets[f + 1] = k;
    }
    return k;
}

/* ------------------------------------------------------------------------ */
/* Drinker-line proximity                                                   */
/* ------------------------------------------------------------------------ */

/* 1 if point (px, py) is strictly closer than t to the closed segment
 * (ax, ay)-(bx, by).  Coordinates within 2^24 in magnitude, 0 <= t < 2^24. */
int32_t oracle_near_segment(int32_t px, int32_t py, int32_t ax, int32_t ay, int32_t bx, int32_t by, int32_t t)
{
    const int64_t ux = (int64_t)bx - ax, uy = (int64_t)by - ay;   /* segment direction */
    const int64_t wx = (int64_t)px - ax, wy = (int64_t)py - ay;   /* a -> p */
    const int64_t t2 = (int64_t)t * t;
    const int64_t len2 = ux * ux + uy * uy;
    const int64_t dot = ux * wx + uy * wy;
    if (len2 == 0 || dot <= 0) return wx * wx + wy * wy < t2;      /* nearest point: a */
    if (dot >= len2) {                                              /* nearest point: b */
        const int64_t vx = (int64_t)px - bx, vy = (int64_t)py - by;
        return vx * vx + vy * vy < t2;
    }
    /* nearest point inside the segment: distance^2 = cross^2 / len2 */
    const int64_t cross = ux * wy - uy * wx;
    const unsigned __int128 c2 = (unsigned __int128)(cross < 0 ? -cross : cross) * (unsigned __int128)(cross < 0 ? -cross : cross);
    const unsigned __int128 lim = (unsigned __int128)t2 * (unsigned __int128)len2;
    return c2 < lim;
}

/* lines: n_lines segments (ax, ay, bx, by).  Per bird: drinking flag and the
 * smallest index of a segment within t (-1 if none); per frame: counts. */
int32_t oracle_drinkers(const int32_t *xy, const int32_t *offsets, int32_t n_frames, const int32_t *lines,
                        int32_t n_lines, int32_t t, uint8_t *drinking, int32_t *line, int32_t *counts)
{
    if (!offsets_ok(offsets, n_frames) || n_lines < 1 || !lines || t < 0) return ORACLE_EINVAL;
    for (int32_t f = 0; f < n_frames; ++f) {
        int32_t c = 0;
        for (int32_t i = offsets[f]; i < offsets[f + 1]; ++i) {
            int32_t hit = -1;
            for (int32_t k = 0; k < n_lines && hit < 0; ++k)
                if (oracle_near_segment(xy[2 * i], xy[2 * i + 1], lines[4 * k], lines[4 * k + 1],
                                        lines[4 * k + 2], lines[4 * k + 3], t))
                    hit = k;
            drinking[i] = hit >= 0;
            line[i] = hit;
            c += hit >= 0;
        }
        counts[f] = c;
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Detection post-processing: mask components with statistics              */
/* ------------------------------------------------------------------------ */

/* prob: [n_frames][h][w] fp32.  labels: [n_frames][h][w].  Components of
 * all frames are listed frame after frame: comp_offsets[n_frames + 1];
 * per component (up to capacity; the count is returned): label (frame
 * pixel index), area, box (x, y, width, height), centroid (x, y), the
 * centroid in 1/16 px as floor(16 * sum / area) in integers (the position
 * layout the clustering consumes), and score, the largest probability of
 * its pixels.  threshold must be finite and >= 0. */
int64_t oracle_mask_components(const float *prob, int32_t n_frames, int32_t w, int32_t h, float threshold,
                               int32_t connectivity, int32_t *labels, int32_t *n_components,
                               int64_t *comp_offsets, int64_t capacity, int32_t *comp_label,
                               int32_t *comp_area, int32_t *comp_box, double *comp_centroid, int32_t *comp_xy,
                               float *comp_score)
{
    if (n_frames < 0 || w < 1 || h < 1 || (connectivity != 4 && connectivity != 8)) return ORACLE_EINVAL;
    if (!(threshold >= 0.0f) || isinf(threshold)) return ORACLE_EINVAL;
    const int64_t px = (int64_t)w * h;
    int64_t *queue = (int64_t *)malloc((size_t)px * sizeof(int64_t));
    if (!queue) return ORACLE_ENOMEM;
    int64_t k = 0;
    comp_offsets[0] = 0;
    for (int32_t f = 0; f < n_frames; ++f) {
        const float *P = prob + f * px;
        int32_t *L = labels + f * px;
        for (int64_t c = 0; c < px; ++c) L[c] = -1;
        int32_t nc = 0;
        /* seeds in raster order: each component is found first at its
         * smallest pixel index, which becomes its label */
        for (int64_t seed = 0; seed < px; ++seed) {
            if (!(P[seed] > threshold) || L[seed] >= 0) continue;
            int64_t head = 0, tail = 0, area = 0, sx = 0, sy = 0;
            int32_t x0 = w, y0 = h, x1 = -1, y1 = -1;
            float best = P[seed];
            queue[tail++] = seed;
            L[seed] = (int32_t)seed;
            while (head < tail) {
                const int64_t c = queue[head++];
                const int32_t cx = (int32_t)(c % w), cy = (int32_t)(c / w);
                ++area;
                sx += cx;
                sy += cy;
                if (cx < x0) x0 = cx;
                if (cx > x1) x1 = cx;
                if (cy < y0) y0 = cy;
                if (cy > y1) y1 = cy;
                if (P[c] > best) best = P[c];
                for (int32_t dy = -1; dy <= 1; ++dy)
                    for (int32_t dx = -1; dx <= 1; ++dx) {
                        if (dx == 0 && dy == 0) continue;
                        if (connectivity == 4 && dx * dy != 0) continue;
                        const int32_t nx = cx + dx, ny = cy + dy;
                        if (nx < 0 || nx >= w || ny < 0 || ny >= h) continue;
                        const int64_t n = (int64_t)ny * w + nx;
                        if (P[n] > threshold && L[n] < 0) {
                            L[n] = (int32_t)seed;
                            queue[tail++] = n;
                        }
                    }
            }
            if (k < capacity) {
                comp_label[k] = (int32_t)seed;
                comp_area[k] = (int32_t)area;
                comp_box[4 * k] = x0;
                comp_box[4 * k + 1] = y0;
                comp_box[4 * k + 2] = x1 - x0 + 1;
                comp_box[4 * k + 3] = y1 - y0 + 1;
                comp_centroid[2 * k] = (double)sx / (double)area;
                comp_centroid[2 * k + 1] = (double)sy / (double)area;
                comp_xy[2 * k] = (int32_t)((16 * sx) / area);
                comp_xy[2 * k + 1] = (int32_t)((16 * sy) / area);
                comp_score[k] = best;
            }
            ++k;
            ++nc;
        }
        n_components[f] = nc;
        comp_offsets[f + 1] = k;
    }
    free(queue);
    return k;
}

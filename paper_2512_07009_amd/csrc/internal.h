// internal.h - declarations shared by the library's own translation units
// (host API and kernel launchers).  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace flock {

// ----------------------------------------------------------------------------
// Clustering
// ----------------------------------------------------------------------------
struct ClusterArgs {
    const int32_t *xy;        // [total][2] 1/16 px
    const int32_t *offsets;   // [n_frames + 1]
    int32_t n_frames;
    int32_t total;
    int32_t eps_q;            // radius in quanta
    int32_t min_pts;
    int32_t cell_side;        // largest s >= 1 with 2 s^2 <= eps_q^2
    int32_t cap_points;       // frames with more points leave the on-chip kernel
    int32_t cap_cells;        // cell-table entries available on chip
    int32_t big_path;         // 1: frames above cap_points go to the multi-workgroup
                              // path; 0: the on-chip kernel clusters them in place
    int32_t big_all;          // 1: the multi-workgroup path takes every frame and also
                              // writes the counts of empty and inconsistent frames
                              // (the on-chip kernel is not launched)
    int32_t union_regs;       // 1: the on-chip unions keep up to 3072 core cells'
                              // edges in registers; 0: always re-read them from LDS
    // Neighbour-cell tables for cells of side cell_side (as the on-chip
    // kernel's build_stencil makes them), packed 6 bits per cell offset
    // ((dx + 2) | (dy + 2) << 3), five per word:
    uint32_t sten_all[5];     // the whole stencil, nearest cells first
    uint32_t sten_fwd[3];     // its forward half, adjacent cells first
    uint32_t sten_meta;       // nsten | nadj << 8 | nfwd << 16 | dxmax[k] << (24 + 2 k)
    int32_t *labels;          // [total]
    uint8_t *kind;            // [total]
    int32_t *n_clusters;      // [n_frames] or nullptr
};

// Bytes of dynamic LDS the resident clustering kernel needs for these caps.
size_t cluster_lds_bytes(int32_t cap_points, int32_t cap_cells);
// Largest point capacity that fits the device's LDS with a cell table of
// at least min_cells entries.
int32_t cluster_max_cap_points(size_t lds_limit);

// Static shared memory of the compact clustering kernel (bytes).
size_t cluster_compact_static_lds();
// Largest frame the compact kernel holds (points per thread x threads).
constexpr int32_t kClusterCompactCap = 5120;
// compact: the two-workgroups-per-compute-unit kernel (frames of at most
// kClusterCompactCap points, lds_bytes at most half a compute unit's LDS
// less its static shared memory).
hipError_t launch_cluster_resident(const ClusterArgs &a, size_t lds_bytes, bool compact, hipStream_t stream);

// Multi-workgroup path for frames above cap_points (cluster_big.hip).
size_t cluster_big_workspace(int32_t n_frames, int32_t total);
hipError_t launch_cluster_big(const ClusterArgs &a, void *workspace, hipStream_t stream);

// ----------------------------------------------------------------------------
// Density
// ----------------------------------------------------------------------------
struct DensityArgs {
    const int32_t *xy;
    const int32_t *offsets;
    int32_t n_frames;
    int32_t total;
    int32_t max_frame_points; // bound used to size the per-frame sort (0: no sort)
    int32_t width_px, height_px;
    int32_t grid_w, grid_h;
    float sigma_px;
    float *density;           // [n_frames][grid_h][grid_w]
};

struct DensityPlan {
    int gather;               // 1: factor tables gathered into registers; 0: recurrence
    int rm;                   // region height in tiles (16 rows gather, 32 recurrence)
    int rn;                   // region width in tiles
    int regions_y, regions_x; // regions per frame
    int split;                // bird slices per (frame, region); > 1 adds partial grids afterwards
    int waves;                // gather: waves sharing one (frame, region, slice)
    long long blocks;         // workgroups of the main kernel
};

DensityPlan plan_density(const DensityArgs &a, int n_cus, size_t lds_limit);
// Workspace for the partial grids of a split launch (0 if none); depends on the
// batch shape and grid only, and bounds every plan for that shape.
size_t density_workspace_bytes(int32_t n_frames, int32_t total, int32_t grid_w, int32_t grid_h, int n_cus);
hipError_t launch_density(const DensityArgs &a, const DensityPlan &p, float *partial, hipStream_t stream);
// The allocation-free entry point's scratch: a file-scope device array of
// kDensityScratchBytes per device (the partial grids of split launches).
// Returns its address on the current device (looked up once per device).
constexpr size_t kDensityScratchBytes = (size_t)16 << 20;
hipError_t density_static_scratch(void **ptr);

// ----------------------------------------------------------------------------
// Heatmap analytics
// ----------------------------------------------------------------------------
struct HeatArgs {
    const float *density;     // [n_frames][grid_h][grid_w]
    int32_t n_frames;
    int32_t grid_w, grid_h;
    int32_t tiles_x, tiles_y; // set by launch_heatmap
    double cell_area;
    float threshold;
    int32_t connectivity;     // 4 or 8
    int32_t *labels;          // [n_frames][grid_h][grid_w]
    int32_t *n_components;    // [n_frames]
    double *entropy;          // [n_frames]
    double *degree;           // [n_frames]
    int32_t *comp_cells;      // [n_frames][grid_h][grid_w]
    double *comp_mass;        // [n_frames][grid_h][grid_w]
};

size_t heatmap_workspace_bytes(int32_t n_frames, int32_t grid_w, int32_t grid_h);
// Dynamic LDS of the frame-resident kernel (one workgroup per frame), and
// its workspace (the per-frame fixed-point scales).
size_t heatmap_frame_lds_bytes(int32_t grid_w, int32_t grid_h);
size_t heatmap_frame_workspace_bytes(int32_t n_frames, int32_t grid_w, int32_t grid_h);
// resident: one workgroup per frame with the grid in LDS (needs
// heatmap_frame_lds_bytes within the device's limit); else the tiled kernels,
// which use the workspace.
hipError_t launch_heatmap(HeatArgs a, void *workspace, bool resident, hipStream_t stream);

// ----------------------------------------------------------------------------
// Region of interest
// ----------------------------------------------------------------------------
constexpr int kRoiMaxVertices = 64;
constexpr int kRoiBlock = 2048;  // birds per block of the ROI kernels

struct RoiArgs {
    const int32_t *xy;        // [total][2]
    const int32_t *offsets;   // [n_frames + 1]
    int32_t n_frames;
    int32_t total;
    int32_t n_vertices;       // 3 .. kRoiMaxVertices
    int32_t vx[kRoiMaxVertices], vy[kRoiMaxVertices];  // polygon, quanta
    int32_t bx0, by0, bx1, by1;                          // its bounding box
    int32_t *counts;          // [n_frames]
    int32_t *out_xy;          // [total][2] capacity
    int32_t *out_offsets;     // [n_frames + 1]
    int32_t *out_index;       // [total] capacity, or nullptr
};

size_t roi_workspace_bytes(int32_t total);
hipError_t launch_roi(const RoiArgs &a, void *workspace, hipStream_t stream);

// ----------------------------------------------------------------------------
// Drinker-line proximity
// ----------------------------------------------------------------------------
constexpr int kDrinkMaxLines = 64;

struct DrinkArgs {
    const int32_t *xy;        // [total][2]
    const int32_t *offsets;   // [n_frames + 1]
    int32_t n_frames;
    int32_t total;
    int32_t n_lines;          // 1 .. kDrinkMaxLines
    int32_t threshold;        // quanta, 0 .. 2^24
    int32_t ax[kDrinkMaxLines], ay[kDrinkMaxLines], bx[kDrinkMaxLines], by[kDrinkMaxLines];
    uint8_t *drinking;        // [total], 16-byte aligned
    int32_t *line;            // [total] or nullptr
    int32_t *counts;          // [n_frames]
};

size_t drink_workspace_bytes(int32_t total);
hipError_t launch_drinkers(const DrinkArgs &a, void *workspace, hipStream_t stream);

// Detection post-processing (mask components with statistics)
constexpr int kMaskTile = 64;  // tile side in pixels

struct MaskArgs {
    const float *prob;         // [n_frames][height][width]
    int32_t n_frames, width, height;
    float threshold;
    int32_t connectivity;
    int32_t tiles_x, tiles_y;  // set by launch_mask
    int64_t n_tiles;
    int64_t frame_slots, band_slots;
    int32_t *labels;           // optional
    int32_t *n_components;     // [n_frames]
    int32_t *comp_offsets;     // [n_frames + 1]
    int64_t capacity;
    int32_t *comp_label, *comp_area, *comp_box;  // each optional
    double *comp_centroid;
    int32_t *comp_xy;
    float *comp_score;
};
size_t mask_workspace_bytes(int32_t n_frames, int32_t width, int32_t height, int32_t connectivity);
hipError_t launch_mask(MaskArgs a, void *workspace, hipStream_t stream);

}  // namespace flock

// api.cpp - the C ABI of libflock (declared in include/flock.h): argument
// validation, launch planning and error reporting.  No computation happens
// here; every step of the path runs in the HIP kernels.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "flock.h"
#include "internal.h"

namespace {

thread_local char g_error[512];

flock_status fail(flock_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
    return st;
}

flock_status hip_fail(hipError_t err, const char *what) {
    return fail(FLOCK_EDEVICE, "%s: %s", what, hipGetErrorString(err));
}

struct DeviceInfo {
    bool valid = false;
    bool gfx950 = false;
    int n_cus = 0;
    size_t lds_per_block = 0;
    size_t lds_per_cu = 0;
    char arch[64] = {0};
};

constexpr int kMaxDevices = 64;
DeviceInfo g_devices[kMaxDevices];
std::once_flag g_device_once[kMaxDevices];

flock_status device_info(const DeviceInfo **out) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return hip_fail(err, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(FLOCK_EUNSUPPORTED, "device index %d", dev);
    std::call_once(g_device_once[dev], [dev] {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return;
        DeviceInfo &d = g_devices[dev];
        std::snprintf(d.arch, sizeof d.arch, "%s", prop.gcnArchName);
        d.gfx950 = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
        d.n_cus = prop.multiProcessorCount;
        d.lds_per_block = prop.sharedMemPerBlock;
        d.lds_per_cu = prop.maxSharedMemoryPerMultiProcessor;
        d.valid = true;
    });
    const DeviceInfo &d = g_devices[dev];
    if (!d.valid) return fail(FLOCK_EDEVICE, "could not read properties of device %d", dev);
    if (!d.gfx950) return fail(FLOCK_EUNSUPPORTED, "device %d is %s; this library is built for gfx950", dev, d.arch);
    *out = &d;
    return FLOCK_OK;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool validate_requested() {
    const char *v = std::getenv("FLOCK_VALIDATE");
    return v && v[0] == '1';
}

// Debug mode: copy offsets (and coordinates) to the host and check them.
flock_status validate_batch(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t total,
                            hipStream_t stream) {
    std::vector<int32_t> off((size_t)n_frames + 1);
    hipError_t err = hipMemcpyAsync(off.data(), offsets, off.size() * sizeof(int32_t),
                                    hipMemcpyDeviceToHost, stream);
    if (err == hipSuccess) err = hipStreamSynchronize(stream);
    if (err != hipSuccess) return hip_fail(err, "FLOCK_VALIDATE offsets copy");
    if (off[0] != 0) return fail(FLOCK_EINVAL, "offsets[0] = %d, expected 0", off[0]);
    for (int32_t f = 0; f < n_frames; ++f)
        if (off[f + 1] < off[f]) return fail(FLOCK_EINVAL, "offsets decrease at frame %d", f);
    if (off[n_frames] != total)
        return fail(FLOCK_EINVAL, "offsets[n_frames] = %d but total = %d", off[n_frames], total);
    if (total > 0) {
        std::vector<int32_t> h((size_t)total * 2);
        err = hipMemcpyAsync(h.data(), xy, h.size() * sizeof(int32_t), hipMemcpyDeviceToHost, stream);
        if (err == hipSuccess) err = hipStreamSynchronize(stream);
        if (err != hipSuccess) return hip_fail(err, "FLOCK_VALIDATE xy copy");
        for (size_t i = 0; i < h.size(); ++i)
            if (h[i] < 0 || h[i] >= (1 << 24))
                return fail(FLOCK_EINVAL, "coordinate %d of bird %zu outside [0, 2^24)", h[i], i / 2);
    }
    return FLOCK_OK;
}

// Largest s >= 1 with 2 s^2 <= e^2 (cell side whose diagonal is <= e).
int32_t diagonal_cell_side(int32_t e) {
    const int64_t half = (int64_t)e * e / 2;
    int64_t s = (int64_t)std::sqrt((double)half);
    while (s * s > half) --s;
    while ((s + 1) * (s + 1) <= half) ++s;
    return s < 1 ? 1 : (int32_t)s;
}

// The on-chip kernel's neighbour-cell tables for cells of side `side`
// (offsets (dx, dy), |dx|, |dy| <= reach <= 2, whose cells can hold points
// within e: gap(|dx|)^2 + gap(|dy|)^2 <= e^2, gap(d) = (d - 1) side + 1 for
// d > 0).  Whole stencil by gap distance, ties in row-major order; forward
// half (dy > 0, or dy = 0 and dx > 0) with the adjacent cells first.
void pack_stencil(int32_t e, int32_t side, flock::ClusterArgs *a) {
    const int reach = e == 0 ? 0 : std::min(1 + (e - 1) / side, 7);
    auto gap = [side](int d) -> int64_t { d = d < 0 ? -d : d; return d == 0 ? 0 : (int64_t)(d - 1) * side + 1; };
    struct Off { int dx, dy; int64_t key; int idx; };
    std::vector<Off> all, adj, far;
    int rowcnt[3] = {0, 0, 0};
    for (int idx = 0; idx < 25; ++idx) {
        const int dx = idx % 5 - 2, dy = idx / 5 - 2;
        if (std::abs(dx) > reach || std::abs(dy) > reach) continue;
        const int64_t d = gap(dx) * gap(dx) + gap(dy) * gap(dy);
        if (d > (int64_t)e * e) continue;
        all.push_back({dx, dy, d, idx});
        if (dy >= 0) rowcnt[dy]++;
        if (dy > 0 || (dy == 0 && dx > 0)) (std::abs(dx) <= 1 && std::abs(dy) <= 1 ? adj : far).push_back({dx, dy, d, idx});
    }
    std::stable_sort(all.begin(), all.end(), [](const Off &x, const Off &y) { return x.key < y.key; });
    auto code = [](const Off &o) { return (uint32_t)((o.dx + 2) | ((o.dy + 2) << 3)); };
    for (uint32_t &w : a->sten_all) w = 0;
    for (uint32_t &w : a->sten_fwd) w = 0;
    for (size_t i = 0; i < all.size(); ++i) a->sten_all[i / 5] |= code(all[i]) << (6 * (i % 5));
    std::vector<Off> fwd = adj;
    fwd.insert(fwd.end(), far.begin(), far.end());
    for (size_t i = 0; i < fwd.size(); ++i) a->sten_fwd[i / 5] |= code(fwd[i]) << (6 * (i % 5));
    uint32_t meta = (uint32_t)all.size() | ((uint32_t)adj.size() << 8) | ((uint32_t)fwd.size() << 16);
    for (int k = 0; k < 3; ++k) meta |= (uint32_t)(rowcnt[k] > 0 ? (rowcnt[k] - 1) / 2 : 0) << (24 + 2 * k);
    a->sten_meta = meta;
}

struct ClusterPlan {
    int32_t cap_points;
    int32_t cap_cells;
    size_t lds_bytes;
    bool compact = false;  // two workgroups per compute unit
};

ClusterPlan plan_cluster(int32_t max_frame_points, size_t lds_limit) {
    ClusterPlan p;
    int32_t limit = flock::cluster_max_cap_points(lds_limit);
    // FLOCK_CLUSTER_CAP lowers the on-chip capacity (for tuning the split
    // between the on-chip and the multi-workgroup paths)
    const char *cap = std::getenv("FLOCK_CLUSTER_CAP");
    if (cap && std::atoi(cap) > 0) limit = std::min(limit, std::atoi(cap));
    p.cap_points = (max_frame_points > 0 && max_frame_points < limit) ? max_frame_points : limit;
    const size_t reserve = 1024;  // static shared variables
    const int64_t avail = (int64_t)lds_limit - (int64_t)reserve - 13 * (int64_t)p.cap_points - 4;
    int64_t cells = std::max<int64_t>(4096, 2 * (int64_t)p.cap_points);
    cells = std::min<int64_t>(cells, avail / 6);
    p.cap_cells = (int32_t)cells;
    p.lds_bytes = flock::cluster_lds_bytes(p.cap_points, p.cap_cells);
    return p;
}

// With more frames than compute units and frames of at most
// kClusterCompactCap points, two workgroups share a compute unit when half
// its LDS holds the frame with a cell table of at least kCompactMinCells
// entries (a 1080p frame at eps 40 px needs 2652).  A frame whose grid has
// more cells than the table runs on a coarsened grid (correct, slower).
// FLOCK_CLUSTER_COMPACT=0 turns this off.
constexpr int64_t kCompactMinCells = 2048;

void plan_compact(ClusterPlan *p, int32_t max_frame_points, int32_t n_frames, const DeviceInfo &dev) {
    const char *env = std::getenv("FLOCK_CLUSTER_COMPACT");
    if (env && std::strcmp(env, "0") == 0) return;
    if (n_frames <= dev.n_cus || max_frame_points <= 0 || max_frame_points > flock::kClusterCompactCap) return;
    if (max_frame_points > p->cap_points) return;
    const size_t half = (dev.lds_per_cu ? dev.lds_per_cu : dev.lds_per_block) / 2;
    const size_t fixed = flock::cluster_compact_static_lds() + 16;  // static variables, alignment
    const int64_t avail = (int64_t)half - (int64_t)fixed - 13 * (int64_t)max_frame_points - 4;
    const int64_t cells = std::min<int64_t>(avail / 6, 2 * (int64_t)max_frame_points + 4096);
    if (cells < kCompactMinCells) return;
    const size_t bytes = flock::cluster_lds_bytes(max_frame_points, (int32_t)cells);
    if (bytes + fixed > half) return;
    p->cap_points = max_frame_points;
    p->cap_cells = (int32_t)cells;
    p->lds_bytes = bytes;
    p->compact = true;
}

}  // namespace

extern "C" {

const char *flock_last_error(void) { return g_error; }

const char *flock_version(void) { return "flock 0.1.0 gfx950"; }

size_t cluster_frames_workspace(int32_t n_frames, int32_t total, int32_t max_frame_points) {
    if (n_frames <= 0 || total <= 0 || max_frame_points < 0) return 0;
    const DeviceInfo *dev = nullptr;
    size_t lds = 160 * 1024;
    if (device_info(&dev) == FLOCK_OK) lds = dev->lds_per_block;
    g_error[0] = '\0';
    const ClusterPlan plan = plan_cluster(max_frame_points, lds);
    const bool big = max_frame_points == 0 || max_frame_points > plan.cap_points;
    return big ? flock::cluster_big_workspace(n_frames, total) : 0;
}

size_t density_frames_workspace(int32_t n_frames, int32_t total, int32_t grid_w, int32_t grid_h) {
    const DeviceInfo *dev = nullptr;
    int n_cus = 256;
    if (device_info(&dev) == FLOCK_OK) n_cus = dev->n_cus;
    g_error[0] = '\0';
    return flock::density_workspace_bytes(n_frames, total, grid_w, grid_h, n_cus);
}

flock_status cluster_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t total,
                            int32_t max_frame_points, int32_t eps_q, int32_t min_pts, int32_t *labels,
                            uint8_t *kind, int32_t *n_clusters, void *workspace, size_t workspace_bytes,
                            void *stream) {
    g_error[0] = '\0';
    if (n_frames < 0) return fail(FLOCK_EINVAL, "n_frames = %d < 0", n_frames);
    if (total < 0) return fail(FLOCK_EINVAL, "total = %d < 0", total);
    if (max_frame_points < 0) return fail(FLOCK_EINVAL, "max_frame_points = %d < 0", max_frame_points);
    if (eps_q < 0 || eps_q > 32766) return fail(FLOCK_EINVAL, "eps_q = %d outside [0, 32766]", eps_q);
    if (min_pts < 1) return fail(FLOCK_EINVAL, "min_pts = %d < 1", min_pts);
    if (n_frames == 0) return FLOCK_OK;
    if (!offsets) return fail(FLOCK_EINVAL, "offsets is NULL");
    if (total > 0 && (!xy || !labels || !kind))
        return fail(FLOCK_EINVAL, "xy, labels and kind must be non-NULL when total > 0");
    if (!aligned(xy, 8)) return fail(FLOCK_EINVAL, "xy must be 8-byte aligned");
    if (!aligned(offsets, 4) || !aligned(labels, 4) || !aligned(n_clusters, 4))
        return fail(FLOCK_EINVAL, "offsets, labels and n_clusters must be 4-byte aligned");
    if (total == 0 && !n_clusters) return FLOCK_OK;

    const DeviceInfo *dev = nullptr;
    flock_status st = device_info(&dev);
    if (st != FLOCK_OK) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (validate_requested()) {
        st = validate_batch(xy, offsets, n_frames, total, s);
        if (st != FLOCK_OK) return st;
    }

    ClusterPlan plan = plan_cluster(max_frame_points, dev->lds_per_block);
    const bool big = max_frame_points == 0 || max_frame_points > plan.cap_points;
    if (!big) plan_compact(&plan, max_frame_points, n_frames, *dev);
    const size_t ws_need = big ? flock::cluster_big_workspace(n_frames, total) : 0;
    if (workspace && workspace_bytes < ws_need)
        return fail(FLOCK_ENOMEM, "workspace of %zu bytes, %zu needed", workspace_bytes, ws_need);
    if (workspace && !aligned(workspace, 256)) return fail(FLOCK_EINVAL, "workspace must be 256-byte aligned");
    flock::ClusterArgs a{};
    a.xy = xy;
    a.offsets = offsets;
    a.n_frames = n_frames;
    a.total = total;
    a.eps_q = eps_q;
    a.min_pts = min_pts;
    a.cell_side = diagonal_cell_side(eps_q);
    pack_stencil(eps_q, a.cell_side, &a);
    a.cap_points = plan.cap_points;
    a.cap_cells = plan.cap_cells;
    a.labels = labels;
    a.kind = kind;
    a.n_clusters = n_clusters;
    a.big_path = big ? 1 : 0;
    {
        // FLOCK_CLUSTER_UNION=lds takes the general union stage for every
        // frame (for tests of that path)
        const char *u = std::getenv("FLOCK_CLUSTER_UNION");
        a.union_regs = (u && std::strcmp(u, "lds") == 0) ? 0 : 1;
    }
    // one frame above the on-chip capacity (offsets[1] = total): the
    // multi-workgroup path alone, without an on-chip launch that would only
    // return
    a.big_all = big && n_frames == 1 && total > plan.cap_points ? 1 : 0;
    hipError_t err = hipSuccess;
    if (!a.big_all) {
        err = flock::launch_cluster_resident(a, plan.lds_bytes, plan.compact, s);
        if (err != hipSuccess) return hip_fail(err, "cluster kernel launch");
    }
    if (big && total > 0) {
        void *ws = workspace;
        if (!ws) {
            err = hipMallocAsync(&ws, ws_need, s);
            if (err != hipSuccess) return fail(FLOCK_ENOMEM, "hipMallocAsync(%zu): %s", ws_need,
                                               hipGetErrorString(err));
        }
        err = flock::launch_cluster_big(a, ws, s);
        if (!workspace) {
            const hipError_t ferr = hipFreeAsync(ws, s);
            if (err == hipSuccess) err = ferr;
        }
        if (err != hipSuccess) return hip_fail(err, "large-frame cluster kernels");
    }
    return FLOCK_OK;
}

}  // extern "C"

namespace {

// density_frames and density_frames_noalloc: the same checks, plan and
// kernels; they differ only in where a split launch keeps its partial grids
// (the caller's workspace or a library allocation, or the static scratch).
flock_status density_run(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t total,
                         int32_t max_frame_points, int32_t width_px, int32_t height_px, int32_t grid_w,
                         int32_t grid_h, float sigma_px, float *density, void *workspace,
                         size_t workspace_bytes, bool noalloc, void *stream) {
    g_error[0] = '\0';
    if (n_frames < 0) return fail(FLOCK_EINVAL, "n_frames = %d < 0", n_frames);
    if (total < 0) return fail(FLOCK_EINVAL, "total = %d < 0", total);
    if (max_frame_points < 0) return fail(FLOCK_EINVAL, "max_frame_points = %d < 0", max_frame_points);
    if (width_px < 1 || height_px < 1)
        return fail(FLOCK_EINVAL, "frame extent %d x %d px must be >= 1", width_px, height_px);
    if (grid_w < 1 || grid_h < 1 || grid_w > 4096 || grid_h > 4096)
        return fail(FLOCK_EINVAL, "grid %d x %d outside 1..4096", grid_w, grid_h);
    if (!std::isfinite(sigma_px) || !(sigma_px > 0.0f))
        return fail(FLOCK_EINVAL, "sigma_px must be finite and > 0");
    if (n_frames == 0) return FLOCK_OK;
    if (!offsets || !density) return fail(FLOCK_EINVAL, "offsets and density must be non-NULL");
    if (total > 0 && !xy) return fail(FLOCK_EINVAL, "xy is NULL with total > 0");
    if (!aligned(xy, 8)) return fail(FLOCK_EINVAL, "xy must be 8-byte aligned");
    if (!aligned(offsets, 4) || !aligned(density, 4))
        return fail(FLOCK_EINVAL, "offsets and density must be 4-byte aligned");

    const DeviceInfo *dev = nullptr;
    flock_status st = device_info(&dev);
    if (st != FLOCK_OK) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    // the debug check copies to the host and synchronises: never on the
    // allocation-free entry point, which may run under graph capture
    if (!noalloc && validate_requested()) {
        st = validate_batch(xy, offsets, n_frames, total, s);
        if (st != FLOCK_OK) return st;
    }

    flock::DensityArgs a;
    a.xy = xy;
    a.offsets = offsets;
    a.n_frames = n_frames;
    a.total = total;
    a.max_frame_points = max_frame_points;
    a.width_px = width_px;
    a.height_px = height_px;
    a.grid_w = grid_w;
    a.grid_h = grid_h;
    a.sigma_px = sigma_px;
    a.density = density;
    const flock::DensityPlan plan = flock::plan_density(a, dev->n_cus, dev->lds_per_block);
    if (plan.blocks > 0x7fffffffLL) return fail(FLOCK_EUNSUPPORTED, "batch too large for one launch");
    // a split launch keeps partial grids in the workspace
    const size_t need = plan.split > 1 ? (size_t)n_frames * plan.split * (size_t)grid_w * grid_h * sizeof(float) : 0;
    void *ws = workspace;
    hipError_t err = hipSuccess;
    if (noalloc) {
        if (need > flock::kDensityScratchBytes)
            return fail(FLOCK_ENOMEM,
                        "this batch needs %zu bytes of partial grids, beyond the %zu bytes of static scratch "
                        "of the allocation-free entry point (density_frames with a workspace takes it)",
                        need, flock::kDensityScratchBytes);
        ws = nullptr;
        if (need > 0) {
            err = flock::density_static_scratch(&ws);
            if (err != hipSuccess || !ws) return hip_fail(err, "static scratch address");
        }
    } else {
        if (workspace && workspace_bytes < need)
            return fail(FLOCK_ENOMEM, "workspace of %zu bytes < %zu needed", workspace_bytes, need);
        if (workspace && !aligned(workspace, 256)) return fail(FLOCK_EINVAL, "workspace must be 256-byte aligned");
        if (need > 0 && !ws) {
            err = hipMallocAsync(&ws, need, s);
            if (err != hipSuccess) return hip_fail(err, "workspace allocation");
        }
    }
    err = flock::launch_density(a, plan, static_cast<float *>(ws), s);
    if (!noalloc && need > 0 && !workspace) {
        const hipError_t ferr = hipFreeAsync(ws, s);
        if (err == hipSuccess) err = ferr;
    }
    if (err != hipSuccess) return hip_fail(err, "density kernel launch");
    return FLOCK_OK;
}

}  // namespace

extern "C" {

flock_status density_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t total,
                            int32_t max_frame_points, int32_t width_px, int32_t height_px,
                            int32_t grid_w, int32_t grid_h,
                            float sigma_px, float *density, void *workspace, size_t workspace_bytes,
                            void *stream) {
    return density_run(xy, offsets, n_frames, total, max_frame_points, width_px, height_px, grid_w, grid_h,
                       sigma_px, density, workspace, workspace_bytes, false, stream);
}

flock_status density_frames_noalloc(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t total,
                                    int32_t max_frame_points, int32_t width_px, int32_t height_px,
                                    int32_t grid_w, int32_t grid_h, float sigma_px, float *density,
                                    void *stream) {
    return density_run(xy, offsets, n_frames, total, max_frame_points, width_px, height_px, grid_w, grid_h,
                       sigma_px, density, nullptr, 0, true, stream);
}

size_t roi_filter_frames_workspace(int32_t n_frames, int32_t total) {
    g_error[0] = '\0';
    return n_frames > 0 ? flock::roi_workspace_bytes(total) : 0;  // flags, block counts and bases, staging
}

flock_status roi_filter_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t total,
                               const int32_t *roi_xy, int32_t n_vertices, int32_t *counts, int32_t *out_xy,
                               int32_t *out_offsets, int32_t *out_index, void *workspace,
                               size_t workspace_bytes, void *stream) {
    g_error[0] = '\0';
    if (n_frames < 0) return fail(FLOCK_EINVAL, "n_frames = %d < 0", n_frames);
    if (total < 0) return fail(FLOCK_EINVAL, "total = %d < 0", total);
    if (n_vertices < 3 || n_vertices > flock::kRoiMaxVertices)
        return fail(FLOCK_EINVAL, "n_vertices = %d outside 3..%d", n_vertices, flock::kRoiMaxVertices);
    if (!roi_xy) return fail(FLOCK_EINVAL, "roi_xy must be non-NULL");
    flock::RoiArgs a;
    for (int v = 0; v < n_vertices; ++v) {
        const int32_t x = roi_xy[2 * v], y = roi_xy[2 * v + 1];
        if (x < -(1 << 24) || x > (1 << 24) || y < -(1 << 24) || y > (1 << 24))
            return fail(FLOCK_EINVAL, "roi vertex %d = (%d, %d) outside |coordinate| <= 2^24", v, x, y);
        a.vx[v] = x;
        a.vy[v] = y;
    }
    for (int v = n_vertices; v < flock::kRoiMaxVertices; ++v) a.vx[v] = a.vy[v] = 0;
    a.bx0 = *std::min_element(a.vx, a.vx + n_vertices);
    a.bx1 = *std::max_element(a.vx, a.vx + n_vertices);
    a.by0 = *std::min_element(a.vy, a.vy + n_vertices);
    a.by1 = *std::max_element(a.vy, a.vy + n_vertices);
    if (n_frames == 0) return FLOCK_OK;
    if (!offsets || !counts || !out_offsets) return fail(FLOCK_EINVAL, "offsets, counts and out_offsets must be non-NULL");
    if ((long long)total / flock::kRoiBlock + 1 > 0x7fffffffLL / 64)
        return fail(FLOCK_EUNSUPPORTED, "batch too large for one launch");
    if (total > 0 && (!xy || !out_xy)) return fail(FLOCK_EINVAL, "xy and out_xy must be non-NULL with total > 0");
    if (!aligned(xy, 8) || !aligned(out_xy, 8)) return fail(FLOCK_EINVAL, "xy and out_xy must be 8-byte aligned");
    if (!aligned(offsets, 4) || !aligned(counts, 4) || !aligned(out_offsets, 4) || !aligned(out_index, 4))
        return fail(FLOCK_EINVAL, "offsets, counts, out_offsets and out_index must be 4-byte aligned");

    const DeviceInfo *dev = nullptr;
    flock_status st = device_info(&dev);
    if (st != FLOCK_OK) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (validate_requested()) {
        st = validate_batch(xy, offsets, n_frames, total, s);
        if (st != FLOCK_OK) return st;
    }
    const size_t need = flock::roi_workspace_bytes(total);
    if (workspace && workspace_bytes < need)
        return fail(FLOCK_ENOMEM, "workspace of %zu bytes < %zu needed", workspace_bytes, need);
    if (workspace && !aligned(workspace, 256)) return fail(FLOCK_EINVAL, "workspace must be 256-byte aligned");
    void *ws = workspace;
    hipError_t err = hipSuccess;
    if (!ws && need > 0) {
        err = hipMallocAsync(&ws, need, s);
        if (err != hipSuccess) return hip_fail(err, "workspace allocation");
    }
    a.xy = xy;
    a.offsets = offsets;
    a.n_frames = n_frames;
    a.total = total;
    a.n_vertices = n_vertices;
    a.counts = counts;
    a.out_xy = out_xy;
    a.out_offsets = out_offsets;
    a.out_index = out_index;
    err = flock::launch_roi(a, ws, s);
    if (!workspace && need > 0) {
        const hipError_t ferr = hipFreeAsync(ws, s);
        if (err == hipSuccess) err = ferr;
    }
    if (err != hipSuccess) return hip_fail(err, "roi kernels");
    return FLOCK_OK;
}

size_t drinker_proximity_frames_workspace(int32_t n_frames, int32_t total) {
    g_error[0] = '\0';
    return n_frames > 0 ? flock::drink_workspace_bytes(total) : 0;  // block counts and bases
}

flock_status drinker_proximity_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t total,
                                      const int32_t *lines, int32_t n_lines, int32_t threshold_q,
                                      uint8_t *drinking, int32_t *line, int32_t *counts, void *workspace,
                                      size_t workspace_bytes, void *stream) {
    g_error[0] = '\0';
    if (n_frames < 0) return fail(FLOCK_EINVAL, "n_frames = %d < 0", n_frames);
    if (total < 0) return fail(FLOCK_EINVAL, "total = %d < 0", total);
    if (n_lines < 1 || n_lines > flock::kDrinkMaxLines)
        return fail(FLOCK_EINVAL, "n_lines = %d outside 1..%d", n_lines, flock::kDrinkMaxLines);
    if (!lines) return fail(FLOCK_EINVAL, "lines must be non-NULL");
    if (threshold_q < 0 || threshold_q > (1 << 24))
        return fail(FLOCK_EINVAL, "threshold_q = %d outside 0..2^24", threshold_q);
    flock::DrinkArgs a;
    for (int l = 0; l < flock::kDrinkMaxLines; ++l) {
        if (l >= n_lines) {
            a.ax[l] = a.ay[l] = a.bx[l] = a.by[l] = 0;
            continue;
        }
        for (int k = 0; k < 4; ++k) {
            const int32_t v = lines[4 * l + k];
            if (v < -(1 << 24) || v > (1 << 24))
                return fail(FLOCK_EINVAL, "line %d coordinate %d outside |coordinate| <= 2^24", l, v);
        }
        a.ax[l] = lines[4 * l];
        a.ay[l] = lines[4 * l + 1];
        a.bx[l] = lines[4 * l + 2];
        a.by[l] = lines[4 * l + 3];
    }
    if (n_frames == 0) return FLOCK_OK;
    if (!offsets || !counts) return fail(FLOCK_EINVAL, "offsets and counts must be non-NULL");
    if (total > 0 && (!xy || !drinking)) return fail(FLOCK_EINVAL, "xy and drinking must be non-NULL with total > 0");
    if (!aligned(xy, 8)) return fail(FLOCK_EINVAL, "xy must be 8-byte aligned");
    if (!aligned(drinking, 16)) return fail(FLOCK_EINVAL, "drinking must be 16-byte aligned");
    if (!aligned(offsets, 4) || !aligned(counts, 4) || !aligned(line, 4))
        return fail(FLOCK_EINVAL, "offsets, counts and line must be 4-byte aligned");
    if ((long long)total / flock::kRoiBlock + 1 > 0x7fffffffLL / 64)
        return fail(FLOCK_EUNSUPPORTED, "batch too large for one launch");

    const DeviceInfo *dev = nullptr;
    flock_status st = device_info(&dev);
    if (st != FLOCK_OK) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (validate_requested()) {
        st = validate_batch(xy, offsets, n_frames, total, s);
        if (st != FLOCK_OK) return st;
    }
    const size_t need = flock::drink_workspace_bytes(total);
    if (workspace && workspace_bytes < need)
        return fail(FLOCK_ENOMEM, "workspace of %zu bytes < %zu needed", workspace_bytes, need);
    if (workspace && !aligned(workspace, 256)) return fail(FLOCK_EINVAL, "workspace must be 256-byte aligned");
    void *ws = workspace;
    hipError_t err = hipSuccess;
    if (!ws) {
        err = hipMallocAsync(&ws, need, s);
        if (err != hipSuccess) return hip_fail(err, "workspace allocation");
    }
    a.xy = xy;
    a.offsets = offsets;
    a.n_frames = n_frames;
    a.total = total;
    a.n_lines = n_lines;
    a.threshold = threshold_q;
    a.drinking = drinking;
    a.line = line;
    a.counts = counts;
    err = flock::launch_drinkers(a, ws, s);
    if (!workspace) {
        const hipError_t ferr = hipFreeAsync(ws, s);
        if (err == hipSuccess) err = ferr;
    }
    if (err != hipSuccess) return hip_fail(err, "drinker kernels");
    return FLOCK_OK;
}

size_t heatmap_frames_workspace(int32_t n_frames, int32_t grid_w, int32_t grid_h) {
    g_error[0] = '\0';
    // enough for either path (which one runs depends on the device's LDS)
    return std::max(flock::heatmap_workspace_bytes(n_frames, grid_w, grid_h),
                    flock::heatmap_frame_workspace_bytes(n_frames, grid_w, grid_h));
}

flock_status heatmap_frames(const float *density, int32_t n_frames, int32_t grid_w, int32_t grid_h,
                            double cell_area_px2, float threshold, int32_t connectivity, int32_t *labels,
                            int32_t *n_components, double *entropy, double *degree, int32_t *comp_cells,
                            double *comp_mass, void *workspace, size_t workspace_bytes, void *stream) {
    g_error[0] = '\0';
    if (n_frames < 0) return fail(FLOCK_EINVAL, "n_frames = %d < 0", n_frames);
    if (grid_w < 1 || grid_h < 1 || grid_w > 4096 || grid_h > 4096)
        return fail(FLOCK_EINVAL, "grid %d x %d outside 1..4096", grid_w, grid_h);
    if (!std::isfinite(cell_area_px2) || cell_area_px2 < 0.0)
        return fail(FLOCK_EINVAL, "cell_area_px2 must be finite and >= 0");
    if (!std::isfinite(threshold) || !(threshold > 0.0f))
        return fail(FLOCK_EINVAL, "threshold must be finite and > 0");
    if (connectivity != 4 && connectivity != 8)
        return fail(FLOCK_EINVAL, "connectivity = %d, expected 4 or 8", connectivity);
    if (n_frames == 0) return FLOCK_OK;
    if (!density || !labels || !n_components || !entropy || !degree || !comp_cells || !comp_mass)
        return fail(FLOCK_EINVAL, "density and every output must be non-NULL");
    if (!aligned(density, 4) || !aligned(labels, 4) || !aligned(n_components, 4) || !aligned(comp_cells, 4))
        return fail(FLOCK_EINVAL, "density, labels, n_components and comp_cells must be 4-byte aligned");
    if (!aligned(entropy, 8) || !aligned(degree, 8) || !aligned(comp_mass, 8))
        return fail(FLOCK_EINVAL, "entropy, degree and comp_mass must be 8-byte aligned");
    const long long tiles = (long long)((grid_w + 31) / 32) * ((grid_h + 31) / 32) * n_frames;
    const long long cells = (long long)grid_w * grid_h * n_frames;
    if (tiles > 0x7fffffffLL || (cells + 255) / 256 > 0x7fffffffLL)
        return fail(FLOCK_EUNSUPPORTED, "batch too large for one launch");

    const DeviceInfo *dev = nullptr;
    flock_status st = device_info(&dev);
    if (st != FLOCK_OK) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    // one workgroup per frame when the grid's forest fits in LDS
    // (FLOCK_HEATMAP_PATH=tiled takes the tiled kernels for every grid)
    const char *hp = std::getenv("FLOCK_HEATMAP_PATH");
    const bool tiled = hp && std::strcmp(hp, "tiled") == 0;
    const bool resident = !tiled && flock::heatmap_frame_lds_bytes(grid_w, grid_h) + 4096 <= dev->lds_per_block;
    const size_t need = resident ? flock::heatmap_frame_workspace_bytes(n_frames, grid_w, grid_h)
                                 : flock::heatmap_workspace_bytes(n_frames, grid_w, grid_h);
    if (workspace && workspace_bytes < need)
        return fail(FLOCK_ENOMEM, "workspace of %zu bytes < %zu needed", workspace_bytes, need);
    if (workspace && !aligned(workspace, 256)) return fail(FLOCK_EINVAL, "workspace must be 256-byte aligned");
    void *ws = workspace;
    hipError_t err = hipSuccess;
    if (!ws && need > 0) {
        err = hipMallocAsync(&ws, need, s);
        if (err != hipSuccess) return hip_fail(err, "workspace allocation");
    }
    flock::HeatArgs a;
    a.density = density;
    a.n_frames = n_frames;
    a.grid_w = grid_w;
    a.grid_h = grid_h;
    a.tiles_x = a.tiles_y = 0;
    a.cell_area = cell_area_px2;
    a.threshold = threshold;
    a.connectivity = connectivity;
    a.labels = labels;
    a.n_components = n_components;
    a.entropy = entropy;
    a.degree = degree;
    a.comp_cells = comp_cells;
    a.comp_mass = comp_mass;
    err = flock::launch_heatmap(a, ws, resident, s);
    if (!workspace && need > 0) {
        const hipError_t ferr = hipFreeAsync(ws, s);
        if (err == hipSuccess) err = ferr;
    }
    if (err != hipSuccess) return hip_fail(err, "heatmap kernels");
    return FLOCK_OK;
}

size_t mask_components_frames_workspace(int32_t n_frames, int32_t width, int32_t height, int32_t connectivity) {
    g_error[0] = '\0';
    return flock::mask_workspace_bytes(n_frames, width, height, connectivity);
}

flock_status mask_components_frames(const float *prob, int32_t n_frames, int32_t width, int32_t height,
                                    float threshold, int32_t connectivity, int32_t *labels,
                                    int32_t *n_components, int32_t *comp_offsets, int32_t capacity,
                                    int32_t *comp_label, int32_t *comp_area, int32_t *comp_box,
                                    double *comp_centroid, int32_t *comp_xy, float *comp_score, void *workspace,
                                    size_t workspace_bytes, void *stream) {
    g_error[0] = '\0';
    if (n_frames < 0) return fail(FLOCK_EINVAL, "n_frames = %d < 0", n_frames);
    if (width < 1 || height < 1 || width > 32768 || height > 32768)
        return fail(FLOCK_EINVAL, "frame %d x %d outside 1..32768", width, height);
    if (!std::isfinite(threshold) || !(threshold >= 0.0f))
        return fail(FLOCK_EINVAL, "threshold must be finite and >= 0");
    if (connectivity != 4 && connectivity != 8)
        return fail(FLOCK_EINVAL, "connectivity = %d, expected 4 or 8", connectivity);
    if (capacity < 0) return fail(FLOCK_EINVAL, "capacity = %d < 0", capacity);
    if ((long long)n_frames * width * height > 0x7fffffffLL)
        return fail(FLOCK_EUNSUPPORTED, "batch of %lld pixels above 2^31 - 1",
                    (long long)n_frames * width * height);
    if (n_frames == 0) return FLOCK_OK;
    if (!prob || !n_components || !comp_offsets)
        return fail(FLOCK_EINVAL, "prob, n_components and comp_offsets must be non-NULL");
    if (!aligned(prob, 4) || !aligned(labels, 4) || !aligned(n_components, 4) || !aligned(comp_offsets, 4) ||
        !aligned(comp_label, 4) || !aligned(comp_area, 4) || !aligned(comp_score, 4))
        return fail(FLOCK_EINVAL, "prob, labels, n_components, comp_offsets, comp_label, comp_area and "
                                  "comp_score must be 4-byte aligned");
    if (!aligned(comp_box, 16) || !aligned(comp_centroid, 16) || !aligned(comp_xy, 8))
        return fail(FLOCK_EINVAL, "comp_box and comp_centroid must be 16-byte aligned, comp_xy 8-byte aligned");

    const DeviceInfo *dev = nullptr;
    flock_status st = device_info(&dev);
    if (st != FLOCK_OK) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const size_t need = flock::mask_workspace_bytes(n_frames, width, height, connectivity);
    if (workspace && workspace_bytes < need)
        return fail(FLOCK_ENOMEM, "workspace of %zu bytes < %zu needed", workspace_bytes, need);
    if (workspace && !aligned(workspace, 256)) return fail(FLOCK_EINVAL, "workspace must be 256-byte aligned");
    void *ws = workspace;
    hipError_t err = hipSuccess;
    if (!ws) {
        err = hipMallocAsync(&ws, need, s);
        if (err != hipSuccess) return hip_fail(err, "workspace allocation");
    }
    flock::MaskArgs a{};
    a.prob = prob;
    a.n_frames = n_frames;
    a.width = width;
    a.height = height;
    a.threshold = threshold;
    a.connectivity = connectivity;
    a.labels = labels;
    a.n_components = n_components;
    a.comp_offsets = comp_offsets;
    a.capacity = capacity;
    a.comp_label = comp_label;
    a.comp_area = comp_area;
    a.comp_box = comp_box;
    a.comp_centroid = comp_centroid;
    a.comp_xy = comp_xy;
    a.comp_score = comp_score;
    err = flock::launch_mask(a, ws, s);
    if (!workspace) {
        const hipError_t ferr = hipFreeAsync(ws, s);
        if (err == hipSuccess) err = ferr;
    }
    if (err != hipSuccess) return hip_fail(err, "mask component kernels");
    return FLOCK_OK;
}

}  // extern "C"

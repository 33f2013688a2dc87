// Calls every entry point of the C ABI with invalid arguments (and with
// empty batches) and checks the status, the error text and that nothing
// touches the (fake, never dereferenced) device pointers.  Built with host
// AddressSanitizer / UndefinedBehaviorSanitizer around the library's host
// code; no GPU is needed, since every one of these calls returns before the
// device is queried.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "flock.h"

static int failures = 0;

static void expect(int32_t st, int32_t want, const char *needle, const char *what) {
    const char *msg = flock_last_error();
    if (st != want || (needle && !std::strstr(msg, needle))) {
        std::printf("%s: status %d (want %d), error \"%s\" (want \"%s\")\n", what, st, want, msg, needle ? needle : "");
        ++failures;
    }
}

int main() {
    void *fake = reinterpret_cast<void *>(0x100000);
    void *fake4 = reinterpret_cast<void *>(0x100004);
    const int32_t *xy = static_cast<const int32_t *>(fake), *off = static_cast<const int32_t *>(fake);
    int32_t *i32 = static_cast<int32_t *>(fake);
    uint8_t *u8 = static_cast<uint8_t *>(fake);
    float *f32 = static_cast<float *>(fake);
    double *f64 = static_cast<double *>(fake);
    // clustering
    expect(cluster_frames(xy, off, -1, 4, 0, 640, 4, i32, u8, i32, nullptr, 0, nullptr), FLOCK_EINVAL, "n_frames", "cluster n_frames");
    expect(cluster_frames(xy, off, 1, -5, 0, 640, 4, i32, u8, i32, nullptr, 0, nullptr), FLOCK_EINVAL, "total", "cluster total");
    expect(cluster_frames(xy, off, 1, 4, 0, 32767, 4, i32, u8, i32, nullptr, 0, nullptr), FLOCK_EINVAL, "eps_q", "cluster eps");
    expect(cluster_frames(xy, off, 1, 4, 0, 640, 0, i32, u8, i32, nullptr, 0, nullptr), FLOCK_EINVAL, "min_pts", "cluster minpts");
    expect(cluster_frames(xy, nullptr, 1, 4, 0, 640, 4, i32, u8, i32, nullptr, 0, nullptr), FLOCK_EINVAL, "offsets", "cluster offsets");
    expect(cluster_frames(static_cast<const int32_t *>(fake4), off, 1, 4, 0, 640, 4, i32, u8, i32, nullptr, 0, nullptr),
           FLOCK_EINVAL, "aligned", "cluster align");
    expect(cluster_frames(nullptr, nullptr, 0, 0, 0, 640, 4, nullptr, nullptr, nullptr, nullptr, 0, nullptr), FLOCK_OK, "", "cluster empty");
    // density
    expect(density_frames(xy, off, 1, 4, 0, 0, 1080, 128, 72, 30.0f, f32, nullptr, 0, nullptr), FLOCK_EINVAL, "extent", "density extent");
    expect(density_frames(xy, off, 1, 4, 0, 1920, 1080, 5000, 72, 30.0f, f32, nullptr, 0, nullptr), FLOCK_EINVAL, "grid", "density grid");
    expect(density_frames(xy, off, 1, 4, 0, 1920, 1080, 128, 72, NAN, f32, nullptr, 0, nullptr), FLOCK_EINVAL, "sigma", "density sigma");
    expect(density_frames(xy, off, 1, 4, 0, 1920, 1080, 128, 72, 30.0f, nullptr, nullptr, 0, nullptr), FLOCK_EINVAL, "non-NULL", "density out");
    expect(density_frames_noalloc(xy, off, 1, 4, 0, 1920, 1080, 128, 72, -1.0f, f32, nullptr), FLOCK_EINVAL, "sigma", "noalloc sigma");
    expect(density_frames_noalloc(nullptr, nullptr, 0, 0, 0, 1920, 1080, 128, 72, 30.0f, nullptr, nullptr), FLOCK_OK, "", "noalloc empty");
    // heatmap
    expect(heatmap_frames(f32, 1, 128, 72, 225.0, 0.0f, 8, i32, i32, f64, f64, i32, f64, nullptr, 0, nullptr), FLOCK_EINVAL,
           "threshold", "heatmap threshold");
    expect(heatmap_frames(f32, 1, 128, 72, 225.0, 1e-4f, 6, i32, i32, f64, f64, i32, f64, nullptr, 0, nullptr), FLOCK_EINVAL,
           "connectivity", "heatmap connectivity");
    // region of interest and drinkers (host polygons and lines)
    const int32_t square[8] = {0, 0, 160, 0, 160, 160, 0, 160};
    const int32_t far_poly[8] = {0, 0, 1 << 25, 0, 160, 160, 0, 160};
    expect(roi_filter_frames(xy, off, 1, 4, square, 2, i32, i32, i32, i32, nullptr, 0, nullptr), FLOCK_EINVAL, "n_vertices", "roi nv");
    expect(roi_filter_frames(xy, off, 1, 4, far_poly, 4, i32, i32, i32, i32, nullptr, 0, nullptr), FLOCK_EINVAL, "2^24", "roi far");
    const int32_t lines[8] = {0, 0, 160, 0, 0, 0, 0, 160};
    expect(drinker_proximity_frames(xy, off, 1, 4, lines, 2, -1, u8, i32, i32, nullptr, 0, nullptr), FLOCK_EINVAL,
           "threshold_q", "drinker threshold");
    expect(drinker_proximity_frames(xy, off, 1, 4, lines, 0, 64, u8, i32, i32, nullptr, 0, nullptr), FLOCK_EINVAL, "n_lines",
           "drinker lines");
    // mask components
    expect(mask_components_frames(f32, 1, 0, 48, 0.5f, 8, i32, i32, i32, 16, i32, i32, i32, f64, i32, f32, nullptr, 0, nullptr),
           FLOCK_EINVAL, "frame", "mask frame");
    expect(mask_components_frames(f32, 1, 64, 48, NAN, 8, i32, i32, i32, 16, i32, i32, i32, f64, i32, f32, nullptr, 0, nullptr),
           FLOCK_EINVAL, "threshold", "mask threshold");
    expect(mask_components_frames(f32, 1024, 32768, 32768, 0.5f, 8, i32, i32, i32, 16, i32, i32, i32, f64, i32, f32, nullptr, 0,
                                  nullptr),
           FLOCK_EUNSUPPORTED, nullptr, "mask size");
    if (std::strlen(flock_last_error()) >= 512) ++failures;  // the error text fits its buffer
    if (std::strncmp(flock_version(), "flock ", 6) != 0) ++failures;
    if (failures) {
        std::printf("%d failures\n", failures);
        return 1;
    }
    std::printf("abi checks ok\n");
    return 0;
}

/* Runs the oracle's threaded batch functions (clustering, density grids,
 * sampled density cells, heatmap analytics) on a seeded synthetic batch with
 * one thread and with several, and checks that the outputs are identical.
 * Built together with oracle.c under a sanitizer (ThreadSanitizer for the
 * worker threads), so any data race in the oracle's threading is reported. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int32_t oracle_cluster_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t eps_q,
                              int32_t min_pts, int32_t *labels, uint8_t *kind, int32_t *n_clusters,
                              int32_t n_threads);
int32_t oracle_density_frames(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t width_px,
                              int32_t height_px, int32_t grid_w, int32_t grid_h, double sigma_px,
                              double *density, int32_t n_threads);
int32_t oracle_density_cells(const int32_t *xy, const int32_t *offsets, int32_t n_frames, int32_t width_px,
                             int32_t height_px, int32_t grid_w, int32_t grid_h, double sigma_px,
                             const int32_t *cell_frame, const int32_t *cell_gx, const int32_t *cell_gy,
                             int64_t m, double *out, int32_t n_threads);
int32_t oracle_heatmap_frames(const float *density, int32_t n_frames, int32_t grid_w, int32_t grid_h,
                              double cell_area, float threshold, int32_t connectivity, int32_t *labels,
                              int32_t *n_components, double *entropy, double *degree, int32_t *comp_cells,
                              double *comp_mass, int32_t n_threads);

static uint64_t state = 0x9e3779b97f4a7c15ull;
static uint32_t next_u32(void) {
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return (uint32_t)(state >> 16);
}

#define F 12
#define GW 64
#define GH 36

int main(void) {
    int32_t offsets[F + 1];
    offsets[0] = 0;
    for (int f = 0; f < F; ++f) offsets[f + 1] = offsets[f] + (f == 3 ? 0 : 100 + (int32_t)(next_u32() % 400));
    const int32_t T = offsets[F];
    int32_t *xy = malloc(sizeof(int32_t) * 2 * (size_t)T);
    for (int32_t i = 0; i < T; ++i) {
        /* clumps plus background, 1920 x 1080 px in 1/16 px */
        const int32_t cx = (int32_t)(next_u32() % 4) * 7000 + 3000, cy = (int32_t)(next_u32() % 3) * 5000 + 2000;
        const int near = next_u32() % 3 != 0;
        xy[2 * i] = near ? cx + (int32_t)(next_u32() % 2000) : (int32_t)(next_u32() % (16 * 1920));
        xy[2 * i + 1] = near ? cy + (int32_t)(next_u32() % 2000) : (int32_t)(next_u32() % (16 * 1080));
    }
    int fails = 0;
    for (int run = 0; run < 2; ++run) {
        const int32_t threads = run == 0 ? 1 : 6;
        static int32_t lab[2][8192], ncl[2][F];
        static uint8_t kind[2][8192];
        static double dens[2][F * GW * GH], cells[2][F * 16];
        static int32_t hl[2][F * GW * GH], hc[2][F * GW * GH], hn[2][F];
        static double hm[2][F * GW * GH], he[2][F], hd[2][F];
        static float densf[F * GW * GH];
        int32_t fr[F * 16], gx[F * 16], gy[F * 16];
        if (oracle_cluster_frames(xy, offsets, F, 640, 4, lab[run], kind[run], ncl[run], threads) != 0) return 2;
        if (oracle_density_frames(xy, offsets, F, 1920, 1080, GW, GH, 30.0, dens[run], threads) != 0) return 2;
        for (int k = 0; k < F * 16; ++k) {
            fr[k] = k / 16;
            gx[k] = (k * 7) % GW;
            gy[k] = (k * 5) % GH;
        }
        if (oracle_density_cells(xy, offsets, F, 1920, 1080, GW, GH, 30.0, fr, gx, gy, F * 16, cells[run], threads) != 0)
            return 2;
        for (int k = 0; k < F * GW * GH; ++k) densf[k] = (float)dens[0][k];
        if (oracle_heatmap_frames(densf, F, GW, GH, 900.0, 2e-5f, 8, hl[run], hn[run], he[run], hd[run], hc[run],
                                  hm[run], threads) != 0)
            return 2;
        if (run == 1) {
            fails += memcmp(lab[0], lab[1], sizeof(int32_t) * (size_t)T) != 0;
            fails += memcmp(kind[0], kind[1], (size_t)T) != 0;
            fails += memcmp(ncl[0], ncl[1], sizeof ncl[0]) != 0;
            fails += memcmp(dens[0], dens[1], sizeof dens[0]) != 0;
            fails += memcmp(cells[0], cells[1], sizeof cells[0]) != 0;
            fails += memcmp(hl[0], hl[1], sizeof hl[0]) != 0;
            fails += memcmp(hn[0], hn[1], sizeof hn[0]) != 0;
            fails += memcmp(he[0], he[1], sizeof he[0]) != 0;
            fails += memcmp(hd[0], hd[1], sizeof hd[0]) != 0;
            fails += memcmp(hc[0], hc[1], sizeof hc[0]) != 0;
            fails += memcmp(hm[0], hm[1], sizeof hm[0]) != 0;
        }
    }
    free(xy);
    if (fails) {
        printf("threaded outputs differ from one thread: %d arrays\n", fails);
        return 1;
    }
    printf("oracle threads ok: %d birds in %d frames\n", T, F);
    return 0;
}

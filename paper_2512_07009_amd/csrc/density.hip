// density.hip - Gaussian density grid per frame as a matrix-core contraction
// on gfx950.
//
// The per-frame density of Algorithm 1 (Section 3.6),
//     D[gy][gx] = c * sum_i exp(-((cx - x_i)^2 + (cy - y_i)^2) / (2 s^2)),
//     c = 1 / (2 pi s^2),
// separates into per-axis factors Fy[gy][i] = exp(-(cy - y_i)^2 / (2 s^2)) and
// Fx[gx][i] = exp(-(cx - x_i)^2 / (2 s^2)), so D = c * Fy . Fx^T: a dense
// contraction over the birds of the frame.
//
// Each workgroup (4 waves) owns one frame and one output region of
// (32 RM) gy rows x (32 RN) gx columns.  Birds stream through in chunks of
// kChunk: the chunk's factors for the region's rows and columns are written
// to LDS as fp16, then each wave runs v_mfma_f32_32x32x16_f16 over its quarter
// of the chunk for every tile of the region, accumulating in fp32.  At the
// end the four waves' partial sums are added in a fixed order through LDS, so
// the result is deterministic.
//
// Factor generation is windowed: a factor below 2^-25 rounds to +0 in fp16,
// and exp(-t^2/2) < 2^-25 for |t| > 5.9, so each bird only evaluates the rows
// within 6 s of it; the rest of the LDS tile is cleared to zero.  The fp16
// operands are those of the dense evaluation (up to fp32 rounding before the
// conversion), and the contraction itself stays dense over all (row, column,
// bird) triples.
//
// Along a window the factor follows a two-multiply recurrence on the row
// spacing h: with d the offset of a row centre from the bird,
//     F(d + h) = F(d) * R(d),   R(d + h) = R(d) * Q,
//     R(d) = exp(-(2 d h + h^2) / (2 s^2)),  Q = exp(-h^2 / s^2),
// started from exact exponentials at the two ends of the window's halves
// (two independent chains per thread) and restarted every kRestart rows,
// which bounds the accumulated fp32 error far below the fp16 rounding.  When
// h > 2 s (windows of a few rows) every factor is an exact exponential.
//
// Accuracy: each fp16 factor carries a relative rounding error <= 2^-11, so
// each term of the sum is within about 2^-10 of exact; all terms are positive,
// so the same relative bound holds for every output, which is <= the frame's
// maximum.

#include <cmath>
#include <cstdio>
#include <cstdlib>

#include "internal.h"

namespace flock {
namespace {

constexpr int kThreads = 256;       // 4 waves
constexpr int kChunk = 128;         // birds per LDS chunk: one (bird, axis) window per thread
constexpr int kPitch = kChunk + 8;  // halves per LDS row (16-byte skew between rows)
constexpr int kRestart = 16;        // rows between exact restarts of the recurrence
constexpr float kCutSigmas = 6.0f;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));

struct Geometry {
    float hx, hy;          // cell size, px
    float inv_hx, inv_hy;
    float neg_k;           // -log2(e) / (2 s^2): exp(-d^2/(2s^2)) = exp2(d^2 * neg_k)
    float cut;             // window half-width, px
    float scale;           // 1 / (2 pi s^2)
    int recur_x, recur_y;  // recurrence usable along the axis (h <= 2 s)
};

template <int RM, int RN>
struct Layout {
    static constexpr int kRowsY = 32 * RM;
    static constexpr int kRowsX = 32 * RN;
    static constexpr int kFactorBytes = (kRowsY + kRowsX) * kPitch * 2;
    static constexpr int kRedBytes = 4 * 32 * 33 * 4;  // one tile from each wave, padded rows
    static constexpr int kBytes = kFactorBytes > kRedBytes ? kFactorBytes : kRedBytes;
};

// Write one bird's factors for rows [row0, row0 + nrows) of one axis into a
// column of buf (row-major, kPitch halves per row); rows outside the window
// are left as they are (cleared).  A row just outside the computed window has
// a factor below 2^-25 (its fp16 value is +0), so float rounding of the
// bounds cannot change the tile.
__device__ __forceinline__ void fill_window(_Float16 *col, float pos, float h, float inv_h, int grid_n,
                                            int row0, int nrows, float neg_k, float cut, bool recur) {
    int lo = max((int)ceilf((pos - cut) * inv_h - 0.5f), row0);
    int hi = min((int)floorf((pos + cut) * inv_h - 0.5f), min(row0 + nrows, grid_n) - 1);
    if (!recur) {
        for (int row = lo; row <= hi; ++row) {
            const float d = ((float)row + 0.5f) * h - pos;
            col[(row - row0) * kPitch] = (_Float16)__builtin_amdgcn_exp2f(d * d * neg_k);
        }
        return;
    }
    const float q = __builtin_amdgcn_exp2f(2.0f * h * h * neg_k);
    // two chains: rows lo.. upward and rows hi.. downward, meeting in the middle
    const int mid = (lo + hi) >> 1;
    for (int base = lo, top = hi; base <= mid; base += kRestart, top -= kRestart) {
        const float da = ((float)base + 0.5f) * h - pos;
        const float db = ((float)top + 0.5f) * h - pos;
        float fa = __builtin_amdgcn_exp2f(da * da * neg_k);
        float ra = __builtin_amdgcn_exp2f((2.0f * da + h) * h * neg_k);
        float fb = __builtin_amdgcn_exp2f(db * db * neg_k);
        float rb = __builtin_amdgcn_exp2f((h - 2.0f * db) * h * neg_k);  // ratio going down
        const int steps = min(kRestart, mid - base + 1);
        for (int i = 0; i < steps; ++i) {
            col[(base + i - row0) * kPitch] = (_Float16)fa;
            if (top - i > mid) col[(top - i - row0) * kPitch] = (_Float16)fb;
            fa *= ra;
            ra *= q;
            fb *= rb;
            rb *= q;
        }
    }
}

template <int RM, int RN>
__global__ __launch_bounds__(kThreads) void density_kernel(DensityArgs a, Geometry g, int regions_y,
                                                           int regions_x) {
    using L = Layout<RM, RN>;
    __shared__ __align__(16) unsigned char lds[L::kBytes];
    _Float16 *fy = reinterpret_cast<_Float16 *>(lds);
    _Float16 *fx = fy + L::kRowsY * kPitch;

    const int regions = regions_y * regions_x;
    const int f = blockIdx.x / regions;
    const int reg = blockIdx.x - f * regions;
    const int gy0 = (reg / regions_x) * L::kRowsY;
    const int gx0 = (reg % regions_x) * L::kRowsX;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    const int32_t b = a.offsets[f];
    const int32_t e = a.offsets[f + 1];
    const bool ok = !(b < 0 || e < b || e > a.total);
    const int32_t n = ok ? e - b : 0;
    const int2 *P = reinterpret_cast<const int2 *>(a.xy) + b;

    float16v acc[RM][RN];
#pragma unroll
    for (int m = 0; m < RM; ++m)
#pragma unroll
        for (int t = 0; t < RN; ++t)
#pragma unroll
            for (int j = 0; j < 16; ++j) acc[m][t][j] = 0.0f;

    const int r32 = lane & 31;
    const int kq = (lane >> 5) * 8;
    // thread -> (bird k of the chunk, axis); the bird is fetched one chunk ahead
    const int k = tid & (kChunk - 1);
    const bool yaxis = tid < kChunk;
    int2 p = make_int2(0, 0);
    if (k < n) p = P[k];
    for (int32_t k0 = 0; k0 < n; k0 += kChunk) {
        // clear both factor tiles (16-byte stores)
        {
            uint4 *z = reinterpret_cast<uint4 *>(lds);
            constexpr int nz = L::kFactorBytes / 16;
            const uint4 zero = make_uint4(0, 0, 0, 0);
#pragma unroll 4
            for (int i = tid; i < nz; i += kThreads) z[i] = zero;
        }
        const int2 pc = p;
        if (k0 + kChunk + k < n) p = P[k0 + kChunk + k];
        __syncthreads();
        if (k0 + k < n) {
            if (yaxis)
                fill_window(fy + k, (float)pc.y * 0.0625f, g.hy, g.inv_hy, a.grid_h, gy0, L::kRowsY,
                            g.neg_k, g.cut, g.recur_y);
            else
                fill_window(fx + k, (float)pc.x * 0.0625f, g.hx, g.inv_hx, a.grid_w, gx0, L::kRowsX,
                            g.neg_k, g.cut, g.recur_x);
        }
        __syncthreads();
        // this wave's 32 birds of the chunk: two k-steps of 16
#pragma unroll
        for (int ks = 0; ks < 32; ks += 16) {
            const int kk = wave * 32 + ks + kq;
            half8 bx[RN];
#pragma unroll
            for (int t = 0; t < RN; ++t)
                bx[t] = *reinterpret_cast<const half8 *>(fx + (t * 32 + r32) * kPitch + kk);
#pragma unroll
            for (int m = 0; m < RM; ++m) {
                const half8 ay = *reinterpret_cast<const half8 *>(fy + (m * 32 + r32) * kPitch + kk);
#pragma unroll
                for (int t = 0; t < RN; ++t)
                    acc[m][t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ay, bx[t], acc[m][t], 0, 0, 0);
            }
        }
        __syncthreads();
    }

    // Sum the four waves' tiles in a fixed order and store.  Lane l of a wave
    // holds column (l & 31) and rows 8*(j/4) + 4*(l/32) + (j%4), j = 0..15.
    float *red = reinterpret_cast<float *>(lds);
    float *out = a.density + (size_t)f * a.grid_h * a.grid_w;
#pragma unroll
    for (int m = 0; m < RM; ++m) {
#pragma unroll
        for (int t = 0; t < RN; ++t) {
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int row = 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3);
                red[(wave * 32 + row) * 33 + r32] = acc[m][t][j];
            }
            __syncthreads();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int el = tid + i * kThreads;  // 0..1023 over the 32x32 tile
                const int row = el >> 5, colx = el & 31;
                const float s = ((red[row * 33 + colx] + red[(32 + row) * 33 + colx]) +
                                 red[(64 + row) * 33 + colx]) + red[(96 + row) * 33 + colx];
                const int gy = gy0 + m * 32 + row;
                const int gx = gx0 + t * 32 + colx;
                if (ok && gy < a.grid_h && gx < a.grid_w) out[(size_t)gy * a.grid_w + gx] = s * g.scale;
            }
            __syncthreads();
        }
    }
}

template <int RM, int RN>
hipError_t launch_rm_rn(const DensityArgs &a, const Geometry &g, const DensityPlan &p, hipStream_t stream) {
    const long long blocks = (long long)a.n_frames * p.regions_y * p.regions_x;
    hipLaunchKernelGGL((density_kernel<RM, RN>), dim3((unsigned)blocks), dim3(kThreads), 0, stream, a, g,
                       p.regions_y, p.regions_x);
    return hipGetLastError();
}

struct Shape {
    int rm, rn;
};
// instantiated region shapes (tiles of 32 x 32; at most 12 tiles per region)
constexpr Shape kShapes[] = {{1, 1}, {1, 2}, {2, 1}, {2, 2}, {1, 4}, {3, 2},
                             {2, 4}, {3, 4}, {4, 2}, {5, 2}, {4, 1}, {5, 1}};

Geometry make_geometry(const DensityArgs &a) {
    Geometry g;
    const double s = (double)a.sigma_px;
    const double hx = (double)a.width_px / a.grid_w, hy = (double)a.height_px / a.grid_h;
    g.hx = (float)hx;
    g.hy = (float)hy;
    g.inv_hx = (float)(1.0 / hx);
    g.inv_hy = (float)(1.0 / hy);
    g.neg_k = (float)(-1.4426950408889634 / (2.0 * s * s));
    g.cut = (float)(kCutSigmas * s);
    g.scale = (float)(1.0 / (2.0 * 3.14159265358979323846 * s * s));
    g.recur_x = hx <= 2.0 * s;
    g.recur_y = hy <= 2.0 * s;
    return g;
}

}  // namespace

// Choose the output region per workgroup with a small cost model: per bird a
// region costs its matrix-core time (RM*RN/2 cycles), the factor rows its
// windows cover and its tile clearing; workgroups spread over the compute
// units, and a launch never finishes before one workgroup does.
// FLOCK_DENSITY_SHAPE="rm,rn" forces a region shape (for tuning).
DensityPlan plan_density(const DensityArgs &a, int n_cus) {
    const int tiles_y = (a.grid_h + 31) / 32;
    const int tiles_x = (a.grid_w + 31) / 32;
    const char *force = std::getenv("FLOCK_DENSITY_SHAPE");
    if (force) {
        int rm = 0, rn = 0;
        if (std::sscanf(force, "%d,%d", &rm, &rn) == 2)
            for (const Shape &sh : kShapes)
                if (sh.rm == rm && sh.rn == rn)
                    return DensityPlan{rm, rn, (tiles_y + rm - 1) / rm, (tiles_x + rn - 1) / rn};
    }
    const double s = (double)a.sigma_px;
    const double hx = (double)a.width_px / a.grid_w, hy = (double)a.height_px / a.grid_h;
    const double lx = std::min(2.0 * kCutSigmas * s / hx + 1.0, (double)a.grid_w);
    const double ly = std::min(2.0 * kCutSigmas * s / hy + 1.0, (double)a.grid_h);
    const double birds = a.n_frames > 0 ? (double)a.total / a.n_frames : 0.0;
    DensityPlan best{1, 1, tiles_y, tiles_x};
    double best_t = 1e300;
    for (const Shape &sh : kShapes) {
        if (sh.rm > tiles_y && sh.rm > 1) continue;
        if (sh.rn > tiles_x && sh.rn > 1) continue;
        const int ry = (tiles_y + sh.rm - 1) / sh.rm, rx = (tiles_x + sh.rn - 1) / sh.rn;
        const double rows_y = std::min(ly, 32.0 * sh.rm) * std::min(1.0, (32.0 * sh.rm + ly) / (32.0 * tiles_y));
        const double rows_x = std::min(lx, 32.0 * sh.rn) * std::min(1.0, (32.0 * sh.rn + lx) / (32.0 * tiles_x));
        const double per_bird = sh.rm * sh.rn * 0.5 + (rows_x + rows_y) / 11.0 + (sh.rm + sh.rn) * 0.0625 + 0.5;
        const double per_block = birds * per_bird + 2000.0;
        const double blocks = (double)a.n_frames * ry * rx;
        const double t = std::max(blocks * per_block / n_cus, per_block);
        if (t < best_t * 0.999) {
            best_t = t;
            best = DensityPlan{sh.rm, sh.rn, ry, rx};
        }
    }
    return best;
}

hipError_t launch_density(const DensityArgs &a, const DensityPlan &p, size_t lds_limit,
                          hipStream_t stream) {
    (void)lds_limit;
    const Geometry g = make_geometry(a);
#define FLOCK_SHAPE(RM, RN) \
    if (p.rm == RM && p.rn == RN) return launch_rm_rn<RM, RN>(a, g, p, stream);
    FLOCK_SHAPE(1, 1) FLOCK_SHAPE(1, 2) FLOCK_SHAPE(2, 1) FLOCK_SHAPE(2, 2) FLOCK_SHAPE(1, 4)
    FLOCK_SHAPE(3, 2) FLOCK_SHAPE(2, 4) FLOCK_SHAPE(3, 4) FLOCK_SHAPE(4, 2) FLOCK_SHAPE(5, 2)
    FLOCK_SHAPE(4, 1) FLOCK_SHAPE(5, 1)
#undef FLOCK_SHAPE
    return hipErrorInvalidValue;
}

}  // namespace flock

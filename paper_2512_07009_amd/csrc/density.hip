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
// (16 TM) gy rows x (64 TNW) gx columns.  Birds stream through in chunks of
// kChunk: the chunk's factors for the region's rows and columns are written
// to LDS as fp16, then every wave runs v_mfma_f32_16x16x32_f16 over the chunk
// for its own TNW column tiles and all TM row tiles, accumulating in fp32.
//
// Factor generation is windowed: a factor below 2^-25 rounds to +0 in fp16,
// and exp(-t^2/2) < 2^-25 for |t| > 5.9, so each bird only evaluates the
// rows within 6 s of it (plus one row of margin); the rest of the LDS tile is
// cleared to zero.  The fp16 operands are therefore exactly those of the
// dense evaluation, while the contraction itself stays dense over all
// (row, column, bird) triples.
//
// Accuracy: each fp16 factor carries a relative rounding error <= 2^-11, so
// each term of the sum is within about 2^-10 of exact; all terms are positive,
// so the same relative bound holds for every output, which is <= the frame's
// maximum.

#include <cmath>

#include "internal.h"

namespace flock {
namespace {

constexpr int kThreads = 256;   // 4 waves
constexpr int kChunk = 128;     // birds per LDS chunk (2 factor items per thread)
constexpr int kPitch = kChunk + 8;  // halves per LDS row (16-byte skew between rows)
constexpr float kCutSigmas = 6.0f;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));

struct Geometry {
    float inv16;          // 1/16: quanta -> px
    float hx, hy;         // cell size, px
    float inv_hx, inv_hy;
    float neg_k;          // -log2(e) / (2 s^2): exp(-d^2/(2s^2)) = exp2(d^2 * neg_k)
    float cut;            // window half-width, px
    float scale;          // 1 / (2 pi s^2)
};

// Write bird k's factors for LDS rows [row0, row0 + nrows) of one axis into
// buf (row-major, kPitch halves per row); rows outside the window stay 0.
__device__ __forceinline__ void fill_window(_Float16 *buf, int k, float pos_px, float h,
                                            float inv_h, int grid_n, int row0, int nrows,
                                            const Geometry &g) {
    // rows whose centres (r + 1/2) h lie within cut of pos, with one row margin
    int lo = (int)floorf((pos_px - g.cut) * inv_h - 0.5f) - 1;
    int hi = (int)ceilf((pos_px + g.cut) * inv_h - 0.5f) + 1;
    lo = max(lo, row0);
    hi = min(hi, min(row0 + nrows, grid_n) - 1);
    for (int row = lo; row <= hi; ++row) {
        const float c = ((float)row + 0.5f) * h;
        const float d = c - pos_px;
        const float v = __builtin_amdgcn_exp2f(d * d * g.neg_k);
        buf[(row - row0) * kPitch + k] = (_Float16)v;
    }
}

template <int TM, int TNW>
__global__ __launch_bounds__(kThreads) void density_kernel(DensityArgs a, Geometry g, int regions_y,
                                                           int regions_x) {
    constexpr int kRowsY = 16 * TM;          // gy rows of the region
    constexpr int kRowsX = 16 * 4 * TNW;     // gx columns of the region
    __shared__ __align__(16) _Float16 fy[kRowsY * kPitch];
    __shared__ __align__(16) _Float16 fx[kRowsX * kPitch];

    const int regions = regions_y * regions_x;
    const int f = blockIdx.x / regions;
    const int reg = blockIdx.x % regions;
    const int gy0 = (reg / regions_x) * kRowsY;
    const int gx0 = (reg % regions_x) * kRowsX;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    const int32_t b = a.offsets[f];
    const int32_t e = a.offsets[f + 1];
    const bool ok = !(b < 0 || e < b || e > a.total);
    const int32_t n = ok ? e - b : 0;

    float4v acc[TM][TNW];
#pragma unroll
    for (int m = 0; m < TM; ++m)
#pragma unroll
        for (int t = 0; t < TNW; ++t) acc[m][t] = float4v{0.f, 0.f, 0.f, 0.f};

    const int2 *P = reinterpret_cast<const int2 *>(a.xy) + b;
    for (int32_t k0 = 0; k0 < n; k0 += kChunk) {
        // clear both factor tiles (16-byte stores)
        {
            uint4 *zy = reinterpret_cast<uint4 *>(fy);
            uint4 *zx = reinterpret_cast<uint4 *>(fx);
            constexpr int ny = kRowsY * kPitch / 8, nx = kRowsX * kPitch / 8;
            const uint4 z = make_uint4(0, 0, 0, 0);
            for (int i = tid; i < ny; i += kThreads) zy[i] = z;
            for (int i = tid; i < nx; i += kThreads) zx[i] = z;
        }
        __syncthreads();
        // windowed factors: thread -> (bird, axis)
        {
            const int k = tid & (kChunk - 1);
            const int axis = tid / kChunk;  // 0: y rows, 1: x columns
            if (k0 + k < n) {
                const int2 p = P[k0 + k];
                if (axis == 0)
                    fill_window(fy, k, (float)p.y * g.inv16, g.hy, g.inv_hy, a.grid_h, gy0, kRowsY, g);
                else
                    fill_window(fx, k, (float)p.x * g.inv16, g.hx, g.inv_hx, a.grid_w, gx0, kRowsX, g);
            }
        }
        __syncthreads();
        // contraction over the chunk: 4 k-steps of 32 birds
        const int r16 = lane & 15;
        const int kq = (lane >> 4) * 8;
#pragma unroll
        for (int ks = 0; ks < kChunk; ks += 32) {
            half8 bx[TNW];
#pragma unroll
            for (int t = 0; t < TNW; ++t) {
                const int col = (wave * TNW + t) * 16 + r16;
                bx[t] = *reinterpret_cast<const half8 *>(fx + col * kPitch + ks + kq);
            }
#pragma unroll
            for (int m = 0; m < TM; ++m) {
                const half8 ay = *reinterpret_cast<const half8 *>(fy + (m * 16 + r16) * kPitch + ks + kq);
#pragma unroll
                for (int t = 0; t < TNW; ++t)
                    acc[m][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ay, bx[t], acc[m][t], 0, 0, 0);
            }
        }
        __syncthreads();
    }

    if (!ok) return;
    // epilogue: lane holds column gx = tile col + (lane & 15), rows 4*(lane>>4) + j
    float *out = a.density + (size_t)f * a.grid_h * a.grid_w;
#pragma unroll
    for (int m = 0; m < TM; ++m) {
#pragma unroll
        for (int t = 0; t < TNW; ++t) {
            const int gx = gx0 + (wave * TNW + t) * 16 + (lane & 15);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int gy = gy0 + m * 16 + (lane >> 4) * 4 + j;
                if (gx < a.grid_w && gy < a.grid_h) out[(size_t)gy * a.grid_w + gx] = acc[m][t][j] * g.scale;
            }
        }
    }
}

template <int TM, int TNW>
hipError_t launch_tm_tnw(const DensityArgs &a, const Geometry &g, const DensityPlan &p,
                         hipStream_t stream) {
    const long long blocks = (long long)a.n_frames * p.regions_y * p.regions_x;
    hipLaunchKernelGGL((density_kernel<TM, TNW>), dim3((unsigned)blocks), dim3(kThreads), 0, stream, a,
                       g, p.regions_y, p.regions_x);
    return hipGetLastError();
}

template <int TM>
hipError_t launch_tm(const DensityArgs &a, const Geometry &g, const DensityPlan &p, hipStream_t s) {
    switch (p.tnw) {
        case 1: return launch_tm_tnw<TM, 1>(a, g, p, s);
        case 2: return launch_tm_tnw<TM, 2>(a, g, p, s);
        case 4: return launch_tm_tnw<TM, 4>(a, g, p, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

// Choose the output region per workgroup: as large as the register budget
// allows (fewer redundant factor evaluations), split further only while the
// launch would leave compute units idle.
DensityPlan plan_density(const DensityArgs &a, int n_cus) {
    const int tiles_y = (a.grid_h + 15) / 16;
    const int tiles_x = (a.grid_w + 15) / 16;
    static const int kTm[] = {9, 5, 3, 2, 1};
    static const int kTnw[] = {4, 2, 1};
    DensityPlan best{1, 1, tiles_y, (tiles_x + 3) / 4};
    // largest region first; keep the first that gives >= n_cus workgroups,
    // else the one with the most workgroups
    long long best_blocks = -1;
    for (int tnw : kTnw) {
        for (int tm : kTm) {
            if (tm > tiles_y && tm != 1) continue;
            if (4 * tnw > tiles_x && tnw != 1) continue;
            DensityPlan p{tm, tnw, (tiles_y + tm - 1) / tm, (tiles_x + 4 * tnw - 1) / (4 * tnw)};
            const long long blocks = (long long)a.n_frames * p.regions_y * p.regions_x;
            if (blocks >= n_cus) return p;
            if (blocks > best_blocks) {
                best = p;
                best_blocks = blocks;
            }
        }
    }
    return best;
}

hipError_t launch_density(const DensityArgs &a, const DensityPlan &p, hipStream_t stream) {
    Geometry g;
    const double s = (double)a.sigma_px;
    g.inv16 = 1.0f / 16.0f;
    g.hx = (float)((double)a.width_px / a.grid_w);
    g.hy = (float)((double)a.height_px / a.grid_h);
    g.inv_hx = (float)((double)a.grid_w / a.width_px);
    g.inv_hy = (float)((double)a.grid_h / a.height_px);
    g.neg_k = (float)(-1.4426950408889634 / (2.0 * s * s));
    g.cut = (float)(kCutSigmas * s);
    g.scale = (float)(1.0 / (2.0 * 3.14159265358979323846 * s * s));
    switch (p.tm) {
        case 1: return launch_tm<1>(a, g, p, stream);
        case 2: return launch_tm<2>(a, g, p, stream);
        case 3: return launch_tm<3>(a, g, p, stream);
        case 5: return launch_tm<5>(a, g, p, stream);
        case 9: return launch_tm<9>(a, g, p, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace flock

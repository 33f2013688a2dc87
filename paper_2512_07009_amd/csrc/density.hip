// density.hip - Gaussian density grid per frame as a matrix-core contraction
// on gfx950.
//
// The per-frame density of Algorithm 1 (Section 3.6),
//     D[gy][gx] = c * sum_i exp(-((cx - x_i)^2 + (cy - y_i)^2) / (2 s^2)),
//     c = 1 / (2 pi s^2),
// separates into per-axis factors Fy[gy][i] = exp(-(cy - y_i)^2 / (2 s^2)) and
// Fx[gx][i] = exp(-(cx - x_i)^2 / (2 s^2)), so D = c * Fy . Fx^T: a dense
// contraction over the birds of the frame, run on the matrix cores with fp16
// factors and fp32 accumulation.
//
// Factors are stored as fp16 values of 2^8 f (kLift; the largest, 256, is
// far from fp16's limit) and the 2^-16 of the product goes into the output
// scale, so fp16's subnormal range starts at f = 2^-22 (5.5 s from the bird)
// instead of 2^-14 (4.4 s).  A bird has nonzero factors only in the rows
// within about 6 s of it (its window: the tables hold the cells up to
// ceil(6 s / cell) + 1 away, exact zeros beyond); the contraction stays
// dense over all (row, column, bird) triples.
//
// Two ways to make the operands:
//
// Gather path (the cell size c = 16 W / G is a whole number of 1/16-px quanta
// on both axes).  A bird at y = G c + r (0 <= r < c, in quanta) sits at the
// same offset (n + 1/2) c - r from the centre of row G + n for every G, so its
// factors are one row of an exact table indexed by r, built in LDS once per
// workgroup.  Each lane of a wave builds its own v_mfma_f32_16x16x32_f16
// operands from that table (one clamped index, one 32-bit read giving the
// factors of two 16-row tiles), with no tile writes and no barriers; the
// next k-step's operands are gathered while the current one's MFMAs run.
// Waves sharing a frame region add their tiles in a fixed order at the end;
// batches with few (frame, region) pairs also split frames into bird slices
// whose partial grids a second kernel adds in slice order.
//
// Recurrence path (any other grid).  Each workgroup generates its factors
// with a two-multiply recurrence along the window,
//     F(d + h) = F(d) * R(d),   R(d + h) = R(d) * Q,
//     R(d) = exp(-(2 d h + h^2) / (2 s^2)),  Q = exp(-h^2 / s^2),
// started from exact exponentials at both ends of the window (two chains per
// thread) and restarted every kRestart rows; when h > 2 s every factor is an
// exact exponential.
//
// Accuracy: a normal fp16 factor (f >= 2^-22) carries a relative rounding
// error <= 2^-11 (plus a few fp32 ulps before the conversion); a subnormal
// one an absolute error <= 2^-25 of 2^8 f, i.e. 2^-33 of f.  A term is a
// product of two factors <= 1, so its error is <= about 2^-10 of the term plus
// 2^-32 absolute; all terms are positive, so an output's error is <= 2^-10 of
// the output plus N 2^-32 c for N birds (c = 1 / (2 pi s^2)), against an
// output <= the frame's maximum.  The window's cut contributes < 2^-25 per
// factor.  Every sum is taken in a fixed order, so results are
// deterministic.

#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <mutex>

#include "internal.h"

namespace flock {
namespace {

// ---------------------------------------------------------------------------
// Recurrence path
// ---------------------------------------------------------------------------

constexpr int kRThreads = 256;       // 4 waves
constexpr int kRChunk = 128;         // birds per LDS chunk: one (bird, axis) window per thread
constexpr int kRPitch = kRChunk + 8; // halves per LDS row (16-byte skew between rows)
constexpr int kRestart = 16;         // rows between exact restarts of the recurrence
constexpr float kCutSigmas = 6.0f;
constexpr float kLift = 256.0f;      // factors are stored as fp16(kLift f)

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));

struct Geometry {
    float hx, hy;          // cell size, px
    float inv_hx, inv_hy;
    float neg_k;           // -log2(e) / (2 s^2): exp(-d^2/(2s^2)) = exp2(d^2 * neg_k)
    float cut;             // window half-width, px
    float scale;           // 1 / (2 pi s^2 kLift^2)
    int recur_x, recur_y;  // recurrence usable along the axis (h <= 2 s)
};

template <int RM, int RN>
struct RecurLayout {
    static constexpr int kRowsY = 32 * RM;
    static constexpr int kRowsX = 32 * RN;
    static constexpr int kFactorBytes = (kRowsY + kRowsX) * kRPitch * 2;
    static constexpr int kRedBytes = 4 * 32 * 33 * 4;  // one tile from each wave, padded rows
    static constexpr int kBytes = kFactorBytes > kRedBytes ? kFactorBytes : kRedBytes;
};

// Write one bird's factors (times kLift) for rows [row0, row0 + nrows) of one
// axis into a column of buf (row-major, kRPitch halves per row); rows outside
// the window (6 s) are left as they are (cleared): their factors are below
// exp(-18) = 1.5e-8 of the peak.
__device__ __forceinline__ void fill_window(_Float16 *col, float pos, float h, float inv_h, int grid_n,
                                            int row0, int nrows, float neg_k, float cut, bool recur) {
    int lo = max((int)ceilf((pos - cut) * inv_h - 0.5f), row0);
    int hi = min((int)floorf((pos + cut) * inv_h - 0.5f), min(row0 + nrows, grid_n) - 1);
    if (!recur) {
        for (int row = lo; row <= hi; ++row) {
            const float d = ((float)row + 0.5f) * h - pos;
            col[(row - row0) * kRPitch] = (_Float16)(kLift * __builtin_amdgcn_exp2f(d * d * neg_k));
        }
        return;
    }
    const float q = __builtin_amdgcn_exp2f(2.0f * h * h * neg_k);
    // two chains: rows lo.. upward and rows hi.. downward, meeting in the middle
    const int mid = (lo + hi) >> 1;
    for (int base = lo, top = hi; base <= mid; base += kRestart, top -= kRestart) {
        const float da = ((float)base + 0.5f) * h - pos;
        const float db = ((float)top + 0.5f) * h - pos;
        float fa = kLift * __builtin_amdgcn_exp2f(da * da * neg_k);
        float ra = __builtin_amdgcn_exp2f((2.0f * da + h) * h * neg_k);
        float fb = kLift * __builtin_amdgcn_exp2f(db * db * neg_k);
        float rb = __builtin_amdgcn_exp2f((h - 2.0f * db) * h * neg_k);  // ratio going down
        const int steps = min(kRestart, mid - base + 1);
        for (int i = 0; i < steps; ++i) {
            col[(base + i - row0) * kRPitch] = (_Float16)fa;
            if (top - i > mid) col[(top - i - row0) * kRPitch] = (_Float16)fb;
            fa *= ra;
            ra *= q;
            fb *= rb;
            rb *= q;
        }
    }
}

template <int RM, int RN>
__global__ __launch_bounds__(kRThreads) void density_recur_kernel(DensityArgs a, Geometry g, int regions_y,
                                                           int regions_x) {
    using L = RecurLayout<RM, RN>;
    __shared__ __align__(16) unsigned char lds[L::kBytes];
    _Float16 *fy = reinterpret_cast<_Float16 *>(lds);
    _Float16 *fx = fy + L::kRowsY * kRPitch;

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
    const int k = tid & (kRChunk - 1);
    const bool yaxis = tid < kRChunk;
    int2 p = make_int2(0, 0);
    if (k < n) p = P[k];
    for (int32_t k0 = 0; k0 < n; k0 += kRChunk) {
        // clear both factor tiles (16-byte stores)
        {
            uint4 *z = reinterpret_cast<uint4 *>(lds);
            constexpr int nz = L::kFactorBytes / 16;
            const uint4 zero = make_uint4(0, 0, 0, 0);
#pragma unroll 4
            for (int i = tid; i < nz; i += kRThreads) z[i] = zero;
        }
        const int2 pc = p;
        if (k0 + kRChunk + k < n) p = P[k0 + kRChunk + k];
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
                bx[t] = *reinterpret_cast<const half8 *>(fx + (t * 32 + r32) * kRPitch + kk);
#pragma unroll
            for (int m = 0; m < RM; ++m) {
                const half8 ay = *reinterpret_cast<const half8 *>(fy + (m * 32 + r32) * kRPitch + kk);
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
                const int el = tid + i * kRThreads;  // 0..1023 over the 32x32 tile
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


// ---------------------------------------------------------------------------
// Gather path
// ---------------------------------------------------------------------------

constexpr int kGWaves = 8;                 // waves per workgroup (two per SIMD)
constexpr int kGThreads = 64 * kGWaves;
constexpr int kGStep = 32;                 // birds per MFMA k-step (16 x 16 x 32)
constexpr int kGRedTiles = 8;              // 16 x 16 tiles per round of the cross-wave sum
constexpr int kGRing = 128;                // staged birds per wave (one k-step left over + one round)
constexpr int kGMaxTableBytes = 96 * 1024; // both factor tables
constexpr int kGMinWaveBirds = 32;         // kept birds per wave, at least, when a launch splits frames
constexpr int32_t kGFar = 1 << 28;         // bird term that clamps every row to a zero entry

typedef float float4v __attribute__((ext_vector_type(4)));

// Factor table of one axis.  Row r (the bird's offset within its cell, in
// quanta, 0 <= r < c) holds the factors of cells G + n, n = -j .. j, as
// T(i) = f((i - 1 - j + 1/2) c - r) for i = 1 .. 2 j + 1 and T(i) = 0
// elsewhere; its entry i (i = -16 .. PW - 1) is the pair (T(i), T(i + 16)), so
// one 32-bit read gives a bird's factors for two 16-row tiles.
struct GatherAxis {
    int32_t c;      // quanta per cell
    int32_t j;      // window half-width, cells (2 j + 3 <= PW)
    int32_t tab;    // byte offset of the table in LDS
};

struct GatherGeom {
    GatherAxis ay, ax;
    int pw;           // 32 or 64
    float neg_k;      // -log2(e) / (2 s^2), px^-2
    float scale;      // 1 / (2 pi s^2 kLift^2)
    int table_bytes;  // the tables (one when both axes agree), 16-byte aligned
    int lds_bytes;
};

// One bird as a lane reads it: per axis the byte offset of its table row and
// 4 (j + 17 - G), G its cell.
struct GBird {
    int32_t rb_y, g_y, rb_x, g_x;
};

// floor(v / c) for |v| < 2^24, 1 <= c < 2^20: a float reciprocal, then one
// correction step either way.
__device__ __forceinline__ int32_t floor_div(int32_t v, int32_t c, float inv_c) {
    int32_t q = (int32_t)floorf((float)v * inv_c);
    if (q * c > v) --q;
    else if ((q + 1) * c <= v) ++q;
    return q;
}

template <int PW>
__device__ __forceinline__ void stage_axis(int32_t q, const GatherAxis &t, float inv_c, int32_t *rb, int32_t *g) {
    // exact for |q| < 2^24; beyond that the bird is far outside any grid and
    // only the table row needs keeping in range
    const int32_t G = floor_div(q, t.c, inv_c);
    const int32_t r = min(max(q - G * t.c, 0), t.c - 1);
    *rb = t.tab + 4 * (PW + 16) * r;
    *g = 4 * (t.j + 17 - G);
}

// A bird's factor pair for tiles M and M + 1 (M even) of a lane: with
// v = 4 (R0 + (lane & 15)) + 4 (j + 17 - G), the entry's byte offset in the
// bird's row is clamp(v + 64 M, 0, 4 (PW + 15)) (16 rows of 4 bytes per
// tile).  An index clamped from below or above holds two zeros, as do the
// true factors there, so the clamp is exact.  Constant bounds make it one
// v_med3, and the 64 M goes into the read's offset field.
template <int M, int PW>
__device__ __forceinline__ uint32_t factor_pair(const unsigned char *lds, int32_t rb, int32_t v) {
    const int32_t o = min(max(v, -64 * M), 4 * (PW + 15) - 64 * M);
    return *reinterpret_cast<const uint32_t *>(lds + rb + o + 64 * M);
}

// Operands of tiles M and M + 1 from the pairs of eight birds.
template <int M, int PW>
__device__ __forceinline__ void operands(half8 &lo, half8 &hi, const int32_t (&rb)[8], const int32_t (&v)[8],
                                         const unsigned char *lds) {
    uint32_t w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) w[e] = factor_pair<M, PW>(lds, rb[e], v[e]);
    uint32_t l4[4], h4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        l4[e] = __builtin_amdgcn_perm(w[2 * e + 1], w[2 * e], 0x05040100u);  // low halves: tile M
        h4[e] = __builtin_amdgcn_perm(w[2 * e + 1], w[2 * e], 0x07060302u);  // high halves: tile M + 1
    }
    lo = __builtin_bit_cast(half8, l4);
    hi = __builtin_bit_cast(half8, h4);
}

template <int TN, int PW, int N = 0>
__device__ __forceinline__ void operands_x(half8 (&bx)[TN], const int32_t (&rb)[8], const int32_t (&v)[8],
                                           const unsigned char *lds) {
    if constexpr (N < TN) {
        half8 hi;
        operands<N, PW>(bx[N], hi, rb, v, lds);
        if constexpr (N + 1 < TN) bx[N + 1] = hi;
        operands_x<TN, PW, N + 2>(bx, rb, v, lds);
    }
}

template <int TM, int TN, int PW, int M = 0>
__device__ __forceinline__ void contract_y(float4v (&acc)[TM][TN], const half8 (&bx)[TN], const int32_t (&rb)[8],
                                           const int32_t (&v)[8], const unsigned char *lds) {
    if constexpr (M < TM) {
        half8 a0, a1;
        operands<M, PW>(a0, a1, rb, v, lds);
#pragma unroll
        for (int n = 0; n < TN; ++n) acc[M][n] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, bx[n], acc[M][n], 0, 0, 0);
        if constexpr (M + 1 < TM) {
#pragma unroll
            for (int n = 0; n < TN; ++n)
                acc[M + 1][n] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, bx[n], acc[M + 1][n], 0, 0, 0);
        }
        contract_y<TM, TN, PW, M + 2>(acc, bx, rb, v, lds);
    }
}

// A work item is (frame, output region of 16 TM rows x 16 TN columns, slice
// of the frame's birds); `waves` waves of a workgroup share an item, and
// their tiles are added in a fixed order at the end (deterministic).  With
// split > 1 the slices' grids go to `partial` for a second kernel to add.
// The slices and waves of a (frame, region) take the frame's 64-bird blocks
// in turn (a fixed assignment).
//
// Only birds whose window of cells (G - j .. G + j on both axes) meets the
// region contribute to it: every other bird's factors there are table zeros.
// Each wave reads its blocks one at a time (one bird per lane), keeps the ones that
// meet the region, in input order, in a ring of staged birds in LDS (ballot
// ranks), and runs a k-step whenever 32 are staged; the last step is padded
// with birds whose factors are all zero.  No barrier is needed until the
// final sum.
template <int TM, int TN, int PW>
__global__ __launch_bounds__(kGThreads) __attribute__((amdgpu_waves_per_eu(2))) void density_gather_kernel(DensityArgs a, GatherGeom gg, int regions_y,
                                                                   int regions_x, int split, int waves,
                                                                   long long items, float *partial) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    // this wave's item and its part of the item's birds
    const int per_wg = kGWaves / waves;
    const long long item = (long long)blockIdx.x * per_wg + wave / waves;
    const int part = wave % waves;
    const bool active = item < items;
    const int regions = regions_y * regions_x;
    int f = 0, reg = 0, sl = 0;
    if (active) {
        sl = (int)(item % split);
        const long long fr = item / split;
        reg = (int)(fr % regions);
        f = (int)(fr / regions);
    }
    const int row0 = (reg / regions_x) * 16 * TM;
    const int col0 = (reg % regions_x) * 16 * TN;
    int32_t b = 0, n = 0;
    if (active) {
        b = a.offsets[f];
        const int32_t e = a.offsets[f + 1];
        n = (b < 0 || e < b || e > a.total) ? 0 : e - b;
    }
    // the split * waves (slice, part) units of a (frame, region) take the
    // frame's 64-bird blocks in turn: unit u = sl * waves + part reads blocks
    // u, u + split * waves, ...  Spatially grouped birds in the input then
    // spread over all units instead of loading one of them.
    const int32_t stride = 64 * split * waves;
    const int2 *P = reinterpret_cast<const int2 *>(a.xy) + b;

    GBird *ring = reinterpret_cast<GBird *>(lds + gg.table_bytes) + wave * kGRing;
    const float inv_cy = 1.0f / (float)gg.ay.c, inv_cx = 1.0f / (float)gg.ax.c;
    const int r16 = lane & 15, grp = lane >> 4;
    const int32_t yoff = 4 * (row0 + r16), xoff = 4 * (col0 + r16);
    // a bird in cell G meets rows [row0, row0 + 16 TM) when
    // row0 - j <= G <= row0 + 16 TM - 1 + j, i.e. when its staged
    // g = 4 (j + 17 - G) lies in [4 (17 - 16 TM + 1 - row0), 4 (2 j + 17 - row0)]
    const int32_t gy_lo = 4 * (18 - 16 * TM - row0), gy_hi = 4 * (2 * gg.ay.j + 17 - row0);
    const int32_t gx_lo = 4 * (18 - 16 * TN - col0), gx_hi = 4 * (2 * gg.ax.j + 17 - col0);

    float4v acc[TM][TN];
#pragma unroll
    for (int m = 0; m < TM; ++m)
#pragma unroll
        for (int t = 0; t < TN; ++t) acc[m][t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};

    // the first round's coordinates are in flight while the tables are built
    int2 qn = make_int2(0, 0);
    int32_t next = 64 * (sl * waves + part);  // first bird of the next round
    if (next + lane < n) qn = P[next + lane];
    // the factor tables (exact: every distance is a multiple of 1/32 px).  A
    // row's PW factors come in PW / 16 chunks of 16, one per thread, the
    // threads of a row in adjacent lanes.  Entries -16 .. PW - 1 of a row form
    // PW / 16 + 1 blocks of 16; block b pairs chunk b - 1 (low halves) with
    // chunk b (high halves), chunks -1 and PW / 16 being zeros.  The thread of
    // chunk k writes block k + 1 with its right neighbour's chunk, and the
    // thread of chunk 0 also writes block 0.
    auto build = [&](const GatherAxis &t) {
        constexpr int kCh = PW / 16;
        const int k = tid % kCh;
        for (int r0 = 0; r0 < t.c; r0 += kGThreads / kCh) {  // uniform over the workgroup
            const int r = r0 + tid / kCh;
            uint32_t mine[8];  // factors 16 k + 2 q (low half) and 16 k + 2 q + 1 (high half)
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                uint32_t h[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int i = 16 * k + 2 * q + u;
                    float f = 0.0f;
                    if (i >= 1 && i <= 2 * t.j + 1) {
                        const float d = (((float)(i - 1 - t.j) + 0.5f) * (float)t.c - (float)r) * 0.0625f;
                        f = kLift * __builtin_amdgcn_exp2f(d * d * gg.neg_k);
                    }
                    h[u] = __builtin_bit_cast(uint16_t, (_Float16)f);
                }
                mine[q] = h[0] | (h[1] << 16);
            }
            uint32_t right[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const uint32_t v = (uint32_t)__shfl_down((int)mine[q], 1, 64);
                right[q] = k + 1 < kCh ? v : 0u;
            }
            if (r < t.c) {
                uint4 *row = reinterpret_cast<uint4 *>(lds + t.tab + r * (PW + 16) * 4);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    // entries 16 k + 4 q .. + 3 of block k + 1: (mine, right) pairs
                    row[4 * (k + 1) + q] = make_uint4(__builtin_amdgcn_perm(right[2 * q], mine[2 * q], 0x05040100u),
                                                      __builtin_amdgcn_perm(right[2 * q], mine[2 * q], 0x07060302u),
                                                      __builtin_amdgcn_perm(right[2 * q + 1], mine[2 * q + 1], 0x05040100u),
                                                      __builtin_amdgcn_perm(right[2 * q + 1], mine[2 * q + 1], 0x07060302u));
                }
                if (k == 0) {
#pragma unroll
                    for (int q = 0; q < 4; ++q)  // block 0: (0, chunk 0)
                        row[q] = make_uint4(mine[2 * q] << 16, mine[2 * q] & 0xffff0000u, mine[2 * q + 1] << 16,
                                            mine[2 * q + 1] & 0xffff0000u);
                }
            }
        }
    };
    build(gg.ay);
    if (gg.ax.tab != gg.ay.tab) build(gg.ax);
    __syncthreads();  // tables written

    // a wave's LDS accesses stay in program order; the fences keep the
    // compiler from moving them across the ring's writes and reads
    auto wave_sync = [] {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };
    const uint64_t below = (1ull << lane) - 1ull;
    int32_t head = 0, tail = 0;  // ring positions, taken modulo kGRing
    // stage rounds of 64 birds until a k-step's worth meets the region (or
    // the birds run out); the last, partial step is filled with birds whose
    // factors are all zero
    auto fill = [&] {
        while (tail - head < kGStep && next < n) {
            const int2 q = qn;
            const bool have = next + lane < n;
            next += stride;
            if (next + lane < n) qn = P[next + lane];  // the following round in flight
            GBird gb{gg.ay.tab, kGFar, gg.ax.tab, kGFar};
            bool keep = false;
            if (have) {
                stage_axis<PW>(q.y, gg.ay, inv_cy, &gb.rb_y, &gb.g_y);
                stage_axis<PW>(q.x, gg.ax, inv_cx, &gb.rb_x, &gb.g_x);
                keep = (gb.g_y >= gy_lo) & (gb.g_y <= gy_hi) & (gb.g_x >= gx_lo) & (gb.g_x <= gx_hi);
            }
            const uint64_t m = __ballot(keep);
            if (keep) ring[(tail + __popcll(m & below)) & (kGRing - 1)] = gb;
            tail += __popcll(m);
        }
        if (tail > head && tail - head < kGStep) {
            if (lane < kGStep && head + lane >= tail)
                ring[(head + lane) & (kGRing - 1)] = GBird{gg.ay.tab, kGFar, gg.ax.tab, kGFar};
            tail = head + kGStep;
        }
        wave_sync();
    };
    fill();
    while (tail > head) {  // wave-uniform
        const GBird *sb = ring + (head & (kGRing - 1)) + 8 * grp;  // this lane's eight birds of the step
        half8 bx[TN];
        {
            int32_t rbx[8], vx[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int2 q = reinterpret_cast<const int2 *>(sb + e)[1];
                rbx[e] = q.x;
                vx[e] = q.y + xoff;
            }
            operands_x<TN, PW>(bx, rbx, vx, lds);
        }
        int32_t rby[8], vy[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int2 q = reinterpret_cast<const int2 *>(sb + e)[0];
            rby[e] = q.x;
            vy[e] = q.y + yoff;
        }
        contract_y<TM, TN, PW>(acc, bx, rby, vy, lds);
        head += kGStep;
        wave_sync();  // the step's reads are done before the ring is written again
        fill();
    }

    const size_t cells = (size_t)a.grid_h * a.grid_w;
    float *out = split > 1 ? partial + ((size_t)f * split + sl) * cells : a.density + (size_t)f * cells;
    const float scale = split > 1 ? 1.0f : gg.scale;
    if (waves == 1) {
        // lane l holds rows 4 (l / 16) + i, column l % 16 of every tile
        if (!active) return;
#pragma unroll
        for (int m = 0; m < TM; ++m)
#pragma unroll
            for (int t = 0; t < TN; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int gy = row0 + 16 * m + 4 * grp + i, gx = col0 + 16 * t + r16;
                    if (gy < a.grid_h && gx < a.grid_w) out[(size_t)gy * a.grid_w + gx] = acc[m][t][i] * scale;
                }
        return;
    }

    // the waves of an item add their tiles in wave order, kGRedTiles at a time
    __syncthreads();  // tables and staging are done with: the space holds the tiles
    float *red = reinterpret_cast<float *>(lds);
    const int w0 = (wave / waves) * waves;
    const int gt = part * 64 + lane;
#pragma unroll
    for (int t0 = 0; t0 < TM * TN; t0 += kGRedTiles) {
#pragma unroll
        for (int q = 0; q < kGRedTiles; ++q) {
            const int t = t0 + q;
            if (t >= TM * TN) break;
#pragma unroll
            for (int i = 0; i < 4; ++i) red[(wave * kGRedTiles + q) * 256 + (4 * grp + i) * 16 + r16] = acc[t / TN][t % TN][i];
        }
        __syncthreads();
        const int nt = min(kGRedTiles, TM * TN - t0);
        for (int el = gt; el < nt * 256; el += 64 * waves) {
            const int q = el >> 8, within = el & 255;
            float v = 0.0f;
            for (int w = 0; w < waves; ++w) v += red[((w0 + w) * kGRedTiles + q) * 256 + within];
            const int t = t0 + q;
            const int gy = row0 + 16 * (t / TN) + (within >> 4), gx = col0 + 16 * (t % TN) + (within & 15);
            if (active && gy < a.grid_h && gx < a.grid_w) out[(size_t)gy * a.grid_w + gx] = v * scale;
        }
        __syncthreads();
    }
}

// density[f][cell] = scale * sum over slices s = 0, 1, ... of partial[f][s][cell].
__global__ __launch_bounds__(256) void density_reduce_kernel(float *density, const float *partial,
                                                             int64_t cells, int64_t total, int split,
                                                             float scale) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        const int64_t f = i / cells, c = i - f * cells;
        const float *src = partial + f * split * cells + c;
        // slices in order, eight loads in flight at a time (a missing slice
        // adds +0, which leaves the non-negative sum unchanged)
        float s = 0.0f;
        for (int k0 = 0; k0 < split; k0 += 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = k0 + u < split ? src[(int64_t)(k0 + u) * cells] : 0.0f;
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        density[i] = s * scale;
    }
}

template <int RM, int RN>
hipError_t launch_recur(const DensityArgs &a, const Geometry &g, const DensityPlan &p, hipStream_t stream) {
    const long long blocks = (long long)a.n_frames * p.regions_y * p.regions_x;
    hipLaunchKernelGGL((density_recur_kernel<RM, RN>), dim3((unsigned)blocks), dim3(kRThreads), 0, stream, a, g,
                       p.regions_y, p.regions_x);
    return hipGetLastError();
}

struct Shape {
    int rm, rn;
};
// instantiated region shapes of the recurrence path (tiles of 32 x 32; at
// most 12 tiles per region)
constexpr Shape kShapes[] = {{1, 1}, {1, 2}, {2, 1}, {2, 2}, {1, 4}, {3, 2},
                             {2, 4}, {3, 4}, {4, 2}, {5, 2}, {4, 1}, {5, 1}};
// instantiated region shapes of the gather path (tiles of 16 x 16; at most 36
// tiles per region, so that the accumulators and operands fit the registers
// of two waves per SIMD without spilling)
constexpr Shape kGShapes[] = {{1, 1}, {2, 2}, {1, 4}, {4, 1}, {2, 4}, {4, 2}, {3, 4},
                              {4, 4}, {5, 4}, {9, 2}, {9, 4}, {3, 8}, {4, 8}};

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
    g.scale = (float)(1.0 / (2.0 * 3.14159265358979323846 * s * s) / ((double)kLift * kLift));
    g.recur_x = hx <= 2.0 * s;
    g.recur_y = hy <= 2.0 * s;
    return g;
}

// Factor-table geometry of the gather path; false when it does not apply (a
// cell is not a whole number of quanta, or the tables exceed their budget).
bool make_gather_geom(const DensityArgs &a, GatherGeom *gg) {
    if ((16LL * a.height_px) % a.grid_h != 0 || (16LL * a.width_px) % a.grid_w != 0) return false;
    const double cut_q = 16.0 * kCutSigmas * (double)a.sigma_px;  // window half-width, quanta
    auto axis = [&](int64_t c, GatherAxis *t) {
        if (c < 1 || c > (1 << 20)) return false;
        // cells G + n with |n| <= j cover every cell centre within cut_q of the bird
        const double jd = std::ceil(cut_q / (double)c) + 1.0;
        if (jd > 64.0) return false;
        t->c = (int32_t)c;
        t->j = (int32_t)jd;
        return true;
    };
    if (!axis(16LL * a.height_px / a.grid_h, &gg->ay) || !axis(16LL * a.width_px / a.grid_w, &gg->ax)) return false;
    const int jmax = std::max(gg->ay.j, gg->ax.j);
    if (2 * jmax + 3 <= 32) gg->pw = 32;
    else if (2 * jmax + 3 <= 64) gg->pw = 64;
    else return false;
    auto bytes16 = [](int64_t pairs) { return (pairs * 4 + 15) / 16 * 16; };
    const int64_t ty = bytes16((int64_t)gg->ay.c * (gg->pw + 16));
    const bool shared = gg->ay.c == gg->ax.c && gg->ay.j == gg->ax.j;
    const int64_t tx = shared ? 0 : bytes16((int64_t)gg->ax.c * (gg->pw + 16));
    if (ty + tx > kGMaxTableBytes) return false;
    gg->ay.tab = 0;
    gg->ax.tab = shared ? 0 : (int32_t)ty;
    gg->table_bytes = (int)(ty + tx);
    const int stage = kGWaves * kGRing * (int)sizeof(GBird);
    gg->lds_bytes = std::max(gg->table_bytes + stage, kGWaves * kGRedTiles * 256 * 4);
    const double s = (double)a.sigma_px;
    gg->neg_k = (float)(-1.4426950408889634 / (2.0 * s * s));
    gg->scale = (float)(1.0 / (2.0 * 3.14159265358979323846 * s * s) / ((double)kLift * kLift));
    return true;
}

long long shape_regions(const Shape &sh, int tile, int grid_w, int grid_h) {
    return ((grid_h + (long long)tile * sh.rm - 1) / ((long long)tile * sh.rm)) *
           ((grid_w + (long long)tile * sh.rn - 1) / ((long long)tile * sh.rn));
}

// Share of a frame's birds whose window of 2 j + 1 cells meets one region
// of `rows` grid rows, `nreg` regions along the axis: about 1 + 2 j / rows
// regions per bird, at most all of them.
double meet_share(int j, int rows, long long nreg) {
    return std::min((double)nreg, 1.0 + 2.0 * j / rows) / (double)nreg;
}

long long axis_regions(int grid_n, int rows) { return (grid_n + rows - 1) / rows; }

// Modelled SIMD cycles of one 32-bird k-step on a region: per lane a pair
// read (read, clamp, address, pack: about 112 cycles for its eight birds)
// for every two tile rows of each axis, and one 16-cycle MFMA per tile.
double step_cycles(const Shape &sh) { return 112.0 * ((sh.rm + 1) / 2 + (sh.rn + 1) / 2) + 16.0 * sh.rm * sh.rn; }

// Gather-path region shape of least modelled cost per frame: each bird's
// k-step share on every region its window meets, the test that keeps or
// drops every bird on every region (about 3 cycles a bird), and a fixed cost
// per region (tables, the final sum and the stores).
Shape gather_shape(int jy, int jx, int grid_w, int grid_h, double birds, int max_tiles = 1 << 30) {
    Shape best = kGShapes[0];
    double best_cost = 1e300;
    for (const Shape &sh : kGShapes) {
        if (sh.rm * sh.rn > max_tiles) continue;
        const long long ry = axis_regions(grid_h, 16 * sh.rm), rx = axis_regions(grid_w, 16 * sh.rn);
        const double meets = ry * meet_share(jy, 16 * sh.rm, ry) * rx * meet_share(jx, 16 * sh.rn, rx);
        const double cost = birds / kGStep * meets * step_cycles(sh) + (3.2 * birds + 4000.0) * (double)(ry * rx);
        if (cost < best_cost * 0.999) {
            best = sh;
            best_cost = cost;
        }
    }
    return best;
}

int env_int(const char *name) {
    const char *v = std::getenv(name);
    return v ? std::atoi(v) : 0;
}

// Waves per work item and slices per (frame, region) of a gather launch.  A
// compute unit holds kGWaves waves (two per SIMD).  Items are spread over
// as few waves as fill the chip (the smallest power of two w, at most
// kGWaves, with items * w >= resident waves): more waves per item only add
// fixed costs (a table build per workgroup, the final sum across waves).
// `birds` is the birds an item keeps (those whose window meets its region),
// on average.  FLOCK_DENSITY_WAVES / FLOCK_DENSITY_SPLIT override (for
// tuning and tests).
void gather_split(int32_t n_frames, double birds, long long regions, int n_cus, int *waves, int *split) {
    const long long items = (long long)n_frames * regions;
    const long long resident = (long long)kGWaves * std::max(n_cus, 1);
    int w = 1;
    while (w < kGWaves && items * w < resident) w *= 2;
    // slices only while one launch would leave most of the chip idle (the
    // partial grids cost traffic), up to one round of waves, with at least
    // kGMinWaveBirds kept birds per wave
    long long sp = 1;
    if (2 * items * w < resident) {
        sp = resident / (items * w);
        sp = std::min<long long>(sp, std::max<long long>(1, (long long)(birds / (w * kGMinWaveBirds))));
        sp = std::min<long long>(sp, 64);
    }
    const int fw = env_int("FLOCK_DENSITY_WAVES"), fs = env_int("FLOCK_DENSITY_SPLIT");
    if (fw == 1 || fw == 2 || fw == 4 || fw == 8) w = fw;
    if (fs >= 1 && fs <= 64) sp = fs;
    *waves = w;
    *split = (int)sp;
}

// Scratch of the allocation-free entry point (density_frames_noalloc): the
// partial grids of split launches, in a file-scope device array instead of a
// workspace.  Each device holds its own copy for the life of the process.
// In host code `scratch` names a host-side stand-in, never the device memory:
// its device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[kDensityScratchBytes];

constexpr int kScratchDevices = 64;
std::once_flag g_scratch_once[kScratchDevices];
void *g_scratch_ptr[kScratchDevices];
hipError_t g_scratch_err[kScratchDevices];

}  // namespace

hipError_t density_static_scratch(void **ptr) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
    std::call_once(g_scratch_once[dev], [dev] {
        void *p = nullptr;
        g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? p : nullptr;
    });
    *ptr = g_scratch_ptr[dev];
    return g_scratch_err[dev];
}

size_t density_workspace_bytes(int32_t n_frames, int32_t total, int32_t grid_w, int32_t grid_h, int n_cus) {
    if (n_frames <= 0 || grid_w < 1 || grid_h < 1) return 0;
    // the shape depends on the frame extent and sigma, which the query does
    // not know: bound the split over every shape, with every bird kept (a
    // split only shrinks when an item keeps fewer birds)
    const double birds = (double)total / n_frames;
    int most = 1;
    for (const Shape &sh : kGShapes) {
        int waves = 1, split = 1;
        gather_split(n_frames, birds, shape_regions(sh, 16, grid_w, grid_h), n_cus, &waves, &split);
        most = std::max(most, split);
    }
    if (most <= 1) return 0;
    return (size_t)n_frames * most * (size_t)grid_w * grid_h * sizeof(float);
}

// Gather path whenever its tables apply; otherwise the recurrence path, whose
// region per workgroup comes from a small cost model: per bird a region costs
// its matrix-core time (RM*RN/2 cycles), the factor rows its windows cover and
// its tile clearing; workgroups spread over the compute units, and a launch
// never finishes before one workgroup does.
// FLOCK_DENSITY_PATH="recur" forces the recurrence path and
// FLOCK_DENSITY_SHAPE="rm,rn" its region shape (for tuning).
DensityPlan plan_density(const DensityArgs &a, int n_cus, size_t lds_limit) {
    const int tiles_y = (a.grid_h + 31) / 32;
    const int tiles_x = (a.grid_w + 31) / 32;
    const char *force = std::getenv("FLOCK_DENSITY_SHAPE");
    const char *path = std::getenv("FLOCK_DENSITY_PATH");
    const bool force_recur = path && std::strcmp(path, "recur") == 0;
    GatherGeom gg;
    if (!force_recur && make_gather_geom(a, &gg) && (size_t)gg.lds_bytes <= lds_limit) {
        const double birds = a.n_frames > 0 ? (double)a.total / a.n_frames : 0.0;
        Shape sh = gather_shape(gg.ay.j, gg.ax.j, a.grid_w, a.grid_h, birds);
        int grm = 0, grn = 0;
        if (force && std::sscanf(force, "%d,%d", &grm, &grn) == 2)
            for (const Shape &k : kGShapes)
                if (k.rm == grm && k.rn == grn) sh = k;
        DensityPlan p{};
        p.gather = 1;
        p.rm = sh.rm;
        p.rn = sh.rn;
        p.regions_y = (a.grid_h + 16 * sh.rm - 1) / (16 * sh.rm);
        p.regions_x = (a.grid_w + 16 * sh.rn - 1) / (16 * sh.rn);
        const double kept = birds * meet_share(gg.ay.j, 16 * sh.rm, p.regions_y) *
                            meet_share(gg.ax.j, 16 * sh.rn, p.regions_x);
        gather_split(a.n_frames, kept, (long long)p.regions_y * p.regions_x, n_cus, &p.waves, &p.split);
        if (p.split > 1 && !(force && grm)) {
            // few frames for the chip: the launch is bound by each wave's own
            // path, whose fixed part grows with the tiles an item's waves add
            // up at the end (kGRedTiles per round); shapes of at most 16 tiles
            // keep that to two rounds
            sh = gather_shape(gg.ay.j, gg.ax.j, a.grid_w, a.grid_h, birds, 16);
            p.rm = sh.rm;
            p.rn = sh.rn;
            p.regions_y = (a.grid_h + 16 * sh.rm - 1) / (16 * sh.rm);
            p.regions_x = (a.grid_w + 16 * sh.rn - 1) / (16 * sh.rn);
            const double kept2 = birds * meet_share(gg.ay.j, 16 * sh.rm, p.regions_y) *
                                 meet_share(gg.ax.j, 16 * sh.rn, p.regions_x);
            gather_split(a.n_frames, kept2, (long long)p.regions_y * p.regions_x, n_cus, &p.waves, &p.split);
        }
        const long long items = (long long)a.n_frames * p.regions_y * p.regions_x * p.split;
        const int per_wg = kGWaves / p.waves;
        p.blocks = (items + per_wg - 1) / per_wg;
        return p;
    }
    int frm = 0, frn = 0;
    if (force && std::sscanf(force, "%d,%d", &frm, &frn) == 2) {
        bool known = false;
        for (const Shape &sh : kShapes) known |= sh.rm == frm && sh.rn == frn;
        if (!known) frm = frn = 0;
    }
    DensityPlan best{};
    best.rm = best.rn = 1;
    best.split = best.waves = 1;
    if (frm) {
        best.rm = frm;
        best.rn = frn;
        best.regions_y = (tiles_y + frm - 1) / frm;
        best.regions_x = (tiles_x + frn - 1) / frn;
        best.blocks = (long long)a.n_frames * best.regions_y * best.regions_x;
        return best;
    }
    const double s = (double)a.sigma_px;
    const double hx = (double)a.width_px / a.grid_w, hy = (double)a.height_px / a.grid_h;
    const double lx = std::min(2.0 * kCutSigmas * s / hx + 1.0, (double)a.grid_w);
    const double ly = std::min(2.0 * kCutSigmas * s / hy + 1.0, (double)a.grid_h);
    const double birds = a.n_frames > 0 ? (double)a.total / a.n_frames : 0.0;
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
            best.rm = sh.rm;
            best.rn = sh.rn;
            best.regions_y = ry;
            best.regions_x = rx;
        }
    }
    if (best.regions_y == 0) {
        best.regions_y = tiles_y;
        best.regions_x = tiles_x;
    }
    best.blocks = (long long)a.n_frames * best.regions_y * best.regions_x;
    return best;
}

hipError_t launch_density(const DensityArgs &a, const DensityPlan &p, float *partial, hipStream_t stream) {
    hipError_t err = hipErrorInvalidValue;
    if (p.gather) {
        GatherGeom gg;
        if (!make_gather_geom(a, &gg)) return hipErrorInvalidValue;
        if (p.split > 1 && !partial) return hipErrorInvalidValue;
        const long long items = (long long)a.n_frames * p.regions_y * p.regions_x * p.split;
#define FLOCK_GSHAPE_PW(TM, TN, PW)                                                                              \
    if (p.rm == TM && p.rn == TN && gg.pw == PW) {                                                               \
        hipLaunchKernelGGL((density_gather_kernel<TM, TN, PW>), dim3((unsigned)p.blocks), dim3(kGThreads),      \
                           (size_t)gg.lds_bytes, stream, a, gg, p.regions_y, p.regions_x, p.split, p.waves, items, \
                           partial);                                                                             \
        err = hipGetLastError();                                                                                 \
    }
#define FLOCK_GSHAPE(TM, TN) FLOCK_GSHAPE_PW(TM, TN, 32) FLOCK_GSHAPE_PW(TM, TN, 64)
        FLOCK_GSHAPE(1, 1) FLOCK_GSHAPE(2, 2) FLOCK_GSHAPE(1, 4) FLOCK_GSHAPE(4, 1) FLOCK_GSHAPE(2, 4)
        FLOCK_GSHAPE(4, 2) FLOCK_GSHAPE(3, 4) FLOCK_GSHAPE(4, 4) FLOCK_GSHAPE(5, 4)
        FLOCK_GSHAPE(9, 2) FLOCK_GSHAPE(9, 4) FLOCK_GSHAPE(3, 8) FLOCK_GSHAPE(4, 8)
#undef FLOCK_GSHAPE
#undef FLOCK_GSHAPE_PW
        if (err != hipSuccess || p.split <= 1) return err;
        const int64_t cells = (int64_t)a.grid_h * a.grid_w;
        const int64_t total = cells * a.n_frames;
        const unsigned blocks = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
        hipLaunchKernelGGL(density_reduce_kernel, dim3(blocks), dim3(256), 0, stream, a.density, partial, cells,
                           total, p.split, gg.scale);
        return hipGetLastError();
    }
    const Geometry g = make_geometry(a);
#define FLOCK_SHAPE(RM, RN) \
    if (p.rm == RM && p.rn == RN) return launch_recur<RM, RN>(a, g, p, stream);
    FLOCK_SHAPE(1, 1) FLOCK_SHAPE(1, 2) FLOCK_SHAPE(2, 1) FLOCK_SHAPE(2, 2) FLOCK_SHAPE(1, 4)
    FLOCK_SHAPE(3, 2) FLOCK_SHAPE(2, 4) FLOCK_SHAPE(3, 4) FLOCK_SHAPE(4, 2) FLOCK_SHAPE(5, 2)
    FLOCK_SHAPE(4, 1) FLOCK_SHAPE(5, 1)
#undef FLOCK_SHAPE
    return err;
}

}  // namespace flock

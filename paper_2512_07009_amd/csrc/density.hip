// density.hip - Gaussian density grid per frame as a matrix-core contraction
// on gfx950.
//
// The per-frame density of Algorithm 1 (Section 3.6),
//     D[gy][gx] = c * sum_i exp(-((cx - x_i)^2 + (cy - y_i)^2) / (2 s^2)),
//     c = 1 / (2 pi s^2),
// separates into per-axis factors Fy[gy][i] = exp(-(cy - y_i)^2 / (2 s^2)) and
// Fx[gx][i] = exp(-(cx - x_i)^2 / (2 s^2)), so D = c * Fy . Fx^T: a dense
// contraction over the birds of the frame, run on v_mfma_f32_32x32x16_f16
// with fp16 factors and fp32 accumulation.
//
// A factor below 2^-25 rounds to +0 in fp16, and exp(-t^2/2) < 2^-25 for
// |t| > 5.9, so a bird has nonzero factors only in the rows within 6 s of it
// (its window); every other factor is +0 in either evaluation, and the
// contraction stays dense over all (row, column, bird) triples.
//
// Two ways to make the factor tiles:
//
// Table path (the cell size c = 16 W / G is a whole number of 1/16-px quanta
// on both axes).  A bird at y = G c + r (0 <= r < c, in quanta) sits at the
// same offset r - c/2 - j c from the centre of row G + j for every G, so its
// window is one row of an exact table T[r][j], built once per workgroup.
// Each of the eight waves of a workgroup works on its own: it copies the
// windows of 16 birds from the table into private factor tiles (a halo of
// one window height above and below the output rows takes the windows of
// birds near or past the region's edge without clipping), then runs one MFMA
// k-step over them; the copy of the next 16 birds overlaps that contraction.
// Workgroups of few-frame batches each take a slice of a frame's birds; a
// second kernel adds the slices' partial grids in slice order.
//
// Recurrence path (any other grid).  Each workgroup generates its factors
// with a two-multiply recurrence along the window,
//     F(d + h) = F(d) * R(d),   R(d + h) = R(d) * Q,
//     R(d) = exp(-(2 d h + h^2) / (2 s^2)),  Q = exp(-h^2 / s^2),
// started from exact exponentials at both ends of the window (two chains per
// thread) and restarted every kRestart rows; when h > 2 s every factor is an
// exact exponential.
//
// Accuracy: each fp16 factor carries a relative rounding error <= 2^-11 (plus
// at most a few fp32 ulps before the conversion), so each term of the sum is
// within about 2^-10 of exact; all terms are positive, so the same relative
// bound holds for every output, which is <= the frame's maximum.  Every sum
// is taken in a fixed order, so results are deterministic.

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>

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
struct RecurLayout {
    static constexpr int kRowsY = 32 * RM;
    static constexpr int kRowsX = 32 * RN;
    static constexpr int kFactorBytes = (kRowsY + kRowsX) * kRPitch * 2;
    static constexpr int kRedBytes = 4 * 32 * 33 * 4;  // one tile from each wave, padded rows
    static constexpr int kBytes = kFactorBytes > kRedBytes ? kFactorBytes : kRedBytes;
};

// Write one bird's factors for rows [row0, row0 + nrows) of one axis into a
// column of buf (row-major, kRPitch halves per row); rows outside the window
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
            col[(row - row0) * kRPitch] = (_Float16)__builtin_amdgcn_exp2f(d * d * neg_k);
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
// Table path
// ---------------------------------------------------------------------------

constexpr int kWWaves = 8;                       // waves per workgroup, each one self-sufficient
constexpr int kWThreads = 64 * kWWaves;
constexpr int kWBirds = 16;                      // birds per wave step: one MFMA k-step
constexpr int kWPitch = kWBirds + 8;             // halves per private tile row (48 B: reads hit 8 bank groups)
constexpr int kMaxWin = 48;                      // window rows per axis (table row width)
constexpr int kSplitTarget = 256;                // workgroups a split launch aims for
constexpr int kMinSliceBirds = 256;              // birds per slice, at least
constexpr int kRedTiles = 3;                     // output tiles per round of the final cross-wave sum

// Per-axis table geometry (quanta per cell c, window half-width j, window rows
// w = 2 j + 1, table row width tw = w rounded up to a multiple of 8 = halo
// rows per side of a tile).
struct TableAxis {
    int32_t c, j, w, tw;
};
struct TableGeom {
    TableAxis ay, ax;
    int rows_y, rows_x;   // tile rows incl. halos: 32 RM + 2 tw_y, 32 RN + 2 tw_x
    int wave_tile;        // halves of one wave's private tiles (Fy then Fx)
    int tab_y, tab_x;     // half offsets of the two tables (tab_x == tab_y when they coincide)
    float neg_k;          // -log2(e) / (2 s^2), in px^-2
    float scale;          // 1 / (2 pi s^2)
    int lds_bytes;
};

// floor(v / c) for |v| < 2^24, 1 <= c < 2^20: a float reciprocal, then one
// correction step either way.
__device__ __forceinline__ int32_t floor_div(int32_t v, int32_t c, float inv_c) {
    int32_t q = (int32_t)floorf((float)v * inv_c);
    if (q * c > v) --q;
    else if ((q + 1) * c <= v) ++q;
    return q;
}

// One lane's half of a bird's window on one axis: table groups [q0, q1) of
// eight rows go to column k of the wave's tile (rows of pitch kWPitch).  The
// table row is zero past w, and the tile's halos are tw rows high, so every
// write stays inside the tile.
__device__ __forceinline__ void put_half_window(_Float16 *tile, const _Float16 *table, int32_t pos_q,
                                                const TableAxis &t, float inv_c, int row0, int nrows, int k,
                                                int q0, int q1, bool have) {
    if (!have) return;
    const int32_t g = floor_div(pos_q, t.c, inv_c);
    // exact for |pos_q| < 2^24; beyond that the bird is far outside any grid
    // this path takes and only the table index needs keeping in range
    const int32_t r = min(max(pos_q - g * t.c, 0), t.c - 1);
    // first window row relative to the output rows, kept inside the halos
    const int32_t lo = min(max(g - t.j - row0, -t.tw), nrows);
    const int off = (lo + t.tw + 8 * q0) * kWPitch + k;
    _Float16 *dst = tile + off;
    const half8 *src = reinterpret_cast<const half8 *>(table + r * t.tw);
    for (int q = q0; q < q1; ++q, dst += 8 * kWPitch) {
        const half8 v = src[q];
#pragma unroll
        for (int e = 0; e < 8; ++e) dst[e * kWPitch] = v[e];
    }
}

// Eight waves, each with private factor tiles for kWBirds birds: a wave takes
// every eighth block of kWBirds birds of its slice, copies their windows from
// the tables into its tiles (lane = bird, axis and half of the window), and
// runs one MFMA k-step over them for every tile of the region.  No barrier is
// needed between waves until the final sum; the next block's copy overlaps
// the current block's matrix-core work.
template <int RM, int RN>
__global__ __launch_bounds__(kWThreads) void density_table_kernel(DensityArgs a, TableGeom tg, int regions_y,
                                                                  int regions_x, int split, float *partial) {
    constexpr int kRowsY = 32 * RM, kRowsX = 32 * RN;
    extern __shared__ __align__(16) unsigned char lds[];
    _Float16 *const sh = reinterpret_cast<_Float16 *>(lds);

    const int per_frame = regions_y * regions_x * split;
    const int f = blockIdx.x / per_frame;
    const int rem = blockIdx.x - f * per_frame;
    const int reg = rem / split;
    const int sl = rem - reg * split;
    const int gy0 = (reg / regions_x) * kRowsY;
    const int gx0 = (reg % regions_x) * kRowsX;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    const int32_t b = a.offsets[f];
    const int32_t e = a.offsets[f + 1];
    const bool ok = !(b < 0 || e < b || e > a.total);
    const int32_t n = ok ? e - b : 0;
    // this workgroup's slice of the frame's birds
    const int32_t k0 = (int32_t)((int64_t)n * sl / split);
    const int32_t k1 = (int32_t)((int64_t)n * (sl + 1) / split);
    const int2 *P = reinterpret_cast<const int2 *>(a.xy) + b;

    _Float16 *const tile = sh + wave * tg.wave_tile;
    {
        // this wave's tiles start at zero (halo rows too: never read, but cheap)
        uint4 *z = reinterpret_cast<uint4 *>(tile);
        const uint4 zero = make_uint4(0, 0, 0, 0);
        for (int i = lane; i < tg.wave_tile / 8; i += 64) z[i] = zero;
        // the tables hold the exact windows
        auto build = [&](const TableAxis &t, _Float16 *tab) {
            for (int r = tid; r < t.c; r += kWThreads) {
                const float base = ((float)r - 0.5f * (float)t.c + (float)(t.j * t.c)) * 0.0625f;
                const float step = (float)t.c * 0.0625f;
                for (int jj = 0; jj < t.tw; ++jj) {
                    const float d = base - (float)jj * step;  // exact: multiples of 1/32 px
                    tab[r * t.tw + jj] =
                        jj < t.w ? (_Float16)__builtin_amdgcn_exp2f(d * d * tg.neg_k) : (_Float16)0.0f;
                }
            }
        };
        build(tg.ay, sh + tg.tab_y);
        if (tg.tab_x != tg.tab_y) build(tg.ax, sh + tg.tab_x);
    }

    float16v acc[RM][RN];
#pragma unroll
    for (int m = 0; m < RM; ++m)
#pragma unroll
        for (int t = 0; t < RN; ++t)
#pragma unroll
            for (int j = 0; j < 16; ++j) acc[m][t][j] = 0.0f;

    // copy roles: lane -> (bird bk of the block, axis, half of the window)
    const int bk = lane & (kWBirds - 1);
    const bool yaxis = (lane & 16) == 0;
    const int half = lane >> 5;
    const TableAxis ta = yaxis ? tg.ay : tg.ax;
    const int groups = ta.tw >> 3;
    const int q0 = half ? (groups + 1) >> 1 : 0;
    const int q1 = half ? groups : (groups + 1) >> 1;
    _Float16 *const atile = tile + (yaxis ? 0 : tg.rows_y * kWPitch);
    const _Float16 *const table = sh + (yaxis ? tg.tab_y : tg.tab_x);
    const int row0 = yaxis ? gy0 : gx0;
    const int nrows = yaxis ? kRowsY : kRowsX;
    // MFMA roles: lane -> (tile row, eight birds)
    const int r32 = lane & 31;
    const int kq = (lane >> 5) * 8;
    const _Float16 *const fy = tile + tg.ay.tw * kWPitch;
    const _Float16 *const fx = tile + (tg.rows_y + tg.ax.tw) * kWPitch;

    const float inv_c = 1.0f / (float)ta.c;
    const int32_t nblk = (k1 - k0 + kWBirds - 1) / kWBirds;
    // each lane's coordinate for this wave's next kAhead blocks (register ring)
    constexpr int kAhead = 4;
    auto coord = [&](int32_t blk) -> int32_t {
        const int32_t kb = k0 + blk * kWBirds + bk;
        return kb < k1 ? (yaxis ? P[kb].y : P[kb].x) : 0;
    };
    int32_t pos[kAhead];
#pragma unroll
    for (int j = 0; j < kAhead; ++j) pos[j] = coord(wave + j * kWWaves);
    __syncthreads();  // tables written

    for (int32_t i = 0; wave + i * kWWaves < nblk; i += kAhead) {
#pragma unroll
        for (int j = 0; j < kAhead; ++j) {
            const int32_t blk = wave + (i + j) * kWWaves;
            if (blk >= nblk) break;
            const int32_t kb = k0 + blk * kWBirds + bk;
            put_half_window(atile, table, pos[j], ta, inv_c, row0, nrows, bk, q0, q1, kb < k1);
            pos[j] = coord(blk + kAhead * kWWaves);  // fetched kAhead blocks ahead
            // this wave's own writes are read back below; LDS keeps one wave's
            // accesses in order, and the fence keeps the compiler from moving them
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            __builtin_amdgcn_wave_barrier();
            half8 bx[RN];
#pragma unroll
            for (int t = 0; t < RN; ++t)
                bx[t] = *reinterpret_cast<const half8 *>(fx + (t * 32 + r32) * kWPitch + kq);
#pragma unroll
            for (int m = 0; m < RM; ++m) {
                const half8 ay = *reinterpret_cast<const half8 *>(fy + (m * 32 + r32) * kWPitch + kq);
#pragma unroll
                for (int t = 0; t < RN; ++t)
                    acc[m][t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ay, bx[t], acc[m][t], 0, 0, 0);
            }
            // clear the output rows for the next block (16-byte stores of whole
            // rows, after this wave's operand reads, which LDS keeps in order);
            // halo rows are never read and keep whatever the windows left there
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int i = lane; i < 2 * (kRowsY + kRowsX); i += 64) {
                const int row = i >> 1;
                const int trow = row < kRowsY ? tg.ay.tw + row : tg.rows_y + tg.ax.tw + (row - kRowsY);
                *reinterpret_cast<half8 *>(tile + trow * kWPitch + (i & 1) * 8) = half8{};
            }
            __builtin_amdgcn_wave_barrier();
        }
    }
    __syncthreads();  // every wave is done with its tiles: the space holds the final sum

    // Sum the waves' tiles in a fixed order and store.  Lane l of a wave holds
    // column (l & 31) and rows 8*(j/4) + 4*(l/32) + (j%4), j = 0..15.
    float *red = reinterpret_cast<float *>(lds);
    const size_t cells = (size_t)a.grid_h * a.grid_w;
    float *out = split > 1 ? partial + ((size_t)f * split + sl) * cells : a.density + (size_t)f * cells;
    const float scale = split > 1 ? 1.0f : tg.scale;
    constexpr int kTiles = RM * RN;
    constexpr int kPerRound = kTiles < kRedTiles ? kTiles : kRedTiles;
    constexpr int kTile = kWWaves * 32 * 33;  // floats per tile: every wave's partial, padded rows
#pragma unroll
    for (int t0 = 0; t0 < kTiles; t0 += kPerRound) {
#pragma unroll
        for (int q = 0; q < kPerRound; ++q) {
            if (t0 + q >= kTiles) break;
            const int m = (t0 + q) / RN, t = (t0 + q) % RN;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int row = 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3);
                red[q * kTile + (wave * 32 + row) * 33 + r32] = acc[m][t][j];
            }
        }
        __syncthreads();
        const int ntiles = min(kPerRound, kTiles - t0);
        for (int el = tid; el < ntiles * 1024; el += kWThreads) {
            const int q = el >> 10, row = (el >> 5) & 31, colx = el & 31;
            const float *rq = red + q * kTile + row * 33 + colx;
            float v = 0.0f;
#pragma unroll
            for (int w = 0; w < kWWaves; ++w) v += rq[w * 32 * 33];
            const int m = (t0 + q) / RN, t = (t0 + q) % RN;
            const int gy = gy0 + m * 32 + row;
            const int gx = gx0 + t * 32 + colx;
            if ((ok || split > 1) && gy < a.grid_h && gx < a.grid_w) out[(size_t)gy * a.grid_w + gx] = v * scale;
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
        float s = 0.0f;
        for (int k = 0; k < split; ++k) s += src[k * cells];
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

template <int RM, int RN>
hipError_t launch_table(const DensityArgs &a, const TableGeom &tg, const DensityPlan &p, float *partial,
                        hipStream_t stream) {
    const long long blocks = (long long)a.n_frames * p.regions_y * p.regions_x * p.split;
    const size_t lds = (size_t)tg.lds_bytes;
    hipLaunchKernelGGL((density_table_kernel<RM, RN>), dim3((unsigned)blocks), dim3(kWThreads), lds, stream, a,
                       tg, p.regions_y, p.regions_x, p.split, partial);
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


// Table geometry for a region shape; false when the table path does not apply
// (a cell is not a whole number of quanta, a window is wider than kMaxWin rows,
// or the tiles and tables exceed the LDS budget).
bool make_table_geom(const DensityArgs &a, int rm, int rn, size_t lds_limit, TableGeom *tg) {
    if ((16LL * a.height_px) % a.grid_h != 0 || (16LL * a.width_px) % a.grid_w != 0) return false;
    const double cut_q = 16.0 * kCutSigmas * (double)a.sigma_px;  // window half-width, quanta
    auto axis = [&](int64_t c, TableAxis *t) {
        if (c < 1 || c > (1 << 20)) return false;
        // rows G + j with |j| <= j cover every row centre within cut_q of the bird
        const double jd = std::ceil(cut_q / (double)c) + 1.0;
        if (jd > (kMaxWin - 1) / 2) return false;
        t->c = (int)c;
        t->j = (int)jd;
        t->w = 2 * t->j + 1;
        t->tw = (t->w + 7) / 8 * 8;
        return true;
    };
    if (!axis(16LL * a.height_px / a.grid_h, &tg->ay) || !axis(16LL * a.width_px / a.grid_w, &tg->ax))
        return false;
    tg->rows_y = 32 * rm + 2 * tg->ay.tw;
    tg->rows_x = 32 * rn + 2 * tg->ax.tw;
    tg->wave_tile = (tg->rows_y + tg->rows_x) * kWPitch;
    tg->tab_y = kWWaves * tg->wave_tile;
    const bool shared = tg->ay.c == tg->ax.c && tg->ay.j == tg->ax.j;
    tg->tab_x = shared ? tg->tab_y : tg->tab_y + tg->ay.c * tg->ay.tw;
    const int64_t halves = (int64_t)tg->tab_x + (shared ? (int64_t)tg->ay.c * tg->ay.tw
                                                        : (int64_t)tg->ax.c * tg->ax.tw);
    const int64_t red = (int64_t)std::min(rm * rn, kRedTiles) * kWWaves * 32 * 33 * 4;
    const int64_t bytes = std::max<int64_t>(2 * halves, red);
    if (bytes > (int64_t)lds_limit) return false;
    tg->lds_bytes = (int)bytes;
    const double s = (double)a.sigma_px;
    tg->neg_k = (float)(-1.4426950408889634 / (2.0 * s * s));
    tg->scale = (float)(1.0 / (2.0 * 3.14159265358979323846 * s * s));
    return true;
}

long long shape_regions(const Shape &sh, int grid_w, int grid_h) {
    return ((grid_h + 32LL * sh.rm - 1) / (32LL * sh.rm)) * ((grid_w + 32LL * sh.rn - 1) / (32LL * sh.rn));
}

// Ordering of region shapes for the table path: least padded area, then
// fewest regions.
bool table_better(const Shape &x, const Shape &y, int grid_w, int grid_h) {
    const long long rx = shape_regions(x, grid_w, grid_h), ry = shape_regions(y, grid_w, grid_h);
    const long long ax = rx * x.rm * x.rn, ay = ry * y.rm * y.rn;
    return ax < ay || (ax == ay && rx < ry);
}

Shape table_shape(int grid_w, int grid_h) {
    Shape best = kShapes[0];
    for (const Shape &sh : kShapes)
        if (table_better(sh, best, grid_w, grid_h)) best = sh;
    return best;
}

// Bird slices per (frame, region): enough workgroups to fill the chip, at
// least kMinSliceBirds birds per slice on average.
int table_split(int32_t n_frames, int32_t total, long long regions) {
    const long long wgs = (long long)n_frames * regions;
    if (n_frames <= 0 || wgs >= kSplitTarget) return 1;
    const long long want = (kSplitTarget + wgs - 1) / wgs;
    const long long cap = std::max<long long>(1, (long long)total / n_frames / kMinSliceBirds);
    return (int)std::max<long long>(1, std::min<long long>(std::min(want, cap), 64));
}

}  // namespace

size_t density_workspace_bytes(int32_t n_frames, int32_t total, int32_t grid_w, int32_t grid_h) {
    if (n_frames <= 0 || grid_w < 1 || grid_h < 1) return 0;
    const Shape sh = table_shape(grid_w, grid_h);
    const int split = table_split(n_frames, total, shape_regions(sh, grid_w, grid_h));
    if (split <= 1) return 0;
    return (size_t)n_frames * split * (size_t)grid_w * grid_h * sizeof(float);
}

// Recurrence path: choose the output region per workgroup with a small cost
// model: per bird a region costs its matrix-core time (RM*RN/2 cycles), the
// factor rows its windows cover and its tile clearing; workgroups spread over
// the compute units, and a launch never finishes before one workgroup does.
// Table path: the least padded region shape whose tiles fit in LDS, and bird
// slices when the batch has few (frame, region) pairs.
// FLOCK_DENSITY_SHAPE="rm,rn" forces a region shape and FLOCK_DENSITY_PATH=
// "recur" or "table" a path where it applies (for tuning).
DensityPlan plan_density(const DensityArgs &a, int n_cus, size_t lds_limit) {
    const int tiles_y = (a.grid_h + 31) / 32;
    const int tiles_x = (a.grid_w + 31) / 32;
    const char *force = std::getenv("FLOCK_DENSITY_SHAPE");
    const char *path = std::getenv("FLOCK_DENSITY_PATH");
    const bool force_recur = path && std::strcmp(path, "recur") == 0;
    const bool force_table = path && std::strcmp(path, "table") == 0;
    int frm = 0, frn = 0;
    if (force && std::sscanf(force, "%d,%d", &frm, &frn) == 2) {
        bool known = false;
        for (const Shape &sh : kShapes) known |= sh.rm == frm && sh.rn == frn;
        if (!known) frm = frn = 0;
    }
    // The table path's single-column LDS writes conflict across banks, so on
    // batches that already fill the chip the recurrence path is faster; the
    // table path serves batches with fewer (frame, region) pairs than
    // workgroups wanted, which it splits by birds.
    const Shape pref = table_shape(a.grid_w, a.grid_h);
    const bool few = (long long)a.n_frames * shape_regions(pref, a.grid_w, a.grid_h) < kSplitTarget;
    if (!force_recur && (few || force_table)) {
        // table path: the forced shape, else the best shape whose tiles fit
        const int split_cap = table_split(a.n_frames, a.total, shape_regions(pref, a.grid_w, a.grid_h));
        TableGeom tg;
        bool found = false;
        Shape best = kShapes[0];
        if (frm) {
            best = Shape{frm, frn};
            found = make_table_geom(a, frm, frn, lds_limit, &tg);
        } else {
            for (const Shape &sh : kShapes)
                if ((!found || table_better(sh, best, a.grid_w, a.grid_h)) &&
                    make_table_geom(a, sh.rm, sh.rn, lds_limit, &tg)) {
                    best = sh;
                    found = true;
                }
        }
        if (found) {
            const long long regions = shape_regions(best, a.grid_w, a.grid_h);
            const int split = std::min(split_cap, table_split(a.n_frames, a.total, regions));
            return DensityPlan{1, best.rm, best.rn, (int)((a.grid_h + 32LL * best.rm - 1) / (32LL * best.rm)),
                               (int)((a.grid_w + 32LL * best.rn - 1) / (32LL * best.rn)), split};
        }
    }
    if (frm) return DensityPlan{0, frm, frn, (tiles_y + frm - 1) / frm, (tiles_x + frn - 1) / frn, 1};
    const double s = (double)a.sigma_px;
    const double hx = (double)a.width_px / a.grid_w, hy = (double)a.height_px / a.grid_h;
    const double lx = std::min(2.0 * kCutSigmas * s / hx + 1.0, (double)a.grid_w);
    const double ly = std::min(2.0 * kCutSigmas * s / hy + 1.0, (double)a.grid_h);
    const double birds = a.n_frames > 0 ? (double)a.total / a.n_frames : 0.0;
    DensityPlan best{0, 1, 1, tiles_y, tiles_x, 1};
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
            best = DensityPlan{0, sh.rm, sh.rn, ry, rx, 1};
        }
    }
    return best;
}

hipError_t launch_density(const DensityArgs &a, const DensityPlan &p, size_t lds_limit, float *partial,
                          hipStream_t stream) {
    hipError_t err = hipErrorInvalidValue;
    if (p.table) {
        TableGeom tg;
        if (!make_table_geom(a, p.rm, p.rn, lds_limit, &tg)) return hipErrorInvalidValue;
        if (p.split > 1 && !partial) return hipErrorInvalidValue;
#define FLOCK_SHAPE(RM, RN) \
    if (p.rm == RM && p.rn == RN) err = launch_table<RM, RN>(a, tg, p, partial, stream);
        FLOCK_SHAPE(1, 1) FLOCK_SHAPE(1, 2) FLOCK_SHAPE(2, 1) FLOCK_SHAPE(2, 2) FLOCK_SHAPE(1, 4)
        FLOCK_SHAPE(3, 2) FLOCK_SHAPE(2, 4) FLOCK_SHAPE(3, 4) FLOCK_SHAPE(4, 2) FLOCK_SHAPE(5, 2)
        FLOCK_SHAPE(4, 1) FLOCK_SHAPE(5, 1)
#undef FLOCK_SHAPE
        if (err != hipSuccess || p.split <= 1) return err;
        const int64_t cells = (int64_t)a.grid_h * a.grid_w;
        const int64_t total = cells * a.n_frames;
        const unsigned blocks = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
        hipLaunchKernelGGL(density_reduce_kernel, dim3(blocks), dim3(256), 0, stream, a.density, partial, cells,
                           total, p.split, tg.scale);
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

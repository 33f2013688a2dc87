// heatmap.hip - heatmap analytics of density grids on gfx950.
//
// What is computed (the clustering module of Section 2.3 thresholds the
// density heatmaps and applies connected component analysis; Algorithm 1
// computes the heatmap, its entropy and a clustering degree per frame):
//   hot cell     density >= threshold;
//   component    connected hot cells under the 4-neighbourhood (shared edge)
//                or the 8-neighbourhood (shared edge or corner), labelled by
//                its smallest row-major cell index gy * grid_w + gx; cold
//                cells get -1;
//   per component  cells and mass = cell_area * sum of density, stored at
//                the label cell (0 elsewhere);
//   entropy      -sum p ln p over positive cells, p = density / S, S the sum
//                of the positive cells (0 when S = 0);
//   degree       (sum of density over hot cells) / S (0 when S = 0).
//
// Design (HBM-bound: a few bytes per cell).  Grids whose int32 forest fits
// in LDS (grid_w * grid_h <= about 39k cells) take heat_frame_kernel, one
// workgroup per frame (described there).  Larger grids take four tiled
// kernels:
//   1. heat_tile_kernel, one 256-thread workgroup per 32 x 32 tile: loads the
//      tile once, unites hot neighbours inside the tile in LDS (smallest
//      index hooking), writes each hot cell's tile root (frame index) into
//      `labels` as a forest, clears the component outputs and writes the
//      tile's partial sums (S, sum D ln D, hot sum, largest D) in a fixed
//      order;
//   2. heat_merge_kernel: threads on tile boundary cells unite hot pairs that
//      cross a tile edge in the global forest (agent-scope CAS hooking, the
//      smaller root wins); extra workgroups add each frame's tile partials in
//      tile order into entropy and degree and pick the frame's fixed-point
//      scale;
//   3. heat_label_kernel, per tile again: each hot cell walks to its root and
//      stores it; cells and fixed-point mass are summed per root in an LDS
//      table, then added once per (tile, root) to the root's outputs (integer
//      atomics, so the sums do not depend on their order);
//   4. heat_mass_kernel: the root cells turn their fixed-point mass into
//      cell_area * sum.
// Every output is a deterministic function of the input.

#include <climits>
#include <cmath>

#include "cluster_common.h"
#include "internal.h"

namespace flock {
namespace {

using namespace cl;

constexpr int kHT = 32;                 // tile side, cells
constexpr int kHThreads = 256;          // 4 cells per thread
constexpr int kHRows = kHThreads / kHT; // rows per pass
constexpr int kHTable = 1024;           // LDS table slots for (root -> sums) per tile

struct TilePart {
    double s, e, hot;  // sum D, sum D ln D over positive cells; sum D over hot cells
    uint32_t maxbits;  // largest positive D, as its float bits (0 if none)
    uint32_t pad;
};

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ uint32_t wave_max_u(uint32_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, 64));
    return v;
}

// Natural log of a positive float in fp64, from a table of bucket centres:
// v = m 2^e exactly (m in [1, 2)), c is the centre of m's bucket of width
// 1/kLnBuckets, and ln v = e ln 2 + ln c + ln(1 + r) with r = m / c - 1,
// |r| <= 2^-8, formed as fma(m, 1/c, -1); ln(1 + r) is its Taylor series
// through r^7 (truncation below 2^-67).  The absolute error is a few 1e-16
// (ln 2 and the table entries are rounded to fp64; |e| <= 149), about the
// library routine's, at a fraction of its instructions.
constexpr int kLnBuckets = 128;
struct LnTable {
    double ln_c[kLnBuckets], inv_c[kLnBuckets];
};

// Filled by threads 0 .. kLnBuckets - 1; the caller syncs before use.
__device__ __forceinline__ void ln_table_init(LnTable &t) {
    const int k = threadIdx.x;
    if (k < kLnBuckets) {
        const double c = 1.0 + ((double)k + 0.5) / kLnBuckets;
        t.ln_c[k] = log(c);
        t.inv_c[k] = 1.0 / c;
    }
}

__device__ __forceinline__ double ln_pos(float vf, const LnTable &t) {
    const uint64_t b = (uint64_t)__double_as_longlong((double)vf);
    const int e = (int)(b >> 52) - 1023;
    const int k = (int)((b >> 45) & (kLnBuckets - 1));
    const double m = __longlong_as_double((long long)((b & 0x000fffffffffffffull) | 0x3ff0000000000000ull));
    const double r = fma(m, t.inv_c[k], -1.0);
    const double p =
        r * (1.0 + r * (-0.5 + r * (1.0 / 3.0 + r * (-0.25 + r * (0.2 + r * (-1.0 / 6.0 + r * (1.0 / 7.0)))))));
    return fma((double)e, 0.69314718055994530942, t.ln_c[k] + p);
}

struct TileGeom {
    int f, x0, y0, w, h;
};

__device__ __forceinline__ TileGeom tile_of(const HeatArgs &a, long long b) {
    const long long per = (long long)a.tiles_x * a.tiles_y;
    TileGeom t;
    t.f = (int)(b / per);
    const int r = (int)(b - (long long)t.f * per);
    t.y0 = (r / a.tiles_x) * kHT;
    t.x0 = (r % a.tiles_x) * kHT;
    t.w = min(kHT, a.grid_w - t.x0);
    t.h = min(kHT, a.grid_h - t.y0);
    return t;
}

__global__ __launch_bounds__(kHThreads) void heat_tile_kernel(HeatArgs a, TilePart *part) {
    __shared__ int32_t par[kHT * kHT];
    __shared__ uint8_t hotm[kHT * kHT];
    __shared__ double s_red[3][kHThreads / 64];
    __shared__ uint32_t s_max[kHThreads / 64];
    __shared__ LnTable lnt;
    ln_table_init(lnt);
    __syncthreads();
    const TileGeom t = tile_of(a, blockIdx.x);
    const int tid = threadIdx.x, lx = tid % kHT, ly0 = tid / kHT;
    const size_t cells = (size_t)a.grid_w * a.grid_h;
    const float *D = a.density + (size_t)t.f * cells;

    double s = 0.0, e = 0.0, hs = 0.0;
    uint32_t mb = 0;
    float v[kHT / kHRows];
    bool hot[kHT / kHRows];
#pragma unroll
    for (int k = 0; k < kHT / kHRows; ++k) {
        const int ly = ly0 + kHRows * k, l = ly * kHT + lx;
        const bool in = lx < t.w && ly < t.h;
        const size_t c = (size_t)(t.y0 + ly) * a.grid_w + t.x0 + lx;
        v[k] = in ? D[c] : 0.0f;
        hot[k] = in && v[k] >= a.threshold;
        par[l] = l;
        hotm[l] = hot[k];
        if (v[k] > 0.0f) {
            s += (double)v[k];
            e += (double)v[k] * ln_pos(v[k], lnt);
            mb = max(mb, __float_as_uint(v[k]));
        }
        if (hot[k]) hs += (double)v[k];
        if (in) {
            a.comp_cells[(size_t)t.f * cells + c] = 0;
            a.comp_mass[(size_t)t.f * cells + c] = 0.0;
        }
    }
    __syncthreads();
    // unite hot neighbours inside the tile: right, down, and for the
    // 8-neighbourhood down-left and down-right
#pragma unroll
    for (int k = 0; k < kHT / kHRows; ++k) {
        if (!hot[k]) continue;
        const int ly = ly0 + kHRows * k, l = ly * kHT + lx;
        if (lx + 1 < t.w && hotm[l + 1]) uf_unite<kGroup>(par, l, l + 1);
        if (ly + 1 < t.h) {
            if (hotm[l + kHT]) uf_unite<kGroup>(par, l, l + kHT);
            if (a.connectivity == 8) {
                if (lx > 0 && hotm[l + kHT - 1]) uf_unite<kGroup>(par, l, l + kHT - 1);
                if (lx + 1 < t.w && hotm[l + kHT + 1]) uf_unite<kGroup>(par, l, l + kHT + 1);
            }
        }
    }
    __syncthreads();
    // each hot cell's tile root (a smaller tile index is a smaller frame
    // index) starts the global forest; cold cells are -1
    int32_t *L = a.labels + (size_t)t.f * cells;
#pragma unroll
    for (int k = 0; k < kHT / kHRows; ++k) {
        const int ly = ly0 + kHRows * k;
        if (!(lx < t.w && ly < t.h)) continue;
        const size_t c = (size_t)(t.y0 + ly) * a.grid_w + t.x0 + lx;
        int32_t lab = -1;
        if (hot[k]) {
            const int r = uf_root<kGroup>(par, ly * kHT + lx);
            lab = (t.y0 + r / kHT) * a.grid_w + t.x0 + r % kHT;
        }
        L[c] = lab;
    }
    // the tile's partial sums, in a fixed order
    s = wave_sum_d(s);
    e = wave_sum_d(e);
    hs = wave_sum_d(hs);
    mb = wave_max_u(mb);
    const int wave = tid >> 6;
    if ((tid & 63) == 0) {
        s_red[0][wave] = s;
        s_red[1][wave] = e;
        s_red[2][wave] = hs;
        s_max[wave] = mb;
    }
    __syncthreads();
    if (tid == 0) {
        TilePart p{0.0, 0.0, 0.0, 0u, 0u};
        for (int w = 0; w < kHThreads / 64; ++w) {
            p.s += s_red[0][w];
            p.e += s_red[1][w];
            p.hot += s_red[2][w];
            p.maxbits = max(p.maxbits, s_max[w]);
        }
        part[blockIdx.x] = p;
    }
}

// Crossing forward edges of cell (gx, gy): right, down, down-left,
// down-right (the last two for the 8-neighbourhood), where the neighbour
// lies in another tile.
__device__ __forceinline__ void merge_cell(const HeatArgs &a, int f, int gx, int gy) {
    const size_t cells = (size_t)a.grid_w * a.grid_h;
    const float *D = a.density + (size_t)f * cells;
    const int32_t c = gy * a.grid_w + gx;
    if (!(D[c] >= a.threshold)) return;
    int32_t *L = a.labels + (size_t)f * cells;
    const bool xe = (gx % kHT) == kHT - 1, x0 = (gx % kHT) == 0, ye = (gy % kHT) == kHT - 1;
    auto take = [&](int nx, int ny) {
        const int32_t n = ny * a.grid_w + nx;
        if (D[n] >= a.threshold) uf_unite<kAgent>(L, c, n);
    };
    if (xe && gx + 1 < a.grid_w) take(gx + 1, gy);
    if (gy + 1 < a.grid_h) {
        if (ye) take(gx, gy + 1);
        if (a.connectivity == 8) {
            if (gx > 0 && (x0 || ye)) take(gx - 1, gy + 1);
            if (gx + 1 < a.grid_w && (xe || ye)) take(gx + 1, gy + 1);
        }
    }
}

__global__ __launch_bounds__(256) void heat_merge_kernel(HeatArgs a, const TilePart *part, int32_t *shift,
                                                         long long merge_blocks) {
    const int tid = threadIdx.x;
    if ((long long)blockIdx.x < merge_blocks) {
        // boundary cells of every frame: for each inner vertical tile edge
        // its two columns, for each inner horizontal edge its upper row
        const long long nv = 2LL * (a.tiles_x - 1) * a.grid_h, nh = (long long)(a.tiles_y - 1) * a.grid_w;
        const long long per = nv + nh;
        const long long i = (long long)blockIdx.x * 256 + tid;
        if (i >= per * a.n_frames) return;
        const int f = (int)(i / per);
        const long long j = i - (long long)f * per;
        int gx, gy;
        if (j < nv) {
            const long long k = j / (2LL * a.grid_h);
            const int side = (int)((j / a.grid_h) % 2);
            gx = (int)(kHT * (k + 1) - 1 + side);
            gy = (int)(j % a.grid_h);
        } else {
            const long long jj = j - nv;
            gy = (int)(kHT * (jj / a.grid_w + 1) - 1);
            gx = (int)(jj % a.grid_w);
        }
        merge_cell(a, f, gx, gy);
        return;
    }
    // one workgroup per frame: tile partials in tile order (strided per lane,
    // then a fixed shuffle tree), entropy, degree, the fixed-point scale
    const int f = (int)((long long)blockIdx.x - merge_blocks);
    if (tid >= 64) return;
    const long long per = (long long)a.tiles_x * a.tiles_y;
    const TilePart *P = part + (size_t)f * per;
    double s = 0.0, e = 0.0, hs = 0.0;
    uint32_t mb = 0;
    for (long long k = tid; k < per; k += 64) {
        s += P[k].s;
        e += P[k].e;
        hs += P[k].hot;
        mb = max(mb, P[k].maxbits);
    }
    s = wave_sum_d(s);
    e = wave_sum_d(e);
    hs = wave_sum_d(hs);
    mb = wave_max_u(mb);
    if (tid == 0) {
        a.entropy[f] = s > 0.0 ? log(s) - e / s : 0.0;
        a.degree[f] = s > 0.0 ? hs / s : 0.0;
        a.n_components[f] = 0;
        // every positive D is below 2^(E + 1), E its float exponent; with
        // 2^lg >= cells, D * 2^sh with sh = 62 - (E + 1) - lg keeps any sum of
        // cells below 2^62
        const int E = mb ? (int)((mb >> 23) & 0xffu) - 127 : 0;
        int lg = 0;
        while ((1LL << lg) < (long long)a.grid_w * a.grid_h) ++lg;
        shift[f] = 62 - (max(E, -126) + 1) - lg;
    }
}

__device__ __forceinline__ uint32_t slot_hash(int32_t root) { return ((uint32_t)root * 2654435761u) >> 22; }

__global__ __launch_bounds__(kHThreads) void heat_label_kernel(HeatArgs a, const int32_t *shift) {
    __shared__ int32_t keys[kHTable];
    __shared__ int32_t cnt[kHTable];
    __shared__ unsigned long long mass[kHTable];
    const TileGeom t = tile_of(a, blockIdx.x);
    const int tid = threadIdx.x, lx = tid % kHT, ly0 = tid / kHT;
    for (int k = tid; k < kHTable; k += kHThreads) {
        keys[k] = -1;
        cnt[k] = 0;
        mass[k] = 0ull;
    }
    __syncthreads();
    const size_t cells = (size_t)a.grid_w * a.grid_h;
    const float *D = a.density + (size_t)t.f * cells;
    int32_t *L = a.labels + (size_t)t.f * cells;
    const int sh = shift[t.f];
#pragma unroll
    for (int k = 0; k < kHT / kHRows; ++k) {
        const int ly = ly0 + kHRows * k;
        if (!(lx < t.w && ly < t.h)) continue;
        const int32_t c = (t.y0 + ly) * a.grid_w + t.x0 + lx;
        const float v = D[c];
        if (!(v >= a.threshold)) continue;
        // read-only walk: concurrent writers only store roots
        const int32_t root = uf_root<kAgent>(L, c);
        st_rlx<kAgent>(L + c, root);
        if (root == c) atomicAdd(a.n_components + t.f, 1);
        const unsigned long long q = (unsigned long long)llrint(ldexp((double)v, sh));
        // this root's slot in the tile table (linear probing; a tile has at
        // most kHT * kHT = kHTable distinct roots, so a slot is always found)
        uint32_t h = slot_hash(root);
        for (;;) {
            const int32_t old = atomicCAS(keys + h, -1, root);
            if (old == -1 || old == root) break;
            h = (h + 1) & (kHTable - 1);
        }
        atomicAdd(cnt + h, 1);
        atomicAdd(mass + h, q);
    }
    __syncthreads();
    int32_t *CC = a.comp_cells + (size_t)t.f * cells;
    unsigned long long *CM = reinterpret_cast<unsigned long long *>(a.comp_mass + (size_t)t.f * cells);
    for (int k = tid; k < kHTable; k += kHThreads) {
        const int32_t root = keys[k];
        if (root < 0) continue;
        atomicAdd(CC + root, cnt[k]);
        atomicAdd(CM + root, mass[k]);
    }
}

__global__ __launch_bounds__(256) void heat_mass_kernel(HeatArgs a, const int32_t *shift) {
    const size_t cells = (size_t)a.grid_w * a.grid_h;
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= cells * (size_t)a.n_frames) return;
    const int f = (int)(i / cells);
    const int32_t c = (int32_t)(i - (size_t)f * cells);
    if (a.labels[i] != c) return;  // not a component's label cell
    const unsigned long long q = reinterpret_cast<const unsigned long long *>(a.comp_mass)[i];
    a.comp_mass[i] = ldexp((double)q, -shift[f]) * a.cell_area;
}

// The same for the frame-resident path, over each frame's list of label
// cells only (one workgroup per frame).
__global__ __launch_bounds__(256) void heat_root_mass_kernel(HeatArgs a, const int32_t *shift,
                                                             const int32_t *roots) {
    const int f = blockIdx.x;
    const size_t cells = (size_t)a.grid_w * a.grid_h;
    const int n = a.n_components[f];
    const int sh = shift[f];
    unsigned long long *CMu = reinterpret_cast<unsigned long long *>(a.comp_mass) + (size_t)f * cells;
    double *CM = a.comp_mass + (size_t)f * cells;
    for (int t = threadIdx.x; t < n; t += 256) {
        const int32_t c = roots[(size_t)f * cells + t];
        CM[c] = ldexp((double)CMu[c], -sh) * a.cell_area;
    }
}

// ---------------------------------------------------------------------------
// Frame-resident path: one workgroup per frame, the whole grid's forest in LDS
// ---------------------------------------------------------------------------

constexpr int kFThreads = 1024;
constexpr int kFWaves = kFThreads / 64;

// Inclusive prefix sum over the wave (64-bit values).
__device__ __forceinline__ unsigned long long wave_incl_scan_u64(unsigned long long v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const unsigned long long t = __shfl_up(v, o, 64);
        if (lane >= o) v += t;
    }
    return v;
}

// One frame per 1024-thread workgroup (grid_w * grid_h int32 parents in LDS):
//   A. one coalesced pass over the grid: hot flags (parent = own index, -1
//      cold), the partial sums, outputs cleared; a fixed-order block sum
//      gives entropy, degree and the fixed-point scale;
//   B. horizontal runs of hot cells, one row per wave at a time and 64 cells
//      per ballot: every cell of a run points at the run's first cell;
//   C. joins between consecutive rows, once per overlap: the vertical pair
//      (c, c + w) unless the pair to its left already joins the same runs,
//      and for the 8-neighbourhood a diagonal pair only where no edge-sharing
//      path through c's row neighbour or the cell below exists;
//   D. labels by read-only walks; per wave, runs of lanes with equal roots
//      add their cells and fixed-point mass with one global atomic each;
//      each root cell appends its index to the frame's list in the workspace.
// heat_root_mass_kernel then converts the listed cells' mass (after the kernel
// boundary every atomic is complete; a device-scope fence inside the kernel
// would instead write back the L2 once per workgroup).
__global__ __launch_bounds__(kFThreads) void heat_frame_kernel(HeatArgs a, int32_t *shift, int32_t *roots) {
    extern __shared__ int32_t P[];
    __shared__ double s_red[3][kFWaves];
    __shared__ uint32_t s_max[kFWaves];
    __shared__ int s_shift, s_ncomp;
    __shared__ LnTable lnt;
    ln_table_init(lnt);
    __syncthreads();
    const int f = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int gw = a.grid_w, gh = a.grid_h;
    const int cells = gw * gh;
    const float *D = a.density + (size_t)f * cells;
    int32_t *L = a.labels + (size_t)f * cells;
    int32_t *CC = a.comp_cells + (size_t)f * cells;
    double *CM = a.comp_mass + (size_t)f * cells;
    unsigned long long *CMu = reinterpret_cast<unsigned long long *>(CM);

    // A
    double s = 0.0, e = 0.0, hs = 0.0;
    uint32_t mb = 0;
    for (int c = tid; c < cells; c += kFThreads) {
        const float v = D[c];
        const bool hot = v >= a.threshold;
        P[c] = hot ? c : -1;
        if (v > 0.0f) {
            s += (double)v;
            e += (double)v * ln_pos(v, lnt);
            mb = max(mb, __float_as_uint(v));
        }
        if (hot) hs += (double)v;
        CC[c] = 0;
        CM[c] = 0.0;
    }
    s = wave_sum_d(s);
    e = wave_sum_d(e);
    hs = wave_sum_d(hs);
    mb = wave_max_u(mb);
    if (lane == 0) {
        s_red[0][wave] = s;
        s_red[1][wave] = e;
        s_red[2][wave] = hs;
        s_max[wave] = mb;
    }
    __syncthreads();
    if (tid == 0) {
        double S = 0.0, E = 0.0, HS = 0.0;
        uint32_t M = 0;
        for (int w = 0; w < kFWaves; ++w) {
            S += s_red[0][w];
            E += s_red[1][w];
            HS += s_red[2][w];
            M = max(M, s_max[w]);
        }
        a.entropy[f] = S > 0.0 ? log(S) - E / S : 0.0;
        a.degree[f] = S > 0.0 ? HS / S : 0.0;
        const int Ex = M ? (int)((M >> 23) & 0xffu) - 127 : 0;
        int lg = 0;
        while ((1LL << lg) < (long long)cells) ++lg;
        s_shift = 62 - (max(Ex, -126) + 1) - lg;
        shift[f] = s_shift;
        s_ncomp = 0;
    }
    // B (reads and writes only this wave's rows)
    for (int row = wave; row < gh; row += kFWaves) {
        int carry = -1;  // first cell of the run still open at the end of the last chunk
        for (int x0 = 0; x0 < gw; x0 += 64) {
            const int x = x0 + lane, c = row * gw + x;
            const bool hot = x < gw && P[c] >= 0;
            const uint64_t hm = __ballot(hot);
            const uint64_t cold_below = ~hm & ((1ull << lane) - 1ull);
            const int start = cold_below ? row * gw + x0 + (63 - __clzll(cold_below)) + 1
                                         : (carry >= 0 ? carry : row * gw + x0);
            if (hot) P[c] = start;
            const int s63 = __shfl(start, 63, 64);
            carry = ((hm >> 63) & 1ull) ? s63 : -1;
        }
    }
    __syncthreads();
    // C
    auto hotc = [&](int c) { return ld_rlx<kGroup>(P + c) >= 0; };
    for (int c = tid; c < cells - gw; c += kFThreads) {
        if (!hotc(c)) continue;
        const int gx = c % gw, d = c + gw;
        const bool dh = hotc(d);
        const bool lh = gx > 0 && hotc(c - 1), rh = gx + 1 < gw && hotc(c + 1);
        if (dh && !(lh && hotc(d - 1))) uf_unite<kGroup>(P, c, d);
        if (a.connectivity == 8 && !dh) {
            if (gx + 1 < gw && !rh && hotc(d + 1)) uf_unite<kGroup>(P, c, d + 1);
            if (gx > 0 && !lh && hotc(d - 1)) uf_unite<kGroup>(P, c, d - 1);
        }
    }
    __syncthreads();
    // D (loop bound rounded up to whole waves: the shuffles need every lane)
    const int sh = s_shift;
    const int cells_up = (cells + 63) & ~63;
    for (int c = tid; c < cells_up; c += kFThreads) {
        const bool in = c < cells;
        const int32_t p0 = in ? P[c] : -1;
        const int32_t r = p0 >= 0 ? uf_root<kGroup>(P, c) : -1;
        unsigned long long q = 0ull;
        if (r >= 0) {
            L[c] = r;
            q = (unsigned long long)llrint(ldexp((double)D[c], sh));
            if (r == c) roots[(size_t)f * cells + atomicAdd(&s_ncomp, 1)] = c;  // for heat_root_mass_kernel
        } else if (in) {
            L[c] = -1;
        }
        const int32_t prev = __shfl_up(r, 1, 64);
        const bool head = lane == 0 || prev != r;
        const uint64_t heads = __ballot(head);
        const uint64_t after = lane == 63 ? 0ull : heads >> (lane + 1);
        const int next = after ? lane + 1 + __ffsll((long long)after) - 1 : 64;  // next run's first lane
        const unsigned long long incl = wave_incl_scan_u64(q);
        const unsigned long long at_end = __shfl(incl, next - 1, 64);
        const unsigned long long before = __shfl(incl, lane > 0 ? lane - 1 : 0, 64);
        if (head && r >= 0) {
            atomicAdd(CC + r, next - lane);
            atomicAdd(CMu + r, at_end - (lane > 0 ? before : 0ull));
        }
    }
    __syncthreads();
    if (tid == 0) a.n_components[f] = s_ncomp;
}

}  // namespace

size_t heatmap_workspace_bytes(int32_t n_frames, int32_t grid_w, int32_t grid_h) {
    if (n_frames <= 0 || grid_w < 1 || grid_h < 1) return 0;
    const long long tiles = (long long)((grid_w + kHT - 1) / kHT) * ((grid_h + kHT - 1) / kHT);
    const size_t parts = ((size_t)n_frames * tiles * sizeof(TilePart) + 255) & ~(size_t)255;
    return parts + (((size_t)n_frames * sizeof(int32_t) + 255) & ~(size_t)255);
}

size_t heatmap_frame_lds_bytes(int32_t grid_w, int32_t grid_h) { return (size_t)grid_w * grid_h * sizeof(int32_t); }

// A shift per frame, then each frame's label cells (at most one per cell).
size_t heatmap_frame_workspace_bytes(int32_t n_frames, int32_t grid_w, int32_t grid_h) {
    if (n_frames <= 0 || grid_w < 1 || grid_h < 1) return 0;
    return (((size_t)n_frames * sizeof(int32_t) + 255) & ~(size_t)255) +
           (size_t)n_frames * grid_w * grid_h * sizeof(int32_t);
}

hipError_t launch_heatmap(HeatArgs a, void *workspace, bool resident, hipStream_t stream) {
    if (resident) {
        int32_t *shift = static_cast<int32_t *>(workspace);
        int32_t *roots = reinterpret_cast<int32_t *>(static_cast<unsigned char *>(workspace) +
                                                     (((size_t)a.n_frames * sizeof(int32_t) + 255) & ~(size_t)255));
        hipLaunchKernelGGL(heat_frame_kernel, dim3((unsigned)a.n_frames), dim3(kFThreads),
                           heatmap_frame_lds_bytes(a.grid_w, a.grid_h), stream, a, shift, roots);
        hipLaunchKernelGGL(heat_root_mass_kernel, dim3((unsigned)a.n_frames), dim3(256), 0, stream, a, shift, roots);
        return hipGetLastError();
    }
    a.tiles_x = (a.grid_w + kHT - 1) / kHT;
    a.tiles_y = (a.grid_h + kHT - 1) / kHT;
    const long long tiles = (long long)a.tiles_x * a.tiles_y * a.n_frames;
    TilePart *part = static_cast<TilePart *>(workspace);
    const size_t parts = ((size_t)tiles * sizeof(TilePart) + 255) & ~(size_t)255;
    int32_t *shift = reinterpret_cast<int32_t *>(static_cast<unsigned char *>(workspace) + parts);
    const long long per = 2LL * (a.tiles_x - 1) * a.grid_h + (long long)(a.tiles_y - 1) * a.grid_w;
    const long long merge_blocks = (per * a.n_frames + 255) / 256;
    const long long cells = (long long)a.grid_w * a.grid_h * a.n_frames;
    hipLaunchKernelGGL(heat_tile_kernel, dim3((unsigned)tiles), dim3(kHThreads), 0, stream, a, part);
    hipLaunchKernelGGL(heat_merge_kernel, dim3((unsigned)(merge_blocks + a.n_frames)), dim3(256), 0, stream, a,
                       part, shift, merge_blocks);
    hipLaunchKernelGGL(heat_label_kernel, dim3((unsigned)tiles), dim3(kHThreads), 0, stream, a, shift);
    hipLaunchKernelGGL(heat_mass_kernel, dim3((unsigned)((cells + 255) / 256)), dim3(256), 0, stream, a, shift);
    return hipGetLastError();
}

}  // namespace flock

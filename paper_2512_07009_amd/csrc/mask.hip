// mask.hip - detection post-processing: the segmentation output of every
// frame thresholded into foreground pixels (probability strictly above the
// threshold), grouped into 4- or 8-connected components, and each component
// listed with its statistics (Section 3.2 replaces region properties by a
// connected-components-with-statistics routine; Section 2.3 turns the
// components into boxes with confidence scores).
//
// A component is labelled by its first pixel in raster order and the list
// is in label order within each frame.  Five launches:
//   1. mask_tile_kernel, one workgroup per 64 x 64 tile.  Each wave loads 16
//      rows (one pixel per lane, 256 contiguous bytes per load) and ballots
//      give each row's foreground bits.  Horizontal runs are listed in raster
//      order; then one thread per run joins it, in an LDS union-find, with
//      each run of the row above that it touches (found from the row's bits
//      with two popcounts), so that all joins of the tile run at once.  The
//      root of a tree is its first run, which holds the piece's first pixel.
//      Pieces (the components restricted to the tile) are numbered in raster
//      order; area, sums of x and y, box and largest probability are
//      accumulated per run in LDS, then written as one record per piece.
//      The labels image gets each pixel's piece root, and the tile's outer
//      rows and columns get the piece's slot (for step 2);
//   2. mask_seam_kernel, one thread per pixel pair across a tile seam: pieces
//      that touch across the seam are united in a global lock-free
//      union-find over 64-bit keys (first pixel, slot), so that every tree's
//      root is the piece holding the component's first pixel;
//   3. mask_resolve_kernel, one wave per tile: each piece that is not a root
//      adds its record into its root's record (integer atomics: the results
//      do not depend on their order); each root sets its first pixel's bit
//      in a bitmap of the batch and counts itself in its block of 512 bits
//      and its superblock of 64 blocks;
//   4. each superblock's first rank, and per frame the rank of its first
//      pixel (the component offsets): in the finish kernel for batches of up
//      to 2^26 pixels (every workgroup scans the superblock counts in LDS),
//      else by mask_scan_kernel, one workgroup;
//   5. mask_finish_kernel, one workgroup per tile: each root writes its
//      component at its rank (the number of roots before its first pixel),
//      and the pixels of the other pieces get their root's label (one wave
//      per piece, within the piece's box).
// Every access is bounded by the tile, the seam arrays or the slot ranges,
// whatever the probabilities are.

#include "cluster_common.h"
#include "internal.h"

namespace flock {
namespace {

using cl::kAgent;
using cl::kGroup;

constexpr int kT = kMaskTile;                   // tile side, px
constexpr int kMThreads = 256;                  // tile workgroup
constexpr int kRows = kT / (kMThreads / 64);    // rows per wave
constexpr int kAccCap = 128;                    // pieces accumulated in LDS per pass
constexpr int kMaxRuns = kT * kT / 2;           // runs a tile can hold
constexpr int kRunsPerThread = kMaxRuns / kMThreads;
constexpr int kBitBlock = 512;                  // bits per count block
constexpr int kBitWords = kBitBlock / 32;
constexpr int kSuper = 64;                      // blocks per superblock
constexpr int kRelabel = 16;                    // relabelled pixels per lane per pass
constexpr int kSuperBits = kBitBlock * kSuper;
constexpr int kLocalSuper = 2048;               // superblocks the finish kernel scans itself (2^26 pixels)

static_assert(kT == 64, "one lane per column of a tile");
static_assert(kAccCap <= kMThreads, "one record per thread per pass");

// Statistics of one piece, then (for a root) of its whole component.
struct MaskRec {
    uint64_t sx, sy;      // sums of x and y over the pixels (frame px)
    uint32_t area;
    uint32_t x0, y0, x1, y1;  // inclusive box
    uint32_t score;       // bits of the largest probability (> 0, so ordered as integers)
    uint32_t root;        // frame pixel index of the piece's first pixel
    uint32_t pad;
};
static_assert(sizeof(MaskRec) == 48, "record layout");

struct MaskAcc {         // LDS accumulator, tile coordinates
    uint32_t area, sx, sy, x0, x1, y1, score, root;
};

struct MaskWs {
    uint64_t *gp;         // [slots] key of the parent: first pixel << 32 | slot
    MaskRec *rec;         // [slots]
    int32_t *tile_np;     // [n_tiles] pieces per tile
    int32_t *hseam;       // [F][tiles_y][2][W] slots of each band's top and bottom rows
    int32_t *vseam;       // [F][tiles_x][2][H] slots of each column's left and right columns
    uint32_t *bitmap;     // [nwords] first pixels of the components
    int32_t *bcount;      // [nbp] components per block of kBitBlock bits
    int32_t *sbcount;     // [nsb] components per superblock of kSuper blocks
    int32_t *sbbase;      // [nsb + 1] components before each superblock
    int64_t nwords, nbp;
    int32_t nsb;
};

__device__ __forceinline__ uint64_t bits_upto(int x) { return x >= 63 ? ~0ull : ((2ull << x) - 1); }

// First pixel of the run of set bits of m that contains bit x.
__device__ __forceinline__ int run_first(uint64_t m, int x) {
    const uint64_t st = m & ~(m << 1);
    return 63 - __builtin_clzll(st & bits_upto(x));
}

// Last pixel of the run of set bits of m that contains bit x.
__device__ __forceinline__ int run_last(uint64_t m, int x) {
    const uint64_t en = m & ~(m >> 1);
    return x + __builtin_ctzll(en >> x);
}

struct TileLoc {
    int f, tx, ty, X0, Y0, tw, th;
    int64_t base;  // first slot of the tile
};

// Slots of a tile hold at most as many pieces as the tile can: with 8
// neighbours every 2 x 2 block of pixels meets one piece at most, with 4 every
// domino of a domino tiling does.  Tiles are laid out frame by frame, band by
// band, so the slot base follows from the tile position in closed form.
__device__ __forceinline__ TileLoc tile_loc(const MaskArgs &a, int64_t tile) {
    TileLoc t;  // 32-bit arithmetic: tiles number below 2^31
    const uint32_t tl = (uint32_t)tile, tx = (uint32_t)a.tiles_x, ty = (uint32_t)a.tiles_y;
    t.tx = (int)(tl % tx);
    const uint32_t rest = tl / tx;
    t.ty = (int)(rest % ty);
    t.f = (int)(rest / ty);
    t.X0 = t.tx * kT;
    t.Y0 = t.ty * kT;
    t.tw = min(kT, a.width - t.X0);
    t.th = min(kT, a.height - t.Y0);
    const int64_t in_band = a.connectivity == 8 ? (int64_t)(kT / 2) * ((t.th + 1) / 2) : (int64_t)(kT / 2) * t.th;
    t.base = (int64_t)t.f * a.frame_slots + (int64_t)t.ty * a.band_slots + in_band * t.tx;
    return t;
}

__device__ __forceinline__ int64_t tile_cap(const MaskArgs &a, const TileLoc &t) {
    return a.connectivity == 8 ? (int64_t)((t.tw + 1) / 2) * ((t.th + 1) / 2) : ((int64_t)t.tw * t.th + 1) / 2;
}

__global__ __launch_bounds__(kMThreads) void mask_tile_kernel(MaskArgs a, MaskWs w) {
    __shared__ uint64_t s_mask[kT];
    __shared__ int32_t s_rowbase[kT + 1];    // first run id of each row; [kT] = number of runs
    __shared__ int32_t s_side[2][kT];        // slots of the tile's left and right columns
    __shared__ uint16_t s_run[kMaxRuns];     // row | first pixel << 6
    __shared__ int32_t s_P[kMaxRuns];        // union-find over runs, then piece | first pixel << 11
    __shared__ uint32_t s_rmax[kMaxRuns];    // largest probability of each run (bits; > 0, ordered as integers)
    __shared__ MaskAcc s_acc[kAccCap];
    __shared__ int32_t s_wtot[kMThreads / 64];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: rows are scalar values
    const TileLoc t = tile_loc(a, blockIdx.x);
    const int64_t WH = (int64_t)a.width * a.height;
    const int64_t fbase = (int64_t)t.f * WH;
    const uint64_t le = bits_upto(lane);  // lanes 0 .. lane

    // 1. rows: foreground bits by ballot
    const bool col_ok = lane < t.tw;
    const float *src = a.prob + fbase + (int64_t)t.Y0 * a.width + t.X0;  // the tile's first row
    float v[kRows];
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        const float *row = src + (int64_t)r * a.width;
        v[i] = (col_ok && r < t.th) ? row[lane] : 0.0f;
    }
    // the bitmap and block counts of steps 3-4 start at zero
    {
        const int64_t g = (int64_t)blockIdx.x * kMThreads + tid;
        const int64_t stride = (int64_t)gridDim.x * kMThreads;
        for (int64_t j = g; j < w.nwords; j += stride) w.bitmap[j] = 0u;
        for (int64_t j = g; j < w.nbp; j += stride) w.bcount[j] = 0;
        for (int64_t j = g; j < w.nsb; j += stride) w.sbcount[j] = 0;
    }
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        const uint64_t mr = __ballot(col_ok && r < t.th && v[i] > a.threshold);
        if (lane == 0) s_mask[r] = mr;
    }
    __syncthreads();

    // 2. runs, numbered in raster order, with their largest probabilities
    //    (the ballots are taken again: row masks do not stay in scalar registers)
    {
        const uint64_t ml = s_mask[lane];
        const int c = __popcll(ml & ~(ml << 1));
        int inc = c;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int u = __shfl_up(inc, o, 64);
            if (lane >= o) inc += u;
        }
        const int excl = inc - c;
        if (wave == 0) {
            s_rowbase[lane] = excl;
            if (lane == 63) s_rowbase[kT] = inc;
        }
#pragma unroll
        for (int i = 0; i < kRows; ++i) {
            const int r = wave * kRows + i;
            const bool fg = col_ok && r < t.th && v[i] > a.threshold;
            const uint64_t mr = __ballot(fg);
            const int rbr = __builtin_amdgcn_readlane(excl, r);  // first run id of row r
            const uint64_t st = mr & ~(mr << 1);
            const int id = rbr + __popcll(st & le) - 1;
            if ((st >> lane) & 1) {
                s_run[id] = (uint16_t)(r | lane << 6);
                s_P[id] = id;
                s_rmax[id] = 0u;
            }
            // after the run's first lane cleared it: one wave's LDS operations run in order
            if (fg) atomicMax(&s_rmax[id], __float_as_uint(v[i]));
        }
    }
    __syncthreads();
    const int nruns = s_rowbase[kT];

    // 3. each run joins the runs above it that it touches (with 8 neighbours
    //    one pixel further on either side); the root of a tree is its first
    //    run in raster order, which holds the piece's first pixel
    const bool eight = a.connectivity == 8;
    for (int j = tid; j < nruns; j += kMThreads) {
        const int ru = s_run[j];
        const int r = ru & 63, s0 = ru >> 6;
        if (r == 0) continue;
        const int s1 = run_last(s_mask[r], s0);
        const int lo = eight && s0 > 0 ? s0 - 1 : s0, hi = eight && s1 < kT - 1 ? s1 + 1 : s1;
        const uint64_t mu = s_mask[r - 1];
        const uint64_t win = mu & bits_upto(hi) & ~(bits_upto(lo) >> 1);
        if (!win) continue;
        // ids of the runs above holding the window's first and last set bits
        const uint64_t st = mu & ~(mu << 1);
        const int a0 = __popcll(st & bits_upto(__builtin_ctzll(win)));
        const int a1 = __popcll(st & bits_upto(63 - __builtin_clzll(win)));
        int base = j - 1;  // the row above's first run: count back over this row's earlier runs
        base -= __popcll(s_mask[r] & ~(s_mask[r] << 1) & (bits_upto(s0) >> 1));
        base -= __popcll(st);
        for (int k = base + a0; k <= base + a1; ++k) cl::uf_unite<kGroup>(s_P, j, k);
    }
    __syncthreads();

    // 4. flatten (run j = tid + k * kMThreads on this thread), number the
    //    pieces in raster order of their first runs, kMThreads runs a pass,
    //    and give every run its piece and the piece's first pixel
    int rt[kRunsPerThread];
#pragma unroll
    for (int k = 0; k < kRunsPerThread; ++k) {
        const int j = tid + k * kMThreads;
        rt[k] = j < nruns ? cl::uf_find<kGroup>(s_P, j) : -1;
    }
    __syncthreads();
    int np = 0;
#pragma unroll
    for (int k = 0; k < kRunsPerThread; ++k) {
        if (k * kMThreads >= nruns) break;
        const int j = tid + k * kMThreads;
        const bool is_first = rt[k] == j;
        const uint64_t b = __ballot(is_first);
        if (lane == 63) s_wtot[wave] = __popcll(b);
        __syncthreads();
        int before = np, total = 0;
#pragma unroll
        for (int q = 0; q < kMThreads / 64; ++q) {
            const int c = s_wtot[q];
            before += q < wave ? c : 0;
            total += c;
        }
        if (is_first) {
            const int ru = s_run[j];
            const int fp = (ru & 63) * kT + (ru >> 6);
            s_P[j] = (before + __popcll(b & (le >> 1))) | fp << 11;
        }
        np += total;
        __syncthreads();
    }
#pragma unroll
    for (int k = 0; k < kRunsPerThread; ++k) {
        const int j = tid + k * kMThreads;
        if (j < nruns && rt[k] != j) s_P[j] = s_P[rt[k]];
    }
    __syncthreads();

    // 5. labels (the piece's first pixel for now) and the tile's outer slots
    const int64_t cap = tile_cap(a, t);
    const int32_t lab0 = t.Y0 * a.width + t.X0;  // frame index of the tile's first pixel
    int32_t *lrow0 = a.labels ? a.labels + fbase + lab0 : nullptr;
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        if (r >= t.th) continue;
        const uint64_t ml = s_mask[r];  // reloaded: the row masks do not stay in scalar registers
        const uint64_t mr = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)ml) |
                            (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(ml >> 32)) << 32;
        const uint64_t st = mr & ~(mr << 1);
        const bool fg = (mr >> lane) & 1;
        const int pk = fg ? s_P[s_rowbase[r] + __popcll(st & le) - 1] : -1;
        const int pc = pk & 0x7ff, fp = pk >> 11;
        const int32_t lab = fg ? lab0 + (int32_t)__umul24((uint32_t)(fp >> 6), (uint32_t)a.width) + (fp & 63) : -1;
        const int32_t slot = fg && pc < cap ? (int32_t)t.base + pc : -1;
        if (lrow0 && col_ok) lrow0[(int64_t)r * a.width + lane] = lab;
        if (r == 0 && col_ok) w.hseam[((int64_t)(t.f * a.tiles_y + t.ty) * 2 + 0) * a.width + t.X0 + lane] = slot;
        if (r == t.th - 1 && col_ok)
            w.hseam[((int64_t)(t.f * a.tiles_y + t.ty) * 2 + 1) * a.width + t.X0 + lane] = slot;
        if (lane == 0) s_side[0][r] = slot;
        if (lane == t.tw - 1) s_side[1][r] = slot;
    }
    __syncthreads();
    if (wave < 2 && lane < t.th)
        w.vseam[((int64_t)(t.f * a.tiles_x + t.tx) * 2 + wave) * a.height + t.Y0 + lane] = s_side[wave][lane];

    // 6. statistics per run, kAccCap pieces per pass
    for (int c0 = 0; c0 < np; c0 += kAccCap) {
        if (tid < kAccCap) s_acc[tid] = MaskAcc{0u, 0u, 0u, 63u, 0u, 0u, 0u, 0u};
        __syncthreads();
        for (int j = tid; j < nruns; j += kMThreads) {
            const int pk = s_P[j];
            const int p = (pk & 0x7ff) - c0;
            if (p < 0 || p >= kAccCap) continue;
            const int ru = s_run[j];
            const int r = ru & 63, s0 = ru >> 6;
            const int s1 = run_last(s_mask[r], s0);
            const uint32_t len = (uint32_t)(s1 - s0 + 1);
            MaskAcc &q = s_acc[p];
            atomicAdd(&q.area, len);
            atomicAdd(&q.sx, (uint32_t)(s0 + s1) * len / 2u);
            atomicAdd(&q.sy, len * (uint32_t)r);
            atomicMin(&q.x0, (uint32_t)s0);
            atomicMax(&q.x1, (uint32_t)s1);
            atomicMax(&q.y1, (uint32_t)r);
            atomicMax(&q.score, s_rmax[j]);
            if (r * kT + s0 == (pk >> 11)) q.root = (uint32_t)(pk >> 11);
        }
        __syncthreads();
        const int p = c0 + tid;
        if (tid < kAccCap && p < np && p < cap) {
            const MaskAcc q = s_acc[tid];
            const int ry = (int)(q.root / kT), rx = (int)(q.root % kT);
            const int64_t fl = (int64_t)(t.Y0 + ry) * a.width + t.X0 + rx;
            const int64_t slot = t.base + p;
            MaskRec R;
            R.sx = (uint64_t)q.sx + (uint64_t)q.area * (uint64_t)t.X0;
            R.sy = (uint64_t)q.sy + (uint64_t)q.area * (uint64_t)t.Y0;
            R.area = q.area;
            R.x0 = q.x0 + t.X0;
            R.y0 = (uint32_t)(ry + t.Y0);
            R.x1 = q.x1 + t.X0;
            R.y1 = q.y1 + t.Y0;
            R.score = q.score;
            R.root = (uint32_t)fl;
            R.pad = 0u;
            w.rec[slot] = R;
            w.gp[slot] = ((uint64_t)(fbase + fl) << 32) | (uint64_t)slot;
        }
        __syncthreads();
    }
    if (tid == 0) w.tile_np[blockIdx.x] = (int32_t)min((int64_t)np, cap);
}

__device__ __forceinline__ uint64_t ld64(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, kAgent);
}

// Key of the root of slot s's tree, halving the path on the way: a slot
// is pointed at its grandparent, an ancestor with a smaller key.
__device__ __forceinline__ uint64_t key_root(uint64_t *gp, uint32_t s) {
    for (;;) {
        const uint64_t k = ld64(gp + s);
        if ((uint32_t)k == s) return k;
        const uint64_t g = ld64(gp + (uint32_t)k);
        if ((uint32_t)g == (uint32_t)k) return g;
        __hip_atomic_store(gp + s, g, __ATOMIC_RELAXED, kAgent);
        s = (uint32_t)g;
    }
}

// Key of the root of slot s's tree, without writes: where other threads set
// slots straight to their roots, a halving step could put back an older
// ancestor over such a store.
__device__ __forceinline__ uint64_t key_root_ro(const uint64_t *gp, uint32_t s) {
    uint64_t k = ld64(gp + s);
    while ((uint32_t)k != s) {
        s = (uint32_t)k;
        k = ld64(gp + s);
    }
    return k;
}

// Unite the trees of slots a and b, hooking the root with the larger key
// under the smaller: every parent key is below its child's, so the root of
// a tree is its smallest first pixel.
__device__ __forceinline__ void key_unite(uint64_t *gp, uint32_t a, uint32_t b) {
    for (;;) {
        uint64_t ka = key_root(gp, a), kb = key_root(gp, b);
        if (ka == kb) return;
        if (ka > kb) {
            const uint64_t u = ka;
            ka = kb;
            kb = u;
        }
        uint64_t expected = kb;
        if (__hip_atomic_compare_exchange_strong(gp + (uint32_t)kb, &expected, ka, __ATOMIC_RELAXED,
                                                 __ATOMIC_RELAXED, kAgent))
            return;
        a = (uint32_t)ka;
        b = (uint32_t)kb;
    }
}

// Slots P[i] and Q[i-1..i+1] (Q[i] only with 4 neighbours) face each other
// across a seam; each touching pair is united at its first position along
// the seam.
__device__ __forceinline__ void join_seam(uint64_t *gp, const int32_t *P, const int32_t *Q, int i, int n,
                                          bool eight) {
    const int32_t p = P[i];
    if (p < 0) return;
    const int32_t pp = i > 0 ? P[i - 1] : -1;
    int32_t prevq = -1;
    for (int d = eight ? -1 : 0; d <= (eight ? 1 : 0); ++d) {
        const int j = i + d;
        if (j < 0 || j >= n) continue;
        const int32_t q = Q[j];
        if (q < 0 || q == prevq) {
            prevq = q;
            continue;
        }
        prevq = q;
        if (pp == p && j > 0 && Q[j - 1] == q) continue;  // same pair one step back
        key_unite(gp, (uint32_t)p, (uint32_t)q);
    }
}

__global__ __launch_bounds__(256) void mask_seam_kernel(MaskArgs a, MaskWs w, int64_t nh, int64_t nv) {
    int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const bool eight = a.connectivity == 8;
    if (g < nh) {  // 32-bit arithmetic: seam positions number below 2^31
        const uint32_t gu = (uint32_t)g, wu = (uint32_t)a.width, bands = (uint32_t)(a.tiles_y - 1);
        const int x = (int)(gu % wu);
        const uint32_t fb = gu / wu;
        const int f = (int)(fb / bands), b = (int)(fb % bands);
        const int32_t *up = w.hseam + ((int64_t)(f * a.tiles_y + b) * 2 + 1) * a.width;
        const int32_t *dn = w.hseam + ((int64_t)(f * a.tiles_y + b + 1) * 2 + 0) * a.width;
        join_seam(w.gp, up, dn, x, a.width, eight);
        return;
    }
    g -= nh;
    if (g < nv) {
        const uint32_t gu = (uint32_t)g, hu = (uint32_t)a.height, cols = (uint32_t)(a.tiles_x - 1);
        const int y = (int)(gu % hu);
        const uint32_t fc = gu / hu;
        const int f = (int)(fc / cols), c = (int)(fc % cols);
        const int32_t *le = w.vseam + ((int64_t)(f * a.tiles_x + c) * 2 + 1) * a.height;
        const int32_t *ri = w.vseam + ((int64_t)(f * a.tiles_x + c + 1) * 2 + 0) * a.height;
        join_seam(w.gp, le, ri, y, a.height, eight);
    }
}

__global__ __launch_bounds__(64) void mask_resolve_kernel(MaskArgs a, MaskWs w) {
    const TileLoc t = tile_loc(a, blockIdx.x);
    const int np = w.tile_np[blockIdx.x];
    for (int p = threadIdx.x; p < np; p += 64) {
        const uint32_t s = (uint32_t)(t.base + p);
        const MaskRec R = w.rec[s];  // in flight during the root search
        const uint64_t own = ld64(w.gp + s);
        if ((uint32_t)own == s) {
            const uint64_t g = own >> 32;
            atomicOr(w.bitmap + (g >> 5), 1u << (g & 31));
            atomicAdd(w.bcount + (g / kBitBlock), 1);
            atomicAdd(w.sbcount + (g / kSuperBits), 1);
            continue;
        }
        const uint64_t rk = key_root_ro(w.gp, s);
        __hip_atomic_store(w.gp + s, rk, __ATOMIC_RELAXED, kAgent);  // step 5 reads the root here
        MaskRec *D = w.rec + (uint32_t)rk;
        // the root holds the component's first pixel, hence its top row
        atomicAdd(&D->area, R.area);
        atomicAdd((unsigned long long *)&D->sx, (unsigned long long)R.sx);
        atomicAdd((unsigned long long *)&D->sy, (unsigned long long)R.sy);
        atomicMin(&D->x0, R.x0);
        atomicMax(&D->x1, R.x1);
        atomicMax(&D->y1, R.y1);
        atomicMax(&D->score, R.score);
    }
}

// Components whose first pixel lies before bit b of the batch: the count
// before b's superblock, the counts of the blocks before b's block in that
// superblock, and the bits before b in its block.  Every load is 16 bytes
// wide and unconditional (the counts are padded to whole superblocks, the
// bitmap to whole blocks plus one), so that they are all in flight at once;
// the parts beyond b are masked off afterwards.
__device__ __forceinline__ int32_t rank_before(const MaskWs &w, const int32_t *sbbase, int64_t b) {
    const int64_t sb = b / kSuperBits;
    const int32_t base = sbbase[sb];
    if (b % kSuperBits == 0) return base;  // also b = total on a superblock edge
    const int64_t blk = b / kBitBlock;
    const int4 *cq = reinterpret_cast<const int4 *>(w.bcount) + sb * (kSuper / 4);
    const uint4 *bq = reinterpret_cast<const uint4 *>(w.bitmap) + blk * (kBitWords / 4);
    int4 c[kSuper / 4];
    uint4 u[kBitWords / 4];
#pragma unroll
    for (int q = 0; q < kSuper / 4; ++q) c[q] = cq[q];
#pragma unroll
    for (int q = 0; q < kBitWords / 4; ++q) u[q] = bq[q];
    const int nblk = (int)(blk - sb * kSuper);  // whole blocks before b in the superblock
    int32_t r = base;
#pragma unroll
    for (int q = 0; q < kSuper / 4; ++q) {
        r += (4 * q < nblk ? c[q].x : 0) + (4 * q + 1 < nblk ? c[q].y : 0) + (4 * q + 2 < nblk ? c[q].z : 0) +
             (4 * q + 3 < nblk ? c[q].w : 0);
    }
    const int bit = (int)(b - blk * kBitBlock);  // bits before b in its block
#pragma unroll
    for (int q = 0; q < kBitWords / 4; ++q) {
        const uint32_t wd[4] = {u[q].x, u[q].y, u[q].z, u[q].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int lo = 32 * (4 * q + e);
            const uint32_t keep = bit >= lo + 32 ? ~0u : bit > lo ? (1u << (bit - lo)) - 1u : 0u;
            r += __popc(wd[e] & keep);
        }
    }
    return r;
}

__global__ __launch_bounds__(1024) void mask_scan_kernel(MaskArgs a, MaskWs w) {
    __shared__ int s_wave[16];
    constexpr int kBatch = 8;  // counts loaded together
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nb = w.nsb;
    const int per = (nb + 1023) / 1024;
    const int b0 = min(tid * per, nb), b1 = min(b0 + per, nb);
    int sum = 0;
    for (int b = b0; b < b1; b += kBatch) {
        int c[kBatch];
#pragma unroll
        for (int q = 0; q < kBatch; ++q) c[q] = b + q < b1 ? w.sbcount[b + q] : 0;
#pragma unroll
        for (int q = 0; q < kBatch; ++q) sum += c[q];
    }
    int inc = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(inc, o, 64);
        if (lane >= o) inc += u;
    }
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    int run = inc - sum;
    for (int k = 0; k < wave; ++k) run += s_wave[k];
    for (int b = b0; b < b1; b += kBatch) {
        int c[kBatch];
#pragma unroll
        for (int q = 0; q < kBatch; ++q) c[q] = b + q < b1 ? w.sbcount[b + q] : 0;
#pragma unroll
        for (int q = 0; q < kBatch; ++q)
            if (b + q < b1) {
                w.sbbase[b + q] = run;
                run += c[q];
            }
    }
    if (tid == 1023) w.sbbase[nb] = run;
    __syncthreads();
    const int64_t WH = (int64_t)a.width * a.height;
    for (int f = tid; f <= a.n_frames; f += 1024) {
        const int32_t r0 = rank_before(w, w.sbbase, (int64_t)f * WH);
        a.comp_offsets[f] = r0;
        if (f < a.n_frames) a.n_components[f] = rank_before(w, w.sbbase, (int64_t)(f + 1) * WH) - r0;
    }
}

__global__ __launch_bounds__(kMThreads) void mask_finish_kernel(MaskArgs a, MaskWs w) {
    __shared__ int32_t s_list[kT * kT / 2];
    __shared__ int32_t s_sbb[kLocalSuper + 1];
    __shared__ int s_wtot[kMThreads / 64];
    __shared__ int32_t s_n;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const TileLoc t = tile_loc(a, blockIdx.x);
    const int np = w.tile_np[blockIdx.x];
    const int64_t WH = (int64_t)a.width * a.height;
    const int64_t fbase = (int64_t)t.f * WH;
    if (tid == 0) s_n = 0;
    // the superblock bases: scanned here from the counts when they fit in
    // LDS (no separate scan launch), else read from the scan kernel
    const int32_t *sbbase = w.sbbase;
    if (w.nsb <= kLocalSuper) {
        constexpr int kPer = kLocalSuper / kMThreads;
        int c[kPer], sum = 0;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int i = tid * kPer + q;
            c[q] = i < w.nsb ? w.sbcount[i] : 0;
            sum += c[q];
        }
        int run = cl::block_exclusive_scan(sum, s_wtot);  // holds barriers
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            s_sbb[tid * kPer + q] = run;
            run += c[q];
        }
        if (tid == kMThreads - 1) s_sbb[kLocalSuper] = run;
        sbbase = s_sbb;
    }
    __syncthreads();
    if (w.nsb <= kLocalSuper) {
        // frame offsets and counts: frame f's by workgroup f (there are at
        // least as many tiles as frames)
        for (int f = blockIdx.x; f <= a.n_frames && tid == 0; f += gridDim.x) {
            const int32_t r0 = rank_before(w, sbbase, (int64_t)f * WH);
            a.comp_offsets[f] = r0;
            if (f < a.n_frames) a.n_components[f] = rank_before(w, sbbase, (int64_t)(f + 1) * WH) - r0;
        }
    }
    for (int p = tid; p < np; p += kMThreads) {
        const uint32_t s = (uint32_t)(t.base + p);
        const uint64_t k = w.gp[s];
        if ((uint32_t)k != s) {
            if (a.labels) {
                // a piece that is not its component's first: its pixels carry
                // the piece's own first pixel, to be replaced by the root's
                s_list[atomicAdd(&s_n, 1)] = p;
            }
            continue;
        }
        const MaskRec R = w.rec[s];  // in flight with the rank's loads
        const int64_t rank = rank_before(w, sbbase, (int64_t)(k >> 32));
        if (rank >= a.capacity) continue;
        if (a.comp_label) a.comp_label[rank] = (int32_t)R.root;
        if (a.comp_area) a.comp_area[rank] = (int32_t)R.area;
        if (a.comp_box)
            reinterpret_cast<int4 *>(a.comp_box)[rank] =
                make_int4((int)R.x0, (int)R.y0, (int)(R.x1 - R.x0 + 1), (int)(R.y1 - R.y0 + 1));
        if (a.comp_centroid)
            reinterpret_cast<double2 *>(a.comp_centroid)[rank] =
                make_double2((double)R.sx / (double)R.area, (double)R.sy / (double)R.area);
        if (a.comp_xy)
            reinterpret_cast<int2 *>(a.comp_xy)[rank] =
                make_int2((int)((16ull * R.sx) / R.area), (int)((16ull * R.sy) / R.area));
        if (a.comp_score) a.comp_score[rank] = __uint_as_float(R.score);
    }
    if (!a.labels) return;
    __syncthreads();
    // each wave relabels one piece's box at a time, kRelabel pixels per lane
    // in flight (loads first, then stores)
    const int n = s_n;
    for (int q = wave; q < n; q += kMThreads / 64) {
        const uint32_t s = (uint32_t)(t.base + s_list[q]);
        const MaskRec R = w.rec[s];
        const int32_t old = (int32_t)R.root;
        const int32_t lab = (int32_t)((int64_t)(w.gp[s] >> 32) - fbase);
        const int bw = (int)(R.x1 - R.x0 + 1), nb = bw * (int)(R.y1 - R.y0 + 1);
        int32_t *row0 = a.labels + fbase + (int64_t)R.y0 * a.width + R.x0;
        for (int e0 = 0; e0 < nb; e0 += 64 * kRelabel) {
            int32_t cur[kRelabel];
            int64_t at[kRelabel];
#pragma unroll
            for (int u = 0; u < kRelabel; ++u) {
                const int e = e0 + u * 64 + lane;
                const int ey = e / bw;
                at[u] = (int64_t)ey * a.width + (e - ey * bw);
                cur[u] = e < nb ? row0[at[u]] : -1;
            }
#pragma unroll
            for (int u = 0; u < kRelabel; ++u)
                if (e0 + u * 64 + lane < nb && cur[u] == old) row0[at[u]] = lab;
        }
    }
}

struct MaskLayout {
    int64_t slots, n_tiles;
    int64_t nwords, nbp;
    int32_t nsb;
    size_t off_gp, off_rec, off_np, off_hs, off_vs, off_bits, off_bc, off_sbc, off_sbb, bytes;
};

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

void mask_geometry(MaskArgs &a) {
    a.tiles_x = (a.width + kT - 1) / kT;
    a.tiles_y = (a.height + kT - 1) / kT;
    a.n_tiles = (int64_t)a.n_frames * a.tiles_x * a.tiles_y;
    const int tw_last = a.width - (a.tiles_x - 1) * kT, th_last = a.height - (a.tiles_y - 1) * kT;
    if (a.connectivity == 8) {
        const int64_t sx = (int64_t)(kT / 2) * (a.tiles_x - 1) + (tw_last + 1) / 2;
        const int64_t sy = (int64_t)(kT / 2) * (a.tiles_y - 1) + (th_last + 1) / 2;
        a.band_slots = (kT / 2) * sx;
        a.frame_slots = sx * sy;
    } else {
        a.band_slots = (int64_t)(kT / 2) * a.width;
        a.frame_slots = a.band_slots * (a.tiles_y - 1) + (int64_t)(kT / 2) * th_last * (a.tiles_x - 1) +
                        ((int64_t)tw_last * th_last + 1) / 2;
    }
}

MaskLayout mask_layout(const MaskArgs &a) {
    MaskLayout L;
    L.n_tiles = a.n_tiles;
    L.slots = (int64_t)a.n_frames * a.frame_slots;
    const int64_t total = (int64_t)a.n_frames * a.width * a.height;
    const int64_t nb = (total + kBitBlock - 1) / kBitBlock;
    L.nsb = (int32_t)((total + kSuperBits - 1) / kSuperBits);
    L.nbp = (int64_t)L.nsb * kSuper;      // whole superblocks, for the 16-byte loads
    L.nwords = (nb + 1) * kBitWords;      // whole blocks and one more, for the 16-byte loads
    size_t o = 0;
    L.off_gp = o;
    o += align256((size_t)L.slots * sizeof(uint64_t));
    L.off_rec = o;
    o += align256((size_t)L.slots * sizeof(MaskRec));
    L.off_np = o;
    o += align256((size_t)L.n_tiles * sizeof(int32_t));
    L.off_hs = o;
    o += align256((size_t)a.n_frames * a.tiles_y * 2 * a.width * sizeof(int32_t));
    L.off_vs = o;
    o += align256((size_t)a.n_frames * a.tiles_x * 2 * a.height * sizeof(int32_t));
    L.off_bits = o;
    o += align256((size_t)L.nwords * sizeof(uint32_t));
    L.off_bc = o;
    o += align256((size_t)L.nbp * sizeof(int32_t));
    L.off_sbc = o;
    o += align256((size_t)L.nsb * sizeof(int32_t));
    L.off_sbb = o;
    o += align256((size_t)(L.nsb + 1) * sizeof(int32_t));
    L.bytes = o;
    return L;
}

}  // namespace

size_t mask_workspace_bytes(int32_t n_frames, int32_t width, int32_t height, int32_t connectivity) {
    if (n_frames <= 0 || width < 1 || height < 1) return 0;
    MaskArgs a{};
    a.n_frames = n_frames;
    a.width = width;
    a.height = height;
    a.connectivity = connectivity == 4 ? 4 : 8;
    mask_geometry(a);
    return mask_layout(a).bytes;
}

hipError_t launch_mask(MaskArgs a, void *workspace, hipStream_t stream) {
    mask_geometry(a);
    const MaskLayout L = mask_layout(a);
    char *base = static_cast<char *>(workspace);
    MaskWs w;
    w.gp = reinterpret_cast<uint64_t *>(base + L.off_gp);
    w.rec = reinterpret_cast<MaskRec *>(base + L.off_rec);
    w.tile_np = reinterpret_cast<int32_t *>(base + L.off_np);
    w.hseam = reinterpret_cast<int32_t *>(base + L.off_hs);
    w.vseam = reinterpret_cast<int32_t *>(base + L.off_vs);
    w.bitmap = reinterpret_cast<uint32_t *>(base + L.off_bits);
    w.bcount = reinterpret_cast<int32_t *>(base + L.off_bc);
    w.sbcount = reinterpret_cast<int32_t *>(base + L.off_sbc);
    w.sbbase = reinterpret_cast<int32_t *>(base + L.off_sbb);
    w.nwords = L.nwords;
    w.nbp = L.nbp;
    w.nsb = L.nsb;
    const unsigned tiles = (unsigned)L.n_tiles;
    hipLaunchKernelGGL(mask_tile_kernel, dim3(tiles), dim3(kMThreads), 0, stream, a, w);
    const int64_t nh = (int64_t)a.n_frames * (a.tiles_y - 1) * a.width;
    const int64_t nv = (int64_t)a.n_frames * (a.tiles_x - 1) * a.height;
    if (nh + nv > 0)
        hipLaunchKernelGGL(mask_seam_kernel, dim3((unsigned)((nh + nv + 255) / 256)), dim3(256), 0, stream, a, w,
                           nh, nv);
    hipLaunchKernelGGL(mask_resolve_kernel, dim3(tiles), dim3(64), 0, stream, a, w);
    if (w.nsb > kLocalSuper) hipLaunchKernelGGL(mask_scan_kernel, dim3(1), dim3(1024), 0, stream, a, w);
    hipLaunchKernelGGL(mask_finish_kernel, dim3(tiles), dim3(kMThreads), 0, stream, a, w);
    return hipGetLastError();
}

}  // namespace flock

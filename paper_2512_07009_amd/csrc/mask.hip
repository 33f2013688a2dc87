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
//      rows (one pixel per lane, 256 contiguous bytes per load), ballots give
//      the row's foreground bits, horizontal runs come from bit operations,
//      and runs of neighbouring rows are joined once per touching pair in an
//      LDS union-find whose root is the piece's first pixel.  Pieces (the
//      components restricted to the tile) are numbered in raster order of
//      their first pixel; area, sums of x and y, box and largest
//      probability are accumulated per run in LDS, then written as one record
//      per piece.  The labels image gets each pixel's piece root, and the
//      tile's outer rows and columns get the piece's slot (for step 2);
//   2. mask_seam_kernel, one thread per pixel pair across a tile seam: pieces
//      that touch across the seam are united in a global lock-free
//      union-find over 64-bit keys (first pixel, slot), so that every tree's
//      root is the piece holding the component's first pixel;
//   3. mask_resolve_kernel, one wave per tile: each piece that is not a root
//      adds its record into its root's record (integer atomics: the results
//      do not depend on their order); each root sets its first pixel's bit
//      in a bitmap of the batch and counts itself in its block of 1024 bits;
//   4. mask_scan_kernel, one workgroup: each block's first rank, and per
//      frame the rank of its first pixel (the component offsets);
//   5. mask_finish_kernel, one workgroup per tile: each root writes its
//      component at its rank (the number of roots before its first pixel),
//      and each other piece relabels its own pixels inside its box.
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
constexpr int kAccCap = 256;                    // pieces accumulated in LDS per pass
constexpr int kBitBlock = 1024;                 // bits per count block
constexpr int kBitWords = kBitBlock / 32;

static_assert(kT == 64, "one lane per column of a tile");
static_assert(kAccCap == kMThreads, "one record per thread per pass");

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
    int32_t *bcount;      // [nb] components per block of kBitBlock bits
    int32_t *bbase;       // [nb + 1] components before each block
    int64_t nwords;
    int32_t nb;
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
    TileLoc t;
    t.tx = (int)(tile % a.tiles_x);
    const int64_t rest = tile / a.tiles_x;
    t.ty = (int)(rest % a.tiles_y);
    t.f = (int)(rest / a.tiles_y);
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
    __shared__ int32_t s_P[kT * kT];
    __shared__ int32_t s_cnt[kT];
    __shared__ MaskAcc s_acc[kAccCap];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const TileLoc t = tile_loc(a, blockIdx.x);
    const int64_t WH = (int64_t)a.width * a.height;
    const int64_t fbase = (int64_t)t.f * WH;

    const bool col_ok = lane < t.tw;
    const float *src = a.prob + fbase + (int64_t)t.Y0 * a.width + t.X0 + lane;
    float v[kRows];
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        v[i] = (col_ok && r < t.th) ? src[(int64_t)r * a.width] : 0.0f;
    }
    // the bitmap and block counts of steps 3-4 start at zero
    {
        const int64_t g = (int64_t)blockIdx.x * kMThreads + threadIdx.x;
        const int64_t stride = (int64_t)gridDim.x * kMThreads;
        for (int64_t j = g; j < w.nwords; j += stride) w.bitmap[j] = 0u;
        for (int64_t j = g; j < w.nb; j += stride) w.bcount[j] = 0;
    }
    uint64_t m[kRows];
    bool fg[kRows], first[kRows];
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        fg[i] = col_ok && r < t.th && v[i] > a.threshold;
        m[i] = __ballot(fg[i]);
        first[i] = fg[i] && !(((m[i] << 1) >> lane) & 1);  // no run pixel on the left
        if (first[i]) s_P[r * kT + lane] = r * kT + lane;
    }
    if (lane == 0) {
#pragma unroll
        for (int i = 0; i < kRows; ++i) s_mask[wave * kRows + i] = m[i];
    }
    __syncthreads();

    // join each run with the runs it touches in the row above, once per pair:
    // a run above that starts under the run (or the run starts under it), and
    // with 8 neighbours a run above that ends just before the run's first
    // pixel or starts just after its last
    const bool eight = a.connectivity == 8;
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        if (r == 0 || !fg[i]) continue;
        const uint64_t mu = i == 0 ? s_mask[r - 1] : m[i - 1];
        const int x = lane;
        const bool up = (mu >> x) & 1;
        const bool upl = ((mu << 1) >> x) & 1;  // above-left (0 at x = 0)
        const bool upr = ((mu >> 1) >> x) & 1;  // above-right (0 at x = 63)
        const int A = r * kT + run_first(m[i], x);
        const int above = (r - 1) * kT;
        int B1 = -1, B2 = -1;
        if (up && !upl) B1 = above + x;
        else if (up && first[i]) B1 = above + run_first(mu, x);
        else if (eight && !up && upl && first[i]) B1 = above + run_first(mu, x - 1);
        if (eight && !up && upr && run_last(m[i], x) == x) B2 = above + x + 1;
        if (B1 >= 0) cl::uf_unite<kGroup>(s_P, A, B1);
        if (B2 >= 0) cl::uf_unite<kGroup>(s_P, A, B2);
    }
    __syncthreads();

    // flatten: every run points at its piece's root, the piece's first pixel
    int root[kRows];
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        root[i] = first[i] ? cl::uf_find<kGroup>(s_P, r * kT + lane) : 0;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        if (first[i]) s_P[r * kT + lane] = root[i];
    }
    __syncthreads();
    bool is_root[kRows];
    uint64_t rm[kRows];
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        if (fg[i] && !first[i]) root[i] = s_P[r * kT + run_first(m[i], lane)];
        is_root[i] = first[i] && root[i] == r * kT + lane;
        rm[i] = __ballot(is_root[i]);
    }
    if (lane == 0) {
#pragma unroll
        for (int i = 0; i < kRows; ++i) s_cnt[wave * kRows + i] = __popcll(rm[i]);
    }
    __syncthreads();

    // pieces numbered in raster order of their roots
    const int c = s_cnt[lane];
    int inc = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(inc, o, 64);
        if (lane >= o) inc += u;
    }
    const int excl = inc - c;
    const int np = __shfl(inc, 63, 64);
    const uint64_t lt = (1ull << lane) - 1;
    int piece[kRows];
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        piece[i] = __shfl(excl, r, 64) + __popcll(rm[i] & lt);
        if (is_root[i]) s_P[r * kT + lane] = -(piece[i] + 1);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kRows; ++i)
        if (fg[i] && !is_root[i]) piece[i] = -s_P[root[i]] - 1;

    // statistics, kAccCap pieces per pass
    const int64_t cap = tile_cap(a, t);
    for (int c0 = 0; c0 < np; c0 += kAccCap) {
        s_acc[threadIdx.x] = MaskAcc{0u, 0u, 0u, 63u, 0u, 0u, 0u, 0u};
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kRows; ++i) {
            const int r = wave * kRows + i;
            const int p = piece[i] - c0;
            if (!fg[i] || p < 0 || p >= kAccCap) continue;
            MaskAcc &q = s_acc[p];
            atomicMax(&q.score, __float_as_uint(v[i]));
            if (first[i]) {
                const int e = run_last(m[i], lane);
                const uint32_t len = (uint32_t)(e - lane + 1);
                atomicAdd(&q.area, len);
                atomicAdd(&q.sx, (uint32_t)(lane + e) * len / 2u);
                atomicAdd(&q.sy, len * (uint32_t)r);
                atomicMin(&q.x0, (uint32_t)lane);
                atomicMax(&q.x1, (uint32_t)e);
                atomicMax(&q.y1, (uint32_t)r);
            }
            if (is_root[i]) q.root = (uint32_t)(r * kT + lane);
        }
        __syncthreads();
        const int p = c0 + threadIdx.x;
        if (p < np && p < cap) {
            const MaskAcc q = s_acc[threadIdx.x];
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

    // labels (the piece's first pixel for now) and the tile's outer slots
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
        const int r = wave * kRows + i;
        if (!col_ok || r >= t.th) continue;
        const int rt = root[i];
        if (a.labels) {
            const int64_t lab = fg[i] ? (int64_t)(t.Y0 + rt / kT) * a.width + t.X0 + rt % kT : -1;
            a.labels[fbase + (int64_t)(t.Y0 + r) * a.width + t.X0 + lane] = (int32_t)lab;
        }
        const int32_t slot = fg[i] && piece[i] < cap ? (int32_t)(t.base + piece[i]) : -1;
        if (r == 0) w.hseam[((int64_t)(t.f * a.tiles_y + t.ty) * 2 + 0) * a.width + t.X0 + lane] = slot;
        if (r == t.th - 1) w.hseam[((int64_t)(t.f * a.tiles_y + t.ty) * 2 + 1) * a.width + t.X0 + lane] = slot;
        if (lane == 0) w.vseam[((int64_t)(t.f * a.tiles_x + t.tx) * 2 + 0) * a.height + t.Y0 + r] = slot;
        if (lane == t.tw - 1) w.vseam[((int64_t)(t.f * a.tiles_x + t.tx) * 2 + 1) * a.height + t.Y0 + r] = slot;
    }
    if (threadIdx.x == 0) w.tile_np[blockIdx.x] = (int32_t)min((int64_t)np, cap);
}

__device__ __forceinline__ uint64_t ld64(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, kAgent);
}

// Key of the root of slot s's tree.
__device__ __forceinline__ uint64_t key_root(const uint64_t *gp, uint32_t s) {
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
    if (g < nh) {
        const int x = (int)(g % a.width);
        const int64_t fb = g / a.width;
        const int f = (int)(fb / (a.tiles_y - 1)), b = (int)(fb % (a.tiles_y - 1));
        const int32_t *up = w.hseam + ((int64_t)(f * a.tiles_y + b) * 2 + 1) * a.width;
        const int32_t *dn = w.hseam + ((int64_t)(f * a.tiles_y + b + 1) * 2 + 0) * a.width;
        join_seam(w.gp, up, dn, x, a.width, eight);
        return;
    }
    g -= nh;
    if (g < nv) {
        const int y = (int)(g % a.height);
        const int64_t fc = g / a.height;
        const int f = (int)(fc / (a.tiles_x - 1)), c = (int)(fc % (a.tiles_x - 1));
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
        const uint64_t own = ld64(w.gp + s);
        if ((uint32_t)own == s) {
            const uint64_t g = own >> 32;
            atomicOr(w.bitmap + (g >> 5), 1u << (g & 31));
            atomicAdd(w.bcount + (g / kBitBlock), 1);
            continue;
        }
        const uint64_t rk = key_root(w.gp, s);
        __hip_atomic_store(w.gp + s, rk, __ATOMIC_RELAXED, kAgent);
        const MaskRec R = w.rec[s];
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

// Components whose first pixel lies before bit b of the batch.
__device__ __forceinline__ int32_t rank_before(const MaskWs &w, int64_t b) {
    const int64_t blk = b / kBitBlock;
    int32_t r = w.bbase[blk];
    const int64_t w1 = b >> 5;
    for (int64_t j = blk * kBitWords; j < w1; ++j) r += __popc(w.bitmap[j]);
    if (b & 31) r += __popc(w.bitmap[w1] & ((1u << (b & 31)) - 1u));
    return r;
}

__global__ __launch_bounds__(1024) void mask_scan_kernel(MaskArgs a, MaskWs w) {
    __shared__ int s_wave[16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nb = w.nb;
    const int per = (nb + 1023) / 1024;
    const int b0 = min(tid * per, nb), b1 = min(b0 + per, nb);
    int sum = 0;
    for (int b = b0; b < b1; ++b) sum += w.bcount[b];
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
    for (int b = b0; b < b1; ++b) {
        w.bbase[b] = run;
        run += w.bcount[b];
    }
    if (tid == 1023) w.bbase[nb] = run;
    __syncthreads();
    const int64_t WH = (int64_t)a.width * a.height;
    for (int f = tid; f <= a.n_frames; f += 1024) {
        const int32_t r0 = rank_before(w, (int64_t)f * WH);
        a.comp_offsets[f] = r0;
        if (f < a.n_frames) a.n_components[f] = rank_before(w, (int64_t)(f + 1) * WH) - r0;
    }
}

__global__ __launch_bounds__(kMThreads) void mask_finish_kernel(MaskArgs a, MaskWs w) {
    __shared__ int32_t s_list[kT * kT / 2];
    __shared__ int32_t s_n;
    const TileLoc t = tile_loc(a, blockIdx.x);
    const int np = w.tile_np[blockIdx.x];
    const int64_t fbase = (int64_t)t.f * a.width * a.height;
    if (threadIdx.x == 0) s_n = 0;
    __syncthreads();
    for (int p = threadIdx.x; p < np; p += kMThreads) {
        const uint32_t s = (uint32_t)(t.base + p);
        const uint64_t k = w.gp[s];
        if ((uint32_t)k != s) {
            if (a.labels) s_list[atomicAdd(&s_n, 1)] = p;
            continue;
        }
        const int64_t rank = rank_before(w, (int64_t)(k >> 32));
        if (rank >= a.capacity) continue;
        const MaskRec R = w.rec[s];
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
    // pieces that are not their component's first: their pixels still carry
    // the piece's own first pixel
    const int n = s_n;
    for (int q = 0; q < n; ++q) {
        const uint32_t s = (uint32_t)(t.base + s_list[q]);
        const MaskRec R = w.rec[s];
        const int32_t old = (int32_t)R.root;
        const int32_t lab = (int32_t)((int64_t)(w.gp[s] >> 32) - fbase);
        const int bw = (int)(R.x1 - R.x0 + 1), bh = (int)(R.y1 - R.y0 + 1);
        for (int e = threadIdx.x; e < bw * bh; e += kMThreads) {
            const int64_t idx = fbase + (int64_t)(R.y0 + e / bw) * a.width + R.x0 + e % bw;
            if (a.labels[idx] == old) a.labels[idx] = lab;
        }
    }
}

struct MaskLayout {
    int64_t slots, n_tiles;
    int64_t nwords;
    int32_t nb;
    size_t off_gp, off_rec, off_np, off_hs, off_vs, off_bits, off_bc, off_bb, bytes;
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
    L.nwords = (total + 31) / 32;
    L.nb = (int32_t)((total + kBitBlock - 1) / kBitBlock);
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
    o += align256((size_t)L.nb * sizeof(int32_t));
    L.off_bb = o;
    o += align256((size_t)(L.nb + 1) * sizeof(int32_t));
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
    w.bbase = reinterpret_cast<int32_t *>(base + L.off_bb);
    w.nwords = L.nwords;
    w.nb = L.nb;
    const unsigned tiles = (unsigned)L.n_tiles;
    hipLaunchKernelGGL(mask_tile_kernel, dim3(tiles), dim3(kMThreads), 0, stream, a, w);
    const int64_t nh = (int64_t)a.n_frames * (a.tiles_y - 1) * a.width;
    const int64_t nv = (int64_t)a.n_frames * (a.tiles_x - 1) * a.height;
    if (nh + nv > 0)
        hipLaunchKernelGGL(mask_seam_kernel, dim3((unsigned)((nh + nv + 255) / 256)), dim3(256), 0, stream, a, w,
                           nh, nv);
    hipLaunchKernelGGL(mask_resolve_kernel, dim3(tiles), dim3(64), 0, stream, a, w);
    hipLaunchKernelGGL(mask_scan_kernel, dim3(1), dim3(1024), 0, stream, a, w);
    hipLaunchKernelGGL(mask_finish_kernel, dim3(tiles), dim3(kMThreads), 0, stream, a, w);
    return hipGetLastError();
}

}  // namespace flock

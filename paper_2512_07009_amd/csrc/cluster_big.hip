// cluster_big.hip - radius-neighbour clustering of frames too large for one
// workgroup's LDS, spread over many workgroups.
//
// Same definition and conventions as cluster.hip (standard DBSCAN with the
// nearest-core border rule and smallest-core-index labels; the paper's
// clustering module, Section 2.3).  Frames with more points than the on-chip
// capacity are processed by a sequence of grid-wide kernels over the whole
// batch; each thread first finds its frame and skips frames that the on-chip
// kernel handles.  All intermediate state is in the workspace:
//
//   frame records  int32[F][16]        bbox, cell grid, stencil
//   rank           int32[T]            rank of a point within its cell
//   spos, ssid     int2[T], int32[T]   points sorted by cell; frame-local index
//   score          uint8[T]            core flag by sorted position
//   cstart, cnode  int32[2T + 2F]      per frame f, entries 2*offsets[f] + 2f
//                                      .. + ncell: cell start (and end
//                                      sentinel); the cell's smallest core index
//
// A frame of n points gets a cell table of at most 2n + 1 cells (the cell
// side doubles from the eps-diagonal side until the grid fits; the same-cell
// shortcut holds only at the undoubled side), so the table never depends on
// anything the host does not know.  The union-find forest lives in the
// caller's labels array (frame-local indices): walks read it through the
// cache, hooks are agent-scope compare-and-swap.
//
// Kernels, in stream order: prep (one workgroup per frame: bounding box,
// grid; the cell clearing there or, for a few frames, in extra workgroups
// beside it), hist (cell counts and ranks), scan (one workgroup per frame),
// scatter, core (neighbour counts with early exit, and each cell's smallest
// core index), union of adjacent cell pairs (blocks of cells joined in LDS
// first), union of the farther cell pairs (and point pairs where the grid
// was coarsened), labels (cores: their tree's root and the cluster counts;
// other points: the root of the nearest core's tree).  A batch of one large frame skips the on-chip kernel, and
// prep then writes the counts of an empty or inconsistent frame.

#include <algorithm>
#include <climits>

#include "cluster_common.h"
#include "internal.h"

namespace flock {
namespace {

using namespace cl;

constexpr int kBlock = 256;
constexpr int kScanThreads = 1024;
constexpr int kPrepThreads = 1024;
constexpr int kUnroll = 32;      // independent loads per thread and step in the bounding box
constexpr int kScanUnroll = 32;  // cells per thread in a scan tile (32768 cells, 132 KiB of LDS)
constexpr int kRec = 16;  // int32 fields per frame record
constexpr int kClearBlocks = 8;  // cell-clearing workgroups per frame beside the bounding box
constexpr int kClearFrames = 64; // ... for batches of at most this many frames

enum RecField {
    kXmin = 0, kYmin, kXmax, kYmax, kSide, kNcx, kNcy, kDense, kReach, kDx0, kDx1, kDx2, kNcell, kBig
};

struct BigWs {
    int32_t *rec;
    int32_t *rank;
    int2 *spos;
    int32_t *ssid;
    uint8_t *score;
    int32_t *cstart;
    int32_t *cnode;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

BigWs carve(void *base, int32_t n_frames, int32_t total) {
    char *p = static_cast<char *>(base);
    BigWs w;
    const size_t cells = 2 * (size_t)total + 2 * (size_t)n_frames;
    w.rec = reinterpret_cast<int32_t *>(p);
    p += align256(sizeof(int32_t) * kRec * (size_t)n_frames);
    w.rank = reinterpret_cast<int32_t *>(p);
    p += align256(sizeof(int32_t) * (size_t)total);
    w.spos = reinterpret_cast<int2 *>(p);
    p += align256(sizeof(int2) * (size_t)total);
    w.ssid = reinterpret_cast<int32_t *>(p);
    p += align256(sizeof(int32_t) * (size_t)total);
    w.score = reinterpret_cast<uint8_t *>(p);
    p += align256((size_t)total);
    w.cstart = reinterpret_cast<int32_t *>(p);
    p += align256(sizeof(int32_t) * cells);
    w.cnode = reinterpret_cast<int32_t *>(p);
    return w;
}

__device__ __forceinline__ bool frame_ok(const ClusterArgs &a, int f, int32_t *b, int32_t *e) {
    *b = a.offsets[f];
    *e = a.offsets[f + 1];
    return !(*b < 0 || *e < *b || *e > a.total);
}

// Frame holding global point index i: the last f with offsets[f] <= i, or -1
// when i lies past that frame's end (points beyond offsets[n_frames], or
// under a frame whose offsets decrease): such points belong to no frame and
// are never read.
__device__ __forceinline__ int frame_of_point(const int32_t *offsets, int n_frames, int32_t i) {
    int lo = 0, hi = n_frames - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (offsets[mid] <= i) lo = mid;
        else hi = mid - 1;
    }
    return (i >= offsets[lo] && i < offsets[lo + 1]) ? lo : -1;
}

// Frame owning cell-table entry c: the last f with 2 offsets[f] + 2 f <= c.
__device__ __forceinline__ int frame_of_cell(const int32_t *offsets, int n_frames, int64_t c) {
    int lo = 0, hi = n_frames - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (2 * (int64_t)offsets[mid] + 2 * (int64_t)mid <= c) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ int64_t cell_base(const int32_t *offsets, int f) {
    return 2 * (int64_t)offsets[f] + 2 * (int64_t)f;
}

struct BigGrid {
    int32_t x0, y0, side, ncx, ncy, dense, reach, dx0, dx1, dx2, ncell;  // dx_k: half-width of stencil row |dy| = k
};

// Half-width of stencil row |dy| (0..2), blended with masks: an indexed
// array, or selects between the record's fields (which the compiler turns
// into a select of their addresses), would put the grid record in scratch
// memory.
__device__ __forceinline__ int32_t dx_of(const BigGrid &g, int ady) {
    const int32_t m0 = -(int32_t)(ady == 0), m1 = -(int32_t)(ady == 1);
    return (g.dx0 & m0) | (g.dx1 & m1) | (g.dx2 & ~(m0 | m1));
}

__device__ __forceinline__ BigGrid load_grid(const int32_t *rec) {
    BigGrid g;
    g.x0 = rec[kXmin];
    g.y0 = rec[kYmin];
    g.side = rec[kSide];
    g.ncx = rec[kNcx];
    g.ncy = rec[kNcy];
    g.dense = rec[kDense];
    g.reach = rec[kReach];
    g.dx0 = rec[kDx0];
    g.dx1 = rec[kDx1];
    g.dx2 = rec[kDx2];
    g.ncell = rec[kNcell];
    return g;
}

__device__ __forceinline__ void cell_xy(int2 p, const BigGrid &g, int32_t *cx, int32_t *cy) {
    *cx = cell_coord_clamped(p.x, g.x0, g.side, g.ncx);
    *cy = cell_coord_clamped(p.y, g.y0, g.side, g.ncy);
}

// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kPrepThreads) void big_prep(ClusterArgs a, BigWs w) {
    __shared__ int s_bbox[4];
    const int f = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    int32_t *rec = w.rec + (size_t)f * kRec;
    int32_t b, e;
    const bool ok = frame_ok(a, f, &b, &e);
    const int32_t n = ok ? e - b : 0;
    const bool big = ok && n > 0 && (n > a.cap_points || a.big_all);
    if (blockIdx.y > 0) {
        // clearing share of a large frame's cell range (2 n + 2 entries, at
        // least the ncell + 1 the grid uses), beside the bounding box
        if (!big) return;
        const int64_t base = cell_base(a.offsets, f), m = 2 * (int64_t)n + 2;
        const int64_t per = (m + gridDim.y - 2) / (gridDim.y - 1);
        const int64_t c0 = (int64_t)(blockIdx.y - 1) * per, c1 = min(m, c0 + per);
        for (int64_t c = c0 + tid; c < c1; c += kPrepThreads) {
            w.cstart[base + c] = 0;
            w.cnode[base + c] = INT_MAX;
        }
        return;
    }
    if (!big) {
        if (tid == 0) {
            rec[kBig] = 0;
            // without the on-chip kernel, the counts of empty and inconsistent frames
            if (a.big_all && a.n_clusters) a.n_clusters[f] = ok ? 0 : -1;
        }
        return;
    }
    if (tid == 0) {
        s_bbox[0] = INT_MAX;
        s_bbox[1] = INT_MAX;
        s_bbox[2] = INT_MIN;
        s_bbox[3] = INT_MIN;
    }
    __syncthreads();
    const int2 *P = reinterpret_cast<const int2 *>(a.xy) + b;
    int xmn = INT_MAX, ymn = INT_MAX, xmx = INT_MIN, ymx = INT_MIN;
    for (int32_t i0 = tid; i0 < n; i0 += kPrepThreads * kUnroll) {
        int2 pv[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int32_t i = i0 + u * kPrepThreads;
            pv[u] = i < n ? P[i] : P[i0];
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            xmn = min(xmn, pv[u].x);
            ymn = min(ymn, pv[u].y);
            xmx = max(xmx, pv[u].x);
            ymx = max(ymx, pv[u].y);
        }
    }
    xmn = wave_min(xmn);
    ymn = wave_min(ymn);
    xmx = wave_max(xmx);
    ymx = wave_max(ymx);
    if (lane == 0) {
        atomicMin(&s_bbox[0], xmn);
        atomicMin(&s_bbox[1], ymn);
        atomicMax(&s_bbox[2], xmx);
        atomicMax(&s_bbox[3], ymx);
    }
    __syncthreads();
    // grid: at most 2n + 1 cells
    const uint32_t wx = (uint32_t)(s_bbox[2] - s_bbox[0]), wy = (uint32_t)(s_bbox[3] - s_bbox[1]);
    uint32_t side = (uint32_t)a.cell_side;
    uint64_t ncx = wx / side + 1, ncy = wy / side + 1;
    while (ncx * ncy > 2 * (uint64_t)n + 1) {
        side *= 2u;
        ncx = wx / side + 1;
        ncy = wy / side + 1;
    }
    const int32_t ncell = (int32_t)(ncx * ncy);
    const int32_t reach = a.eps_q == 0 ? 0 : min(1 + (a.eps_q - 1) / (int32_t)side, 2);
    if (tid == 0) {
        rec[kXmin] = s_bbox[0];
        rec[kYmin] = s_bbox[1];
        rec[kXmax] = s_bbox[2];
        rec[kYmax] = s_bbox[3];
        rec[kSide] = (int32_t)side;
        rec[kNcx] = (int32_t)ncx;
        rec[kNcy] = (int32_t)ncy;
        rec[kDense] = side == (uint32_t)a.cell_side;
        rec[kReach] = reach;
        const int64_t e2 = (int64_t)a.eps_q * a.eps_q;
        for (int dy = 0; dy < 3; ++dy) {
            int dx = 0;
            if (dy <= reach) {
                const int64_t gy = cell_gap(dy, (int32_t)side);
                dx = reach;
                while (dx > 0) {
                    const int64_t gx = cell_gap(dx, (int32_t)side);
                    if (gx * gx + gy * gy <= e2) break;
                    --dx;
                }
            }
            rec[kDx0 + dy] = dx;
        }
        rec[kNcell] = ncell;
        rec[kBig] = 1;
        if (a.n_clusters) a.n_clusters[f] = 0;
    }
    if (gridDim.y == 1) {  // no clearing workgroups beside this one
        const int64_t base = cell_base(a.offsets, f);
        for (int32_t c = tid; c <= ncell; c += kPrepThreads) {
            w.cstart[base + c] = 0;
            w.cnode[base + c] = INT_MAX;
        }
    }
}

__global__ __launch_bounds__(kBlock) void big_hist(ClusterArgs a, BigWs w) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= a.total) return;
    const int f = frame_of_point(a.offsets, a.n_frames, i);
    if (f < 0) return;
    const int32_t *rec = w.rec + (size_t)f * kRec;
    if (!rec[kBig]) return;
    const BigGrid g = load_grid(rec);
    const int2 p = reinterpret_cast<const int2 *>(a.xy)[i];
    int32_t cx, cy;
    cell_xy(p, g, &cx, &cy);
    w.rank[i] = atomicAdd(&w.cstart[cell_base(a.offsets, f) + (int64_t)cy * g.ncx + cx], 1);
}

// Exclusive scan of a frame's cell counts, in tiles of kScanThreads *
// kScanUnroll cells: coalesced loads into LDS, kScanUnroll consecutive cells
// per thread, a workgroup scan plus the carry of the earlier tiles, coalesced
// stores.
__global__ __launch_bounds__(kScanThreads) void big_scan(ClusterArgs a, BigWs w) {
    constexpr int kTileCells = kScanThreads * kScanUnroll;
    // cell c of a tile sits at (c / 32) * 33 + c % 32: both the coalesced
    // passes (consecutive c per lane) and the per-thread runs (32 consecutive
    // c per lane) then touch 64 different banks per wave
    __shared__ int s_wave[kScanThreads / 64];
    __shared__ int s_tile[kTileCells / 32 * 33];
    __shared__ int s_carry;
    auto at = [](int c) { return (c >> 5) * 33 + (c & 31); };
    const int f = blockIdx.x, tid = threadIdx.x;
    const int32_t *rec = w.rec + (size_t)f * kRec;
    if (!rec[kBig]) return;
    const int32_t ncell = rec[kNcell];
    int32_t *cs = w.cstart + cell_base(a.offsets, f);
    int carry = 0;
    for (int32_t t0 = 0; t0 < ncell; t0 += kTileCells) {
        // every load in flight before the first use: indexes are clamped
        // (cs[ncell] exists), values past ncell replaced by 0
        int ld[kScanUnroll];
#pragma unroll
        for (int u = 0; u < kScanUnroll; ++u) ld[u] = cs[min(t0 + u * kScanThreads + tid, ncell)];
#pragma unroll
        for (int u = 0; u < kScanUnroll; ++u)
            s_tile[at(u * kScanThreads + tid)] = t0 + u * kScanThreads + tid < ncell ? ld[u] : 0;
        __syncthreads();
        int v[kScanUnroll], sum = 0;
#pragma unroll
        for (int u = 0; u < kScanUnroll; ++u) {
            v[u] = s_tile[at(tid * kScanUnroll + u)];
            sum += v[u];
        }
        int run = carry + block_exclusive_scan(sum, s_wave);  // ends with a barrier
#pragma unroll
        for (int u = 0; u < kScanUnroll; ++u) {
            s_tile[at(tid * kScanUnroll + u)] = run;
            run += v[u];
        }
        if (tid == kScanThreads - 1) s_carry = run;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kScanUnroll; ++u) {
            const int32_t c = t0 + u * kScanThreads + tid;
            if (c < ncell) cs[c] = s_tile[at(u * kScanThreads + tid)];
        }
        carry = s_carry;
        __syncthreads();  // s_tile and s_carry are rewritten by the next tile
    }
    if (tid == 0) cs[ncell] = carry;
}

__global__ __launch_bounds__(kBlock) void big_scatter(ClusterArgs a, BigWs w) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= a.total) return;
    const int f = frame_of_point(a.offsets, a.n_frames, i);
    if (f < 0) return;
    const int32_t *rec = w.rec + (size_t)f * kRec;
    if (!rec[kBig]) return;
    const BigGrid g = load_grid(rec);
    const int2 p = reinterpret_cast<const int2 *>(a.xy)[i];
    int32_t cx, cy;
    cell_xy(p, g, &cx, &cy);
    const int32_t b = a.offsets[f];
    const int32_t pos = b + w.cstart[cell_base(a.offsets, f) + (int64_t)cy * g.ncx + cx] + w.rank[i];
    w.spos[pos] = p;
    w.ssid[pos] = i - b;
}

// Neighbour counts (dense cells are all core, the rest stop at min_pts), the
// union-find parents and kinds, and each core cell's node.
__global__ __launch_bounds__(kBlock) void big_core(ClusterArgs a, BigWs w) {
    const int32_t p = blockIdx.x * kBlock + threadIdx.x;
    if (p >= a.total) return;
    const int f = frame_of_point(a.offsets, a.n_frames, p);
    if (f < 0) return;
    const int32_t *rec = w.rec + (size_t)f * kRec;
    if (!rec[kBig]) return;
    const BigGrid g = load_grid(rec);
    const int32_t b = a.offsets[f];
    const int32_t *cs = w.cstart + cell_base(a.offsets, f);
    const int2 *S = w.spos + b;
    const Radius r{a.eps_q, a.eps_q + 1, a.eps_q * a.eps_q};
    const int2 v = w.spos[p];
    int32_t cx, cy;
    cell_xy(v, g, &cx, &cy);
    const int32_t own = cy * g.ncx + cx;
    int32_t cnt = g.dense ? cs[own + 1] - cs[own] : 0;
    if (cnt < a.min_pts) {
        cnt = 0;
        for (int k = 0; k <= 2 * g.reach && cnt < a.min_pts; ++k) {
            const int dy = (k & 1) ? -((k + 1) >> 1) : (k >> 1);  // 0, -1, 1, -2, 2
            const int32_t ry = cy + dy;
            if (ry < 0 || ry >= g.ncy) continue;
            const int dxm = dx_of(g, dy < 0 ? -dy : dy);
            const int32_t rx0 = max(cx - dxm, 0), rx1 = min(cx + dxm, g.ncx - 1);
            const int32_t q1 = cs[ry * g.ncx + rx1 + 1];
            int32_t q = cs[ry * g.ncx + rx0];
            // four loads in flight per step (the count may pass min_pts)
            for (; q + 4 <= q1 && cnt < a.min_pts; q += 4) {
                const int2 s0 = S[q], s1 = S[q + 1], s2 = S[q + 2], s3 = S[q + 3];
                cnt += (within(v, s0, r) ? 1 : 0) + (within(v, s1, r) ? 1 : 0) + (within(v, s2, r) ? 1 : 0) +
                       (within(v, s3, r) ? 1 : 0);
            }
            for (; q < q1 && cnt < a.min_pts; ++q) cnt += within(v, S[q], r) ? 1 : 0;
        }
    }
    const bool core = cnt >= a.min_pts;
    w.score[p] = core ? 1 : 0;
    const int32_t o = w.ssid[p];
    a.labels[b + o] = o;  // union-find parent
    a.kind[b + o] = core ? 2 : 0;
    // a core cell's node: its smallest core index (eps-diagonal grid)
    if (core && g.dense) atomicMin(&w.cnode[cell_base(a.offsets, f) + own], o);
}

// k-th forward stencil offset (cells after this one in row-major order).
__device__ __forceinline__ bool forward_offset(const BigGrid &g, int k, int *odx, int *ody) {
    for (int dy = 0; dy <= g.reach; ++dy) {
        const int lo = dy == 0 ? 1 : -dx_of(g, dy);
        const int cnt = dx_of(g, dy) - lo + 1;
        if (cnt > 0 && k < cnt) {
            *odx = lo + k;
            *ody = dy;
            return true;
        }
        k -= max(cnt, 0);
    }
    return false;
}

constexpr int kMaxForward = 12;
constexpr int kAdjacent = 4;  // forward adjacent cells

// Walks a and b to their roots through cached parents, in step (one load
// latency per level of the deeper tree).  Path splitting here (plain
// stores of grandparents) made both the unions and the later label walks
// slower.
__device__ __forceinline__ void roots_cached(const int32_t *parent, int32_t *a, int32_t *b) {
    int32_t x = *a, y = *b;
    for (;;) {
        const int32_t px = ld_rlx<kGroup>(parent + x), py = ld_rlx<kGroup>(parent + y);
        if ((px == x) & (py == y)) break;
        x = px;
        y = py;
    }
    *a = x;
    *b = y;
}

// Merge the trees of nodes a and b in a frame's global forest.  The walks
// read parents through the cache of this workgroup's XCD, so they may miss
// what workgroups on other XCDs hooked during this launch; every value they
// see is still an ancestor (a parent only ever moves to a smaller node of
// the same tree), so a walk ends at some ancestor.  Only the compare-and-swap
// that hooks a root under a smaller node is coherent (agent scope); when it
// fails, the parent it returns is current and the walk goes on from there.
// Each failure lowers the larger of the two nodes, so the loop ends, and
// every tree's root stays its smallest node.
__device__ __forceinline__ void uf_unite_cached(int32_t *parent, int32_t a, int32_t b) {
    roots_cached(parent, &a, &b);
    for (;;) {
        if (a == b) return;
        if (a < b) {
            const int32_t t = a;
            a = b;
            b = t;
        }
        int32_t expected = a;
        if (__hip_atomic_compare_exchange_strong(parent + a, &expected, b, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                 kAgent))
            return;
        a = uf_root<kGroup>(parent, expected);
    }
}

// Point-pair unions of point p when its frame's grid was coarsened.
__device__ void union_points_one(const ClusterArgs &a, const BigWs &w, int32_t p) {
    if (p >= a.total || !w.score[p]) return;
    const int f = frame_of_point(a.offsets, a.n_frames, p);
    if (f < 0) return;
    const int32_t *rec = w.rec + (size_t)f * kRec;
    if (!rec[kBig] || rec[kDense]) return;
    const BigGrid g = load_grid(rec);
    const int32_t b = a.offsets[f];
    const int32_t *cs = w.cstart + cell_base(a.offsets, f);
    const int2 *S = w.spos + b;
    const uint8_t *core = w.score + b;
    int32_t *parent = a.labels + b;
    const Radius r{a.eps_q, a.eps_q + 1, a.eps_q * a.eps_q};
    const int32_t lp = p - b;
    const int2 v = S[lp];
    const int32_t op = w.ssid[p];
    int32_t cx, cy;
    cell_xy(v, g, &cx, &cy);
    const int32_t own = cy * g.ncx + cx;
    for (int32_t q = cs[own]; q < lp; ++q)
        if (core[q] && within(v, S[q], r)) uf_unite_cached(parent, op, w.ssid[b + q]);
    for (int dy = 0; dy <= g.reach; ++dy) {
        const int32_t ry = cy + dy;
        if (ry >= g.ncy) break;
        const int32_t rx0 = dy == 0 ? cx + 1 : max(cx - dx_of(g, dy), 0);
        const int32_t rx1 = min(cx + dx_of(g, dy), g.ncx - 1);
        if (rx0 > rx1) continue;
        const int32_t q1 = cs[ry * g.ncx + rx1 + 1];
        for (int32_t q = cs[ry * g.ncx + rx0]; q < q1; ++q)
            if (core[q] && within(v, S[q], r)) uf_unite_cached(parent, op, w.ssid[b + q]);
    }
}

// True if some core of sorted points [a0, a1) lies within eps of some core
// of [b0, b1), whose cell covers [rx0, rx1] x [ry0, ry1]: A's cores out of
// reach of that rectangle are skipped, B is read four points per step (the
// scan of a large pair is bound by the latency of these loads).
__device__ __forceinline__ bool cores_touch(const int2 *S, const uint8_t *core, int32_t a0, int32_t a1, int32_t b0,
                                            int32_t b1, int32_t rx0, int32_t rx1, int32_t ry0, int32_t ry1,
                                            const Radius &r) {
    for (int32_t qa = a0; qa < a1; ++qa) {
        if (!core[qa]) continue;
        const int2 va = S[qa];
        const int32_t ddx = min(max(max(rx0 - va.x, va.x - rx1), 0), r.e1);
        const int32_t ddy = min(max(max(ry0 - va.y, va.y - ry1), 0), r.e1);
        if (__mul24(ddx, ddx) + __mul24(ddy, ddy) > r.e2) continue;
        int32_t qb = b0;
        bool hit = false;
        for (; qb + 4 <= b1 && !hit; qb += 4) {
            const int2 s0 = S[qb], s1 = S[qb + 1], s2 = S[qb + 2], s3 = S[qb + 3];
            const uint8_t c0 = core[qb], c1 = core[qb + 1], c2 = core[qb + 2], c3 = core[qb + 3];
            hit = (c0 && within(va, s0, r)) | (c1 && within(va, s1, r)) | (c2 && within(va, s2, r)) |
                  (c3 && within(va, s3, r));
        }
        for (; qb < b1 && !hit; ++qb) hit = core[qb] && within(va, S[qb], r);
        if (hit) return true;
    }
    return false;
}

// Adjacent cell-pair unions, tiled.  A workgroup takes blocks of kTileW x
// kTileH cells of one frame; with their forward adjacent neighbours (one
// more column each side, one more row below) they form its region.  It
// tests the adjacent pairs of its cells (one per thread), joins them in a
// forest over the region in LDS (synchronous hook-and-jump rounds), and
// then hooks every region cell's node to the smallest node of its local
// tree in the frame's global forest (uf_unite_cached), so that each
// compare-and-swap meets the node's own root.  Every local edge is a true
// edge and every adjacent pair is tested by the block owning its first
// cell, so the global forest ends with the components of the adjacent
// edges, with far fewer global hooks than one per edge.
constexpr int kTileW = 16, kTileH = 8;
constexpr int kTileCells = kTileW * kTileH;
constexpr int kTileThreads = kTileCells * kAdjacent;   // one adjacent pair per thread
constexpr int kRegW = kTileW + 2, kRegH = kTileH + 1, kRegionCells = kRegW * kRegH;

// Workgroups of frame f in the tiled launch: [slot(f), slot(f + 1)), at
// least one per frame (the + f), about one per kTileCells cell-table entries.
__device__ __forceinline__ int64_t tile_slot(const int32_t *offsets, int f) {
    return cell_base(offsets, f) / kTileCells + f;
}

__device__ __forceinline__ int frame_of_slot(const int32_t *offsets, int n_frames, int64_t wg) {
    int lo = 0, hi = n_frames - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tile_slot(offsets, mid) <= wg) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

__global__ __launch_bounds__(kTileThreads) void big_union_tiles(ClusterArgs a, BigWs w) {
    __shared__ int32_t s_node[kRegionCells];  // node of each region cell; INT_MAX: no core, or off the grid
    __shared__ int32_t s_par[kRegionCells];   // local forest over region cells
    __shared__ int32_t s_min[kRegionCells];   // smallest node of each local tree (at its root)
    __shared__ uint32_t s_edge[kTileCells];   // bit k: an edge to adjacent neighbour k
    __shared__ int s_hook[3];
    const int tid = threadIdx.x;
    const int64_t wg = blockIdx.x;
    const int f = frame_of_slot(a.offsets, a.n_frames, wg);
    const int32_t *rec = w.rec + (size_t)f * kRec;
    if (!rec[kBig]) return;
    const BigGrid g = load_grid(rec);
    const int32_t b = a.offsets[f];
    const int64_t s0 = tile_slot(a.offsets, f), nslots = tile_slot(a.offsets, f + 1) - s0;
    if (wg >= s0 + nslots || !g.dense) return;  // past the last frame's slots; coarsened grids: far launch
    if (tid == 0) s_hook[0] = 0;
    const int64_t base = cell_base(a.offsets, f);
    const int32_t *cs = w.cstart + base;
    const int32_t *cn = w.cnode + base;
    const int2 *S = w.spos + b;
    const uint8_t *core = w.score + b;
    int32_t *parent = a.labels + b;
    const Radius r{a.eps_q, a.eps_q + 1, a.eps_q * a.eps_q};
    const int tiles_x = (g.ncx + kTileW - 1) / kTileW, tiles_y = (g.ncy + kTileH - 1) / kTileH;
    auto region = [](int ox, int oy) { return oy * kRegW + ox + 1; };
    // adjacent neighbour k: (1, 0), (-1, 1), (0, 1), (1, 1)
    auto adx = [](int k) { return k == 0 ? 1 : k - 2; };
    auto ady = [](int k) { return k == 0 ? 0 : 1; };
    auto root = [&](int i) {
        while (s_par[i] != i) i = s_par[i];
        return i;
    };
    // tests the pair (owned cell j, its adjacent neighbour k) and sets bit k on a hit
    auto test = [&](int tx0, int ty0, int j, int k) {
        const int ox = j % kTileW, oy = j / kTileW;
        const int odx = adx(k), ody = ady(k);
        const int ia = region(ox, oy), ib = region(ox + odx, oy + ody);
        if ((s_node[ia] == INT_MAX) | (s_node[ib] == INT_MAX)) return;
        const int32_t ax = tx0 + ox, ay = ty0 + oy, bx = ax + odx, by = ay + ody;
        const int32_t ca = ay * g.ncx + ax, cb = by * g.ncx + bx;
        const int32_t rx0 = g.x0 + bx * g.side, ry0 = g.y0 + by * g.side;
        if (cores_touch(S, core, cs[ca], cs[ca + 1], cs[cb], cs[cb + 1], rx0, rx0 + g.side - 1, ry0,
                        ry0 + g.side - 1, r))
            atomicOr(&s_edge[j], 1u << k);
    };
    // hook-and-jump rounds over the block's edges (each round that hooks
    // leaves fewer local roots, so the loop ends)
    int round = 0;
    auto rounds = [&]() {
        for (int guard = 0; guard <= kRegionCells; ++guard, ++round) {
            if (tid == 0) s_hook[(round + 1) % 3] = 0;
            bool any = false;
            if (tid < kTileCells && s_edge[tid]) {
                const uint32_t m = s_edge[tid];
                const int ox = tid % kTileW, oy = tid / kTileW;
                const int32_t pa = s_par[region(ox, oy)];
                int32_t pb[kAdjacent];
                int32_t lo = pa;
#pragma unroll
                for (int k = 0; k < kAdjacent; ++k) {
                    pb[k] = ((m >> k) & 1u) ? s_par[region(ox + adx(k), oy + ady(k))] : pa;
                    lo = min(lo, pb[k]);
                }
                if (pa != lo) {
                    atomicMin(&s_par[pa], lo);
                    any = true;
                }
#pragma unroll
                for (int k = 0; k < kAdjacent; ++k)
                    if (pb[k] != lo) {
                        atomicMin(&s_par[pb[k]], lo);
                        any = true;
                    }
            }
            if (any) s_hook[round % 3] = 1;
            __syncthreads();
            if (!s_hook[round % 3]) break;
            for (int i = tid; i < kRegionCells; i += kTileThreads) s_par[i] = root(i);
            __syncthreads();
        }
        ++round;
    };
    for (int64_t t = wg - s0; t < (int64_t)tiles_x * tiles_y; t += nslots) {
        const int tx0 = (int)(t % tiles_x) * kTileW, ty0 = (int)(t / tiles_x) * kTileH;
        for (int i = tid; i < kRegionCells; i += kTileThreads) {
            const int32_t rx = tx0 - 1 + i % kRegW, ry = ty0 + i / kRegW;
            s_node[i] = (rx >= 0 && rx < g.ncx && ry < g.ncy) ? cn[ry * g.ncx + rx] : INT_MAX;
            s_par[i] = i;
        }
        if (tid < kTileCells) s_edge[tid] = 0;
        __syncthreads();
        test(tx0, ty0, tid / kAdjacent, tid % kAdjacent);
        __syncthreads();
        rounds();
        // every node of a local tree is hooked to the tree's smallest node,
        // so that each compare-and-swap meets the node's own root
        for (int i = tid; i < kRegionCells; i += kTileThreads) s_min[i] = INT_MAX;
        __syncthreads();
        for (int i = tid; i < kRegionCells; i += kTileThreads)
            if (s_node[i] != INT_MAX) atomicMin(&s_min[root(i)], s_node[i]);
        __syncthreads();
        for (int i = tid; i < kRegionCells; i += kTileThreads) {
            const int32_t m = s_min[root(i)];
            if (s_node[i] != INT_MAX && s_node[i] != m) uf_unite_cached(parent, s_node[i], m);
        }
        __syncthreads();  // the next block rewrites the region
    }
}

// Farther cell-pair unions (forward offsets beyond the adjacent ones), one
// item per (cell, offset), after the adjacent unions: most pairs find their
// two nodes already joined (cached walks: a common ancestor in a stale view
// is still one) and skip the point tests.  Also the point unions of frames
// whose grid was coarsened.
__global__ __launch_bounds__(kBlock) void big_union_far(ClusterArgs a, BigWs w, int64_t n_items) {
    const int64_t item = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (item < a.total) union_points_one(a, w, (int32_t)item);  // n_items >= total
    if (item >= n_items) return;
    const int64_t c = item / kMaxForward;
    const int k = (int)(item - c * kMaxForward);
    const int f = frame_of_cell(a.offsets, a.n_frames, c);
    const int32_t *rec = w.rec + (size_t)f * kRec;
    if (!rec[kBig] || !rec[kDense]) return;
    const BigGrid g = load_grid(rec);
    const int64_t base = cell_base(a.offsets, f);
    const int32_t ca = (int32_t)(c - base);
    if (ca >= g.ncell) return;
    int odx, ody;
    if (!forward_offset(g, k, &odx, &ody)) return;
    if (odx >= -1 && odx <= 1 && ody <= 1) return;  // adjacent: the tiled launch's
    const int32_t ay = ca / g.ncx, ax = ca - ay * g.ncx;
    const int32_t bx = ax + odx, by = ay + ody;
    if (bx < 0 || bx >= g.ncx || by >= g.ncy) return;
    const int32_t cb = by * g.ncx + bx;
    int32_t na = w.cnode[base + ca], nb = w.cnode[base + cb];  // both loads in flight
    if ((na == INT_MAX) | (nb == INT_MAX)) return;
    const int32_t b = a.offsets[f];
    int32_t *parent = a.labels + b;
    int32_t ra = na, rb = nb;
    roots_cached(parent, &ra, &rb);
    if (ra == rb) return;
    const int32_t *cs = w.cstart + base;
    const int32_t rx0 = g.x0 + bx * g.side, ry0 = g.y0 + by * g.side;
    if (cores_touch(w.spos + b, w.score + b, cs[ca], cs[ca + 1], cs[cb], cs[cb + 1], rx0, rx0 + g.side - 1, ry0,
                    ry0 + g.side - 1, Radius{a.eps_q, a.eps_q + 1, a.eps_q * a.eps_q}))
        uf_unite_cached(parent, na, nb);
}

// Labels, one thread per sorted point, after the unions have ended: a core
// takes its tree's root (its cell's node on the eps-diagonal grid, else the
// point itself, walked to the root) and counts the cluster if it is that
// root; a non-core point searches its stencil for the nearest core within
// eps (ties by smaller (y, x)) and takes the root of that core's node.  The
// walks read parents through the cache: the forest no longer changes but
// for cores storing their roots, which leaves every walk's end the same.
__device__ __forceinline__ int32_t node_of(const BigWs &w, const ClusterArgs &a, const BigGrid &g, int f, int32_t b,
                                           int32_t q, int2 v) {
    if (!g.dense) return w.ssid[b + q];
    int32_t cx, cy;
    cell_xy(v, g, &cx, &cy);
    return w.cnode[cell_base(a.offsets, f) + (int64_t)cy * g.ncx + cx];
}

__global__ __launch_bounds__(kBlock) void big_label(ClusterArgs a, BigWs w) {
    const int32_t p = blockIdx.x * kBlock + threadIdx.x;
    if (p >= a.total) return;
    const int f = frame_of_point(a.offsets, a.n_frames, p);
    if (f < 0) return;
    const int32_t *rec = w.rec + (size_t)f * kRec;
    if (!rec[kBig]) return;
    const BigGrid g = load_grid(rec);
    const int32_t b = a.offsets[f];
    int32_t *parent = a.labels + b;
    const int32_t o = w.ssid[p];
    const int2 v = w.spos[p];
    if (w.score[p]) {
        const int32_t root = uf_root<kGroup>(parent, node_of(w, a, g, f, b, p - b, v));
        st_rlx<kAgent>(parent + o, root);
        if (root == o && a.n_clusters) atomicAdd(&a.n_clusters[f], 1);
        return;
    }
    const int64_t base = cell_base(a.offsets, f);
    const int32_t *cs = w.cstart + base;
    const int2 *S = w.spos + b;
    const uint8_t *core = w.score + b;
    const Radius r{a.eps_q, a.eps_q + 1, a.eps_q * a.eps_q};
    int32_t cx, cy;
    cell_xy(v, g, &cx, &cy);
    int32_t best = -1, best_d2 = INT32_MAX, by = 0, bx = 0;
    for (int dy = -g.reach; dy <= g.reach; ++dy) {
        const int32_t ry = cy + dy;
        if (ry < 0 || ry >= g.ncy) continue;
        const int dxm = dx_of(g, dy < 0 ? -dy : dy);
        const int32_t rx0 = max(cx - dxm, 0), rx1 = min(cx + dxm, g.ncx - 1);
        const int32_t q1 = cs[ry * g.ncx + rx1 + 1];
        // four candidates loaded per step (indices past the span repeat its
        // last point and are masked), then tested in order
        for (int32_t q = cs[ry * g.ncx + rx0]; q < q1; q += 4) {
            int2 qv[4];
            bool cv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int32_t qi = min(q + u, q1 - 1);
                qv[u] = S[qi];
                cv[u] = (q + u < q1) & (core[qi] != 0);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int32_t d2 = sq_dist_clamped(v, qv[u], r);
                const bool take = cv[u] & (d2 <= r.e2) & core_before(d2, qv[u].y, qv[u].x, best_d2, by, bx);
                best = take ? q + u : best;
                best_d2 = take ? d2 : best_d2;
                by = take ? qv[u].y : by;
                bx = take ? qv[u].x : bx;
            }
        }
    }
    if (best >= 0) {
        parent[o] = uf_root<kGroup>(parent, node_of(w, a, g, f, b, best, make_int2(bx, by)));
        a.kind[b + o] = 1;
    } else {
        parent[o] = -1;
    }
}

unsigned blocks_for(int64_t n) { return (unsigned)((n + kBlock - 1) / kBlock); }

}  // namespace

size_t cluster_big_workspace(int32_t n_frames, int32_t total) {
    const size_t cells = 2 * (size_t)total + 2 * (size_t)n_frames;
    return align256(sizeof(int32_t) * kRec * (size_t)n_frames) + align256(sizeof(int32_t) * (size_t)total) +
           align256(sizeof(int2) * (size_t)total) + align256(sizeof(int32_t) * (size_t)total) +
           align256((size_t)total) + 2 * align256(sizeof(int32_t) * cells) + 256;
}

hipError_t launch_cluster_big(const ClusterArgs &a, void *workspace, hipStream_t stream) {
    const BigWs w = carve(workspace, a.n_frames, a.total);
    const int64_t cells = 2 * (int64_t)a.total + 2 * (int64_t)a.n_frames;
    const unsigned pts = blocks_for(a.total);
    // a few frames: each frame's cell range is cleared by kClearBlocks
    // workgroups beside the one that finds its bounding box
    const unsigned prep_y = a.n_frames <= kClearFrames ? 1 + kClearBlocks : 1;
    hipLaunchKernelGGL(big_prep, dim3(a.n_frames, prep_y), dim3(kPrepThreads), 0, stream, a, w);
    if (a.total > 0) {
        hipLaunchKernelGGL(big_hist, dim3(pts), dim3(kBlock), 0, stream, a, w);
        hipLaunchKernelGGL(big_scan, dim3(a.n_frames), dim3(kScanThreads), 0, stream, a, w);
        hipLaunchKernelGGL(big_scatter, dim3(pts), dim3(kBlock), 0, stream, a, w);
        hipLaunchKernelGGL(big_core, dim3(pts), dim3(kBlock), 0, stream, a, w);
        // one more slot per frame than the cell table's blocks (tile_slot)
        const int64_t slots = cells / kTileCells + a.n_frames, items = cells * kMaxForward;
        hipLaunchKernelGGL(big_union_tiles, dim3((unsigned)slots), dim3(kTileThreads), 0, stream, a, w);
        hipLaunchKernelGGL(big_union_far, dim3(blocks_for(items)), dim3(kBlock), 0, stream, a, w, items);
        hipLaunchKernelGGL(big_label, dim3(pts), dim3(kBlock), 0, stream, a, w);
    }
    return hipGetLastError();
}

}  // namespace flock

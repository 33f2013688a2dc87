// cluster.hip - radius-neighbour (DBSCAN-style) clustering of ragged frames
// on gfx950.
//
// What is computed (the paper's clustering module, Section 2.3, at point
// level; standard DBSCAN of Ester et al. 1996 with fixed tie rules):
//   neighbours  dx^2 + dy^2 <= E^2 on integer 1/16-px coordinates (E = eps_q),
//               self included;
//   core        >= min_pts neighbours;
//   cluster     connected component of core points, labelled by its smallest
//               frame-local core index;
//   border      non-core point with a core neighbour: label of the nearest
//               core, ties by smaller (y, x) of that core;
//   noise       label -1.
//
// Design (one workgroup per frame, everything on chip):
//   1. bounding box of the frame's points;
//   2. counting sort of the points into square cells of side s, the largest
//      integer with 2 s^2 <= E^2, so any two points of one cell are
//      neighbours (a cell holding >= min_pts points is all core, and all
//      cores of a cell are connected);
//   3. neighbour counts with early exit at min_pts, scanning for each point
//      the contiguous run of sorted points that covers each row of
//      neighbouring cells (the cells whose nearest corners are within E);
//   4. union-find over core points with min-index hooking: a root is only
//      ever hooked under a smaller index, so every component's final root is
//      its smallest core index whatever the order of the atomic operations;
//   5. flatten, nearest-core border assignment, coalesced output writes.
// Frames with more points than the on-chip capacity go to the multi-workgroup
// path (cluster_big.hip) when the caller's plan provides its workspace;
// otherwise, and for frames wider than 16-bit coordinates, an in-place path
// keeps the union-find forest in the caller's labels array and runs
// brute-force pair tests through LDS tiles (correct for any size, slow).
//
// All results are independent of the order of points within a cell, so the
// nondeterministic order of the LDS atomics in the counting sort cannot
// change any output.

#include <climits>

#include "cluster_common.h"
#include "internal.h"

namespace flock {
namespace {

using namespace cl;

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kTile = 1024;  // points per LDS tile on the in-place path

// ---------------------------------------------------------------------------
// In-place path for frames above the on-chip capacity
// ---------------------------------------------------------------------------

__device__ __forceinline__ void cluster_frame_inplace(const ClusterArgs &a, int f, int32_t b, int32_t n,
                                      unsigned char *smem, int *red) {
    const int2 *P = reinterpret_cast<const int2 *>(a.xy) + b;
    int32_t *par = a.labels + b;
    uint8_t *knd = a.kind + b;
    int2 *tile = reinterpret_cast<int2 *>(smem);
    uint8_t *tcore = reinterpret_cast<uint8_t *>(tile + kTile);
    const Radius r{a.eps_q, a.eps_q + 1, a.eps_q * a.eps_q};
    const int tid = threadIdx.x;

    // A: neighbour counts -> core flags; parent[i] = i
    for (int32_t base = 0; base < n; base += kThreads) {
        const int32_t i = base + tid;
        const bool valid = i < n;
        const int2 pi = valid ? P[i] : make_int2(0, 0);
        int32_t cnt = 0;
        for (int32_t t0 = 0; t0 < n; t0 += kTile) {
            const int32_t tn = min(kTile, n - t0);
            __syncthreads();
            for (int j = tid; j < tn; j += kThreads) tile[j] = P[t0 + j];
            __syncthreads();
            if (valid && cnt < a.min_pts)
                for (int j = 0; j < tn; ++j) cnt += within(pi, tile[j], r) ? 1 : 0;
        }
        if (valid) {
            knd[i] = cnt >= a.min_pts ? 2 : 0;
            st_rlx<kAgent>(par + i, i);
        }
    }
    __syncthreads();

    // B: unite every core pair within eps (each unordered pair once: j < i)
    for (int32_t base = 0; base < n; base += kThreads) {
        const int32_t i = base + tid;
        const bool valid = i < n && knd[i] == 2;
        const int2 pi = i < n ? P[i] : make_int2(0, 0);
        for (int32_t t0 = 0; t0 < base + kThreads && t0 < n; t0 += kTile) {
            const int32_t tn = min(kTile, n - t0);
            __syncthreads();
            for (int j = tid; j < tn; j += kThreads) {
                tile[j] = P[t0 + j];
                tcore[j] = knd[t0 + j];
            }
            __syncthreads();
            if (valid) {
                const int jn = min(tn, i - t0);
                for (int j = 0; j < jn; ++j)
                    if (tcore[j] == 2 && within(pi, tile[j], r)) uf_unite<kAgent>(par, i, t0 + j);
            }
        }
    }
    __syncthreads();

    // C: flatten (read-only traversals; each thread writes only its own root)
    int roots = 0;
    for (int32_t i = tid; i < n; i += kThreads) {
        if (knd[i] != 2) continue;
        int32_t root = uf_root<kAgent>(par, i);
        st_rlx<kAgent>(par + i, root);
        roots += root == i;
    }
    __syncthreads();

    // D: border points take the nearest core's label
    for (int32_t base = 0; base < n; base += kThreads) {
        const int32_t i = base + tid;
        const bool valid = i < n && knd[i] != 2;
        const int2 pi = i < n ? P[i] : make_int2(0, 0);
        int32_t best = -1, best_d2 = INT32_MAX, by = 0, bx = 0;
        for (int32_t t0 = 0; t0 < n; t0 += kTile) {
            const int32_t tn = min(kTile, n - t0);
            __syncthreads();
            for (int j = tid; j < tn; j += kThreads) {
                tile[j] = P[t0 + j];
                tcore[j] = knd[t0 + j];
            }
            __syncthreads();
            if (valid) {
                for (int j = 0; j < tn; ++j) {
                    if (tcore[j] != 2) continue;
                    const int2 q = tile[j];
                    const int32_t d2 = sq_dist_clamped(pi, q, r);
                    if (d2 > r.e2) continue;
                    const bool take = core_before(d2, q.y, q.x, best_d2, by, bx);
                    best = take ? t0 + j : best;
                    best_d2 = take ? d2 : best_d2;
                    by = take ? q.y : by;
                    bx = take ? q.x : bx;
                }
            }
        }
        // all reads of knd by tile loads are done before anyone rewrites it
        __syncthreads();
        if (valid) {
            if (best >= 0) {
                st_rlx<kAgent>(par + i, ld_rlx<kAgent>(par + best));
                knd[i] = 1;
            } else {
                st_rlx<kAgent>(par + i, -1);
                knd[i] = 0;
            }
        }
    }

    roots = wave_sum(roots);
    if ((tid & 63) == 0) atomicAdd(red, roots);
    __syncthreads();
    if (tid == 0 && a.n_clusters) a.n_clusters[f] = *red;
}

// ---------------------------------------------------------------------------
// Resident path: one frame per workgroup, all state in LDS
// ---------------------------------------------------------------------------

constexpr uint16_t kNone = 0xffff;
// Per-point kind byte (by sorted position): the output kinds, plus a marker
// for a non-core point with no neighbour but itself (noise, no border search).
constexpr uint8_t kBorder = 1;
constexpr uint8_t kCore = 2;
constexpr uint8_t kIsolated = 3;
constexpr int kMaxOffsets = 16;
// Neighbour cells lie within +-reach cells, and reach <= 2 for every eps:
// reach = 1 + (E - 1) / side with side >= max(1, floor(E / sqrt 2)) > (E - 1) / 2.
// So the full stencil has at most 5 x 5 cells.
constexpr int kMaxStencil = 25;
constexpr int kBorderLanes = 8;  // lanes that share one border candidate
// Points per thread held in registers during the sort: the planner keeps a
// resident frame at <= kThreads * kPtsPerThread points.  The compact kernel
// (two workgroups per compute unit) holds kPtsCompact per thread, which
// keeps it within 64 VGPRs (8 waves per SIMD).
constexpr int kPtsPerThread = 10;
constexpr int kPtsCompact = 5;
static_assert(kClusterCompactCap == kThreads * kPtsCompact, "compact capacity");

// Coordinates relative to the frame's bounding-box corner, packed as
// x | y << 16 (the resident path takes frames whose extent fits 16 bits).
__device__ __forceinline__ int32_t pk_x(uint32_t v) { return (int32_t)(v & 0xffffu); }
__device__ __forceinline__ int32_t pk_y(uint32_t v) { return (int32_t)(v >> 16); }

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Squared distance of two packed points, per axis clamped to E + 1, on both
// 16-bit halves at once: |a - b| = max - min, then dx^2 + dy^2 by one 16-bit
// dot product (<= 2 (E + 1)^2 < 2^31 for E <= 32766).
__device__ __forceinline__ int32_t sq_dist_pk(uint32_t a, uint32_t b, int32_t e1) {
    const u16x2 ua = __builtin_bit_cast(u16x2, a), ub = __builtin_bit_cast(u16x2, b);
    const u16x2 lim = {(unsigned short)e1, (unsigned short)e1};
    const u16x2 d = __builtin_elementwise_min(__builtin_elementwise_max(ua, ub) - __builtin_elementwise_min(ua, ub),
                                              lim);
    return (int32_t)__builtin_amdgcn_udot2(d, d, 0u, false);
}

// Cell geometry of one frame (relative coordinates).
struct Grid {
    int32_t side;        // cell side (quanta)
    float inv_side;
    int32_t ncx, ncy;    // cells per axis
    int32_t ncell;
    int32_t reach;       // neighbour cells lie within +-reach cells
    const int32_t *dxmax;  // [reach + 1] in LDS: per |dy|, widest |dx| whose cells can hold neighbours
    bool dense_ok;       // side is the eps-diagonal side: same cell => neighbours
};

// floor(v / side) for 0 <= v < 2^16, via a float reciprocal and one
// branch-free correction (the product is within one of the quotient, and
// c * side stays below 2^24, so 24-bit multiplies are exact).
__device__ __forceinline__ int32_t cell_coord(int32_t v, const Grid &g, int32_t ncoord) {
    int32_t c = (int32_t)((float)v * g.inv_side);
    const int32_t cs = __mul24(c, g.side);
    c += (int32_t)(cs + g.side <= v) - (int32_t)(cs > v);
    return min(max(c, 0), ncoord - 1);
}

__device__ __forceinline__ int32_t cell_id(uint32_t v, const Grid &g, int32_t *cx, int32_t *cy) {
    *cx = cell_coord(pk_x(v), g, g.ncx);
    *cy = cell_coord(pk_y(v), g, g.ncy);
    return *cy * g.ncx + *cx;
}

// Neighbours of v among sorted points [q0, q1), stopping once `need` are seen.
__device__ __forceinline__ int32_t count_span(const uint32_t *pxy, int32_t q0, int32_t q1, uint32_t v,
                                              const Radius &r, int32_t need) {
    int32_t cnt = 0;
    int32_t q = q0;
    for (; q + 4 <= q1; q += 4) {
        const uint32_t w0 = pxy[q], w1 = pxy[q + 1], w2 = pxy[q + 2], w3 = pxy[q + 3];
        cnt += (sq_dist_pk(v, w0, r.e1) <= r.e2) + (sq_dist_pk(v, w1, r.e1) <= r.e2) +
               (sq_dist_pk(v, w2, r.e1) <= r.e2) + (sq_dist_pk(v, w3, r.e1) <= r.e2);
        if (cnt >= need) return cnt;
    }
    for (; q < q1; ++q) cnt += sq_dist_pk(v, pxy[q], r.e1) <= r.e2;
    return cnt;
}

// floor(x / d) for 0 <= x < 2^22, 1 <= d, from a float reciprocal and one
// correction step.
__device__ __forceinline__ int32_t div_small(int32_t x, int32_t d, float inv_d) {
    int32_t q = (int32_t)((float)x * inv_d);
    const int32_t qd = __mul24(q, d);  // below 2^23: exact
    q += (int32_t)(qd + d <= x) - (int32_t)(qd > x);
    return q;
}

// Neighbour-cell tables of one frame, built by the 64 lanes of one wave.
// Cell offset (dx, dy), |dx|, |dy| <= reach <= 2, can hold a neighbour iff the
// gap between the two cells, gap(|dx|)^2 + gap(|dy|)^2, is <= E^2.
//   sdx/sdy   the whole stencil, nearest cells first (ties in lane order)
//   fdx/fdy   its forward half (cells later in row-major order), the
//             nadj adjacent cells first, nfwd in all (at most 4 + 8)
//   dxmax[k]  the widest |dx| in row |dy| = k
__device__ __forceinline__ void build_stencil(int32_t reach, int32_t side, const Radius &r, int lane, int *dxmax, int *sdx,
                              int *sdy, int *nsten, int *fdx, int *fdy, int *nadj, int *nfwd) {
    const int dx = lane % 5 - 2, dy = lane / 5 - 2;
    const int adx = dx < 0 ? -dx : dx, ady = dy < 0 ? -dy : dy;
    bool valid = false;
    uint32_t key = 0xffffffffu;
    if (lane < kMaxStencil && adx <= reach && ady <= reach) {
        const int64_t gx = cell_gap(adx, side), gy = cell_gap(ady, side);
        const int64_t d = gx * gx + gy * gy;
        valid = d <= (int64_t)r.e2;
        key = valid ? (uint32_t)d : key;
    }
    int rank = 0;
    for (int u = 0; u < kMaxStencil; ++u) {
        const uint32_t ku = __shfl(key, u, 64);
        rank += (ku < key) | ((ku == key) & (u < lane));
    }
    const uint64_t vm = __ballot(valid);
    if (valid) {
        sdx[rank] = dx;
        sdy[rank] = dy;
    }
    const bool fwd = valid && (dy > 0 || (dy == 0 && dx > 0));
    const bool adj = adx <= 1 && ady <= 1;
    const uint64_t m0 = __ballot(fwd && adj), m1 = __ballot(fwd && !adj);
    const uint64_t below = (1ull << lane) - 1ull;
    if (fwd) {
        const int at = adj ? __popcll(m0 & below) : __popcll(m0) + __popcll(m1 & below);
        fdx[at] = dx;
        fdy[at] = dy;
    }
    if (lane <= 2) {  // row dy = lane: valid cells are |dx| <= dxmax, a symmetric run
        const int cnt = __popcll((vm >> ((lane + 2) * 5)) & 31ull);
        dxmax[lane] = cnt > 0 ? (cnt - 1) / 2 : 0;
    }
    if (lane == 0) {
        *nsten = __popcll(vm);
        *nadj = __popcll(m0);
        *nfwd = __popcll(m0) + __popcll(m1);
    }
}

// The first two points of a cell (the first one twice in a one-point cell)
// and their core flags.
struct CellHead {
    uint32_t p0, p1;
    bool c0, c1;
};

__device__ __forceinline__ CellHead cell_head(const uint32_t *pxy, const uint8_t *score, int32_t q0, int32_t q1) {
    const int32_t q = min(q0 + 1, q1 - 1);
    return CellHead{pxy[q0], pxy[q], score[q0] == kCore, score[q] == kCore};
}

// Some core pair among the first two points of each cell within eps: in
// clustered frames this settles about nine adjacent cell pairs in ten.
__device__ __forceinline__ bool heads_touch(const CellHead &A, const CellHead &B, const Radius &r) {
    return (A.c0 & B.c0 & (sq_dist_pk(A.p0, B.p0, r.e1) <= r.e2)) |
           (A.c0 & B.c1 & (sq_dist_pk(A.p0, B.p1, r.e1) <= r.e2)) |
           (A.c1 & B.c0 & (sq_dist_pk(A.p1, B.p0, r.e1) <= r.e2)) |
           (A.c1 & B.c1 & (sq_dist_pk(A.p1, B.p1, r.e1) <= r.e2));
}

// True if some core of sorted points [a0, a1) lies within eps of some core of
// [b0, b1) (scalar loops with early exit).
__device__ __forceinline__ bool cells_touch(const uint32_t *pxy, const uint8_t *score, int32_t a0, int32_t a1,
                                            int32_t b0, int32_t b1, const Radius &r) {
    for (int32_t qa = a0; qa < a1; ++qa) {
        if (score[qa] != kCore) continue;
        const uint32_t va = pxy[qa];
        for (int32_t qb = b0; qb < b1; ++qb)
            if ((score[qb] == kCore) & (sq_dist_pk(va, pxy[qb], r.e1) <= r.e2)) return true;
    }
    return false;
}

// A core cell of the work list: its id, column and row, sorted range
// [a0, a1), node (smallest core index) and first two points.
struct CoreCell {
    int32_t ca, ax, ay, a0, a1, node;
    CellHead head;
};

constexpr uint32_t kDeadPair = 0xffffffffu;

// Exclusive prefix sum and total over the wave of per-lane counts below 16
// (wave-uniform call): one ballot per bit of the count.
__device__ __forceinline__ int wave_prefix16(int cnt, int *total) {
    const uint64_t below = (1ull << (threadIdx.x & 63)) - 1ull;
    int pre = 0, tot = 0;
#pragma unroll
    for (int bit = 0; bit < 4; ++bit) {
        const uint64_t m = __ballot((cnt >> bit) & 1);
        pre += __popcll(m & below) << bit;
        tot += __popcll(m) << bit;
    }
    *total = tot;
    return pre;
}

// Edges from core cell A (if `have`) to its neighbours at the forward offsets
// fdx/fdy[o0 + k], k < NO, o0 + k < o1 (wave-uniform call): bit k of the
// result is set when some core of A lies within eps of some core of the
// neighbour.  All cores of a cell are neighbours, so a cell's cores form one
// node of the graph (its smallest core index).
//   far = false: every neighbour holding a core;
//   far = true:  only neighbours whose root differs from A's (the forest is
//                flat here, so equal roots mean already connected).
// The first two points of both cells settle most pairs.  The pairs they leave
// open go to `queue` as (cell A | cell B << 16), to be tested after a barrier
// by one lane each, so that the few long scans share a few waves instead of
// holding up every wave; pairs beyond its capacity are tested here.
template <int NO, bool far>
__device__ __forceinline__ uint32_t cell_edges(bool have, const CoreCell &A, const uint32_t *cell,
                                               const int32_t *parent, const uint32_t *pxy, const uint8_t *score,
                                               const Grid &g, const Radius &r, const int *fdx, const int *fdy,
                                               int o0, int o1, uint32_t *queue, int *nq, int qcap) {
    const int32_t ra = far && have ? ld_rlx<kGroup>(parent + A.node) : 0;
    uint32_t touch = 0, open = 0;
    int32_t cbs[NO];
#pragma unroll
    for (int k = 0; k < NO; ++k) {
        cbs[k] = 0;
        const int o = o0 + k;
        if (!have || o >= o1) continue;
        const int32_t bx = A.ax + fdx[o], by = A.ay + fdy[o];
        if ((bx < 0) | (bx >= g.ncx) | (by >= g.ncy)) continue;
        const int32_t cb = by * g.ncx + bx;
        cbs[k] = cb;
        const uint32_t wb = cell[cb];
        const int32_t nb = (int32_t)(wb >> 16);
        if (nb == (int32_t)kNone) continue;
        if (far && ld_rlx<kGroup>(parent + nb) == ra) continue;
        const int32_t b0 = (int32_t)(wb & 0xffffu), b1 = (int32_t)(cell[cb + 1] & 0xffffu);
        const CellHead B = cell_head(pxy, score, b0, b1);
        if (heads_touch(A.head, B, r)) touch |= 1u << k;
        else if ((A.a1 - A.a0 > 2) | (b1 - b0 > 2)) open |= 1u << k;
    }
    int total;
    const int pre = wave_prefix16(__popc(open), &total);
    if (total == 0) return touch;  // wave-uniform
    int base = 0;
    if ((threadIdx.x & 63) == 0) base = atomicAdd(nq, total);
    base = __shfl(base, 0, 64);
    int at = base + pre;
#pragma unroll
    for (int k = 0; k < NO; ++k) {
        if (!((open >> k) & 1u)) continue;
        const int32_t cb = cbs[k];
        if (at < qcap) {
            queue[at] = (uint32_t)A.ca | ((uint32_t)cb << 16);
        } else if (cells_touch(pxy, score, A.a0, A.a1, (int32_t)(cell[cb] & 0xffffu),
                               (int32_t)(cell[cb + 1] & 0xffffu), r)) {
            touch |= 1u << k;
        }
        ++at;
    }
    return touch;
}

// Tests the queued cell pairs, one lane each; a pair with no core pair within
// eps is marked dead.
__device__ __forceinline__ void resolve_queue(uint32_t *queue, int nq, const uint32_t *cell, const uint32_t *pxy,
                                              const uint8_t *score, const Radius &r) {
    for (int t = threadIdx.x; t < nq; t += kThreads) {
        const uint32_t e = queue[t];
        const int32_t ca = (int32_t)(e & 0xffffu), cb = (int32_t)(e >> 16);
        if (!cells_touch(pxy, score, (int32_t)(cell[ca] & 0xffffu), (int32_t)(cell[ca + 1] & 0xffffu),
                         (int32_t)(cell[cb] & 0xffffu), (int32_t)(cell[cb + 1] & 0xffffu), r))
            queue[t] = kDeadPair;
    }
}

// Hook step of the connected-components rounds for node a and its neighbours
// nb[k] (bit k of m): their parents (roots as of the last jump step, or
// parents lowered since, all within the components of these nodes) are
// joined under the smallest of them by an atomic minimum, which keeps
// parent[x] <= x.  Returns true if any two differed.
template <int NO>
__device__ __forceinline__ bool hook_node(int32_t *parent, int32_t a, const int32_t (&nb)[NO], uint32_t m) {
    const int32_t pa = ld_rlx<kGroup>(parent + a);
    int32_t pb[NO];
    int32_t lo = pa;
#pragma unroll
    for (int k = 0; k < NO; ++k) {
        pb[k] = ((m >> k) & 1u) ? ld_rlx<kGroup>(parent + nb[k]) : pa;
        lo = min(lo, pb[k]);
    }
    bool any = false;
    if (pa != lo) {
        __hip_atomic_fetch_min(parent + pa, lo, __ATOMIC_RELAXED, kGroup);
        any = true;
    }
#pragma unroll
    for (int k = 0; k < NO; ++k)
        if (pb[k] != lo) {
            __hip_atomic_fetch_min(parent + pb[k], lo, __ATOMIC_RELAXED, kGroup);
            any = true;
        }
    return any;
}

// hook_node for the register stages, whose neighbour nodes are kept two to a
// register (node ids are below 2^16): entry k is the low half of nbp[k / 2]
// for even k, the high half for odd k.
template <int NO>
__device__ __forceinline__ bool hook_node_packed(int32_t *parent, int32_t a, const uint32_t (&nbp)[NO / 2],
                                                 uint32_t m) {
    int32_t nb[NO];
#pragma unroll
    for (int k = 0; k < NO; ++k) nb[k] = (int32_t)((k & 1) ? nbp[k >> 1] >> 16 : nbp[k >> 1] & 0xffffu);
    return hook_node<NO>(parent, a, nb, m);
}

template <int NO>
__device__ __forceinline__ void pack_nodes(const int32_t (&nb)[NO], uint32_t (&nbp)[NO / 2]) {
#pragma unroll
    for (int k = 0; k < NO / 2; ++k) nbp[k] = ((uint32_t)nb[2 * k] & 0xffffu) | ((uint32_t)nb[2 * k + 1] << 16);
}

// Jump step: node a's parent becomes its root (read-only walk; concurrent
// writers only store roots, so every walk ends at the same root).
__device__ __forceinline__ void jump_node(int32_t *parent, int32_t a) {
    int32_t x = ld_rlx<kGroup>(parent + a);
    for (;;) {
        const int32_t p = ld_rlx<kGroup>(parent + x);
        if (p == x) break;
        x = p;
    }
    st_rlx<kGroup>(parent + a, x);
}

// Core cells per lane whose node, neighbour nodes and edge bits stay in
// registers through the connected-components rounds.
constexpr int kRegCells = 3;

// State of one frame that the union stages share.
struct UnionCtx {
    uint32_t *cell;  // the node half holds roots after the adjacent stage
    int32_t *parent;
    const uint32_t *pxy;
    const uint8_t *score;
    const uint16_t *clist;
    uint16_t *emask;  // edge bits per core cell; 4-byte aligned
    uint32_t *queue;  // open pairs: core-cell index j | offset index k << 16
    int qcap;
    int *nq;
    int *hook3;
    const int *fdx, *fdy;
    Grid g;
    Radius r;
    int32_t ncl;
    float inv_ncx;
};

__device__ __forceinline__ CoreCell load_core_cell(const UnionCtx &u, int32_t j, bool have) {
    CoreCell A{};
    if (have) {
        A.ca = u.clist[j];
        A.ay = div_small(A.ca, u.g.ncx, u.inv_ncx);
        A.ax = A.ca - A.ay * u.g.ncx;
        const uint32_t wa = u.cell[A.ca];
        A.a0 = (int32_t)(wa & 0xffffu);
        A.a1 = (int32_t)(u.cell[A.ca + 1] & 0xffffu);
        A.node = (int32_t)(wa >> 16);
        A.head = cell_head(u.pxy, u.score, A.a0, A.a1);
    }
    return A;
}

// cell_edges for the register stages: also returns every neighbour's node in
// nb[k] (A's own node where there is none), and queues open pairs as
// (j | k << 16) for resolve_queue_coop.
template <int NO, bool far>
__device__ __forceinline__ uint32_t cell_edges_nb(bool have, const CoreCell &A, int32_t j, const UnionCtx &u, int o0,
                                                  int o1, int32_t (&nb)[NO]) {
    const int32_t ra = far && have ? ld_rlx<kGroup>(u.parent + A.node) : 0;
    uint32_t touch = 0, open = 0;
    int32_t cbs[NO];
#pragma unroll
    for (int k = 0; k < NO; ++k) {
        nb[k] = A.node;
        cbs[k] = 0;
        const int o = o0 + k;
        if (!have || o >= o1) continue;
        const int32_t bx = A.ax + u.fdx[o], by = A.ay + u.fdy[o];
        if ((bx < 0) | (bx >= u.g.ncx) | (by >= u.g.ncy)) continue;
        const int32_t cb = by * u.g.ncx + bx;
        cbs[k] = cb;
        const uint32_t wb = u.cell[cb];
        const int32_t n = (int32_t)(wb >> 16);
        if (n == (int32_t)kNone) continue;
        nb[k] = n;
        if (far && ld_rlx<kGroup>(u.parent + n) == ra) continue;
        const int32_t b0 = (int32_t)(wb & 0xffffu), b1 = (int32_t)(u.cell[cb + 1] & 0xffffu);
        const CellHead B = cell_head(u.pxy, u.score, b0, b1);
        if (heads_touch(A.head, B, u.r)) touch |= 1u << k;
        else if ((A.a1 - A.a0 > 2) | (b1 - b0 > 2)) open |= 1u << k;
    }
    int total;
    const int pre = wave_prefix16(__popc(open), &total);
    if (total == 0) return touch;  // wave-uniform
    int base = 0;
    if ((threadIdx.x & 63) == 0) base = atomicAdd(u.nq, total);
    base = __shfl(base, 0, 64);
    int at = base + pre;
#pragma unroll
    for (int k = 0; k < NO; ++k) {
        if (!((open >> k) & 1u)) continue;
        const int32_t cb = cbs[k];
        if (at < u.qcap) {
            u.queue[at] = (uint32_t)j | ((uint32_t)k << 16);
        } else if (cells_touch(u.pxy, u.score, A.a0, A.a1, (int32_t)(u.cell[cb] & 0xffffu),
                               (int32_t)(u.cell[cb + 1] & 0xffffu), u.r)) {
            touch |= 1u << k;
        }
        ++at;
    }
    return touch;
}

// True if core point va has a core neighbour among the sorted points q0,
// q0 + step, ... below q1 (four loads in flight at a time).
__device__ __forceinline__ bool core_near_strided(const UnionCtx &u, uint32_t va, int32_t q0, int32_t q1,
                                                  int32_t step) {
    int32_t q = q0;
    for (; q + 3 * step < q1; q += 4 * step) {
        const uint32_t w0 = u.pxy[q], w1 = u.pxy[q + step], w2 = u.pxy[q + 2 * step], w3 = u.pxy[q + 3 * step];
        const bool h = ((u.score[q] == kCore) & (sq_dist_pk(va, w0, u.r.e1) <= u.r.e2)) |
                       ((u.score[q + step] == kCore) & (sq_dist_pk(va, w1, u.r.e1) <= u.r.e2)) |
                       ((u.score[q + 2 * step] == kCore) & (sq_dist_pk(va, w2, u.r.e1) <= u.r.e2)) |
                       ((u.score[q + 3 * step] == kCore) & (sq_dist_pk(va, w3, u.r.e1) <= u.r.e2));
        if (h) return true;
    }
    for (; q < q1; q += step)
        if ((u.score[q] == kCore) & (sq_dist_pk(va, u.pxy[q], u.r.e1) <= u.r.e2)) return true;
    return false;
}

// Most lanes that share one queued pair in resolve_queue_coop.
constexpr int kMaxPairLanes = 8;

// Tests the queued pairs (j | k << 16) in one pass where they fit: G lanes
// per pair (a power of two, at most kMaxPairLanes, with nq G <= kThreads where
// possible).  Lane i of a group takes core cell j's points i, i + G, ... and
// scans all of cell B (at offset o0 + k) for a core within eps, stopping at
// its first hit; a hit in the group sets bit k of cell j's edge bits.
// Wave-uniform call.
__device__ __forceinline__ void resolve_queue_coop(const UnionCtx &u, int nq, int o0) {
    uint32_t *mask32 = reinterpret_cast<uint32_t *>(u.emask);
    const int tid = threadIdx.x, lane = tid & 63;
    int G = 1;
    while (G < kMaxPairLanes && nq * 2 * G <= kThreads) G *= 2;
    const int gl = lane & (G - 1);
    const uint64_t gmask = ((1ull << G) - 1ull) << (lane & ~(G - 1));
    for (int t0 = (tid - lane) / G; t0 < nq; t0 += kThreads / G) {
        const int t = t0 + lane / G;
        bool hit = false;
        int32_t j = 0, k = 0;
        if (t < nq) {
            const uint32_t e = u.queue[t];
            j = (int32_t)(e & 0xffffu);
            k = (int32_t)(e >> 16);
            const int32_t ca = u.clist[j];
            const int32_t ay = div_small(ca, u.g.ncx, u.inv_ncx), ax = ca - ay * u.g.ncx;
            const int32_t cb = (ay + u.fdy[o0 + k]) * u.g.ncx + ax + u.fdx[o0 + k];
            const int32_t a1 = (int32_t)(u.cell[ca + 1] & 0xffffu);
            const int32_t b0 = (int32_t)(u.cell[cb] & 0xffffu), b1 = (int32_t)(u.cell[cb + 1] & 0xffffu);
            for (int32_t qa = (int32_t)(u.cell[ca] & 0xffffu) + gl; qa < a1 && !hit; qa += G)
                if (u.score[qa] == kCore) hit = core_near_strided(u, u.pxy[qa], b0, b1, 1);
        }
        const uint64_t hits = __ballot(hit);
        if (gl == 0 && (hits & gmask)) atomicOr(mask32 + (j >> 1), (1u << k) << (16 * (j & 1)));
    }
}

// Far-stage candidates of core cell A (cell ca at column ax, row ay, root ra
// in the cell table): the neighbours at offsets o0 + k, k < NO, o0 + k < o1,
// that hold a core and have another root; nb[k] gets that root (ra where
// there is none).  Candidates go to the queue as (j | k << 16), or, beyond its
// capacity, are tested here (bit k of the result).  Wave-uniform call.
template <int NO>
__device__ __forceinline__ uint32_t far_candidates(bool have, int32_t ca, int32_t ax, int32_t ay, int32_t ra,
                                                   int32_t j, const UnionCtx &u, int o0, int o1,
                                                   int32_t (&nb)[NO]) {
    uint32_t cand = 0;
    int32_t cbs[NO];
#pragma unroll
    for (int k = 0; k < NO; ++k) {
        nb[k] = ra;
        cbs[k] = 0;
        const int o = o0 + k;
        if (!have || o >= o1) continue;
        const int32_t bx = ax + u.fdx[o], by = ay + u.fdy[o];
        if ((bx < 0) | (bx >= u.g.ncx) | (by >= u.g.ncy)) continue;
        const int32_t cb = by * u.g.ncx + bx;
        const int32_t rb = (int32_t)(u.cell[cb] >> 16);
        if ((rb == (int32_t)kNone) | (rb == ra)) continue;
        nb[k] = rb;
        cbs[k] = cb;
        cand |= 1u << k;
    }
    int total;
    const int pre = wave_prefix16(__popc(cand), &total);
    if (total == 0) return 0;  // wave-uniform
    int base = 0;
    if ((threadIdx.x & 63) == 0) base = atomicAdd(u.nq, total);
    base = __shfl(base, 0, 64);
    int at = base + pre;
    uint32_t touch = 0;
#pragma unroll
    for (int k = 0; k < NO; ++k) {
        if (!((cand >> k) & 1u)) continue;
        if (at < u.qcap) {
            u.queue[at] = (uint32_t)j | ((uint32_t)k << 16);
        } else {
            const int32_t cb = cbs[k];
            if (cells_touch(u.pxy, u.score, (int32_t)(u.cell[ca] & 0xffffu), (int32_t)(u.cell[ca + 1] & 0xffffu),
                            (int32_t)(u.cell[cb] & 0xffffu), (int32_t)(u.cell[cb + 1] & 0xffffu), u.r))
                touch |= 1u << k;
        }
        ++at;
    }
    return touch;
}

// Connected-components rounds over every lane's core cells (j = tid +
// c kThreads; node, neighbour nodes nb and edge bits m in registers): hook
// every edge's two roots under the smaller, then every node jumps to its
// root, until a round hooks nothing.  `round` numbers the rounds across
// stages (hook3[round % 3] says whether round `round` hooked; three slots, so
// that one is cleared while the previous one may still be read).
// Wave-uniform call.
template <int NO>
__device__ __forceinline__ void cc_rounds(const UnionCtx &u, const int32_t (&node)[kRegCells],
                                          const uint32_t (&nbp)[kRegCells][NO / 2], const uint32_t (&m)[kRegCells],
                                          int &round) {
    const int tid = threadIdx.x;
    // a round that hooks leaves fewer roots, so ncl + 1 rounds always
    // suffice; the bound only guarantees that the loop ends
    const int last = round + u.ncl + 1;
    for (;; ++round) {
        if (tid == 0) u.hook3[(round + 1) % 3] = 0;
        bool any = false;
#pragma unroll
        for (int c = 0; c < kRegCells; ++c)
            if (m[c]) any |= hook_node_packed<NO>(u.parent, node[c], nbp[c], m[c]);
        if (any) u.hook3[round % 3] = 1;
        __syncthreads();
        if (!u.hook3[round % 3] || round >= last) break;  // every edge joins equal roots
#pragma unroll
        for (int c = 0; c < kRegCells; ++c)
            if (tid + c * kThreads < u.ncl) jump_node(u.parent, node[c]);
        __syncthreads();
    }
    ++round;
}

// The cell unions with every lane's core cells (j = tid + c kThreads) in
// registers.  Adjacent stage: edges from the first two points of both cells,
// open pairs tested by resolve_queue_coop, then rounds.  Each core cell's
// root then replaces its node in the cell table (any member of a tree serves
// as its node from here on).  Far stage: only pairs with different roots are
// candidates, all tested by resolve_queue_coop, then rounds.  Wave-uniform
// call.
__device__ __forceinline__ void union_regs(const UnionCtx &u, int nadj, int nfwd, int &round) {
    const int tid = threadIdx.x, lane = tid & 63;
    int32_t ca[kRegCells], node[kRegCells];
    {
        uint32_t nbp[kRegCells][2];
        uint32_t m[kRegCells];
        if (tid == 0) *u.nq = 0;
        __syncthreads();
#pragma unroll
        for (int c = 0; c < kRegCells; ++c) {
            const int32_t j = tid + c * kThreads;
            const bool have = j < u.ncl;
            ca[c] = 0;
            node[c] = 0;
#pragma unroll
            for (int k = 0; k < 2; ++k) nbp[c][k] = 0;
            if (tid - lane + c * kThreads >= u.ncl) continue;  // wave-uniform
            const CoreCell A = load_core_cell(u, j, have);
            ca[c] = A.ca;
            node[c] = A.node;
            int32_t nb[4];
            const uint32_t t = cell_edges_nb<4, false>(have, A, j, u, 0, nadj, nb);
            pack_nodes<4>(nb, nbp[c]);
            if (have) u.emask[j] = (uint16_t)t;
        }
        __syncthreads();
        resolve_queue_coop(u, min(*u.nq, u.qcap), 0);
        __syncthreads();
#pragma unroll
        for (int c = 0; c < kRegCells; ++c) m[c] = tid + c * kThreads < u.ncl ? u.emask[tid + c * kThreads] : 0u;
        cc_rounds<4>(u, node, nbp, m, round);
    }
#pragma unroll
    for (int c = 0; c < kRegCells; ++c)
        if (tid + c * kThreads < u.ncl)
            u.cell[ca[c]] = (u.cell[ca[c]] & 0xffffu) | ((uint32_t)ld_rlx<kGroup>(u.parent + node[c]) << 16);
    if (tid == 0) *u.nq = 0;
    __syncthreads();
    {
        uint32_t nbp[kRegCells][4];
        uint32_t m[kRegCells];
#pragma unroll
        for (int c = 0; c < kRegCells; ++c) {
            const int32_t j = tid + c * kThreads;
            const bool have = j < u.ncl;
#pragma unroll
            for (int k = 0; k < 4; ++k) nbp[c][k] = 0;
            if (tid - lane + c * kThreads >= u.ncl) continue;  // wave-uniform
            const int32_t ay = div_small(ca[c], u.g.ncx, u.inv_ncx), ax = ca[c] - ay * u.g.ncx;
            const int32_t ra = have ? (int32_t)(u.cell[ca[c]] >> 16) : 0;
            int32_t nb[8];
            const uint32_t t = far_candidates<8>(have, ca[c], ax, ay, ra, j, u, nadj, nfwd, nb);
            pack_nodes<8>(nb, nbp[c]);
            if (have) u.emask[j] = (uint16_t)t;
        }
        __syncthreads();
        resolve_queue_coop(u, min(*u.nq, u.qcap), nadj);
        __syncthreads();
#pragma unroll
        for (int c = 0; c < kRegCells; ++c) m[c] = tid + c * kThreads < u.ncl ? u.emask[tid + c * kThreads] : 0u;
        cc_rounds<8>(u, node, nbp, m, round);
    }
}

// Append `flag` lanes' values to list[] (wave-uniform call: every lane of the
// wave must reach it).
__device__ __forceinline__ void wave_append(bool flag, uint16_t value, uint16_t *list, int *counter) {
    const uint64_t m = __ballot(flag);
    if (m == 0) return;
    const int lane = threadIdx.x & 63;
    int base = 0;
    if (lane == 0) base = atomicAdd(counter, __popcll(m));
    base = __shfl(base, 0, 64);
    if (flag) list[base + __popcll(m & ((1ull << lane) - 1ull))] = value;
}

// One frame per workgroup, PTS points per thread in the register sort (a
// frame of up to kThreads * PTS points fits).
template <int PTS>
__device__ __forceinline__ void cluster_resident(const ClusterArgs &a) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ int s_bbox[4];
    __shared__ int s_wave[kWaves];
    __shared__ int s_red;
    __shared__ int s_nlist;
    __shared__ int s_ncells;
    __shared__ int s_nadj, s_nfwd;
    __shared__ int s_nq;
    __shared__ int s_hook[3];
    __shared__ int s_fdx[kMaxOffsets];
    __shared__ int s_fdy[kMaxOffsets];
    __shared__ int s_nsten;
    __shared__ int s_sdx[kMaxStencil];
    __shared__ int s_sdy[kMaxStencil];
    __shared__ int s_dxmax[8];

    const int f = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int32_t b = a.offsets[f];
    const int32_t e = a.offsets[f + 1];
    if (b < 0 || e < b || e > a.total) {
        if (tid == 0 && a.n_clusters) a.n_clusters[f] = -1;
        return;
    }
    const int32_t n = e - b;
    if (n == 0) {
        if (tid == 0 && a.n_clusters) a.n_clusters[f] = 0;
        return;
    }
    if (tid == 0) {
        s_bbox[0] = INT_MAX;
        s_bbox[1] = INT_MAX;
        s_bbox[2] = INT_MIN;
        s_bbox[3] = INT_MIN;
        s_red = 0;
        s_nlist = 0;
        s_ncells = 0;
    }
    if (n > a.cap_points && a.big_path) return;  // the multi-workgroup path owns this frame

    const int2 *P = reinterpret_cast<const int2 *>(a.xy) + b;
    const Radius r{a.eps_q, a.eps_q + 1, a.eps_q * a.eps_q};

    // 1. bounding box; each thread keeps its points (i = tid + k * kThreads)
    //    in registers for the sort
    const bool fits = n <= a.cap_points;
    int2 pt[PTS];
#pragma unroll
    for (int k = 0; k < PTS; ++k) {
        const int32_t i = tid + k * kThreads;
        pt[k] = fits && i < n ? P[i] : make_int2(0, 0);
    }
    if (fits) {
        int xmn = INT_MAX, ymn = INT_MAX, xmx = INT_MIN, ymx = INT_MIN;
#pragma unroll
        for (int k = 0; k < PTS; ++k) {
            if (tid + k * kThreads >= n) break;
            xmn = min(xmn, pt[k].x);
            ymn = min(ymn, pt[k].y);
            xmx = max(xmx, pt[k].x);
            ymx = max(ymx, pt[k].y);
        }
        xmn = wave_min(xmn);
        ymn = wave_min(ymn);
        xmx = wave_max(xmx);
        ymx = wave_max(ymx);
        __syncthreads();  // s_bbox initialised
        if (lane == 0) {
            atomicMin(&s_bbox[0], xmn);
            atomicMin(&s_bbox[1], ymn);
            atomicMax(&s_bbox[2], xmx);
            atomicMax(&s_bbox[3], ymx);
        }
        __syncthreads();
    }
    const int32_t x0 = s_bbox[0], y0 = s_bbox[1];
    const uint32_t wx = (uint32_t)(s_bbox[2] - x0), wy = (uint32_t)(s_bbox[3] - y0);
    // frames above the LDS capacity, or whose extent needs more than 16 bits,
    // keep their data off chip
    if (!fits || wx > 0xffffu || wy > 0xffffu) {
        __syncthreads();
        cluster_frame_inplace(a, f, b, n, smem, &s_red);
        return;
    }

    // LDS layout (cap points, cc cells):
    //   pxy    uint32[cap]   packed relative coordinates, sorted by cell
    //   parent int32 [cap]   union-find forest, then labels (original index)
    //   cell   uint32[cc+1]  first sorted position (low 16 bits) | smallest
    //                        core index in the cell, 0xffff if none (high 16)
    //   sid    uint16[cap]   original index of each sorted position
    //   list   uint16[cap]   work list (then edge bits and queue, then the
    //                        border list, then kinds by original index)
    //   clist  uint16[cc]    each cell's offset in the work list (sort),
    //                        then the cells that hold a core
    //   score  uint8 [cap]   kind by sorted position (kCore, kBorder,
    //                        kIsolated, 0 for noise)
    const int32_t cap = a.cap_points, cc = a.cap_cells;
    uint32_t *pxy = reinterpret_cast<uint32_t *>(smem);
    int32_t *parent = reinterpret_cast<int32_t *>(pxy + cap);
    uint32_t *cell = reinterpret_cast<uint32_t *>(parent + cap);
    uint16_t *sid = reinterpret_cast<uint16_t *>(cell + cc + 1);
    uint16_t *list = sid + cap;
    uint16_t *clist = list + cap;
    uint8_t *score = reinterpret_cast<uint8_t *>(clist + cc);
    auto cstart = [cell](int32_t c) -> int32_t { return (int32_t)(cell[c] & 0xffffu); };
    auto cnode = [cell](int32_t c) -> uint32_t { return cell[c] >> 16; };

    // 2. cell grid (every thread derives the same values)
    Grid g;
    {
        uint32_t side = (uint32_t)a.cell_side;
        uint32_t ncx = wx / side + 1, ncy = wy / side + 1;
        while ((uint64_t)ncx * ncy > (uint64_t)cc) {
            side *= 2u;
            ncx = wx / side + 1;
            ncy = wy / side + 1;
        }
        g.side = (int32_t)side;
        g.inv_side = 1.0f / (float)side;
        g.ncx = (int32_t)ncx;
        g.ncy = (int32_t)ncy;
        g.ncell = g.ncx * g.ncy;
        g.dense_ok = side == (uint32_t)a.cell_side;
        // side >= floor(E / sqrt 2) keeps reach <= 2 for every E
        g.reach = r.e == 0 ? 0 : min(1 + (r.e - 1) / g.side, 7);
        g.dxmax = s_dxmax;
    }

    // 3. counting sort by cell (the stencil tables come from the host for
    //    cells of side cell_side; wave 0 builds them for a coarsened grid)
    for (int32_t c = tid; c <= g.ncell; c += kThreads) cell[c] = 0;
    if (g.dense_ok) {
        if (tid < kMaxStencil) {
            const uint32_t w = tid < 5 ? a.sten_all[0] : tid < 10 ? a.sten_all[1] : tid < 15 ? a.sten_all[2]
                             : tid < 20 ? a.sten_all[3] : a.sten_all[4];
            const uint32_t c6 = (w >> (6 * (tid % 5))) & 63u;
            s_sdx[tid] = (int)(c6 & 7u) - 2;
            s_sdy[tid] = (int)(c6 >> 3) - 2;
        } else if (tid >= 32 && tid < 32 + kMaxOffsets) {
            const int t = tid - 32;  // at most 12 forward offsets: entries 15 and up stay 0
            const uint32_t w = t < 5 ? a.sten_fwd[0] : t < 10 ? a.sten_fwd[1] : t < 15 ? a.sten_fwd[2] : 0x12u;
            const uint32_t c6 = (w >> (6 * (t % 5))) & 63u;
            s_fdx[t] = (int)(c6 & 7u) - 2;
            s_fdy[t] = (int)(c6 >> 3) - 2;
        } else if (tid == 64) {
            s_nsten = (int)(a.sten_meta & 0xffu);
            s_nadj = (int)((a.sten_meta >> 8) & 0xffu);
            s_nfwd = (int)((a.sten_meta >> 16) & 0xffu);
#pragma unroll
            for (int k = 0; k < 3; ++k) s_dxmax[k] = (int)((a.sten_meta >> (24 + 2 * k)) & 3u);
        }
    } else if (tid < 64) {
        build_stencil(g.reach, g.side, r, lane, s_dxmax, s_sdx, s_sdy, &s_nsten, s_fdx, s_fdy, &s_nadj, &s_nfwd);
    }
    __syncthreads();
    // each point's cell (below 2^16: the table fits LDS) and rank in it,
    // packed as cell << 16 | rank
    uint32_t pv[PTS], pcr[PTS];
#pragma unroll
    for (int k = 0; k < PTS; ++k) {
        if (tid + k * kThreads >= n) break;
        pv[k] = (uint32_t)(pt[k].x - x0) | ((uint32_t)(pt[k].y - y0) << 16);
        int32_t cx, cy;
        const int32_t c = cell_id(pv[k], g, &cx, &cy);
        pcr[k] = ((uint32_t)c << 16) | atomicAdd(&cell[c], 1u);
    }
    __syncthreads();
    {
        // one scan of two counts per cell, packed (each total is below
        // 2^16): its points (low half) and, unless it is a dense cell, its
        // points again (high half), which go to the work list; the list's
        // offset of each cell waits in clist, unused until step 5
        const int32_t chunk = (g.ncell + kThreads - 1) / kThreads;
        const int32_t c0 = min(tid * chunk, g.ncell);
        const int32_t c1 = min(c0 + chunk, g.ncell);
        auto both = [&](int v) { return v | (g.dense_ok && v >= a.min_pts ? 0 : v << 16); };
        int sum = 0;
        for (int32_t c = c0; c < c1; ++c) sum += both((int)cell[c]);
        int run = block_exclusive_scan(sum, s_wave);
        for (int32_t c = c0; c < c1; ++c) {
            const int v = (int)cell[c];
            cell[c] = (uint32_t)(run & 0xffff) | 0xffff0000u;
            clist[c] = (uint16_t)(run >> 16);
            run += both(v);
        }
        if (tid == kThreads - 1) {
            cell[g.ncell] = (uint32_t)(run & 0xffff) | 0xffff0000u;
            s_nlist = run >> 16;
        }
    }
    __syncthreads();
    // scatter into sorted order; 4a. on the way, a cell holding >= min_pts
    // points is all core, and the other points go to the work list, in
    // sorted order too (so that the lanes of a wave count neighbours of
    // nearby points, with similar scans)
#pragma unroll
    for (int k = 0; k < PTS; ++k) {
        const int32_t i = tid + k * kThreads;
        if (i >= n) break;
        const int32_t c = (int32_t)(pcr[k] >> 16), rank = (int32_t)(pcr[k] & 0xffffu);
        const int32_t c0 = cstart(c);
        const int32_t pos = c0 + rank;
        pxy[pos] = pv[k];
        sid[pos] = (uint16_t)i;
        const bool dense = g.dense_ok && cstart(c + 1) - c0 >= a.min_pts;
        score[pos] = dense ? kCore : 0;
        if (!dense) list[clist[c] + rank] = (uint16_t)pos;
        // a dense cell's node (smallest core index): the start half of the
        // word is the same on both sides, so the minimum acts on the node
        else atomicMin(&cell[c], (uint32_t)c0 | ((uint32_t)i << 16));
    }
    __syncthreads();
    // 4b. count the listed points' neighbours, nearest rows first, stopping
    //     at min_pts; the bounds of all 2 reach + 1 <= 5 row spans are
    //     loaded before the first scan
    {
        const int32_t nl = s_nlist;
        const int dxm0 = g.dxmax[0], dxm1 = g.reach >= 1 ? g.dxmax[1] : 0, dxm2 = g.reach >= 2 ? g.dxmax[2] : 0;
        for (int32_t j = tid; j < nl; j += kThreads) {
            const int32_t p = list[j];
            const uint32_t v = pxy[p];
            int32_t cx, cy;
            cell_id(v, g, &cx, &cy);
            int32_t q0[5], q1[5];
#pragma unroll
            for (int k = 0; k < 5; ++k) {
                const int dy = (k & 1) ? -((k + 1) >> 1) : (k >> 1);  // 0, -1, 1, -2, 2
                const int ady = dy < 0 ? -dy : dy;
                const int dxm = ady == 0 ? dxm0 : ady == 1 ? dxm1 : dxm2;
                const int32_t ry = cy + dy;
                const bool ok = (k <= 2 * g.reach) & (ry >= 0) & (ry < g.ncy);
                const int32_t row = min(max(ry, 0), g.ncy - 1) * g.ncx;
                q0[k] = cstart(row + max(cx - dxm, 0));
                const int32_t e = cstart(row + min(cx + dxm, g.ncx - 1) + 1);
                q1[k] = ok ? e : q0[k];
            }
            int32_t cnt = 0;
#pragma unroll
            for (int k = 0; k < 5; ++k)
                if (cnt < a.min_pts) cnt += count_span(pxy, q0[k], q1[k], v, r, a.min_pts - cnt);
            if (cnt >= a.min_pts) score[p] = kCore;
            else if (cnt == 1) score[p] = kIsolated;  // no neighbour but itself: noise, no border search
        }
    }
    __syncthreads();

    // 5. forest roots, and the smallest core index of each cell whose cores
    //    came from the counts (dense cells had theirs set in the scatter)
    for (int32_t p = tid; p < n; p += kThreads) parent[p] = p;
    for (int32_t j = tid; j < s_nlist; j += kThreads) {
        const int32_t p = list[j];
        if (score[p] == kCore) {
            int32_t cx, cy;
            const int32_t c = cell_id(pxy[p], g, &cx, &cy);
            atomicMin(&cell[c], (cell[c] & 0xffffu) | ((uint32_t)sid[p] << 16));
        }
    }
    if (tid == 0) s_nlist = 0;
    __syncthreads();
    for (int32_t c0 = tid - lane; c0 < g.ncell; c0 += kThreads) {
        const int32_t c = c0 + lane;
        wave_append(c < g.ncell && cnode(c) != kNone, (uint16_t)c, clist, &s_ncells);
    }
    __syncthreads();

    // 6. union-find over core points (the smaller index always becomes the root)
    if (g.dense_ok) {
        // All cores of a cell are neighbours, so a cell's cores form one node
        // (its smallest core index), and the graph is one of core cells.
        // First its edges to adjacent cells, then connected components in
        // synchronous rounds (hook every edge's two roots under the smaller,
        // then every node jumps to its root) until a round hooks nothing;
        // then the same for the farther cells, whose pairs mostly have equal
        // roots by then and are skipped.  A lane takes one core cell in the
        // edge passes (wave-uniform loops).  The work list is free here: it
        // holds each core cell's edge bits, then the queue of open pairs.
        const int32_t ncl = s_ncells;
        const float inv_ncx = 1.0f / (float)g.ncx;
        const int nadj = s_nadj, nfwd = s_nfwd;
        // Edge bits (ncl entries; 4-byte aligned on the register stage, which
        // sets bits with 32-bit atomics), then the 4-byte aligned queue in
        // what is left of the list's cap entries (ncl <= cap: a core cell
        // holds a core point).
        const int shift0 = (int)((reinterpret_cast<uintptr_t>(list) >> 1) & 1u);
        const bool regs = a.union_regs && ncl <= kRegCells * kThreads && shift0 + ncl + 1 <= cap;
        uint16_t *emask = list + (regs ? shift0 : 0);
        uint16_t *qbase = emask + ncl;
        if (reinterpret_cast<uintptr_t>(qbase) & 2u) ++qbase;
        uint32_t *queue = reinterpret_cast<uint32_t *>(qbase);
        const int qcap = max((int)((list + cap - qbase) / 2), 0);
        int round = 0;
        if (tid == 0) s_hook[0] = 0;
        if (regs) {
            const UnionCtx u{cell, parent, pxy, score, clist, emask, queue, qcap, &s_nq, s_hook,
                             s_fdx, s_fdy, g, r, ncl, inv_ncx};
            union_regs(u, nadj, nfwd, round);
        } else {
            // more core cells than registers hold: the same stages with the
            // edge bits re-read from LDS in every round, and queued pairs
            // kept as (cell A | cell B << 16) and hooked from the queue
            auto core_cell = [&](int32_t j, bool have) {
                CoreCell A{};
                if (have) {
                    A.ca = clist[j];
                    A.ay = div_small(A.ca, g.ncx, inv_ncx);
                    A.ax = A.ca - A.ay * g.ncx;
                    const uint32_t wa = cell[A.ca];
                    A.a0 = (int32_t)(wa & 0xffffu);
                    A.a1 = (int32_t)(cell[A.ca + 1] & 0xffffu);
                    A.node = (int32_t)(wa >> 16);
                    A.head = cell_head(pxy, score, A.a0, A.a1);
                }
                return A;
            };
            auto components = [&](int o0, int nq) {
                const int last = round + ncl + 1;  // as in the register stage
                for (;; ++round) {
                    if (tid == 0) s_hook[(round + 1) % 3] = 0;
                    bool any = false;
                    for (int32_t j = tid; j < ncl; j += kThreads) {
                        const uint32_t m = emask[j];
                        if (!m) continue;
                        const int32_t ca = clist[j];
                        const int32_t ay = div_small(ca, g.ncx, inv_ncx), ax = ca - ay * g.ncx;
                        int32_t nb[8];
#pragma unroll
                        for (int k = 0; k < 8; ++k)
                            nb[k] = ((m >> k) & 1u)
                                        ? (int32_t)cnode((ay + s_fdy[o0 + k]) * g.ncx + ax + s_fdx[o0 + k])
                                        : 0;
                        any |= hook_node<8>(parent, (int32_t)cnode(ca), nb, m);
                    }
                    for (int t = tid; t < nq; t += kThreads) {
                        const uint32_t e = queue[t];
                        if (e == kDeadPair) continue;
                        const int32_t nb[1] = {(int32_t)cnode(e >> 16)};
                        any |= hook_node<1>(parent, (int32_t)cnode(e & 0xffffu), nb, 1u);
                    }
                    if (any) s_hook[round % 3] = 1;
                    __syncthreads();
                    if (!s_hook[round % 3] || round >= last) break;  // every edge joins equal roots
                    for (int32_t j = tid; j < ncl; j += kThreads) jump_node(parent, (int32_t)cnode(clist[j]));
                    __syncthreads();
                }
                ++round;
            };
            if (tid == 0) s_nq = 0;
            __syncthreads();
            for (int32_t j0 = tid - lane; j0 < ncl; j0 += kThreads) {
                const bool have = j0 + lane < ncl;
                const uint32_t m = cell_edges<4, false>(have, core_cell(j0 + lane, have), cell, parent, pxy, score,
                                                        g, r, s_fdx, s_fdy, 0, nadj, queue, &s_nq, qcap);
                if (have) emask[j0 + lane] = (uint16_t)m;
            }
            __syncthreads();
            int nq = min(s_nq, qcap);
            resolve_queue(queue, nq, cell, pxy, score, r);
            __syncthreads();
            components(0, nq);
            if (tid == 0) s_nq = 0;
            __syncthreads();
            for (int32_t j0 = tid - lane; j0 < ncl; j0 += kThreads) {
                const bool have = j0 + lane < ncl;
                const uint32_t m = cell_edges<8, true>(have, core_cell(j0 + lane, have), cell, parent, pxy, score,
                                                       g, r, s_fdx, s_fdy, nadj, nfwd, queue, &s_nq, qcap);
                if (have) emask[j0 + lane] = (uint16_t)m;
            }
            __syncthreads();
            nq = min(s_nq, qcap);
            resolve_queue(queue, nq, cell, pxy, score, r);
            __syncthreads();
            components(nadj, nq);
        }
    } else {
        // coarsened grid: point-level unions (each pair once: the later point
        // of a cell, or the point in the earlier cell, does the work)
        for (int32_t p = tid; p < n; p += kThreads) {
            if (score[p] != kCore) continue;
            const uint32_t v = pxy[p];
            const int32_t op = sid[p];
            int32_t cx, cy;
            const int32_t own = cell_id(v, g, &cx, &cy);
            for (int32_t q = cstart(own); q < p; ++q)
                if (score[q] == kCore && sq_dist_pk(v, pxy[q], r.e1) <= r.e2) uf_unite<kGroup>(parent, op, sid[q]);
            for (int dy = 0; dy <= g.reach; ++dy) {
                const int32_t ry = cy + dy;
                if (ry >= g.ncy) break;
                const int dxm = g.dxmax[dy];
                const int32_t rx0 = dy == 0 ? cx + 1 : max(cx - dxm, 0);
                const int32_t rx1 = min(cx + dxm, g.ncx - 1);
                if (rx0 > rx1) continue;
                const int32_t q1 = cstart(ry * g.ncx + rx1 + 1);
                for (int32_t q = cstart(ry * g.ncx + rx0); q < q1; ++q)
                    if (score[q] == kCore && sq_dist_pk(v, pxy[q], r.e1) <= r.e2) uf_unite<kGroup>(parent, op, sid[q]);
            }
        }
        __syncthreads();
    }

    // 7. every core's label is its tree's root (read-only walks; each thread
    //    writes only roots), and roots are counted once
    int roots = 0;
    for (int32_t p = tid; p < n; p += kThreads) {
        if (score[p] != kCore) continue;
        const int32_t o = sid[p];
        int32_t node = o;
        if (g.dense_ok) {
            int32_t cx, cy;
            node = (int32_t)cnode(cell_id(pxy[p], g, &cx, &cy));
        }
        const int32_t root = uf_root<kGroup>(parent, node);
        st_rlx<kGroup>(parent + o, root);
        roots += root == o;
    }
    __syncthreads();

    // 8. border points: nearest core, ties by smaller (y, x)
    for (int32_t p0 = tid - lane; p0 < n; p0 += kThreads) {
        const int32_t p = p0 + lane;
        wave_append(p < n && score[p] == 0, (uint16_t)p, list, &s_nlist);
    }
    __syncthreads();
    {
        // kBorderLanes consecutive lanes share a point: lane g scans stencil
        // cells g, g + kBorderLanes, ...; the group keeps the smallest key
        // d^2 << 32 | packed (y, x), then the smallest sorted index among
        // equal keys (coincident cores, one cluster).
        const int32_t nl = s_nlist;
        const int ns = s_nsten;
        const int gl = lane & (kBorderLanes - 1);
        // this lane's stencil cells gl, gl + kBorderLanes, ... are the same
        // for every point: their offsets stay in registers
        constexpr int kSlots = (kMaxStencil + kBorderLanes - 1) / kBorderLanes;
        int32_t sdx[kSlots], sdy[kSlots];
        bool sv[kSlots];
#pragma unroll
        for (int k = 0; k < kSlots; ++k) {
            const int st = gl + k * kBorderLanes;
            sv[k] = st < ns;
            sdx[k] = sv[k] ? s_sdx[st] : 0;
            sdy[k] = sv[k] ? s_sdy[st] : 0;
        }
        for (int32_t j = tid / kBorderLanes; j < nl; j += kThreads / kBorderLanes) {
            const int32_t p = list[j];
            const uint32_t v = pxy[p];
            const int32_t vx = pk_x(v), vy = pk_y(v);
            int32_t cx, cy;
            cell_id(v, g, &cx, &cy);
            uint64_t bestk = ~0ull;
            int32_t best = -1;
            // every cell word of the lane's cells first (one round of LDS loads)
            uint32_t cw[kSlots], ce[kSlots];
            bool ok[kSlots];
#pragma unroll
            for (int k = 0; k < kSlots; ++k) {
                const int32_t rx = cx + sdx[k], ry = cy + sdy[k];
                ok[k] = sv[k] & (rx >= 0) & (rx < g.ncx) & (ry >= 0) & (ry < g.ncy);
                const int32_t c = ok[k] ? ry * g.ncx + rx : 0;
                cw[k] = cell[c];
                ce[k] = cell[c + 1];
            }
#pragma unroll
            for (int k = 0; k < kSlots; ++k) {
                if (!ok[k] || (cw[k] >> 16) == kNone) continue;  // no core in this cell
                const int32_t rx = cx + sdx[k], ry = cy + sdy[k];
                const int32_t x0c = rx * g.side, y0c = ry * g.side;
                const int32_t ddx = min(max(max(x0c - vx, vx - (x0c + g.side - 1)), 0), r.e1);
                const int32_t ddy = min(max(max(y0c - vy, vy - (y0c + g.side - 1)), 0), r.e1);
                if (__mul24(ddx, ddx) + __mul24(ddy, ddy) > r.e2) continue;  // cell out of reach
                const int32_t q1 = (int32_t)(ce[k] & 0xffffu);
                int32_t q = (int32_t)(cw[k] & 0xffffu);
                for (; q + 1 < q1; q += 2) {  // two candidates per step, in order
                    const uint32_t w0 = pxy[q], w1 = pxy[q + 1];
                    const bool c0 = score[q] == kCore, c1 = score[q + 1] == kCore;
                    const int32_t d0 = sq_dist_pk(v, w0, r.e1), d1 = sq_dist_pk(v, w1, r.e1);
                    const uint64_t k0 = ((uint64_t)(uint32_t)d0 << 32) | w0;
                    const uint64_t k1 = ((uint64_t)(uint32_t)d1 << 32) | w1;
                    const bool t0 = (d0 <= r.e2) & c0 & (k0 < bestk);
                    best = t0 ? q : best;
                    bestk = t0 ? k0 : bestk;
                    const bool t1 = (d1 <= r.e2) & c1 & (k1 < bestk);
                    best = t1 ? q + 1 : best;
                    bestk = t1 ? k1 : bestk;
                }
                if (q < q1) {
                    const uint32_t w = pxy[q];
                    const int32_t d2 = sq_dist_pk(v, w, r.e1);
                    const uint64_t key = ((uint64_t)(uint32_t)d2 << 32) | w;
                    const bool take = (d2 <= r.e2) & (score[q] == kCore) & (key < bestk);
                    best = take ? q : best;
                    bestk = take ? key : bestk;
                }
            }
#pragma unroll
            for (int o = 1; o < kBorderLanes; o <<= 1) {
                const uint64_t ok = __shfl_xor(bestk, o, 64);
                const int32_t ob = __shfl_xor(best, o, 64);
                const bool take = (ok < bestk) | ((ok == bestk) & (ob < best));
                best = take ? ob : best;
                bestk = take ? ok : bestk;
            }
            if (gl == 0) {
                const int32_t o = sid[p];
                if (best >= 0) {
                    parent[o] = parent[sid[best]];
                    score[p] = kBorder;  // 0 -> kBorder: concurrent core tests see no change
                } else {
                    parent[o] = -1;
                }
            }
        }
    }
    roots = wave_sum(roots);
    if (lane == 0) atomicAdd(&s_red, roots);
    __syncthreads();

    // 9. kinds into original order (in the list's space, free now), then the
    //    outputs in original order (coalesced)
    uint8_t *kindo = reinterpret_cast<uint8_t *>(list);
    for (int32_t p = tid; p < n; p += kThreads) kindo[sid[p]] = score[p];
    __syncthreads();
    for (int32_t i = tid; i < n; i += kThreads) {
        const uint8_t k = kindo[i];
        a.labels[b + i] = k == kIsolated ? -1 : parent[i];
        a.kind[b + i] = k == kIsolated ? 0 : k;
    }
    if (tid == 0 && a.n_clusters) a.n_clusters[f] = s_red;
}

__global__ __launch_bounds__(kThreads) void cluster_resident_kernel(ClusterArgs a) {
    cluster_resident<kPtsPerThread>(a);
}

// Two workgroups per compute unit: 8 waves per SIMD (at most 64 VGPRs) and
// half the LDS each.
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(8))) void cluster_compact_kernel(
    ClusterArgs a) {
    cluster_resident<kPtsCompact>(a);
}

}  // namespace

size_t cluster_lds_bytes(int32_t cap_points, int32_t cap_cells) {
    // per point: packed coords 4, parent 4, sid 2, list 2, kind 1;
    // per cell: start|node 4, cell list 2
    size_t bytes = (size_t)cap_points * 13 + (size_t)cap_cells * 6 + 4;
    const size_t inplace = (size_t)kTile * (8 + 1);
    if (bytes < inplace) bytes = inplace;
    return (bytes + 15) & ~(size_t)15;
}

int32_t cluster_max_cap_points(size_t lds_limit) {
    // reserve room for the static shared variables and a 4096-entry cell table
    const size_t reserve = 1024 + 4096 * 6 + 4;
    if (lds_limit <= reserve) return 0;
    size_t cap = (lds_limit - reserve) / 13;
    if (cap > (size_t)kThreads * kPtsPerThread) cap = (size_t)kThreads * kPtsPerThread;  // register sort
    return (int32_t)cap;
}

size_t cluster_compact_static_lds() {
    static const size_t bytes = [] {
        hipFuncAttributes attr{};
        if (hipFuncGetAttributes(&attr, reinterpret_cast<const void *>(&cluster_compact_kernel)) != hipSuccess)
            return (size_t)4096;  // a safe over-estimate of the kernel's static shared variables
        return (size_t)attr.sharedSizeBytes;
    }();
    return bytes;
}

hipError_t launch_cluster_resident(const ClusterArgs &a, size_t lds_bytes, bool compact, hipStream_t stream) {
    if (compact)
        hipLaunchKernelGGL(cluster_compact_kernel, dim3(a.n_frames), dim3(kThreads), lds_bytes, stream, a);
    else
        hipLaunchKernelGGL(cluster_resident_kernel, dim3(a.n_frames), dim3(kThreads), lds_bytes, stream, a);
    return hipGetLastError();
}

}  // namespace flock

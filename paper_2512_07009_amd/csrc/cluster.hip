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
// Frames with more points than the on-chip capacity take an in-place path
// that keeps the union-find forest in the caller's labels array and runs
// brute-force pair tests through LDS tiles (correct for any size, slow).
//
// All results are independent of the order of points within a cell, so the
// nondeterministic order of the LDS atomics in the counting sort cannot
// change any output.

#include <climits>

#include "internal.h"

namespace flock {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kTile = 1024;  // points per LDS tile on the in-place path

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------

template <int Scope>
__device__ __forceinline__ int32_t ld_rlx(const int32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, Scope);
}
template <int Scope>
__device__ __forceinline__ void st_rlx(int32_t *p, int32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, Scope);
}

// Root of x with path halving.  Invariant kept by every writer:
// parent[x] <= x, and parent[x] is an ancestor of x.
template <int Scope>
__device__ int32_t uf_find(int32_t *parent, int32_t x) {
    for (;;) {
        int32_t p = ld_rlx<Scope>(parent + x);
        if (p == x) return x;
        int32_t gp = ld_rlx<Scope>(parent + p);
        if (gp == p) return p;
        st_rlx<Scope>(parent + x, gp);
        x = gp;
    }
}

// Root of x without writes (safe while other threads set parent[i] = root).
template <int Scope>
__device__ int32_t uf_root(const int32_t *parent, int32_t x) {
    for (;;) {
        int32_t p = ld_rlx<Scope>(parent + x);
        if (p == x) return x;
        x = p;
    }
}

// Merge the trees of a and b, hooking the larger root under the smaller.
template <int Scope>
__device__ void uf_unite(int32_t *parent, int32_t a, int32_t b) {
    for (;;) {
        a = uf_find<Scope>(parent, a);
        b = uf_find<Scope>(parent, b);
        if (a == b) return;
        if (a < b) {
            int32_t t = a;
            a = b;
            b = t;
        }
        int32_t expected = a;
        if (__hip_atomic_compare_exchange_strong(parent + a, &expected, b, __ATOMIC_RELAXED,
                                                 __ATOMIC_RELAXED, Scope))
            return;
    }
}

// Exact neighbour test.  Per axis the distance is clamped to E + 1, which
// cannot change the outcome and keeps dx^2 + dy^2 below 2^31 (E <= 32766).
struct Radius {
    int32_t e;       // E
    int32_t e1;      // E + 1
    int32_t e2;      // E^2
};

__device__ __forceinline__ int32_t clamp_abs(int32_t d, int32_t e1) {
    d = d < 0 ? -d : d;
    return d < e1 ? d : e1;
}

__device__ __forceinline__ int32_t sq_dist_clamped(int2 a, int2 b, const Radius &r) {
    int32_t dx = clamp_abs(a.x - b.x, r.e1);
    int32_t dy = clamp_abs(a.y - b.y, r.e1);
    return __mul24(dx, dx) + __mul24(dy, dy);
}

__device__ __forceinline__ bool within(int2 a, int2 b, const Radius &r) {
    return sq_dist_clamped(a, b, r) <= r.e2;
}

// true if core q beats the current best core for a border point:
// key (d^2, y, x) ascending.
__device__ __forceinline__ bool better_core(int32_t d2, int2 q, int32_t best_d2, int2 best) {
    if (d2 != best_d2) return d2 < best_d2;
    if (q.y != best.y) return q.y < best.y;
    return q.x < best.x;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
    return v;
}

// Exclusive scan of one int per thread across the workgroup.
__device__ int block_exclusive_scan(int v, int *wave_tot) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    int inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int t = __shfl_up(inc, o, 64);
        if (lane >= o) inc += t;
    }
    if (lane == 63) wave_tot[wave] = inc;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += wave_tot[w];
    __syncthreads();
    return base + inc - v;
}

// Cell geometry of one frame.
struct Grid {
    int32_t x0, y0;      // bbox origin (quanta)
    int32_t side;        // cell side (quanta)
    int32_t ncx, ncy;    // cells per axis
    int32_t ncell;
    int32_t reach;       // R: neighbour cells lie within +-R cells
    int32_t dxmax[8];    // per |dy| <= R: widest |dx| whose cells can hold neighbours
    bool dense_ok;       // side is the eps-diagonal side: same cell => neighbours
};

__device__ __forceinline__ int64_t cell_gap(int32_t d, int32_t side) {
    d = d < 0 ? -d : d;
    return d == 0 ? 0 : (int64_t)(d - 1) * side + 1;
}

__device__ __forceinline__ int2 cell_of(int2 p, const Grid &g) {
    uint32_t ux = (uint32_t)(p.x - g.x0);
    uint32_t uy = (uint32_t)(p.y - g.y0);
    int32_t cx = (int32_t)(ux / (uint32_t)g.side);
    int32_t cy = (int32_t)(uy / (uint32_t)g.side);
    // bbox-derived, so in range; clamp anyway so no index can leave the table
    cx = min(max(cx, 0), g.ncx - 1);
    cy = min(max(cy, 0), g.ncy - 1);
    return make_int2(cx, cy);
}

// ---------------------------------------------------------------------------
// In-place path for frames above the on-chip capacity
// ---------------------------------------------------------------------------

constexpr int kAgent = __HIP_MEMORY_SCOPE_AGENT;
constexpr int kGroup = __HIP_MEMORY_SCOPE_WORKGROUP;

__device__ void cluster_frame_inplace(const ClusterArgs &a, int f, int32_t b, int32_t n,
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
        int32_t best = -1, best_d2 = 0;
        int2 bestp = make_int2(0, 0);
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
                    if (best < 0 || better_core(d2, q, best_d2, bestp)) {
                        best = t0 + j;
                        best_d2 = d2;
                        bestp = q;
                    }
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

__global__ __launch_bounds__(kThreads) void cluster_resident_kernel(ClusterArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ int s_bbox[4];
    __shared__ int s_wave[kWaves];
    __shared__ int s_red;

    const int f = blockIdx.x;
    const int tid = threadIdx.x;
    const int32_t b = a.offsets[f];
    const int32_t e = a.offsets[f + 1];
    if (b < 0 || e < b || e > a.total) {
        if (tid == 0 && a.n_clusters) a.n_clusters[f] = -1;
        return;
    }
    const int32_t n = e - b;
    if (tid == 0) {
        s_bbox[0] = INT_MAX;
        s_bbox[1] = INT_MAX;
        s_bbox[2] = INT_MIN;
        s_bbox[3] = INT_MIN;
        s_red = 0;
    }
    if (n == 0) {
        if (tid == 0 && a.n_clusters) a.n_clusters[f] = 0;
        return;
    }
    if (n > a.cap_points) {
        __syncthreads();
        cluster_frame_inplace(a, f, b, n, smem, &s_red);
        return;
    }

    const int32_t cap = a.cap_points;
    int2 *sxy = reinterpret_cast<int2 *>(smem);            // [cap] sorted coords
    int32_t *parent = reinterpret_cast<int32_t *>(sxy + cap);  // [cap] by original index
    int32_t *cstart = parent + cap;                          // [cap_cells + 1]
    uint16_t *sid = reinterpret_cast<uint16_t *>(cstart + a.cap_cells + 1);  // [cap]
    uint8_t *score = reinterpret_cast<uint8_t *>(sid + cap);  // [cap] core flag, sorted
    uint8_t *kindo = score + cap;                             // [cap] kind, original order

    const int2 *P = reinterpret_cast<const int2 *>(a.xy) + b;
    const Radius r{a.eps_q, a.eps_q + 1, a.eps_q * a.eps_q};

    // 1. bounding box
    {
        int xmn = INT_MAX, ymn = INT_MAX, xmx = INT_MIN, ymx = INT_MIN;
        for (int32_t i = tid; i < n; i += kThreads) {
            int2 p = P[i];
            xmn = min(xmn, p.x);
            ymn = min(ymn, p.y);
            xmx = max(xmx, p.x);
            ymx = max(ymx, p.y);
        }
        xmn = wave_min(xmn);
        ymn = wave_min(ymn);
        xmx = wave_max(xmx);
        ymx = wave_max(ymx);
        __syncthreads();  // s_bbox initialised
        if ((tid & 63) == 0) {
            atomicMin(&s_bbox[0], xmn);
            atomicMin(&s_bbox[1], ymn);
            atomicMax(&s_bbox[2], xmx);
            atomicMax(&s_bbox[3], ymx);
        }
        __syncthreads();
    }

    // 2. cell grid (every thread derives the same values)
    Grid g;
    {
        g.x0 = s_bbox[0];
        g.y0 = s_bbox[1];
        const uint32_t wx = (uint32_t)(s_bbox[2] - s_bbox[0]);
        const uint32_t wy = (uint32_t)(s_bbox[3] - s_bbox[1]);
        uint32_t side = (uint32_t)a.cell_side;
        uint64_t ncx = wx / side + 1, ncy = wy / side + 1;
        while (ncx * ncy > (uint64_t)a.cap_cells) {
            side *= 2u;
            ncx = wx / side + 1;
            ncy = wy / side + 1;
        }
        g.side = (int32_t)side;
        g.ncx = (int32_t)ncx;
        g.ncy = (int32_t)ncy;
        g.ncell = g.ncx * g.ncy;
        g.dense_ok = side == (uint32_t)a.cell_side;
        g.reach = r.e == 0 ? 0 : 1 + (r.e - 1) / g.side;
        if (g.reach > 7) g.reach = 7;  // side >= s >= E/2 when E >= 2, so reach <= 2
        for (int dy = 0; dy <= g.reach; ++dy) {
            const int64_t gy = cell_gap(dy, g.side);
            int dx = g.reach;
            while (dx > 0) {
                const int64_t gx = cell_gap(dx, g.side);
                if (gx * gx + gy * gy <= (int64_t)r.e2) break;
                --dx;
            }
            g.dxmax[dy] = dx;  // dx = 0 always qualifies for the rows kept below
        }
    }

    // 3. counting sort by cell
    for (int32_t c = tid; c <= g.ncell; c += kThreads) cstart[c] = 0;
    __syncthreads();
    for (int32_t i = tid; i < n; i += kThreads) {
        const int2 c = cell_of(P[i], g);
        parent[i] = atomicAdd(&cstart[c.y * g.ncx + c.x], 1);  // rank within cell
    }
    __syncthreads();
    {
        const int32_t chunk = (g.ncell + kThreads - 1) / kThreads;
        const int32_t c0 = min(tid * chunk, g.ncell);
        const int32_t c1 = min(c0 + chunk, g.ncell);
        int sum = 0;
        for (int32_t c = c0; c < c1; ++c) sum += cstart[c];
        int run = block_exclusive_scan(sum, s_wave);
        for (int32_t c = c0; c < c1; ++c) {
            const int v = cstart[c];
            cstart[c] = run;
            run += v;
        }
        if (tid == kThreads - 1) cstart[g.ncell] = run;
    }
    __syncthreads();
    for (int32_t i = tid; i < n; i += kThreads) {
        const int2 p = P[i];
        const int2 c = cell_of(p, g);
        const int32_t pos = cstart[c.y * g.ncx + c.x] + parent[i];
        sxy[pos] = p;
        sid[pos] = (uint16_t)i;
    }
    __syncthreads();

    // 4. neighbour counts -> core flags
    for (int32_t p = tid; p < n; p += kThreads) {
        const int2 pp = sxy[p];
        const int2 c = cell_of(pp, g);
        const int32_t own = c.y * g.ncx + c.x;
        int32_t cnt = 0;
        if (g.dense_ok) cnt = cstart[own + 1] - cstart[own];
        if (cnt < a.min_pts) {
            cnt = 0;
            for (int dy = -g.reach; dy <= g.reach && cnt < a.min_pts; ++dy) {
                const int32_t cy = c.y + dy;
                if (cy < 0 || cy >= g.ncy) continue;
                const int dxm = g.dxmax[dy < 0 ? -dy : dy];
                const int32_t cx0 = max(c.x - dxm, 0), cx1 = min(c.x + dxm, g.ncx - 1);
                const int32_t q0 = cstart[cy * g.ncx + cx0], q1 = cstart[cy * g.ncx + cx1 + 1];
                for (int32_t q = q0; q < q1; ++q) {
                    cnt += within(pp, sxy[q], r) ? 1 : 0;
                    if (cnt >= a.min_pts) break;
                }
            }
        }
        const bool core = cnt >= a.min_pts;
        score[p] = core ? 1 : 0;
        kindo[sid[p]] = core ? 2 : 0;
    }
    for (int32_t i = tid; i < n; i += kThreads) parent[i] = i;
    __syncthreads();

    // 5. union-find over core points
    for (int32_t p = tid; p < n; p += kThreads) {
        if (!score[p]) continue;
        const int2 pp = sxy[p];
        const int32_t op = sid[p];
        const int2 c = cell_of(pp, g);
        const int32_t own = c.y * g.ncx + c.x;
        // same cell
        if (g.dense_ok) {
            int32_t q = cstart[own];
            while (!score[q]) ++q;  // p itself is core, so this stops by p
            if (q != p) uf_unite<kGroup>(parent, op, sid[q]);
        } else {
            for (int32_t q = cstart[own]; q < p; ++q)
                if (score[q] && within(pp, sxy[q], r)) uf_unite<kGroup>(parent, op, sid[q]);
        }
        // cells after this one in row-major order
        for (int dy = 0; dy <= g.reach; ++dy) {
            const int32_t cy = c.y + dy;
            if (cy >= g.ncy) break;
            const int dxm = g.dxmax[dy];
            const int32_t cx0 = dy == 0 ? c.x + 1 : max(c.x - dxm, 0);
            const int32_t cx1 = min(c.x + dxm, g.ncx - 1);
            for (int32_t cx = cx0; cx <= cx1; ++cx) {
                const int32_t cc = cy * g.ncx + cx;
                const int32_t q0 = cstart[cc], q1 = cstart[cc + 1];
                for (int32_t q = q0; q < q1; ++q) {
                    if (score[q] && within(pp, sxy[q], r)) {
                        uf_unite<kGroup>(parent, op, sid[q]);
                        if (g.dense_ok) break;  // the cell's cores are already one tree
                    }
                }
            }
        }
    }
    __syncthreads();

    // 6. flatten the core forest; count roots
    int roots = 0;
    for (int32_t i = tid; i < n; i += kThreads) {
        if (kindo[i] != 2) continue;
        const int32_t root = uf_root<kGroup>(parent, i);
        st_rlx<kGroup>(parent + i, root);
        roots += root == i;
    }
    __syncthreads();

    // 7. border points: nearest core, ties by (y, x)
    for (int32_t p = tid; p < n; p += kThreads) {
        if (score[p]) continue;
        const int2 pp = sxy[p];
        const int2 c = cell_of(pp, g);
        int32_t best = -1, best_d2 = 0;
        int2 bestp = make_int2(0, 0);
        for (int dy = -g.reach; dy <= g.reach; ++dy) {
            const int32_t cy = c.y + dy;
            if (cy < 0 || cy >= g.ncy) continue;
            const int dxm = g.dxmax[dy < 0 ? -dy : dy];
            const int32_t cx0 = max(c.x - dxm, 0), cx1 = min(c.x + dxm, g.ncx - 1);
            const int32_t q0 = cstart[cy * g.ncx + cx0], q1 = cstart[cy * g.ncx + cx1 + 1];
            for (int32_t q = q0; q < q1; ++q) {
                if (!score[q]) continue;
                const int2 qq = sxy[q];
                const int32_t d2 = sq_dist_clamped(pp, qq, r);
                if (d2 > r.e2) continue;
                if (best < 0 || better_core(d2, qq, best_d2, bestp)) {
                    best = q;
                    best_d2 = d2;
                    bestp = qq;
                }
            }
        }
        const int32_t o = sid[p];
        if (best >= 0) {
            parent[o] = parent[sid[best]];
            kindo[o] = 1;
        } else {
            parent[o] = -1;
        }
    }
    roots = wave_sum(roots);
    if ((tid & 63) == 0) atomicAdd(&s_red, roots);
    __syncthreads();

    // 8. outputs in original order (coalesced)
    for (int32_t i = tid; i < n; i += kThreads) {
        a.labels[b + i] = parent[i];
        a.kind[b + i] = kindo[i];
    }
    if (tid == 0 && a.n_clusters) a.n_clusters[f] = s_red;
}

}  // namespace

size_t cluster_lds_bytes(int32_t cap_points, int32_t cap_cells) {
    size_t bytes = (size_t)cap_points * (8 + 4 + 2 + 1 + 1) + ((size_t)cap_cells + 1) * 4;
    const size_t inplace = (size_t)kTile * (8 + 1);
    if (bytes < inplace) bytes = inplace;
    return (bytes + 15) & ~(size_t)15;
}

int32_t cluster_max_cap_points(size_t lds_limit) {
    // reserve room for the static shared variables and a 4096-entry cell table
    const size_t reserve = 1024 + 4097 * 4;
    if (lds_limit <= reserve) return 0;
    size_t cap = (lds_limit - reserve) / 16;
    if (cap > 65535) cap = 65535;  // original indices are kept as uint16
    return (int32_t)cap;
}

hipError_t launch_cluster_resident(const ClusterArgs &a, size_t lds_bytes, hipStream_t stream) {
    hipLaunchKernelGGL(cluster_resident_kernel, dim3(a.n_frames), dim3(kThreads), lds_bytes, stream,
                       a);
    return hipGetLastError();
}

}  // namespace flock

// cluster_common.h - device helpers shared by the clustering kernels
// (on-chip and multi-workgroup paths): exact integer neighbour tests, the
// min-index union-find, wave reductions and the cell-gap geometry.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace flock {
namespace cl {

constexpr int kAgent = __HIP_MEMORY_SCOPE_AGENT;
constexpr int kGroup = __HIP_MEMORY_SCOPE_WORKGROUP;

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
__device__ __forceinline__ int32_t uf_find(int32_t *parent, int32_t x) {
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
__device__ __forceinline__ int32_t uf_root(const int32_t *parent, int32_t x) {
    for (;;) {
        int32_t p = ld_rlx<Scope>(parent + x);
        if (p == x) return x;
        x = p;
    }
}

// Merge the trees of a and b, hooking the larger root under the smaller.
template <int Scope>
__device__ __forceinline__ void uf_unite(int32_t *parent, int32_t a, int32_t b) {
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

// Candidate order for a border point's core: key (d^2, y, x) ascending.
// Evaluated as bitwise logic with no short-circuit so that the caller's
// running-minimum update compiles to selects: the branchy form of this test
// (nested ifs under a divergent loop) has been compiled on gfx950 into code
// that updated the key but kept the old index.  Callers start best_d2 at
// INT32_MAX, above every accepted d^2 (<= eps_q^2 < 2^31).
__device__ __forceinline__ bool core_before(int32_t d2, int32_t qy, int32_t qx, int32_t best_d2,
                                            int32_t by, int32_t bx) {
    const bool yx = (qy < by) | ((qy == by) & (qx < bx));
    return (d2 < best_d2) | ((d2 == best_d2) & yx);
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
__device__ inline int block_exclusive_scan(int v, int *wave_tot) {
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

// Cell coordinate of v on an axis whose grid starts at v0 with cells of
// `side` quanta and `ncoord` cells: floor((v - v0) / side), clamped into
// [0, ncoord - 1].  The difference is taken in unsigned arithmetic, so a
// value below v0 (which a frame's own points never are) lands in the last
// cell instead of a negative index.
__host__ __device__ __forceinline__ int32_t cell_coord_clamped(int32_t v, int32_t v0, int32_t side, int32_t ncoord) {
    const uint32_t q = ((uint32_t)v - (uint32_t)v0) / (uint32_t)side;
    const uint32_t last = (uint32_t)(ncoord - 1);
    return (int32_t)(q < last ? q : last);
}

// Smallest per-axis distance between points of two cells |d| cells apart.
__device__ __forceinline__ int64_t cell_gap(int32_t d, int32_t side) {
    d = d < 0 ? -d : d;
    return d == 0 ? 0 : (int64_t)(d - 1) * side + 1;
}

}  // namespace cl
}  // namespace flock

// roi.hip - region-of-interest filter and per-frame region counts, and
// drinker-line proximity, on gfx950.
//
// What is computed (the wall pipeline counts the birds in a region near the
// wall, Section 2.2; Algorithm 1 filters the birds to the region of
// interest): a bird is kept when its point lies in the closed ROI polygon,
// edges and vertices included, under the even-odd rule; kept birds keep
// their input order.  Integer coordinates in 1/16 px, exact 64-bit products.
//
// Four kernels over fixed blocks of 2048 birds, whatever the frames
// (HBM-bound: 8 bytes read per bird, 12 written per kept bird):
//   1. roi_flag_kernel: the inside test per bird (polygon in LDS), a flag
//      byte per bird and a count per block;
//   2. roi_scan_kernel, one workgroup: each block's first output position;
//   3. roi_write_kernel: each block's kept birds, which the flag kernel
//      staged in input order (ballots and wave totals give each its rank in
//      the block), are copied to the block's base + rank, so kept birds keep
//      their input order;
//   4. frame_counts_kernel, one wave per frame boundary: the output position
//      of the boundary bird (its block's base plus the flags before it in the
//      block) gives out_offsets, and neighbouring boundaries give counts.
// Drinker-line proximity reuses steps 2 and 4 on its own flags (see
// drink_flag_kernel).

#include <climits>

#include "internal.h"

namespace flock {
namespace {

constexpr int kRThreadsR = 256;
constexpr int kRWaves = kRThreadsR / 64;

// Closed polygon test, even-odd rule.  A point outside the polygon's
// bounding box is outside, and edges whose y range excludes the point are
// skipped.  Otherwise an edge on which the point lies decides
// at once (inside), and each edge whose ends lie on different sides of the
// horizontal line through the point (one strictly above it, so that a vertex
// on the line is counted once) toggles the result when it meets the line to
// the right of the point.  Coordinates and vertices are within 2^24 in
// magnitude, so every difference is below 2^25 and the cross product
// ex qy - ey qx below 2^51: exact in fp64 (two exact products, an exact
// difference), one fp64 multiply per product where a 64-bit integer product
// takes several instructions.
__device__ __forceinline__ bool in_box(const RoiArgs &a, int px, int py) {
    return px >= a.bx0 && px <= a.bx1 && py >= a.by0 && py <= a.by1;
}

// The test for a point inside the bounding box.
__device__ __forceinline__ bool in_polygon_boxed(const RoiArgs &a, const int2 *poly, int px, int py) {
    const int n = a.n_vertices;
    bool in = false;
    for (int i = 0; i < n; ++i) {
        const int2 A = poly[i], B = poly[i + 1 == n ? 0 : i + 1];
        // an edge whose y range excludes py neither holds the point nor
        // crosses its line (both ends lie on one side)
        if (py < min(A.y, B.y) || py > max(A.y, B.y)) continue;
        const double ex = (double)(B.x - A.x), ey = (double)(B.y - A.y);
        const double qx = (double)(px - A.x), qy = (double)(py - A.y);
        const double cr = ex * qy - ey * qx;
        if (cr == 0 && px >= min(A.x, B.x) && px <= max(A.x, B.x) && py >= min(A.y, B.y) && py <= max(A.y, B.y))
            return true;
        const bool a_above = A.y > py, b_above = B.y > py;
        if (a_above != b_above) {
            // crossing at x = A.x + qy ex / ey; right of px iff qx ey < qy ex
            // for ey > 0 (reversed for ey < 0); qy ex - qx ey = cr
            const bool right = ey > 0 ? cr > 0 : cr < 0;
            if (right) in = !in;
        }
    }
    return in;
}

__device__ __forceinline__ void load_polygon(const RoiArgs &a, int2 *poly) {
    if ((int)threadIdx.x < a.n_vertices) poly[threadIdx.x] = make_int2(a.vx[threadIdx.x], a.vy[threadIdx.x]);
    __syncthreads();
}

constexpr int kRBlock = kRoiBlock;             // birds per block
constexpr int kRPer = kRBlock / kRThreadsR;    // birds per thread, consecutive chunks of 256

// Flags of one block of birds.  The bounding-box test runs on every bird;
// the birds inside the box (a small share for a region along a wall) are
// queued in LDS and the edge tests run on the queue, so that whole waves
// test in-box birds instead of every wave running the edge loop for the
// few in-box lanes it holds.  The kept birds then go, in input order, to the
// block's staging area (coordinates and input index), for the write kernel
// to copy to their final places without reading every bird again.
__global__ __launch_bounds__(kRThreadsR) void roi_flag_kernel(RoiArgs a, uint8_t *flag, int32_t *bcount,
                                                             int2 *stage_xy, int32_t *stage_idx) {
    __shared__ int2 poly[kRoiMaxVertices];
    __shared__ int2 s_pt[kRBlock];        // in-box birds: coordinates
    __shared__ uint16_t s_at[kRBlock];    // and their index in the block
    __shared__ uint8_t s_f[kRBlock];      // every bird's flag
    __shared__ int s_tot[kRPer][kRWaves];
    __shared__ int s_nq;
    if (threadIdx.x == 0) s_nq = 0;
    load_polygon(a, poly);  // holds a barrier
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const long long i0 = (long long)blockIdx.x * kRBlock;
    const int2 *P = reinterpret_cast<const int2 *>(a.xy);
    // all loads first, so that their latencies overlap
    int2 pts[kRPer];
#pragma unroll
    for (int k = 0; k < kRPer; ++k) {
        const long long i = i0 + k * kRThreadsR + tid;
        pts[k] = i < a.total ? P[i] : make_int2(INT_MIN, INT_MIN);
    }
    // box test; birds outside are out, the others queued
#pragma unroll
    for (int k = 0; k < kRPer; ++k) {
        const bool box = in_box(a, pts[k].x, pts[k].y);  // a padding lane's point is outside every box
        const uint64_t m = __ballot(box);
        int base = 0;
        if (lane == 0 && m) base = atomicAdd(&s_nq, __popcll(m));
        base = __shfl(base, 0, 64);
        if (box) {
            const int q = base + __popcll(m & ((1ull << lane) - 1));
            s_pt[q] = pts[k];
            s_at[q] = (uint16_t)(k * kRThreadsR + tid);
        } else {
            s_f[k * kRThreadsR + tid] = 0;
        }
    }
    __syncthreads();
    const int nq = s_nq;
    for (int q = tid; q < nq; q += kRThreadsR) {
        const int2 pt = s_pt[q];
        s_f[s_at[q]] = in_polygon_boxed(a, poly, pt.x, pt.y);
    }
    __syncthreads();
    // flags out, and the kept birds' ranks in the block (input order)
    bool in[kRPer];
    uint64_t m[kRPer];
#pragma unroll
    for (int k = 0; k < kRPer; ++k) {
        const long long i = i0 + k * kRThreadsR + tid;
        in[k] = s_f[k * kRThreadsR + tid] != 0;
        if (i < a.total) flag[i] = in[k];
        m[k] = __ballot(in[k]);
        if (lane == 0) s_tot[k][wave] = __popcll(m[k]);
    }
    __syncthreads();
    int at = 0;
    const long long sbase = (long long)blockIdx.x * kRBlock;
#pragma unroll
    for (int k = 0; k < kRPer; ++k) {
        int before = 0, chunk = 0;
#pragma unroll
        for (int w = 0; w < kRWaves; ++w) {
            before += w < wave ? s_tot[k][w] : 0;
            chunk += s_tot[k][w];
        }
        if (in[k]) {
            const long long r = sbase + at + before + __popcll(m[k] & ((1ull << lane) - 1ull));
            stage_xy[r] = pts[k];
            stage_idx[r] = (int32_t)(i0 + k * kRThreadsR + tid);
        }
        at += chunk;
    }
    if (tid == 0) bcount[blockIdx.x] = at;
}

// bbase[b] = bcount[0] + ... + bcount[b - 1]; bbase[nb] = all kept birds.
__global__ __launch_bounds__(1024) void roi_scan_kernel(const int32_t *bcount, int32_t *bbase, int nb) {
    __shared__ int s_wave[16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int per = (nb + 1023) / 1024;
    const int b0 = min(tid * per, nb), b1 = min(b0 + per, nb);
    int sum = 0;
    for (int b = b0; b < b1; ++b) sum += bcount[b];
    int inc = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(inc, o, 64);
        if (lane >= o) inc += t;
    }
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    int run = inc - sum;
    for (int w = 0; w < wave; ++w) run += s_wave[w];
    for (int b = b0; b < b1; ++b) {
        bbase[b] = run;
        run += bcount[b];
    }
    if (tid == 1023) bbase[nb] = run;  // the last thread's chunk ends at nb
}

// Each block's kept birds, staged in input order by the flag kernel, go to
// base + rank.
__global__ __launch_bounds__(kRThreadsR) void roi_write_kernel(RoiArgs a, const int32_t *bbase,
                                                              const int2 *stage_xy, const int32_t *stage_idx) {
    const int32_t base = bbase[blockIdx.x], n = bbase[blockIdx.x + 1] - base;
    const long long sbase = (long long)blockIdx.x * kRBlock;
    int2 *O = reinterpret_cast<int2 *>(a.out_xy);
    for (int t = threadIdx.x; t < n; t += kRThreadsR) {
        O[base + t] = stage_xy[sbase + t];
        if (a.out_index) a.out_index[base + t] = stage_idx[sbase + t];
    }
}

// Per-frame counts of flagged birds, for the ROI filter (which also needs
// the CSR offsets of its output) and the drinker flags.
struct FrameCounts {
    const uint8_t *flag;      // [total] 0 or 1, padded to 256 bytes
    const int32_t *bbase;     // [nb + 1] flagged birds before each 2048-bird block
    const int32_t *offsets;   // [n_frames + 1]
    int32_t n_frames, total;
    int32_t *counts;          // [n_frames]
    int32_t *out_offsets;     // [n_frames + 1] or nullptr
};

// Flagged birds before input bird i0 (0 <= i0 <= total): its block's base
// plus the flags before it in the block (wave-uniform call).
__device__ __forceinline__ int32_t flagged_before(const FrameCounts &fc, int32_t i0) {
    const int lane = threadIdx.x & 63;
    const int32_t b = i0 / kRBlock;
    const int32_t s0 = b * kRBlock;
    // 16 flags per lane and load (a block is 2048 = 2 x 64 x 16 flags; the
    // flag array is 16-byte aligned), bytes at or past i0 masked; the last
    // partial word of the array is read byte by byte, never past total
    int c = 0;
#pragma unroll
    for (int j = 0; j < kRBlock / (64 * 16); ++j) {
        const int32_t base = s0 + 16 * (lane + 64 * j);
        if (base >= i0) continue;
        if (base + 16 > fc.total) {
            for (int32_t i = base; i < i0; ++i) c += fc.flag[i];
            continue;
        }
        const uint4 w = *reinterpret_cast<const uint4 *>(fc.flag + base);
        const int valid = min(16, i0 - base);
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int nb = min(max(valid - 4 * q, 0), 4);  // valid bytes in this word
            const uint32_t keep = nb >= 4 ? 0xffffffffu : ((1u << (8 * nb)) - 1u);
            c += (int)(((ws[q] & keep) * 0x01010101u) >> 24);  // bytes are 0 or 1
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    return fc.bbase[b] + c;  // bbase has nb + 1 entries, and i0 = total gives b <= nb
}

// One wave per frame boundary f = 0 .. n_frames.
__global__ __launch_bounds__(256) void frame_counts_kernel(FrameCounts fc) {
    const int f = (int)(((long long)blockIdx.x * 256 + threadIdx.x) >> 6);
    if (f > fc.n_frames) return;  // wave-uniform
    // frame boundaries clamped into [0, total] (offsets are only validated
    // with FLOCK_VALIDATE; this keeps every read in bounds)
    auto bound = [&](int g) { return g == fc.n_frames ? fc.total : min(max(fc.offsets[g], 0), fc.total); };
    const int32_t v = flagged_before(fc, bound(f));
    if (fc.out_offsets && (threadIdx.x & 63) == 0) fc.out_offsets[f] = v;
    if (f < fc.n_frames) {
        const int32_t v1 = flagged_before(fc, bound(f + 1));
        if ((threadIdx.x & 63) == 0) fc.counts[f] = max(v1 - v, 0);
    }
}

// ---------------------------------------------------------------------------
// Drinker-line proximity
// ---------------------------------------------------------------------------

// Is (px, py) strictly closer than t to the closed segment s = (ax, ay, bx,
// by)?  The nearest point of the segment is a when the projection of p
// falls before a (or the segment is a point), b when it falls past b, and
// otherwise the foot of the perpendicular, at squared distance
// cross^2 / len2.  Coordinates within 2^24: squared end distances, len2 and
// the projection fit int64, and cross^2 < t^2 len2 is compared as a 128-bit
// product (high and low halves).
__device__ __forceinline__ bool near_segment(int4 s, int px, int py, long long t2) {
    const long long ux = (long long)s.z - s.x, uy = (long long)s.w - s.y;
    const long long wx = (long long)px - s.x, wy = (long long)py - s.y;
    const long long len2 = ux * ux + uy * uy, dot = ux * wx + uy * wy;
    if (len2 == 0 || dot <= 0) return wx * wx + wy * wy < t2;
    if (dot >= len2) {
        const long long vx = (long long)px - s.z, vy = (long long)py - s.w;
        return vx * vx + vy * vy < t2;
    }
    const long long cr = ux * wy - uy * wx;
    const unsigned long long c = (unsigned long long)(cr < 0 ? -cr : cr);
    const unsigned long long ch = __umul64hi(c, c), cl = c * c;
    const unsigned long long lh = __umul64hi((unsigned long long)t2, (unsigned long long)len2),
                             ll = (unsigned long long)t2 * (unsigned long long)len2;
    return ch < lh || (ch == lh && cl < ll);
}

// Flags of one block of birds.  A bird within T of a segment lies in the
// segment's bounding box widened by T on every side, so birds outside all
// widened boxes (most of them, for lines across the frame) are not drinking;
// the others are queued in LDS and tested exactly on the queue, so that whole
// waves run the exact tests.
__global__ __launch_bounds__(kRThreadsR) void drink_flag_kernel(DrinkArgs a, int32_t *bcount) {
    __shared__ int4 seg[kDrinkMaxLines];
    __shared__ int4 box[kDrinkMaxLines];  // x0, y0, x1, y1 widened by T
    __shared__ int2 s_pt[kRBlock];
    __shared__ uint16_t s_at[kRBlock];
    __shared__ int s_nq, s_in;
    const int tid = threadIdx.x, lane = tid & 63;
    if (tid == 0) s_nq = s_in = 0;
    if (tid < a.n_lines) {
        seg[tid] = make_int4(a.ax[tid], a.ay[tid], a.bx[tid], a.by[tid]);
        const int t = a.threshold;  // |coordinates|, T <= 2^24: no overflow
        box[tid] = make_int4(min(a.ax[tid], a.bx[tid]) - t, min(a.ay[tid], a.by[tid]) - t,
                             max(a.ax[tid], a.bx[tid]) + t, max(a.ay[tid], a.by[tid]) + t);
    }
    __syncthreads();
    const long long i0 = (long long)blockIdx.x * kRBlock;
    const int2 *P = reinterpret_cast<const int2 *>(a.xy);
    const long long t2 = (long long)a.threshold * a.threshold;
    int2 pts[kRPer];
#pragma unroll
    for (int k = 0; k < kRPer; ++k) {
        const long long i = i0 + k * kRThreadsR + tid;
        pts[k] = i < a.total ? P[i] : make_int2(0, 0);
    }
    bool cands[kRPer];
#pragma unroll
    for (int k = 0; k < kRPer; ++k) cands[k] = false;
    for (int l = 0; l < a.n_lines; ++l) {  // each box read once, for all of the thread's birds
        const int4 b = box[l];
#pragma unroll
        for (int k = 0; k < kRPer; ++k)
            cands[k] |= (pts[k].x > b.x) & (pts[k].x < b.z) & (pts[k].y > b.y) & (pts[k].y < b.w);
    }
#pragma unroll
    for (int k = 0; k < kRPer; ++k) {
        const long long i = i0 + k * kRThreadsR + tid;
        const bool cand = cands[k] & (i < a.total);
        const uint64_t m = __ballot(cand);
        int base = 0;
        if (lane == 0 && m) base = atomicAdd(&s_nq, __popcll(m));
        base = __shfl(base, 0, 64);
        if (cand) {
            const int q = base + __popcll(m & ((1ull << lane) - 1));
            s_pt[q] = pts[k];
            s_at[q] = (uint16_t)(k * kRThreadsR + tid);
        } else if (i < a.total) {
            a.drinking[i] = 0;
            if (a.line) a.line[i] = -1;
        }
    }
    __syncthreads();
    const int nq = s_nq;
    int cnt = 0;
    for (int q = tid; q < nq; q += kRThreadsR) {
        const int2 pt = s_pt[q];
        int32_t hit = -1;
        for (int l = 0; l < a.n_lines && hit < 0; ++l)
            if (near_segment(seg[l], pt.x, pt.y, t2)) hit = l;
        const long long i = i0 + s_at[q];
        a.drinking[i] = hit >= 0;
        if (a.line) a.line[i] = hit;
        cnt += hit >= 0;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
    if (lane == 0 && cnt) atomicAdd(&s_in, cnt);
    __syncthreads();
    if (tid == 0) bcount[blockIdx.x] = s_in;
}

}  // namespace

// Workspace: a flag per bird; a count and a base per block; per block a
// staging area of kRBlock coordinates and kRBlock input indices.
size_t roi_workspace_bytes(int32_t total) {
    if (total <= 0) return 256;
    const size_t nb = ((size_t)total + kRBlock - 1) / kRBlock;
    return (((size_t)total + 255) & ~(size_t)255) + (((2 * nb + 1) * sizeof(int32_t) + 255) & ~(size_t)255) +
           nb * kRBlock * (sizeof(int2) + sizeof(int32_t));
}

hipError_t launch_roi(const RoiArgs &a, void *workspace, hipStream_t stream) {
    const int nb = (int)(((long long)a.total + kRBlock - 1) / kRBlock);
    uint8_t *flag = static_cast<uint8_t *>(workspace);
    int32_t *bcount = reinterpret_cast<int32_t *>(flag + (a.total > 0 ? (((size_t)a.total + 255) & ~(size_t)255) : 0));
    int32_t *bbase = bcount + nb;
    char *stage = reinterpret_cast<char *>(bcount) + (((2 * (size_t)nb + 1) * sizeof(int32_t) + 255) & ~(size_t)255);
    int2 *stage_xy = reinterpret_cast<int2 *>(stage);
    int32_t *stage_idx = reinterpret_cast<int32_t *>(stage + (size_t)nb * kRBlock * sizeof(int2));
    if (nb > 0)
        hipLaunchKernelGGL(roi_flag_kernel, dim3((unsigned)nb), dim3(kRThreadsR), 0, stream, a, flag, bcount, stage_xy,
                           stage_idx);
    hipLaunchKernelGGL(roi_scan_kernel, dim3(1), dim3(1024), 0, stream, bcount, bbase, nb);
    if (nb > 0)
        hipLaunchKernelGGL(roi_write_kernel, dim3((unsigned)nb), dim3(kRThreadsR), 0, stream, a, bbase, stage_xy,
                           stage_idx);
    const FrameCounts fc{flag, bbase, a.offsets, a.n_frames, a.total, a.counts, a.out_offsets};
    const long long waves = (long long)a.n_frames + 1;
    hipLaunchKernelGGL(frame_counts_kernel, dim3((unsigned)((waves * 64 + 255) / 256)), dim3(256), 0, stream, fc);
    return hipGetLastError();
}

size_t drink_workspace_bytes(int32_t total) {
    const size_t nb = total > 0 ? ((size_t)total + kRBlock - 1) / kRBlock : 0;
    return (((2 * nb + 1) * sizeof(int32_t) + 255) & ~(size_t)255);
}

hipError_t launch_drinkers(const DrinkArgs &a, void *workspace, hipStream_t stream) {
    const int nb = (int)(((long long)a.total + kRBlock - 1) / kRBlock);
    int32_t *bcount = static_cast<int32_t *>(workspace);
    int32_t *bbase = bcount + nb;
    if (nb > 0) hipLaunchKernelGGL(drink_flag_kernel, dim3((unsigned)nb), dim3(kRThreadsR), 0, stream, a, bcount);
    hipLaunchKernelGGL(roi_scan_kernel, dim3(1), dim3(1024), 0, stream, bcount, bbase, nb);
    const FrameCounts fc{a.drinking, bbase, a.offsets, a.n_frames, a.total, a.counts, nullptr};
    const long long waves = (long long)a.n_frames + 1;
    hipLaunchKernelGGL(frame_counts_kernel, dim3((unsigned)((waves * 64 + 255) / 256)), dim3(256), 0, stream, fc);
    return hipGetLastError();
}

}  // namespace flock

// roi.hip - region-of-interest filter and per-frame region counts on gfx950.
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
//   3. roi_write_kernel: ballots and wave totals give each kept bird its rank
//      in its block; coordinates and input index go to base + rank, so kept
//      birds keep their input order;
//   4. roi_offsets_kernel, one wave per frame boundary: the output position
//      of the boundary bird (its block's base plus the flags before it in the
//      block) gives out_offsets, and neighbouring boundaries give counts.

#include "internal.h"

namespace flock {
namespace {

constexpr int kRThreadsR = 256;
constexpr int kRWaves = kRThreadsR / 64;

// Closed polygon test, even-odd rule.  An edge on which the point lies
// decides at once (inside).  Otherwise each edge whose ends lie on
// different sides of the horizontal line through the point (one strictly
// above it, so that a vertex on the line is counted once) toggles the
// result when it meets the line to the right of the point.
__device__ __forceinline__ bool in_polygon(const int2 *poly, int n, int px, int py) {
    bool in = false;
    for (int i = 0; i < n; ++i) {
        const int2 A = poly[i], B = poly[i + 1 == n ? 0 : i + 1];
        const long long ex = (long long)B.x - A.x, ey = (long long)B.y - A.y;
        const long long qx = (long long)px - A.x, qy = (long long)py - A.y;
        const long long cr = ex * qy - ey * qx;
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

__global__ __launch_bounds__(kRThreadsR) void roi_flag_kernel(RoiArgs a, uint8_t *flag, int32_t *bcount) {
    __shared__ int2 poly[kRoiMaxVertices];
    __shared__ int s_cnt[kRWaves];
    load_polygon(a, poly);
    const int tid = threadIdx.x;
    const long long i0 = (long long)blockIdx.x * kRBlock;
    const int2 *P = reinterpret_cast<const int2 *>(a.xy);
    int cnt = 0;
#pragma unroll
    for (int k = 0; k < kRPer; ++k) {
        const long long i = i0 + k * kRThreadsR + tid;
        if (i >= a.total) break;
        const int2 p = P[i];
        const bool in = in_polygon(poly, a.n_vertices, p.x, p.y);
        flag[i] = in;
        cnt += in;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
    if ((tid & 63) == 0) s_cnt[tid >> 6] = cnt;
    __syncthreads();
    if (tid == 0) {
        int t = 0;
        for (int w = 0; w < kRWaves; ++w) t += s_cnt[w];
        bcount[blockIdx.x] = t;
    }
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

__global__ __launch_bounds__(kRThreadsR) void roi_write_kernel(RoiArgs a, const uint8_t *flag,
                                                              const int32_t *bbase) {
    __shared__ int s_tot[kRWaves];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const long long i0 = (long long)blockIdx.x * kRBlock;
    const int2 *P = reinterpret_cast<const int2 *>(a.xy);
    int2 *O = reinterpret_cast<int2 *>(a.out_xy);
    int32_t at = bbase[blockIdx.x];
    for (int k = 0; k < kRPer; ++k) {
        const long long i = i0 + k * kRThreadsR + tid;
        const bool in = i < a.total && flag[i];
        const uint64_t m = __ballot(in);
        if (lane == 0) s_tot[wave] = __popcll(m);
        __syncthreads();
        int before = 0, chunk = 0;
        for (int w = 0; w < kRWaves; ++w) {
            before += w < wave ? s_tot[w] : 0;
            chunk += s_tot[w];
        }
        if (in) {
            const int32_t r = at + before + __popcll(m & ((1ull << lane) - 1ull));
            O[r] = P[i];
            if (a.out_index) a.out_index[r] = (int32_t)i;
        }
        at += chunk;
        __syncthreads();  // s_tot is rewritten by the next chunk
    }
}

// Output position of input bird i0 (0 <= i0 <= total): its block's base plus
// the kept birds before it in the block (wave-uniform call).
__device__ __forceinline__ int32_t out_position(const RoiArgs &a, const uint8_t *flag, const int32_t *bbase,
                                                int32_t i0) {
    const int lane = threadIdx.x & 63;
    const int32_t b = i0 / kRBlock;
    const int32_t s0 = b * kRBlock;
    int c = 0;
    for (int32_t i = s0 + lane; i < i0; i += 64) c += flag[i];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    return bbase[b] + c;  // bbase has nb + 1 entries, and i0 = total gives b <= nb
}

__global__ __launch_bounds__(256) void roi_offsets_kernel(RoiArgs a, const uint8_t *flag, const int32_t *bbase) {
    const int f = (int)(((long long)blockIdx.x * 256 + threadIdx.x) >> 6);
    if (f > a.n_frames) return;  // wave-uniform
    // frame boundaries clamped into [0, total] (offsets are only validated
    // with FLOCK_VALIDATE; this keeps every read in bounds)
    auto bound = [&](int g) { return g == a.n_frames ? a.total : min(max(a.offsets[g], 0), a.total); };
    const int32_t v = out_position(a, flag, bbase, bound(f));
    if ((threadIdx.x & 63) == 0) a.out_offsets[f] = v;
    if (f < a.n_frames) {
        const int32_t v1 = out_position(a, flag, bbase, bound(f + 1));
        if ((threadIdx.x & 63) == 0) a.counts[f] = max(v1 - v, 0);
    }
}

}  // namespace

size_t roi_workspace_bytes(int32_t total) {
    if (total <= 0) return 256;
    const size_t nb = ((size_t)total + kRBlock - 1) / kRBlock;
    return (((size_t)total + 255) & ~(size_t)255) + (((2 * nb + 1) * sizeof(int32_t) + 255) & ~(size_t)255);
}

hipError_t launch_roi(const RoiArgs &a, void *workspace, hipStream_t stream) {
    const int nb = (int)(((long long)a.total + kRBlock - 1) / kRBlock);
    uint8_t *flag = static_cast<uint8_t *>(workspace);
    int32_t *bcount = reinterpret_cast<int32_t *>(flag + (a.total > 0 ? (((size_t)a.total + 255) & ~(size_t)255) : 0));
    int32_t *bbase = bcount + nb;
    if (nb > 0) hipLaunchKernelGGL(roi_flag_kernel, dim3((unsigned)nb), dim3(kRThreadsR), 0, stream, a, flag, bcount);
    hipLaunchKernelGGL(roi_scan_kernel, dim3(1), dim3(1024), 0, stream, bcount, bbase, nb);
    if (nb > 0) hipLaunchKernelGGL(roi_write_kernel, dim3((unsigned)nb), dim3(kRThreadsR), 0, stream, a, flag, bbase);
    const long long waves = (long long)a.n_frames + 1;
    hipLaunchKernelGGL(roi_offsets_kernel, dim3((unsigned)((waves * 64 + 255) / 256)), dim3(256), 0, stream, a, flag,
                       bbase);
    return hipGetLastError();
}

}  // namespace flock

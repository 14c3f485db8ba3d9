// Exact fp64 fallback scan of the assignment (gfx950): the rows whose nearest
// centroid the screening kernels could not certify get it here from the
// exact distance of every centroid, evaluated as the definition states
// (squared L2 in fp64, one subtraction and one fma per dimension in
// ascending order, ties to the lower id). The rows come from the screens'
// worklist or, when the worklist overflowed, from a scan for labels of -1
// (every screen writes the label of every row it is given: the nearest
// centroid, or -1 for a row it hands on).
#include "ivf_internal.h"
#include "exact.h"

#include <math.h>

namespace ivf {
namespace {

constexpr double kInfD = __builtin_huge_val();

// Exact fp64 argmin over all centroids for rows whose top-1 could not be
// certified. Work items are 8 rows (8 worklist entries, or, if the worklist
// overflowed, the -1 labels found in a 1024-row window). Centroids stream
// through LDS in chunks of 128 rows (coalesced loads, row stride D+1 so that
// lanes reading the same dimension of different centroids hit different
// banks); thread (r, j) evaluates row r against chunk centroid j with the
// exact operation sequence, keeps its best (distance, id), and the 128
// threads of each row reduce in a fixed order.
constexpr int kFbRows = 8;
constexpr int kFbChunk = 128;
constexpr int kFbThreads = kFbRows * kFbChunk;

size_t assign_fallback_lds(int D)
{
    return (size_t)(kFbChunk + kFbRows) * (D + 1) * sizeof(float) + kFbThreads * sizeof(int) +
           2 * kFbRows * (kFbChunk / 64) * sizeof(double);
}

// Smallest (distance, id) over centroids [c0, c1) for the nr <= kFbRows rows
// found[0 .. nr): rows staged in LDS (exact as fp32), centroids staged 128 at
// a time, thread (r, j) keeps row r's best over centroids j, j + 128, ...;
// afterwards wd/wi hold each row's best of the two waves that served it.
template <typename XT>
__device__ void fb_scan(const XT *__restrict__ rows, int D, const float *__restrict__ cent, int64_t c0,
                        int64_t c1, const int *found, int nr, float *cs, float *xs, double *wd, int *wi)
{
    const int LW = D + 1;
    const int r = threadIdx.x / kFbChunk;   // row slot of this thread
    const int j = threadIdx.x % kFbChunk;   // centroid slot within a chunk
    const int lane = threadIdx.x & 63;
    for (int i = threadIdx.x; i < kFbRows * D; i += blockDim.x) {
        const int rr = i / D, d = i - rr * D;
        xs[rr * LW + d] = rr < nr ? (float)rows[(int64_t)found[rr] * D + d] : 0.f;
    }
    double bd = kInfD;
    int bi = 0x7fffffff;
    for (int64_t base = c0; base < c1; base += kFbChunk) {
        __syncthreads();
        const int nc = (int)min((int64_t)kFbChunk, c1 - base);
        const int V4 = D / 4;
        for (int i = threadIdx.x; i < nc * V4; i += blockDim.x) {
            const int cc = i / V4, d4 = i - cc * V4;
            const float4 v = *reinterpret_cast<const float4 *>(cent + (base + cc) * D + 4 * d4);
            float *dst = cs + cc * LW + 4 * d4;
            dst[0] = v.x;
            dst[1] = v.y;
            dst[2] = v.z;
            dst[3] = v.w;
        }
        __syncthreads();
        if (r < nr && j < nc) {
            const float *xr = xs + r * LW;
            const float *cr = cs + j * LW;
            double acc = 0.0;
            for (int d = 0; d < D; ++d) {
                const double t = (double)xr[d] - (double)cr[d];
                acc = fma(t, t, acc);
            }
            const int id = (int)(base + j);
            if (dist_lt(acc, id, bd, bi)) {
                bd = acc;
                bi = id;
            }
        }
    }
    // reduce the 128 candidates of each row: two waves per row
    for (int o = 32; o > 0; o >>= 1) {
        const double od = __shfl_xor(bd, o);
        const int oi = __shfl_xor(bi, o);
        if (dist_lt(od, oi, bd, bi)) {
            bd = od;
            bi = oi;
        }
    }
    if (lane == 0) {
        wd[r * 2 + j / 64] = bd;
        wi[r * 2 + j / 64] = bi;
    }
    __syncthreads();
}

// The first kFbSplitWindows windows of kFbRows worklist rows are scanned by
// (window, centroid segment) items spread over the whole grid (a few rows
// need many workgroups to finish quickly); each item leaves its rows' best
// in sd/si[(window * kFbSeg + segment) * kFbRows + row], and
// assign_fallback_merge_kernel reduces them. Nothing to do when the worklist
// overflowed (the full kernel then scans every row whose label is -1).
template <typename XT>
__global__ __launch_bounds__(kFbThreads) void assign_fallback_split_kernel(const XT *__restrict__ rows, int D,
                                                                           const float *__restrict__ cent,
                                                                           int64_t C, const int32_t *wl,
                                                                           const uint32_t *wl_cnt,
                                                                           int64_t wl_cap, double *sd,
                                                                           int32_t *si)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char fb_lds[];
    const int LW = D + 1;
    float *cs = reinterpret_cast<float *>(fb_lds);
    float *xs = cs + kFbChunk * LW;
    int *found = reinterpret_cast<int *>(xs + kFbRows * LW);
    double *wd = reinterpret_cast<double *>(found + kFbThreads);
    int *wi = reinterpret_cast<int *>(wd + kFbRows * (kFbChunk / 64));

    const uint32_t total = *wl_cnt;
    if ((int64_t)total > wl_cap) return;
    const int64_t nwin = min((int64_t)kFbSplitWindows, ((int64_t)total + kFbRows - 1) / kFbRows);
    const int64_t seg = (C + kFbSeg - 1) / kFbSeg;
    for (int64_t item = blockIdx.x; item < nwin * kFbSeg; item += gridDim.x) {
        const int64_t w = item / kFbSeg, sg = item - w * kFbSeg;
        const int nr = (int)min((int64_t)kFbRows, (int64_t)total - w * kFbRows);
        __syncthreads();
        if (threadIdx.x < kFbRows) found[threadIdx.x] = threadIdx.x < nr ? wl[w * kFbRows + threadIdx.x] : 0;
        __syncthreads();
        const int64_t c0 = min(C, sg * seg), c1 = min(C, c0 + seg);
        fb_scan(rows, D, cent, c0, c1, found, nr, cs, xs, wd, wi);
        if (threadIdx.x < nr) {
            const int rr = threadIdx.x;
            const double d0 = wd[rr * 2], d1 = wd[rr * 2 + 1];
            const int i0 = wi[rr * 2], i1 = wi[rr * 2 + 1];
            const bool second = dist_lt(d1, i1, d0, i0);
            sd[item * kFbRows + rr] = second ? d1 : d0;
            si[item * kFbRows + rr] = second ? i1 : i0;
        }
    }
}

// One thread per row of the split windows: the best of its kFbSeg segments.
__global__ __launch_bounds__(256) void assign_fallback_merge_kernel(int32_t *labels, const int32_t *wl,
                                                                    const uint32_t *wl_cnt, int64_t wl_cap,
                                                                    const double *sd, const int32_t *si)
{
    const uint32_t total = *wl_cnt;
    if ((int64_t)total > wl_cap) return;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // worklist entry
    if (e >= min((int64_t)total, (int64_t)kFbSplitWindows * kFbRows)) return;
    const int64_t w = e / kFbRows, rr = e - w * kFbRows;
    double bd = kInfD;
    int bi = 0x7fffffff;
    for (int sg = 0; sg < kFbSeg; ++sg) {
        const int64_t k = (w * kFbSeg + sg) * kFbRows + rr;
        if (dist_lt(sd[k], si[k], bd, bi)) {
            bd = sd[k];
            bi = si[k];
        }
    }
    labels[wl[e]] = bi;
}

// Worklist windows from kFbSplitWindows on (or, when the worklist
// overflowed, every row whose label is -1): one workgroup per window of
// kFbRows rows scans all centroids.
template <typename XT>
__global__ __launch_bounds__(kFbThreads) void assign_fallback_kernel(const XT *__restrict__ rows,
                                                                     int64_t N, int D,
                                                                     const float *__restrict__ cent,
                                                                     int64_t C, int32_t *labels,
                                                                     const int32_t *wl,
                                                                     const uint32_t *wl_cnt,
                                                                     int64_t wl_cap)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char fb_lds[];
    const int LW = D + 1;
    float *cs = reinterpret_cast<float *>(fb_lds);          // [kFbChunk][LW]
    float *xs = cs + kFbChunk * LW;                         // [kFbRows][LW]
    int *found = reinterpret_cast<int *>(xs + kFbRows * LW); // [kFbThreads]
    double *wd = reinterpret_cast<double *>(found + kFbThreads);  // [kFbRows][2]
    int *wi = reinterpret_cast<int *>(wd + kFbRows * (kFbChunk / 64));
    __shared__ int s_n;

    const uint32_t total = *wl_cnt;
    const bool overflow = (int64_t)total > wl_cap;
    const int64_t nwin = overflow ? (N + kFbThreads - 1) / kFbThreads : ((int64_t)total + kFbRows - 1) / kFbRows;
    const int64_t w0 = overflow ? 0 : kFbSplitWindows;

    for (int64_t w = w0 + blockIdx.x; w < nwin; w += gridDim.x) {
        // rows of this work window
        if (threadIdx.x == 0) s_n = 0;
        __syncthreads();
        if (overflow) {
            const int64_t row = w * kFbThreads + threadIdx.x;
            if (row < N && labels[row] < 0) found[atomicAdd(&s_n, 1)] = (int)row;
        } else if (threadIdx.x < kFbRows) {
            const int64_t e = w * kFbRows + threadIdx.x;
            if (e < (int64_t)total) found[atomicAdd(&s_n, 1)] = wl[e];
        }
        __syncthreads();
        const int nfound = s_n;
        for (int g = 0; g < nfound; g += kFbRows) {
            const int nr = min(kFbRows, nfound - g);
            fb_scan(rows, D, cent, 0, C, found + g, nr, cs, xs, wd, wi);
            if (threadIdx.x < nr) {
                const int rr = threadIdx.x;
                double d0 = wd[rr * 2], d1 = wd[rr * 2 + 1];
                int i0 = wi[rr * 2], i1 = wi[rr * 2 + 1];
                labels[found[g + rr]] = dist_lt(d1, i1, d0, i0) ? i1 : i0;
            }
            __syncthreads();
        }
    }
}

}  // namespace

hipError_t launch_assign_fallback(const void *rows, int rowtype, int64_t N, int D,
                                  const float *cent, int64_t C, int32_t *labels,
                                  const int32_t *wl, const uint32_t *wl_cnt, int64_t wl_cap,
                                  double *split_d, int32_t *split_i, int grid, hipStream_t s)
{
    const size_t lds = assign_fallback_lds(D);
    const int merge_grid = (kFbSplitWindows * kFbRows + 255) / 256;
    if (rowtype == kRowU8) {
        hipLaunchKernelGGL(assign_fallback_split_kernel<uint8_t>, dim3(grid), dim3(kFbThreads), lds, s,
                           (const uint8_t *)rows, D, cent, C, wl, wl_cnt, wl_cap, split_d, split_i);
        hipLaunchKernelGGL(assign_fallback_kernel<uint8_t>, dim3(grid), dim3(kFbThreads), lds, s,
                           (const uint8_t *)rows, N, D, cent, C, labels, wl, wl_cnt, wl_cap);
    } else {
        hipLaunchKernelGGL(assign_fallback_split_kernel<float>, dim3(grid), dim3(kFbThreads), lds, s,
                           (const float *)rows, D, cent, C, wl, wl_cnt, wl_cap, split_d, split_i);
        hipLaunchKernelGGL(assign_fallback_kernel<float>, dim3(grid), dim3(kFbThreads), lds, s,
                           (const float *)rows, N, D, cent, C, labels, wl, wl_cnt, wl_cap);
    }
    hipLaunchKernelGGL(assign_fallback_merge_kernel, dim3(merge_grid), dim3(256), 0, s, labels, wl, wl_cnt,
                       wl_cap, split_d, split_i);
    return hipGetLastError();
}

}  // namespace ivf

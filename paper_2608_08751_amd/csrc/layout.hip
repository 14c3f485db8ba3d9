// List-major layout of the base vectors (Sec. "List-major contiguous scans":
// each IVF list becomes one contiguous range) and their residuals x - c(x)
// (Sec. "Residual-PQ Candidate Reduction", residual encoding), on gfx950.
//
// Output position p holds base row perm[p]; its list is the j with
// offsets[j] <= p < offsets[j+1], and c(x) is centroid j. A workgroup takes a
// contiguous range of positions: one thread finds the range's first list by
// binary search over the offsets, and every row group then only moves its
// list index forward, so no per-row label is read and a centroid is reloaded
// only at list boundaries. A thread handles a 4-element unit of a row (one
// float4 of residual, so every residual store of a wave is contiguous); a
// uint8 copy without residuals uses 16-byte units. Every thread keeps
// several rows in flight to cover the latency of the dependent id -> row
// loads. The kernel is bound by HBM bandwidth.
#include "ivf_internal.h"

#include <math.h>

namespace ivf {
namespace {

constexpr int kLmThreads = 256;
constexpr int kLmRows = 512;   // output positions per workgroup
constexpr int kLmFlight = 4;   // rows each thread has in flight

// A unit is 16 bytes of a row: 16 uint8 elements (D % 16 == 0) or 4 fp32.
template <typename XT>
struct Unit;
template <>
struct Unit<uint8_t> {
    static constexpr int kElems = 16;
    typedef uint4 type;
    __device__ static void to_float(const uint4 &w, float (&f)[16])
    {
        const uint32_t v[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f[4 * k + 0] = (float)(v[k] & 0xFFu);
            f[4 * k + 1] = (float)((v[k] >> 8) & 0xFFu);
            f[4 * k + 2] = (float)((v[k] >> 16) & 0xFFu);
            f[4 * k + 3] = (float)(v[k] >> 24);
        }
    }
};
template <>
struct Unit<float> {
    static constexpr int kElems = 4;
    typedef float4 type;
    __device__ static void to_float(const float4 &w, float (&f)[4])
    {
        f[0] = w.x;
        f[1] = w.y;
        f[2] = w.z;
        f[3] = w.w;
    }
};
// uint8 rows whose length is not a multiple of 16 use 4-byte units
struct NarrowU8 {
    static constexpr int kElems = 4;
    typedef uint32_t type;
    __device__ static void to_float(const uint32_t &w, float (&f)[4])
    {
        f[0] = (float)(w & 0xFFu);
        f[1] = (float)((w >> 8) & 0xFFu);
        f[2] = (float)((w >> 16) & 0xFFu);
        f[3] = (float)(w >> 24);
    }
};

template <typename XT, typename UT>
__global__ __launch_bounds__(kLmThreads) void list_major_kernel(
    const XT *__restrict__ base, int64_t N, const float *__restrict__ cent, int64_t C, int D,
    const int64_t *__restrict__ offsets, const uint32_t *__restrict__ perm, int64_t pos0,
    int64_t n, XT *__restrict__ out_rows, float *__restrict__ out_res)
{
    typedef typename UT::type U;
    constexpr int E = UT::kElems;
    __shared__ int64_t first_list;
    const int units = D / E;
    const int groups = kLmThreads / units;  // rows per sweep of the workgroup
    const int g = threadIdx.x / units;
    const int e0 = (threadIdx.x - g * units) * E;  // first element of this thread's unit
    const int64_t p0 = pos0 + (int64_t)blockIdx.x * kLmRows;
    const int64_t p1 = min(p0 + kLmRows, pos0 + n);
    if (threadIdx.x == 0) {
        // the last list j with offsets[j] <= p0 (offsets[0] = 0 <= p0)
        int64_t lo = 0, hi = C - 1;
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo + 1) / 2;
            if (offsets[mid] <= p0)
                lo = mid;
            else
                hi = mid - 1;
        }
        first_list = lo;
    }
    __syncthreads();
    if (g >= groups) return;
    int64_t j = first_list;
    int64_t next = j + 1 < C ? offsets[j + 1] : INT64_MAX;
    const float nan = __builtin_nanf("");
    for (int64_t pb = p0 + g; pb < p1; pb += (int64_t)groups * kLmFlight) {
        // ids and lists of up to kLmFlight rows, then all their loads, then the stores
        uint32_t src[kLmFlight];
        int64_t lst[kLmFlight];
#pragma unroll
        for (int k = 0; k < kLmFlight; ++k) {
            const int64_t p = pb + (int64_t)k * groups;
            src[k] = p < p1 ? perm[p] : 0xFFFFFFFFu;
            if (p < p1) {
                while (p >= next) {  // lists are visited in order (empty ones skipped)
                    ++j;
                    next = j + 1 < C ? offsets[j + 1] : INT64_MAX;
                }
            }
            lst[k] = j;
        }
        U w[kLmFlight];
#pragma unroll
        for (int k = 0; k < kLmFlight; ++k) {
            w[k] = U{};
            if (src[k] < (uint64_t)N) w[k] = *reinterpret_cast<const U *>(base + (int64_t)src[k] * D + e0);
        }
#pragma unroll
        for (int k = 0; k < kLmFlight; ++k) {
            const int64_t p = pb + (int64_t)k * groups;
            if (p >= p1) break;
            const int64_t q = p - pos0;  // output row
            const bool ok = src[k] < (uint64_t)N;
            if (out_rows) *reinterpret_cast<U *>(out_rows + q * D + e0) = w[k];
            if (out_res) {
                float x[E];
                UT::to_float(w[k], x);
                const float *c = cent + lst[k] * D + e0;
                float *r = out_res + q * D + e0;
#pragma unroll
                for (int t = 0; t < E; t += 4) {
                    const float4 cv = *reinterpret_cast<const float4 *>(c + t);
                    const float4 rv = ok ? make_float4(x[t] - cv.x, x[t + 1] - cv.y, x[t + 2] - cv.z,
                                                       x[t + 3] - cv.w)
                                         : make_float4(nan, nan, nan, nan);
                    *reinterpret_cast<float4 *>(r + t) = rv;
                }
            }
        }
    }
}

}  // namespace

hipError_t launch_list_major(const void *base, int rowtype, int64_t N, const float *cent, int64_t C,
                             int D, const int64_t *offsets, const uint32_t *perm, int64_t pos0,
                             int64_t n, void *out_rows, float *out_res, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    const int64_t grid = (n + kLmRows - 1) / kLmRows;
    if (rowtype == kRowU8 && D % 16 == 0 && !out_res)
        hipLaunchKernelGGL((list_major_kernel<uint8_t, Unit<uint8_t>>), dim3((unsigned)grid),
                           dim3(kLmThreads), 0, s, (const uint8_t *)base, N, cent, C, D, offsets, perm,
                           pos0, n, (uint8_t *)out_rows, out_res);
    else if (rowtype == kRowU8)
        hipLaunchKernelGGL((list_major_kernel<uint8_t, NarrowU8>), dim3((unsigned)grid),
                           dim3(kLmThreads), 0, s, (const uint8_t *)base, N, cent, C, D, offsets, perm,
                           pos0, n, (uint8_t *)out_rows, out_res);
    else
        hipLaunchKernelGGL((list_major_kernel<float, Unit<float>>), dim3((unsigned)grid),
                           dim3(kLmThreads), 0, s, (const float *)base, N, cent, C, D, offsets, perm,
                           pos0, n, (float *)out_rows, out_res);
    return hipGetLastError();
}

}  // namespace ivf

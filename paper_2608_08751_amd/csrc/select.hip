// Norms, routing threshold, certified top-k selection with fp64 refinement,
// and the exact fp64 fallback scans (gfx950).
//
// Coarse search returns, per query, the nprobe centroids of smallest squared
// L2 distance (Eq. 1), selected on the device so that only O(B*P) ids and
// distances leave the GPU ("On-device list selection", Sec. "GPU coarse
// search"). The screening keys from the MFMA kernel carry a rounding error of
// at most B per key; the selection below only trusts them as far as B allows
// and decides the final order with exact fp64 distances.
#include "ivf_internal.h"

#include <math.h>

namespace ivf {
namespace {

constexpr float kInfF = __builtin_huge_valf();
constexpr double kInfD = __builtin_huge_val();

__device__ __forceinline__ bool dist_lt(double da, int ia, double db, int ib)
{
    return da < db || (da == db && ia < ib);
}

__device__ __forceinline__ bool key_lt(float ka, int ia, float kb, int ib)
{
    return ka < kb || (ka == kb && ia < ib);
}

// The distance of the exactness contract: fp64, ascending dims, fma.
template <typename XT>
__device__ __forceinline__ double exact_dist(const XT *__restrict__ x, const float *__restrict__ c,
                                             int D)
{
    double s = 0.0;
    for (int d = 0; d < D; ++d) {
        const double t = (double)x[d] - (double)c[d];
        s = fma(t, t, s);
    }
    return s;
}

__device__ __forceinline__ double key_bound(double coef, uint32_t mc2_bits, double xn2)
{
    const double M = (double)__uint_as_float(mc2_bits) * (1.0 + 0x1p-20);
    return coef * (M + 2.0 * sqrt(xn2 * (1.0 + 0x1p-40)) * sqrt(M)) + 0x1p-100;
}

__device__ __forceinline__ int pow2_at_least(int n)
{
    int p = 1;
    while (p < n) p <<= 1;
    return p;
}

// Bitonic sort of P (power of two) entries in LDS by (key, id) ascending.
template <typename K, typename LT>
__device__ void bitonic_sort(K *key, int *id, int P, LT lt)
{
    for (int k = 2; k <= P; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < P; i += blockDim.x) {
                const int ixj = i ^ j;
                if (ixj > i) {
                    const bool up = (i & k) == 0;
                    const K ka = key[i], kb = key[ixj];
                    const int ia = id[i], ib = id[ixj];
                    const bool swap = up ? lt(kb, ib, ka, ia) : lt(ka, ia, kb, ib);
                    if (swap) {
                        key[i] = kb;
                        key[ixj] = ka;
                        id[i] = ib;
                        id[ixj] = ia;
                    }
                }
            }
            __syncthreads();
        }
    }
}

__global__ void fill_u32_kernel(uint32_t *p, int64_t n, uint32_t v)
{
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// fl32(||c||^2) per centroid (fp64 accumulation, one wave per row) and the
// maximum over all rows (as float bits; floats >= 0 order like their bits).
__global__ __launch_bounds__(256) void centroid_norms_kernel(const float *__restrict__ cent,
                                                             int64_t C, int D,
                                                             float *__restrict__ cnorm,
                                                             uint32_t *__restrict__ mc2_bits)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    __shared__ uint32_t wmax[4];
    uint32_t mx = 0;
    for (int64_t r = (int64_t)blockIdx.x * 4 + wave; r < C; r += (int64_t)gridDim.x * 4) {
        double s = 0.0;
        for (int d = lane; d < D; d += 64) {
            const double v = (double)cent[r * D + d];
            s = fma(v, v, s);
        }
        for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
        const float n = (float)s;
        if (lane == 0) cnorm[r] = n;
        mx = max(mx, __float_as_uint(n));
    }
    if (lane == 0) wmax[wave] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t m = max(max(wmax[0], wmax[1]), max(wmax[2], wmax[3]));
        atomicMax(mc2_bits, m);
    }
}

__global__ __launch_bounds__(256) void row_norms_kernel(const float *__restrict__ rows, int64_t n,
                                                        int D, double *__restrict__ out)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    for (int64_t r = (int64_t)blockIdx.x * 4 + wave; r < n; r += (int64_t)gridDim.x * 4) {
        double s = 0.0;
        for (int d = lane; d < D; d += 64) {
            const double v = (double)rows[r * D + d];
            s = fma(v, v, s);
        }
        for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
        if (lane == 0) out[r] = s;
    }
}

// Routing threshold from the sample keys [0, Cs) of one query: the keys are cut
// into groups of 16 consecutive centroids, tau = the rank_j-th smallest group
// minimum (so about rank_j sample keys lie at or below tau), and every sample
// key <= tau is emitted as a candidate. With Cs == 0, tau = +inf.
constexpr int kMaxGroups = 4096;

__global__ __launch_bounds__(256) void route_threshold_kernel(RouteArgs a)
{
    const int64_t q = blockIdx.x;
    __shared__ float gm[kMaxGroups];
    __shared__ int gid[kMaxGroups];
    __shared__ uint32_t s_cnt;
    if (a.Cs == 0) {
        if (threadIdx.x == 0) {
            a.tau[q] = kInfF;
            a.cand_cnt[q] = 0;
        }
        return;
    }
    const int G = (int)(a.Cs / 16);
    const int P = pow2_at_least(G);
    const float *kr = a.keys + q * a.Cs;
    for (int g = threadIdx.x; g < P; g += blockDim.x) {
        float m = kInfF;
        if (g < G) {
            const float4 *p = reinterpret_cast<const float4 *>(kr + 16 * (int64_t)g);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float4 v = p[i];
                m = fminf(m, fminf(fminf(v.x, v.y), fminf(v.z, v.w)));
            }
        }
        gm[g] = m;
        gid[g] = g;
    }
    if (threadIdx.x == 0) s_cnt = 0;
    __syncthreads();
    bitonic_sort(gm, gid, P, key_lt);
    const float th = gm[min(a.rank_j, G) - 1];
    for (int64_t i = threadIdx.x; i < a.Cs; i += blockDim.x) {
        const float k = kr[i];
        if (k <= th) {
            const uint32_t slot = atomicAdd(&s_cnt, 1u);
            if (slot < (uint32_t)a.L) a.cand[q * a.L + slot] = make_uint2(__float_as_uint(k), (uint32_t)i);
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a.tau[q] = th;
        a.cand_cnt[q] = s_cnt;
    }
}

// Certified selection of one query's top-k from its screened candidates.
// Candidates = every centroid with key <= tau. Let kth = the k-th smallest key.
// If tau >= kth + 2B, every centroid outside {key <= kth + 2B} is strictly
// farther (exactly) than k candidates, so the exact top-k lies in that set;
// its members are re-evaluated in fp64 and sorted by (distance, id).
// Otherwise (or on overflow / underflow) the query goes to the fallback scan.
constexpr int kMaxCand = 4096;

__global__ __launch_bounds__(256) void route_select_kernel(RouteArgs a)
{
    const int64_t q = blockIdx.x;
    __shared__ float sk[kMaxCand];
    __shared__ int si[kMaxCand];
    __shared__ double sd[kMaxCand];
    __shared__ float qrow[256];
    __shared__ int s_nr;
    const uint32_t n = a.cand_cnt[q];
    if (threadIdx.x == 0) atomicAdd(a.stats + kStatCandidates, (unsigned long long)n);
    const bool overflow = n > (uint32_t)a.L;
    if (a.force_fallback || overflow || n < (uint32_t)a.k) {
        if (threadIdx.x == 0) {
            const uint32_t slot = atomicAdd(a.wl_cnt, 1u);
            a.wl[slot] = (int32_t)q;
            atomicAdd(a.stats + kStatFallback, 1ull);
            if (overflow) atomicAdd(a.stats + kStatOverflow, 1ull);
        }
        return;
    }
    const int P = pow2_at_least((int)n);
    for (int i = threadIdx.x; i < P; i += blockDim.x) {
        if (i < (int)n) {
            const uint2 c = a.cand[q * a.L + i];
            sk[i] = __uint_as_float(c.x);
            si[i] = (int)c.y;
        } else {
            sk[i] = kInfF;
            si[i] = 0x7fffffff;
        }
    }
    for (int d = threadIdx.x; d < a.D; d += blockDim.x) qrow[d] = a.queries[q * a.D + d];
    if (threadIdx.x == 0) s_nr = 0;
    __syncthreads();
    bitonic_sort(sk, si, P, key_lt);
    const double kth = (double)sk[a.k - 1];
    const double B2 = 2.0 * key_bound(a.bound_coef, *a.mc2_bits, a.qn2[q]);
    if (!((double)a.tau[q] >= kth + B2)) {
        if (threadIdx.x == 0) {
            const uint32_t slot = atomicAdd(a.wl_cnt, 1u);
            a.wl[slot] = (int32_t)q;
            atomicAdd(a.stats + kStatFallback, 1ull);
        }
        return;
    }
    const double thr = kth + B2;
    int cnt = 0;
    for (int i = threadIdx.x; i < (int)n; i += blockDim.x) cnt += ((double)sk[i] <= thr) ? 1 : 0;
    atomicAdd(&s_nr, cnt);
    __syncthreads();
    const int nr = s_nr;  // a prefix of the sorted candidates, nr >= k
    const int PR = pow2_at_least(nr);
    // exact distances of the prefix (in place of the keys' storage order)
    for (int i = threadIdx.x; i < PR; i += blockDim.x) {
        if (i < nr) {
            sd[i] = exact_dist(qrow, a.cent + (int64_t)si[i] * a.D, a.D);
        } else {
            sd[i] = kInfD;
            si[i] = 0x7fffffff;
        }
    }
    __syncthreads();
    bitonic_sort(sd, si, PR, dist_lt);
    for (int i = threadIdx.x; i < a.k; i += blockDim.x) {
        a.out_ids[q * a.k + i] = si[i];
        if (a.out_dist) a.out_dist[q * a.k + i] = (float)sd[i];
    }
}

// Exact fp64 scan of all centroids for the queries on the worklist: a running
// best list of K2 entries plus a buffer of new entries that beat its k-th
// element; the union is re-sorted whenever the buffer fills.
__global__ __launch_bounds__(256) void route_fallback_kernel(RouteArgs a)
{
    __shared__ double bd[2048];
    __shared__ int bi[2048];
    __shared__ float qrow[256];
    __shared__ uint32_t s_cnt;
    const uint32_t total = *a.wl_cnt;
    int K2 = 256;
    while (K2 < a.k) K2 <<= 1;
    for (uint32_t w = blockIdx.x; w < total; w += gridDim.x) {
        const int64_t q = a.wl[w];
        for (int i = threadIdx.x; i < 2 * K2; i += blockDim.x) {
            bd[i] = kInfD;
            bi[i] = 0x7fffffff;
        }
        for (int d = threadIdx.x; d < a.D; d += blockDim.x) qrow[d] = a.queries[q * a.D + d];
        if (threadIdx.x == 0) s_cnt = 0;
        __syncthreads();
        double wd = kInfD;
        int wi = 0x7fffffff;
        for (int64_t base = 0; base < a.C; base += blockDim.x) {
            const int64_t c = base + threadIdx.x;
            if (c < a.C) {
                const double d = exact_dist(qrow, a.cent + c * a.D, a.D);
                if (dist_lt(d, (int)c, wd, wi)) {
                    const uint32_t slot = atomicAdd(&s_cnt, 1u);
                    bd[K2 + slot] = d;
                    bi[K2 + slot] = (int)c;
                }
            }
            __syncthreads();
            const bool last = base + blockDim.x >= a.C;
            if (s_cnt > (uint32_t)(K2 - blockDim.x) || last) {
                bitonic_sort(bd, bi, 2 * K2, dist_lt);
                for (int i = K2 + threadIdx.x; i < 2 * K2; i += blockDim.x) {
                    bd[i] = kInfD;
                    bi[i] = 0x7fffffff;
                }
                if (threadIdx.x == 0) s_cnt = 0;
                __syncthreads();
                wd = bd[a.k - 1];
                wi = bi[a.k - 1];
            }
            __syncthreads();
        }
        for (int i = threadIdx.x; i < a.k; i += blockDim.x) {
            a.out_ids[q * a.k + i] = bi[i];
            if (a.out_dist) a.out_dist[q * a.k + i] = (float)bd[i];
        }
        __syncthreads();
    }
}

// Exact fp64 argmin over all centroids for rows whose top-1 could not be
// certified. Rows come from the worklist, or, if it overflowed, from a scan of
// the labels for the -1 marker.
template <typename XT>
__global__ __launch_bounds__(256) void assign_fallback_kernel(const XT *__restrict__ rows,
                                                              int64_t N, int D,
                                                              const float *__restrict__ cent,
                                                              int64_t C, int32_t *labels,
                                                              const int32_t *wl,
                                                              const uint32_t *wl_cnt,
                                                              int64_t wl_cap)
{
    __shared__ double rd[4];
    __shared__ int ri[4];
    __shared__ int s_rows[256];
    __shared__ int s_n;
    const uint32_t total = *wl_cnt;
    const bool overflow = (int64_t)total > wl_cap;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nitems = overflow ? (N + 255) / 256 : (int64_t)total;
    for (int64_t w = blockIdx.x; w < nitems; w += gridDim.x) {
        // gather the rows of this work item
        if (threadIdx.x == 0) s_n = 0;
        __syncthreads();
        if (overflow) {
            const int64_t r = w * 256 + threadIdx.x;
            if (r < N && labels[r] < 0) s_rows[atomicAdd(&s_n, 1)] = (int)r;
        } else if (threadIdx.x == 0) {
            s_rows[0] = wl[w];
            s_n = 1;
        }
        __syncthreads();
        const int nrow = s_n;
        for (int t = 0; t < nrow; ++t) {
            const int64_t r = s_rows[t];
            const XT *x = rows + r * D;
            double bd = kInfD;
            int bi = 0x7fffffff;
            for (int64_t c = threadIdx.x; c < C; c += blockDim.x) {
                const double d = exact_dist(x, cent + c * D, D);
                if (dist_lt(d, (int)c, bd, bi)) {
                    bd = d;
                    bi = (int)c;
                }
            }
            for (int o = 32; o > 0; o >>= 1) {
                const double od = __shfl_xor(bd, o);
                const int oi = __shfl_xor(bi, o);
                if (dist_lt(od, oi, bd, bi)) {
                    bd = od;
                    bi = oi;
                }
            }
            if (lane == 0) {
                rd[wave] = bd;
                ri[wave] = bi;
            }
            __syncthreads();
            if (threadIdx.x == 0) {
                for (int v = 1; v < 4; ++v)
                    if (dist_lt(rd[v], ri[v], rd[0], ri[0])) {
                        rd[0] = rd[v];
                        ri[0] = ri[v];
                    }
                labels[r] = ri[0];
            }
            __syncthreads();
        }
    }
}

int grid_for(int64_t n, int per_block, int cap)
{
    int64_t g = (n + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

}  // namespace

hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(n, 256, 4096)), dim3(256), 0, s, p, n, v);
    return hipGetLastError();
}

hipError_t launch_centroid_norms(const float *cent, int64_t C, int D, float *cnorm,
                                 uint32_t *mc2_bits, hipStream_t s)
{
    hipLaunchKernelGGL(centroid_norms_kernel, dim3(grid_for(C, 4, 2048)), dim3(256), 0, s, cent, C, D,
                       cnorm, mc2_bits);
    return hipGetLastError();
}

hipError_t launch_row_norms(const float *rows, int64_t n, int D, double *out, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(row_norms_kernel, dim3(grid_for(n, 4, 4096)), dim3(256), 0, s, rows, n, D, out);
    return hipGetLastError();
}

hipError_t launch_route_threshold(const RouteArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(route_threshold_kernel, dim3((unsigned)a.nq), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_route_select(const RouteArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(route_select_kernel, dim3((unsigned)a.nq), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_route_fallback(const RouteArgs &a, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(route_fallback_kernel, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_assign_fallback(const void *rows, int rowtype, int64_t N, int D,
                                  const float *cent, int64_t C, int32_t *labels,
                                  const int32_t *wl, const uint32_t *wl_cnt, int64_t wl_cap,
                                  int grid, hipStream_t s)
{
    if (rowtype == kRowU8)
        hipLaunchKernelGGL(assign_fallback_kernel<uint8_t>, dim3(grid), dim3(256), 0, s,
                           (const uint8_t *)rows, N, D, cent, C, labels, wl, wl_cnt, wl_cap);
    else
        hipLaunchKernelGGL(assign_fallback_kernel<float>, dim3(grid), dim3(256), 0, s,
                           (const float *)rows, N, D, cent, C, labels, wl, wl_cnt, wl_cap);
    return hipGetLastError();
}

}  // namespace ivf

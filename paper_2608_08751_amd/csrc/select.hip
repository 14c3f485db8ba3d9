// Norms, routing threshold, certified top-k selection with fp64 refinement,
// and the exact fp64 fallback scan of queries (gfx950).
//
// Coarse search returns, per query, the nprobe centroids of smallest squared
// L2 distance (Eq. 1), selected on the device so that only O(B*P) ids and
// distances leave the GPU ("On-device list selection", Sec. "GPU coarse
// search"). The screening keys from the MFMA kernel carry a rounding error of
// at most B per key; the selection below only trusts them as far as B allows
// and decides the final order with exact fp64 distances.
#include "ivf_internal.h"
#include "exact.h"

#include <math.h>

namespace ivf {
namespace {

constexpr float kInfF = __builtin_huge_valf();
constexpr double kInfD = __builtin_huge_val();

__device__ __forceinline__ bool key_lt(float ka, int ia, float kb, int ib)
{
    return ka < kb || (ka == kb && ia < ib);
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

// fl32(||c||^2) per centroid (fp64 accumulation in dimension order, one
// thread per row, 16-byte loads; D % 4 == 0) and the maximum over all rows
// (as float bits; floats >= 0 order like their bits).
__global__ __launch_bounds__(256) void centroid_norms_kernel(const float *__restrict__ cent,
                                                             int64_t C, int D,
                                                             float *__restrict__ cnorm,
                                                             uint32_t *__restrict__ mc2_bits)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    __shared__ uint32_t wmax[4];
    uint32_t mx = 0;
    for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < C; r += (int64_t)gridDim.x * 256) {
        const float4 *p = reinterpret_cast<const float4 *>(cent + r * D);
        double s = 0.0;
        for (int d4 = 0; d4 < D / 4; d4 += 8) {
            float4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (d4 + u < D / 4) v[u] = p[d4 + u];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                if (d4 + u < D / 4) {
                    s = fma((double)v[u].x, (double)v[u].x, s);
                    s = fma((double)v[u].y, (double)v[u].y, s);
                    s = fma((double)v[u].z, (double)v[u].z, s);
                    s = fma((double)v[u].w, (double)v[u].w, s);
                }
            }
        }
        const float n = (float)s;
        cnorm[r] = n;
        mx = max(mx, __float_as_uint(n));
    }
    for (int o = 32; o > 0; o >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, o));
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

// Order-preserving map between non-NaN floats and uint32 keys.
__device__ __forceinline__ uint32_t f2o(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float o2f(uint32_t u)
{
    return __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);
}

// k-th smallest (1-based, k <= number of values) of the values spread over
// the workgroup (thread t holds v[e] for e < nv): MSD radix select, four
// passes of 8 bits with a 256-bin LDS histogram each; one wave locates the
// bin that contains rank k with a prefix scan. Returns the exact value.
template <int V>
__device__ uint32_t block_select(const uint32_t (&v)[V], int nv, int k, uint32_t *hist,
                                 uint32_t *sh)
{
    uint32_t prefix = 0, mask = 0, krem = (uint32_t)k;
    const int lane = threadIdx.x & 63;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
        __syncthreads();
#pragma unroll
        for (int e = 0; e < V; ++e)
            if (e < nv && (v[e] & mask) == prefix) atomicAdd(&hist[(v[e] >> shift) & 0xFFu], 1u);
        __syncthreads();
        if (threadIdx.x < 64) {
            const uint32_t c0 = hist[4 * lane], c1 = hist[4 * lane + 1];
            const uint32_t c2 = hist[4 * lane + 2], c3 = hist[4 * lane + 3];
            const uint32_t own = c0 + c1 + c2 + c3;
            uint32_t incl = own;
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t up = __shfl_up(incl, o);
                if (lane >= o) incl += up;
            }
            const uint32_t before = incl - own;
            if (before < krem && krem <= incl) {
                uint32_t r = krem - before;
                int bin = 4 * lane;
                if (r > c0) { r -= c0; ++bin;
                    if (r > c1) { r -= c1; ++bin;
                        if (r > c2) { r -= c2; ++bin; } } }
                sh[0] = (uint32_t)bin;
                sh[1] = r;
            }
        }
        __syncthreads();
        prefix |= sh[0] << shift;
        mask |= 0xFFu << shift;
        krem = sh[1];
        __syncthreads();
    }
    return prefix;
}

// Routing threshold from the Cs sample keys of one query: the keys are cut
// into groups of 16 consecutive sample centroids, tau = the rank_j-th smallest group
// minimum (so about rank_j sample keys lie at or below tau), and every sample
// key <= tau is emitted as a candidate. With Cs == 0, tau = +inf.
constexpr int kMaxGroups = 4096;
constexpr int kGroupsPerThread = kMaxGroups / 256;

// true when the int8 route kernels produce this call's keys (group minima)
__device__ __forceinline__ bool int8_keys(const RouteArgs &a) { return a.i8_off && *a.i8_off == 0u; }

// Centroid id of sample key s: the sample is the chunks j * sstride of kChunk
// centroids, its keys in that order.
__device__ __forceinline__ uint32_t sample_id(const RouteArgs &a, int64_t s)
{
    const int64_t st = a.sstride > 1 ? a.sstride : 1;
    return (uint32_t)((s / kChunk) * st * kChunk + s % kChunk);
}

__global__ __launch_bounds__(256) void route_threshold_kernel(RouteArgs a)
{
    if (int8_keys(a)) return;
    const int64_t q = blockIdx.x;
    __shared__ uint32_t hist[256];
    __shared__ uint32_t sh[2];
    __shared__ uint32_t s_cnt;
    if (a.Cs == 0) {
        if (threadIdx.x == 0) {
            a.tau[q] = kInfF;
            a.cand_cnt[q] = 0;
        }
        return;
    }
    const int G = (int)(a.Cs / 16);
    const float *kr = a.keys + q * a.Cs;
    uint32_t v[kGroupsPerThread];
    int nv = 0;
#pragma unroll
    for (int e = 0; e < kGroupsPerThread; ++e) {
        const int g = threadIdx.x + 256 * e;
        v[e] = 0xFFFFFFFFu;
        if (g < G) {
            const float4 *p = reinterpret_cast<const float4 *>(kr + 16 * (int64_t)g);
            float m = kInfF;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float4 w = p[i];
                m = fminf(m, fminf(fminf(w.x, w.y), fminf(w.z, w.w)));
            }
            v[e] = f2o(m);
            nv = e + 1;
        }
    }
    if (threadIdx.x == 0) s_cnt = 0;
    const float th = o2f(block_select(v, nv, min(a.rank_j, G), hist, sh));
    const float4 *k4 = reinterpret_cast<const float4 *>(kr);
    for (int64_t i = threadIdx.x; i < a.Cs / 4; i += blockDim.x) {
        const float4 w = k4[i];
        const float kk[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (kk[e] <= th) {
                const uint32_t slot = atomicAdd(&s_cnt, 1u);
                if (slot < (uint32_t)a.L)
                    a.cand[q * a.L + slot] = make_uint2(__float_as_uint(kk[e]), sample_id(a, 4 * i + e));
            }
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a.tau[q] = th;
        a.cand_cnt[q] = s_cnt;
    }
}

// The same threshold with the query's sample keys read once: thread t keeps
// groups t, t + 256, ... (GPT of them, 16 keys each) in registers, takes
// their minima for the selection and then emits its own keys <= tau. Used
// when the sample has at most 256 * GPT groups.
template <int GPT>
__global__ __launch_bounds__(256) void route_threshold_reg_kernel(RouteArgs a)
{
    if (int8_keys(a)) return;
    const int64_t q = blockIdx.x;
    __shared__ uint32_t hist[256];
    __shared__ uint32_t sh[2];
    __shared__ uint32_t s_cnt;
    const int G = (int)(a.Cs / 16);
    const float4 *k4 = reinterpret_cast<const float4 *>(a.keys + q * a.Cs);
    float4 w[GPT][4];
    uint32_t v[GPT];
    int nv = 0;
#pragma unroll
    for (int e = 0; e < GPT; ++e) {
        const int g = threadIdx.x + 256 * e;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[e][i] = g < G ? k4[4 * (int64_t)g + i] : make_float4(kInfF, kInfF, kInfF, kInfF);
    }
#pragma unroll
    for (int e = 0; e < GPT; ++e) {
        float m = kInfF;
#pragma unroll
        for (int i = 0; i < 4; ++i) m = fminf(m, fminf(fminf(w[e][i].x, w[e][i].y), fminf(w[e][i].z, w[e][i].w)));
        v[e] = 0xFFFFFFFFu;
        if (threadIdx.x + 256 * e < G) {
            v[e] = f2o(m);
            nv = e + 1;
        }
    }
    if (threadIdx.x == 0) s_cnt = 0;
    const float th = o2f(block_select(v, nv, min(a.rank_j, G), hist, sh));
#pragma unroll
    for (int e = 0; e < GPT; ++e) {
        const int g = threadIdx.x + 256 * e;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float kk[4] = {w[e][i].x, w[e][i].y, w[e][i].z, w[e][i].w};
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if (g < G && kk[c] <= th) {
                    const uint32_t slot = atomicAdd(&s_cnt, 1u);
                    if (slot < (uint32_t)a.L)
                        a.cand[q * a.L + slot] = make_uint2(__float_as_uint(kk[c]), sample_id(a, 16 * g + 4 * i + c));
                }
            }
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a.tau[q] = th;
        a.cand_cnt[q] = s_cnt;
    }
}

// The threshold from the group minima the fp32 keys pass wrote: tau = the
// rank_j-th smallest minimum, then only the groups whose minimum is <= tau
// (about rank_j of them) are read for their keys <= tau, which become
// candidates (a group whose minimum exceeds tau holds none).
__global__ __launch_bounds__(256) void route_threshold_gmin_kernel(RouteArgs a)
{
    if (int8_keys(a)) return;
    const int64_t q = blockIdx.x;
    __shared__ uint32_t hist[256];
    __shared__ uint32_t sh[2];
    __shared__ uint32_t s_cnt;
    const int G = (int)(a.Cs / 16);
    const float *gmin = a.kmin + q * G;
    uint32_t v[kGroupsPerThread];
    int nv = 0;
#pragma unroll
    for (int e = 0; e < kGroupsPerThread; ++e) {
        const int g = threadIdx.x + 256 * e;
        v[e] = 0xFFFFFFFFu;
        if (g < G) {
            v[e] = f2o(gmin[g]);
            nv = e + 1;
        }
    }
    if (threadIdx.x == 0) s_cnt = 0;
    const uint32_t tho = block_select(v, nv, min(a.rank_j, G), hist, sh);
    const float th = o2f(tho);
    const float4 *k4 = reinterpret_cast<const float4 *>(a.keys + q * a.Cs);
#pragma unroll
    for (int e = 0; e < kGroupsPerThread; ++e) {
        const int g = threadIdx.x + 256 * e;
        if (g < G && v[e] <= tho) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float4 w = k4[4 * (int64_t)g + i];
                const float kk[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    if (kk[c] <= th) {
                        const uint32_t slot = atomicAdd(&s_cnt, 1u);
                        if (slot < (uint32_t)a.L)
                            a.cand[q * a.L + slot] = make_uint2(__float_as_uint(kk[c]), sample_id(a, 16 * g + 4 * i + c));
                    }
                }
            }
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a.tau[q] = th;
        a.cand_cnt[q] = s_cnt;
    }
}

// The threshold when the int8 route kernels ran: the keys buffer holds the
// sample's group minima [nq, Cs / 16] directly, tau = the rank_j-th smallest,
// and the sample's centroids are left to the filter, which then covers every
// centroid (the candidate list starts empty).
__global__ __launch_bounds__(256) void route_threshold_min_kernel(RouteArgs a)
{
    if (!int8_keys(a)) return;
    const int64_t q = blockIdx.x;
    __shared__ uint32_t hist[256];
    __shared__ uint32_t sh[2];
    const int G = (int)(a.Cs / 16);
    const float *kr = a.keys + q * G;
    uint32_t v[kGroupsPerThread];
    int nv = 0;
#pragma unroll
    for (int e = 0; e < kGroupsPerThread; ++e) {
        const int g = threadIdx.x + 256 * e;
        v[e] = 0xFFFFFFFFu;
        if (g < G) {
            v[e] = f2o(kr[g]);
            nv = e + 1;
        }
    }
    const float th = o2f(block_select(v, nv, min(a.rank_j, G), hist, sh));
    if (threadIdx.x == 0) {
        a.tau[q] = th;
        a.cand_cnt[q] = 0;
    }
}

// Certified selection of one query's top-k from its screened candidates.
// Candidates = every centroid with key <= tau. Let kth = the k-th smallest key
// (radix select). If tau >= kth + 2B, every centroid outside
// R = {key <= kth + 2B} is strictly farther (exactly) than k candidates, so the
// exact top-k lies in R; R's members are re-evaluated in fp64 and ranked by
// (distance, id). Otherwise (or on overflow / underflow) the query goes to
// the fallback scan.
constexpr int kMaxCand = 4096;
constexpr int kCandPerThread = kMaxCand / 256;

__device__ __forceinline__ void push_fallback(const RouteArgs &a, int64_t q, bool overflow)
{
    const uint32_t slot = atomicAdd(a.wl_cnt, 1u);
    a.wl[slot] = (int32_t)q;
    atomicAdd(a.stats + kStatFallback, 1ull);
    if (overflow) atomicAdd(a.stats + kStatOverflow, 1ull);
}

__global__ __launch_bounds__(256) void route_select_kernel(RouteArgs a)
{
    const int64_t q = blockIdx.x;
    __shared__ uint32_t hist[256];
    __shared__ uint32_t sh[2];
    __shared__ __attribute__((aligned(16))) float qrow[256];
    __shared__ int s_nr;
    // R (at most L <= kMaxCand entries): fp64 distances, then ids
    extern __shared__ __attribute__((aligned(16))) unsigned char sel_lds[];
    double *rd = reinterpret_cast<double *>(sel_lds);
    int *rid = reinterpret_cast<int *>(rd + a.L);
    const uint32_t n = a.cand_cnt[q];
    const bool overflow = n > (uint32_t)a.L;
    if (a.force_fallback || overflow || n < (uint32_t)a.k) {
        if (threadIdx.x == 0) push_fallback(a, q, overflow);
        return;
    }
    uint32_t v[kCandPerThread];
    int cid[kCandPerThread];
    int nv = 0;
#pragma unroll
    for (int e = 0; e < kCandPerThread; ++e) {
        const int i = threadIdx.x + 256 * e;
        v[e] = 0xFFFFFFFFu;
        cid[e] = 0;
        if (i < (int)n) {
            const uint2 c = a.cand[q * a.L + i];
            v[e] = f2o(__uint_as_float(c.x));
            cid[e] = (int)c.y;
            nv = e + 1;
        }
    }
    for (int d = threadIdx.x; d < a.D; d += blockDim.x) qrow[d] = a.queries[q * a.D + d];
    if (threadIdx.x == 0) s_nr = 0;
    const double kth = (double)o2f(block_select(v, nv, a.k, hist, sh));
    const double B2 = a.i8_off && *a.i8_off == 0u ? 2.0 * (double)a.qbound[q]
                                                  : 2.0 * key_bound(a.bound_coef, *a.mc2_bits, a.qn2[q]);
    if (!((double)a.tau[q] >= kth + B2)) {
        if (threadIdx.x == 0) push_fallback(a, q, false);
        return;
    }
    const double thr = kth + B2;
#pragma unroll
    for (int e = 0; e < kCandPerThread; ++e)
        if (e < nv && (double)o2f(v[e]) <= thr) rid[atomicAdd(&s_nr, 1)] = cid[e];
    __syncthreads();
    const int nr = s_nr;  // >= k
    for (int i = threadIdx.x; i < nr; i += blockDim.x)
        rd[i] = exact_dist(qrow, a.cent + (int64_t)rid[i] * a.D, a.D);
    __syncthreads();
    // rank of each re-evaluated candidate in (distance, id) order
    for (int i = threadIdx.x; i < nr; i += blockDim.x) {
        const double di = rd[i];
        const int ii = rid[i];
        int rank = 0;
        for (int j = 0; j < nr; ++j) rank += dist_lt(rd[j], rid[j], di, ii) ? 1 : 0;
        if (rank < a.k) {
            a.out_ids[q * a.k + rank] = ii;
            if (a.out_dist) a.out_dist[q * a.k + rank] = (float)di;
        }
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
    __shared__ unsigned long long s_sum[4];
    {
        // the candidate total of the batch for the statistics (one atomic
        // per workgroup instead of one per query)
        unsigned long long sum = 0;
        for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < a.nq; q += (int64_t)gridDim.x * blockDim.x)
            sum += a.cand_cnt[q];
        for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
        if ((threadIdx.x & 63) == 0) s_sum[threadIdx.x >> 6] = sum;
        __syncthreads();
        if (threadIdx.x == 0) {
            const unsigned long long t = s_sum[0] + s_sum[1] + s_sum[2] + s_sum[3];
            if (t) atomicAdd(a.stats + kStatCandidates, t);
        }
    }
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
    hipLaunchKernelGGL(centroid_norms_kernel, dim3(grid_for(C, 256, 4096)), dim3(256), 0, s, cent, C, D,
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
    const int64_t G = a.Cs / 16;
    if (a.i8_off && a.Cs > 0) hipLaunchKernelGGL(route_threshold_min_kernel, dim3((unsigned)a.nq), dim3(256), 0, s, a);
    if (a.Cs > 0 && a.kmin && G <= kMaxGroups)
        hipLaunchKernelGGL(route_threshold_gmin_kernel, dim3((unsigned)a.nq), dim3(256), 0, s, a);
    else if (a.Cs > 0 && G <= 256)
        hipLaunchKernelGGL(route_threshold_reg_kernel<1>, dim3((unsigned)a.nq), dim3(256), 0, s, a);
    else if (a.Cs > 0 && G <= 512)
        hipLaunchKernelGGL(route_threshold_reg_kernel<2>, dim3((unsigned)a.nq), dim3(256), 0, s, a);
    else if (a.Cs > 0 && G <= 1024)
        hipLaunchKernelGGL(route_threshold_reg_kernel<4>, dim3((unsigned)a.nq), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(route_threshold_kernel, dim3((unsigned)a.nq), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_route_select(const RouteArgs &a, hipStream_t s)
{
    const size_t lds = (size_t)a.L * (sizeof(double) + sizeof(int));
    hipLaunchKernelGGL(route_select_kernel, dim3((unsigned)a.nq), dim3(256), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_route_fallback(const RouteArgs &a, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(route_fallback_kernel, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}


}  // namespace ivf

// Residual-PQ approximate-distance scan on gfx950 (Sec. "Residual-PQ
// Candidate Reduction": lookup tables and ADC sums; Sec. "Compact PQ-Code
// Offloading": chunked scan with local top-K, hierarchical merge to a
// bounded per-query handoff of N_rerank candidates).
//
// For query b and probed list l: r = q - c_l (fp32), LUT[m][j] = the fp64
// distance of the contract between r^(m) and codeword j of subspace m,
// rounded to fp32, and for every position p of list l
//     d~ = ((0 + LUT[0][a_0]) + LUT[1][a_1]) + ... ,   a = codes[p],
// with candidate id perm[p]. Candidates are ordered by (d~, id) through one
// 64-bit key: (order-preserving bits of d~) << 32 | id.
//
// Level 1 (adc_list_kernel): one workgroup per (query, probe slot) builds
// the LUT in LDS, scans the list in chunks of kAdcChunk codes and keeps its
// k smallest keys in an LDS pool (an exact MSD radix select trims the pool
// whenever it holds more than k), then hands them to the workspace. Level 2
// (adc_merge_kernel): one workgroup per query runs the same pool over its
// P * k handed-over keys and sorts the k smallest. Ids are unique within a
// query (lists are disjoint), so "the k smallest keys" is exact.
#include "ivf_internal.h"

namespace ivf {
namespace {

constexpr int kAdcThreads = 256;
constexpr int kAdcChunk = 1024;                          // codes appended per round
constexpr int kAdcPool = kAdcMaxK + kAdcChunk;            // LDS pool capacity (keys)
constexpr int kAdcKeysPerThread = kAdcPool / kAdcThreads;
constexpr uint64_t kNoKey = ~0ull;

__device__ __forceinline__ uint32_t f2o(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float o2f(uint32_t u)
{
    return __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);
}

struct PoolLds {
    uint64_t key[kAdcPool];
    uint32_t hist[256];
    uint32_t sel_digit, sel_below;
    uint32_t n;  // keys in the pool
};

// Leaves exactly the k smallest of the pool's n (> k) unique keys in it.
__device__ void pool_trim(PoolLds &P, int k)
{
    const int t = threadIdx.x;
    const int n = (int)P.n;
    uint64_t prefix = 0, mask = 0;
    uint32_t kk = (uint32_t)k;  // rank of the target inside the current prefix
    for (int shift = 56; shift >= 0; shift -= 8) {
        P.hist[t] = 0;
        __syncthreads();
        for (int i = t; i < n; i += kAdcThreads) {
            const uint64_t v = P.key[i];
            if ((v & mask) == prefix) atomicAdd(&P.hist[(v >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (t < 64) {  // one wave: the digit whose cumulative count reaches kk
            const uint32_t h0 = P.hist[4 * t], h1 = P.hist[4 * t + 1], h2 = P.hist[4 * t + 2],
                           h3 = P.hist[4 * t + 3];
            const uint32_t own = h0 + h1 + h2 + h3;
            uint32_t incl = own;
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t up = __shfl_up(incl, o);
                if (t >= o) incl += up;
            }
            uint32_t before = incl - own;
            if (before < kk && kk <= incl) {
                int dgt = 4 * t;
                uint32_t b = before;
                if (b + h0 < kk) {
                    b += h0;
                    ++dgt;
                    if (b + h1 < kk) {
                        b += h1;
                        ++dgt;
                        if (b + h2 < kk) {
                            b += h2;
                            ++dgt;
                        }
                    }
                }
                P.sel_digit = (uint32_t)dgt;
                P.sel_below = b;
            }
        }
        __syncthreads();
        prefix |= (uint64_t)P.sel_digit << shift;
        mask |= 255ull << shift;
        kk -= P.sel_below;
        __syncthreads();
    }
    // prefix is now the k-th smallest key: keep the keys <= prefix
    uint64_t mine[kAdcKeysPerThread];
#pragma unroll
    for (int e = 0; e < kAdcKeysPerThread; ++e) {
        const int i = t + e * kAdcThreads;
        mine[e] = i < n ? P.key[i] : kNoKey;
    }
    if (t == 0) P.n = 0;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < kAdcKeysPerThread; ++e)
        if (mine[e] <= prefix && mine[e] != kNoKey) P.key[atomicAdd(&P.n, 1u)] = mine[e];
    __syncthreads();
    // with unique keys exactly k remain; repeated ids (not a valid list
    // layout) must not let the pool outgrow its capacity
    if (t == 0 && P.n > (uint32_t)k) P.n = (uint32_t)k;
    __syncthreads();
}

__global__ __launch_bounds__(kAdcThreads) void adc_list_kernel(
    const float *__restrict__ Q, int D, const float *__restrict__ cent, int64_t C,
    const int32_t *__restrict__ probes, int P, const int64_t *__restrict__ offsets,
    const uint32_t *__restrict__ perm, int64_t N, const uint8_t *__restrict__ codes, int M,
    const float *__restrict__ codebooks, int k, uint64_t *__restrict__ handoff)
{
    extern __shared__ float dyn[];  // r [D] then LUT [M][256]
    __shared__ PoolLds pool;
    float *r = dyn;
    float *lut = dyn + D;
    const int t = threadIdx.x;
    const int64_t b = blockIdx.x / P;
    const int s = (int)(blockIdx.x - b * P);
    uint64_t *out = handoff + (int64_t)blockIdx.x * k;
    const int32_t l = probes[b * P + s];
    if (l < 0 || l >= C) {  // not a list: hand over nothing
        for (int i = t; i < k; i += kAdcThreads) out[i] = kNoKey;
        return;
    }
    const int dsub = D / M;
    for (int d = t; d < D; d += kAdcThreads) r[d] = Q[b * D + d] - cent[(int64_t)l * D + d];
    if (t == 0) pool.n = 0;
    __syncthreads();
    for (int e = t; e < M * kPqK; e += kAdcThreads) {
        const int m = e >> 8;
        const float *w = codebooks + (int64_t)e * dsub;
        const float *rm = r + m * dsub;
        double acc = 0.0;
        for (int d = 0; d < dsub; ++d) {
            const double u = (double)rm[d] - (double)w[d];
            acc = fma(u, u, acc);
        }
        lut[e] = (float)acc;
    }
    __syncthreads();
    // positions of list l, kept inside [0, N) whatever the offsets hold
    const int64_t o0 = min(max(offsets[l], (int64_t)0), N);
    const int64_t o1 = min(max(offsets[l + 1], o0), N);
    for (int64_t c0 = o0; c0 < o1; c0 += kAdcChunk) {
        const int len = (int)min((int64_t)kAdcChunk, o1 - c0);
        const int base = (int)pool.n;
        for (int i = t; i < len; i += kAdcThreads) {
            const int64_t p = c0 + i;
            const uint8_t *a = codes + p * M;
            float acc = 0.0f;
            if ((M & 3) == 0) {
                for (int m = 0; m < M; m += 4) {
                    const uint32_t w = *reinterpret_cast<const uint32_t *>(a + m);
                    acc = acc + lut[(m + 0) * kPqK + (w & 0xFFu)];
                    acc = acc + lut[(m + 1) * kPqK + ((w >> 8) & 0xFFu)];
                    acc = acc + lut[(m + 2) * kPqK + ((w >> 16) & 0xFFu)];
                    acc = acc + lut[(m + 3) * kPqK + (w >> 24)];
                }
            } else {
                for (int m = 0; m < M; ++m) acc = acc + lut[m * kPqK + a[m]];
            }
            pool.key[base + i] = ((uint64_t)f2o(acc) << 32) | perm[p];
        }
        __syncthreads();
        if (t == 0) pool.n = (uint32_t)(base + len);
        __syncthreads();
        if ((int)pool.n > k) pool_trim(pool, k);
    }
    const int n = (int)pool.n;
    for (int i = t; i < k; i += kAdcThreads) out[i] = i < n ? pool.key[i] : kNoKey;
}

__global__ __launch_bounds__(kAdcThreads) void adc_merge_kernel(const uint64_t *__restrict__ handoff,
                                                               int P, int k, uint32_t *__restrict__ ids,
                                                               float *__restrict__ dist)
{
    __shared__ PoolLds pool;
    const int t = threadIdx.x;
    const int64_t b = blockIdx.x;
    const uint64_t *in = handoff + b * (int64_t)P * k;
    const int64_t total = (int64_t)P * k;
    if (t == 0) pool.n = 0;
    __syncthreads();
    for (int64_t c0 = 0; c0 < total; c0 += kAdcChunk) {
        const int len = (int)min((int64_t)kAdcChunk, total - c0);
        // append the chunk's real keys (missing entries are skipped)
        for (int i = t; i < len; i += kAdcThreads) {
            const uint64_t v = in[c0 + i];
            if (v != kNoKey) pool.key[atomicAdd(&pool.n, 1u)] = v;
        }
        __syncthreads();
        if ((int)pool.n > k) pool_trim(pool, k);
    }
    // bitonic sort of the pool (at most k <= kAdcMaxK keys) ascending
    const int n = (int)pool.n;
    int np = 1;
    while (np < n) np <<= 1;
    for (int i = n + t; i < np; i += kAdcThreads) pool.key[i] = kNoKey;
    __syncthreads();
    for (int size = 2; size <= np; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = t; i < np; i += kAdcThreads) {
                const int j = i ^ stride;
                if (j > i) {
                    const bool up = (i & size) == 0;
                    const uint64_t a = pool.key[i], c = pool.key[j];
                    if ((a > c) == up) {
                        pool.key[i] = c;
                        pool.key[j] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
    for (int i = t; i < k; i += kAdcThreads) {
        const bool have = i < n;
        const uint64_t v = have ? pool.key[i] : kNoKey;
        ids[b * k + i] = have ? (uint32_t)v : 0xFFFFFFFFu;
        dist[b * k + i] = have ? o2f((uint32_t)(v >> 32)) : __builtin_huge_valf();
    }
}

}  // namespace

hipError_t launch_adc_scan(const float *Q, int64_t B, int D, const float *cent, int64_t C,
                           const int32_t *probes, int P, const int64_t *offsets, const uint32_t *perm,
                           int64_t N, const uint8_t *codes, int M, const float *codebooks, int k,
                           uint64_t *handoff, uint32_t *ids, float *dist, hipStream_t s)
{
    if (B <= 0) return hipSuccess;
    const size_t lds = (size_t)(D + M * kPqK) * sizeof(float);
    hipLaunchKernelGGL(adc_list_kernel, dim3((unsigned)(B * P)), dim3(kAdcThreads), lds, s, Q, D, cent, C,
                       probes, P, offsets, perm, N, codes, M, codebooks, k, handoff);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(adc_merge_kernel, dim3((unsigned)B), dim3(kAdcThreads), 0, s, handoff, P, k, ids, dist);
    return hipGetLastError();
}

}  // namespace ivf

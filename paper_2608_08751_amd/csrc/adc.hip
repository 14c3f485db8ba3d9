// Residual-PQ approximate-distance scan on gfx950 (Sec. "Residual-PQ
// Candidate Reduction": lookup tables and ADC sums; Sec. "Compact PQ-Code
// Offloading": GPU-side task setup, chunked scan with local top-K, fused
// first merge, hierarchical merge to a bounded per-query handoff of N_rerank
// candidates).
//
// For query b and probed list l: r = q - c_l (fp32), LUT[m][j] = the fp64
// distance of the contract between r^(m) and codeword j of subspace m,
// rounded to fp32, and for every position p of list l
//     d~ = ((0 + LUT[0][a_0]) + LUT[1][a_1]) + ... ,   a = codes[p],
// with candidate id perm[p]. Candidates are ordered by (d~, id) through one
// 64-bit key: (order-preserving bits of d~) << 32 | id.
//
// Work decomposition. Every probed list is cut into chunks of kAdcChunk
// codes (the last one partial); the chunks of a list are taken in runs of
// G_b (the group size of query b, max(kAdcMinGroup, ceil(chunks_b / P))), so a
// short list is one group and a long one is spread over several groups, and a
// query has at most 2P groups (the workspace holds 2P * k handoff keys per
// query).
//   adc_setup_kernel   one workgroup per query: the chunk counts of its
//                      probed lists, G_b, the groups of every list and their
//                      exclusive scan over the probes (each group's slot),
//                      and one descriptor per group (list, code range);
//   adc_group_kernel   one workgroup per group slot (slots past the query's
//                      group count return at once): builds the list's LUT,
//                      scans the group's chunks and keeps the k smallest keys
//                      in an LDS pool (an exact MSD radix select trims it
//                      whenever it holds more than k), then hands over those k
//                      keys: the chunk scan and the first merge are one
//                      kernel, chunk-level candidates never leave LDS;
//   adc_merge_kernel   one workgroup per query merges its groups' keys into
//                      the k smallest and sorts them.
// Ids are unique within a query (lists are disjoint), so "the k smallest
// keys" is exact whatever the grouping.
#include "ivf_internal.h"

#include <algorithm>

namespace ivf {
namespace {

constexpr int kAdcThreads = 256;
constexpr int kAdcChunk = 1024;                          // codes per chunk (appended per round)
constexpr int kAdcMinGroup = 8;                          // chunks per group at least
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
    uint64_t thr;  // the k-th smallest key at the last trim (keys >= thr cannot enter)
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
    if (t == 0) {
        P.n = 0;
        P.thr = prefix;
    }
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

// Positions [o0, o1) of list l, kept inside [0, N) whatever the offsets hold;
// an id outside [0, C) is an empty list.
__device__ __forceinline__ void list_range(const int64_t *__restrict__ offsets, int64_t C, int64_t N, int32_t l,
                                           int64_t &o0, int64_t &o1)
{
    if (l < 0 || l >= C) {
        o0 = o1 = 0;
        return;
    }
    o0 = min(max(offsets[l], (int64_t)0), N);
    o1 = min(max(offsets[l + 1], o0), N);
}

// Task setup of query b: the group size, the groups of each probed list
// (prefix over the probes gives each group's slot j < 2P), and for every
// group its list and code range: dl[b][j], dpos[b][j] = (first, end).
__global__ __launch_bounds__(kAdcThreads) void adc_setup_kernel(const int32_t *__restrict__ probes, int P,
                                                                const int64_t *__restrict__ offsets, int64_t C,
                                                                int64_t N, int32_t *__restrict__ gcnt,
                                                                int32_t *__restrict__ dl,
                                                                longlong2 *__restrict__ dpos)
{
    __shared__ int32_t wsum[kAdcThreads / 64];
    __shared__ int32_t s_g;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t b = blockIdx.x;
    // thread t takes the contiguous probes [t * per, (t + 1) * per)
    const int per = (P + kAdcThreads - 1) / kAdcThreads;  // <= 16
    int32_t nch[16];
    int64_t o0s[16], o1s[16];
    int32_t tot = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int p = t * per + e;
        nch[e] = 0;
        o0s[e] = o1s[e] = 0;
        if (e < per && p < P) {
            list_range(offsets, C, N, probes[b * P + p], o0s[e], o1s[e]);
            nch[e] = (int32_t)((o1s[e] - o0s[e] + kAdcChunk - 1) / kAdcChunk);
        }
        tot += nch[e];
    }
    // chunks of the query -> group size
    int32_t s = tot;
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) wsum[wave] = s;
    __syncthreads();
    if (t == 0) {
        int32_t n = 0;
        for (int w = 0; w < kAdcThreads / 64; ++w) n += wsum[w];
        s_g = max(kAdcMinGroup, (n + P - 1) / P);
    }
    __syncthreads();
    const int32_t G = s_g;
    // groups per list and their exclusive scan over the probes
    int32_t ng = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) ng += (nch[e] + G - 1) / G;
    int32_t incl = ng;
    for (int o = 1; o < 64; o <<= 1) {
        const int32_t up = __shfl_up(incl, o);
        if (lane >= o) incl += up;
    }
    __syncthreads();
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int32_t j = incl - ng;
    for (int w = 0; w < wave; ++w) j += wsum[w];
    const int64_t base = b * 2 * (int64_t)P;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        if (nch[e] == 0) continue;
        const int32_t l = probes[b * P + t * per + e];
        for (int64_t f = o0s[e]; f < o1s[e]; f += (int64_t)G * kAdcChunk, ++j) {
            dl[base + j] = l;
            dpos[base + j] = make_longlong2(f, min(o1s[e], f + (int64_t)G * kAdcChunk));
        }
    }
    if (t == kAdcThreads - 1) gcnt[b] = j;  // the last thread ends past every group
}

// Group slot (b, j) of every query (grid B * 2P).
__global__ __launch_bounds__(kAdcThreads) void adc_group_kernel(
    const float *__restrict__ Q, int D, const float *__restrict__ cent, int P, const uint32_t *__restrict__ perm,
    const uint8_t *__restrict__ codes, int M, const float *__restrict__ codebooks, int k,
    const int32_t *__restrict__ gcnt, const int32_t *__restrict__ dl, const longlong2 *__restrict__ dpos,
    uint64_t *__restrict__ handoff, int32_t *__restrict__ hcnt)
{
    extern __shared__ double dyn[];  // r [D] (fp64) then LUT [M][256] (fp32)
    __shared__ PoolLds pool;
    double *r = dyn;
    float *lut = reinterpret_cast<float *>(dyn + D);
    const int t = threadIdx.x;
    const int64_t b = blockIdx.x / (2 * P);
    const int j = (int)(blockIdx.x - b * 2 * P);
    if (j >= gcnt[b]) return;  // no such group
    const int64_t slot = b * 2 * (int64_t)P + j;
    const int32_t l = dl[slot];
    const longlong2 range = dpos[slot];
    const int dsub = D / M;
    // the residual in fp32 (as defined), held in fp64 for the table's sums
    for (int d = t; d < D; d += kAdcThreads) r[d] = (double)(Q[b * D + d] - cent[(int64_t)l * D + d]);
    if (t == 0) {
        pool.n = 0;
        pool.thr = kNoKey;
    }
    __syncthreads();
    if (dsub == 8) {
        // the common 8-dimension subspace: two 16-byte codebook loads per entry
        for (int e = t; e < M * kPqK; e += kAdcThreads) {
            const float4 *wr = reinterpret_cast<const float4 *>(codebooks + (int64_t)e * 8);
            const float4 w0 = wr[0], w1 = wr[1];
            const float w[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
            const double *rm = r + (e >> 8) * 8;
            double acc = 0.0;
#pragma unroll
            for (int d = 0; d < 8; ++d) {
                const double v = rm[d] - (double)w[d];
                acc = fma(v, v, acc);
            }
            lut[e] = (float)acc;
        }
    } else {
        for (int e = t; e < M * kPqK; e += kAdcThreads) {
            const float *wr = codebooks + (int64_t)e * dsub;
            const double *rm = r + (e >> 8) * dsub;
            double acc = 0.0;
            for (int d = 0; d < dsub; ++d) {
                const double v = rm[d] - (double)wr[d];
                acc = fma(v, v, acc);
            }
            lut[e] = (float)acc;
        }
    }
    __syncthreads();
    // Keys are unique (distance bits, then the row id), so once a trim has
    // left the k smallest, a key at or above the k-th of them cannot enter:
    // only smaller keys are appended (a wave reserves its slots with one LDS
    // atomic), and the pool is trimmed when the next chunk might not fit.
    const int lane = t & 63;
    for (int64_t c0 = range.x; c0 < range.y; c0 += kAdcChunk) {
        const int len = (int)min((int64_t)kAdcChunk, range.y - c0);
        const uint64_t thr = pool.thr;
        for (int i0 = 0; i0 < len; i0 += kAdcThreads) {
            const int i = i0 + t;
            uint64_t key = kNoKey;
            if (i < len) {
                const int64_t pos = c0 + i;
                const uint8_t *a = codes + pos * M;
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
                key = ((uint64_t)f2o(acc) << 32) | perm[pos];
            }
            const bool keep = i < len && key < thr;
            const uint64_t want = __ballot(keep);
            if (want != 0) {
                uint32_t wbase = 0;
                if (lane == 0) wbase = atomicAdd(&pool.n, (uint32_t)__popcll(want));
                wbase = __shfl(wbase, 0);
                if (keep) pool.key[wbase + __popcll(want & ((1ull << lane) - 1))] = key;
            }
        }
        __syncthreads();
        if ((int)pool.n > kAdcPool - kAdcChunk) pool_trim(pool, k);
    }
    if ((int)pool.n > k) pool_trim(pool, k);
    // the group's keys (at most k) and their count
    uint64_t *out = handoff + slot * k;
    const int n = (int)pool.n;
    for (int i = t; i < n; i += kAdcThreads) out[i] = pool.key[i];
    if (t == 0) hcnt[slot] = n;
}

__global__ __launch_bounds__(kAdcThreads) void adc_merge_kernel(const uint64_t *__restrict__ handoff,
                                                               const int32_t *__restrict__ hcnt, int P, int k,
                                                               const int32_t *__restrict__ gcnt,
                                                               uint32_t *__restrict__ ids, float *__restrict__ dist)
{
    __shared__ PoolLds pool;
    const int t = threadIdx.x;
    const int64_t b = blockIdx.x;
    const uint64_t *in = handoff + b * 2 * (int64_t)P * k;
    const int32_t *hc = hcnt + b * 2 * (int64_t)P;
    const int G = gcnt[b];  // the query's groups
    if (t == 0) pool.n = 0;
    __syncthreads();
    // append the groups' keys (n <= k each) while they fit the pool; trim it
    // to the k smallest only when the next group would not fit
    for (int g = 0; g < G; ++g) {
        const int n = hc[g];
        if ((int)pool.n + n > kAdcPool) pool_trim(pool, k);  // then pool.n = k, and k + n <= kAdcPool
        const int base = (int)pool.n;
        for (int i = t; i < n; i += kAdcThreads) pool.key[base + i] = in[(int64_t)g * k + i];
        __syncthreads();
        if (t == 0) pool.n = (uint32_t)(base + n);
        __syncthreads();
    }
    if ((int)pool.n > k) pool_trim(pool, k);
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
                           const AdcScratch &w, uint32_t *ids, float *dist, hipStream_t s)
{
    if (B <= 0) return hipSuccess;
    hipLaunchKernelGGL(adc_setup_kernel, dim3((unsigned)B), dim3(kAdcThreads), 0, s, probes, P, offsets, C, N,
                       w.gcnt, w.dl, w.dpos);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t lds = (size_t)D * sizeof(double) + (size_t)M * kPqK * sizeof(float);
    hipLaunchKernelGGL(adc_group_kernel, dim3((unsigned)(B * 2 * P)), dim3(kAdcThreads), lds, s, Q, D, cent, P,
                       perm, codes, M, codebooks, k, w.gcnt, w.dl, w.dpos, w.handoff, w.hcnt);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(adc_merge_kernel, dim3((unsigned)B), dim3(kAdcThreads), 0, s, w.handoff, w.hcnt, P, k,
                       w.gcnt, ids, dist);
    return hipGetLastError();
}

}  // namespace ivf

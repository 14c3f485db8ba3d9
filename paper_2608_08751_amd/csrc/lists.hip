// Inverted-list build on gfx950: counts, exclusive-scan offsets and the
// stable permutation of row ids grouped by list (the cluster-major layout with
// per-list offset, length and vector ids, Sec. "System Architecture").
//
// Rows are cut into nblocks contiguous blocks and buckets into slices of
// kSlice lists; workgroup (block b, slice s) owns LDS counters for its slice.
//   1. hist      cnt[b][j] = #{rows of block b with label j}      (LDS atomics)
//   2. colscan   cnt[b][j] <- sum_{b' < b} cnt[b'][j]; counts[j] = column total
//   3. offsets   offsets = exclusive prefix sum of counts, offsets[C] = N
//   4. scatter   rows of block b are placed at offsets[j] + cnt[b][j] + rank,
//                where rank counts earlier rows of block b with label j; the
//                block is walked in sub-chunks of kSub rows in row order, and
//                ranks among equal labels inside a sub-chunk are fixed
//                explicitly (not by atomic order), so the result is the
//                stable order, identical on every run.
// Labels are read with coalesced 16-byte loads; the slices of one block are
// mapped to the same XCD so that their reads of the same labels share an L2.
#include "ivf_internal.h"

namespace ivf {
namespace {

__device__ __forceinline__ void decode_block(int w, int nblocks, int nslices, int &b, int &s)
{
    if (nblocks % 8 == 0) {
        // consecutive workgroup ids go to different XCDs (round robin by 8):
        // give all slices of a block the same id modulo 8
        b = (w % 8) + 8 * (w / (8 * nslices));
        s = (w / 8) % nslices;
    } else {
        b = w / nslices;
        s = w % nslices;
    }
}

// Four consecutive labels starting at r (r % 4 == 0); -1 beyond r1.
__device__ __forceinline__ int4 load_labels4(const int32_t *__restrict__ labels, int64_t r, int64_t r1)
{
    if (r + 3 < r1) return *reinterpret_cast<const int4 *>(labels + r);
    int4 v;
    v.x = r < r1 ? labels[r] : -1;
    v.y = r + 1 < r1 ? labels[r + 1] : -1;
    v.z = r + 2 < r1 ? labels[r + 2] : -1;
    v.w = r + 3 < r1 ? labels[r + 3] : -1;
    return v;
}

__global__ __launch_bounds__(kBuildThreads) void hist_kernel(const int32_t *__restrict__ labels,
                                                             int64_t N, int64_t R, int64_t C,
                                                             int nblocks, int nslices,
                                                             uint32_t *__restrict__ cntmat)
{
    __shared__ uint32_t cnt[kSlice];
    int b, s;
    decode_block(blockIdx.x, nblocks, nslices, b, s);
    const int64_t j0 = (int64_t)s * kSlice;
    const int width = (int)min((int64_t)kSlice, C - j0);
    for (int i = threadIdx.x; i < width; i += blockDim.x) cnt[i] = 0;
    __syncthreads();
    const int64_t r0 = (int64_t)b * R;
    const int64_t r1 = min(N, r0 + R);
    const int64_t step = 4 * (int64_t)blockDim.x;
    for (int64_t r = r0 + 4 * (int64_t)threadIdx.x; r < r1; r += 4 * step) {
        int4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = load_labels4(labels, r + u * step, r1);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int l[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t rel = (uint32_t)((int64_t)l[e] - j0);
                if (l[e] >= 0 && rel < (uint32_t)width) atomicAdd(&cnt[rel], 1u);
            }
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < width; i += blockDim.x) cntmat[(int64_t)b * C + j0 + i] = cnt[i];
}

__global__ __launch_bounds__(256) void colscan_kernel(uint32_t *__restrict__ cntmat, int64_t C,
                                                      int nblocks, int64_t *__restrict__ counts)
{
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < C;
         j += (int64_t)gridDim.x * blockDim.x) {
        uint32_t run = 0;
        for (int b = 0; b < nblocks; ++b) {
            const uint32_t v = cntmat[(int64_t)b * C + j];
            cntmat[(int64_t)b * C + j] = run;
            run += v;
        }
        counts[j] = run;
    }
}

// Exclusive scan of counts by one workgroup of 1,024 threads, in passes of
// 16,384 counts: each thread loads 16 consecutive counts at once (one memory
// latency per pass), scans them in registers, and the thread totals are
// scanned across the wave (shuffles) and the 16 waves (LDS); a carry links
// the passes.
constexpr int kOffPer = 16;

__global__ __launch_bounds__(1024) void offsets_kernel(const int64_t *__restrict__ counts,
                                                       int64_t C, int64_t *__restrict__ offsets)
{
    __shared__ int64_t wtot[16];
    __shared__ int64_t carry_s;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t carry = 0;
    for (int64_t base = 0; base < C; base += 1024 * kOffPer) {
        const int64_t j0 = base + (int64_t)threadIdx.x * kOffPer;
        int64_t v[kOffPer];
        if (j0 + kOffPer <= C) {
#pragma unroll
            for (int k = 0; k < kOffPer; k += 2) {
                const longlong2 u = *reinterpret_cast<const longlong2 *>(counts + j0 + k);
                v[k] = u.x;
                v[k + 1] = u.y;
            }
        } else {
#pragma unroll
            for (int k = 0; k < kOffPer; ++k) v[k] = j0 + k < C ? counts[j0 + k] : 0;
        }
        int64_t tot = 0;
#pragma unroll
        for (int k = 0; k < kOffPer; ++k) tot += v[k];
        // inclusive scan of the thread totals over the wave
        int64_t incl = tot;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int64_t up = __shfl_up(incl, o);
            if (lane >= o) incl += up;
        }
        if (lane == 63) wtot[wave] = incl;
        __syncthreads();
        int64_t before = carry;
        for (int w = 0; w < wave; ++w) before += wtot[w];
        if (threadIdx.x == 1023) carry_s = before + incl;
        int64_t run = before + incl - tot;
        if (j0 + kOffPer <= C && ((j0 & 1) == 0)) {
#pragma unroll
            for (int k = 0; k < kOffPer; k += 2) {
                longlong2 u;
                u.x = run;
                u.y = run + v[k];
                run += v[k] + v[k + 1];
                *reinterpret_cast<longlong2 *>(offsets + j0 + k) = u;
            }
        } else {
#pragma unroll
            for (int k = 0; k < kOffPer; ++k) {
                if (j0 + k < C) offsets[j0 + k] = run;
                run += v[k];
            }
        }
        __syncthreads();
        carry = carry_s;
    }
    if (threadIdx.x == 0) offsets[C] = carry;
}

constexpr int kLinearDupMax = 128;

__global__ __launch_bounds__(kBuildThreads) void scatter_kernel(
    const int32_t *__restrict__ labels, int64_t N, int64_t R, int64_t C, int nblocks, int nslices,
    const uint32_t *__restrict__ colpre, const int64_t *__restrict__ offsets,
    uint32_t *__restrict__ perm)
{
    __shared__ uint32_t cur[kSlice];       // next free position per list of the slice
    __shared__ uint32_t mult[kSlice / 2];  // 16-bit multiplicities in the sub-chunk
    __shared__ uint32_t dupk[kSub];        // (rel << 12) | row-in-sub-chunk of repeated labels
    __shared__ uint16_t rnk[kSub];
    __shared__ uint32_t ndup;
    int b, s;
    decode_block(blockIdx.x, nblocks, nslices, b, s);
    const int64_t j0 = (int64_t)s * kSlice;
    const int width = (int)min((int64_t)kSlice, C - j0);
    for (int i = threadIdx.x; i < width; i += blockDim.x)
        cur[i] = (uint32_t)(offsets[j0 + i] + colpre[(int64_t)b * C + j0 + i]);
    for (int i = threadIdx.x; i < kSlice / 2; i += blockDim.x) mult[i] = 0;
    if (threadIdx.x == 0) ndup = 0;
    __syncthreads();

    const int64_t r0 = (int64_t)b * R;
    const int64_t r1 = min(N, r0 + R);
    const int t4 = 4 * threadIdx.x;
    // labels of the next sub-chunk are loaded one sub-chunk ahead
    int4 nxt = load_labels4(labels, r0 + t4, r1);
    for (int64_t base = r0; base < r1; base += kSub) {
        const int64_t r = base + t4;
        const int4 cur4 = nxt;
        if (base + kSub < r1) nxt = load_labels4(labels, base + kSub + t4, r1);
        const int l[4] = {cur4.x, cur4.y, cur4.z, cur4.w};
        uint32_t rel[4], old[4], m[4];
        bool mine[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            rel[e] = (uint32_t)((int64_t)l[e] - j0);
            mine[e] = l[e] >= 0 && rel[e] < (uint32_t)width;
            if (mine[e]) {
                old[e] = atomicAdd(&cur[rel[e]], 1u);
                atomicAdd(&mult[rel[e] >> 1], 1u << (16 * (rel[e] & 1)));
            }
        }
        __syncthreads();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (mine[e]) {
                m[e] = (mult[rel[e] >> 1] >> (16 * (rel[e] & 1))) & 0xFFFFu;
                if (m[e] > 1) dupk[atomicAdd(&ndup, 1u)] = (rel[e] << 12) | (uint32_t)(t4 + e);
            }
        }
        __syncthreads();
        const int nd = (int)ndup;
        if (nd > 0) {
            if (nd <= kLinearDupMax) {
                for (int i = threadIdx.x; i < nd; i += blockDim.x) {
                    const uint32_t k = dupk[i];
                    int rank = 0;
                    for (int i2 = 0; i2 < nd; ++i2) {
                        const uint32_t k2 = dupk[i2];
                        rank += ((k2 >> 12) == (k >> 12) && k2 < k) ? 1 : 0;
                    }
                    rnk[k & 0xFFFu] = (uint16_t)rank;
                }
            } else {
                int P = 1;
                while (P < nd) P <<= 1;
                for (int i = nd + threadIdx.x; i < P; i += blockDim.x) dupk[i] = 0xFFFFFFFFu;
                __syncthreads();
                for (int k = 2; k <= P; k <<= 1) {
                    for (int j = k >> 1; j > 0; j >>= 1) {
                        for (int i = threadIdx.x; i < P; i += blockDim.x) {
                            const int ixj = i ^ j;
                            if (ixj > i) {
                                const uint32_t a = dupk[i], c = dupk[ixj];
                                if (((i & k) == 0) == (a > c)) {
                                    dupk[i] = c;
                                    dupk[ixj] = a;
                                }
                            }
                        }
                        __syncthreads();
                    }
                }
                for (int i = threadIdx.x; i < nd; i += blockDim.x) {
                    const uint32_t k = dupk[i];
                    const uint32_t lo_key = k & ~0xFFFu;
                    int lo = 0, hi = i;  // first index whose key >= lo_key
                    while (lo < hi) {
                        const int mid = (lo + hi) >> 1;
                        if (dupk[mid] < lo_key) lo = mid + 1; else hi = mid;
                    }
                    rnk[k & 0xFFFu] = (uint16_t)(i - lo);
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (mine[e]) {
                const uint32_t pos = m[e] == 1 ? old[e] : cur[rel[e]] - m[e] + rnk[t4 + e];
                perm[pos] = (uint32_t)(r + e);
            }
        }
        __syncthreads();
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (mine[e]) mult[rel[e] >> 1] = 0;
        if (threadIdx.x == 0) ndup = 0;
        __syncthreads();
    }
}

}  // namespace

BuildPlan plan_build(int64_t N, int64_t C, int num_cus, int max_blocks)
{
    BuildPlan p;
    p.N = N;
    p.C = C;
    p.nslices = (int)((C + kSlice - 1) / kSlice);
    // one workgroup per CU in total: nblocks * nslices ~ num_cus
    int64_t nb = num_cus / p.nslices;
    if (max_blocks > 0 && nb > max_blocks) nb = max_blocks;
    if (nb >= 8) nb -= nb % 8;
    if (nb < 1) nb = 1;
    int64_t R = (N + nb - 1) / nb;
    R = ((R + kSub - 1) / kSub) * kSub;
    if (R < kSub) R = kSub;
    p.R = R;
    p.nblocks = (int)((N + R - 1) / R);
    if (p.nblocks < 1) p.nblocks = 1;
    return p;
}

size_t build_scratch_bytes(const BuildPlan &p)
{
    return (size_t)p.nblocks * (size_t)p.C * sizeof(uint32_t);
}

hipError_t launch_build_hist(const BuildPlan &p, const int32_t *labels, uint32_t *cntmat,
                             hipStream_t s)
{
    hipLaunchKernelGGL(hist_kernel, dim3(p.nblocks * p.nslices), dim3(kBuildThreads), 0, s, labels,
                       p.N, p.R, p.C, p.nblocks, p.nslices, cntmat);
    return hipGetLastError();
}

hipError_t launch_build_scan(const BuildPlan &p, uint32_t *cntmat, int64_t *counts, int64_t *offsets,
                             hipStream_t s)
{
    int g = (int)((p.C + 255) / 256);
    if (g > 4096) g = 4096;
    hipLaunchKernelGGL(colscan_kernel, dim3(g), dim3(256), 0, s, cntmat, p.C, p.nblocks, counts);
    hipLaunchKernelGGL(offsets_kernel, dim3(1), dim3(1024), 0, s, counts, p.C, offsets);
    return hipGetLastError();
}

hipError_t launch_offsets(const int64_t *counts, int64_t C, int64_t *offsets, hipStream_t st)
{
    hipLaunchKernelGGL(offsets_kernel, dim3(1), dim3(1024), 0, st, counts, C, offsets);
    return hipGetLastError();
}

hipError_t launch_build_scatter(const BuildPlan &p, const int32_t *labels, const uint32_t *cntmat,
                                const int64_t *offsets, uint32_t *perm, hipStream_t s)
{
    if (p.N > 0)
        hipLaunchKernelGGL(scatter_kernel, dim3(p.nblocks * p.nslices), dim3(kBuildThreads), 0, s,
                           labels, p.N, p.R, p.C, p.nblocks, p.nslices, cntmat, offsets, perm);
    return hipGetLastError();
}

}  // namespace ivf

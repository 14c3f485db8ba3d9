// Inverted-list build for C <= 65,536 lists as a two-level most-significant-
// digit radix partition (gfx950). Produces the same counts, offsets and stable
// permutation as the single-pass build in lists.hip (the cluster-major layout
// with per-list offset, length and vector ids, Sec. "System Architecture"),
// but writes its outputs as contiguous runs instead of scattered 4-byte
// stores.
//
// Level 0: digit = label >> 8 (at most 256 buckets). Rows are cut into blocks;
//   hist0 counts each block's digits, scan0 turns the counts into each block's
//   start per digit (bucket-major), scatter0 moves (row id, label & 255) into
//   the bucket regions of two scratch arrays, keeping row order inside each
//   bucket.
// Level 1: digit = label & 255 inside each bucket region. plan1 cuts every
//   region into sub-blocks; hist1 counts their digits; scan1 gives the
//   per-list counts and each sub-block's start per digit; the offsets are the
//   exclusive scan of the counts; scatter1 writes the row ids into the
//   permutation.
// Inside a block, rows are taken in 4,096-row tiles: wave w ranks its 1,024
// rows column by column (64 consecutive rows per column) with an LDS
// match-any on the digit, the 4 waves' digit counts are combined with a prefix, the tile
// is staged in LDS in (digit, row) order and written out so that consecutive
// threads store consecutive addresses of one digit run. Both levels keep row
// order within a digit, so the final order is (label, row id).
#include "ivf_internal.h"

#include <algorithm>

namespace ivf {
namespace {

constexpr int kRThreads = 256;           // 4 waves
constexpr int kRTile = 4096;             // rows per tile of level 1
constexpr int kRTile0 = 8192;            // rows per tile of level 0 (longer runs per digit)

template <bool FIRST>
constexpr int tile_rows()
{
    return FIRST ? kRTile0 : kRTile;
}

// Exclusive scan of v over the 256 threads of the block; returns the prefix.
__device__ __forceinline__ uint32_t block_exscan256(uint32_t v, uint32_t *wsum)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t incl = v;
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t up = __shfl_up(incl, o);
        if (lane >= o) incl += up;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    uint32_t before = 0;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    __syncthreads();
    return before + incl - v;
}

template <int RT>
struct TileLds {
    unsigned long long peers[4][256];  // per-wave match-any scratch (lane bits per digit)
    uint32_t wcnt[4][256];   // per-wave digit counts, then their exclusive prefix
    uint32_t start[256];     // digit start inside the tile
    uint32_t gbase[256];     // global start of this tile's digit run
    uint32_t run[256];       // block running offset per digit
    uint32_t wsum[4];
    uint32_t sid[RT];        // staged row ids
    uint8_t slo[RT];         // staged low bytes (level 0)
    uint8_t sdig[RT];        // staged digits
};

// A tile's inputs, loaded one tile ahead: row r = base + wave*RT/4 + e*64 + lane.
template <int RT>
struct TileIn {
    static constexpr int kItems = RT / kRThreads;  // rows per thread
    uint32_t v[kItems];        // level 0: label; level 1: row id
    uint32_t lo4[kItems / 4];  // level 1: low bytes, four per word
};

template <bool FIRST, bool FULL, int RT = tile_rows<FIRST>()>
__device__ __forceinline__ void load_tile(TileIn<RT> &in, int64_t base, int64_t end,
                                          const int32_t *__restrict__ labels,
                                          const uint32_t *__restrict__ in_ids,
                                          const uint8_t *__restrict__ in_lo)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int e = 0; e < TileIn<RT>::kItems / 4; ++e) in.lo4[e] = 0;
#pragma unroll
    for (int e = 0; e < TileIn<RT>::kItems; ++e) {
        const int64_t r = base + wave * (RT / 4) + e * 64 + lane;
        const bool ok = FULL || r < end;
        if (FIRST) {
            in.v[e] = ok ? (uint32_t)labels[r] : 0xFFFFFFFFu;
        } else {
            in.v[e] = ok ? in_ids[r] : 0u;
            in.lo4[e / 4] |= (ok ? (uint32_t)in_lo[r] : 0u) << (8 * (e % 4));
        }
    }
}

// One tile: rank, stage and write. Level 0 (FIRST): the digit is label >> 8,
// the payload is (row id, label & 255). Level 1: the digit is the stored low
// byte, the payload is the stored row id.
template <bool FIRST, bool FULL, int RT = tile_rows<FIRST>()>
__device__ void radix_tile(TileLds<RT> &t, const TileIn<RT> &in, int64_t base, int64_t end, int C,
                           uint32_t *__restrict__ out_ids, uint8_t *__restrict__ out_lo)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    constexpr int kItems = TileIn<RT>::kItems;
    uint32_t dp[kItems];  // (digit << 16) | position in the wave's run, 0xFFFF = none
    // rank column by column
#pragma unroll
    for (int e = 0; e < kItems; ++e) {
        const int64_t r = base + wave * (RT / 4) + e * 64 + lane;
        bool valid = FULL || r < end;
        uint32_t d;
        if (FIRST) {
            const int32_t l = (int32_t)in.v[e];
            valid = valid && l >= 0 && l < C;  // labels outside [0, C) are skipped
            d = valid ? ((uint32_t)l >> 8) : 0u;
        } else {
            d = (in.lo4[e / 4] >> (8 * (e % 4))) & 0xFFu;
        }
        // lanes of this wave with the same digit: every lane ORs its bit into
        // peers[wave][d], reads the union back, and the group leader clears it
        uint16_t p = 0xFFFFu;
        if (valid) {
            atomicOr(&t.peers[wave][d], 1ull << lane);
            const uint64_t m = t.peers[wave][d];
            const uint32_t b = t.wcnt[wave][d];
            p = (uint16_t)(b + (uint32_t)__popcll(m & lt));
            if ((m & lt) == 0) {
                t.wcnt[wave][d] = b + (uint32_t)__popcll(m);
                t.peers[wave][d] = 0ull;
            }
        }
        dp[e] = (d << 16) | p;
    }
    __syncthreads();
    // combine the waves: per digit (one thread per digit)
    {
        const int d = threadIdx.x;
        const uint32_t c0 = t.wcnt[0][d], c1 = t.wcnt[1][d], c2 = t.wcnt[2][d], c3 = t.wcnt[3][d];
        const uint32_t tot = c0 + c1 + c2 + c3;
        t.wcnt[0][d] = 0;
        t.wcnt[1][d] = c0;
        t.wcnt[2][d] = c0 + c1;
        t.wcnt[3][d] = c0 + c1 + c2;
        const uint32_t st = block_exscan256(tot, t.wsum);
        t.start[d] = st;
        t.gbase[d] = t.run[d];
        t.run[d] += tot;
    }
    __syncthreads();
    // stage in (digit, row) order
#pragma unroll
    for (int e = 0; e < kItems; ++e) {
        if ((dp[e] & 0xFFFFu) != 0xFFFFu) {
            const uint32_t d = dp[e] >> 16;
            const uint32_t li = t.start[d] + t.wcnt[wave][d] + (dp[e] & 0xFFFFu);
            t.sid[li] = FIRST ? (uint32_t)(base + wave * (RT / 4) + e * 64 + lane) : in.v[e];
            t.sdig[li] = (uint8_t)d;
            if (FIRST) t.slo[li] = (uint8_t)(in.v[e] & 0xFFu);
        }
    }
    __syncthreads();
    // write the runs: consecutive staged entries of a digit go to consecutive
    // addresses
    const uint32_t total = t.start[255] + (t.run[255] - t.gbase[255]);
#pragma unroll
    for (int e = 0; e < kItems; ++e) {
        const uint32_t i = threadIdx.x + e * kRThreads;
        if (i < total) {
            const uint32_t d = t.sdig[i];
            const uint32_t g = t.gbase[d] + (i - t.start[d]);
            out_ids[g] = t.sid[i];
            if (FIRST) out_lo[g] = t.slo[i];
        }
    }
    // the next tile counts from zero (nothing reads wcnt in this phase; the
    // barrier below orders the reset before the next tile's ranking)
    t.wcnt[0][threadIdx.x] = t.wcnt[1][threadIdx.x] = t.wcnt[2][threadIdx.x] = t.wcnt[3][threadIdx.x] = 0;
    __syncthreads();
}

template <int RT>
__device__ __forceinline__ void init_run(TileLds<RT> &t)
{
    for (int i = threadIdx.x; i < 256; i += kRThreads) {
        t.wcnt[0][i] = t.wcnt[1][i] = t.wcnt[2][i] = t.wcnt[3][i] = 0;
        t.peers[0][i] = t.peers[1][i] = t.peers[2][i] = t.peers[3][i] = 0ull;
    }
}

// ---- level 0 ----------------------------------------------------------------

__global__ __launch_bounds__(kRThreads) void hist0_kernel(const int32_t *__restrict__ labels, int64_t N,
                                                          int64_t R0, int C, int nblocks,
                                                          uint32_t *__restrict__ cnt0)
{
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t r0 = (int64_t)blockIdx.x * R0, r1 = min(N, r0 + R0);  // r0 % 4 == 0
    const int64_t step = 4 * (int64_t)kRThreads;
    for (int64_t r = r0 + 4 * (int64_t)threadIdx.x; r < r1; r += 4 * step) {
        int l[16];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t q = r + u * step;
            if (q + 3 < r1) {
                const int4 v = *reinterpret_cast<const int4 *>(labels + q);
                l[4 * u] = v.x;
                l[4 * u + 1] = v.y;
                l[4 * u + 2] = v.z;
                l[4 * u + 3] = v.w;
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) l[4 * u + k] = q + k < r1 ? labels[q + k] : -1;
            }
        }
#pragma unroll
        for (int k = 0; k < 16; ++k)
            if (l[k] >= 0 && l[k] < C) atomicAdd(&h[(uint32_t)l[k] >> 8], 1u);
    }
    __syncthreads();
    cnt0[(int64_t)threadIdx.x * nblocks + blockIdx.x] = h[threadIdx.x];  // digit-major
}

// Digit d (one workgroup): cnt0[d][b] <- exclusive prefix over the blocks;
// tot0[d] = the digit's total.
__global__ __launch_bounds__(kRThreads) void scan0_kernel(uint32_t *__restrict__ cnt0, int nblocks,
                                                          uint32_t *__restrict__ tot0)
{
    __shared__ uint32_t wsum[4];
    __shared__ uint32_t carry;
    const int d = blockIdx.x;
    uint32_t *row = cnt0 + (int64_t)d * nblocks;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int b0 = 0; b0 < nblocks; b0 += kRThreads) {
        const int b = b0 + threadIdx.x;
        const uint32_t v = b < nblocks ? row[b] : 0u;
        const uint32_t ex = block_exscan256(v, wsum);
        const uint32_t c = carry;
        if (b < nblocks) row[b] = c + ex;
        __syncthreads();
        if (threadIdx.x == kRThreads - 1) carry = c + ex + v;
        __syncthreads();
    }
    if (threadIdx.x == 0) tot0[d] = carry;
}

// astart[d] = start of bucket d (exclusive scan of the digit totals),
// astart[256] = number of valid rows.
__global__ __launch_bounds__(kRThreads) void starts0_kernel(const uint32_t *__restrict__ tot0,
                                                            uint32_t *__restrict__ astart)
{
    __shared__ uint32_t wsum[4];
    const int d = threadIdx.x;
    const uint32_t v = tot0[d];
    const uint32_t st = block_exscan256(v, wsum);
    astart[d] = st;
    if (d == 255) astart[256] = st + v;
}

__global__ __launch_bounds__(kRThreads, 2) void scatter0_kernel(const int32_t *__restrict__ labels, int64_t N,
                                                             int64_t R0, int C, int nblocks,
                                                             const uint32_t *__restrict__ base0,
                                                             const uint32_t *__restrict__ astart,
                                                             uint32_t *__restrict__ tmp_ids,
                                                             uint8_t *__restrict__ tmp_lo)
{
    constexpr int RT = kRTile0;
    __shared__ TileLds<RT> t;
    init_run(t);
    t.run[threadIdx.x] = astart[threadIdx.x] + base0[(int64_t)threadIdx.x * nblocks + blockIdx.x];
    __syncthreads();
    const int64_t r0 = (int64_t)blockIdx.x * R0, r1 = min(N, r0 + R0);
    TileIn<RT> cur, nxt;
    if (r0 + RT <= r1) load_tile<true, true>(cur, r0, r1, labels, nullptr, nullptr);
    else load_tile<true, false>(cur, r0, r1, labels, nullptr, nullptr);
    for (int64_t base = r0; base < r1; base += RT) {
        const int64_t nb = base + RT;
        if (nb + RT <= r1) load_tile<true, true>(nxt, nb, r1, labels, nullptr, nullptr);
        else if (nb < r1) load_tile<true, false>(nxt, nb, r1, labels, nullptr, nullptr);
        if (base + RT <= r1)
            radix_tile<true, true>(t, cur, base, base + RT, C, tmp_ids, tmp_lo);
        else
            radix_tile<true, false>(t, cur, base, r1, C, tmp_ids, tmp_lo);
        cur = nxt;
    }
}

// ---- level 1 ----------------------------------------------------------------

// Sub-blocks of R1 rows inside every bucket region: sbstart[d] = index of the
// first sub-block of bucket d, sbstart[256] = their number.
__global__ __launch_bounds__(kRThreads) void plan1_kernel(const uint32_t *__restrict__ astart, int64_t R1,
                                                          uint32_t *__restrict__ sbstart)
{
    __shared__ uint32_t wsum[4];
    const int d = threadIdx.x;
    const uint32_t sz = astart[d + 1] - astart[d];
    const uint32_t n = (uint32_t)((sz + R1 - 1) / R1);
    const uint32_t st = block_exscan256(n, wsum);
    sbstart[d] = st;
    if (d == 255) sbstart[256] = st + n;
}

// Sub-block w -> (bucket, row range) by binary search over sbstart.
__device__ __forceinline__ bool locate_sub(const uint32_t *__restrict__ sbstart,
                                           const uint32_t *__restrict__ astart, int64_t R1, int w,
                                           int &bucket, int64_t &lo, int64_t &hi)
{
    if ((uint32_t)w >= sbstart[256]) return false;
    int a = 0, b = 256;  // last bucket with sbstart[bucket] <= w
    while (b - a > 1) {
        const int m = (a + b) >> 1;
        if (sbstart[m] <= (uint32_t)w) a = m; else b = m;
    }
    // empty buckets share their sbstart with the next bucket: move to the
    // bucket that actually owns sub-block w
    while (a < 255 && sbstart[a + 1] <= (uint32_t)w) ++a;
    bucket = a;
    const int64_t k = w - sbstart[a];
    lo = (int64_t)astart[a] + k * R1;
    hi = min((int64_t)astart[a + 1], lo + R1);
    return true;
}

__global__ __launch_bounds__(kRThreads) void hist1_kernel(const uint8_t *__restrict__ tmp_lo,
                                                          const uint32_t *__restrict__ astart,
                                                          const uint32_t *__restrict__ sbstart, int64_t R1,
                                                          uint32_t *__restrict__ cnt1)
{
    __shared__ uint32_t h[4][256];  // one histogram per wave
    int bucket;
    int64_t lo, hi;
    if (!locate_sub(sbstart, astart, R1, blockIdx.x, bucket, lo, hi)) return;
    const int wave = threadIdx.x >> 6;
    for (int w = 0; w < 4; ++w) h[w][threadIdx.x] = 0;
    __syncthreads();
    // 16-byte loads over the aligned middle, single bytes at the two ends
    const int64_t a0 = min(hi, (lo + 15) & ~(int64_t)15);
    const int64_t a1 = max(a0, hi & ~(int64_t)15);
    for (int64_t r = lo + threadIdx.x; r < a0; r += kRThreads) atomicAdd(&h[wave][tmp_lo[r]], 1u);
    for (int64_t r = a1 + threadIdx.x; r < hi; r += kRThreads) atomicAdd(&h[wave][tmp_lo[r]], 1u);
    const uint4 *v = reinterpret_cast<const uint4 *>(tmp_lo + a0);
    const int64_t n16 = (a1 - a0) >> 4;
    for (int64_t i = threadIdx.x; i < n16; i += kRThreads) {
        const uint4 w4 = v[i];
        const uint32_t ws[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int b = 0; b < 4; ++b) atomicAdd(&h[wave][(ws[k] >> (8 * b)) & 0xFFu], 1u);
    }
    __syncthreads();
    cnt1[(int64_t)blockIdx.x * 256 + threadIdx.x] = h[0][threadIdx.x] + h[1][threadIdx.x] + h[2][threadIdx.x] +
                                                    h[3][threadIdx.x];
}

// Per bucket b and low byte d: prefix of cnt1 over the bucket's sub-blocks;
// counts[b*256 + d] = the list length (for lists < C).
__global__ __launch_bounds__(kRThreads) void scan1_kernel(uint32_t *__restrict__ cnt1,
                                                          const uint32_t *__restrict__ sbstart, int C,
                                                          int64_t *__restrict__ counts)
{
    const int b = blockIdx.x, d = threadIdx.x;
    uint32_t run = 0;
    for (uint32_t w = sbstart[b]; w < sbstart[b + 1]; ++w) {
        const uint32_t v = cnt1[(int64_t)w * 256 + d];
        cnt1[(int64_t)w * 256 + d] = run;
        run += v;
    }
    const int j = b * 256 + d;
    if (j < C) counts[j] = run;
}

__global__ __launch_bounds__(kRThreads) void scatter1_kernel(const uint32_t *__restrict__ tmp_ids,
                                                             const uint8_t *__restrict__ tmp_lo,
                                                             const uint32_t *__restrict__ astart,
                                                             const uint32_t *__restrict__ sbstart,
                                                             int64_t R1, const uint32_t *__restrict__ base1,
                                                             const int64_t *__restrict__ offsets, int C,
                                                             uint32_t *__restrict__ perm)
{
    __shared__ TileLds<kRTile> t;
    int bucket;
    int64_t lo, hi;
    if (!locate_sub(sbstart, astart, R1, blockIdx.x, bucket, lo, hi)) return;
    init_run(t);
    {
        const int d = threadIdx.x;
        const int j = bucket * 256 + d;
        t.run[d] = j < C ? (uint32_t)offsets[j] + base1[(int64_t)blockIdx.x * 256 + d] : 0u;
    }
    __syncthreads();
    TileIn<kRTile> cur, nxt;
    if (lo + kRTile <= hi) load_tile<false, true>(cur, lo, hi, nullptr, tmp_ids, tmp_lo);
    else load_tile<false, false>(cur, lo, hi, nullptr, tmp_ids, tmp_lo);
    for (int64_t base = lo; base < hi; base += kRTile) {
        const int64_t nb = base + kRTile;
        if (nb + kRTile <= hi) load_tile<false, true>(nxt, nb, hi, nullptr, tmp_ids, tmp_lo);
        else if (nb < hi) load_tile<false, false>(nxt, nb, hi, nullptr, tmp_ids, tmp_lo);
        if (base + kRTile <= hi)
            radix_tile<false, true>(t, cur, base, base + kRTile, C, perm, nullptr);
        else
            radix_tile<false, false>(t, cur, base, hi, C, perm, nullptr);
        cur = nxt;
    }
}

}  // namespace

RadixPlan plan_radix(int64_t N, int64_t C, int num_cus)
{
    // Blocks of at most 16 tiles: many more workgroups than resident slots,
    // so the last round is short; each digit still gets long write runs
    // (about 256 rows per digit per block at the largest block size).
    RadixPlan p;
    p.N = N;
    p.C = C;
    int64_t R0 = (N + 8 * (int64_t)num_cus - 1) / (8 * (int64_t)num_cus);
    R0 = (R0 + kRTile0 - 1) / kRTile0 * kRTile0;
    R0 = std::min<int64_t>(std::max<int64_t>(R0, kRTile0), 16 * (int64_t)kRTile0);
    p.R0 = R0;
    p.nblocks0 = (int)std::max<int64_t>(1, (N + R0 - 1) / R0);
    p.R1 = std::min<int64_t>(R0, 16 * (int64_t)kRTile);
    p.max_sub1 = (int)((N + p.R1 - 1) / p.R1) + 256;
    return p;
}

size_t radix_scratch_bytes(const RadixPlan &p)
{
    // cnt0 [nblocks0][256], astart [257], sbstart [257], cnt1 [max_sub1][256],
    // tmp ids [N], tmp low bytes [N]
    const size_t a = 256;
    auto up = [&](size_t x) { return (x + a - 1) / a * a; };
    return up((size_t)p.nblocks0 * 256 * 4) + up(256 * 4) + up(257 * 4) + up(257 * 4) +
           up((size_t)p.max_sub1 * 256 * 4) + up((size_t)p.N * 4) + up((size_t)p.N) + a;
}

RadixScratch carve_radix(const RadixPlan &p, void *base)
{
    const size_t a = 256;
    auto up = [&](size_t x) { return (x + a - 1) / a * a; };
    char *c = (char *)base;
    RadixScratch s;
    s.cnt0 = (uint32_t *)c;
    c += up((size_t)p.nblocks0 * 256 * 4);
    s.tot0 = (uint32_t *)c;
    c += up(256 * 4);
    s.astart = (uint32_t *)c;
    c += up(257 * 4);
    s.sbstart = (uint32_t *)c;
    c += up(257 * 4);
    s.cnt1 = (uint32_t *)c;
    c += up((size_t)p.max_sub1 * 256 * 4);
    s.tmp_ids = (uint32_t *)c;
    c += up((size_t)p.N * 4);
    s.tmp_lo = (uint8_t *)c;
    return s;
}

hipError_t launch_radix_level0(const RadixPlan &p, const int32_t *labels, const RadixScratch &s,
                               hipStream_t st)
{
    hipLaunchKernelGGL(hist0_kernel, dim3(p.nblocks0), dim3(kRThreads), 0, st, labels, p.N, p.R0, (int)p.C,
                       p.nblocks0, s.cnt0);
    hipLaunchKernelGGL(scan0_kernel, dim3(256), dim3(kRThreads), 0, st, s.cnt0, p.nblocks0, s.tot0);
    hipLaunchKernelGGL(starts0_kernel, dim3(1), dim3(kRThreads), 0, st, s.tot0, s.astart);
    hipLaunchKernelGGL(scatter0_kernel, dim3(p.nblocks0), dim3(kRThreads), 0, st, labels, p.N, p.R0, (int)p.C,
                       p.nblocks0, s.cnt0, s.astart, s.tmp_ids, s.tmp_lo);
    return hipGetLastError();
}

hipError_t launch_radix_level1_counts(const RadixPlan &p, const RadixScratch &s, int64_t *counts,
                                      hipStream_t st)
{
    hipLaunchKernelGGL(plan1_kernel, dim3(1), dim3(kRThreads), 0, st, s.astart, p.R1, s.sbstart);
    hipLaunchKernelGGL(hist1_kernel, dim3(p.max_sub1), dim3(kRThreads), 0, st, s.tmp_lo, s.astart, s.sbstart,
                       p.R1, s.cnt1);
    const int nb = (int)((p.C + 255) / 256);
    hipLaunchKernelGGL(scan1_kernel, dim3(nb), dim3(kRThreads), 0, st, s.cnt1, s.sbstart, (int)p.C, counts);
    return hipGetLastError();
}

hipError_t launch_radix_level1_scatter(const RadixPlan &p, const RadixScratch &s, const int64_t *offsets,
                                       uint32_t *perm, hipStream_t st)
{
    hipLaunchKernelGGL(scatter1_kernel, dim3(p.max_sub1), dim3(kRThreads), 0, st, s.tmp_ids, s.tmp_lo,
                       s.astart, s.sbstart, p.R1, s.cnt1, offsets, (int)p.C, perm);
    return hipGetLastError();
}

}  // namespace ivf

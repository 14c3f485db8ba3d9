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
// Inside a block, rows are taken in tiles (8,192 rows at level 0, 4,096 at
// level 1): wave w ranks its quarter column by column (64 consecutive rows per
// column) with an LDS match-any on the digit, keeping cumulative per-wave
// digit counts; after one workgroup barrier every wave reads all four waves'
// counts and derives the tile's digit starts itself (no further barrier), the
// tile is staged in LDS in (digit, row) order and, after a second barrier,
// written out so that consecutive threads store consecutive addresses of one
// digit run. Both levels keep row order within a digit, so the final order is
// (label, row id).
#include "ivf_internal.h"

#include <algorithm>

namespace ivf {
namespace {

constexpr int kRThreads = 256;           // 4 waves (histogram and scan kernels)
// Partition kernels: one workgroup of kPW waves per CU, each wave ranking
// kItems0 / kItems1 columns of 64 rows per tile. Long tiles give long write
// runs per digit, and few blocks in flight keep the runs being filled (about
// 256 per block) within the L2 until their cache lines are complete.
constexpr int kPW = 12;
constexpr int kRTile0 = kPW * 64 * 32;   // rows per tile of level 0 (24,576)
constexpr int kRTile = kPW * 64 * 16;    // rows per tile of level 1 (12,288)
constexpr int kPosBits = 15;             // tile position bits of a staged level-0 entry
static_assert(kRTile0 <= (1 << kPosBits), "tile positions must fit the staged entry");

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

// LDS of one partition workgroup. Ranking state is per wave; the combine is
// done by every wave for itself (each lane owns digits 4 lane .. 4 lane + 3),
// so a tile needs two workgroup barriers: after the ranking (the digit counts
// of all waves are complete) and after the staging (the tile is in LDS).
template <bool FIRST, int RT, int W>
struct TileLds {
    unsigned long long peers[W][256];  // per-wave match-any scratch (lane bits per digit), zero between columns
    uint32_t wcnt[W][256];   // entries of each digit ranked by each wave in this tile
    uint32_t wbase[W][256];  // wave w: staged index of its first digit-d entry of the tile
    uint32_t woff[W][256];   // wave w's copy: global index of staged index 0 of digit d (mod 2^32)
    uint32_t sw[RT];         // staged entries: level 0 (label << kPosBits | tile position), level 1 row id
    uint8_t sdig[FIRST ? 4 : RT];  // level 1: staged digits
};

// A tile's inputs: row r = base + wave*RT/W + e*64 + lane.
template <int RT, int W>
struct TileIn {
    static constexpr int kItems = RT / (W * 64);  // rows per thread
    uint32_t v[kItems];        // level 0: label; level 1: row id
    uint32_t lo4[kItems / 4];  // level 1: low bytes, four per word
};

template <bool FIRST, bool FULL, int RT, int W>
__device__ __forceinline__ void load_tile(TileIn<RT, W> &in, int64_t base, int64_t end,
                                          const int32_t *__restrict__ labels,
                                          const uint32_t *__restrict__ in_ids,
                                          const uint8_t *__restrict__ in_lo)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int e = 0; e < TileIn<RT, W>::kItems / 4; ++e) in.lo4[e] = 0;
#pragma unroll
    for (int e = 0; e < TileIn<RT, W>::kItems; ++e) {
        const int64_t r = base + wave * (RT / W) + e * 64 + lane;
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
// byte, the payload is the stored row id. Outputs are written only below
// n_out. `next` loads the following tile into `in` once the tile no longer
// needs it (after the ranking at level 0, after the staging at level 1), so
// its loads overlap the rest of the tile.
template <bool FIRST, bool FULL, int RT, int W, class Next>
__device__ void radix_tile(TileLds<FIRST, RT, W> &t, uint32_t (&run)[4], TileIn<RT, W> &in, int64_t base, int64_t end,
                           int C, uint32_t n_out, uint32_t *__restrict__ out_ids, uint8_t *__restrict__ out_lo,
                           Next &&next)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    constexpr int kItems = TileIn<RT, W>::kItems;
    // (label << 16 | rank) at level 0, (digit << 16 | rank) at level 1, where
    // rank is the entry's position among the wave's digit-d entries of the
    // tile; ~0 = none
    uint32_t dp[kItems];
    // this wave's counts start from zero (every wave has read them in the
    // previous tile's combine, before its second barrier)
    *reinterpret_cast<uint4 *>(&t.wcnt[wave][4 * lane]) = make_uint4(0u, 0u, 0u, 0u);
    // rank column by column: the lanes of a column with the same digit OR
    // their bits into peers[wave][d] and read the union back; the group's
    // lowest lane adds the group to the wave's count and clears the entry.
    // (A wave's LDS instructions execute in order, for all lanes at once.)
#pragma unroll
    for (int e = 0; e < kItems; ++e) {
        const int64_t r = base + wave * (RT / W) + e * 64 + lane;
        bool valid = FULL || r < end;
        uint32_t d, key;
        if (FIRST) {
            const int32_t l = (int32_t)in.v[e];
            valid = valid && l >= 0 && l < C;  // labels outside [0, C) are skipped
            d = valid ? ((uint32_t)l >> 8) : 0u;
            key = (uint32_t)l;
        } else {
            d = (in.lo4[e / 4] >> (8 * (e % 4))) & 0xFFu;
            key = d;
        }
        uint32_t rk = 0xFFFFFFFFu;
        if (valid) {
            atomicOr(&t.peers[wave][d], 1ull << lane);
            const uint64_t m = t.peers[wave][d];
            const uint32_t b = t.wcnt[wave][d];
            rk = (key << 16) | (b + (uint32_t)__popcll(m & lt));
            if ((m & lt) == 0) {
                t.wcnt[wave][d] = b + (uint32_t)__popcll(m);
                t.peers[wave][d] = 0ull;
            }
        }
        dp[e] = rk;
    }
    if (FIRST) next();
    __syncthreads();
    // combine, in every wave: the tile's count of each digit, their exclusive
    // scan over the digits, this wave's staging base per digit and the global
    // offsets
    uint32_t total;
    {
        uint32_t tot[4] = {0u, 0u, 0u, 0u}, before[4] = {0u, 0u, 0u, 0u}, s = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const uint4 v = *reinterpret_cast<const uint4 *>(&t.wcnt[w][4 * lane]);
            const uint32_t c[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                tot[j] += c[j];
                before[j] += w < wave ? c[j] : 0u;
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) s += tot[j];
        uint32_t incl = s;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t up = __shfl_up(incl, o);
            if (lane >= o) incl += up;
        }
        total = __shfl(incl, 63);
        uint32_t st = incl - s;
        uint32_t wb[4], wo[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            wb[j] = st + before[j];
            wo[j] = run[j] - st;
            run[j] += tot[j];
            st += tot[j];
        }
        *reinterpret_cast<uint4 *>(&t.wbase[wave][4 * lane]) = make_uint4(wb[0], wb[1], wb[2], wb[3]);
        *reinterpret_cast<uint4 *>(&t.woff[wave][4 * lane]) = make_uint4(wo[0], wo[1], wo[2], wo[3]);
    }
    // stage in (digit, row) order (wbase of this wave was written by this wave)
#pragma unroll
    for (int e = 0; e < kItems; ++e) {
        if (dp[e] != 0xFFFFFFFFu) {
            const uint32_t key = dp[e] >> 16;
            const uint32_t d = FIRST ? key >> 8 : key;
            const uint32_t li = t.wbase[wave][d] + (dp[e] & 0xFFFFu);
            if (li < (uint32_t)RT) {
                if (FIRST) {
                    t.sw[li] = (key << kPosBits) | (uint32_t)(wave * (RT / W) + e * 64 + lane);
                } else {
                    t.sw[li] = in.v[e];
                    t.sdig[li] = (uint8_t)d;
                }
            }
        }
    }
    if (!FIRST) next();
    __syncthreads();
    // write the runs: consecutive staged entries of a digit go to consecutive
    // addresses
#pragma unroll 8
    for (int e = 0; e < kItems; ++e) {
        const uint32_t i = threadIdx.x + e * (W * 64);
        if (i < total) {
            const uint32_t w = t.sw[i];
            const uint32_t d = FIRST ? (w >> (kPosBits + 8)) & 0xFFu : t.sdig[i];
            const uint32_t g = t.woff[wave][d] + i;
            if (g < n_out) {
                if (FIRST) {
                    out_ids[g] = (uint32_t)base + (w & ((1u << kPosBits) - 1));
                    out_lo[g] = (uint8_t)(w >> kPosBits);
                } else {
                    out_ids[g] = w;
                }
            }
        }
    }
}

// Zeroes the match-any scratch (the caller's next barrier publishes it).
template <bool FIRST, int RT, int W>
__device__ __forceinline__ void init_block(TileLds<FIRST, RT, W> &t)
{
    for (int i = threadIdx.x; i < W * 256; i += W * 64) (&t.peers[0][0])[i] = 0ull;
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

__global__ __launch_bounds__(kPW * 64) void scatter0_kernel(const int32_t *__restrict__ labels, int64_t N,
                                                             int64_t R0, int C, int nblocks,
                                                             const uint32_t *__restrict__ base0,
                                                             const uint32_t *__restrict__ astart,
                                                             uint32_t *__restrict__ tmp_ids,
                                                             uint8_t *__restrict__ tmp_lo)
{
    constexpr int RT = kRTile0, W = kPW;
    __shared__ TileLds<true, RT, W> t;
    uint32_t run[4];  // running global offsets of this lane's digits 4 lane .. 4 lane + 3
    init_block(t);
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int d = 4 * lane + j;
        run[j] = astart[d] + base0[(int64_t)d * nblocks + blockIdx.x];
    }
    __syncthreads();
    const uint32_t n_out = (uint32_t)N;
    const int64_t r0 = (int64_t)blockIdx.x * R0, r1 = min(N, r0 + R0);
    TileIn<RT, W> cur;
    if (r0 + RT <= r1) load_tile<true, true, RT, W>(cur, r0, r1, labels, nullptr, nullptr);
    else load_tile<true, false, RT, W>(cur, r0, r1, labels, nullptr, nullptr);
    for (int64_t base = r0; base < r1; base += RT) {
        const int64_t nb = base + RT;
        auto next = [&]() {
            if (nb + RT <= r1) load_tile<true, true, RT, W>(cur, nb, r1, labels, nullptr, nullptr);
            else if (nb < r1) load_tile<true, false, RT, W>(cur, nb, r1, labels, nullptr, nullptr);
        };
        if (base + RT <= r1)
            radix_tile<true, true, RT, W>(t, run, cur, base, base + RT, C, n_out, tmp_ids, tmp_lo, next);
        else
            radix_tile<true, false, RT, W>(t, run, cur, base, r1, C, n_out, tmp_ids, tmp_lo, next);
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

__global__ __launch_bounds__(kPW * 64) void scatter1_kernel(const uint32_t *__restrict__ tmp_ids,
                                                             const uint8_t *__restrict__ tmp_lo,
                                                             const uint32_t *__restrict__ astart,
                                                             const uint32_t *__restrict__ sbstart,
                                                             int64_t R1, const uint32_t *__restrict__ base1,
                                                             const int64_t *__restrict__ offsets, int C,
                                                             uint32_t *__restrict__ perm)
{
    constexpr int RT = kRTile, W = kPW;
    __shared__ TileLds<false, RT, W> t;
    int bucket;
    int64_t lo, hi;
    if (!locate_sub(sbstart, astart, R1, blockIdx.x, bucket, lo, hi)) return;
    uint32_t run[4];  // running global offsets of this lane's digits 4 lane .. 4 lane + 3
    init_block(t);
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int d = 4 * lane + j;
        const int l = bucket * 256 + d;
        run[j] = l < C ? (uint32_t)offsets[l] + base1[(int64_t)blockIdx.x * 256 + d] : 0u;
    }
    __syncthreads();
    const uint32_t n_out = astart[256];
    TileIn<RT, W> cur;
    if (lo + RT <= hi) load_tile<false, true, RT, W>(cur, lo, hi, nullptr, tmp_ids, tmp_lo);
    else load_tile<false, false, RT, W>(cur, lo, hi, nullptr, tmp_ids, tmp_lo);
    for (int64_t base = lo; base < hi; base += RT) {
        const int64_t nb = base + RT;
        auto next = [&]() {
            if (nb + RT <= hi) load_tile<false, true, RT, W>(cur, nb, hi, nullptr, tmp_ids, tmp_lo);
            else if (nb < hi) load_tile<false, false, RT, W>(cur, nb, hi, nullptr, tmp_ids, tmp_lo);
        };
        if (base + RT <= hi)
            radix_tile<false, true, RT, W>(t, run, cur, base, base + RT, C, n_out, perm, nullptr, next);
        else
            radix_tile<false, false, RT, W>(t, run, cur, base, hi, C, n_out, perm, nullptr, next);
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
    hipLaunchKernelGGL(scatter0_kernel, dim3(p.nblocks0), dim3(kPW * 64), 0, st, labels, p.N, p.R0, (int)p.C,
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
    hipLaunchKernelGGL(scatter1_kernel, dim3(p.max_sub1), dim3(kPW * 64), 0, st, s.tmp_ids, s.tmp_lo,
                       s.astart, s.sbstart, p.R1, s.cnt1, offsets, (int)p.C, perm);
    return hipGetLastError();
}

}  // namespace ivf

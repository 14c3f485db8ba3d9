// Nearest-centroid screening of uint8 rows on int8 MFMA (gfx950).
//
// The assignment step of Lloyd's iteration and of the base-vector assignment
// (Sec. "Fast Index Construction") needs, per row x, the centroid c of least
// ||x - c||^2. With x' = x - 128 and c' = c - 128 the distance is
// ||x'||^2 + k(c) with k(c) = ||c'||^2 - 2 x'.c', so the nearest centroid is
// the one of least k. Rows are integers in [0, 255], so x' is exact in int8;
// centroids are quantised once per call to 16-bit fixed point,
//     P = rint(256 c')  (-32768 <= P <= 32767),  P = 256 H + (Ls + 128),
// with H = floor(P / 256) and Ls = (P mod 256) - 128 both in [-128, 127].
// Two int8 MFMA products give exact int32 sums, and the screening score of a
// centroid is the exact integer
//     s(c) = 256 (x'.H - Bh) + x'.Ls,   Bh = rint(||c'||^2 / 2),
// which equals -128 k(c) up to a per-row constant and an error e(c) with
//     |e(c)| <= |128 ||c'||^2 - 256 Bh| + sum_d |x'_d| |256 c'_d - P_d|
//            <  129 + ||x'||_1 / 2 < R := 131 + ||x'||_1 / 2.
// If the best score beats the second by more than 2R, its centroid is the
// unique nearest; if it beats the third by more than 2R, the nearest is one of
// the two best and an exact fp64 evaluation of both decides with the
// (distance, id) order; otherwise the row goes to the exact fallback scan.
// Labels therefore equal those of the fp64 definition, while the contraction
// runs on int8 MFMA (v_mfma_i32_32x32x32_i8) instead of fp32 MFMA.
//
// Centroids whose quantisation would overflow (a coordinate c with
// rint(256 (c - 128)) outside [-32768, 32767], i.e. roughly c outside
// [0, 255.998], or a non-finite value) set a device flag; this kernel then does nothing and the
// fp32 screening kernel, which reads the same flag, takes the call.
//
// MFMA operands: A = 32 centroids of a staged chunk (lane l supplies centroid
// l % 32, bytes 16 (l / 32) .. +15 of a 32-byte K-step), B = 32 rows held in
// registers (same byte mapping); accumulator register r of lane l holds
// centroid 8 (r / 4) + 4 (l / 32) + r % 4 of the block for row l % 32.
#include "exact.h"
#include "wave_ops.h"
#include "ivf_internal.h"

#include <algorithm>
#include <type_traits>
#include <utility>

namespace ivf {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

constexpr int kQChunk = kQuantChunk;  // centroids per staged chunk (sub-chunk of the single plane)
constexpr int kS1Sub = 4;            // 64-centroid sub-chunks per staged chunk of the single plane
constexpr int kS1Chunk = kS1Sub * kQChunk;
constexpr int kOrder1PartRows = 32;  // centroids per column-sum block of the visiting order
constexpr int kNoScore = INT32_MIN;  // score of a padded centroid (below any real score)
constexpr int kNoBias = -(1 << 23);  // H accumulator start of a padded centroid: s = kNoScore

// Row blocks of 32 rows per wave: two for DP <= 128 (each staged centroid
// fragment then feeds two MFMAs), one above (register budget).
template <int DP>
constexpr int rows_blocks()
{
    return DP <= 128 ? 2 : 1;
}

// ------------------------------------------------------------ quantisation
// One wave per centroid (grid-stride). Writes the two planes [H | Ls] of
// DP bytes each (zero beyond D), the bias -Bh, and raises *q_bad on any value
// that does not fit. Centroids C .. Cpad-1 are padding: zero planes and the
// lowest score.
__global__ __launch_bounds__(256) void quantize_kernel(const float *__restrict__ cent, int64_t C, int D,
                                                       int DP, int64_t Cpad, int8_t *__restrict__ qc,
                                                       int32_t *__restrict__ negb, uint32_t *__restrict__ q_bad,
                                                       const uint32_t *__restrict__ skip)
{
    if (skip && *skip) return;  // no int8 screen reads the planes in this call
    const int lane = threadIdx.x & 63;
    const int64_t w0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t j = w0; j < Cpad; j += nw) {
        double n2 = 0.0;
        bool bad = false;
        int8_t *q = qc + j * 2 * DP;
        for (int d = lane; d < DP; d += 64) {
            int hb = 0, lb = 0;
            if (j < C && d < D) {
                const double cp = (double)cent[j * D + d] - 128.0;
                const double p = rint(256.0 * cp);
                if (!(p >= -32768.0 && p <= 32767.0)) {  // also true for NaN
                    bad = true;
                } else {
                    const int P = (int)p;
                    const int H = P >> 8;  // floor(P / 256)
                    hb = H;
                    lb = P - 256 * H - 128;
                    n2 = fma(cp, cp, n2);
                }
            }
            q[d] = (int8_t)hb;
            q[DP + d] = (int8_t)lb;
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) n2 += __shfl_xor(n2, o);
        if (__any(bad) && lane == 0) *q_bad = 1u;
        if (lane == 0) negb[j] = j < C ? -(int32_t)llrint(0.5 * n2) : kNoBias;
    }
}

// ------------------------------------------------------------ staging
// A chunk of kQChunk quantised centroids (both planes) and their biases is
// copied from the padded global arrays straight into LDS by buffer loads with
// an LDS destination (16 bytes per lane, a wave writes 1 KiB of consecutive
// LDS per instruction): no register staging and no LDS stores by the vector
// unit. LDS layout of a chunk: centroid rows of PL planes with a pitch of
// PL DP + 16 bytes (the 16 spread the rows over the banks), then the 64
// biases. Slot s (16 bytes) of the row area holds unit s % (PL DP / 16 + 1)
// of row s / (PL DP / 16 + 1); the pad unit and the bias instruction's lanes past the
// biases read beyond the buffer range and receive zeros. Loads go through
// buffer resources over the chunk's valid rows, so a ragged last chunk and
// the chunk after the last one read zeros and every load is unconditional.
// The loads of a chunk are complete (and visible to every wave) after the
// next workgroup barrier, which waits for all outstanding vector memory
// operations.
template <int DP, int NT, int PL = 2>
struct QStager {
    static constexpr int kRowB = PL * DP;                // bytes per centroid
    static constexpr int kRowU = kRowB / 16;             // 16-byte units per centroid
    static constexpr int kPitch = kRowB + 16;
    static constexpr int kRowInst = kRowU + 1;           // 64 rows x (kRowU + 1) slots / 64 lanes
    static constexpr int kInst = kRowInst + 1;           // plus one for the biases
    static constexpr int kBias = kQChunk * kPitch;       // byte offset of the biases (= kRowInst KiB)
    static constexpr int kBytes = kInst * 1024;
    static constexpr int kW = NT / 64;
    static constexpr int kIPW = (kInst + kW - 1) / kW;   // load instructions per wave
    int voff[kIPW];
    int wave;  // wave-uniform

    __device__ __forceinline__ void init()
    {
        const int lane = threadIdx.x & 63;
        wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
#pragma unroll
        for (int i = 0; i < kIPW; ++i) {
            const int inst = wave + i * kW;
            int off = 1 << 30;  // beyond any buffer range: reads zero
            if (inst < kRowInst) {
                const int slot = 64 * inst + lane;
                const int r = slot / (kRowU + 1), u = slot % (kRowU + 1);
                if (u < kRowU) off = r * kRowB + 16 * u;
            } else if (inst == kRowInst && lane < kQChunk / 4) {
                off = 16 * lane;
            }
            voff[i] = off;
        }
    }

    // Enqueues the loads of the chunk starting at centroid cbase into the LDS
    // buffer buf.
    __device__ __forceinline__ void fetch(const int8_t *__restrict__ qc, const int32_t *__restrict__ negb,
                                          int64_t cbase, int64_t cpad, char *buf) const
    {
        const int64_t left = cpad - cbase;
        const int valid = (int)(left < 0 ? 0 : left < kQChunk ? left : kQChunk);
        const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<int8_t *>(qc + cbase * kRowB), (short)0, valid * kRowB, 0x00020000);
        const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<int32_t *>(negb + cbase), (short)0, valid * 4, 0x00020000);
#pragma unroll
        for (int i = 0; i < kIPW; ++i) {
            const int inst = wave + i * kW;
            if (inst < kInst)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(inst < kRowInst ? rq : rb,
                                                         (__attribute__((address_space(3))) void *)(buf + inst * 1024),
                                                         16, voff[i], 0, 0, 0);
        }
    }
};

// ------------------------------------------------------------ rows
// Row block rb of this wave: K-step k of row (wave * RB + rb) * 32 + l % 32
// as x' = x - 128 (a byte xor), dimensions >= D zero; l1 += sum |x'_d| over
// the lane's bytes (v_sad_u8 against 128).
template <int DP, int RB>
__device__ __forceinline__ void load_rows(const uint8_t *__restrict__ X, int64_t row0, int64_t nrows, int D,
                                          int wave, int jl, int h, i32x4 (&xf)[RB][DP / 32],
                                          uint32_t (&l1)[RB])
{
    constexpr int KS = DP / 32;
    const int64_t left = nrows - row0;
    const int rows_here = (int)(left < 0 ? 0 : left < 2048 ? left : 2048);
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t *>(X + row0 * (int64_t)D), (short)0, rows_here * D, 0x00020000);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int base = ((wave * RB + rb) * 32 + jl) * D + 16 * h;
        uint32_t s = 0;
#pragma unroll
        for (int k = 0; k < KS; ++k) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const int d = 32 * k + 16 * h + 4 * w;
                const uint32_t raw = __builtin_amdgcn_raw_buffer_load_b32(rr, base + 32 * k + 4 * w, 0, 0);
                const bool ok = d < D;
                xf[rb][k][w] = ok ? (int)(raw ^ 0x80808080u) : 0;
                s = ok ? __builtin_amdgcn_sad_u8(raw, 0x80808080u, s) : s;
            }
        }
        l1[rb] = s;
    }
}

// The same for a list of rows: tile position t holds row ids[t] (t < n);
// rowid[rb] receives this lane's row, or -1 past the end of the list.
template <int DP, int RB>
__device__ __forceinline__ void load_rows_ids(const uint8_t *__restrict__ X, int64_t N, const int32_t *__restrict__ ids,
                                              int64_t t0, int64_t n, int D, int wave, int jl, int h,
                                              i32x4 (&xf)[RB][DP / 32], uint32_t (&l1)[RB], int64_t (&rowid)[RB])
{
    constexpr int KS = DP / 32;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int64_t t = t0 + (wave * RB + rb) * 32 + jl;
        int64_t r = t < n ? (int64_t)ids[t] : -1;
        if (r >= N) r = -1;
        rowid[rb] = r;
        const uint8_t *xr = X + (r < 0 ? 0 : r) * (int64_t)D + 16 * h;
        uint32_t s = 0;
#pragma unroll
        for (int k = 0; k < KS; ++k) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const int d = 32 * k + 16 * h + 4 * w;
                const bool ok = r >= 0 && d < D;
                const uint32_t raw = ok ? *reinterpret_cast<const uint32_t *>(xr + 32 * k + 4 * w) : 0x80808080u;
                xf[rb][k][w] = ok ? (int)(raw ^ 0x80808080u) : 0;
                s = ok ? __builtin_amdgcn_sad_u8(raw, 0x80808080u, s) : s;
            }
        }
        l1[rb] = s;
    }
}

// ------------------------------------------------------------ top-1 epilogue
// The three largest scores a lane has kept for its row and the ids of two.
// The certificate only asks whether the second and third scores are below
// best - 2R, and the best only grows, so a lane keeps just the scores above
// thr = max(k3, k1 - 2R - 1) at the time they are seen: every score that
// ends up at or above final best - 2R is kept exactly, and every score kept
// in its place or dropped lies below final best - 2R, so the decisions are
// those of the exact three largest.
// t3 = (thr - lmax) >> 8 is the prefilter threshold on the H accumulators
// (lmax = 128 ||x'||_1 >= x'.Ls, so an H value h <= t3 has s <= thr);
// twoR = 262 + ||x'||_1, so lmax = 128 (twoR - 262).
// Largest value over the two half-lanes of a row (lanes l and l ^ 32).
// v_permlane32_swap exchanges the upper 32 lanes of its first operand with
// the lower 32 lanes of its second; with v in both, each lane finds v of
// lanes l and l ^ 32 in its two results. A VALU exchange, where a shuffle
// would take a round trip through the LDS crossbar.
__device__ __forceinline__ int halves_max(int v)
{
    const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
    return max((int)r[0], (int)r[1]);
}

struct Top3i {
    int k1, k2, k3;
    int i1, i2;
    int t3, twoR;
    int ks;  // single plane: score of the row's hinted centroid (kNoScore: none)
};

__device__ __forceinline__ int keep_threshold(const Top3i &st)
{
    return st.k1 > kNoScore ? max(st.k3, st.k1 - st.twoR - 1) : kNoScore;
}

// Plain integer expressions (the compiler forms v_med3_i32 and v_max3_i32
// from them): the operands include MFMA results, and only instructions the
// compiler sees get the wait states that reading them requires.
__device__ __forceinline__ int med3i(int a, int b, int c)
{
    return min(max(a, b), max(min(a, b), c));
}

__device__ __forceinline__ int max3i(int a, int b, int c) { return max(max(a, b), c); }

__device__ __forceinline__ int max4i(int a, int b, int c, int d)
{
    return max(max(max(a, b), c), d);
}

// Branch-free insertion (v <= k3 leaves the state unchanged): with
// k1 >= k2 >= k3, med3(v, k2, k3) is the new third and med3(v, k1, k2) the
// new second; strict comparisons keep the lower id on equal scores because a
// lane visits ids in ascending order.
__device__ __forceinline__ void top3i_push(Top3i &t, int v, int id)
{
    const bool gt1 = v > t.k1;
    const bool gt2 = v > t.k2;
    t.k3 = med3i(v, t.k2, t.k3);
    t.k2 = med3i(v, t.k1, t.k2);
    t.k1 = gt1 ? v : t.k1;
    const int j2 = gt2 ? id : t.i2;
    t.i2 = gt1 ? t.i1 : j2;
    t.i1 = gt1 ? id : t.i1;
}

__device__ __forceinline__ bool score_gt(int ka, int ia, int kb, int ib)
{
    return ka > kb || (ka == kb && ia < ib);
}

// Merges two lists sorted by (score descending, id ascending).
__device__ __forceinline__ Top3i top3i_merge(Top3i a, Top3i b)
{
    if (score_gt(b.k1, b.i1, a.k1, a.i1)) {
        const Top3i t = a;
        a = b;
        b = t;
    }
    Top3i m;
    m.k1 = a.k1;
    m.i1 = a.i1;
    if (score_gt(b.k1, b.i1, a.k2, a.i2)) {
        m.k2 = b.k1;
        m.i2 = b.i1;
        m.k3 = max(a.k2, b.k2);
    } else {
        m.k2 = a.k2;
        m.i2 = a.i2;
        m.k3 = max(a.k3, b.k1);
    }
    return m;
}

// Group g (0..3) of a finished tile: registers 4g .. 4g + 3, centroids
// idp + 8g + e. The group's H values are tested against the prefilter
// threshold (three instructions for four centroids); only when some lane of
// the wave passes are the exact scores formed (one shift-add each), tested
// against the third largest and inserted.
template <int g>
__device__ __forceinline__ void i8_group(const i32x16 &pH, const i32x16 &pL, int idp, Top3i &st)
{
    const int m = max4i(pH[4 * g], pH[4 * g + 1], pH[4 * g + 2], pH[4 * g + 3]);
    if (__any(m > st.t3)) {
        int v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (int)((uint32_t)pH[4 * g + e] << 8) + pL[4 * g + e];
        if (__any(max4i(v[0], v[1], v[2], v[3]) > keep_threshold(st))) {
#pragma unroll
            for (int e = 0; e < 4; ++e) top3i_push(st, v[e], idp + 8 * g + e);
            const int thr = keep_threshold(st);
            st.t3 = thr > kNoScore ? (thr - ((st.twoR - 262) << 7)) >> 8 : kNoScore;
        }
    }
    // keeps the group at this point of the MFMA stream
    asm volatile("" : "+v"(st.k1), "+v"(st.k2), "+v"(st.k3), "+v"(st.i1), "+v"(st.i2), "+v"(st.t3));
}

// Routing epilogues of the two-plane tile (uint8-valued queries): keys of
// the threshold sample, or the filter that lists every centroid whose key is
// at most the query's threshold. The key of a centroid is -(float)s, which
// orders the centroids like their distances up to the bound of the routing
// certificate (the screening error of s plus the rounding to fp32).
// The keys pass writes, per row, the minimum key of every 16 consecutive
// centroids of the sample (the two half-lanes of a row each hold 8 of them),
// which is all the threshold needs.
struct RouteKeysState {
    float *krow;      // the row's group minima, indexed by (centroid id - c_begin) / 16; null: no row
    int64_t c_begin, c_end;
    int acc;          // largest score of the current group of 16 on this half-lane
};

// Candidates are queued per thread and row block in LDS (kRouteQueue
// entries (s, id); entry e of thread t at q[e * threads + t] of the row
// block's queue) and moved to the query's list with one atomic per thread
// when some lane of the wave could overflow its queue and at the end of the
// range. The queue takes every score with s >= sthr, a necessary condition
// for -(float)s <= tau; the flush keeps the exact ones.
constexpr int kRouteQueue = 12;

struct RouteFilterState {
    int t3;           // prefilter on the H accumulators: a key <= tau needs H >= t3
    int sthr;         // and s >= sthr
    float tau;
    int64_t row;      // -1: no row
    uint32_t *cand_cnt;
    uint2 *cand;
    int L;
    uint2 *q;         // this thread's queue (stride qstride)
    int qstride;
    int qn;
};

__device__ __forceinline__ void route_flush(RouteFilterState &st)
{
    if (st.qn > 0 && st.row >= 0) {
        uint32_t n = 0;
        for (int i = 0; i < st.qn; ++i) n += -(float)(int)st.q[i * st.qstride].x <= st.tau ? 1u : 0u;
        if (n) {
            uint32_t slot = atomicAdd(st.cand_cnt + st.row, n);
            uint2 *dst = st.cand + st.row * st.L;
            for (int i = 0; i < st.qn; ++i) {
                const uint2 e = st.q[i * st.qstride];
                const float k = -(float)(int)e.x;
                if (k <= st.tau) {
                    if (slot < (uint32_t)st.L) dst[slot] = make_uint2(__float_as_uint(k), e.y);
                    ++slot;
                }
            }
        }
    }
    st.qn = 0;
}

template <int g>
__device__ __forceinline__ void i8_group(const i32x16 &pH, const i32x16 &pL, int idp, RouteKeysState &st)
{
    // registers of groups 2m and 2m + 1 hold, over both half-lanes, the
    // centroids 16m .. 16m + 15 of the 32-centroid block at idp - 4h
    int m = (int)((uint32_t)pH[4 * g] << 8) + pL[4 * g];
#pragma unroll
    for (int e = 1; e < 4; ++e) m = max(m, (int)((uint32_t)pH[4 * g + e] << 8) + pL[4 * g + e]);
    if constexpr (g % 2 == 0) {
        st.acc = m;
    } else {
        m = max(m, st.acc);
        m = halves_max(m);
        const int64_t id0 = (int64_t)(idp & ~31) + 16 * (g / 2);
        if (st.krow && (threadIdx.x & 32) == 0 && id0 >= st.c_begin && id0 + 15 < st.c_end)
            st.krow[(id0 - st.c_begin) >> 4] = -(float)m;
    }
}

template <int g>
__device__ __forceinline__ void i8_group(const i32x16 &pH, const i32x16 &pL, int idp, RouteFilterState &st)
{
    const int m = max4i(pH[4 * g], pH[4 * g + 1], pH[4 * g + 2], pH[4 * g + 3]);
    if (__any(m >= st.t3)) {
        if (__any(st.qn > kRouteQueue - 4)) route_flush(st);
        // branch-free: every value is written at the queue's end, which
        // advances only for those that pass (sthr excludes rows past the
        // queries and padded centroids, whose score is INT_MIN)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int v = (int)((uint32_t)pH[4 * g + e] << 8) + pL[4 * g + e];
            st.q[st.qn * st.qstride] = make_uint2((uint32_t)v, (uint32_t)(idp + 8 * g + e));
            st.qn += v >= st.sthr ? 1 : 0;
        }
    }
    // keeps the group at this point of the MFMA stream
    asm volatile("" : "+v"(st.t3), "+v"(st.qn));
}

template <int g, int T, int KS, class S>
__device__ __forceinline__ void i8_groups_at(const i32x16 &pH, const i32x16 &pL, int idp, S &st)
{
    if constexpr (g < 4) {
        if constexpr (g * KS / 4 == T) i8_group<g>(pH, pL, idp, st);
        i8_groups_at<g + 1, T, KS>(pH, pL, idp, st);
    }
}

// The fragments of one staged 32-centroid block for every K-step: plane H at
// Ar + 32k, plane Ls at Ar + DP + 32k (Ar = this lane's row, offset 16 h).
template <int DP>
struct Frags {
    i32x4 h[DP / 32], l[DP / 32];
};

template <int DP>
__device__ __forceinline__ void load_frags(const char *Ar, Frags<DP> &f)
{
#pragma unroll
    for (int k = 0; k < DP / 32; ++k) {
        f.h[k] = *reinterpret_cast<const i32x4 *>(Ar + 32 * k);
        f.l[k] = *reinterpret_cast<const i32x4 *>(Ar + DP + 32 * k);
    }
}

__device__ __forceinline__ i32x16 load_bias(const int *Bh)
{
    i32x16 bias;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const i32x4 u = *reinterpret_cast<const i32x4 *>(Bh + 8 * g);
        bias[4 * g + 0] = u[0];
        bias[4 * g + 1] = u[1];
        bias[4 * g + 2] = u[2];
        bias[4 * g + 3] = u[3];
    }
    return bias;
}

// K-steps T .. KS-1 of one tile: a 32-centroid block against one 32-row
// block, both planes, into (cH, cL); at T = 0, cH starts from the biases and
// cL from zero. With EP, the epilogue of the previous tile (pH, pL; ids from
// idp; state sp) runs between the K-steps. With PF (the last tile that uses
// this block's fragments), each fragment register is refilled from the next
// block (nA, nB) as soon as its last MFMA has been issued, so the LDS reads
// of the next block overlap this tile's MFMAs.
template <int DP, bool PF, int T = 0, class S>
__device__ __forceinline__ void i8_tile(Frags<DP> &f, const i32x4 (&x)[DP / 32], i32x16 &bias, i32x16 &cH,
                                        i32x16 &cL, const i32x16 &pH, const i32x16 &pL, int idp, S &sp,
                                        const char *nA, const int *nB)
{
    constexpr int KS = DP / 32;
    if constexpr (T < KS) {
        if constexpr (T == 0) {
            const i32x16 zero = {0};
            cH = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.h[0], x[0], bias, 0, 0, 0);
            cL = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.l[0], x[0], zero, 0, 0, 0);
            if constexpr (PF) bias = load_bias(nB);
        } else {
            cH = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.h[T], x[T], cH, 0, 0, 0);
            cL = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.l[T], x[T], cL, 0, 0, 0);
        }
        if constexpr (PF) {
            f.h[T] = *reinterpret_cast<const i32x4 *>(nA + 32 * T);
            f.l[T] = *reinterpret_cast<const i32x4 *>(nA + DP + 32 * T);
        }
        i8_groups_at<0, T, KS>(pH, pL, idp, sp);
        __builtin_amdgcn_sched_barrier(0);
        i8_tile<DP, PF, T + 1>(f, x, bias, cH, cL, pH, pL, idp, sp, nA, nB);
    }
}

template <int g = 0, class S>
__device__ __forceinline__ void i8_drain(const i32x16 &pH, const i32x16 &pL, int idp, S &st)
{
    if constexpr (g < 4) {
        i8_group<g>(pH, pL, idp, st);
        i8_drain<g + 1>(pH, pL, idp, st);
    }
}


// Merges the two half-lanes of a row, certifies with the bound 2R = 262 + ||x'||_1,
// settles two-way near-ties exactly in fp64 and queues the rest for the
// full fp64 fallback.
__device__ __forceinline__ void i8_finish(const ScreenI8Args &a, int64_t row, bool rvalid, int h, const Top3i &st)
{
    Top3i o;
    o.k1 = __shfl_xor(st.k1, 32);
    o.k2 = __shfl_xor(st.k2, 32);
    o.k3 = __shfl_xor(st.k3, 32);
    o.i1 = __shfl_xor(st.i1, 32);
    o.i2 = __shfl_xor(st.i2, 32);
    const Top3i m = top3i_merge(st, o);
    int label = -1;
    bool refined = false;
    if (rvalid && h == 0) {
        const int64_t twoR = st.twoR;
        // a centroid id is used only when it names a real centroid; any other
        // state sends the row to the exact fallback scan
        const bool ok1 = m.i1 >= 0 && m.i1 < a.ncent;
        const bool ok2 = m.i2 >= 0 && m.i2 < a.ncent;
        if (!a.force_fallback && ok1) {
            if ((int64_t)m.k1 - (int64_t)m.k2 > twoR) {
                label = m.i1;
            } else if ((int64_t)m.k1 - (int64_t)m.k3 > twoR && ok2) {
                const uint8_t *x = a.rows + row * (int64_t)a.D;
                const double d1 = exact_dist(x, a.cent + (int64_t)m.i1 * a.D, a.D);
                const double d2 = exact_dist(x, a.cent + (int64_t)m.i2 * a.D, a.D);
                label = dist_lt(d2, m.i2, d1, m.i1) ? m.i2 : m.i1;
                refined = true;
            }
        }
        a.labels[row] = label;
    }
    // statistics and worklist slots: one atomic per wave
    const bool to_fallback = rvalid && h == 0 && label < 0;
    wave_count(a.stats + kStatRefine2, refined);
    wave_count(a.stats + kStatFallback, to_fallback);
    const uint32_t slot = wave_append(a.wl_cnt, to_fallback);
    if (to_fallback && slot < (uint64_t)a.wl_cap) a.wl[slot] = (int32_t)row;
}

// One workgroup tile: W * 32 * RB rows against every centroid. Chunk j sits
// in LDS buffer j & 1. Tiles (32 centroids x 32 rows) run block by block and
// within a block row block by row block, alternating between the
// accumulator sets T0 and T1; each tile's K-steps carry the epilogue of the
// tile before it, and the last tile of a block loads the next block's
// fragments and biases. The barrier before the last tile of chunk j, the
// first tile that reads chunk j + 1, completes the loads of chunk j + 1
// (issued right after the previous such barrier) and ends every read of
// chunk j's buffer, whose loads for chunk j + 2 are issued right after it, a
// whole chunk ahead of their first use. The loop is rotated so that an
// iteration starts right after a barrier (no LDS read outstanding) with the
// last tile of chunk j, then runs chunk j + 1 up to its last tile; all LDS
// waits inside are then exact.
template <int DP, int W>
__device__ void screen_i8_tile(const ScreenI8Args &a, int64_t tile, char *__restrict__ lds, const int32_t *ids,
                               int64_t n)
{
    constexpr int RB = rows_blocks<DP>();
    constexpr int NT = W * 64;
    using St = QStager<DP, NT>;
    constexpr int CS = (St::kBytes + 15) / 16 * 16;
    constexpr int BLK = 32 * St::kPitch;  // bytes of one 32-centroid block
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int h = lane >> 5;
    const int jl = lane & 31;
    const int64_t row0 = tile * (W * 32 * RB);

    i32x4 xf[RB][DP / 32];
    uint32_t l1[RB];
    int64_t rowid[RB];
    if (ids) {
        load_rows_ids<DP, RB>(a.rows, a.nrows, ids, row0, n, a.D, wave, jl, h, xf, l1, rowid);
    } else {
        load_rows<DP, RB>(a.rows, row0, a.nrows, a.D, wave, jl, h, xf, l1);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int64_t row = row0 + (wave * RB + rb) * 32 + jl;
            rowid[rb] = row < a.nrows ? row : -1;
        }
    }

    Top3i st[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        l1[rb] += __shfl_xor(l1[rb], 32);
        st[rb] = Top3i{kNoScore, kNoScore, kNoScore, -1, -1, kNoScore, (int)(262 + l1[rb]), kNoScore};
    }

    const char *A0 = lds + jl * St::kPitch + 16 * h;  // block 0 of buffer 0
    const char *B0 = lds + St::kBias + 16 * h;        // its biases (4 h ints in)
    const int idh = 4 * h;
    const int nch = (int)a.nchunks;
    auto abuf = [&](int jj) { return A0 + (jj & 1) * CS; };
    auto bbuf = [&](int jj) { return reinterpret_cast<const int *>(B0 + (jj & 1) * CS); };

    St q;
    q.init();
    q.fetch(a.qc, a.negb, 0, a.cpad, lds);
    __syncthreads();
    q.fetch(a.qc, a.negb, kQChunk, a.cpad, lds + CS);
    // the barrier completes the loads of chunk jj (issued one stage earlier)
    // and ends every read of the other buffer, which then receives chunk jj + 1
    auto stage = [&](int jj) {
        __syncthreads();
        q.fetch(a.qc, a.negb, (int64_t)(jj + 1) * kQChunk, a.cpad, lds + ((jj + 1) & 1) * CS);
    };

    // T1 starts as a tile of lowest scores, so the first epilogue inserts nothing
    i32x16 h0, l0, h1, l1acc = {0};
#pragma unroll
    for (int r = 0; r < 16; ++r) h1[r] = kNoBias;
    i32x16 bias = load_bias(bbuf(0));
    Frags<DP> f;
    load_frags<DP>(abuf(0), f);

    if constexpr (RB == 2) {
        // (jj, cb, rows 0) -> T0 while T1 = the tile before drains
        auto rows0 = [&](int jj, int cb) {
            i8_tile<DP, false>(f, xf[0], bias, h0, l0, h1, l1acc, idh + jj * kQChunk + 32 * cb - 32, st[1],
                               nullptr, nullptr);
        };
        // (jj, cb, rows 1) -> T1 while T0 = (jj, cb, rows 0) drains; loads the next block
        auto rows1 = [&](int jj, int cb, const char *nA, const int *nB) {
            i8_tile<DP, true>(f, xf[1], bias, h1, l1acc, h0, l0, idh + jj * kQChunk + 32 * cb, st[0], nA, nB);
        };
        rows0(0, 0);
        rows1(0, 0, abuf(0) + BLK, bbuf(0) + 32);
        rows0(0, 1);
        stage(1);
        for (int j = 0;; ++j) {
            rows1(j, 1, abuf(j + 1), bbuf(j + 1));
            if (j + 1 == nch) break;
            rows0(j + 1, 0);
            rows1(j + 1, 0, abuf(j + 1) + BLK, bbuf(j + 1) + 32);
            rows0(j + 1, 1);
            stage(j + 2);
        }
    } else {
        // (jj, 0) -> T0 while T1 = (jj - 1, 1) drains; (jj, 1) -> T1 while T0 drains
        auto blk0 = [&](int jj) {
            i8_tile<DP, true>(f, xf[0], bias, h0, l0, h1, l1acc, idh + jj * kQChunk - 32, st[0], abuf(jj) + BLK,
                              bbuf(jj) + 32);
        };
        auto blk1 = [&](int jj) {
            i8_tile<DP, true>(f, xf[0], bias, h1, l1acc, h0, l0, idh + jj * kQChunk, st[0], abuf(jj + 1),
                              bbuf(jj + 1));
        };
        blk0(0);
        stage(1);
        for (int j = 0;; ++j) {
            blk1(j);
            if (j + 1 == nch) break;
            blk0(j + 1);
            stage(j + 2);
        }
    }
    i8_drain(h1, l1acc, idh + (nch - 1) * kQChunk + 32, st[RB - 1]);

#pragma unroll
    for (int rb = 0; rb < RB; ++rb) i8_finish(a, rowid[rb], rowid[rb] >= 0, h, st[rb]);
}

template <int DP, int W>
__global__ __launch_bounds__(W * 64, 2) void screen_i8_kernel(ScreenI8Args a)
{
    using St = QStager<DP, W * 64>;
    constexpr int CS = (St::kBytes + 15) / 16 * 16;
    __shared__ __attribute__((aligned(16))) char lds[2 * CS];
    if (*a.q_bad) return;  // the fp32 screen takes this call
    if (blockIdx.x == 0 && threadIdx.x == 0) a.stats[kStatScreenI8] = 1ull;
    // after the single-plane screen: only the rows it left (its list), or
    // every row when the list overflowed or the single plane did not apply
    const int32_t *ids = nullptr;
    int64_t n = a.nrows;
    if (a.list && *a.q_bad1 == 0) {
        const uint32_t c = *a.list_cnt;
        if (c <= (uint64_t)a.list_cap) {
            ids = a.list;
            n = c;
        }
    }
    constexpr int rows_per_tile = W * 32 * rows_blocks<DP>();
    const int64_t ntiles = (n + rows_per_tile - 1) / rows_per_tile;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        screen_i8_tile<DP, W>(a, tile, lds, ids, n);
        __syncthreads();
    }
}

template <int DP, int W>
hipError_t launch_i8(const ScreenI8Args &a, int num_cus, hipStream_t s)
{
    constexpr int rows_per_tile = W * 32 * rows_blocks<DP>();
    const int64_t ntiles = (a.nrows + rows_per_tile - 1) / rows_per_tile;
    const int per_cu = 8 / W;  // two waves per SIMD
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(ntiles, (int64_t)per_cu * num_cus));
    hipLaunchKernelGGL((screen_i8_kernel<DP, W>), dim3(grid), dim3(W * 64), 0, s, a);
    return hipGetLastError();
}

template <int W>
hipError_t launch_i8_w(int DP, const ScreenI8Args &a, int num_cus, hipStream_t s)
{
    switch (DP) {
    case 32: return launch_i8<32, W>(a, num_cus, s);
    case 64: return launch_i8<64, W>(a, num_cus, s);
    case 96: return launch_i8<96, W>(a, num_cus, s);
    case 128: return launch_i8<128, W>(a, num_cus, s);
    case 192: return launch_i8<192, W>(a, num_cus, s);
    case 256: return launch_i8<256, W>(a, num_cus, s);
    default: return hipErrorInvalidValue;
    }
}

// ============================================================ routing
// Routing of uint8-valued queries (integers in [0, 255] stored as fp32) on
// the two planes: x' = q - 128 is exact in int8, and the key -(float)s of a
// centroid differs from 128 k(c) minus a per-query constant by less than
// R + 64 (R = 131 + ||x'||_1 / 2 from the screening, 64 from rounding s to
// fp32), so the routing certificate of the fp32 path holds with the bound
// B = R + 64 in these key units (Sec. "GPU coarse search": the routing
// contraction; the exactness argument is that of the assignment screens).
// route_i8_check checks every query value before the centroids are
// quantised, route_i8_bound writes B per query; when some value is not an
// integer in [0, 255] or some centroid does not quantise (*q_bad), *off is
// raised and the fp32 kernels, which check the same flag, take the call.

// Raises *off when some value of the nq queries is not an integer in
// [0, 255] (one wave per query, grid-stride).
__global__ __launch_bounds__(256) void route_i8_check_kernel(const float *__restrict__ Q, int64_t nq, int D,
                                                             uint32_t *__restrict__ off)
{
    const int lane = threadIdx.x & 63;
    const int64_t w0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
    bool bad = false;
    for (int64_t q = w0; q < nq; q += nw) {
        for (int d = lane; d < D; d += 64) {
            const float v = Q[q * D + d];
            if (!(v >= 0.0f && v <= 255.0f && v == rintf(v))) bad = true;  // also true for NaN
        }
    }
    if (__syncthreads_or(bad) && threadIdx.x == 0) atomicOr(off, 1u);  // one atomic per workgroup
}

// Per query of a batch (one wave each): qbound[q] = B = (390 + ||x'||_1) / 2;
// raises *off when *q_bad (a centroid outside the two planes' range) is set.
__global__ __launch_bounds__(256) void route_i8_bound_kernel(const float *__restrict__ Q, int64_t nq, int D,
                                                             const uint32_t *__restrict__ q_bad,
                                                             uint32_t *__restrict__ off, float *__restrict__ qbound)
{
    // (the bounds are written whatever *off says: a wave must not read the
    // flag this kernel itself raises to decide whether to take part)
    const int lane = threadIdx.x & 63;
    const int64_t w0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
    if (w0 == 0 && lane == 0 && *q_bad) atomicOr(off, 1u);
    for (int64_t q = w0; q < nq; q += nw) {
        uint32_t l1 = 0;
        for (int d = lane; d < D; d += 64) {
            const float v = Q[q * D + d];  // (a value outside [0, 255] has raised *off already)
            const int x = v >= 0.0f && v <= 255.0f ? (int)v - 128 : 0;
            l1 += (uint32_t)(x < 0 ? -x : x);
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) l1 += __shfl_xor(l1, o);
        if (lane == 0) qbound[q] = 0.5f * (float)(390u + l1);
    }
}

// Row block rb of this wave from fp32 queries that hold integers in
// [0, 255]: x' = q - 128 as int8 (dimensions >= D zero), l1 = ||x'||_1 of
// the lane's half (the caller adds the other half).
template <int DP, int RB>
__device__ __forceinline__ void load_queries(const float *__restrict__ Q, int64_t row0, int64_t nrows, int D,
                                             int wave, int jl, int h, i32x4 (&xf)[RB][DP / 32],
                                             uint32_t (&l1)[RB], int64_t (&rowid)[RB])
{
    constexpr int KS = DP / 32;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int64_t row = row0 + (wave * RB + rb) * 32 + jl;
        const bool rv = row < nrows;
        rowid[rb] = rv ? row : -1;
        const float *qr = Q + (rv ? row : 0) * (int64_t)D + 16 * h;
        uint32_t s = 0;
#pragma unroll
        for (int k = 0; k < KS; ++k) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const int d = 32 * k + 16 * h + 4 * w;
                uint32_t packed = 0;
                if (rv && d < D) {
                    const float4 v = *reinterpret_cast<const float4 *>(qr + 32 * k + 4 * w);
                    const float va[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int x = (int)va[e] - 128;
                        packed |= ((uint32_t)x & 0xFFu) << (8 * e);
                        s += (uint32_t)(x < 0 ? -x : x);
                    }
                }
                xf[rb][k][w] = (int)packed;
            }
        }
        l1[rb] = s;
    }
}

// Chunks [ch_lo, ch_hi) of the range's 64-centroid chunks (chunk j starts at
// centroid c_begin + 64 j) against one tile of queries, with the keys or
// the filter epilogue; the staging and the MFMA stream are those of
// screen_i8_tile.
template <int DP, int W, int MODE>
__device__ void route_i8_range(const RouteI8Args &a, int64_t tile, int64_t ch_lo, int64_t ch_hi,
                               char *__restrict__ lds, uint2 *__restrict__ queue)
{
    constexpr int RB = rows_blocks<DP>();
    constexpr int NT = W * 64;
    using St = QStager<DP, NT>;
    constexpr int CS = (St::kBytes + 15) / 16 * 16;
    constexpr int BLK = 32 * St::kPitch;
    using S = typename std::conditional<MODE == kRouteKeys, RouteKeysState, RouteFilterState>::type;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int h = lane >> 5;
    const int jl = lane & 31;
    const int64_t row0 = tile * (W * 32 * RB);

    i32x4 xf[RB][DP / 32];
    uint32_t l1[RB];
    int64_t rowid[RB];
    load_queries<DP, RB>(a.queries, row0, a.nq, a.D, wave, jl, h, xf, l1, rowid);

    S st[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        l1[rb] += __shfl_xor(l1[rb], 32);
        const int64_t row = rowid[rb];
        if constexpr (MODE == kRouteKeys) {
            st[rb].krow = row >= 0 ? a.keys + row * ((a.c_end - a.c_begin) / 16) : nullptr;
            st[rb].c_begin = a.c_begin;
            st[rb].c_end = a.c_end;
            st[rb].acc = INT_MIN;
        } else {
            st[rb].row = row;
            st[rb].cand_cnt = a.cand_cnt;
            st[rb].cand = a.cand;
            st[rb].L = a.L;
            st[rb].tau = row >= 0 ? a.tau[row] : -__builtin_huge_valf();
            // a key <= tau needs s >= -tau - 64, and s <= 256 H + 128 ||x'||_1
            const double t = floor((-(double)st[rb].tau - 64.0 - 128.0 * (double)l1[rb]) / 256.0);
            st[rb].t3 = row < 0 || !(t <= 2147483647.0) ? INT_MAX : t < -2147483648.0 ? INT_MIN : (int)t;
            // s > INT_MIN for every real centroid: padded ones (s = INT_MIN) never pass
            const double u = ceil(-(double)st[rb].tau - 64.0);
            st[rb].sthr = row < 0 || !(u <= 2147483647.0) ? INT_MAX : u < -2147483647.0 ? INT_MIN + 1 : (int)u;
            st[rb].q = queue + rb * kRouteQueue * NT + threadIdx.x;
            st[rb].qstride = NT;
            st[rb].qn = 0;
        }
    }

    const char *A0 = lds + jl * St::kPitch + 16 * h;
    const char *B0 = lds + St::kBias + 16 * h;
    // ids count chunks in visiting order (the keys' slots); chunk jj of the
    // range is read from physical chunk (ch_lo + jj) * cstride (keys of a
    // spread sample; 1 otherwise)
    const int64_t cb0 = a.c_begin + ch_lo * kQChunk;
    const int idh = (int)cb0 + 4 * h;
    const int nch = (int)(ch_hi - ch_lo);
    const int64_t cst = a.cstride > 1 ? a.cstride : 1;
    auto pbase = [&](int64_t jj) { return a.c_begin + (ch_lo + jj) * cst * kQChunk; };
    auto abuf = [&](int jj) { return A0 + (jj & 1) * CS; };
    auto bbuf = [&](int jj) { return reinterpret_cast<const int *>(B0 + (jj & 1) * CS); };

    St q;
    q.init();
    q.fetch(a.qc, a.negb, pbase(0), a.cpad, lds);
    __syncthreads();
    q.fetch(a.qc, a.negb, pbase(1), a.cpad, lds + CS);
    auto stage = [&](int jj) {
        __syncthreads();
        q.fetch(a.qc, a.negb, pbase(jj + 1), a.cpad, lds + ((jj + 1) & 1) * CS);
    };

    // T1 starts as a tile of lowest scores: the first epilogue keeps nothing
    // (its ids lie before the range)
    i32x16 h0, l0, h1, l1acc = {0};
#pragma unroll
    for (int r = 0; r < 16; ++r) h1[r] = kNoBias;
    i32x16 bias = load_bias(bbuf(0));
    Frags<DP> f;
    load_frags<DP>(abuf(0), f);
    // the block before the range: keys are written only inside the range and
    // the filter's first drain sees only lowest scores
    S none = st[RB - 1];
    if constexpr (MODE == kRouteKeys) {
        none.krow = nullptr;
    } else {
        none.row = -1;
        none.sthr = INT_MAX;
    }

    if constexpr (RB == 2) {
        auto rows0 = [&](int jj, int cb, S &sp) {
            i8_tile<DP, false>(f, xf[0], bias, h0, l0, h1, l1acc, idh + jj * kQChunk + 32 * cb - 32, sp,
                               nullptr, nullptr);
        };
        auto rows1 = [&](int jj, int cb, const char *nA, const int *nB) {
            i8_tile<DP, true>(f, xf[1], bias, h1, l1acc, h0, l0, idh + jj * kQChunk + 32 * cb, st[0], nA, nB);
        };
        rows0(0, 0, none);
        rows1(0, 0, abuf(0) + BLK, bbuf(0) + 32);
        rows0(0, 1, st[1]);
        stage(1);
        for (int j = 0;; ++j) {
            rows1(j, 1, abuf(j + 1), bbuf(j + 1));
            if (j + 1 == nch) break;
            rows0(j + 1, 0, st[1]);
            rows1(j + 1, 0, abuf(j + 1) + BLK, bbuf(j + 1) + 32);
            rows0(j + 1, 1, st[1]);
            stage(j + 2);
        }
    } else {
        auto blk0 = [&](int jj, S &sp) {
            i8_tile<DP, true>(f, xf[0], bias, h0, l0, h1, l1acc, idh + jj * kQChunk - 32, sp, abuf(jj) + BLK,
                              bbuf(jj) + 32);
        };
        auto blk1 = [&](int jj) {
            i8_tile<DP, true>(f, xf[0], bias, h1, l1acc, h0, l0, idh + jj * kQChunk, st[0], abuf(jj + 1),
                              bbuf(jj + 1));
        };
        blk0(0, none);
        stage(1);
        for (int j = 0;; ++j) {
            blk1(j);
            if (j + 1 == nch) break;
            blk0(j + 1, st[0]);
            stage(j + 2);
        }
    }
    i8_drain(h1, l1acc, idh + (nch - 1) * kQChunk + 32, st[RB - 1]);
    if constexpr (MODE == kRouteFilter) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) route_flush(st[rb]);
    }
}

template <int DP, int W, int MODE>
__global__ __launch_bounds__(W * 64, 2) void route_i8_kernel(RouteI8Args a)
{
    using St = QStager<DP, W * 64>;
    constexpr int CS = (St::kBytes + 15) / 16 * 16;
    __shared__ __attribute__((aligned(16))) char lds[2 * CS];
    __shared__ uint2 queue[MODE == kRouteFilter ? rows_blocks<DP>() * kRouteQueue * W * 64 : 1];
    if (*a.off) return;  // the fp32 kernels take this call
    if (MODE == kRouteFilter && blockIdx.x == 0 && threadIdx.x == 0 && a.stats) a.stats[kStatScreenI8] = 1ull;
    constexpr int rows_per_tile = W * 32 * rows_blocks<DP>();
    const int64_t ntiles = (a.nq + rows_per_tile - 1) / rows_per_tile;
    // a contiguous range of (tile, chunk) units in tile-major order
    const int64_t units = ntiles * a.nchunks;
    int64_t u = units * blockIdx.x / gridDim.x;
    const int64_t u1 = units * (blockIdx.x + 1) / gridDim.x;
    while (u < u1) {
        const int64_t tile = u / a.nchunks;
        const int64_t ch = u - tile * a.nchunks;
        const int64_t ch_end = min(a.nchunks, ch + (u1 - u));
        route_i8_range<DP, W, MODE>(a, tile, ch, ch_end, lds, queue);
        u += ch_end - ch;
        __syncthreads();
    }
}

template <int DP, int MODE>
hipError_t launch_route_i8_dp(const RouteI8Args &a, int num_cus, hipStream_t s)
{
    constexpr int W = 8;
    constexpr int rows_per_tile = W * 32 * rows_blocks<DP>();
    const int64_t ntiles = (a.nq + rows_per_tile - 1) / rows_per_tile;
    const int64_t units = ntiles * a.nchunks;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(units, (int64_t)num_cus));
    hipLaunchKernelGGL((route_i8_kernel<DP, W, MODE>), dim3(grid), dim3(W * 64), 0, s, a);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_route_i8_mode(int DP, const RouteI8Args &a, int num_cus, hipStream_t s)
{
    switch (DP) {
    case 32: return launch_route_i8_dp<32, MODE>(a, num_cus, s);
    case 64: return launch_route_i8_dp<64, MODE>(a, num_cus, s);
    case 96: return launch_route_i8_dp<96, MODE>(a, num_cus, s);
    case 128: return launch_route_i8_dp<128, MODE>(a, num_cus, s);
    case 192: return launch_route_i8_dp<192, MODE>(a, num_cus, s);
    case 256: return launch_route_i8_dp<256, MODE>(a, num_cus, s);
    default: return hipErrorInvalidValue;
    }
}

// ============================================================ single plane
// Screening on one int8 plane: half the MFMA work of the two planes. Every
// centroid is quantised to H1 = rint(c') in [-128, 127] (c' = c - 128) with
// the bias b1 = rint(||c'||^2 / 2), and the score of a centroid is the exact
// integer
//     s1(c) = x'.H1 - b1,
// which differs from g(c) = x'.c' - ||c'||^2 / 2 = -k(c) / 2 by at most
//     W = min(E ||x'||_1, R2 ||x'||_2) + 1/2,
//     E = max_{c,d} |c'_d - H1_d|,   R2 = max_c ||c' - H1||_2
// (Cauchy-Schwarz for the second; E = R2 = 0 for integer-valued centroids,
// such as rows sampled as the k-means initialisation). With T >= 2W: if the
// best score beats the second by more
// than T, its centroid is the unique nearest; if it beats the third by more
// than T, the nearest is one of the two best and an exact fp64 evaluation
// decides; otherwise the row is listed for the two-plane screen, whose bound
// is 256 times finer. Centroids with rint(c') outside [-128, 127] set *q_bad1
// and the two-plane screen takes every row.
constexpr int kNoBias1 = -(1 << 26);  // bias of a padded centroid: below every real score (|s1| < 2^23)

__global__ __launch_bounds__(256) void quantize1_kernel(const float *__restrict__ cent, int64_t C, int D, int DP,
                                                        int64_t Cpad, int8_t *__restrict__ q1,
                                                        int32_t *__restrict__ negb1, uint32_t *__restrict__ q_bad1,
                                                        uint32_t *__restrict__ e_bits, uint32_t *__restrict__ r2_bits,
                                                        const uint32_t *__restrict__ ord, int32_t *__restrict__ pos)
{
    const int lane = threadIdx.x & 63;
    const int64_t w0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t j = w0; j < Cpad; j += nw) {
        // plane row j holds centroid c (rows past C are padding)
        const int64_t c = ord && j < C ? (int64_t)ord[j] : j;
        if (pos && j < C && lane == 0) pos[c] = (int32_t)j;
        double n2 = 0.0, e = 0.0, q2 = 0.0;
        bool bad = false;
        int8_t *q = q1 + j * DP;
        for (int d = lane; d < DP; d += 64) {
            int hb = 0;
            if (j < C && d < D) {
                const double cp = (double)cent[c * D + d] - 128.0;
                const double p = rint(cp);
                if (!(p >= -128.0 && p <= 127.0)) {  // also true for NaN
                    bad = true;
                } else {
                    hb = (int)p;
                    e = fmax(e, fabs(cp - p));
                    q2 = fma(cp - p, cp - p, q2);  // cp - p is exact
                    n2 = fma(cp, cp, n2);
                }
            }
            q[d] = (int8_t)hb;
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            n2 += __shfl_xor(n2, o);
            q2 += __shfl_xor(q2, o);
            e = fmax(e, __shfl_xor(e, o));
        }
        if (__any(bad) && lane == 0) *q_bad1 = 1u;
        if (lane == 0) {
            negb1[j] = j < C ? -(int32_t)llrint(0.5 * n2) : kNoBias1;
            // non-negative floats order like their bit patterns; the read
            // skips the atomic once a larger residual is recorded
            const uint32_t eb = __float_as_uint(__double2float_ru(e));
            if (j < C && e > 0.0 && eb > __atomic_load_n(e_bits, __ATOMIC_RELAXED)) atomicMax(e_bits, eb);
            // the residual vector's norm, rounded up (2^-40 covers the
            // rounding of the sum of squares and of the square root)
            const uint32_t rb = __float_as_uint(__double2float_ru(sqrt(q2) * (1.0 + 0x1p-40)));
            if (r2_bits && j < C && q2 > 0.0 && rb > __atomic_load_n(r2_bits, __ATOMIC_RELAXED))
                atomicMax(r2_bits, rb);
        }
    }
}

// ------------------------------------------------------------ visiting order
// The single plane's scan inserts a score only when it comes near the row's
// best so far, so the cost of insertions follows how often that best rises.
// Centroids near the middle of the data score well for most rows; visiting
// them first raises every row's best early. The order is a heuristic (any
// order gives the same certified results): ascending ||c - mean||^2 with the
// mean taken over the centroids, in 15-bit buckets of the float's bits,
// stable by id within a bucket (a counting sort, the list build's kernels).

// Column sums of rows [b * R, (b + 1) * R): one thread per dimension, fp64,
// a fixed order (the result is the same on every run).
__global__ __launch_bounds__(128) void order1_part_kernel(const float *__restrict__ cent, int64_t C, int D,
                                                          double *__restrict__ part)
{
    const int d = threadIdx.x;
    if (d >= D) return;
    const int64_t c0 = (int64_t)blockIdx.x * kOrder1PartRows;
    const int64_t c1 = c0 + kOrder1PartRows < C ? c0 + kOrder1PartRows : C;
    double sum = 0.0;
#pragma unroll 8
    for (int64_t c = c0; c < c1; ++c) sum += (double)cent[c * D + d];
    part[(int64_t)blockIdx.x * D + d] = sum;
}

// One block per dimension: strided partial sums, then a tree in LDS (a fixed
// order).
__global__ __launch_bounds__(256) void order1_mean_kernel(const double *__restrict__ part, int64_t parts, int64_t C,
                                                          int D, float *__restrict__ mean)
{
    __shared__ double red[256];
    const int d = blockIdx.x;
    const int t = threadIdx.x;
    double sum = 0.0;
#pragma unroll 4
    for (int64_t b = t; b < parts; b += 256) sum += part[b * D + d];
    red[t] = sum;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) red[t] += red[t + w];
        __syncthreads();
    }
    if (t == 0) mean[d] = (float)(red[0] / (double)C);
}

// One wave per centroid: key = the top 15 bits of fl32(||c - mean||^2)
// (non-negative floats order like their bit patterns; NaN takes the last
// bucket).
__global__ __launch_bounds__(256) void order1_keys_kernel(const float *__restrict__ cent, int64_t C, int D,
                                                          const float *__restrict__ mean, int32_t *__restrict__ keys)
{
    const int lane = threadIdx.x & 63;
    const int64_t w0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t c = w0; c < C; c += nw) {
        float s2 = 0.0f;
        for (int d = lane; d < D; d += 64) {
            const float t = cent[c * D + d] - mean[d];
            s2 += t * t;
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) s2 += __shfl_xor(s2, o);
        if (lane == 0) {
            const uint32_t b = __float_as_uint(s2) >> 16;
            keys[c] = (int32_t)(b < (uint32_t)kOrder1Keys ? b : (uint32_t)kOrder1Keys - 1u);
        }
    }
}

// The fragments of one staged 32-centroid block of the single plane.
template <int DP>
struct Frags1 {
    i32x4 h[DP / 32];
};

template <int DP>
__device__ __forceinline__ void load_frags1(const char *Ar, Frags1<DP> &f)
{
#pragma unroll
    for (int k = 0; k < DP / 32; ++k) f.h[k] = *reinterpret_cast<const i32x4 *>(Ar + 32 * k);
}

// Group g (0..3) of a finished single-plane tile: registers 4g .. 4g + 3,
// centroids idp + 8g + e. st.t3 holds the keep threshold (scores at or
// below it cannot change the certificate's decision); only when some lane
// of the wave has a score above it are the four values inserted. The
// insertion is rare once a row has met its nearest centroids, so it is laid
// out off the straight-line path.
template <int g>
__device__ __forceinline__ void s1_group(const i32x16 &p, int idp, Top3i &st)
{
    const int v0 = p[4 * g], v1 = p[4 * g + 1], v2 = p[4 * g + 2], v3 = p[4 * g + 3];
    const int m = max4i(v0, v1, v2, v3);
    if (__builtin_expect(__any(m > st.t3), 0)) {
        // the group's best (the lowest position among equal scores) first
        const int e1 = v0 == m ? 0 : v1 == m ? 1 : v2 == m ? 2 : 3;
        top3i_push(st, m, idp + 8 * g + e1);
        int kb = max(halves_max(st.k1), st.ks);
        st.t3 = kb > kNoScore ? max(st.k3, kb - st.twoR - 1) : kNoScore;
        // the other three only when some lane still needs one of them
        const int r0 = e1 == 0 ? kNoScore : v0, r1 = e1 == 1 ? kNoScore : v1;
        const int r2 = e1 == 2 ? kNoScore : v2, r3 = e1 == 3 ? kNoScore : v3;
        if (__builtin_expect(__any(max4i(r0, r1, r2, r3) > st.t3), 0)) {
            top3i_push(st, r0, idp + 8 * g);
            top3i_push(st, r1, idp + 8 * g + 1);
            top3i_push(st, r2, idp + 8 * g + 2);
            top3i_push(st, r3, idp + 8 * g + 3);
            kb = max(halves_max(st.k1), st.ks);
            st.t3 = kb > kNoScore ? max(st.k3, kb - st.twoR - 1) : kNoScore;
        }
    }
}

// A whole finished tile of one row block (16 scores per lane) in one test:
// only when some lane of the wave has a score above its keep threshold are
// the four groups tested and inserted one by one.
__device__ __forceinline__ void s1_tile_test(const i32x16 &p, int idp, Top3i &st)
{
    const int m = max(max(max3i(max3i(p[0], p[1], p[2]), max3i(p[3], p[4], p[5]), max3i(p[6], p[7], p[8])),
                          max3i(max3i(p[9], p[10], p[11]), max3i(p[12], p[13], p[14]), p[15])),
                      kNoScore);
    if (__builtin_expect(__any(m > st.t3), 0)) {
        s1_group<0>(p, idp, st);
        s1_group<1>(p, idp, st);
        s1_group<2>(p, idp, st);
        s1_group<3>(p, idp, st);
    }
}

// K-step at which the previous block's row block rb is tested: one step
// after an even spread, so that the test does not read an accumulator whose
// last MFMA was issued just before (no wait states for its result).
template <int RB, int KS, int rb>
constexpr int s1_test_step()
{
    return rb * KS / RB + 1 < KS ? rb * KS / RB + 1 : KS - 1;
}

template <int RB, int T, int KS, int rb = 0>
__device__ __forceinline__ void s1_tests_at(const i32x16 (&p)[RB], int idp, Top3i (&st)[RB])
{
    if constexpr (rb < RB) {
        if constexpr (s1_test_step<RB, KS, rb>() == T) s1_tile_test(p[rb], idp, st[rb]);
        s1_tests_at<RB, T, KS, rb + 1>(p, idp, st);
    }
}

// K-steps T .. KS-1 of one 32-centroid block against the RB 32-row blocks of
// the wave (c[rb]: RB independent MFMA chains), all starting from the biases
// at T = 0. The epilogue of the previous block (p; ids from idp) runs between
// the K-steps, and each fragment register is refilled from the next block
// (nA, nB) as soon as its last MFMA has been issued.
template <int DP, int RB, int T = 0>
__device__ __forceinline__ void s1_block(Frags1<DP> &f, const i32x4 (&x)[RB][DP / 32], i32x16 &bias,
                                         i32x16 (&c)[RB], const i32x16 (&p)[RB], int idp, Top3i (&st)[RB],
                                         const char *nA, const int *nB)
{
    constexpr int KS = DP / 32;
    if constexpr (T < KS) {
        if constexpr (T == 0) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) c[rb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.h[0], x[rb][0], bias, 0, 0, 0);
            // an empty use of the biases after the MFMAs: none is their last
            // reader, so the compiler gives each a separate destination instead
            // of copying the biases into one accumulator first
            asm volatile("" ::"v"(bias));
            bias = load_bias(nB);
        } else {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) c[rb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.h[T], x[rb][T], c[rb], 0, 0, 0);
        }
        f.h[T] = *reinterpret_cast<const i32x4 *>(nA + 32 * T);
        s1_tests_at<RB, T, KS>(p, idp, st);
        __builtin_amdgcn_sched_barrier(0);
        s1_block<DP, RB, T + 1>(f, x, bias, c, p, idp, st, nA, nB);
    }
}

// Merges the two half-lanes of a row and certifies with the window T:
// settled rows get their label (two-way near-ties decided in fp64), the
// others are listed for the two-plane screen. The scan's ids are plane rows;
// one is used only when it names a real centroid, through the visiting
// order. Equal scores may rank in plane-row order, which never decides a
// label: a gap above T excludes ties, and the fp64 decision breaks them by
// centroid id.
__device__ __forceinline__ void s1_finish(const ScreenI8Args &a, int64_t row, bool rvalid, int h, const Top3i &st)
{
    Top3i o;
    o.k1 = __shfl_xor(st.k1, 32);
    o.k2 = __shfl_xor(st.k2, 32);
    o.k3 = __shfl_xor(st.k3, 32);
    o.i1 = __shfl_xor(st.i1, 32);
    o.i2 = __shfl_xor(st.i2, 32);
    const Top3i m = top3i_merge(st, o);
    int label = -1;
    bool refined = false;
    if (rvalid && h == 0) {
        const int64_t T = st.twoR;
        const bool ok1 = m.i1 >= 0 && m.i1 < a.ncent;
        const bool ok2 = m.i2 >= 0 && m.i2 < a.ncent;
        if (!a.force_rescreen && ok1) {
            const int c1 = a.ord1 ? (int)a.ord1[m.i1] : m.i1;
            if ((int64_t)m.k1 - (int64_t)m.k2 > T) {
                label = c1;
            } else if ((int64_t)m.k1 - (int64_t)m.k3 > T && ok2) {
                const int c2 = a.ord1 ? (int)a.ord1[m.i2] : m.i2;
                const uint8_t *x = a.rows + row * (int64_t)a.D;
                const double d1 = exact_dist(x, a.cent + (int64_t)c1 * a.D, a.D);
                const double d2 = exact_dist(x, a.cent + (int64_t)c2 * a.D, a.D);
                label = dist_lt(d2, c2, d1, c1) ? c2 : c1;
                refined = true;
            }
        }
        if (label >= 0) a.labels[row] = label;
    }
    // statistics and list slots: one atomic per wave; past the list's
    // capacity the two-plane screen takes every row
    const bool listed = rvalid && h == 0 && label < 0;
    wave_count(a.stats + kStatRefine2, refined);
    wave_count(a.stats + kStatRescreen, listed);
    const uint32_t slot = wave_append(const_cast<uint32_t *>(a.list_cnt), listed);
    if (listed && slot < (uint64_t)a.list_cap) const_cast<int32_t *>(a.list)[slot] = (int32_t)row;
}

// Row blocks of 32 rows per wave in the single-plane screen: three at
// DP = 128 (a block's fragments and biases feed three MFMA chains, within
// the register file), two below.
template <int DP>
constexpr int s1_row_blocks()
{
    return DP == 128 ? 3 : 2;
}

template <class F, int... I>
__device__ __forceinline__ void for_each_index(F &&f, std::integer_sequence<int, I...>)
{
    (f(std::integral_constant<int, I>{}), ...);
}

// One workgroup tile of the single-plane screen: W * 32 * RB rows against
// every centroid. A block's fragments feed every row block of the wave;
// blocks alternate between the accumulator sets A and B, and each block's
// K-steps carry the epilogue of the block before it. A staged chunk holds
// kS1Sub sub-chunks of 64 centroids in the two-plane tile's LDS layout (2 *
// kS1Sub blocks of 32 per workgroup barrier); two chunk buffers alternate.
// The barrier before the last block of chunk j makes chunk j + 1 visible
// (that block refills its fragments from it) and then chunk j + 2 is
// fetched into chunk j's buffer, which no wave reads any more.
template <int DP, int W>
__device__ void screen1_tile(const ScreenI8Args &a, int64_t tile, char *__restrict__ lds)
{
    static_assert(DP <= 128, "the single-plane screen keeps several row blocks per wave");
    constexpr int RB = s1_row_blocks<DP>();
    constexpr int NT = W * 64;
    using St = QStager<DP, NT, 1>;
    constexpr int CS = (St::kBytes + 15) / 16 * 16;  // one 64-centroid sub-chunk
    constexpr int SB = kS1Sub * CS;                  // one staged chunk
    constexpr int NB = 2 * kS1Sub;                   // 32-centroid blocks per staged chunk
    constexpr int BLK = 32 * St::kPitch;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int h = lane >> 5;
    const int jl = lane & 31;
    const int64_t row0 = tile * (W * 32 * RB);

    i32x4 xf[RB][DP / 32];
    uint32_t l1[RB];
    load_rows<DP, RB>(a.rows, row0, a.nrows, a.D, wave, jl, h, xf, l1);

    // T = ceil(2 min(E ||x'||_1, R2 ||x'||_2) + 1) + 1 >= 2W (E and R2
    // rounded up; one unit of margin): |x'.(c' - H1)| is at most both
    // E ||x'||_1 and, by Cauchy-Schwarz, ||x'||_2 ||c' - H1||_2 <= ||x'||_2 R2
    const double E = (double)__uint_as_float(*a.e_bits);
    const double R2 = a.r2_bits ? (double)__uint_as_float(*a.r2_bits) : __builtin_huge_val();
    Top3i st[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        l1[rb] += __shfl_xor(l1[rb], 32);
        int q2 = 0;  // ||x'||_2^2 (exact; the lane's half of the dimensions, then both)
#pragma unroll
        for (int k = 0; k < DP / 32; ++k)
#pragma unroll
            for (int w = 0; w < 4; ++w) q2 = __builtin_amdgcn_sdot4(xf[rb][k][w], xf[rb][k][w], q2, false);
        q2 += __shfl_xor(q2, 32);
        const double wb = fmin(E * (double)l1[rb], sqrt((double)q2) * R2);
        const int T = (int)ceil(2.0 * wb) + 2;
        st[rb] = Top3i{kNoScore, kNoScore, kNoScore, -1, -1, kNoScore, T, kNoScore};
    }
    // A hinted label (an earlier step's) starts the keep threshold from that
    // centroid's exact score s_h <= the row's best: every score the
    // certificate needs (at or above best - T) still lies above s_h - T - 1,
    // and the scan meets far fewer new bests. The score is the plane row's
    // dot with x' (the two half-lanes' halves added) plus its bias, the same
    // integer the MFMA chain produces.
    if (a.hint) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int64_t row = row0 + (wave * RB + rb) * 32 + jl;
            const int hl = row < a.nrows ? a.hint[row] : -1;
            const bool ok = hl >= 0 && hl < a.ncent;
            int dot = 0;
            int hp = 0;  // the hinted centroid's plane row
            if (ok) {
                hp = a.pos1 ? a.pos1[hl] : hl;
                const int8_t *qr = a.qc1 + (int64_t)hp * DP + 16 * h;
#pragma unroll
                for (int k = 0; k < DP / 32; ++k) {
                    const i32x4 v = *reinterpret_cast<const i32x4 *>(qr + 32 * k);
#pragma unroll
                    for (int w = 0; w < 4; ++w) dot = __builtin_amdgcn_sdot4(v[w], xf[rb][k][w], dot, false);
                }
            }
            dot += __shfl_xor(dot, 32);
            if (ok) {
                st[rb].ks = dot + a.negb1[hp];
                st[rb].t3 = st[rb].ks - st[rb].twoR - 1;
            }
        }
    }

    const char *A0 = lds + jl * St::kPitch + 16 * h;
    const char *B0 = lds + St::kBias + 16 * h;
    const int idh = 4 * h;
    const int nch = (int)a.nchunks;
    // block b (0 .. NB - 1) of staged chunk jj
    auto abuf = [&](int jj, int b) { return A0 + (jj & 1) * SB + (b >> 1) * CS + (b & 1) * BLK; };
    auto bbuf = [&](int jj, int b) {
        return reinterpret_cast<const int *>(B0 + (jj & 1) * SB + (b >> 1) * CS) + 32 * (b & 1);
    };

    St q;
    q.init();
    auto fetch = [&](int jj) {
        char *buf = lds + (jj & 1) * SB;
#pragma unroll
        for (int u = 0; u < kS1Sub; ++u)
            q.fetch(a.qc1, a.negb1, (int64_t)jj * kS1Chunk + u * kQChunk, a.cpad, buf + u * CS);
    };
    fetch(0);
    __syncthreads();
    fetch(1);

    // set B starts as a block of lowest scores: the first epilogue inserts nothing
    i32x16 sa[RB], sb[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sb[rb][r] = kNoScore;
    i32x16 bias = load_bias(bbuf(0, 0));
    Frags1<DP> f;
    load_frags1<DP>(abuf(0, 0), f);

    // block b of chunk jj into set A (b even) or B while the other set (the
    // block before) drains; fragments refill from the next block
    auto block = [&](int jj, auto bc) {
        constexpr int b = decltype(bc)::value;
        const char *nA = b + 1 < NB ? abuf(jj, b + 1) : abuf(jj + 1, 0);
        const int *nB = b + 1 < NB ? bbuf(jj, b + 1) : bbuf(jj + 1, 0);
        const int idp = idh + jj * kS1Chunk + 32 * b - 32;
        if constexpr (b % 2 == 0)
            s1_block<DP, RB>(f, xf, bias, sa, sb, idp, st, nA, nB);
        else
            s1_block<DP, RB>(f, xf, bias, sb, sa, idp, st, nA, nB);
    };
    for (int j = 0;; ++j) {
        for_each_index([&](auto bc) { block(j, bc); }, std::make_integer_sequence<int, NB - 1>{});
        __syncthreads();
        fetch(j + 2);
        block(j, std::integral_constant<int, NB - 1>{});
        if (j + 1 == nch) break;
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) s1_tile_test(sb[rb], idh + (nch - 1) * kS1Chunk + 32 * (NB - 1), st[rb]);

#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int64_t row = row0 + (wave * RB + rb) * 32 + jl;
        s1_finish(a, row, row < a.nrows, h, st[rb]);
    }
}

template <int DP, int W>
__global__ __launch_bounds__(W * 64, 2) void screen1_kernel(ScreenI8Args a)
{
    using St = QStager<DP, W * 64, 1>;
    constexpr int CS = (St::kBytes + 15) / 16 * 16;
    __shared__ __attribute__((aligned(16))) char lds[2 * kS1Sub * CS];
    if (*a.q_bad || *a.q_bad1) return;  // another screen takes every row
    constexpr int rows_per_tile = W * 32 * s1_row_blocks<DP>();
    const int64_t ntiles = (a.nrows + rows_per_tile - 1) / rows_per_tile;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        screen1_tile<DP, W>(a, tile, lds);
        __syncthreads();
    }
}

template <int DP>
hipError_t launch_s1(const ScreenI8Args &a, int num_cus, hipStream_t s)
{
    constexpr int W = 8;
    constexpr int rows_per_tile = W * 32 * s1_row_blocks<DP>();
    const int64_t ntiles = (a.nrows + rows_per_tile - 1) / rows_per_tile;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(ntiles, (int64_t)num_cus));
    hipLaunchKernelGGL((screen1_kernel<DP, W>), dim3(grid), dim3(W * 64), 0, s, a);
    return hipGetLastError();
}

}  // namespace

int64_t quantized_pad(int64_t C) { return (C + kQChunk - 1) / kQChunk * kQChunk; }

int64_t quantized_pad1(int64_t C) { return (C + kS1Chunk - 1) / kS1Chunk * kS1Chunk; }

hipError_t launch_quantize_centroids(const float *cent, int64_t C, int D, int DP, int8_t *qc, int32_t *negb,
                                     uint32_t *q_bad, hipStream_t s, const uint32_t *skip)
{
    const int64_t cpad = quantized_pad(C);
    const int64_t blocks = std::min<int64_t>((cpad + 3) / 4, 8192);
    hipLaunchKernelGGL(quantize_kernel, dim3((unsigned)blocks), dim3(256), 0, s, cent, C, D, DP, cpad, qc, negb,
                       q_bad, skip);
    return hipGetLastError();
}

hipError_t launch_quantize_centroids1(const float *cent, int64_t C, int D, int DP, int8_t *q1, int32_t *negb1,
                                      uint32_t *q_bad1, uint32_t *e_bits, uint32_t *r2_bits, hipStream_t s,
                                      const uint32_t *ord, int32_t *pos)
{
    const int64_t cpad = quantized_pad1(C);
    const int64_t blocks = std::min<int64_t>((cpad + 3) / 4, 65536);
    hipLaunchKernelGGL(quantize1_kernel, dim3((unsigned)blocks), dim3(256), 0, s, cent, C, D, DP, cpad, q1, negb1,
                       q_bad1, e_bits, r2_bits, ord, pos);
    return hipGetLastError();
}

int64_t order1_parts(int64_t C) { return (C + kOrder1PartRows - 1) / kOrder1PartRows; }

hipError_t launch_order1_keys(const float *cent, int64_t C, int D, double *part, float *mean, int32_t *keys,
                              hipStream_t s)
{
    if (C <= 0) return hipSuccess;
    if (D > 128) return hipErrorInvalidValue;  // the single plane's dimensions
    const int64_t parts = order1_parts(C);
    hipLaunchKernelGGL(order1_part_kernel, dim3((unsigned)parts), dim3(128), 0, s, cent, C, D, part);
    hipLaunchKernelGGL(order1_mean_kernel, dim3((unsigned)D), dim3(256), 0, s, part, parts, C, D, mean);
    const int64_t blocks = std::min<int64_t>((C + 3) / 4, 65536);
    hipLaunchKernelGGL(order1_keys_kernel, dim3((unsigned)blocks), dim3(256), 0, s, cent, C, D, mean, keys);
    return hipGetLastError();
}

hipError_t launch_screen_i8_single(int DP, const ScreenI8Args &a0, int num_cus, hipStream_t s)
{
    if (a0.nrows <= 0) return hipSuccess;
    // the single plane is padded to whole staged chunks
    ScreenI8Args a = a0;
    a.cpad = quantized_pad1(a0.ncent);
    a.nchunks = a.cpad / kS1Chunk;
    switch (DP) {
    case 32: return launch_s1<32>(a, num_cus, s);
    case 64: return launch_s1<64>(a, num_cus, s);
    case 96: return launch_s1<96>(a, num_cus, s);
    case 128: return launch_s1<128>(a, num_cus, s);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_screen_i8(int DP, const ScreenI8Args &a, int num_cus, hipStream_t s)
{
    if (a.nrows <= 0) return hipSuccess;
    return launch_i8_w<8>(DP, a, num_cus, s);
}

hipError_t launch_route_i8_check(const float *queries, int64_t nq, int D, uint32_t *off, hipStream_t s)
{
    if (nq <= 0) return hipSuccess;
    const int64_t blocks = std::min<int64_t>((nq + 3) / 4, 1024);
    hipLaunchKernelGGL(route_i8_check_kernel, dim3((unsigned)blocks), dim3(256), 0, s, queries, nq, D, off);
    return hipGetLastError();
}

hipError_t launch_route_i8_bound(const float *queries, int64_t nq, int D, const uint32_t *q_bad, uint32_t *off,
                                 float *qbound, hipStream_t s)
{
    if (nq <= 0) return hipSuccess;
    const int64_t blocks = std::min<int64_t>((nq + 3) / 4, 65536);
    hipLaunchKernelGGL(route_i8_bound_kernel, dim3((unsigned)blocks), dim3(256), 0, s, queries, nq, D, q_bad, off,
                       qbound);
    return hipGetLastError();
}

hipError_t launch_route_i8(int mode, int DP, const RouteI8Args &a, int num_cus, hipStream_t s)
{
    if (a.nq <= 0 || a.nchunks <= 0) return hipSuccess;
    return mode == kRouteKeys ? launch_route_i8_mode<kRouteKeys>(DP, a, num_cus, s)
                              : launch_route_i8_mode<kRouteFilter>(DP, a, num_cus, s);
}

}  // namespace ivf

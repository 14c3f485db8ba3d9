// Fused fp32-MFMA distance screening for gfx950.
//
// Computes, for a tile of rows x (queries or data vectors) against a range of
// centroids c, the screening key
//     key(x, c) = fl(fl32(||c||^2) - 2 * acc(x, c)),   acc = fp32 MFMA dot product,
// i.e. Eq. (6) of the paper without the per-row constant ||x||^2 (it does not
// change the order within a row), and consumes the keys in one of three
// epilogues without ever writing the distance matrix:
//   kModeKeys    write the keys (used for the routing threshold sample);
//   kModeFilter  keep (key, id) whenever key <= tau(row) (routing candidates);
//   kModeTop1    keep the three smallest keys per row (assignment), then
//                certify the nearest centroid with a rounding-error bound and
//                settle near-ties by exact fp64 re-evaluation.
//
// MFMA: v_mfma_f32_32x32x2_f32. A operand = centroids (M = 32 rows of a
// chunk), B operand = rows (N = 32 rows of a wave), K split into two halves:
// lane half h contributes dimensions [h*DP/2, (h+1)*DP/2), so every lane walks
// contiguous memory and one ds_read_b128 feeds four K-steps. Output layout of
// the 32x32 accumulator: lane l holds column l % 32 (one row x), register r
// holds centroid 8*(r/4) + 4*(l/32) + r%4 of the block.
#include "ivf_internal.h"
#include "exact.h"
#include "wave_ops.h"

#include <math.h>

#include <algorithm>

namespace ivf {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kInf = __builtin_huge_valf();

__device__ __forceinline__ bool key_lt(float ka, int ia, float kb, int ib)
{
    return ka < kb || (ka == kb && ia < ib);
}

// Lane's half-row as fp32 B fragments: b[s] = x[row][h*KH + s], zero padded.
template <int DP>
__device__ __forceinline__ void load_row(const float *__restrict__ X, int64_t row, bool valid,
                                         int D, int h, float (&b)[DP / 2])
{
    constexpr int KH = DP / 2;
    const float *p = X + row * (int64_t)D + h * KH;
#pragma unroll
    for (int t = 0; t < KH / 4; ++t) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (valid && h * KH + 4 * t < D) v = *reinterpret_cast<const float4 *>(p + 4 * t);
        b[4 * t + 0] = v.x;
        b[4 * t + 1] = v.y;
        b[4 * t + 2] = v.z;
        b[4 * t + 3] = v.w;
    }
}

template <int DP>
__device__ __forceinline__ void load_row(const uint8_t *__restrict__ X, int64_t row, bool valid,
                                         int D, int h, float (&b)[DP / 2])
{
    constexpr int KH = DP / 2;
    const uint8_t *p = X + row * (int64_t)D + h * KH;
#pragma unroll
    for (int t = 0; t < KH / 4; ++t) {
        uint32_t w = 0;
        if (valid && h * KH + 4 * t < D) w = *reinterpret_cast<const uint32_t *>(p + 4 * t);
        b[4 * t + 0] = (float)(w & 0xFFu);
        b[4 * t + 1] = (float)((w >> 8) & 0xFFu);
        b[4 * t + 2] = (float)((w >> 16) & 0xFFu);
        b[4 * t + 3] = (float)(w >> 24);
    }
}

// Stages chunks of kChunk centroids (and their norms) from HBM/L2 into LDS.
// Loads go through a buffer resource that spans only the chunk's valid rows:
// reads past it return zeros, which gives the zero padding of a ragged last
// chunk (and of the dimensions D..DP-1, whose offsets are pointed out of
// range) without per-element bounds arithmetic. Per thread, the byte offsets
// within a chunk and the LDS slots are fixed, so a chunk costs kVec loads.
template <int DP, int NT>
struct Stager {
    static constexpr int V4 = DP / 4;
    static constexpr int kVec = kChunk * V4 / NT;  // float4 per thread
    static constexpr int kOut = 1 << 30;           // an offset past any chunk
    int goff[kVec];  // byte offset of this thread's float4 in the chunk
    int loff[kVec];  // float offset of its slot in a staged chunk
    float4 v[kVec];
    float n;    // norm of centroid threadIdx.x of the chunk (threads < kChunk)
    int valid;  // rows of the chunk below c_end

    __device__ __forceinline__ void init(int D)
    {
#pragma unroll
        for (int i = 0; i < kVec; ++i) {
            const int idx = threadIdx.x + i * NT;
            const int rr = idx / V4, c4 = idx - rr * V4;
            goff[i] = 4 * c4 < D ? (rr * D + 4 * c4) * 4 : kOut;
            loff[i] = rr * (DP + 4) + 4 * c4;
        }
    }

    __device__ __forceinline__ void fetch(const float *__restrict__ cent, const float *__restrict__ cnorm,
                                          int64_t cbase, int64_t c_end, int D)
    {
        const int64_t left = c_end - cbase;  // <= 0 past the range: nothing is read
        valid = (int)(left < 0 ? 0 : left < kChunk ? left : kChunk);
        const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(cent + cbase * D), (short)0, valid * D * 4, 0x00020000);
#pragma unroll
        for (int i = 0; i < kVec; ++i)
            v[i] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rc, goff[i], 0, 0));
        if (threadIdx.x < kChunk) {
            const __amdgpu_buffer_rsrc_t rn = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<float *>(cnorm + cbase), (short)0, valid * 4, 0x00020000);
            n = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rn, threadIdx.x * 4, 0, 0));
        }
    }

    // NEG_HALF stages -||c||^2/2 instead of ||c||^2 (exact: a power-of-two scaling).
    template <bool NEG_HALF = false>
    __device__ __forceinline__ void store(float *__restrict__ lc, float *__restrict__ ln) const
    {
#pragma unroll
        for (int i = 0; i < kVec; ++i) *reinterpret_cast<float4 *>(lc + loff[i]) = v[i];
        if (threadIdx.x < kChunk) {
            // padded rows get an infinite norm, so they never win a selection
            const float m = (int)threadIdx.x < valid ? n : kInf;
            ln[threadIdx.x] = NEG_HALF ? -0.5f * m : m;
        }
    }
};

// Per-row state of the top-1 epilogue: the three smallest keys, ids of two.
struct Top3 {
    float k1, k2, k3;
    int i1, i2;
};

// Merges this lane's list with the partner lane's (both sorted by (key, id)).
__device__ __forceinline__ Top3 top3_merge(Top3 a, Top3 b)
{
    if (key_lt(b.k1, b.i1, a.k1, a.i1)) {
        Top3 t = a;
        a = b;
        b = t;
    }
    Top3 m;
    m.k1 = a.k1;
    m.i1 = a.i1;
    if (key_lt(b.k1, b.i1, a.k2, a.i2)) {
        m.k2 = b.k1;
        m.i2 = b.i1;
        m.k3 = fminf(a.k2, b.k2);
    } else {
        m.k2 = a.k2;
        m.i2 = a.i2;
        m.k3 = fminf(a.k3, b.k1);
    }
    return m;
}

// Rigorous bound on |key - (||c||^2 - 2 x.c)| for every centroid c:
// gamma_{DP+2} * (M + 2 ||x|| sqrt(M)), M >= max ||c||^2 (slightly inflated to
// cover the fp32 rounding of the stored norms), plus an absolute term for
// possible flushes of subnormal products.
__device__ __forceinline__ double key_bound(double coef, uint32_t mc2_bits, double xn2)
{
    const double M = (double)__uint_as_float(mc2_bits) * (1.0 + 0x1p-20);
    return coef * (M + 2.0 * sqrt(xn2 * (1.0 + 0x1p-40)) * sqrt(M)) + 0x1p-100;
}

// Survivors of the filter epilogue: a lane whose group of four values holds
// one at or above its threshold queues the whole group (the four values and
// the first id) in LDS, entry i of lane l of a wave at [wave][i][l] so that
// the lanes of one store hit consecutive addresses; one 16-byte and one
// 4-byte store per group, no per-value work on the MFMA path. A flush (before
// a lane's queue would overflow, and at the end of a range) keeps the values
// that pass: a lane's entries all belong to its own row, so one atomic on the
// row's counter reserves room for all of them.
template <int W>
constexpr int filter_queue_cap()
{
    return W == 8 ? 8 : 4;  // 80 KiB (8 waves) or 20 KiB (4 waves, wide rows)
}

template <int W>
struct FilterQueue {
    float4 v[W][filter_queue_cap<W>()][64];  // the group's four values
    int id[W][filter_queue_cap<W>()][64];    // id of its first value
};

// ---------------------------------------------------------------- top-1 path
//
// The accumulators start from -fl32(||c||^2)/2 (staged in LDS instead of the
// norms), so after the MFMAs an accumulator holds v = -key/2 exactly (scaling
// by a power of two is exact) and the key never needs to be formed: the three
// smallest keys are the three largest v. The epilogue of chunk j-1 (the
// branch-free three-largest update) is interleaved with the MFMAs of chunk j,
// so the matrix pipe keeps running while a wave consumes the previous
// accumulators. Centroid data stays double-buffered; the norms take three
// LDS slots because the first MFMAs of chunk j+1 read its norms while a slower
// wave may still be loading chunk j's.

// Inserts (v, id) into a lane's three largest values without branches (a
// value <= v3 leaves the state unchanged): with v1 >= v2 >= v3,
// med3(v, v2, v3) is the new third value and med3(v, v1, v2) the new second.
// Strict comparisons keep the lower id on equal values because a lane visits
// ids in ascending order.
__device__ __forceinline__ void top3_push(Top3 &t, float v, int id)
{
    const bool gt1 = v > t.k1;
    const bool gt2 = v > t.k2;
    t.k3 = __builtin_amdgcn_fmed3f(v, t.k2, t.k3);
    t.k2 = __builtin_amdgcn_fmed3f(v, t.k1, t.k2);
    t.k1 = gt1 ? v : t.k1;
    const int j2 = gt2 ? id : t.i2;
    t.i2 = gt1 ? t.i1 : j2;
    t.i1 = gt1 ? id : t.i1;
}

// max(a, b, c, d) in two v_maximum3_f32. fmaxf would first canonicalise each
// operand (an extra instruction per value); maximum differs from it only for
// NaN and for -0 against +0, and the values here are never NaN while the
// compares that follow treat -0 and +0 alike. Being ordinary compiler
// operations, the reads of MFMA results get their wait states from the
// compiler's hazard recognizer.
__device__ __forceinline__ float max4(float a, float b, float c, float d)
{
    return __builtin_elementwise_maximum(__builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c), d);
}

// Group G (0..7) of the previous chunk's accumulators: block rb = G / 4 (p0
// or p1), registers 4g..4g+3 with g = G % 4, centroids rb*32 + 8g + 4h + e.
// Fp32 MFMA and other vector instructions share the SIMD, so every vector
// instruction here costs matrix throughput: the group is first tested as a
// whole (two instructions), and the insertion runs only when some lane of the
// wave holds a value above its third largest.
template <int G>
__device__ __forceinline__ void top1_group(const f32x16 &p0, const f32x16 &p1, int idp, Top3 &st)
{
    constexpr int rb = G >> 2;
    constexpr int g = G & 3;
    constexpr int off = rb * 32 + 8 * g;  // centroid offset (h excluded)
    const f32x16 &p = rb ? p1 : p0;
    const float m = max4(p[4 * g], p[4 * g + 1], p[4 * g + 2], p[4 * g + 3]);
    if (__any(m > st.k3)) {
        top3_push(st, p[4 * g + 0], idp + off + 0);
        top3_push(st, p[4 * g + 1], idp + off + 1);
        top3_push(st, p[4 * g + 2], idp + off + 2);
        top3_push(st, p[4 * g + 3], idp + off + 3);
    }
    // keeps the test at this point of the MFMA stream (the compiler would
    // otherwise sink the whole epilogue below the chunk's last MFMA)
    asm volatile("" : "+v"(st.k1), "+v"(st.k2), "+v"(st.k3), "+v"(st.i1), "+v"(st.i2));
}

template <int G, int T, int KB>
__device__ __forceinline__ void top1_groups_at(const f32x16 &p0, const f32x16 &p1, int idp, Top3 &st)
{
    if constexpr (G < 8) {
        if constexpr (G * KB / 8 == T) top1_group<G>(p0, p1, idp, st);
        top1_groups_at<G + 1, T, KB>(p0, p1, idp, st);
    }
}

// MFMAs of one staged chunk into (c0, c1); with EP, the epilogue of the
// previous chunk (p0, p1, first id idp) spread over the K-blocks.
template <int DP, bool EP, int T = 0>
__device__ __forceinline__ void top1_kblocks(const float *A0, const float *A1, const float (&b)[DP / 2],
                                             f32x16 &c0, f32x16 &c1, float4 a0, float4 a1,
                                             const f32x16 &p0, const f32x16 &p1, int idp, Top3 &st)
{
    constexpr int KB = DP / 8;
    if constexpr (T < KB) {
        float4 n0 = a0, n1 = a1;
        if constexpr (T + 1 < KB) {
            n0 = *reinterpret_cast<const float4 *>(A0 + 4 * (T + 1));
            n1 = *reinterpret_cast<const float4 *>(A1 + 4 * (T + 1));
        }
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0.x, b[4 * T + 0], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1.x, b[4 * T + 0], c1, 0, 0, 0);
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0.y, b[4 * T + 1], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1.y, b[4 * T + 1], c1, 0, 0, 0);
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0.z, b[4 * T + 2], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1.z, b[4 * T + 2], c1, 0, 0, 0);
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0.w, b[4 * T + 3], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1.w, b[4 * T + 3], c1, 0, 0, 0);
        if constexpr (EP) top1_groups_at<0, T, KB>(p0, p1, idp, st);
        __builtin_amdgcn_sched_barrier(0);
        top1_kblocks<DP, EP, T + 1>(A0, A1, b, c0, c1, n0, n1, p0, p1, idp, st);
    }
}

// One chunk: A0 = this lane's row of the staged centroids, Nh = the staged
// -||c||^2/2 values of the chunk offset by 4h.
template <int DP, bool EP>
__device__ __forceinline__ void mfma_chunk(const float *A0, const float *Nh, const float (&b)[DP / 2],
                                           f32x16 &c0, f32x16 &c1, const f32x16 &p0, const f32x16 &p1,
                                           int idp, Top3 &st)
{
    const float *A1 = A0 + 32 * (DP + 4);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const float4 u = *reinterpret_cast<const float4 *>(Nh + 8 * g);
        const float4 w = *reinterpret_cast<const float4 *>(Nh + 32 + 8 * g);
        c0[4 * g + 0] = u.x;
        c0[4 * g + 1] = u.y;
        c0[4 * g + 2] = u.z;
        c0[4 * g + 3] = u.w;
        c1[4 * g + 0] = w.x;
        c1[4 * g + 1] = w.y;
        c1[4 * g + 2] = w.z;
        c1[4 * g + 3] = w.w;
    }
    const float4 a0 = *reinterpret_cast<const float4 *>(A0);
    const float4 a1 = *reinterpret_cast<const float4 *>(A1);
    top1_kblocks<DP, EP>(A0, A1, b, c0, c1, a0, a1, p0, p1, idp, st);
}

template <int G = 0>
__device__ __forceinline__ void top1_drain(const f32x16 &p0, const f32x16 &p1, int idp, Top3 &st)
{
    if constexpr (G < 8) {
        top1_group<G>(p0, p1, idp, st);
        top1_drain<G + 1>(p0, p1, idp, st);
    }
}

// Merges the two half-lanes of each row, certifies the nearest centroid with
// the rounding-error bound, settles two-way near-ties exactly in fp64 and
// queues everything else for the full fp64 fallback.
template <typename XT>
__device__ __forceinline__ void top1_finish(const ScreenArgs &a, int64_t row, bool rvalid, int h,
                                            double xpart, const Top3 &st)
{
    const double xn2 = xpart + __shfl_xor(xpart, 32);
    Top3 o;
    o.k1 = __shfl_xor(st.k1, 32);
    o.k2 = __shfl_xor(st.k2, 32);
    o.k3 = __shfl_xor(st.k3, 32);
    o.i1 = __shfl_xor(st.i1, 32);
    o.i2 = __shfl_xor(st.i2, 32);
    const Top3 m = top3_merge(st, o);
    int label = -1;
    bool refined = false;
    if (rvalid && h == 0) {
        const double B2 = 2.0 * key_bound(a.bound_coef, *a.mc2_bits, xn2);
        // a centroid id is used only when it names a real centroid; any other
        // state sends the row to the exact fallback scan
        const bool ok1 = m.i1 >= a.c_begin && m.i1 < a.c_end;
        const bool ok2 = m.i2 >= a.c_begin && m.i2 < a.c_end;
        if (!a.force_fallback && ok1) {
            if ((double)m.k2 > (double)m.k1 + B2) {
                label = m.i1;
            } else if ((double)m.k3 > (double)m.k1 + B2 && ok2) {
                const XT *x = reinterpret_cast<const XT *>(a.rows) + row * (int64_t)a.D;
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

template <int DP, int W, typename XT>
__device__ void screen_top1(const ScreenArgs &a, int64_t tile, float *__restrict__ lds_c,
                            float *__restrict__ lds_n)
{
    constexpr int NT = W * 64;
    constexpr int KH = DP / 2;
    constexpr int CS = kChunk * (DP + 4);  // floats per staged chunk
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int h = lane >> 5;
    const int jl = lane & 31;
    const int64_t row = tile * (32 * W) + wave * 32 + jl;
    const bool rvalid = row < a.nrows;

    float b[KH];
    load_row<DP>(reinterpret_cast<const XT *>(a.rows), row, rvalid, a.D, h, b);
    // this lane's half of ||x||^2 (exact fp32 values, fp64 sum) for the bound
    double xpart = 0.0;
#pragma unroll
    for (int s = 0; s < KH; ++s) xpart = fma((double)b[s], (double)b[s], xpart);

    Top3 st{-kInf, -kInf, -kInf, -1, -1};  // three largest v = -key/2
    const int nch = (int)a.nchunks;         // < 2^25: centroid ids fit int32
    const float *Ab = lds_c + jl * (DP + 4) + h * KH;  // this lane's A row in buffer 0
    const float *Nb = lds_n + 4 * h;
    const int idh = (int)a.c_begin + 4 * h;

    Stager<DP, NT> cr;
    cr.init(a.D);
    cr.fetch(a.cent, a.cnorm, a.c_begin, a.c_end, a.D);
    cr.template store<true>(lds_c, lds_n);
    __syncthreads();

    // chunk j of the range sits in buffer j & 1 (data and -||c||^2/2)
    // (the chunk after the last one is fetched and staged too: its loads read
    // nothing and return zeros, which keeps every load unconditional)
    auto step = [&](int j, f32x16 &c0, f32x16 &c1, const f32x16 &p0, const f32x16 &p1) {
        cr.fetch(a.cent, a.cnorm, a.c_begin + (int64_t)(j + 1) * kChunk, a.c_end, a.D);
        const int bj = j & 1;
        mfma_chunk<DP, true>(Ab + bj * CS, Nb + bj * kChunk, b, c0, c1, p0, p1, idh + (j - 1) * kChunk, st);
        cr.template store<true>(lds_c + (bj ^ 1) * CS, lds_n + (bj ^ 1) * kChunk);
        __syncthreads();
    };

    f32x16 x0, x1, y0, y1;
    cr.fetch(a.cent, a.cnorm, a.c_begin + kChunk, a.c_end, a.D);
    mfma_chunk<DP, false>(Ab, Nb, b, x0, x1, x0, x1, 0, st);
    cr.template store<true>(lds_c + CS, lds_n + kChunk);
    __syncthreads();
    int j = 1;
    for (; j + 1 < nch; j += 2) {
        step(j, y0, y1, x0, x1);
        step(j + 1, x0, x1, y0, y1);
    }
    if (j < nch) {
        step(j, y0, y1, x0, x1);
        top1_drain(y0, y1, idh + j * kChunk, st);
    } else {
        top1_drain(x0, x1, idh + (j - 1) * kChunk, st);
    }
    // back to keys: key = -2 v exactly, ascending
    st.k1 *= -2.0f;
    st.k2 *= -2.0f;
    st.k3 *= -2.0f;
    top1_finish<XT>(a, row, rvalid, h, xpart, st);
}

// ------------------------------------------------------------ filter path
//
// The filter's epilogue runs like the top-1 one: the previous chunk's
// accumulators are tested group by group between the MFMAs of the current
// chunk. A group of four values is tested as a whole (max and one compare);
// only when some lane of the wave holds a survivor are its values staged.
template <int W>
struct FilterState {
    uint32_t *cand_cnt;  // the candidate lists (copies of the launch
    uint2 *cand;         // arguments: a pointer to the arguments themselves
    int L;               // would put them in private memory)
    FilterQueue<W> *q;
    int64_t row;  // this lane's row
    float tv;     // keep v >= tv
    int qn;       // entries in this lane's queue
    int wave, lane;
};

// Moves every lane's queued values that pass into its row's candidate list:
// one atomic per lane reserves their number of slots (entries past the
// list's capacity are dropped; the selection sees the count and sends the
// row to the fallback). Keys are -2v, exactly.
template <int W>
__device__ __forceinline__ void filter_flush(FilterState<W> &fs)
{
    if (fs.qn > 0) {
        uint32_t n = 0;
        for (int i = 0; i < fs.qn; ++i) {
            const float4 v = fs.q->v[fs.wave][i][fs.lane];
            n += (v.x >= fs.tv) + (v.y >= fs.tv) + (v.z >= fs.tv) + (v.w >= fs.tv);
        }
        const uint32_t slot = atomicAdd(fs.cand_cnt + fs.row, n);
        uint2 *dst = fs.cand + fs.row * fs.L;
        uint32_t k = slot;
        for (int i = 0; i < fs.qn; ++i) {
            const float4 v4 = fs.q->v[fs.wave][i][fs.lane];
            const int id = fs.q->id[fs.wave][i][fs.lane];
            const float va[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (va[e] >= fs.tv) {
                    if (k < (uint32_t)fs.L) dst[k] = make_uint2(__float_as_uint(-2.0f * va[e]), (uint32_t)(id + e));
                    ++k;
                }
            }
        }
    }
    fs.qn = 0;
}

template <int G, int W>
__device__ __forceinline__ void filter_group(const f32x16 &p0, const f32x16 &p1, int idp, FilterState<W> &fs)
{
    constexpr int rb = G >> 2;
    constexpr int g = G & 3;
    constexpr int off = rb * 32 + 8 * g;  // centroid offset (h excluded)
    const f32x16 &p = rb ? p1 : p0;
    const float m = max4(p[4 * g], p[4 * g + 1], p[4 * g + 2], p[4 * g + 3]);
    const bool pass = m >= fs.tv;
    if (__any(pass)) {
        if (__any(fs.qn >= filter_queue_cap<W>())) filter_flush(fs);
        if (pass) {
            fs.q->v[fs.wave][fs.qn][fs.lane] = make_float4(p[4 * g], p[4 * g + 1], p[4 * g + 2], p[4 * g + 3]);
            fs.q->id[fs.wave][fs.qn][fs.lane] = idp + off;
            ++fs.qn;
        }
    }
    // keeps the test at this point of the MFMA stream
    asm volatile("" : "+v"(fs.tv));
}

template <int G, int T, int KB, int W>
__device__ __forceinline__ void filter_groups_at(const f32x16 &p0, const f32x16 &p1, int idp, FilterState<W> &fs)
{
    if constexpr (G < 8) {
        if constexpr (G * KB / 8 == T) filter_group<G, W>(p0, p1, idp, fs);
        filter_groups_at<G + 1, T, KB, W>(p0, p1, idp, fs);
    }
}

template <int DP, bool EP, int W, int T = 0>
__device__ __forceinline__ void filter_kblocks(const float *A0, const float *A1, const float (&b)[DP / 2],
                                               f32x16 &c0, f32x16 &c1, float4 a0, float4 a1,
                                               const f32x16 &p0, const f32x16 &p1, int idp, FilterState<W> &fs)
{
    constexpr int KB = DP / 8;
    if constexpr (T < KB) {
        float4 n0 = a0, n1 = a1;
        if constexpr (T + 1 < KB) {
            n0 = *reinterpret_cast<const float4 *>(A0 + 4 * (T + 1));
            n1 = *reinterpret_cast<const float4 *>(A1 + 4 * (T + 1));
        }
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0.x, b[4 * T + 0], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1.x, b[4 * T + 0], c1, 0, 0, 0);
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0.y, b[4 * T + 1], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1.y, b[4 * T + 1], c1, 0, 0, 0);
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0.z, b[4 * T + 2], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1.z, b[4 * T + 2], c1, 0, 0, 0);
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0.w, b[4 * T + 3], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1.w, b[4 * T + 3], c1, 0, 0, 0);
        if constexpr (EP) filter_groups_at<0, T, KB, W>(p0, p1, idp, fs);
        __builtin_amdgcn_sched_barrier(0);
        filter_kblocks<DP, EP, W, T + 1>(A0, A1, b, c0, c1, n0, n1, p0, p1, idp, fs);
    }
}

// One chunk into (c0, c1) with the filter epilogue of the previous chunk
// (p0, p1, first id idp) spread over its K-blocks.
template <int DP, int W>
__device__ __forceinline__ void filter_chunk(const float *A0, const float *Nh, const float (&b)[DP / 2],
                                             f32x16 &c0, f32x16 &c1, const f32x16 &p0, const f32x16 &p1,
                                             int idp, FilterState<W> &fs)
{
    const float *A1 = A0 + 32 * (DP + 4);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const float4 u = *reinterpret_cast<const float4 *>(Nh + 8 * g);
        const float4 w = *reinterpret_cast<const float4 *>(Nh + 32 + 8 * g);
        c0[4 * g + 0] = u.x;
        c0[4 * g + 1] = u.y;
        c0[4 * g + 2] = u.z;
        c0[4 * g + 3] = u.w;
        c1[4 * g + 0] = w.x;
        c1[4 * g + 1] = w.y;
        c1[4 * g + 2] = w.z;
        c1[4 * g + 3] = w.w;
    }
    const float4 a0 = *reinterpret_cast<const float4 *>(A0);
    const float4 a1 = *reinterpret_cast<const float4 *>(A1);
    filter_kblocks<DP, true, W>(A0, A1, b, c0, c1, a0, a1, p0, p1, idp, fs);
}

template <int G = 0, int W>
__device__ __forceinline__ void filter_drain(const f32x16 &p0, const f32x16 &p1, int idp, FilterState<W> &fs)
{
    if constexpr (G < 8) {
        filter_group<G, W>(p0, p1, idp, fs);
        filter_drain<G + 1, W>(p0, p1, idp, fs);
    }
}

// First centroid of visited chunk k (the maps of ScreenArgs).
__device__ __forceinline__ int64_t keys_chunk_base(const ScreenArgs &a, int64_t k)
{
    return a.c_begin + k * (a.cstride > 1 ? a.cstride : 1) * kChunk;
}

// The filter's chunks in visiting order: every chunk but the sampled ones
// j * skip_s (j < skip_n). One division to start, then steps; chunk indices
// fit int32 (centroid ids do).
struct ChunkWalk {
    int phys;    // physical chunk of the current visit
    int next_s;  // next sampled chunk after it (INT_MAX: none)
    int left_s;  // sampled chunks from next_s on
    int stride;

    // every member assigned once, without early returns (the compiler keeps
    // the walk in registers)
    __device__ __forceinline__ void init(const ScreenArgs &a, int64_t k64)
    {
        const int k = (int)k64;
        const int ns = (int)a.skip_n;
        const bool on = ns > 0;
        const int st = on ? (int)a.skip_s : 2;
        const int run = st - 1;  // unsampled chunks after each sampled one
        const int p = !on ? k : k < ns * run ? (k / run) * st + 1 + k % run : k + ns;
        const int j = p / st + 1;  // the first sampled chunk after p (p is not sampled)
        const int left = on ? ns - j : 0;
        phys = p;
        left_s = left;
        next_s = left > 0 ? j * st : INT_MAX;
        stride = st;
    }

    __device__ __forceinline__ void next()
    {
        ++phys;
        if (phys == next_s) {
            ++phys;  // skip_s >= 2: the chunk after a sampled one is not sampled
            --left_s;
            next_s = left_s > 0 ? next_s + stride : INT_MAX;
        }
    }
};

// Filter over the chunks [ch_lo, ch_hi) of one tile: chunk j's MFMAs carry
// chunk j-1's epilogue; the last chunk's accumulators are drained after.
template <int DP, int W>
__device__ __forceinline__ void screen_filter_range(const ScreenArgs &a, int64_t tile, int64_t ch_lo, int64_t ch_hi,
                                    float *__restrict__ lds_c, float *__restrict__ lds_n, FilterQueue<W> &fq)
{
    constexpr int NT = W * 64;
    constexpr int KH = DP / 2;
    constexpr int CS = kChunk * (DP + 4);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int h = lane >> 5;
    const int jl = lane & 31;
    const int64_t row = tile * (32 * W) + wave * 32 + jl;
    const bool rvalid = row < a.nrows;

    float b[KH];
    load_row<DP>(reinterpret_cast<const float *>(a.rows), row, rvalid, a.D, h, b);

    FilterState<W> fs;
    fs.cand_cnt = a.cand_cnt;
    fs.cand = a.cand;
    fs.L = a.L;
    fs.q = &fq;
    fs.row = row;
    fs.tv = kInf;  // rows past the end keep nothing
    if (rvalid) fs.tv = fmaxf(-0.5f * a.tau[row], -__FLT_MAX__);
    fs.qn = 0;
    fs.wave = wave;
    fs.lane = lane;

    const float *Ab = lds_c + jl * (DP + 4) + h * KH;
    const float *Nb = lds_n + 4 * h;
    // centroid ids fit int32; the id of register r of block rb of a chunk at
    // cbase is cbase + 4h + rb*32 + 8*(r/4) + r%4
    const int nch = (int)(ch_hi - ch_lo);
    // first centroids of the last three fetched chunks: visits k - 1, k, k + 1
    // once chunk k + 1 is fetched
    ChunkWalk cw;
    cw.init(a, ch_lo);
    const int cb = (int)a.c_begin;
    int b_prev2 = 0, b_prev1 = 0, b_cur = cb + cw.phys * kChunk;
    auto advance = [&]() __attribute__((always_inline)) {
        cw.next();
        b_prev2 = b_prev1;
        b_prev1 = b_cur;
        b_cur = cb + cw.phys * kChunk;
    };
    auto idp_of = [&](int base) { return base + 4 * h; };

    Stager<DP, NT> cr;
    cr.init(a.D);
    cr.fetch(a.cent, a.cnorm, b_cur, a.c_end, a.D);
    cr.template store<true>(lds_c, lds_n);
    __syncthreads();

    Top3 unused{};
    f32x16 x0, x1, y0, y1;
    advance();
    cr.fetch(a.cent, a.cnorm, b_cur, a.c_end, a.D);
    mfma_chunk<DP, false>(Ab, Nb, b, x0, x1, x0, x1, 0, unused);
    cr.template store<true>(lds_c + CS, lds_n + kChunk);
    __syncthreads();

    // chunk j (relative to ch_lo) sits in buffer j & 1
    auto step = [&](int j, f32x16 &c0, f32x16 &c1, const f32x16 &p0, const f32x16 &p1) __attribute__((always_inline)) {
        advance();  // b_cur: visit j + 1, b_prev2: visit j - 1
        cr.fetch(a.cent, a.cnorm, b_cur, a.c_end, a.D);
        const int bj = j & 1;
        filter_chunk<DP, W>(Ab + bj * CS, Nb + bj * kChunk, b, c0, c1, p0, p1, idp_of(b_prev2), fs);
        cr.template store<true>(lds_c + (bj ^ 1) * CS, lds_n + (bj ^ 1) * kChunk);
        __syncthreads();
    };
    int j = 1;
    for (; j + 1 < nch; j += 2) {
        step(j, y0, y1, x0, x1);
        step(j + 1, x0, x1, y0, y1);
    }
    if (j < nch) {
        step(j, y0, y1, x0, x1);
        filter_drain(y0, y1, idp_of(b_prev1), fs);  // visit j
    } else {
        filter_drain(x0, x1, idp_of(b_prev1), fs);  // visit j - 1
    }
    filter_flush(fs);
}

// Keys over the chunks [ch_lo, ch_hi) of one tile (the routing threshold
// sample). As on the top-1 path the accumulators start from -||c||^2/2, so
// v = -key/2 exactly and the key written is -2v. Padded centroids have v =
// -inf, i.e. an infinite key.
template <int DP, int W, typename XT>
__device__ void screen_keys_range(const ScreenArgs &a, int64_t tile, int64_t ch_lo, int64_t ch_hi,
                                  float *__restrict__ lds_c, float *__restrict__ lds_n)
{
    constexpr int NT = W * 64;
    constexpr int KH = DP / 2;
    constexpr int CS = kChunk * (DP + 4);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int h = lane >> 5;
    const int jl = lane & 31;
    const int64_t row = tile * (32 * W) + wave * 32 + jl;
    const bool rvalid = row < a.nrows;

    float b[KH];
    load_row<DP>(reinterpret_cast<const XT *>(a.rows), row, rvalid, a.D, h, b);
    Top3 unused{};

    Stager<DP, NT> cr;
    cr.init(a.D);
    cr.fetch(a.cent, a.cnorm, keys_chunk_base(a, ch_lo), a.c_end, a.D);
    cr.template store<true>(lds_c, lds_n);
    __syncthreads();

    const float *Ab = lds_c + jl * (DP + 4) + h * KH;
    const float *Nb = lds_n + 4 * h;
    for (int64_t ch = ch_lo; ch < ch_hi; ++ch) {
        const int buf = (int)((ch - ch_lo) & 1);
        cr.fetch(a.cent, a.cnorm, keys_chunk_base(a, ch + 1), a.c_end, a.D);  // unconditional; see screen_top1

        f32x16 acc0, acc1;
        mfma_chunk<DP, false>(Ab + buf * CS, Nb + buf * kChunk, b, acc0, acc1, acc0, acc1, 0, unused);

        // the minimum key of each 16 consecutive sample positions: group m
        // of the chunk is registers 8(m%2) .. 8(m%2)+7 of block m/2 in both
        // half-lanes, and min(-2v) = -2 max(v) exactly
        float gm[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const f32x16 &p = m < 2 ? acc0 : acc1;
            const int r0 = 8 * (m & 1);
            float v = fmaxf(fmaxf(fmaxf(p[r0], p[r0 + 1]), fmaxf(p[r0 + 2], p[r0 + 3])),
                            fmaxf(fmaxf(p[r0 + 4], p[r0 + 5]), fmaxf(p[r0 + 6], p[r0 + 7])));
            v = fmaxf(v, __shfl_xor(v, 32));
            gm[m] = -2.0f * v;
        }
        // register r of block rb holds centroid rb*32 + 8*(r/4) + 4*h + r%4
        if (rvalid) {
            const int64_t ld = a.nchunks * kChunk;  // keys in visiting order
            if (h == 0 && a.kmin)
                *reinterpret_cast<float4 *>(a.kmin + row * (ld / 16) + ch * (kChunk / 16)) =
                    make_float4(gm[0], gm[1], gm[2], gm[3]);
            float *out = a.keys + row * ld + ch * kChunk + 4 * h;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                *reinterpret_cast<float4 *>(out + 8 * g) =
                    make_float4(-2.0f * acc0[4 * g + 0], -2.0f * acc0[4 * g + 1],
                                -2.0f * acc0[4 * g + 2], -2.0f * acc0[4 * g + 3]);
                *reinterpret_cast<float4 *>(out + 32 + 8 * g) =
                    make_float4(-2.0f * acc1[4 * g + 0], -2.0f * acc1[4 * g + 1],
                                -2.0f * acc1[4 * g + 2], -2.0f * acc1[4 * g + 3]);
            }
        }

        cr.template store<true>(lds_c + (buf ^ 1) * CS, lds_n + (buf ^ 1) * kChunk);
        __syncthreads();
    }
}

// Waves per SIMD: two, so that one wave's staging and epilogue overlap the
// other's MFMAs; one for DP >= 192, whose row fragments need the whole
// register file (those sizes always run W = 4, one workgroup per CU).
template <int DP>
constexpr int waves_per_simd()
{
    return DP >= 192 ? 1 : 2;
}

template <int DP, int W, typename XT, int MODE>
__global__ __launch_bounds__(W * 64, waves_per_simd<DP>()) void screen_kernel(ScreenArgs a)
{
    __shared__ __attribute__((aligned(16))) float lds_c[2 * kChunk * (DP + 4)];
    __shared__ __attribute__((aligned(16))) float lds_n[2 * kChunk];
    const int64_t ntiles = (a.nrows + 32 * W - 1) / (32 * W);
    if (a.gate && *a.gate == 0u) return;  // screened on int8 MFMA instead
    if constexpr (MODE == kModeTop1) {
        for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
            screen_top1<DP, W, XT>(a, tile, lds_c, lds_n);
            __syncthreads();
        }
    } else {
        // a contiguous range of (tile, chunk) units in tile-major order
        const int64_t units = ntiles * a.nchunks;
        int64_t u = units * blockIdx.x / gridDim.x;
        const int64_t u1 = units * (blockIdx.x + 1) / gridDim.x;
        while (u < u1) {
            const int64_t tile = u / a.nchunks;
            const int64_t ch = u - tile * a.nchunks;
            const int64_t ch_end = min(a.nchunks, ch + (u1 - u));
            if constexpr (MODE == kModeFilter) {
                __shared__ FilterQueue<W> fq;
                screen_filter_range<DP, W>(a, tile, ch, ch_end, lds_c, lds_n, fq);
            } else {
                screen_keys_range<DP, W, XT>(a, tile, ch, ch_end, lds_c, lds_n);
            }
            u += ch_end - ch;
            __syncthreads();
        }
    }
}

template <int DP, int W, typename XT, int MODE>
hipError_t launch_one(const ScreenArgs &a, int num_cus, hipStream_t s)
{
    const int64_t ntiles = (a.nrows + 32 * W - 1) / (32 * W);
    const int64_t work = MODE == kModeTop1 ? ntiles : ntiles * a.nchunks;
    const int per_cu = 4 * waves_per_simd<DP>() / W;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(work, (int64_t)per_cu * num_cus));
    hipLaunchKernelGGL((screen_kernel<DP, W, XT, MODE>), dim3(grid), dim3(W * 64), 0, s, a);
    return hipGetLastError();
}

template <int DP, int W>
hipError_t launch_dp(int mode, int rowtype, const ScreenArgs &a, int num_cus, hipStream_t s)
{
    if (mode == kModeTop1)
        return rowtype == kRowU8 ? launch_one<DP, W, uint8_t, kModeTop1>(a, num_cus, s)
                                 : launch_one<DP, W, float, kModeTop1>(a, num_cus, s);
    if (rowtype != kRowF32) return hipErrorInvalidValue;
    if (mode == kModeKeys) return launch_one<DP, W, float, kModeKeys>(a, num_cus, s);
    return launch_one<DP, W, float, kModeFilter>(a, num_cus, s);
}

template <int W>
hipError_t launch_w(int mode, int rowtype, int DP, const ScreenArgs &a, int num_cus, hipStream_t s)
{
    switch (DP) {
    case 32: return launch_dp<32, W>(mode, rowtype, a, num_cus, s);
    case 64: return launch_dp<64, W>(mode, rowtype, a, num_cus, s);
    case 96: return launch_dp<96, W>(mode, rowtype, a, num_cus, s);
    case 128: return launch_dp<128, W>(mode, rowtype, a, num_cus, s);
    case 192: return launch_dp<192, 4>(mode, rowtype, a, num_cus, s);
    case 256: return launch_dp<256, 4>(mode, rowtype, a, num_cus, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_screen(int mode, int rowtype, int DP, const ScreenArgs &a, int waves, int num_cus,
                         hipStream_t s)
{
    return waves == 4 ? launch_w<4>(mode, rowtype, DP, a, num_cus, s)
                      : launch_w<8>(mode, rowtype, DP, a, num_cus, s);
}

}  // namespace ivf

// Candidate-restricted assignment on gfx950 (the fast construction mode of
// Sec. "Fast Index Construction": every vector is scored against a few
// candidate centroids instead of all of them). The candidates of row i are
// graph[prev[i]][0 .. S) (for instance each centroid's S nearest centroids,
// from ivf_route of the centroids against themselves, and the row's previous
// label); the label is the candidate of smallest exact distance by
// (distance, id), the distance evaluated in fp64 exactly as everywhere in
// this library (t = (double)x_d - (double)c_d; s = fma(t, t, s), d
// ascending).
//
// Without a processing order (or for S > 16) a row owns a group of SP = next
// power of two >= S lanes of one wave; lane s of the group evaluates
// candidate s with one sequential fma chain over the dims (float4 loads of
// the centroid row; the lanes of a group read the same row addresses, which
// the memory system merges), and a shuffle butterfly inside the group takes
// the (distance, id) minimum. With an order that groups rows by previous
// label, one row per lane and the label's candidates shared by the wave
// (assign_graph_tile_kernel below).
#include "ivf_internal.h"
#include "exact.h"

#include <limits.h>

#include <algorithm>

namespace ivf {
namespace {

constexpr int kAgThreads = 256;

__device__ __forceinline__ void load4(const uint8_t *p, float (&v)[4])
{
    const uint32_t w = *reinterpret_cast<const uint32_t *>(p);
    v[0] = (float)(w & 0xFFu);
    v[1] = (float)((w >> 8) & 0xFFu);
    v[2] = (float)((w >> 16) & 0xFFu);
    v[3] = (float)(w >> 24);
}

__device__ __forceinline__ void load4(const float *p, float (&v)[4])
{
    const float4 w = *reinterpret_cast<const float4 *>(p);
    v[0] = w.x;
    v[1] = w.y;
    v[2] = w.z;
    v[3] = w.w;
}

template <typename XT>
__global__ __launch_bounds__(kAgThreads) void assign_graph_kernel(
    const XT *__restrict__ X, int64_t N, const float *__restrict__ cent, int64_t C, int D,
    const int32_t *__restrict__ graph, int S, int sp_log2, const int32_t *__restrict__ prev,
    const uint32_t *__restrict__ order, int32_t *__restrict__ labels, float *__restrict__ dist)
{
    const int SP = 1 << sp_log2;
    const int s = threadIdx.x & (SP - 1);
    // processing position -> row (rows with the same previous label next to
    // each other share their candidates' loads); order entries >= N are skipped
    const int64_t pos = ((int64_t)blockIdx.x * kAgThreads + threadIdx.x) >> sp_log2;
    const int64_t i = (order && pos < N) ? (int64_t)order[pos] : pos;
    const bool live = pos < N && i < N;
    double d = __builtin_huge_val();
    int id = INT_MAX;  // loses every comparison against a real candidate
    if (live && s < S) {
        const int32_t p = prev[i];
        const int32_t j = (p >= 0 && p < C) ? graph[(int64_t)p * S + s] : -1;
        if (j >= 0 && j < C) {
            const XT *x = X + i * D;
            const float *c = cent + (int64_t)j * D;
            double acc = 0.0;
            for (int k0 = 0; k0 < D; k0 += 32) {
                // the loads of 32 dims first, then their fma chain in dim order
                float xv[8][4], cv[8][4];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    if (k0 + 4 * q < D) {
                        load4(x + k0 + 4 * q, xv[q]);
                        load4(c + k0 + 4 * q, cv[q]);
                    }
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    if (k0 + 4 * q < D) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const double t = (double)xv[q][e] - (double)cv[q][e];
                            acc = fma(t, t, acc);
                        }
                    }
                }
            }
            d = acc;
            id = j;
        }
    }
    // (distance, id) minimum over the SP lanes of the row's group
    for (int off = SP >> 1; off > 0; off >>= 1) {
        const double od = __shfl_xor(d, off);
        const int oid = __shfl_xor(id, off);
        if (od < d || (od == d && oid < id)) {
            d = od;
            id = oid;
        }
    }
    if (live && s == 0) {
        const bool none = id == INT_MAX;
        labels[i] = none ? -1 : id;
        if (dist) dist[i] = none ? __builtin_huge_valf() : (float)d;
    }
}

// Cell-and-walk assignment: candidates for rows that have no previous label
// (the graph-assisted assignment of the full base set, Sec. "Fast Index
// Building Details"). Row i first takes the member of its coarse cell
// cell[i] of smallest (distance, id) (members[offsets[c] .. offsets[c + 1]),
// both offsets clamped into [0, M]), then up to `hops` times moves to the
// graph neighbour of smallest (distance, id) while that neighbour comes
// before the current choice. Ids outside [0, C) are skipped; a row without a
// valid member gets -1 and an infinite distance.
//
// A wave holds a tile of eight rows, each in its LDS slot as fp64 (exact for
// uint8 and fp32 rows, so the chain needs no conversion of the row). When
// every live row of the tile lies in the same cell (nearly always when the
// rows come in cell order), the 64 lanes share the cell's members: lane l
// takes members l, l + 64, ... and runs the exact sequential fp64 chain of
// each against all eight rows at once, so one load of a centroid element
// serves eight distances (the rows' LDS reads are broadcasts); a last pass
// of at most 32 members gives each half of the wave four of the rows, so it
// issues half the instructions of a full pass. A reduce-
// scatter over the lanes then leaves each group of eight lanes (lanes 8r ..
// 8r + 7) with row r's partial minima. Otherwise each row's eight lanes go
// over the row's own members s, s + 8, .... Either way a butterfly inside the
// group gives the row's (distance, id) minimum, and on a hop lane s of the
// group evaluates neighbours s, s + 8, ...; the rows of a wave walk until
// none of them moves. The slots are D + 2 doubles apart (four banks), so
// the eight groups' reads of the walk do not collide.
constexpr int kAcRows = 8;  // rows per wave

__host__ __device__ constexpr int ac_pitch(int D) { return D + 2; }

// waves per workgroup: four, or fewer where the slots would exceed 64 KiB
int ac_waves(int D)
{
    const int w = 65536 / (kAcRows * ac_pitch(D) * (int)sizeof(double));
    return w < 1 ? 1 : (w > 4 ? 4 : w);
}

__device__ __forceinline__ double dist_lds(const double *__restrict__ xs, const float *__restrict__ c, int D)
{
    double acc = 0.0;
    for (int k0 = 0; k0 < D; k0 += 32) {
        float4 cv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q)
            if (k0 + 4 * q < D) cv[q] = *reinterpret_cast<const float4 *>(c + k0 + 4 * q);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (k0 + 4 * q < D) {
                const double2 xa = *reinterpret_cast<const double2 *>(xs + k0 + 4 * q);
                const double2 xb = *reinterpret_cast<const double2 *>(xs + k0 + 4 * q + 2);
                const double xv[4] = {xa.x, xa.y, xb.x, xb.y};
                const float ca[4] = {cv[q].x, cv[q].y, cv[q].z, cv[q].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double t = xv[e] - (double)ca[e];
                    acc = fma(t, t, acc);
                }
            }
        }
    }
    return acc;
}

// The exact distances of centroid c to the NR rows of a tile from `rows` on
// (slots `pitch` doubles apart), each its own sequential chain in dim order.
template <int NR>
__device__ __forceinline__ void dist_tile(const double *__restrict__ rows, int pitch, const float *__restrict__ c,
                                          int D, double (&acc)[NR])
{
#pragma unroll
    for (int r = 0; r < NR; ++r) acc[r] = 0.0;
    for (int k0 = 0; k0 < D; k0 += 16) {
        float4 cv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (k0 + 4 * q < D) cv[q] = *reinterpret_cast<const float4 *>(c + k0 + 4 * q);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (k0 + 4 * q < D) {
                const double cd[4] = {(double)cv[q].x, (double)cv[q].y, (double)cv[q].z, (double)cv[q].w};
#pragma unroll
                for (int r = 0; r < NR; ++r) {
                    const double *xs = rows + r * pitch + k0 + 4 * q;
                    const double2 xa = *reinterpret_cast<const double2 *>(xs);
                    const double2 xb = *reinterpret_cast<const double2 *>(xs + 2);
                    const double xv[4] = {xa.x, xa.y, xb.x, xb.y};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const double t = xv[e] - cd[e];
                        acc[r] = fma(t, t, acc[r]);
                    }
                }
            }
        }
    }
}

__device__ __forceinline__ void take_min(double &d, int &id, double od, int oid)
{
    if (dist_lt(od, oid, d, id)) {
        d = od;
        id = oid;
    }
}

// Reduce-scatter of the eight rows' (distance, id) minima over the lane bits
// 5, 4, 3: lane l keeps row (l >> 3), minimised over the lanes l ^ 8k.
__device__ __forceinline__ void tile_scatter_min(const double (&bd)[kAcRows], const int (&bi)[kAcRows], int lane,
                                                 double &d, int &id)
{
    const bool h5 = lane & 32, h4 = lane & 16, h3 = lane & 8;
    double d4[4];
    int i4[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {  // rows 4 * bit5 + k stay
        const double sd = h5 ? bd[k] : bd[k + 4];
        const int si = h5 ? bi[k] : bi[k + 4];
        d4[k] = h5 ? bd[k + 4] : bd[k];
        i4[k] = h5 ? bi[k + 4] : bi[k];
        take_min(d4[k], i4[k], __shfl_xor(sd, 32), __shfl_xor(si, 32));
    }
    double d2[2];
    int i2[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {  // of those, 2 * bit4 + k stay
        const double sd = h4 ? d4[k] : d4[k + 2];
        const int si = h4 ? i4[k] : i4[k + 2];
        d2[k] = h4 ? d4[k + 2] : d4[k];
        i2[k] = h4 ? i4[k + 2] : i4[k];
        take_min(d2[k], i2[k], __shfl_xor(sd, 16), __shfl_xor(si, 16));
    }
    const double sd = h3 ? d2[0] : d2[1];
    const int si = h3 ? i2[0] : i2[1];
    d = h3 ? d2[1] : d2[0];
    id = h3 ? i2[1] : i2[0];
    take_min(d, id, __shfl_xor(sd, 8), __shfl_xor(si, 8));
}

// (distance, id) minimum over the eight lanes of a row
__device__ __forceinline__ void row_min(double &d, int &id)
{
    for (int off = 4; off > 0; off >>= 1) {
        const double od = __shfl_xor(d, off);
        const int oid = __shfl_xor(id, off);
        take_min(d, id, od, oid);
    }
}

template <typename XT>
__global__ __launch_bounds__(256) void assign_cells_kernel(
    const XT *__restrict__ X, int64_t N, const float *__restrict__ cent, int64_t C, int D,
    const int32_t *__restrict__ cell, int64_t G, const int64_t *__restrict__ offsets,
    const uint32_t *__restrict__ members, int64_t M, const int32_t *__restrict__ graph, int S, int hops,
    const uint32_t *__restrict__ order, int32_t *__restrict__ labels, float *__restrict__ dist)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char ac_lds[];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int slot = lane >> 3;  // the row of this lane within the tile
    const int sub = lane & 7;    // its lane within the row
    const int pitch = ac_pitch(D);
    double *tile = reinterpret_cast<double *>(ac_lds) + (size_t)wave * kAcRows * pitch;
    double *xs = tile + slot * pitch;
    // a contiguous range of processing positions per workgroup: with rows in
    // cell order, consecutive rows of a workgroup read the same members
    const int per_tile = (int)(blockDim.x >> 6) * kAcRows;
    const int64_t per = ((N + gridDim.x - 1) / gridDim.x + per_tile - 1) / per_tile * per_tile;
    const int64_t p0 = (int64_t)blockIdx.x * per, p1 = min(N, p0 + per);
    for (int64_t pb = p0 + wave * kAcRows; pb < p1; pb += per_tile) {
        const int64_t p = pb + slot;
        const int64_t i = p < p1 ? (order ? (int64_t)order[p] : p) : N;
        const bool live = i < N;  // order entries >= N are not rows
        // the rows into their slots (a dead slot holds zeros); the wave's own
        // LDS operations run in order, the fence keeps the compiler from
        // moving reads above writes
        __builtin_amdgcn_wave_barrier();
        for (int d = sub; d < D; d += kAcRows) xs[d] = live ? (double)X[i * D + d] : 0.0;
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();

        double bd = __builtin_huge_val();
        int bi = INT_MAX;  // loses every comparison against a real candidate
        const int32_t g = live ? cell[i] : -1;
        const uint64_t lm = __ballot(live);
        const int32_t g0 = __shfl(g, lm ? __ffsll((unsigned long long)lm) - 1 : 0);
        const bool shared = lm != 0 && g0 >= 0 && g0 < G && !__any(live && g != g0);
        if (shared) {
            int64_t m0 = offsets[g0], m1 = offsets[g0 + 1];
            m0 = min(max(m0, (int64_t)0), M);
            m1 = min(max(m1, m0), M);
            double td[kAcRows];
            int ti[kAcRows];
#pragma unroll
            for (int r = 0; r < kAcRows; ++r) {
                td[r] = __builtin_huge_val();
                ti[r] = INT_MAX;
            }
            for (int64_t eb = m0; eb < m1; eb += 64) {
                if (m1 - eb > 32) {
                    const int64_t e = eb + lane;
                    const uint32_t j = e < m1 ? members[e] : UINT32_MAX;
                    if ((int64_t)j < C) {
                        double acc[kAcRows];
                        dist_tile<kAcRows>(tile, pitch, cent + (int64_t)j * D, D, acc);
#pragma unroll
                        for (int r = 0; r < kAcRows; ++r) take_min(td[r], ti[r], acc[r], (int)j);
                    }
                } else {
                    // a last pass of at most 32 members: half h of the wave
                    // takes rows 4h .. 4h + 3, each lane half the chains
                    const bool h = lane & 32;
                    const int64_t e = eb + (lane & 31);
                    const uint32_t j = e < m1 ? members[e] : UINT32_MAX;
                    if ((int64_t)j < C) {
                        double acc[4];
                        dist_tile<4>(tile + (h ? 4 * pitch : 0), pitch, cent + (int64_t)j * D, D, acc);
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            if (h)
                                take_min(td[4 + r], ti[4 + r], acc[r], (int)j);
                            else
                                take_min(td[r], ti[r], acc[r], (int)j);
                        }
                    }
                }
            }
            tile_scatter_min(td, ti, lane, bd, bi);
            if (!live) {  // a dead slot's row is not one
                bd = __builtin_huge_val();
                bi = INT_MAX;
            }
        } else if (g >= 0 && g < G) {
            int64_t m0 = offsets[g], m1 = offsets[g + 1];
            m0 = min(max(m0, (int64_t)0), M);
            m1 = min(max(m1, m0), M);
            for (int64_t e = m0 + sub; e < m1; e += kAcRows) {
                const uint32_t j = members[e];
                if ((int64_t)j < C) take_min(bd, bi, dist_lds(xs, cent + (int64_t)j * D, D), (int)j);
            }
        }
        row_min(bd, bi);
        // greedy walk; a row that did not move stays where it is (its
        // neighbours, and so its decision, do not change)
        bool moving = bi != INT_MAX && graph != nullptr;
        for (int h = 0; h < hops && __any(moving); ++h) {
            double nd = __builtin_huge_val();
            int ni = INT_MAX;
            if (moving) {
                for (int n = sub; n < S; n += kAcRows) {
                    const int32_t j = graph[(int64_t)bi * S + n];
                    if (j >= 0 && j < C) take_min(nd, ni, dist_lds(xs, cent + (int64_t)j * D, D), j);
                }
            }
            row_min(nd, ni);
            const bool better = moving && ni != INT_MAX && dist_lt(nd, ni, bd, bi);
            if (better) {
                bd = nd;
                bi = ni;
            }
            moving = better;
        }
        if (live && sub == 0) {
            const bool none = bi == INT_MAX;
            labels[i] = none ? -1 : bi;
            if (dist) dist[i] = none ? __builtin_huge_valf() : (float)bd;
        }
    }
}

// The exact distance of a row (global) to a centroid, loads of 32 dims
// ahead of each block of the chain.
template <typename XT>
__device__ __forceinline__ double dist_row(const XT *__restrict__ x, const float *__restrict__ c, int D)
{
    double acc = 0.0;
    for (int k0 = 0; k0 < D; k0 += 32) {
        float xv[8][4], cv[8][4];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (k0 + 4 * q < D) {
                load4(x + k0 + 4 * q, xv[q]);
                load4(c + k0 + 4 * q, cv[q]);
            }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (k0 + 4 * q < D) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double t = (double)xv[q][e] - (double)cv[q][e];
                    acc = fma(t, t, acc);
                }
            }
        }
    }
    return acc;
}

// Candidate-restricted assignment with one row per lane, for S <= SM (8 or
// 16). Rows grouped by previous label (the previous step's list permutation
// as `order`) share their candidates: for each label that covers at least
// kAgMinLanes lanes of the wave (at most kAgPasses labels per wave), the
// candidates' ids and values are the same for every lane (scalar loads) and
// each lane runs its row's exact chain against each of them. The rows of the
// other labels (label boundaries, orders that do not group) take their own
// candidates' rows one lane per row. Used when a processing order is given:
// in row order nearly every row would take that path, which exposes the
// latency of its eight sequential candidates (18 ms for 10M rows against
// 10 ms for the lane-group kernel).
constexpr int kAgPasses = 4;
constexpr int kAgMinLanes = 8;

template <typename XT, int SM>
__global__ __launch_bounds__(256) void assign_graph_tile_kernel(
    const XT *__restrict__ X, int64_t N, const float *__restrict__ cent, int64_t C, int D,
    const int32_t *__restrict__ graph, int S, const int32_t *__restrict__ prev,
    const uint32_t *__restrict__ order, int32_t *__restrict__ labels, float *__restrict__ dist)
{
    const int lane = threadIdx.x & 63;
    const int64_t pos = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * 64 + lane;
    const int64_t i = (order && pos < N) ? (int64_t)order[pos] : pos;
    const bool live = pos < N && i < N;  // order entries >= N are not rows
    const int32_t p = live ? prev[i] : -1;
    const bool has = p >= 0 && p < C;
    const XT *x = X + (live ? i : 0) * (int64_t)D;
    double bd = __builtin_huge_val();
    int bi = INT_MAX;  // loses every comparison against a real candidate
    uint64_t todo = __ballot(has), rest = 0;
    for (int pass = 0; pass < kAgPasses && todo != 0; ++pass) {
        const int32_t L = __builtin_amdgcn_readfirstlane(__shfl(p, __ffsll((unsigned long long)todo) - 1));
        const uint64_t group = __ballot(has && p == L);
        todo &= ~group;
        if (__popcll(group) < kAgMinLanes) {
            rest |= group;
            continue;
        }
        int32_t js[SM];
#pragma unroll
        for (int s = 0; s < SM; ++s) {
            const int32_t j = s < S ? graph[(int64_t)L * S + s] : -1;
            js[s] = __builtin_amdgcn_readfirstlane((j >= 0 && j < C) ? j : -1);
        }
        double acc[SM];
#pragma unroll
        for (int s = 0; s < SM; ++s) acc[s] = 0.0;
        for (int k0 = 0; k0 < D; k0 += 32) {
            double xd[32];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                if (k0 + 4 * q < D) {
                    float v[4];
                    load4(x + k0 + 4 * q, v);
#pragma unroll
                    for (int e = 0; e < 4; ++e) xd[4 * q + e] = (double)v[e];
                }
            }
#pragma unroll
            for (int s = 0; s < SM; ++s) {
                if (js[s] < 0) continue;  // the same for every lane
                const float *c = cent + (int64_t)js[s] * D + k0;
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    if (k0 + 4 * q < D) {
                        const float4 cv = *reinterpret_cast<const float4 *>(c + 4 * q);
                        const float ca[4] = {cv.x, cv.y, cv.z, cv.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const double t = xd[4 * q + e] - (double)ca[e];
                            acc[s] = fma(t, t, acc[s]);
                        }
                    }
                }
            }
        }
        if ((group >> lane) & 1) {
#pragma unroll
            for (int s = 0; s < SM; ++s)
                if (js[s] >= 0) take_min(bd, bi, acc[s], js[s]);
        }
    }
    rest |= todo;
    if ((rest >> lane) & 1) {
        for (int s = 0; s < S; ++s) {
            const int32_t j = graph[(int64_t)p * S + s];
            if (j >= 0 && j < C) take_min(bd, bi, dist_row(x, cent + (int64_t)j * D, D), j);
        }
    }
    if (live) {
        const bool none = bi == INT_MAX;
        labels[i] = none ? -1 : bi;
        if (dist) dist[i] = none ? __builtin_huge_valf() : (float)bd;
    }
}

}  // namespace

hipError_t launch_assign_graph(const void *rows, int rowtype, int64_t N, const float *cent, int64_t C,
                               int D, const int32_t *graph, int S, const int32_t *prev, const uint32_t *order,
                               int32_t *labels, float *dist, hipStream_t s)
{
    if (N <= 0) return hipSuccess;
    // with a processing order (rows grouped by previous label) the waves
    // share candidates; in row order the lane-group kernel is faster
    if (S <= 16 && order) {
        const unsigned tiles = (unsigned)((N + 255) / 256);
#define IVF_AG_TILE(XT, SM)                                                                                  \
    hipLaunchKernelGGL((assign_graph_tile_kernel<XT, SM>), dim3(tiles), dim3(256), 0, s, (const XT *)rows, N, \
                       cent, C, D, graph, S, prev, order, labels, dist)
        if (rowtype == kRowU8) {
            if (S <= 8)
                IVF_AG_TILE(uint8_t, 8);
            else
                IVF_AG_TILE(uint8_t, 16);
        } else {
            if (S <= 8)
                IVF_AG_TILE(float, 8);
            else
                IVF_AG_TILE(float, 16);
        }
#undef IVF_AG_TILE
        return hipGetLastError();
    }
    int sp_log2 = 0;
    while ((1 << sp_log2) < S) ++sp_log2;
    const int64_t threads = N << sp_log2;
    const unsigned grid = (unsigned)((threads + kAgThreads - 1) / kAgThreads);
    if (rowtype == kRowU8)
        hipLaunchKernelGGL(assign_graph_kernel<uint8_t>, dim3(grid), dim3(kAgThreads), 0, s,
                           (const uint8_t *)rows, N, cent, C, D, graph, S, sp_log2, prev, order, labels, dist);
    else
        hipLaunchKernelGGL(assign_graph_kernel<float>, dim3(grid), dim3(kAgThreads), 0, s,
                           (const float *)rows, N, cent, C, D, graph, S, sp_log2, prev, order, labels, dist);
    return hipGetLastError();
}

}  // namespace ivf

namespace ivf {

hipError_t launch_assign_cells(const void *rows, int rowtype, int64_t N, const float *cent, int64_t C, int D,
                               const int32_t *cell, int64_t G, const int64_t *offsets, const uint32_t *members,
                               int64_t M, const int32_t *graph, int S, int hops, const uint32_t *order,
                               int32_t *labels, float *dist, int num_cus, hipStream_t s)
{
    if (N <= 0) return hipSuccess;
    if (D < 4 || D > kCellsMaxDim || D % 4) return hipErrorInvalidValue;
    const int waves = ac_waves(D);
    const size_t lds = (size_t)waves * kAcRows * ac_pitch(D) * sizeof(double);
    const int64_t blocks = (N + waves * kAcRows - 1) / (waves * kAcRows);
    const unsigned grid = (unsigned)std::min<int64_t>(blocks, (int64_t)num_cus * 32);
    if (rowtype == kRowU8)
        hipLaunchKernelGGL(assign_cells_kernel<uint8_t>, dim3(grid), dim3(waves * 64), lds, s,
                           (const uint8_t *)rows, N, cent, C, D, cell, G, offsets, members, M, graph, S, hops,
                           order, labels, dist);
    else
        hipLaunchKernelGGL(assign_cells_kernel<float>, dim3(grid), dim3(waves * 64), lds, s,
                           (const float *)rows, N, cent, C, D, cell, G, offsets, members, M, graph, S, hops,
                           order, labels, dist);
    return hipGetLastError();
}

}  // namespace ivf

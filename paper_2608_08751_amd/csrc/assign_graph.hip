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
// A row owns a group of SP = next power of two >= S lanes of one wave; lane s
// of the group evaluates candidate s with one sequential fma chain over the
// dims (float4 loads of the centroid row; the lanes of a group read the same
// row addresses, which the memory system merges), and a shuffle butterfly
// inside the group takes the (distance, id) minimum.
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
// Eight rows per wave, eight lanes per row: each row goes to its LDS slot as
// fp32 (exact for uint8), lane s of the row evaluates members s, s + 8, ...
// and, on a hop, neighbours s, s + 8, ..., each with the exact sequential
// fp64 chain (the row's ds_read_b128 is a broadcast within its eight lanes;
// the slots are padded apart by four banks), and a butterfly over the eight
// lanes takes the row's (distance, id) minimum. Every lane is busy in both
// phases (one row per wave left 49 of 128 member lanes and 56 of 64 walk
// lanes idle); the rows of a wave walk until none of them moves.
constexpr int kAcWaves = 4;
constexpr int kAcRows = 8;                      // rows per wave
constexpr int kAcPitch = kCellsMaxDim + 4;      // floats per row slot

__device__ __forceinline__ double dist_lds(const float *__restrict__ xs, const float *__restrict__ c, int D)
{
    double acc = 0.0;
    for (int k0 = 0; k0 < D; k0 += 32) {
        float4 xv[8], cv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (k0 + 4 * q < D) {
                xv[q] = *reinterpret_cast<const float4 *>(xs + k0 + 4 * q);
                cv[q] = *reinterpret_cast<const float4 *>(c + k0 + 4 * q);
            }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (k0 + 4 * q < D) {
                const float xa[4] = {xv[q].x, xv[q].y, xv[q].z, xv[q].w};
                const float ca[4] = {cv[q].x, cv[q].y, cv[q].z, cv[q].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double t = (double)xa[e] - (double)ca[e];
                    acc = fma(t, t, acc);
                }
            }
        }
    }
    return acc;
}

// (distance, id) minimum over the eight lanes of a row
__device__ __forceinline__ void row_min(double &d, int &id)
{
    for (int off = 4; off > 0; off >>= 1) {
        const double od = __shfl_xor(d, off);
        const int oid = __shfl_xor(id, off);
        if (dist_lt(od, oid, d, id)) {
            d = od;
            id = oid;
        }
    }
}

template <typename XT>
__global__ __launch_bounds__(kAcWaves * 64) void assign_cells_kernel(
    const XT *__restrict__ X, int64_t N, const float *__restrict__ cent, int64_t C, int D,
    const int32_t *__restrict__ cell, int64_t G, const int64_t *__restrict__ offsets,
    const uint32_t *__restrict__ members, int64_t M, const int32_t *__restrict__ graph, int S, int hops,
    const uint32_t *__restrict__ order, int32_t *__restrict__ labels, float *__restrict__ dist)
{
    __shared__ __attribute__((aligned(16))) float xs_all[kAcWaves][kAcRows][kAcPitch];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int slot = lane >> 3;  // the row of this lane within the wave
    const int sub = lane & 7;    // its lane within the row
    float *xs = xs_all[wave][slot];
    // a contiguous range of processing positions per workgroup: with rows in
    // cell order, consecutive rows of a workgroup read the same members
    constexpr int kPer = kAcWaves * kAcRows;
    const int64_t per = ((N + gridDim.x - 1) / gridDim.x + kPer - 1) / kPer * kPer;
    const int64_t p0 = (int64_t)blockIdx.x * per, p1 = min(N, p0 + per);
    for (int64_t pb = p0 + wave * kAcRows; pb < p1; pb += kPer) {
        const int64_t p = pb + slot;
        const int64_t i = p < p1 ? (order ? (int64_t)order[p] : p) : N;
        const bool live = i < N;  // order entries >= N are not rows
        // the rows into their slots; the wave's own LDS operations run in
        // order, the fence keeps the compiler from moving reads above writes
        __builtin_amdgcn_wave_barrier();
        if (live)
            for (int d = sub; d < D; d += kAcRows) xs[d] = (float)X[i * D + d];
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();

        double bd = __builtin_huge_val();
        int bi = INT_MAX;  // loses every comparison against a real candidate
        const int32_t g = live ? cell[i] : -1;
        if (g >= 0 && g < G) {
            int64_t m0 = offsets[g], m1 = offsets[g + 1];
            m0 = min(max(m0, (int64_t)0), M);
            m1 = min(max(m1, m0), M);
            for (int64_t e = m0 + sub; e < m1; e += kAcRows) {
                const uint32_t j = members[e];
                if ((int64_t)j < C) {
                    const double d = dist_lds(xs, cent + (int64_t)j * D, D);
                    if (dist_lt(d, (int)j, bd, bi)) {
                        bd = d;
                        bi = (int)j;
                    }
                }
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
                    if (j >= 0 && j < C) {
                        const double d = dist_lds(xs, cent + (int64_t)j * D, D);
                        if (dist_lt(d, j, nd, ni)) {
                            nd = d;
                            ni = j;
                        }
                    }
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

}  // namespace

hipError_t launch_assign_graph(const void *rows, int rowtype, int64_t N, const float *cent, int64_t C,
                               int D, const int32_t *graph, int S, const int32_t *prev, const uint32_t *order,
                               int32_t *labels, float *dist, hipStream_t s)
{
    if (N <= 0) return hipSuccess;
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
    const int64_t blocks = (N + kAcWaves * kAcRows - 1) / (kAcWaves * kAcRows);
    const unsigned grid = (unsigned)std::min<int64_t>(blocks, (int64_t)num_cus * 32);
    if (rowtype == kRowU8)
        hipLaunchKernelGGL(assign_cells_kernel<uint8_t>, dim3(grid), dim3(kAcWaves * 64), 0, s,
                           (const uint8_t *)rows, N, cent, C, D, cell, G, offsets, members, M, graph, S, hops,
                           order, labels, dist);
    else
        hipLaunchKernelGGL(assign_cells_kernel<float>, dim3(grid), dim3(kAcWaves * 64), 0, s,
                           (const float *)rows, N, cent, C, D, cell, G, offsets, members, M, graph, S, hops,
                           order, labels, dist);
    return hipGetLastError();
}

}  // namespace ivf

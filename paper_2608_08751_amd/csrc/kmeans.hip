// Lloyd mean update on gfx950 (k-means centroid training, Sec. "Fast Index
// Construction"), run after the assignment and the list build.
//
// Cluster j's rows are perm[offsets[j] .. offsets[j+1]), ascending by row id
// (the stable list build), so one wave per cluster sums them in exactly the
// order "ascending row id": uint64 integer sums for uint8 data (exact), fp64
// left-to-right sums for fp32 data. The new centroid is
// (float)(sum / (double)count); an empty cluster takes training row
//     r = SplitMix64 output (((iter << 32) | j) + 1) of a generator seeded with
//         `seed`, mod N
// (SplitMix64: Steele, Lea & Flood 2014). The wave also accumulates the
// squared distances of its rows to the input centroid j; a one-workgroup
// kernel adds the per-cluster parts in a fixed order into the objective.
// Rows are D elements at a stride of ld elements (ld = D for whole vectors;
// a subspace of product quantisation passes its first column and the full
// row length).
#include "ivf_internal.h"

namespace ivf {
namespace {

__device__ __forceinline__ uint64_t splitmix_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

__device__ __forceinline__ int64_t reseed_row(uint64_t seed, int32_t iter, int64_t j, int64_t N)
{
    const uint64_t key = ((uint64_t)(uint32_t)iter << 32) | (uint64_t)(uint32_t)j;
    const uint64_t z = splitmix_mix(seed + (key + 1) * 0x9E3779B97F4A7C15ULL);
    return (int64_t)(z % (uint64_t)N);
}

template <typename T> struct SumType;
template <> struct SumType<uint8_t> { typedef unsigned long long type; };
template <> struct SumType<float> { typedef double type; };


// Group g = blockIdx.y is an independent problem (a subspace of product
// quantisation): its rows start g * gs.x elements further, its centroids
// g * C * D floats, its counts, offsets and permutation g * C, g * (C + 1)
// and g * N entries further, and its reseed uses seed + g.
// K dims per lane (D <= 64 K), 32 / K member rows in flight.
template <typename XT, int K>
__global__ __launch_bounds__(256) void update_kernel(const XT *__restrict__ X, int64_t N, int D,
                                                     int64_t ld,
                                                     const float *__restrict__ cin, int64_t C,
                                                     const int64_t *__restrict__ counts,
                                                     const int64_t *__restrict__ offsets,
                                                     const uint32_t *__restrict__ perm,
                                                     uint64_t seed, int32_t iter,
                                                     float *__restrict__ cout,
                                                     double *__restrict__ jpart, int64_t x_group)
{
    typedef typename SumType<XT>::type S;
    const int lane = threadIdx.x & 63;
    const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= C) return;
    {
        const int64_t g = blockIdx.y;
        X += g * x_group;
        cin += g * C * D;
        cout += g * C * D;
        counts += g * C;
        offsets += g * (C + 1);
        perm += g * N;
        jpart += g * C;
        seed += (uint64_t)g;
    }
    const int64_t n = counts[j];
    const int64_t o = offsets[j];
    S sum[K];
    double cj[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        sum[k] = 0;
        const int d = lane + 64 * k;
        cj[k] = d < D ? (double)cin[j * D + d] : 0.0;
    }
    double jp = 0.0;
    for (int64_t t0 = 0; t0 < n; t0 += 64) {
        const int64_t cnt = min((int64_t)64, n - t0);
        const uint32_t myidx = lane < cnt ? perm[o + t0 + lane] : 0u;
        int u = 0;
        // B member rows in flight, then their values added in row order
        constexpr int B = 32 / K;
        for (; u + B <= cnt; u += B) {
            XT v[B][K];
#pragma unroll
            for (int q = 0; q < B; ++q) {
                const int64_t i = (int64_t)(uint32_t)__shfl((int)myidx, u + q);
                const XT *x = X + i * ld;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    const int d = lane + 64 * k;
                    v[q][k] = d < D ? x[d] : (XT)0;
                }
            }
#pragma unroll
            for (int q = 0; q < B; ++q) {
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    const int d = lane + 64 * k;
                    if (d < D) {
                        sum[k] += (S)v[q][k];
                        const double t = (double)v[q][k] - cj[k];
                        jp = fma(t, t, jp);
                    }
                }
            }
        }
        for (; u < cnt; ++u) {
            const int64_t i = (int64_t)(uint32_t)__shfl((int)myidx, u);
            const XT *x = X + i * ld;
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int d = lane + 64 * k;
                if (d < D) {
                    const XT v = x[d];
                    sum[k] += (S)v;
                    const double t = (double)v - cj[k];
                    jp = fma(t, t, jp);
                }
            }
        }
    }
    int64_t r = -1;
    if (n == 0) r = reseed_row(seed, iter, j, N);
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int d = lane + 64 * k;
        if (d < D) {
            float v;
            if (n > 0)
                v = (float)((double)sum[k] / (double)n);
            else
                v = (float)X[r * ld + d];
            cout[j * D + d] = v;
        }
    }
    for (int off = 32; off > 0; off >>= 1) jp += __shfl_xor(jp, off);
    if (lane == 0) jpart[j] = jp;
}

// D = DS dividing 64 (1 ... 32): every lane loads. Lane (q, d) = (lane / DS,
// lane % DS) reads dim d of member b * (64 / DS) + q of each chunk of 64
// members into register b, P chunks in flight (64 P member rows per round
// trip, against 32 / K above); the sums then take the members in list order,
// each value fetched from its lane by a shuffle, so every sum and the
// objective are those of update_kernel bit for bit (lanes q > 0 run copies
// of the chains and drop them).
template <typename XT, int DS>
__global__ __launch_bounds__(256) void update_small_kernel(const XT *__restrict__ X, int64_t N, int D, int64_t ld,
                                                           const float *__restrict__ cin, int64_t C,
                                                           const int64_t *__restrict__ counts,
                                                           const int64_t *__restrict__ offsets,
                                                           const uint32_t *__restrict__ perm, uint64_t seed,
                                                           int32_t iter, float *__restrict__ cout,
                                                           double *__restrict__ jpart, int64_t x_group)
{
    typedef typename SumType<XT>::type S;
    constexpr int R = 64 / DS;                       // members per wave load
    constexpr int P = DS <= 8 ? 4 : DS == 16 ? 2 : 1;  // chunks in flight
    const int lane = threadIdx.x & 63;
    const int q = lane / DS, d = lane % DS;
    const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= C) return;
    {
        const int64_t g = blockIdx.y;
        X += g * x_group;
        cin += g * C * D;
        cout += g * C * D;
        counts += g * C;
        offsets += g * (C + 1);
        perm += g * N;
        jpart += g * C;
        seed += (uint64_t)g;
    }
    const int64_t n = counts[j];
    const int64_t o = offsets[j];
    S sum = 0;
    const double cj = (double)cin[j * D + d];
    double jp = 0.0;
    for (int64_t t0 = 0; t0 < n; t0 += 64 * P) {
        XT v[P][DS];
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int64_t c0 = t0 + 64 * p;
            const int64_t cnt = n - c0;  // members left from this chunk on (may be <= 0)
            const uint32_t myidx = lane < cnt ? perm[o + c0 + lane] : 0u;
#pragma unroll
            for (int b = 0; b < DS; ++b) {
                const int mm = b * R + q;
                const int64_t i = (int64_t)(uint32_t)__shfl((int)myidx, mm);
                v[p][b] = mm < cnt ? X[i * ld + d] : (XT)0;
            }
        }
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int64_t cnt = n - (t0 + 64 * p);
#pragma unroll
            for (int m = 0; m < 64; ++m) {
                // member m of the chunk: register m / R of lane (m % R) * DS + d
                const XT w = __shfl(v[p][m / R], (m % R) * DS + d);
                if (m < cnt) {
                    sum += (S)w;
                    const double t = (double)w - cj;
                    jp = fma(t, t, jp);
                }
            }
        }
    }
    if (q == 0) {
        float r;
        if (n > 0)
            r = (float)((double)sum / (double)n);
        else
            r = (float)X[reseed_row(seed, iter, j, N) * ld + d];
        cout[j * D + d] = r;
    } else {
        jp = 0.0;
    }
    for (int off = 32; off > 0; off >>= 1) jp += __shfl_xor(jp, off);
    if (lane == 0) jpart[j] = jp;
}

// uint8 rows with D = 16 U (U = 1, 2, 4, 8 or 16 lanes per row) and 16-byte
// aligned rows: lane l reads the 16 bytes of dimensions 16 (l % U) .. + 15 of
// member l / U of each group of 64 / U members (one 16-byte load per lane,
// 64 / U rows per wave instruction), P groups in flight. The per-dimension
// sums are exact integers, so their order does not matter and the means are
// those of the byte-wise kernel bit for bit; the objective is the same fp64
// sum in another order.
template <int U>
__global__ __launch_bounds__(256) void update_u8v_kernel(const uint8_t *__restrict__ X, int64_t N, int D,
                                                         int64_t ld, const float *__restrict__ cin, int64_t C,
                                                         const int64_t *__restrict__ counts,
                                                         const int64_t *__restrict__ offsets,
                                                         const uint32_t *__restrict__ perm, uint64_t seed,
                                                         int32_t iter, float *__restrict__ cout,
                                                         double *__restrict__ jpart, int64_t x_group)
{
    constexpr int R = 64 / U;  // members per wave load
    constexpr int P = 4;       // loads in flight per lane
    const int lane = threadIdx.x & 63;
    const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= C) return;
    {
        const int64_t g = blockIdx.y;
        X += g * x_group;
        cin += g * C * D;
        cout += g * C * D;
        counts += g * C;
        offsets += g * (C + 1);
        perm += g * N;
        jpart += g * C;
        seed += (uint64_t)g;
    }
    const int64_t n = counts[j];
    const int64_t o = offsets[j];
    const int u = lane % U, r = lane / U;
    double cj[16];
    unsigned long long sum[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        cj[e] = (double)cin[j * D + 16 * u + e];
        sum[e] = 0;
    }
    double jp = 0.0;
    for (int64_t t0 = 0; t0 < n; t0 += 64) {
        const int cnt = (int)min((int64_t)64, n - t0);
        const uint32_t myidx = lane < cnt ? perm[o + t0 + lane] : 0u;
        for (int q0 = 0; q0 < cnt; q0 += P * R) {
            uint4 v[P];
#pragma unroll
            for (int p = 0; p < P; ++p) {
                const int m = q0 + p * R + r;  // member within the chunk of 64
                const int64_t i = (int64_t)(uint32_t)__shfl((int)myidx, m & 63);
                v[p] = m < cnt ? *reinterpret_cast<const uint4 *>(X + i * ld + 16 * u) : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int p = 0; p < P; ++p) {
                if (q0 + p * R + r < cnt) {
                    const uint32_t w[4] = {v[p].x, v[p].y, v[p].z, v[p].w};
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const uint32_t b = (w[e >> 2] >> (8 * (e & 3))) & 0xFFu;
                        sum[e] += b;
                        const double t = (double)b - cj[e];
                        jp = fma(t, t, jp);
                    }
                }
            }
        }
    }
    // lanes with the same dimensions (same l % U) add their partial sums
#pragma unroll
    for (int off = U; off < 64; off <<= 1)
#pragma unroll
        for (int e = 0; e < 16; ++e) sum[e] += __shfl_xor(sum[e], off);
    int64_t rr = -1;
    if (n == 0) rr = reseed_row(seed, iter, j, N);
    if (r == 0) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int d = 16 * u + e;
            cout[j * D + d] = n > 0 ? (float)((double)sum[e] / (double)n) : (float)X[rr * ld + d];
        }
    }
    for (int off = 32; off > 0; off >>= 1) jp += __shfl_xor(jp, off);
    if (lane == 0) jpart[j] = jp;
}

// Block g adds the C parts of group g in a fixed order into out[g].
__global__ __launch_bounds__(1024) void sum_parts_kernel(const double *__restrict__ part,
                                                         int64_t C, double *__restrict__ out)
{
    __shared__ double s[1024];
    part += (int64_t)blockIdx.x * C;
    out += blockIdx.x;
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < C; j += blockDim.x) acc += part[j];
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
        if (threadIdx.x < (unsigned)w) s[threadIdx.x] += s[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = s[0];
}

}  // namespace

hipError_t launch_kmeans_update(const void *rows, int rowtype, int64_t N, int D, int64_t ld,
                                const float *cent_in, int64_t C, const int64_t *counts,
                                const int64_t *offsets, const uint32_t *perm, uint64_t seed,
                                int32_t iter, float *cent_out, double *jpart, double *objective,
                                hipStream_t s, int groups, int64_t x_group)
{
    const dim3 grid((unsigned)((C + 3) / 4), (unsigned)groups);
    const int U = D / 16;
    const bool vec = rowtype == kRowU8 && D % 16 == 0 && (U == 1 || U == 2 || U == 4 || U == 8 || U == 16) &&
                     ld % 16 == 0 && x_group % 16 == 0 && (uintptr_t)rows % 16 == 0;
    if (vec) {
        auto k = U == 1 ? update_u8v_kernel<1> : U == 2 ? update_u8v_kernel<2> : U == 4 ? update_u8v_kernel<4>
                 : U == 8 ? update_u8v_kernel<8> : update_u8v_kernel<16>;
        hipLaunchKernelGGL(k, grid, dim3(256), 0, s, (const uint8_t *)rows, N, D, ld, cent_in, C, counts, offsets,
                           perm, seed, iter, cent_out, jpart, x_group);
    } else {
        // dims per lane: 1, 2 or 4 (D <= 64, 128, 256), member rows in flight 32, 16, 8
        const int K = D <= 64 ? 1 : D <= 128 ? 2 : 4;
        const bool small = D == 1 || D == 2 || D == 4 || D == 8 || D == 16 || D == 32;
#define IVF_UPDATE_SMALL(XT, DS_)                                                                              \
    hipLaunchKernelGGL((update_small_kernel<XT, DS_>), grid, dim3(256), 0, s, (const XT *)rows, N, D, ld, cent_in, \
                       C, counts, offsets, perm, seed, iter, cent_out, jpart, x_group)
#define IVF_UPDATE_SMALL_ALL(XT)         \
    do {                                 \
        if (D == 1)                      \
            IVF_UPDATE_SMALL(XT, 1);     \
        else if (D == 2)                 \
            IVF_UPDATE_SMALL(XT, 2);     \
        else if (D == 4)                 \
            IVF_UPDATE_SMALL(XT, 4);     \
        else if (D == 8)                 \
            IVF_UPDATE_SMALL(XT, 8);     \
        else if (D == 16)                \
            IVF_UPDATE_SMALL(XT, 16);    \
        else                             \
            IVF_UPDATE_SMALL(XT, 32);    \
    } while (0)
#define IVF_UPDATE_LAUNCH(XT, K_)                                                                              \
    hipLaunchKernelGGL((update_kernel<XT, K_>), grid, dim3(256), 0, s, (const XT *)rows, N, D, ld, cent_in, C, \
                       counts, offsets, perm, seed, iter, cent_out, jpart, x_group)
        if (small) {
            if (rowtype == kRowU8)
                IVF_UPDATE_SMALL_ALL(uint8_t);
            else
                IVF_UPDATE_SMALL_ALL(float);
        } else if (rowtype == kRowU8) {
            if (K == 1)
                IVF_UPDATE_LAUNCH(uint8_t, 1);
            else if (K == 2)
                IVF_UPDATE_LAUNCH(uint8_t, 2);
            else
                IVF_UPDATE_LAUNCH(uint8_t, 4);
        } else {
            if (K == 1)
                IVF_UPDATE_LAUNCH(float, 1);
            else if (K == 2)
                IVF_UPDATE_LAUNCH(float, 2);
            else
                IVF_UPDATE_LAUNCH(float, 4);
        }
#undef IVF_UPDATE_LAUNCH
#undef IVF_UPDATE_SMALL_ALL
#undef IVF_UPDATE_SMALL
    }
    if (objective)
        hipLaunchKernelGGL(sum_parts_kernel, dim3((unsigned)groups), dim3(1024), 0, s, jpart, C, objective);
    return hipGetLastError();
}

}  // namespace ivf

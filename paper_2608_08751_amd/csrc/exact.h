// The exact distance of the results (the definition the screening kernels are
// certified against): squared L2 in fp64, dimensions in ascending order, one
// subtraction and one fma per dimension, and the (distance, id) order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ivf {

__device__ __forceinline__ bool dist_lt(double da, int ia, double db, int ib)
{
    return da < db || (da == db && ia < ib);
}

// The operands are loaded 32 dimensions at a time before their fma chain,
// so that a row costs D / 32 memory latencies instead of D; the arithmetic
// is the same sequence in the same order.
template <typename XT>
__device__ __forceinline__ double exact_dist(const XT *__restrict__ x, const float *__restrict__ c,
                                             int D)
{
    constexpr int kB = 32;
    double s = 0.0;
    int d = 0;
#pragma unroll 1
    for (; d + kB <= D; d += kB) {
        float cv[kB];
        XT xv[kB];
#pragma unroll
        for (int k = 0; k < kB; ++k) {
            cv[k] = c[d + k];
            xv[k] = x[d + k];
        }
#pragma unroll
        for (int k = 0; k < kB; ++k) {
            const double t = (double)xv[k] - (double)cv[k];
            s = fma(t, t, s);
        }
    }
#pragma unroll 1
    for (; d < D; ++d) {
        const double t = (double)x[d] - (double)c[d];
        s = fma(t, t, s);
    }
    return s;
}

// The same distance for a row staged in LDS (fp32) and a centroid row whose
// address is 16-byte aligned (D % 4 == 0): the centroid is read 64 dims at a
// time in 16-byte loads, all issued before their fma chain.
__device__ __forceinline__ double exact_dist_lds4(const float *__restrict__ x, const float *__restrict__ c, int D)
{
    double s = 0.0;
#pragma unroll 1
    for (int d0 = 0; d0 < D; d0 += 64) {
        float4 cv[16];
#pragma unroll
        for (int q = 0; q < 16; ++q)
            if (d0 + 4 * q < D) cv[q] = *reinterpret_cast<const float4 *>(c + d0 + 4 * q);
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            if (d0 + 4 * q < D) {
                const float4 xv = *reinterpret_cast<const float4 *>(x + d0 + 4 * q);
                const float xa[4] = {xv.x, xv.y, xv.z, xv.w};
                const float ca[4] = {cv[q].x, cv[q].y, cv[q].z, cv[q].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double t = (double)xa[e] - (double)ca[e];
                    s = fma(t, t, s);
                }
            }
        }
    }
    return s;
}

}  // namespace ivf

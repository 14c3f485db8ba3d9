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

}  // namespace ivf

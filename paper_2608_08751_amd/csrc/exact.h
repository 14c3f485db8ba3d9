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

template <typename XT>
__device__ __forceinline__ double exact_dist(const XT *__restrict__ x, const float *__restrict__ c,
                                             int D)
{
    double s = 0.0;
#pragma unroll 1
    for (int d = 0; d < D; ++d) {
        const double t = (double)x[d] - (double)c[d];
        s = fma(t, t, s);
    }
    return s;
}

}  // namespace ivf

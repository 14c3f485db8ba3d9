// Throughput probes for the MFMA pipes of gfx950 that the screening kernels
// use: every wave runs rounds of sixteen MFMAs (v_mfma_f32_32x32x2_f32, or
// v_mfma_i32_32x32x32_i8) on two independent accumulators with the A and B
// operands in registers, two waves per SIMD on every CU. This is the rate
// the screening kernels' MFMA stream could reach with no loads and no other
// vector instructions; bench reports the screening kernels against it next
// to the published peak. The int8 probe feeds pseudo-random operands (four
// register sets per operand, rotated): with data that toggles like real
// rows and centroids the part runs the int8 pipe at a lower, power-limited
// clock than with constant operands.
#include "ivf_internal.h"

namespace ivf {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256, 2) void mfma_probe_kernel(int iters, float a, float b, int write,
                                                            float *sink)
{
    f32x16 acc0 = {0.f}, acc1 = {0.f};
    const float av = a + threadIdx.x * 1e-7f;
    const float bv = b - threadIdx.x * 1e-7f;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc1, 0, 0, 0);
        }
    }
    float r = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) r += acc0[e] + acc1[e];
    // the host passes write = 0: the store only keeps the MFMAs alive
    if (write) sink[blockIdx.x * blockDim.x + threadIdx.x] = r;
}

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(512, 2) void mfma_probe_i8_kernel(int iters, int seed, int write, int *sink)
{
    i32x16 acc0 = {0}, acc1 = {0};
    i32x4 av[4], bv[4];
    uint32_t s = (uint32_t)seed * 2654435761u + threadIdx.x * 40503u + blockIdx.x;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            s = s * 1664525u + 1013904223u;  // LCG (Numerical Recipes constants)
            av[i][j] = (int)s;
            s = s * 1664525u + 1013904223u;
            bv[i][j] = (int)s;
        }
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(av[k], bv[(k + r) & 3], acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(av[(k + 1) & 3], bv[(k + r + 2) & 3], acc1, 0, 0, 0);
            }
        }
    }
    int t = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) t += acc0[e] + acc1[e];
    if (write) sink[blockIdx.x * blockDim.x + threadIdx.x] = t;
}

}  // namespace

hipError_t launch_mfma_probe_i8(int iters, int num_cus, hipStream_t s, double *ops)
{
    const int grid = num_cus;  // 8 waves per workgroup: two waves per SIMD
    hipLaunchKernelGGL(mfma_probe_i8_kernel, dim3(grid), dim3(512), 0, s, iters, 1, 0, (int *)nullptr);
    *ops = (double)grid * 8 * iters * 16 * (2.0 * 32 * 32 * 32);
    return hipGetLastError();
}

hipError_t launch_mfma_probe(int iters, int num_cus, hipStream_t s, double *flops)
{
    const int grid = 2 * num_cus;  // 4 waves per workgroup: two waves per SIMD
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(grid), dim3(256), 0, s, iters, 1.0f, 2.0f, 0,
                       (float *)nullptr);
    *flops = (double)grid * 4 * iters * 16 * (2.0 * 32 * 32 * 2);
    return hipGetLastError();
}

}  // namespace ivf

// Product quantisation on gfx950: the PQ encoding equation (Sec. "ANN Search
// and IVF") applied to residuals (Sec. "Residual-PQ Candidate Reduction").
// For every row and subspace m, the nearest of the K = 256 codewords of
// subspace m by (distance, index), with the distance evaluated in fp64 as
// everywhere in this library:
//     t = (double)x_d - (double)c_d; s = fma(t, t, s), d ascending.
// Subspaces have at most 16 dims, so the exact search is cheap enough for
// the vector ALUs (256 codewords x dsub fp64 FMAs per row and subspace); no
// screening or certificate is needed.
//
// A workgroup takes 256 rows (one per thread) and walks the subspaces of its
// range: it stages codebook m in LDS as doubles (every thread then reads the
// same codeword, a broadcast), each thread holds its sub-vector in
// registers, and the result goes to a uint8 code matrix [n, M] and/or to
// int32 labels [m1 - m0][n] (the codebook update of a subspace needs them).
#include "ivf_internal.h"

namespace ivf {
namespace {

constexpr int kPqThreads = 256;

template <int DS>  // upper bound on the dims per subspace
__global__ __launch_bounds__(kPqThreads) void pq_assign_kernel(
    const float *__restrict__ X, int64_t n, int D, int dsub, int m0, int m1,
    const float *__restrict__ codebooks, uint8_t *__restrict__ codes, int M,
    int32_t *__restrict__ labels)
{
    extern __shared__ double cb[];  // [kPqK][dsub] doubles of the current subspace
    const int64_t i = (int64_t)blockIdx.x * kPqThreads + threadIdx.x;
    const bool valid = i < n;
    for (int m = m0; m < m1; ++m) {
        __syncthreads();  // everyone is done with the previous codebook
        const float *src = codebooks + (int64_t)m * kPqK * dsub;
        for (int t = threadIdx.x; t < kPqK * dsub; t += kPqThreads) cb[t] = (double)src[t];
        __syncthreads();
        double x[DS];
#pragma unroll
        for (int d = 0; d < DS; ++d)
            x[d] = (valid && d < dsub) ? (double)X[i * D + (int64_t)m * dsub + d] : 0.0;
        double best = __builtin_huge_val();
        int bj = 0;
        for (int j = 0; j < kPqK; ++j) {
            const double *c = cb + j * dsub;
            double s = 0.0;
#pragma unroll
            for (int d = 0; d < DS; ++d) {
                if (d < dsub) {
                    const double t = x[d] - c[d];
                    s = fma(t, t, s);
                }
            }
            if (s < best) {  // strict: the lower index wins a tie
                best = s;
                bj = j;
            }
        }
        if (valid) {
            if (codes) codes[i * M + m] = (uint8_t)bj;
            if (labels) labels[(int64_t)(m - m0) * n + i] = bj;
        }
    }
}

}  // namespace

hipError_t launch_pq_assign(const float *X, int64_t n, int D, int dsub, int m0, int m1,
                            const float *codebooks, uint8_t *codes, int M, int32_t *labels,
                            hipStream_t s)
{
    if (n <= 0 || m1 <= m0) return hipSuccess;
    const unsigned grid = (unsigned)((n + kPqThreads - 1) / kPqThreads);
    const size_t lds = (size_t)kPqK * dsub * sizeof(double);
    if (dsub <= 4)
        hipLaunchKernelGGL(pq_assign_kernel<4>, dim3(grid), dim3(kPqThreads), lds, s, X, n, D, dsub, m0,
                           m1, codebooks, codes, M, labels);
    else if (dsub <= 8)
        hipLaunchKernelGGL(pq_assign_kernel<8>, dim3(grid), dim3(kPqThreads), lds, s, X, n, D, dsub, m0,
                           m1, codebooks, codes, M, labels);
    else
        hipLaunchKernelGGL(pq_assign_kernel<16>, dim3(grid), dim3(kPqThreads), lds, s, X, n, D, dsub, m0,
                           m1, codebooks, codes, M, labels);
    return hipGetLastError();
}

}  // namespace ivf

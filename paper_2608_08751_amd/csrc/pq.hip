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
// A workgroup takes 256 R rows (R per thread: 4 for subspaces of 4 or 8
// dims, 2 for 16, 1 for other widths) and walks the subspaces of its range: it stages codebook m in
// LDS as doubles (every thread then reads the same codeword, a broadcast, and
// one read serves its R rows' chains), each thread holds its sub-vectors in
// registers, and the result goes to a uint8 code matrix [n, M] and/or to
// int32 labels [m1 - m0][n] (the codebook update of a subspace needs them).
#include "ivf_internal.h"

namespace ivf {
namespace {

constexpr int kPqThreads = 256;

// DS: the dims per subspace (EXACT) or an upper bound on them; R: rows per
// thread. With EXACT the chains have no guards, so the compiler interleaves
// the R rows' chains.
template <int DS, int R, bool EXACT>
__global__ __launch_bounds__(kPqThreads) void pq_assign_kernel(
    const float *__restrict__ X, int64_t n, int D, int dsub_arg, int m0, int m1,
    const float *__restrict__ codebooks, uint8_t *__restrict__ codes, int M,
    int32_t *__restrict__ labels)
{
    const int dsub = EXACT ? DS : dsub_arg;
    extern __shared__ double cb[];  // [kPqK][dsub] doubles of the current subspace
    // rows i0 + r * kPqThreads, r < R: consecutive threads take consecutive rows
    const int64_t i0 = (int64_t)blockIdx.x * kPqThreads * R + threadIdx.x;
    for (int m = m0; m < m1; ++m) {
        __syncthreads();  // everyone is done with the previous codebook
        const float *src = codebooks + (int64_t)m * kPqK * dsub;
        for (int t = threadIdx.x; t < kPqK * dsub; t += kPqThreads) cb[t] = (double)src[t];
        __syncthreads();
        double x[R][DS];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t i = i0 + (int64_t)r * kPqThreads;
#pragma unroll
            for (int d = 0; d < DS; ++d)
                x[r][d] = (i < n && d < dsub) ? (double)X[i * D + (int64_t)m * dsub + d] : 0.0;
        }
        double best[R];
        int bj[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            best[r] = __builtin_huge_val();
            bj[r] = 0;
        }
        for (int j = 0; j < kPqK; ++j) {
            // one read of the codeword (a broadcast) serves the R rows' chains
            double c[DS];
#pragma unroll
            for (int d = 0; d < DS; ++d) c[d] = d < dsub ? cb[j * dsub + d] : 0.0;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                double s = 0.0;
#pragma unroll
                for (int d = 0; d < DS; ++d) {
                    if (d < dsub) {
                        const double t = x[r][d] - c[d];
                        s = fma(t, t, s);
                    }
                }
                if (s < best[r]) {  // strict: the lower index wins a tie
                    best[r] = s;
                    bj[r] = j;
                }
            }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t i = i0 + (int64_t)r * kPqThreads;
            if (i < n) {
                if (codes) codes[i * M + m] = (uint8_t)bj[r];
                if (labels) labels[(int64_t)(m - m0) * n + i] = bj[r];
            }
        }
    }
}

}  // namespace

hipError_t launch_pq_assign(const float *X, int64_t n, int D, int dsub, int m0, int m1,
                            const float *codebooks, uint8_t *codes, int M, int32_t *labels,
                            hipStream_t s)
{
    if (n <= 0 || m1 <= m0) return hipSuccess;
    const size_t lds = (size_t)kPqK * dsub * sizeof(double);
    // subspaces of 4, 8 or 16 dims: 4 rows per thread (2 at 16 dims, whose
    // sub-vectors take 32 registers a row); other widths one row per thread
    auto grid = [n](int r) { return (unsigned)((n + (int64_t)kPqThreads * r - 1) / ((int64_t)kPqThreads * r)); };
#define IVF_PQ_LAUNCH(DS, R, EXACT)                                                                              \
    hipLaunchKernelGGL((pq_assign_kernel<DS, R, EXACT>), dim3(grid(R)), dim3(kPqThreads), lds, s, X, n, D, dsub, \
                       m0, m1, codebooks, codes, M, labels)
    if (dsub == 4)
        IVF_PQ_LAUNCH(4, 4, true);
    else if (dsub == 8)
        IVF_PQ_LAUNCH(8, 4, true);
    else if (dsub == 16)
        IVF_PQ_LAUNCH(16, 2, true);
    else if (dsub < 4)
        IVF_PQ_LAUNCH(4, 1, false);
    else if (dsub < 8)
        IVF_PQ_LAUNCH(8, 1, false);
    else
        IVF_PQ_LAUNCH(16, 1, false);
#undef IVF_PQ_LAUNCH
    return hipGetLastError();
}

}  // namespace ivf

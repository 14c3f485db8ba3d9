// Device-side generator of the uint8 Gaussian-mixture rows used as k-means
// training data and as the 1e9-row base set. Input generation only: nothing
// here computes any part of the IVF method.
//
// Row i (global index) takes component a_i = SplitMix64 output (i + 1) of the
// component stream mod C; dims (2p, 2p+1) take one SplitMix64 output of the
// noise stream, split into two 24-bit uniforms for the Box-Muller transform
// (Box & Muller 1958). x = clip(rint(mean_a + 20 z), 0, 255).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ULL;

__device__ __forceinline__ uint64_t splitmix_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint8_t to_u8(float v)
{
    v = rintf(v);
    v = fminf(fmaxf(v, 0.0f), 255.0f);
    return (uint8_t)v;
}

// One thread writes 8 consecutive bytes (4 normal pairs) of one row.
__global__ void mixture_rows_kernel(const float *__restrict__ means, int64_t C, int D,
                                    uint64_t comp_seed, uint64_t noise_seed, int64_t row0,
                                    int64_t nrows, uint8_t *__restrict__ out)
{
    const int groups = D / 8;
    const int64_t total = nrows * groups;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int64_t r = t / groups;
        const int g = (int)(t - r * groups);
        const uint64_t row = (uint64_t)(row0 + r);
        const uint64_t a = splitmix_mix(comp_seed + (row + 1) * kGamma) % (uint64_t)C;
        const float *m = means + a * (uint64_t)D + g * 8;
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint64_t n = row * (uint64_t)(D / 2) + (uint64_t)(g * 4 + p) + 1;
            const uint64_t h = splitmix_mix(noise_seed + n * kGamma);
            const float u1 = (float)((h >> 40) + 1) * (1.0f / 16777216.0f);
            const float u2 = (float)(h & 0xFFFFFFULL) * (1.0f / 16777216.0f);
            const float rr = sqrtf(-2.0f * logf(u1));
            const float ang = 6.283185307179586f * u2;
            const float z0 = rr * cosf(ang);
            const float z1 = rr * sinf(ang);
            const uint32_t b0 = to_u8(m[2 * p] + 20.0f * z0);
            const uint32_t b1 = to_u8(m[2 * p + 1] + 20.0f * z1);
            const uint32_t pair = b0 | (b1 << 8);
            if (p < 2)
                lo |= pair << (16 * p);
            else
                hi |= pair << (16 * (p - 2));
        }
        *reinterpret_cast<uint2 *>(out + r * D + g * 8) = make_uint2(lo, hi);
    }
}

// Uniform labels in [0, C): label_i = SplitMix64 output (i + 1) mod C.
__global__ void labels_kernel(uint64_t seed, int64_t C, int64_t n, int32_t *__restrict__ out)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        out[i] = (int32_t)(splitmix_mix(seed + (uint64_t)(i + 1) * kGamma) % (uint64_t)C);
}

} // namespace

extern "C" int synth_labels_i32(uint64_t seed, int64_t C, int64_t n, int32_t *out, void *stream)
{
    if (C < 1 || n < 0 || (!out && n > 0)) return 1;
    if (n == 0) return 0;
    int64_t grid = (n + 255) / 256;
    if (grid > 65536) grid = 65536;
    hipLaunchKernelGGL(labels_kernel, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream, seed, C, n, out);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" int synth_mixture_u8(const float *means, int64_t C, int D, uint64_t comp_seed,
                                uint64_t noise_seed, int64_t row0, int64_t nrows, uint8_t *out,
                                void *stream)
{
    if (C < 1 || D < 8 || D % 8 != 0 || nrows < 0 || row0 < 0 || !means || (!out && nrows > 0))
        return 1;
    if (nrows == 0) return 0;
    const int block = 256;
    const int64_t total = nrows * (D / 8);
    int64_t grid = (total + block - 1) / block;
    if (grid > 65536) grid = 65536;
    hipLaunchKernelGGL(mixture_rows_kernel, dim3((unsigned)grid), dim3(block), 0,
                       (hipStream_t)stream, means, C, D, comp_seed, noise_seed, row0, nrows, out);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

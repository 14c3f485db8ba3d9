// Wave-aggregated global atomics: one atomic per wave and counter instead of
// one per lane (many lanes adding to the same address serialise in L2).
// Every lane of the wave must call these (they use ballots and shuffles).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ivf {

// Adds the number of lanes with `pred` to *ctr.
__device__ __forceinline__ void wave_count(unsigned long long *ctr, bool pred)
{
    const uint64_t m = __ballot(pred);
    if (m != 0 && (int)(threadIdx.x & 63) == __ffsll((unsigned long long)m) - 1)
        atomicAdd(ctr, (unsigned long long)__popcll(m));
}

// Reserves one slot of *ctr per lane with `pred` and returns the lane's slot
// (the wave's slots are consecutive, in lane order); other lanes get an
// unspecified value.
__device__ __forceinline__ uint32_t wave_append(uint32_t *ctr, bool pred)
{
    const uint64_t m = __ballot(pred);
    if (m == 0) return 0;
    const int leader = __ffsll((unsigned long long)m) - 1;
    uint32_t base = 0;
    if ((int)(threadIdx.x & 63) == leader) base = atomicAdd(ctr, (uint32_t)__popcll(m));
    base = __shfl(base, leader);
    return base + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

}  // namespace ivf

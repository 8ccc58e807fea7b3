// Exact, order-independent accumulation of float contributions: each value
// is scaled by 2^k and rounded to a 64-bit integer, integers are added (in
// any order, with the same result), and the sum is scaled back once.  The
// shift k is chosen from a bound on the magnitudes so that no sum can exceed
// 2^62; the rounding grid is then about 2^-61 * n * (largest magnitude).
#pragma once

#include "cd_internal.h"

namespace cdk {

// Shift k such that n values of magnitude at most m, each scaled by 2^k and
// rounded to an integer, sum to less than 2^62 in magnitude.  m = 0 gives 0.
__device__ __forceinline__ int fixed_shift(float m, int64_t n)
{
    if (!(m > 0.0f)) return 0;
    int e;
    frexpf(m, &e);                                 // m < 2^e
    const int lg = 64 - __clzll(static_cast<unsigned long long>(n));   // n < 2^lg
    return 61 - e - lg;
}

__device__ __forceinline__ long long to_fixed(float x, int k)
{
    return static_cast<long long>(rintf(ldexpf(x, k)));
}

// Maximum of m over the workgroup (kThreadsPerGroup threads, all of which
// must call it); red holds one float per wave.  Ends with a barrier, so red
// may be reused afterwards.
template <int kThreadsPerGroup>
__device__ __forceinline__ float group_max(float m, float *red)
{
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, kWave));
    if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = m;
    __syncthreads();
    m = red[0];
#pragma unroll
    for (int w = 1; w < kThreadsPerGroup / kWave; ++w) m = fmaxf(m, red[w]);
    __syncthreads();
    return m;
}

}  // namespace cdk

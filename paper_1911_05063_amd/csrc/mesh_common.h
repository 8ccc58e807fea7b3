// Device helpers shared by the mesh kernels (surface sampling, point to
// surface, and the barycentric scatter of their backward passes).
#pragma once

#include "cd_internal.h"

namespace cdk {

__device__ __forceinline__ bool face_ok(const int32_t *t, int64_t nv)
{
    return t[0] >= 0 && t[0] < nv && t[1] >= 0 && t[1] < nv && t[2] >= 0 && t[2] < nv;
}

__device__ __forceinline__ void bary(float r1, float r2, float &wa, float &wb, float &wc)
{
    const float s1 = sqrtf(r1);
    wa = 1.0f - s1;
    wb = s1 * (1.0f - r2);
    wc = s1 * r2;
}

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
    return m;
}

}  // namespace cdk

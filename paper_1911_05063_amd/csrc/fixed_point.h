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

// Maximum over the wave, in every lane: DPP moves within rows of 16 lanes
// (quad permutations, then the half-row and row mirrors), then gfx950's row
// swaps across rows (register moves only, no LDS round trips).
template <int kCtrl>
__device__ __forceinline__ float dpp_f(float v)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kCtrl, 0xF, 0xF, true));
}

__device__ __forceinline__ float wave_max(float m)
{
    m = fmaxf(m, dpp_f<0xB1>(m));    // quad_perm [1,0,3,2]
    m = fmaxf(m, dpp_f<0x4E>(m));    // quad_perm [2,3,0,1]
    m = fmaxf(m, dpp_f<0x141>(m));   // row_half_mirror
    m = fmaxf(m, dpp_f<0x140>(m));   // row_mirror
    const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    m = fmaxf(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
    const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    return fmaxf(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
}

// Maximum of m over the workgroup (kThreadsPerGroup threads, all of which
// must call it); red holds one float per wave.  Ends with a barrier, so red
// may be reused afterwards.
template <int kThreadsPerGroup>
__device__ __forceinline__ float group_max(float m, float *red)
{
    m = wave_max(m);
    if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = m;
    __syncthreads();
    m = red[0];
#pragma unroll
    for (int w = 1; w < kThreadsPerGroup / kWave; ++w) m = fmaxf(m, red[w]);
    __syncthreads();
    return m;
}

}  // namespace cdk

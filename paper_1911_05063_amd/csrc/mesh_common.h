// Device helpers shared by the mesh kernels (surface sampling, point to
// surface, and the barycentric scatter of their backward passes).
#pragma once

#include "cd_internal.h"
#include "fixed_point.h"

namespace cdk {

__device__ __forceinline__ bool face_ok(const int32_t *t, int64_t nv)
{
    return t[0] >= 0 && t[0] < nv && t[1] >= 0 && t[1] < nv && t[2] >= 0 && t[2] < nv;
}

// face_ok without short-circuit evaluation (no branch).
__device__ __forceinline__ bool face_ok_nb(const int32_t t[3], int64_t nv)
{
    return (t[0] >= 0) & (t[0] < nv) & (t[1] >= 0) & (t[1] < nv) & (t[2] >= 0) & (t[2] < nv);
}

__device__ __forceinline__ void bary(float r1, float r2, float &wa, float &wb, float &wc)
{
    const float s1 = sqrtf(r1);
    wa = 1.0f - s1;
    wb = s1 * (1.0f - r2);
    wc = s1 * r2;
}

}  // namespace cdk

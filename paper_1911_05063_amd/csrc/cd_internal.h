// Internal interface between the C-ABI layer (cd_api.cpp) and the gfx950
// kernels.  Not installed; callers use include/cd.h.
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace cdk {

// Sub-tile length of the deferred argmin: the search keeps, per query, only
// the running minimum and the first target of the sub-tile that last lowered
// it; the exact lowest index is recovered by rescanning that sub-tile.
constexpr int kSubTile = 32;
// Queries held in registers by each lane of the search kernel.
constexpr int kQueriesPerLane = 8;
constexpr int kWave = 64;

// One search direction: queries P against targets Q (both [B, n, 3] float32).
struct NNDir {
    const float *P;
    const float *Q;
    float *dist;                 // [B, NP]   written when nsplit == 1
    int32_t *idx;                // [B, NP]   written when nsplit == 1
    unsigned long long *keys;    // [B, NP]   merged with atomicMin when nsplit > 1
    int32_t NP, NQ;
    int32_t nqb;                 // query blocks (kWave * kQueriesPerLane queries) per item
    int32_t nsplit;              // target splits per item
    int32_t chunk;               // targets per split, a multiple of kSubTile
    int32_t pad;
    int64_t items;               // B * nqb * nsplit work items (one wave each)
};

struct NNPlan {
    NNDir d[2];
    int64_t B;
};

// Layout of the forward workspace: the packed (distance, index) merge keys
// of both directions, each segment 256-byte aligned.
struct WsLayout {
    size_t keys_xy, keys_yx, total;
};
WsLayout workspace_layout(int64_t B, int64_t N, int64_t M);

// Fill `plan` for the given shape on a device with `cu_count` compute units.
void make_plan(NNPlan &plan, int64_t B, int64_t N, int64_t M, int cu_count);

hipError_t launch_forward(const NNPlan &plan, hipStream_t stream);

hipError_t launch_reduce(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                         const float *dist_yx, double w1, double w2, float *chamfer,
                         hipStream_t stream);

hipError_t launch_fscore(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                         const float *dist_yx, float thr, float *f, float *precision,
                         float *recall, hipStream_t stream);

// g_xy/g_yx per point when `pointwise`, else per item (grad_out) scaled by
// sxy = w1/N and syx = w2/M.
hipError_t launch_backward(int64_t B, int64_t N, int64_t M, const float *g_xy,
                           const float *g_yx, bool pointwise, float sxy, float syx,
                           const float *X, const float *Y, const int32_t *idx_xy,
                           const int32_t *idx_yx, float *gX, float *gY, hipStream_t stream);

}  // namespace cdk

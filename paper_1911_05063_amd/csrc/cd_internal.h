// Internal interface between the C-ABI layer (cd_api.cpp) and the gfx950
// kernels.  Not installed; callers use include/cd.h.
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace cdk {

constexpr int kWave = 64;

// Tiling of the fused nearest-neighbour search (nn_search.hip).  The X cloud
// is cut into query groups (rows), the Y cloud into target blocks (columns);
// one workgroup computes every distance of one (item, group, block) tile.
struct FwdPlan {
    int64_t B;
    int32_t N, M;
    int32_t nQG;   // query groups per item
    int32_t nTB;   // target blocks per item
    int32_t TB;    // targets per large block (a multiple of the batch length)
    int32_t nBig;  // large blocks per item; the nTB - nBig others hold TS targets
    int32_t TS;    // targets per small block (a multiple of the batch length)
};

struct FwdArgs {
    const float *X;      // [B, N, 3]
    const float *Y;      // [B, M, 3]
    float *dist_xy;      // [B, N]
    int32_t *idx_xy;     // [B, N]
    float *dist_yx;      // [B, M]
    int32_t *idx_yx;     // [B, M]
    void *ws;            // forward_workspace_bytes(plan) bytes, 256-byte aligned
};

// The plan depends on the shape only, so the workspace size does too.
FwdPlan plan_forward(int64_t B, int64_t N, int64_t M);
size_t forward_workspace_bytes(const FwdPlan &plan);
// Number of tiles (workgroups) the search launches; must fit the grid.
int64_t forward_tiles(const FwdPlan &plan);

hipError_t launch_forward(const FwdPlan &plan, const FwdArgs &args, hipStream_t stream);

// The no-allocation forward's workspace: a static device array of this many
// bytes per GPU.  forward_scratch() gives its address on the device of
// `stream` (looked up once per device, with that device current).
constexpr size_t kForwardScratchBytes = size_t(64) << 20;
hipError_t forward_scratch(hipStream_t stream, void **ptr);

hipError_t launch_reduce(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                         const float *dist_yx, double w1, double w2, float *chamfer,
                         hipStream_t stream);

hipError_t launch_fscore(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                         const float *dist_yx, float thr, float *f, float *precision,
                         float *recall, hipStream_t stream);

constexpr int kMaxTaus = 16;

// Chamfer (w1, w2 given) and F-score counts for ntau thresholds (thr[] are the
// float32 thresholds compared against the squared distances) in one launch.
hipError_t launch_metrics(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                          const float *dist_yx, double w1, double w2, const float *thr,
                          int ntau, float *chamfer, float *f, float *precision, float *recall,
                          hipStream_t stream);

// g_xy/g_yx per point when `pointwise`, else per item (grad_out) scaled by
// sxy = w1/N and syx = w2/M.
size_t backward_workspace_bytes(int64_t B, int64_t N, int64_t M);
hipError_t launch_backward(int64_t B, int64_t N, int64_t M, const float *g_xy,
                           const float *g_yx, bool pointwise, float sxy, float syx,
                           const float *X, const float *Y, const int32_t *idx_xy,
                           const int32_t *idx_yx, float *gX, float *gY, void *ws,
                           hipStream_t stream);

// Backward of barycentric interpolation onto mesh vertices (bary_scatter.hip):
// gV[v] = sum of w_{s,v} gP[s] (negated if `negate`) over the samples whose
// face holds v; weights from w [B, S, 3] if given, else from the sampling
// uniforms (r1, r2).  ws: bary_scatter_workspace_bytes(B, nv, S) bytes.
size_t bary_scatter_workspace_bytes(int64_t B, int64_t nv, int64_t S);
hipError_t launch_bary_scatter(int64_t B, int64_t nv, int64_t nf, const int32_t *F, int64_t S,
                               const int32_t *fidx, const float *r1, const float *r2,
                               const float *w, const float *gP, bool negate, float *gV, void *ws,
                               hipStream_t stream);

// Mesh surface sampling (mesh_sample.hip).
size_t mesh_workspace_bytes(int64_t B, int64_t nv, int64_t nf, int64_t S);
hipError_t launch_mesh_choose_faces(int64_t B, int64_t nv, int64_t nf, const float *V,
                                    const int32_t *F, int64_t S, const float *u, int32_t *fidx,
                                    void *ws, hipStream_t stream);
hipError_t launch_mesh_sample_points(int64_t B, int64_t nv, int64_t nf, const float *V,
                                     const int32_t *F, int64_t S, const int32_t *fidx,
                                     const float *r1, const float *r2, float *P,
                                     hipStream_t stream);
hipError_t launch_mesh_sample_backward(int64_t B, int64_t nv, int64_t nf, const int32_t *F,
                                       int64_t S, const int32_t *fidx, const float *r1,
                                       const float *r2, const float *gP, float *gV, void *ws,
                                       hipStream_t stream);

// Point-to-surface distance (p2s.hip).  Points are cut into groups of 2048,
// faces into blocks; one workgroup per (item, group, block).
struct P2SPlan {
    int nQG;   // point groups per item
    int nFB;   // face blocks per item
    int FB;    // faces per large block
    int nBig;  // large blocks per item; the nFB - nBig others hold FS faces
    int FS;    // faces per small block
};
P2SPlan plan_p2s(int64_t B, int64_t S, int64_t nf);
size_t p2s_workspace_bytes(int64_t B, int64_t S, int64_t nv, int64_t nf);
hipError_t launch_p2s_forward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                              const float *V, const int32_t *F, float *dist, int32_t *fidx,
                              void *ws, hipStream_t stream);
hipError_t launch_p2s_backward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                               const float *V, const int32_t *F, const int32_t *fidx,
                               const float *g, float *gP, float *gV, void *ws, hipStream_t stream);

// Approximate Earth-mover's distance (emd.hip): scheduled log-domain Sinkhorn.
size_t emd_workspace_bytes(int64_t B, int64_t N, int64_t M);
float emd_eps(double eps_start, double eps_end, int n_iters, int t);
hipError_t launch_emd_forward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                              double eps_start, double eps_end, int n_iters, bool warm, float *f,
                              float *g, float *cost, void *ws, hipStream_t stream);
hipError_t launch_emd_backward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                               const float *f, const float *g, double eps, const float *go,
                               float *gX, float *gY, void *ws, hipStream_t stream);

}  // namespace cdk

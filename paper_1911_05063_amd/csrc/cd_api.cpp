// C ABI of the batched Chamfer-distance library (declared in include/cd.h):
// argument checking, workspace layout, launch planning and error reporting.
// All device work is enqueued by the launchers in the .hip files.
#include "cd.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>

#include "cd_internal.h"

namespace {

thread_local char g_last_error[512] = "";

cd_status invalid(const char *what)
{
    std::snprintf(g_last_error, sizeof(g_last_error), "invalid argument: %s", what);
    return CD_ERR_INVALID_ARG;
}

cd_status hip_failed(hipError_t e, const char *where)
{
    std::snprintf(g_last_error, sizeof(g_last_error), "%s: %s (%d)", where, hipGetErrorString(e),
                  static_cast<int>(e));
    return CD_ERR_HIP;
}

constexpr int64_t kMaxPoints = 2147483647LL;  // indices are int32

// Shape checks shared by every entry point.
cd_status check_shape(int64_t B, int64_t N, int64_t M)
{
    if (B < 0) return invalid("B < 0");
    if (N < 1) return invalid("N < 1 (nearest neighbour over an empty cloud is undefined)");
    if (M < 1) return invalid("M < 1 (nearest neighbour over an empty cloud is undefined)");
    if (N > kMaxPoints || M > kMaxPoints) return invalid("N or M >= 2^31 (indices are int32)");
    // One thread per point of both clouds (the forward's merge, the backward's
    // passes) must fit a launch: at most 2^31 points in all.
    if (B > 0 && B > (int64_t(1) << 31) / (N + M))
        return invalid("B * (N + M) > 2^31 points for one launch");
    return CD_OK;
}

// a * b > lim for a, b >= 0, without forming a product that could overflow.
bool product_exceeds(int64_t a, int64_t b, int64_t lim) { return a > 0 && b > lim / a; }

bool aligned256(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }

// A float32 squared distance d satisfies d < tau^2 (exact in double for a
// float tau) iff d < thr, where thr is the smallest float32 >= tau^2.
float threshold_of(float tau)
{
    const double t2 = static_cast<double>(tau) * static_cast<double>(tau);
    float thr = static_cast<float>(t2);
    if (static_cast<double>(thr) < t2) thr = std::nextafter(thr, INFINITY);
    return thr;
}

}  // namespace

extern "C" {

const char *cd_status_string(cd_status s)
{
    switch (s) {
    case CD_OK: return "CD_OK";
    case CD_ERR_INVALID_ARG: return "CD_ERR_INVALID_ARG";
    case CD_ERR_WORKSPACE: return "CD_ERR_WORKSPACE";
    case CD_ERR_HIP: return "CD_ERR_HIP";
    }
    return "CD_UNKNOWN_STATUS";
}

const char *cd_last_error(void) { return g_last_error; }

const char *cd_version(void) { return "0.1.0"; }

size_t cd_workspace_bytes(int64_t B, int64_t N, int64_t M)
{
    if (check_shape(B, N, M) != CD_OK) return 0;
    if (B == 0) return 0;
    return cdk::forward_workspace_bytes(cdk::plan_forward(B, N, M));
}

cd_status cd_forward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                     float *dist_xy, int32_t *idx_xy, float *dist_yx, int32_t *idx_yx, void *ws,
                     size_t ws_bytes, hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (B == 0) return CD_OK;
    if (!X || !Y || !dist_xy || !idx_xy || !dist_yx || !idx_yx) return invalid("NULL array pointer");
    const cdk::FwdPlan plan = cdk::plan_forward(B, N, M);
    const size_t need = cdk::forward_workspace_bytes(plan);
    if (!ws || ws_bytes < need) {
        std::snprintf(g_last_error, sizeof(g_last_error),
                      "workspace too small: %zu bytes given, %zu needed", ws_bytes, need);
        return CD_ERR_WORKSPACE;
    }
    if (!aligned256(ws)) return invalid("workspace not 256-byte aligned");
    if (cdk::forward_tiles(plan) > 2147483647LL) return invalid("too many tiles for one launch");
    const cdk::FwdArgs args{X, Y, dist_xy, idx_xy, dist_yx, idx_yx, ws};
    const hipError_t e = cdk::launch_forward(plan, args, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_forward launch");
    return CD_OK;
}

static_assert(CD_FORWARD_NOALLOC_MAX_BYTES == cdk::kForwardScratchBytes,
              "the header's limit is the scratch array's size");

cd_status cd_forward_noalloc(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                             float *dist_xy, int32_t *idx_xy, float *dist_yx, int32_t *idx_yx,
                             hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (B == 0) return CD_OK;
    if (!X || !Y || !dist_xy || !idx_xy || !dist_yx || !idx_yx) return invalid("NULL array pointer");
    const cdk::FwdPlan plan = cdk::plan_forward(B, N, M);
    const size_t need = cdk::forward_workspace_bytes(plan);
    if (need > cdk::kForwardScratchBytes) {
        std::snprintf(g_last_error, sizeof(g_last_error),
                      "cd_forward_noalloc: this shape needs %zu bytes of workspace, more than "
                      "the %zu of the static scratch array (use cd_forward)",
                      need, cdk::kForwardScratchBytes);
        return CD_ERR_WORKSPACE;
    }
    if (cdk::forward_tiles(plan) > 2147483647LL) return invalid("too many tiles for one launch");
    void *ws = nullptr;
    hipError_t e = cdk::forward_scratch(stream, &ws);
    if (e != hipSuccess) return hip_failed(e, "cd_forward_noalloc scratch address");
    const cdk::FwdArgs args{X, Y, dist_xy, idx_xy, dist_yx, idx_yx, ws};
    e = cdk::launch_forward(plan, args, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_forward_noalloc launch");
    return CD_OK;
}

cd_status cd_reduce(int64_t B, int64_t N, int64_t M, const float *dist_xy, const float *dist_yx,
                    float w1, float w2, float *chamfer, hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (B == 0) return CD_OK;
    if (!dist_xy || !dist_yx || !chamfer) return invalid("NULL array pointer");
    const hipError_t e = cdk::launch_reduce(B, N, M, dist_xy, dist_yx, static_cast<double>(w1),
                                            static_cast<double>(w2), chamfer, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_reduce launch");
    return CD_OK;
}

cd_status cd_fscore(int64_t B, int64_t N, int64_t M, const float *dist_xy, const float *dist_yx,
                    float tau, float *f, float *precision, float *recall, hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (std::isnan(tau) || tau < 0.0f) return invalid("tau must be >= 0 and not NaN");
    if (B == 0) return CD_OK;
    if (!dist_xy || !dist_yx || !f) return invalid("NULL array pointer");
    const float thr = threshold_of(tau);
    const hipError_t e =
        cdk::launch_fscore(B, N, M, dist_xy, dist_yx, thr, f, precision, recall, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_fscore launch");
    return CD_OK;
}

cd_status cd_metrics(int64_t B, int64_t N, int64_t M, const float *dist_xy, const float *dist_yx,
                     float w1, float w2, const float *taus, int ntau, float *chamfer, float *f,
                     float *precision, float *recall, hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (!taus || ntau < 1 || ntau > cdk::kMaxTaus) return invalid("need 1 <= ntau <= 16 and taus");
    float thr[cdk::kMaxTaus];
    for (int t = 0; t < ntau; ++t) {
        if (std::isnan(taus[t]) || taus[t] < 0.0f) return invalid("tau must be >= 0 and not NaN");
        thr[t] = threshold_of(taus[t]);
    }
    if (B == 0) return CD_OK;
    if (!dist_xy || !dist_yx || !chamfer || !f) return invalid("NULL array pointer");
    const hipError_t e = cdk::launch_metrics(B, N, M, dist_xy, dist_yx, static_cast<double>(w1),
                                             static_cast<double>(w2), thr, ntau, chamfer, f,
                                             precision, recall, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_metrics launch");
    return CD_OK;
}

size_t cd_backward_workspace_bytes(int64_t B, int64_t N, int64_t M)
{
    if (check_shape(B, N, M) != CD_OK || B == 0) return 0;
    return (cdk::backward_workspace_bytes(B, N, M) + 255) & ~static_cast<size_t>(255);
}

static cd_status check_backward_ws(int64_t B, int64_t N, int64_t M, const void *ws,
                                   size_t ws_bytes)
{
    const size_t need = cd_backward_workspace_bytes(B, N, M);
    if (!ws || ws_bytes < need) {
        std::snprintf(g_last_error, sizeof(g_last_error),
                      "workspace too small: %zu bytes given, %zu needed", ws_bytes, need);
        return CD_ERR_WORKSPACE;
    }
    if (!aligned256(ws)) return invalid("workspace not 256-byte aligned");
    return CD_OK;
}

cd_status cd_backward(int64_t B, int64_t N, int64_t M, const float *grad_out, float w1, float w2,
                      const float *X, const float *Y, const int32_t *idx_xy,
                      const int32_t *idx_yx, float *gX, float *gY, void *ws, size_t ws_bytes,
                      hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (B == 0) return CD_OK;
    if (!grad_out || !X || !Y || !idx_xy || !idx_yx || !gX || !gY)
        return invalid("NULL array pointer");
    s = check_backward_ws(B, N, M, ws, ws_bytes);
    if (s != CD_OK) return s;
    const float sxy = static_cast<float>(static_cast<double>(w1) / static_cast<double>(N));
    const float syx = static_cast<float>(static_cast<double>(w2) / static_cast<double>(M));
    const hipError_t e = cdk::launch_backward(B, N, M, grad_out, grad_out, false, sxy, syx, X, Y,
                                              idx_xy, idx_yx, gX, gY, ws, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_backward launch");
    return CD_OK;
}

cd_status cd_backward_pointwise(int64_t B, int64_t N, int64_t M, const float *g_xy,
                                const float *g_yx, const float *X, const float *Y,
                                const int32_t *idx_xy, const int32_t *idx_yx, float *gX,
                                float *gY, void *ws, size_t ws_bytes, hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (B == 0) return CD_OK;
    if (!g_xy || !g_yx || !X || !Y || !idx_xy || !idx_yx || !gX || !gY)
        return invalid("NULL array pointer");
    s = check_backward_ws(B, N, M, ws, ws_bytes);
    if (s != CD_OK) return s;
    const hipError_t e = cdk::launch_backward(B, N, M, g_xy, g_yx, true, 1.0f, 1.0f, X, Y, idx_xy,
                                              idx_yx, gX, gY, ws, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_backward_pointwise launch");
    return CD_OK;
}

static cd_status check_mesh(int64_t B, int64_t nv, int64_t nf, int64_t S)
{
    if (B < 0) return invalid("B < 0");
    if (nv < 1 || nf < 1) return invalid("a mesh needs nv >= 1 and nf >= 1");
    if (S < 0) return invalid("S < 0");
    if (nv > kMaxPoints || nf > kMaxPoints || S > kMaxPoints) return invalid("nv, nf or S >= 2^31");
    // Per-sample kernels launch B * S threads and the backward B * ceil(nv / 2048)
    // workgroups (times a bounded number of sample chunks).
    if (product_exceeds(B, S, int64_t(1) << 31) ||
        product_exceeds(B, (nv + 2047) / 2048, int64_t(1) << 23))
        return invalid("B * S > 2^31 or B * ceil(nv / 2048) > 2^23");
    return CD_OK;
}

size_t cd_mesh_workspace_bytes(int64_t B, int64_t nv, int64_t nf, int64_t S)
{
    if (check_mesh(B, nv, nf, S) != CD_OK) return 0;
    return (cdk::mesh_workspace_bytes(B, nv, nf, S) + 255) & ~static_cast<size_t>(255);
}

static cd_status check_mesh_ws(int64_t B, int64_t nv, int64_t nf, int64_t S, const void *ws,
                               size_t ws_bytes)
{
    const size_t need = cd_mesh_workspace_bytes(B, nv, nf, S);
    if (need == 0) return CD_OK;
    if (!ws || ws_bytes < need) {
        std::snprintf(g_last_error, sizeof(g_last_error),
                      "workspace too small: %zu bytes given, %zu needed", ws_bytes, need);
        return CD_ERR_WORKSPACE;
    }
    if (!aligned256(ws)) return invalid("workspace not 256-byte aligned");
    return CD_OK;
}

cd_status cd_mesh_sample_faces(int64_t B, int64_t nv, int64_t nf, const float *V, const int32_t *F,
                               int64_t S, const float *u, int32_t *fidx, void *ws, size_t ws_bytes,
                               hipStream_t stream)
{
    cd_status s = check_mesh(B, nv, nf, S);
    if (s != CD_OK) return s;
    if (B == 0) return CD_OK;
    if (!V || !F || (S > 0 && (!u || !fidx))) return invalid("NULL array pointer");
    s = check_mesh_ws(B, nv, nf, S, ws, ws_bytes);
    if (s != CD_OK) return s;
    const hipError_t e = cdk::launch_mesh_choose_faces(B, nv, nf, V, F, S, u, fidx, ws, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_mesh_sample_faces launch");
    return CD_OK;
}

cd_status cd_mesh_sample_points(int64_t B, int64_t nv, int64_t nf, const float *V,
                                const int32_t *F, int64_t S, const int32_t *fidx, const float *r1,
                                const float *r2, float *P, hipStream_t stream)
{
    cd_status s = check_mesh(B, nv, nf, S);
    if (s != CD_OK) return s;
    if (B == 0 || S == 0) return CD_OK;
    if (!V || !F || !fidx || !r1 || !r2 || !P) return invalid("NULL array pointer");
    const hipError_t e = cdk::launch_mesh_sample_points(B, nv, nf, V, F, S, fidx, r1, r2, P, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_mesh_sample_points launch");
    return CD_OK;
}

cd_status cd_mesh_sample_backward(int64_t B, int64_t nv, int64_t nf, const int32_t *F, int64_t S,
                                  const int32_t *fidx, const float *r1, const float *r2,
                                  const float *gP, float *gV, void *ws, size_t ws_bytes,
                                  hipStream_t stream)
{
    cd_status s = check_mesh(B, nv, nf, S);
    if (s != CD_OK) return s;
    if (B == 0) return CD_OK;
    if (!F || !gV || (S > 0 && (!fidx || !r1 || !r2 || !gP))) return invalid("NULL array pointer");
    s = check_mesh_ws(B, nv, nf, S, ws, ws_bytes);
    if (s != CD_OK) return s;
    const hipError_t e =
        cdk::launch_mesh_sample_backward(B, nv, nf, F, S, fidx, r1, r2, gP, gV, ws, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_mesh_sample_backward launch");
    return CD_OK;
}

static cd_status check_p2s(int64_t B, int64_t S, int64_t nv, int64_t nf)
{
    if (B < 0) return invalid("B < 0");
    if (S < 0) return invalid("S < 0");
    if (nv < 1 || nf < 1) return invalid("a mesh needs nv >= 1 and nf >= 1");
    if (nv > kMaxPoints || nf > kMaxPoints || S > kMaxPoints) return invalid("nv, nf or S >= 2^31");
    if (product_exceeds(B, S, int64_t(1) << 31) || product_exceeds(B, nf, int64_t(1) << 31) ||
        product_exceeds(B, (nv + 2047) / 2048, int64_t(1) << 23))
        return invalid("B * S > 2^31, B * nf > 2^31 or B * ceil(nv / 2048) > 2^23");
    return CD_OK;
}

static cd_status check_ws(size_t need, const void *ws, size_t ws_bytes)
{
    if (!ws || ws_bytes < need) {
        std::snprintf(g_last_error, sizeof(g_last_error),
                      "workspace too small: %zu bytes given, %zu needed", ws_bytes, need);
        return CD_ERR_WORKSPACE;
    }
    if (!aligned256(ws)) return invalid("workspace not 256-byte aligned");
    return CD_OK;
}

size_t cd_p2s_workspace_bytes(int64_t B, int64_t S, int64_t nv, int64_t nf)
{
    if (check_p2s(B, S, nv, nf) != CD_OK) return 0;
    return (cdk::p2s_workspace_bytes(B, S, nv, nf) + 255) & ~static_cast<size_t>(255);
}

cd_status cd_p2s_forward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                         const float *V, const int32_t *F, float *dist, int32_t *fidx, void *ws,
                         size_t ws_bytes, hipStream_t stream)
{
    cd_status s = check_p2s(B, S, nv, nf);
    if (s != CD_OK) return s;
    if (B == 0 || S == 0) return CD_OK;
    if (!P || !V || !F || !dist || !fidx) return invalid("NULL array pointer");
    s = check_ws(cd_p2s_workspace_bytes(B, S, nv, nf), ws, ws_bytes);
    if (s != CD_OK) return s;
    const hipError_t e = cdk::launch_p2s_forward(B, S, nv, nf, P, V, F, dist, fidx, ws, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_p2s_forward launch");
    return CD_OK;
}

cd_status cd_p2s_backward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                          const float *V, const int32_t *F, const int32_t *fidx, const float *g,
                          float *gP, float *gV, void *ws, size_t ws_bytes, hipStream_t stream)
{
    cd_status s = check_p2s(B, S, nv, nf);
    if (s != CD_OK) return s;
    if (B == 0 || (!gP && !gV)) return CD_OK;
    if (!F || (S > 0 && (!P || !V || !fidx || !g))) return invalid("NULL array pointer");
    s = check_ws(cd_p2s_workspace_bytes(B, S, nv, nf), ws, ws_bytes);
    if (s != CD_OK) return s;
    const hipError_t e =
        cdk::launch_p2s_backward(B, S, nv, nf, P, V, F, fidx, g, gP, gV, ws, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_p2s_backward launch");
    return CD_OK;
}

size_t cd_emd_workspace_bytes(int64_t B, int64_t N, int64_t M)
{
    if (check_shape(B, N, M) != CD_OK || B == 0) return 0;
    return (cdk::emd_workspace_bytes(B, N, M) + 255) & ~static_cast<size_t>(255);
}

static bool positive_finite(float v) { return v > 0.0f && std::isfinite(v); }

cd_status cd_emd_forward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                         float eps_start, float eps_end, int n_iters, int warm_start, float *f,
                         float *g, float *cost, void *ws, size_t ws_bytes, hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (!positive_finite(eps_start) || !positive_finite(eps_end))
        return invalid("eps_start and eps_end must be positive and finite");
    if (n_iters < 1) return invalid("n_iters < 1");
    if (product_exceeds(B, 3 * std::max(N, M), (int64_t(1) << 32) - (int64_t(1) << 20)))
        return invalid("3 B max(N, M) >= 2^32 (one thread per gradient component)");
    if (B == 0) return CD_OK;
    if (!X || !Y || !f || !g || !cost) return invalid("NULL array pointer");
    s = check_ws(cd_emd_workspace_bytes(B, N, M), ws, ws_bytes);
    if (s != CD_OK) return s;
    const hipError_t e = cdk::launch_emd_forward(B, N, M, X, Y, eps_start, eps_end, n_iters,
                                                 warm_start != 0, f, g, cost, ws, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_emd_forward launch");
    return CD_OK;
}

cd_status cd_emd_backward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                          const float *f, const float *g, float eps, const float *grad_out,
                          float *gX, float *gY, void *ws, size_t ws_bytes, hipStream_t stream)
{
    cd_status s = check_shape(B, N, M);
    if (s != CD_OK) return s;
    if (!positive_finite(eps)) return invalid("eps must be positive and finite");
    if (product_exceeds(B, 3 * std::max(N, M), (int64_t(1) << 32) - (int64_t(1) << 20)))
        return invalid("3 B max(N, M) >= 2^32 (one thread per gradient component)");
    if (B == 0) return CD_OK;
    if (!X || !Y || !f || !g || !grad_out || !gX || !gY) return invalid("NULL array pointer");
    s = check_ws(cd_emd_workspace_bytes(B, N, M), ws, ws_bytes);
    if (s != CD_OK) return s;
    const hipError_t e =
        cdk::launch_emd_backward(B, N, M, X, Y, f, g, eps, grad_out, gX, gY, ws, stream);
    if (e != hipSuccess) return hip_failed(e, "cd_emd_backward launch");
    return CD_OK;
}

}  // extern "C"

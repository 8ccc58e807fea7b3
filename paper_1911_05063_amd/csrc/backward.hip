// Backward of the Chamfer loss (Kaolin Sec. 2.5: Chamfer distance as a loss
// that supervises networks) for the neighbours the forward chose.
//
// d dist_xy[i] / d x_i = 2 (x_i - y_j) and d dist_xy[i] / d y_j = -2 (x_i - y_j)
// for j = idx_xy[i]; symmetrically for dist_yx.  Two launches on the stream:
//  1. own terms: every gX[i] / gY[j] is overwritten with its own direction's
//     term (plain stores, so no clearing pass is needed);
//  2. scatter terms: each point subtracts its term from its neighbour's
//     gradient with a hardware float atomic add (global_atomic_add_f32).
// Both are O(B (N + M)) and memory/atomic-latency bound.
#include "cd_internal.h"

namespace cdk {
namespace {

constexpr int kBlock = 256;

struct BwdArgs {
    const float *gxy;   // [B] (per item) or [B, N] (pointwise)
    const float *gyx;   // [B] or [B, M]
    const float *X;
    const float *Y;
    const int32_t *idx_xy;
    const int32_t *idx_yx;
    float *gX;
    float *gY;
    int64_t B, N, M;
    float sxy, syx;     // per-item scale (w1/N, w2/M) when not pointwise
    int pointwise;
};

// Thread t < B*N handles x-point t (direction X->Y); the rest handle y-points.
template <bool kScatter>
__global__ __launch_bounds__(kBlock) void backward_kernel(BwdArgs a)
{
    const int64_t t = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int64_t nx = a.B * a.N;
    const int64_t total = nx + a.B * a.M;
    if (t >= total) return;
    const bool xdir = t < nx;
    const int64_t p = xdir ? t : t - nx;                 // query point (flat)
    const int64_t NP = xdir ? a.N : a.M;
    const int64_t NQ = xdir ? a.M : a.N;
    const int64_t b = p / NP;
    const float *P = xdir ? a.X : a.Y;
    const float *Q = xdir ? a.Y : a.X;
    const int32_t nb = xdir ? a.idx_xy[p] : a.idx_yx[p];
    if (nb < 0 || nb >= NQ) {  // not a neighbour index: the point contributes nothing
        if (!kScatter) {
            float *own = xdir ? a.gX : a.gY;
            own[3 * p + 0] = 0.0f;
            own[3 * p + 1] = 0.0f;
            own[3 * p + 2] = 0.0f;
        }
        return;
    }
    const int64_t q = b * NQ + nb;  // neighbour (flat)
    float g;
    if (a.pointwise)
        g = xdir ? a.gxy[p] : a.gyx[p];
    else
        g = (xdir ? a.gxy[b] : a.gyx[b]) * (xdir ? a.sxy : a.syx);
    const float g2 = 2.0f * g;
    float *own = xdir ? a.gX : a.gY;
    float *nbr = xdir ? a.gY : a.gX;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
        const float term = g2 * (P[3 * p + c] - Q[3 * q + c]);
        if (kScatter)
            unsafeAtomicAdd(nbr + 3 * q + c, -term);
        else
            own[3 * p + c] = term;
    }
}

}  // namespace

hipError_t launch_backward(int64_t B, int64_t N, int64_t M, const float *g_xy,
                           const float *g_yx, bool pointwise, float sxy, float syx,
                           const float *X, const float *Y, const int32_t *idx_xy,
                           const int32_t *idx_yx, float *gX, float *gY, hipStream_t stream)
{
    BwdArgs a{g_xy, g_yx, X, Y, idx_xy, idx_yx, gX, gY, B, N, M, sxy, syx, pointwise ? 1 : 0};
    const int64_t total = B * (N + M);
    const uint32_t grid = static_cast<uint32_t>((total + kBlock - 1) / kBlock);
    backward_kernel<false><<<grid, kBlock, 0, stream>>>(a);
    backward_kernel<true><<<grid, kBlock, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace cdk

// Backward of the Chamfer loss (Kaolin Sec. 2.5: Chamfer distance as a loss
// that supervises networks) for the neighbours the forward chose.
//
// d dist_xy[i] / d x_i = 2 (x_i - y_j) and d dist_xy[i] / d y_j = -2 (x_i - y_j)
// for j = idx_xy[i]; symmetrically for dist_yx.  So
//   gX[i] = 2 g_xy(i) (x_i - y_{idx_xy[i]}) - sum_{j: idx_yx[j] = i} 2 g_yx(j) (y_j - x_i)
//   gY[j] = 2 g_yx(j) (y_j - x_{idx_yx[j]}) - sum_{i: idx_xy[i] = j} 2 g_xy(i) (x_i - y_j)
//
// One launch, no global atomics.  A workgroup owns a slice of kSlice points of
// one cloud (the receiving side) of one item: it scans the other cloud's
// neighbour indices, adds the scatter terms that land in its slice to LDS
// accumulators (ds_add_f32), then writes own term + accumulated scatter once
// per point.  Global float atomics on this chip are executed far from the CU
// (about 20 G/s measured), LDS atomics next to it.  The order of the LDS
// additions varies from run to run, so the last bits may too.
#include "cd_internal.h"

namespace cdk {
namespace {

constexpr int kBlock = 512;
constexpr int kSlice = 2048;
constexpr int kUnroll = 8;

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
    int nsx, nsy;       // slices of X and of Y per item
};

// dL/d dist of point p (flat index) of cloud X (xdir) or Y, item b.
__device__ __forceinline__ float weight(const BwdArgs &a, bool xdir, int64_t b, int64_t p)
{
    if (a.pointwise) return xdir ? a.gxy[p] : a.gyx[p];
    return (xdir ? a.gxy[b] : a.gyx[b]) * (xdir ? a.sxy : a.syx);
}

// Workgroup (b, side, slice).  side 0 writes gX[b, slice], side 1 gY[b, slice].
__global__ __launch_bounds__(kBlock) void backward_kernel(BwdArgs a)
{
    __shared__ float acc[3][kSlice];
    const int per_item = a.nsx + a.nsy;
    const int64_t b = blockIdx.x / per_item;
    const int r = blockIdx.x % per_item;
    const bool xside = r < a.nsx;                 // receiving cloud is X
    const int64_t s0 = static_cast<int64_t>(xside ? r : r - a.nsx) * kSlice;
    const int64_t nrecv = xside ? a.N : a.M;      // points of the receiving cloud
    const int64_t nsend = xside ? a.M : a.N;      // points of the other cloud
    const int64_t s1 = min(s0 + kSlice, nrecv);
    const float *R = (xside ? a.X : a.Y) + b * nrecv * 3;              // receiving, item b
    const float *S = (xside ? a.Y : a.X) + b * nsend * 3;              // sending, item b
    const int32_t *sidx = (xside ? a.idx_yx : a.idx_xy) + b * nsend;   // sender -> receiver
    const int32_t *ridx = (xside ? a.idx_xy : a.idx_yx) + b * nrecv;   // receiver -> sender
    float *out = (xside ? a.gX : a.gY) + b * nrecv * 3;

    for (int t = threadIdx.x; t < kSlice; t += kBlock) {
        acc[0][t] = 0.0f;
        acc[1][t] = 0.0f;
        acc[2][t] = 0.0f;
    }
    __syncthreads();

    // Scatter terms of senders whose neighbour lies in this slice:
    // -2 g(s) (s - r) added to r.  kUnroll senders per thread per round, with
    // every load issued before the first wait (out-of-slice lanes read a
    // clamped, valid address and add nothing).
    const bool spw = a.pointwise != 0;
    const float g2s_item = spw ? 0.0f : 2.0f * weight(a, !xside, b, 0);
    const float *gsend = (xside ? a.gyx : a.gxy) + (spw ? b * nsend : 0);  // [B, n] only if pointwise
    for (int64_t base = 0; base < nsend; base += static_cast<int64_t>(kBlock) * kUnroll) {
        int64_t qs[kUnroll], is[kUnroll];
        bool in[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t q = base + static_cast<int64_t>(u) * kBlock + threadIdx.x;
            qs[u] = min(q, nsend - 1);
            const int64_t i = sidx[qs[u]];
            in[u] = q < nsend && i >= s0 && i < s1;
            is[u] = in[u] ? i : s0;
        }
        float sv[kUnroll][3], rv[kUnroll][3], g2[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
            for (int c = 0; c < 3; ++c) {
                sv[u][c] = S[3 * qs[u] + c];
                rv[u][c] = R[3 * is[u] + c];
            }
            g2[u] = spw ? 2.0f * gsend[qs[u]] : g2s_item;
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            if (in[u]) {
                const int64_t l = is[u] - s0;
#pragma unroll
                for (int c = 0; c < 3; ++c) atomicAdd(&acc[c][l], -(g2[u] * (sv[u][c] - rv[u][c])));
            }
        }
    }
    __syncthreads();

    // Own term plus the accumulated scatter, written once per point.  A point
    // whose neighbour index is out of range contributes nothing.
    const float g2r_item = spw ? 0.0f : 2.0f * weight(a, xside, b, 0);
    const float *grecv = (xside ? a.gxy : a.gyx) + (spw ? b * nrecv : 0);
#pragma unroll 4
    for (int64_t p = s0 + threadIdx.x; p < s1; p += kBlock) {
        const int64_t l = p - s0;
        const int32_t nb = ridx[p];
        const bool ok = nb >= 0 && nb < nsend;
        const int64_t qn = ok ? nb : 0;
        const float g2 = ok ? (spw ? 2.0f * grecv[p] : g2r_item) : 0.0f;
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            const float own = g2 * (R[3 * p + c] - S[3 * qn + c]);
            out[3 * p + c] = own + acc[c][l];
        }
    }
}

}  // namespace

hipError_t launch_backward(int64_t B, int64_t N, int64_t M, const float *g_xy,
                           const float *g_yx, bool pointwise, float sxy, float syx,
                           const float *X, const float *Y, const int32_t *idx_xy,
                           const int32_t *idx_yx, float *gX, float *gY, hipStream_t stream)
{
    BwdArgs a{g_xy, g_yx, X, Y, idx_xy, idx_yx, gX, gY, B, N, M, sxy, syx, pointwise ? 1 : 0,
              static_cast<int>((N + kSlice - 1) / kSlice),
              static_cast<int>((M + kSlice - 1) / kSlice)};
    const int64_t grid = B * (a.nsx + a.nsy);
    backward_kernel<<<static_cast<uint32_t>(grid), kBlock, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace cdk

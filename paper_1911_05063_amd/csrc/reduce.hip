// Per-item reductions over the nearest-neighbour distances (Kaolin Sec. 2.5):
// the Chamfer reduction (sum of the two directional means) and the F-score
// match counts.  One kernel serves cd_reduce (Chamfer only), cd_fscore (one
// threshold) and cd_metrics (Chamfer and up to 4 thresholds per pass), so the
// three share one accumulation order and agree bitwise.  One 1024-thread
// workgroup per item: each thread sums its elements in order (in double: the
// rows are long, and a float32 running sum over 1e5 terms could drift past
// 1e-5 relative) with 16 loads in flight (32 for the first group: both
// arrays at once), counts come from wave ballots, and
// a single reduction (wave shuffles, then the 16 waves in order) combines
// everything, so the results are bitwise reproducible.
#include "cd_internal.h"

#include <algorithm>

namespace cdk {
namespace {

constexpr int kBlock = 1024;
constexpr int kWaves = kBlock / kWave;
constexpr int kGroup = 16;          // loads in flight per thread

struct Thresholds {
    float thr[kMaxTaus];
};

// Chamfer sums (if do_chamfer) and the match counts of thresholds
// first_tau .. first_tau+NT-1 (NT = 0..4).
template <int NT>
__global__ __launch_bounds__(kBlock) void metrics_kernel(int64_t N, int64_t M, const float *dxy,
                                                         const float *dyx, double w1, double w2,
                                                         Thresholds th, int first_tau,
                                                         int do_chamfer, int64_t B,
                                                         float *chamfer, float *f, float *prec,
                                                         float *rec)
{
    __shared__ double dred[kWaves][2];
    __shared__ unsigned long long ured[kWaves][2 * (NT > 0 ? NT : 1)];
    const int64_t b = blockIdx.x;
    const float *a = dxy + b * N;
    const float *c = dyx + b * M;
    float thr[NT > 0 ? NT : 1];
#pragma unroll
    for (int t = 0; t < NT; ++t) thr[t] = th.thr[first_tau + t];
    double sx = 0.0, sy = 0.0;
    unsigned long long cp[NT > 0 ? NT : 1], cr[NT > 0 ? NT : 1];
#pragma unroll
    for (int t = 0; t < (NT > 0 ? NT : 1); ++t) cp[t] = cr[t] = 0ull;
    // Groups of kGroup full strides (no bounds checks, all loads in flight;
    // unrolled by hand because loops holding ballots are not unrolled by the
    // compiler), then the remaining full strides as one guarded group, then
    // one partial stride.  Every lane runs the same trip counts, so the
    // ballots see the full wave.
    auto take = [&](float v, double &sum, unsigned long long (&cnt)[NT > 0 ? NT : 1]) {
        if (do_chamfer) sum += static_cast<double>(v);
#pragma unroll
        for (int t = 0; t < NT; ++t) cnt[t] += __popcll(__ballot(v < thr[t]));
    };
    auto pass = [&](const float *p, int64_t n, double &sum, unsigned long long (&cnt)[NT > 0 ? NT : 1],
                    int64_t s) {
        const int64_t full = n / kBlock;
        for (; s + kGroup <= full; s += kGroup) {
            float v[kGroup];
#pragma unroll
            for (int u = 0; u < kGroup; ++u) v[u] = p[(s + u) * kBlock + threadIdx.x];
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                if (do_chamfer) sum += static_cast<double>(v[u]);
#pragma unroll
                for (int t = 0; t < NT; ++t) cnt[t] += __popcll(__ballot(v[u] < thr[t]));
            }
        }
        if (s < full) {
            // The remaining (fewer than kGroup) full strides, loads in flight
            // together; the guard is the same for every lane.
            float v[kGroup];
#pragma unroll
            for (int u = 0; u < kGroup; ++u)
                v[u] = s + u < full ? p[(s + u) * kBlock + threadIdx.x] : 0.0f;
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                if (s + u < full) {
                    if (do_chamfer) sum += static_cast<double>(v[u]);
#pragma unroll
                    for (int t = 0; t < NT; ++t) cnt[t] += __popcll(__ballot(v[u] < thr[t]));
                }
            }
            s = full;
        }
        const int64_t i = full * kBlock + threadIdx.x;
        const bool in = i < n;
        const float v = in ? p[i] : 0.0f;
        if (do_chamfer && in) sum += static_cast<double>(v);
#pragma unroll
        for (int t = 0; t < NT; ++t) cnt[t] += __popcll(__ballot(in && v < thr[t]));
    };
    // The first group of each array is loaded together (one memory round
    // instead of two when both arrays have a full group); the sums still take
    // every array's elements in order.
    int64_t s0 = 0;
    if (N / kBlock >= kGroup && M / kBlock >= kGroup) {
        float va[kGroup], vc[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            va[u] = a[u * kBlock + threadIdx.x];
            vc[u] = c[u * kBlock + threadIdx.x];
        }
#pragma unroll
        for (int u = 0; u < kGroup; ++u) take(va[u], sx, cp);
#pragma unroll
        for (int u = 0; u < kGroup; ++u) take(vc[u], sy, cr);
        s0 = kGroup;
    }
    pass(a, N, sx, cp, s0);
    pass(c, M, sy, cr, s0);
    // One reduction for everything: sums over the wave by shuffles (counts are
    // already per wave: every lane holds the wave's ballot totals), then the
    // waves in order.
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        sx += __shfl_xor(sx, off, kWave);
        sy += __shfl_xor(sy, off, kWave);
    }
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) {
        dred[w][0] = sx;
        dred[w][1] = sy;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            ured[w][2 * t] = cp[t];
            ured[w][2 * t + 1] = cr[t];
        }
    }
    __syncthreads();
    if (threadIdx.x == 0 && do_chamfer) {
        double tx = 0.0, ty = 0.0;
        for (int v = 0; v < kWaves; ++v) {
            tx += dred[v][0];
            ty += dred[v][1];
        }
        chamfer[b] = static_cast<float>(w1 * (tx / static_cast<double>(N)) +
                                        w2 * (ty / static_cast<double>(M)));
    }
    if (threadIdx.x >= 1 && threadIdx.x <= NT) {
        const int t = threadIdx.x - 1;
        unsigned long long np = 0, nr = 0;
        for (int v = 0; v < kWaves; ++v) {
            np += ured[v][2 * t];
            nr += ured[v][2 * t + 1];
        }
        const double P = static_cast<double>(np) / static_cast<double>(N);
        const double R = static_cast<double>(nr) / static_cast<double>(M);
        const double F = (P + R > 0.0) ? (2.0 * P * R) / (P + R) : 0.0;
        const int64_t o = static_cast<int64_t>(first_tau + t) * B + b;
        f[o] = static_cast<float>(F);
        if (prec) prec[o] = static_cast<float>(P);
        if (rec) rec[o] = static_cast<float>(R);
    }
}

}  // namespace

hipError_t launch_metrics(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                          const float *dist_yx, double w1, double w2, const float *thr,
                          int ntau, float *chamfer, float *f, float *precision, float *recall,
                          hipStream_t stream)
{
    Thresholds th;
    for (int t = 0; t < kMaxTaus; ++t) th.thr[t] = (t < ntau) ? thr[t] : 0.0f;
    const uint32_t grid = static_cast<uint32_t>(B);
    for (int t0 = 0; t0 < ntau; t0 += 4) {
        const int ch = (t0 == 0 && chamfer) ? 1 : 0;
        switch (std::min(4, ntau - t0)) {
        case 1:
            metrics_kernel<1><<<grid, kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, w1, w2, th, t0,
                                                          ch, B, chamfer, f, precision, recall);
            break;
        case 2:
            metrics_kernel<2><<<grid, kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, w1, w2, th, t0,
                                                          ch, B, chamfer, f, precision, recall);
            break;
        case 3:
            metrics_kernel<3><<<grid, kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, w1, w2, th, t0,
                                                          ch, B, chamfer, f, precision, recall);
            break;
        default:
            metrics_kernel<4><<<grid, kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, w1, w2, th, t0,
                                                          ch, B, chamfer, f, precision, recall);
            break;
        }
    }
    return hipGetLastError();
}

hipError_t launch_reduce(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                         const float *dist_yx, double w1, double w2, float *chamfer,
                         hipStream_t stream)
{
    Thresholds th{};
    metrics_kernel<0><<<static_cast<uint32_t>(B), kBlock, 0, stream>>>(
        N, M, dist_xy, dist_yx, w1, w2, th, 0, 1, B, chamfer, nullptr, nullptr, nullptr);
    return hipGetLastError();
}

hipError_t launch_fscore(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                         const float *dist_yx, float thr, float *f, float *precision,
                         float *recall, hipStream_t stream)
{
    Thresholds th{};
    th.thr[0] = thr;
    metrics_kernel<1><<<static_cast<uint32_t>(B), kBlock, 0, stream>>>(
        N, M, dist_xy, dist_yx, 1.0, 1.0, th, 0, 0, B, nullptr, f, precision, recall);
    return hipGetLastError();
}

}  // namespace cdk

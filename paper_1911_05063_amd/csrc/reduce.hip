// Per-item reductions over the nearest-neighbour distances (Kaolin Sec. 2.5):
// the Chamfer reduction (sum of the two directional means) and the F-score
// match counts, separately or fused (metrics_kernel).  One 1024-thread workgroup per item; wave shuffles, then LDS,
// combine the per-lane partials in a fixed order, so the results are bitwise
// reproducible.  Chamfer sums are carried in double (the rows are long: a
// float32 running sum over 1e5 terms could drift past 1e-5 relative).
#include "cd_internal.h"

#include <algorithm>

namespace cdk {
namespace {

constexpr int kBlock = 1024;
constexpr int kWaves = kBlock / kWave;

template <typename T>
__device__ __forceinline__ T wave_sum(T v)
{
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Sum over the workgroup; the total is returned to every thread.
template <typename T>
__device__ __forceinline__ T block_sum(T v, T *scratch)
{
    v = wave_sum(v);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0) scratch[w] = v;
    __syncthreads();
    T t = (threadIdx.x < kWaves) ? scratch[threadIdx.x] : T(0);
    if (threadIdx.x < kWave) t = wave_sum(t);
    if (threadIdx.x == 0) scratch[0] = t;
    __syncthreads();
    const T r = scratch[0];
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(kBlock) void chamfer_reduce_kernel(int64_t N, int64_t M,
                                                                const float *dxy,
                                                                const float *dyx, double w1,
                                                                double w2, float *out)
{
    __shared__ double scratch[kWaves];
    const int64_t b = blockIdx.x;
    const float *a = dxy + b * N;
    const float *c = dyx + b * M;
    double sx = 0.0, sy = 0.0;
#pragma unroll 16
    for (int64_t i = threadIdx.x; i < N; i += kBlock) sx += static_cast<double>(a[i]);
#pragma unroll 16
    for (int64_t j = threadIdx.x; j < M; j += kBlock) sy += static_cast<double>(c[j]);
    sx = block_sum(sx, scratch);
    sy = block_sum(sy, scratch);
    if (threadIdx.x == 0)
        out[b] = static_cast<float>(w1 * (sx / static_cast<double>(N)) +
                                    w2 * (sy / static_cast<double>(M)));
}

__global__ __launch_bounds__(kBlock) void fscore_kernel(int64_t N, int64_t M, const float *dxy,
                                                        const float *dyx, float thr, float *f,
                                                        float *prec, float *rec)
{
    __shared__ unsigned long long scratch[kWaves];
    const int64_t b = blockIdx.x;
    const float *a = dxy + b * N;
    const float *c = dyx + b * M;
    unsigned long long cp = 0, cr = 0;
#pragma unroll 16
    for (int64_t i = threadIdx.x; i < N; i += kBlock) cp += (a[i] < thr) ? 1u : 0u;
#pragma unroll 16
    for (int64_t j = threadIdx.x; j < M; j += kBlock) cr += (c[j] < thr) ? 1u : 0u;
    cp = block_sum(cp, scratch);
    cr = block_sum(cr, scratch);
    if (threadIdx.x == 0) {
        const double P = static_cast<double>(cp) / static_cast<double>(N);
        const double R = static_cast<double>(cr) / static_cast<double>(M);
        const double F = (P + R > 0.0) ? (2.0 * P * R) / (P + R) : 0.0;
        f[b] = static_cast<float>(F);
        if (prec) prec[b] = static_cast<float>(P);
        if (rec) rec[b] = static_cast<float>(R);
    }
}

struct Thresholds {
    float thr[kMaxTaus];
};

// Chamfer reduction and F-score counts for up to 4 thresholds (NT) per pass;
// the same accumulation order and reduction tree as the two kernels above, so
// the results are bitwise equal to theirs.  Counts are taken per wave with
// ballots.  Pass `first_tau` handles thresholds first_tau .. first_tau+NT-1;
// the Chamfer value is written by the first pass only.
template <int NT>
__global__ __launch_bounds__(kBlock) void metrics_kernel(int64_t N, int64_t M, const float *dxy,
                                                         const float *dyx, double w1, double w2,
                                                         Thresholds th, int first_tau, int64_t B,
                                                         float *chamfer, float *f, float *prec,
                                                         float *rec)
{
    __shared__ double dscratch[kWaves];
    __shared__ unsigned long long uscratch[kWaves];
    const int64_t b = blockIdx.x;
    const float *a = dxy + b * N;
    const float *c = dyx + b * M;
    const bool do_chamfer = first_tau == 0;
    float thr[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) thr[t] = th.thr[first_tau + t];
    double sx = 0.0, sy = 0.0;
    unsigned long long cp[NT], cr[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) cp[t] = cr[t] = 0ull;
    // Full strides in groups of kGroup (no bounds checks: the group's loads
    // are all in flight together; unrolled by hand because loops holding
    // ballots are not unrolled by the compiler), then single full strides,
    // then one partial stride.  Every lane runs the same trip counts, so the
    // ballots see the full wave.
    constexpr int kGroup = 8;
    auto pass = [&](const float *p, int64_t n, double &sum, unsigned long long (&cnt)[NT]) {
        const int64_t full = n / kBlock;
        int64_t s = 0;
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
        for (; s < full; ++s) {
            const float v = p[s * kBlock + threadIdx.x];
            if (do_chamfer) sum += static_cast<double>(v);
#pragma unroll
            for (int t = 0; t < NT; ++t) cnt[t] += __popcll(__ballot(v < thr[t]));
        }
        const int64_t i = full * kBlock + threadIdx.x;
        const bool in = i < n;
        const float v = in ? p[i] : 0.0f;
        if (do_chamfer && in) sum += static_cast<double>(v);
#pragma unroll
        for (int t = 0; t < NT; ++t) cnt[t] += __popcll(__ballot(in && v < thr[t]));
    };
    pass(a, N, sx, cp);
    pass(c, M, sy, cr);
    if (do_chamfer) {
        sx = block_sum(sx, dscratch);
        sy = block_sum(sy, dscratch);
        if (threadIdx.x == 0)
            chamfer[b] = static_cast<float>(w1 * (sx / static_cast<double>(N)) +
                                            w2 * (sy / static_cast<double>(M)));
    }
    // Each wave counted its lanes once per element; lane 0 carries the wave's
    // counts into the block sum.
    const bool lead = (threadIdx.x % kWave) == 0;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const unsigned long long np = block_sum(lead ? cp[t] : 0ull, uscratch);
        const unsigned long long nr = block_sum(lead ? cr[t] : 0ull, uscratch);
        if (threadIdx.x == 0) {
            const double P = static_cast<double>(np) / static_cast<double>(N);
            const double R = static_cast<double>(nr) / static_cast<double>(M);
            const double F = (P + R > 0.0) ? (2.0 * P * R) / (P + R) : 0.0;
            const int64_t o = static_cast<int64_t>(first_tau + t) * B + b;
            f[o] = static_cast<float>(F);
            if (prec) prec[o] = static_cast<float>(P);
            if (rec) rec[o] = static_cast<float>(R);
        }
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
        switch (std::min(4, ntau - t0)) {
        case 1:
            metrics_kernel<1><<<grid, kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, w1, w2, th, t0,
                                                          B, chamfer, f, precision, recall);
            break;
        case 2:
            metrics_kernel<2><<<grid, kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, w1, w2, th, t0,
                                                          B, chamfer, f, precision, recall);
            break;
        case 3:
            metrics_kernel<3><<<grid, kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, w1, w2, th, t0,
                                                          B, chamfer, f, precision, recall);
            break;
        default:
            metrics_kernel<4><<<grid, kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, w1, w2, th, t0,
                                                          B, chamfer, f, precision, recall);
            break;
        }
    }
    return hipGetLastError();
}

hipError_t launch_reduce(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                         const float *dist_yx, double w1, double w2, float *chamfer,
                         hipStream_t stream)
{
    chamfer_reduce_kernel<<<static_cast<uint32_t>(B), kBlock, 0, stream>>>(N, M, dist_xy, dist_yx,
                                                                          w1, w2, chamfer);
    return hipGetLastError();
}

hipError_t launch_fscore(int64_t B, int64_t N, int64_t M, const float *dist_xy,
                         const float *dist_yx, float thr, float *f, float *precision,
                         float *recall, hipStream_t stream)
{
    fscore_kernel<<<static_cast<uint32_t>(B), kBlock, 0, stream>>>(N, M, dist_xy, dist_yx, thr, f,
                                                                  precision, recall);
    return hipGetLastError();
}

}  // namespace cdk

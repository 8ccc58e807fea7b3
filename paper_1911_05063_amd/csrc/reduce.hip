// Per-item reductions over the nearest-neighbour distances (Kaolin Sec. 2.5):
// the Chamfer reduction (sum of the two directional means) and the F-score
// match counts.  One 1024-thread workgroup per item; wave shuffles, then LDS,
// combine the per-lane partials in a fixed order, so the results are bitwise
// reproducible.  Chamfer sums are carried in double (the rows are long: a
// float32 running sum over 1e5 terms could drift past 1e-5 relative).
#include "cd_internal.h"

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

}  // namespace

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

// Approximate Earth-mover's distance between point clouds (Kaolin Sec. 2.5
// names an approximate EMD among its point-cloud metrics, citing Fan et al.): the optimal
// transport problem with uniform masses a = 1/N, b = 1/M and Euclidean cost
// C_ij = |x_i - y_j|, regularised by entropy and solved with log-domain
// Sinkhorn iterations, each touching all N*M pairs.  With a scheduled eps:
//     f_i <- -eps log sum_j b exp((g_j - C_ij) / eps)
//     g_j <- -eps log sum_i a exp((f_i - C_ij) / eps)
// and the plan P_ij = a b exp((f_i + g_j - C_ij) / eps), the cost is
// sum_ij P_ij C_ij; its backward holds P fixed:
//     d cost / d x_i = sum_j P_ij (x_i - y_j) / C_ij,  d cost / d y_j = the opposite sum.
//
//  * lse_kernel: one half-update.  A workgroup holds 1024 queries (4 per
//    lane) in VGPRs and walks a block of targets; the target index is
//    wave-uniform, so coordinates and potentials arrive by scalar loads.  The
//    log-sum-exp runs in base 2 online over batches of 16 targets: the batch
//    maximum rescales the running sum once per batch, then each pair adds
//    exp2(z - max), z = (g_j - C_ij) log2(e) / eps.  With several target
//    blocks a half-update leaves (max, sum) partials per query; the next
//    half-update merges them for its own target block (1024 targets at a time
//    into LDS) instead of reading finished potentials, and lse_merge_kernel
//    merges them, with the same function, only where finished potentials are
//    needed (the outputs).
//  * plan_kernel: per (query block, target block) tile, either the tile's
//    sum of P_ij C_ij (in double, reduced in a fixed order) or per query
//    the sum of P_ij (q_i - t_j) / C_ij; partial sums over target blocks are
//    added in order by cost_reduce_kernel / grad_merge_kernel.
// Square roots and exponentials use the hardware approximations (v_sqrt_f32,
// v_rsq_f32, v_exp_f32).  Exponents are bounded: after each half-update the
// updated side's sums equal its mass, so every a b exp(z) is at most 1.
#include <algorithm>
#include <cmath>

#include "cd_internal.h"

namespace cdk {
namespace {

constexpr int kEQ = 4;                      // queries per lane
constexpr int kEThreads = 256;              // 4 waves
constexpr int kEGroup = kEQ * kEThreads;    // queries per workgroup
constexpr int kEBatch = 16;                 // targets per online-LSE batch
constexpr int kEMinTB = 64;                 // targets per block, at least
constexpr int64_t kETargetTiles = 512;
constexpr int kEChunk = 1024;               // target potentials merged into LDS at a time
constexpr int kThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;

struct LseArgs {
    const float *Q, *T;     // [B, nq, 3], [B, nt, 3]
    const float *pt;        // [B, nt] potentials of the targets (finished)
    const float2 *tpart;    // or their partials [B, tnTB, nt] from the previous half-update
    float *pq;              // [B, nq] updated potentials of the queries
    float2 *part;           // [B, nTB, nq] (max, sum) partials, base 2
    int64_t nq, nt;
    float k;                // log2(e) / eps
    float out_scale;        // -eps ln 2
    float out_bias;         // eps log(nt)  (= -eps log b)
    float t_scale, t_bias;  // out_scale, out_bias of the half-update that left tpart
    int nQG, nTB, TB, tnTB;
};

// A finished potential from its nTB (max, sum) partials, stride apart:
// -eps log(b sum exp(...)) = scale (M + log2 S) + bias.
__device__ __forceinline__ float merged_potential(const float2 *p, int nTB, int64_t stride,
                                                  float scale, float bias)
{
    float M = -__builtin_inff();
    for (int t = 0; t < nTB; ++t) M = __builtin_fmaxf(M, p[static_cast<int64_t>(t) * stride].x);
    float S = 0.0f;
    for (int t = 0; t < nTB; ++t) {
        const float2 v = p[static_cast<int64_t>(t) * stride];
        S += v.y * __builtin_amdgcn_exp2f(v.x - M);
    }
    return __builtin_fmaf(scale, M + __log2f(S), bias);
}

__device__ __forceinline__ float dist2(float qx, float qy, float qz, float tx, float ty, float tz)
{
    const float dx = qx - tx, dy = qy - ty, dz = qz - tz;
    return __builtin_fmaf(dz, dz, __builtin_fmaf(dy, dy, dx * dx));
}

// One batch of kEBatch targets for kEQ queries: running max m and sum s.
__device__ __forceinline__ void lse_batch(const float (&qx)[kEQ], const float (&qy)[kEQ],
                                          const float (&qz)[kEQ], float (&m)[kEQ],
                                          float (&s)[kEQ], const float (&tx)[kEBatch],
                                          const float (&ty)[kEBatch], const float (&tz)[kEBatch],
                                          const float (&tk)[kEBatch], float kk)
{
#pragma unroll
    for (int k = 0; k < kEQ; ++k) {
        float z[kEBatch];
        float bm = -__builtin_inff();
#pragma unroll
        for (int u = 0; u < kEBatch; ++u) {
            const float c = __builtin_amdgcn_sqrtf(dist2(qx[k], qy[k], qz[k], tx[u], ty[u], tz[u]));
            z[u] = __builtin_fmaf(-c, kk, tk[u]);
            bm = __builtin_fmaxf(bm, z[u]);
        }
        const float mn = __builtin_fmaxf(m[k], bm);
        float acc = s[k] * __builtin_amdgcn_exp2f(m[k] - mn);
#pragma unroll
        for (int u = 0; u < kEBatch; ++u) acc += __builtin_amdgcn_exp2f(z[u] - mn);
        s[k] = acc;
        m[k] = mn;
    }
}

// kFromParts: the targets' potentials come as the previous half-update's
// partials, merged here a chunk at a time into LDS.
template <bool kFromParts>
__global__ __launch_bounds__(kEThreads) void lse_kernel(LseArgs a)
{
    __shared__ float lpt[kFromParts ? kEChunk : 1];
    const int64_t per_item = static_cast<int64_t>(a.nQG) * a.nTB;
    const int64_t b = blockIdx.x / per_item;
    const int rest = static_cast<int>(blockIdx.x % per_item);
    const int qg = rest / a.nTB, tb = rest % a.nTB;
    const int64_t q0 = static_cast<int64_t>(qg) * kEGroup;
    float qx[kEQ], qy[kEQ], qz[kEQ], m[kEQ], s[kEQ];
#pragma unroll
    for (int k = 0; k < kEQ; ++k) {
        const int64_t q = std::min<int64_t>(q0 + k * kEThreads + threadIdx.x, a.nq - 1);
        const float *p = a.Q + (b * a.nq + q) * 3;
        qx[k] = p[0];
        qy[k] = p[1];
        qz[k] = p[2];
        m[k] = -__builtin_inff();
        s[k] = 0.0f;
    }
    // Targets [j0, j1) of item b; 32-bit offsets within the item.
    const int j0 = tb * a.TB;
    const int j1 = static_cast<int>(std::min<int64_t>(static_cast<int64_t>(j0) + a.TB, a.nt));
    const float *Tb = a.T + b * a.nt * 3;
    const float *pb = kFromParts ? nullptr : a.pt + b * a.nt;
    const float kk = a.k;
    // Chunks of kEChunk targets (a multiple of kEBatch, so only the last
    // chunk has a tail); without partials the whole block is one chunk.
    for (int c0 = j0; c0 < j1; c0 += (kFromParts ? kEChunk : j1 - j0)) {
        const int c1 = kFromParts ? std::min(c0 + kEChunk, j1) : j1;
        if (kFromParts) {
            __syncthreads();  // the previous chunk is consumed
            const float2 *tp = a.tpart + b * a.tnTB * a.nt;
            for (int j = c0 + static_cast<int>(threadIdx.x); j < c1; j += kEThreads)
                lpt[j - c0] = merged_potential(tp + j, a.tnTB, a.nt, a.t_scale, a.t_bias);
            __syncthreads();
        }
        auto pot = [&](int j) { return kFromParts ? lpt[j - c0] : pb[j]; };
        const int cfull = c0 + (c1 - c0) / kEBatch * kEBatch;
        for (int jb = c0; jb < cfull; jb += kEBatch) {
            // A full batch: contiguous wave-uniform loads, no per-target guards.
            float tx[kEBatch], ty[kEBatch], tz[kEBatch], tk[kEBatch];
#pragma unroll
            for (int u = 0; u < kEBatch; ++u) {
                tx[u] = Tb[3 * (jb + u) + 0];
                ty[u] = Tb[3 * (jb + u) + 1];
                tz[u] = Tb[3 * (jb + u) + 2];
                tk[u] = pot(jb + u) * kk;
            }
            lse_batch(qx, qy, qz, m, s, tx, ty, tz, tk, kk);
        }
        if (cfull < c1) {
            // The tail: clamped loads, weight 0 past the end.
            float tx[kEBatch], ty[kEBatch], tz[kEBatch], tk[kEBatch];
#pragma unroll
            for (int u = 0; u < kEBatch; ++u) {
                const int j = std::min(cfull + u, c1 - 1);
                tx[u] = Tb[3 * j + 0];
                ty[u] = Tb[3 * j + 1];
                tz[u] = Tb[3 * j + 2];
                tk[u] = cfull + u < c1 ? pot(j) * kk : -__builtin_inff();
            }
            lse_batch(qx, qy, qz, m, s, tx, ty, tz, tk, kk);
        }
    }
#pragma unroll
    for (int k = 0; k < kEQ; ++k) {
        const int64_t q = q0 + k * kEThreads + threadIdx.x;
        if (q >= a.nq) continue;
        if (a.nTB == 1)
            a.pq[b * a.nq + q] = __builtin_fmaf(a.out_scale, m[k] + __log2f(s[k]), a.out_bias);
        else
            a.part[(b * a.nTB + tb) * a.nq + q] = make_float2(m[k], s[k]);
    }
}

__global__ __launch_bounds__(kThreads) void lse_merge_kernel(LseArgs a, int64_t B)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= B * a.nq) return;
    const int64_t b = k / a.nq, q = k - b * a.nq;
    a.pq[k] = merged_potential(a.part + b * a.nTB * a.nq + q, a.nTB, a.nq, a.out_scale,
                               a.out_bias);
}

__global__ __launch_bounds__(kThreads) void fill_kernel(float *p, int64_t n, float v)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k < n) p[k] = v;
}

struct PlanArgs {
    const float *Q, *T;     // [B, nq, 3], [B, nt, 3]
    const float *pq, *pt;   // potentials of queries and targets
    const float *go;        // [B] (gradient mode)
    double *cost_part;      // [B, nQG, nTB] (cost mode)
    float *grad_part;       // [B, nTB, nq, 3] (gradient mode, nTB > 1)
    float *grad;            // [B, nq, 3] (gradient mode, nTB == 1)
    int64_t nq, nt;
    float k;                // log2(e) / eps
    float mass;             // a b = 1 / (nq nt)
    int nQG, nTB, TB;
};

template <bool kGrad>
__device__ __forceinline__ void plan_batch(const float (&qx)[kEQ], const float (&qy)[kEQ],
                                           const float (&qz)[kEQ], const float (&qk)[kEQ],
                                           float (&acc)[kEQ], float (&gx)[kEQ], float (&gy)[kEQ],
                                           float (&gz)[kEQ], const float (&tx)[kEBatch],
                                           const float (&ty)[kEBatch], const float (&tz)[kEBatch],
                                           const float (&tk)[kEBatch], float kk)
{
#pragma unroll
    for (int u = 0; u < kEBatch; ++u) {
#pragma unroll
        for (int k = 0; k < kEQ; ++k) {
            const float d2 = dist2(qx[k], qy[k], qz[k], tx[u], ty[u], tz[u]);
            const float r = d2 > 0.0f ? __builtin_amdgcn_rsqf(d2) : 0.0f;
            const float c = d2 * r;
            const float w = __builtin_amdgcn_exp2f(__builtin_fmaf(-c, kk, qk[k] + tk[u]));
            if (kGrad) {
                const float wr = w * r;
                gx[k] = __builtin_fmaf(wr, qx[k] - tx[u], gx[k]);
                gy[k] = __builtin_fmaf(wr, qy[k] - ty[u], gy[k]);
                gz[k] = __builtin_fmaf(wr, qz[k] - tz[u], gz[k]);
            } else {
                acc[k] = __builtin_fmaf(w, c, acc[k]);
            }
        }
    }
}

template <bool kGrad>
__global__ __launch_bounds__(kEThreads) void plan_kernel(PlanArgs a)
{
    __shared__ double red[kEThreads / kWave];
    const int64_t per_item = static_cast<int64_t>(a.nQG) * a.nTB;
    const int64_t b = blockIdx.x / per_item;
    const int rest = static_cast<int>(blockIdx.x % per_item);
    const int qg = rest / a.nTB, tb = rest % a.nTB;
    const int64_t q0 = static_cast<int64_t>(qg) * kEGroup;
    float qx[kEQ], qy[kEQ], qz[kEQ], qk[kEQ], acc[kEQ], gx[kEQ], gy[kEQ], gz[kEQ];
#pragma unroll
    for (int k = 0; k < kEQ; ++k) {
        const int64_t q = q0 + k * kEThreads + threadIdx.x;
        const bool in = q < a.nq;
        const int64_t qc = in ? q : 0;
        const float *p = a.Q + (b * a.nq + qc) * 3;
        qx[k] = p[0];
        qy[k] = p[1];
        qz[k] = p[2];
        qk[k] = in ? a.pq[b * a.nq + qc] * a.k : -__builtin_inff();   // outside: weight 0
        acc[k] = gx[k] = gy[k] = gz[k] = 0.0f;
    }
    const int j0 = tb * a.TB;
    const int j1 = static_cast<int>(std::min<int64_t>(static_cast<int64_t>(j0) + a.TB, a.nt));
    const int jfull = j0 + (j1 - j0) / kEBatch * kEBatch;
    const float *Tb = a.T + b * a.nt * 3;
    const float *pb = a.pt + b * a.nt;
    const float kk = a.k;
    for (int jb = j0; jb < jfull; jb += kEBatch) {
        float tx[kEBatch], ty[kEBatch], tz[kEBatch], tk[kEBatch];
#pragma unroll
        for (int u = 0; u < kEBatch; ++u) {
            tx[u] = Tb[3 * (jb + u) + 0];
            ty[u] = Tb[3 * (jb + u) + 1];
            tz[u] = Tb[3 * (jb + u) + 2];
            tk[u] = pb[jb + u] * kk;
        }
        plan_batch<kGrad>(qx, qy, qz, qk, acc, gx, gy, gz, tx, ty, tz, tk, kk);
    }
    if (jfull < j1) {
        float tx[kEBatch], ty[kEBatch], tz[kEBatch], tk[kEBatch];
#pragma unroll
        for (int u = 0; u < kEBatch; ++u) {
            const int j = std::min(jfull + u, j1 - 1);
            tx[u] = Tb[3 * j + 0];
            ty[u] = Tb[3 * j + 1];
            tz[u] = Tb[3 * j + 2];
            tk[u] = jfull + u < j1 ? pb[j] * kk : -__builtin_inff();
        }
        plan_batch<kGrad>(qx, qy, qz, qk, acc, gx, gy, gz, tx, ty, tz, tk, kk);
    }
    if (kGrad) {
        const float sc = a.mass * a.go[b];
#pragma unroll
        for (int k = 0; k < kEQ; ++k) {
            const int64_t q = q0 + k * kEThreads + threadIdx.x;
            if (q >= a.nq) continue;
            float *dst = a.nTB == 1 ? a.grad + (b * a.nq + q) * 3
                                    : a.grad_part + ((b * a.nTB + tb) * a.nq + q) * 3;
            const float sv = a.nTB == 1 ? sc : 1.0f;
            dst[0] = sv * gx[k];
            dst[1] = sv * gy[k];
            dst[2] = sv * gz[k];
        }
        return;
    }
    // Cost mode: the tile's sum, reduced in a fixed order.
    double t = 0.0;
#pragma unroll
    for (int k = 0; k < kEQ; ++k) t += static_cast<double>(acc[k]);
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) t += __shfl_xor(t, off, kWave);
    if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
        double sum = 0.0;
        for (int w = 0; w < kEThreads / kWave; ++w) sum += red[w];
        a.cost_part[(b * a.nQG + qg) * a.nTB + tb] = sum;
    }
}

__global__ __launch_bounds__(kThreads) void cost_reduce_kernel(const double *part, int64_t tiles,
                                                               float mass, float *cost)
{
    __shared__ double red[kThreads / kWave];
    const int64_t b = blockIdx.x;
    double t = 0.0;
    for (int64_t i = threadIdx.x; i < tiles; i += kThreads) t += part[b * tiles + i];
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) t += __shfl_xor(t, off, kWave);
    if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
        double s = 0.0;
        for (int w = 0; w < kThreads / kWave; ++w) s += red[w];
        cost[b] = static_cast<float>(s * static_cast<double>(mass));
    }
}

__global__ __launch_bounds__(kThreads) void grad_merge_kernel(PlanArgs a, int64_t B)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= B * a.nq * 3) return;
    const int64_t b = k / (a.nq * 3), e = k - b * a.nq * 3;
    const float *p = a.grad_part + b * a.nTB * a.nq * 3 + e;
    float s = 0.0f;
    for (int t = 0; t < a.nTB; ++t) s += p[static_cast<int64_t>(t) * a.nq * 3];
    a.grad[k] = s * (a.mass * a.go[b]);
}

int64_t ceil_div(int64_t x, int64_t y) { return (x + y - 1) / y; }

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Query groups and target blocks for queries of size nq against nt targets.
struct Tiles {
    int nQG, nTB, TB;
};

Tiles tiles_for(int64_t B, int64_t nq, int64_t nt)
{
    Tiles t;
    t.nQG = static_cast<int>(ceil_div(nq, kEGroup));
    int64_t want = std::max<int64_t>(1, ceil_div(kETargetTiles, B * t.nQG));
    want = std::min(want, std::max<int64_t>(1, ceil_div(nt, kEMinTB)));
    const int64_t tb = ceil_div(ceil_div(nt, want), kEBatch) * kEBatch;
    t.TB = static_cast<int>(tb);
    t.nTB = static_cast<int>(ceil_div(nt, tb));
    return t;
}

struct EmdLayout {
    Tiles xy, yx;               // queries X against Y; queries Y against X
    size_t fpart_bytes;         // f's partials; g's follow (a half-update reads one, writes the other)
    size_t part_bytes, cost_bytes, grad_bytes;
};

EmdLayout layout(int64_t B, int64_t N, int64_t M)
{
    EmdLayout L;
    L.xy = tiles_for(B, N, M);
    L.yx = tiles_for(B, M, N);
    const size_t p1 = L.xy.nTB > 1 ? static_cast<size_t>(B * L.xy.nTB * N) * 8 : 0;
    const size_t p2 = L.yx.nTB > 1 ? static_cast<size_t>(B * L.yx.nTB * M) * 8 : 0;
    L.fpart_bytes = align256(p1);
    L.part_bytes = L.fpart_bytes + align256(p2);
    L.cost_bytes = align256(static_cast<size_t>(B * L.xy.nQG * L.xy.nTB) * 8);
    const size_t g1 = L.xy.nTB > 1 ? static_cast<size_t>(B * L.xy.nTB * N) * 12 : 0;
    const size_t g2 = L.yx.nTB > 1 ? static_cast<size_t>(B * L.yx.nTB * M) * 12 : 0;
    L.grad_bytes = align256(std::max(g1, g2));
    return L;
}

// The potentials of one cloud between half-updates: finished values, or the
// (max, sum) partials a half-update left with the transform that finishes them.
struct Potentials {
    const float *fin = nullptr;     // [B, n], or
    const float2 *part = nullptr;   // [B, nTB, n]
    int nTB = 1;
    float scale = 0.0f, bias = 0.0f;
};

// One half-update of the queries' potentials (written to pq when the targets
// form one block, else left as partials in `part`) against the targets'.
Potentials lse_pass(int64_t B, const float *Q, int64_t nq, const float *T, int64_t nt,
                    const Potentials &tp, float *pq, float eps, const Tiles &t, float2 *part,
                    hipStream_t stream)
{
    LseArgs a{};
    a.Q = Q;
    a.T = T;
    a.pt = tp.fin;
    a.tpart = tp.part;
    a.tnTB = tp.nTB;
    a.t_scale = tp.scale;
    a.t_bias = tp.bias;
    a.pq = pq;
    a.part = part;
    a.nq = nq;
    a.nt = nt;
    a.k = kLog2e / eps;
    a.out_scale = -eps * 0.6931471805599453f;
    a.out_bias = static_cast<float>(static_cast<double>(eps) * std::log(static_cast<double>(nt)));
    a.nQG = t.nQG;
    a.nTB = t.nTB;
    a.TB = t.TB;
    const uint32_t grid = static_cast<uint32_t>(B * t.nQG * t.nTB);
    if (tp.fin)
        lse_kernel<false><<<grid, kEThreads, 0, stream>>>(a);
    else
        lse_kernel<true><<<grid, kEThreads, 0, stream>>>(a);
    Potentials out;
    if (t.nTB == 1) {
        out.fin = pq;
    } else {
        out.part = part;
        out.nTB = t.nTB;
        out.scale = a.out_scale;
        out.bias = a.out_bias;
    }
    return out;
}

// Finished potentials [B, n] into `out` (a no-op if they are there already).
void finish(int64_t B, int64_t n, const Potentials &p, float *out, hipStream_t stream)
{
    if (p.fin) return;
    LseArgs a{};
    a.part = const_cast<float2 *>(p.part);
    a.pq = out;
    a.nq = n;
    a.nTB = p.nTB;
    a.out_scale = p.scale;
    a.out_bias = p.bias;
    lse_merge_kernel<<<static_cast<uint32_t>(ceil_div(B * n, kThreads)), kThreads, 0, stream>>>(
        a, B);
}

hipError_t plan_pass(int64_t B, const float *Q, int64_t nq, const float *T, int64_t nt,
                     const float *pq, const float *pt, float eps, const Tiles &t, bool gradient,
                     const float *go, double *cost_part, float *grad_part, float *grad,
                     hipStream_t stream)
{
    PlanArgs a{};
    a.Q = Q;
    a.T = T;
    a.pq = pq;
    a.pt = pt;
    a.go = go;
    a.cost_part = cost_part;
    a.grad_part = grad_part;
    a.grad = grad;
    a.nq = nq;
    a.nt = nt;
    a.k = kLog2e / eps;
    a.mass = static_cast<float>(1.0 / (static_cast<double>(nq) * static_cast<double>(nt)));
    a.nQG = t.nQG;
    a.nTB = t.nTB;
    a.TB = t.TB;
    const uint32_t grid = static_cast<uint32_t>(B * t.nQG * t.nTB);
    if (gradient)
        plan_kernel<true><<<grid, kEThreads, 0, stream>>>(a);
    else
        plan_kernel<false><<<grid, kEThreads, 0, stream>>>(a);
    if (gradient && t.nTB > 1)
        grad_merge_kernel<<<static_cast<uint32_t>(ceil_div(B * nq * 3, kThreads)), kThreads, 0,
                            stream>>>(a, B);
    return hipGetLastError();
}

}  // namespace

size_t emd_workspace_bytes(int64_t B, int64_t N, int64_t M)
{
    const EmdLayout L = layout(B, N, M);
    return L.part_bytes + L.cost_bytes + L.grad_bytes;
}

float emd_eps(double eps_start, double eps_end, int n_iters, int t)
{
    if (n_iters <= 1) return static_cast<float>(eps_end);
    const double e = eps_start * std::pow(eps_end / eps_start,
                                          static_cast<double>(t) / static_cast<double>(n_iters - 1));
    return static_cast<float>(e);
}

hipError_t launch_emd_forward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                              double eps_start, double eps_end, int n_iters, bool warm, float *f,
                              float *g, float *cost, void *ws, hipStream_t stream)
{
    const EmdLayout L = layout(B, N, M);
    char *base = static_cast<char *>(ws);
    float2 *fpart = reinterpret_cast<float2 *>(base);
    float2 *gpart = reinterpret_cast<float2 *>(base + L.fpart_bytes);
    double *cost_part = reinterpret_cast<double *>(base + L.part_bytes);
    if (!warm)
        fill_kernel<<<static_cast<uint32_t>(ceil_div(B * M, kThreads)), kThreads, 0, stream>>>(
            g, B * M, 0.0f);
    Potentials pf, pg;
    pf.fin = f;
    pg.fin = g;
    for (int t = 0; t < n_iters; ++t) {
        const float eps = emd_eps(eps_start, eps_end, n_iters, t);
        pf = lse_pass(B, X, N, Y, M, pg, f, eps, L.xy, fpart, stream);
        pg = lse_pass(B, Y, M, X, N, pf, g, eps, L.yx, gpart, stream);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    finish(B, N, pf, f, stream);
    finish(B, M, pg, g, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const float eps = emd_eps(eps_start, eps_end, n_iters, n_iters - 1);
    e = plan_pass(B, X, N, Y, M, f, g, eps, L.xy, false, nullptr, cost_part, nullptr,
                             nullptr, stream);
    if (e != hipSuccess) return e;
    cost_reduce_kernel<<<static_cast<uint32_t>(B), kThreads, 0, stream>>>(
        cost_part, static_cast<int64_t>(L.xy.nQG) * L.xy.nTB,
        static_cast<float>(1.0 / (static_cast<double>(N) * static_cast<double>(M))), cost);
    return hipGetLastError();
}

hipError_t launch_emd_backward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                               const float *f, const float *g, double eps, const float *go,
                               float *gX, float *gY, void *ws, hipStream_t stream)
{
    const EmdLayout L = layout(B, N, M);
    char *base = static_cast<char *>(ws);
    float *grad_part = reinterpret_cast<float *>(base + L.part_bytes + L.cost_bytes);
    const float e32 = static_cast<float>(eps);
    hipError_t e = plan_pass(B, X, N, Y, M, f, g, e32, L.xy, true, go, nullptr, grad_part, gX,
                             stream);
    if (e != hipSuccess) return e;
    return plan_pass(B, Y, M, X, N, g, f, e32, L.yx, true, go, nullptr, grad_part, gY, stream);
}

}  // namespace cdk

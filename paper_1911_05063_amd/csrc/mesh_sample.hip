// Differentiable surface sampling of triangle meshes (Kaolin Sec. 2.1: mesh
// to point-cloud conversion with the reparameterization trick), the step that
// feeds the Chamfer loss in mesh reconstruction.
//
//  * face_cdf_kernel: one workgroup per item computes every face's area,
//    |(b - a) x (c - a)| / 2 in float32, rounds it to a fixed-point integer on
//    a grid of 2^-k (k from the item's largest area, so the total stays below
//    2^62) and writes the exact inclusive prefix sums as int64.  Integer sums
//    do not depend on the scan order, and a zero-area face has exactly the
//    cumulative value of the face before it, so it can never be chosen.
//  * choose_faces_kernel: thread per sample; the first face whose cumulative
//    area exceeds u * total (binary search); a zero-area mesh yields -1.
//  * sample_points_kernel: thread per sample;
//    p = (1 - sqrt(r1)) a + sqrt(r1)(1 - r2) b + sqrt(r1) r2 c.
//  * sample_backward_kernel: a workgroup owns a slice of the vertices of one
//    item and a chunk of that item's samples, and adds w_i * gP to its
//    vertices in LDS as 64-bit fixed-point integers (ds_add_u64; the scale 2^k
//    comes from the chunk's largest |gP| so no sum can overflow).  Integer
//    addition is exact, so the order in which lanes add does not matter and
//    the result is bitwise reproducible; it is also several times faster than
//    float LDS atomics.  With one chunk per item the slice goes straight to
//    gV; otherwise each chunk's slice goes to the workspace in double and
//    sum_chunks_kernel adds the chunks in order.
// A face with a vertex index outside [0, nv), or a sample whose face index is
// outside [0, nf), is given area 0 / a NaN point and contributes no gradient.
#include <algorithm>

#include "cd_internal.h"

namespace cdk {
namespace {

constexpr int kCdfThreads = 1024;
constexpr int kThreads = 256;
constexpr int kBwdThreads = 256;
constexpr int kBwdUnroll = 2;
constexpr int kVertSlice = 2048;
// The backward splits each item's samples into chunks until about this many
// workgroups run; each chunk's per-vertex sums go to the workspace and are
// added in chunk order afterwards.
constexpr int64_t kBwdTargetGroups = 512;

__device__ __forceinline__ bool face_ok(const int32_t *t, int64_t nv)
{
    return t[0] >= 0 && t[0] < nv && t[1] >= 0 && t[1] < nv && t[2] >= 0 && t[2] < nv;
}

__device__ __forceinline__ float face_area(const float *Vb, const int32_t *t)
{
    const float *a = Vb + 3 * static_cast<int64_t>(t[0]);
    const float *b = Vb + 3 * static_cast<int64_t>(t[1]);
    const float *c = Vb + 3 * static_cast<int64_t>(t[2]);
    const float e1x = b[0] - a[0], e1y = b[1] - a[1], e1z = b[2] - a[2];
    const float e2x = c[0] - a[0], e2y = c[1] - a[1], e2z = c[2] - a[2];
    const float cx = e1y * e2z - e1z * e2y;
    const float cy = e1z * e2x - e1x * e2z;
    const float cz = e1x * e2y - e1y * e2x;
    return 0.5f * sqrtf(cx * cx + cy * cy + cz * cz);
}

// Shift k such that n values of magnitude at most m, each scaled by 2^k and
// rounded to an integer, sum to less than 2^62 in magnitude.  m = 0 gives 0.
__device__ __forceinline__ int fixed_shift(float m, int64_t n)
{
    if (!(m > 0.0f)) return 0;
    int e;
    frexpf(m, &e);                                 // m < 2^e
    const int lg = 64 - __clzll(static_cast<unsigned long long>(n));   // n < 2^lg
    return 61 - e - lg;
}

__device__ __forceinline__ long long to_fixed(float x, int k)
{
    return static_cast<long long>(rintf(ldexpf(x, k)));
}

template <int kThreadsPerGroup>
__device__ __forceinline__ float group_max(float m, float *red)
{
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, kWave));
    if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = m;
    __syncthreads();
    m = red[0];
#pragma unroll
    for (int w = 1; w < kThreadsPerGroup / kWave; ++w) m = fmaxf(m, red[w]);
    return m;
}

__global__ __launch_bounds__(kCdfThreads) void face_cdf_kernel(int64_t nv, int64_t nf,
                                                               const float *V, const int32_t *F,
                                                               long long *cdf)
{
    __shared__ float red[kCdfThreads / kWave];
    __shared__ long long wsum[kCdfThreads / kWave];
    const int64_t b = blockIdx.x;
    const float *Vb = V + b * nv * 3;
    const int32_t *Fb = F + b * nf * 3;
    long long *out = cdf + b * nf;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    // Thread t owns the contiguous run of faces [f0, f1).
    const int64_t run = (nf + kCdfThreads - 1) / kCdfThreads;
    const int64_t f0 = std::min<int64_t>(nf, threadIdx.x * run), f1 = std::min<int64_t>(nf, f0 + run);
    // Pass 1: areas (stashed as float bits in the output) and their maximum.
    float m = 0.0f;
    for (int64_t f = f0; f < f1; ++f) {
        const int32_t *t = Fb + 3 * f;
        const float a = face_ok(t, nv) ? face_area(Vb, t) : 0.0f;
        out[f] = static_cast<long long>(__float_as_uint(a));
        m = fmaxf(m, a);
    }
    const int k = fixed_shift(group_max<kCdfThreads>(m, red), nf);
    // Pass 2: the run's integer total, then an exact exclusive scan of the totals.
    long long own = 0;
    for (int64_t f = f0; f < f1; ++f) own += to_fixed(__uint_as_float(static_cast<uint32_t>(out[f])), k);
    long long incl = own;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const long long o = __shfl_up(incl, off, kWave);
        if (lane >= off) incl += o;
    }
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    long long acc = incl - own;
    for (int w = 0; w < wave; ++w) acc += wsum[w];
    // Pass 3: the inclusive prefix sums of the run.
    for (int64_t f = f0; f < f1; ++f) {
        acc += to_fixed(__uint_as_float(static_cast<uint32_t>(out[f])), k);
        out[f] = acc;
    }
}

__global__ __launch_bounds__(kThreads) void choose_faces_kernel(int64_t B, int64_t nf, int64_t S,
                                                                const long long *cdf,
                                                                const float *u, int32_t *fidx)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= B * S) return;
    const int64_t b = k / S;
    const long long *c = cdf + b * nf;
    const long long total = c[nf - 1];
    const double target = fmax(0.0, static_cast<double>(u[k]) * static_cast<double>(total));
    // First f with c[f] > target: c[f] > c[f - 1], so face f has positive
    // area.  If none (u * total rounds up to total, or u is NaN), the first f
    // with c[f] == total, i.e. the last face with positive area.
    int64_t lo = 0, hi = nf;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (static_cast<double>(c[mid]) > target) hi = mid; else lo = mid + 1;
    }
    if (lo == nf) {
        lo = 0;
        hi = nf;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (c[mid] >= total) hi = mid; else lo = mid + 1;
        }
    }
    fidx[k] = (total > 0 && lo < nf) ? static_cast<int32_t>(lo) : -1;
}

__device__ __forceinline__ void bary(float r1, float r2, float &wa, float &wb, float &wc)
{
    const float s1 = sqrtf(r1);
    wa = 1.0f - s1;
    wb = s1 * (1.0f - r2);
    wc = s1 * r2;
}

__global__ __launch_bounds__(kThreads) void sample_points_kernel(int64_t B, int64_t nv,
                                                                 int64_t nf, int64_t S,
                                                                 const float *V, const int32_t *F,
                                                                 const int32_t *fidx,
                                                                 const float *r1, const float *r2,
                                                                 float *P)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= B * S) return;
    const int64_t b = k / S;
    const int32_t f = fidx[k];
    const int32_t *t = F + (b * nf + (f >= 0 && f < nf ? f : 0)) * 3;
    if (f < 0 || f >= nf || !face_ok(t, nv)) {
        P[3 * k + 0] = P[3 * k + 1] = P[3 * k + 2] = __builtin_nanf("");
        return;
    }
    float wa, wb, wc;
    bary(r1[k], r2[k], wa, wb, wc);
    const float *Vb = V + b * nv * 3;
    const float *a = Vb + 3 * static_cast<int64_t>(t[0]);
    const float *bb = Vb + 3 * static_cast<int64_t>(t[1]);
    const float *c = Vb + 3 * static_cast<int64_t>(t[2]);
#pragma unroll
    for (int d = 0; d < 3; ++d)
        P[3 * k + d] = __builtin_fmaf(wc, c[d], __builtin_fmaf(wb, bb[d], wa * a[d]));
}

// Workgroup (b, slice, chunk) owns vertices [v0, v1) of item b and scans the
// samples [s0, s1) of that item; it writes its slice of the per-chunk partial
// sums (or gV itself when there is one chunk).  Dynamic LDS: 24 (v1 - v0) bytes.
__global__ __launch_bounds__(kBwdThreads) void sample_backward_kernel(
    int64_t nv, int64_t nf, int64_t S, int nslice, int nchunk, int64_t chunk, const int32_t *F,
    const int32_t *fidx, const float *r1, const float *r2, const float *gP, double *part,
    float *gV)
{
    extern __shared__ unsigned long long acc[];
    __shared__ float red[kBwdThreads / kWave];
    const int64_t c = blockIdx.x % nchunk;
    const int64_t rest = blockIdx.x / nchunk;
    const int64_t b = rest / nslice;
    const int64_t v0 = static_cast<int64_t>(rest % nslice) * kVertSlice;
    const int64_t v1 = std::min<int64_t>(v0 + kVertSlice, nv);
    const int n3 = static_cast<int>(3 * (v1 - v0));
    const int64_t s0 = c * chunk, s1 = std::min<int64_t>(s0 + chunk, S);
    for (int t = threadIdx.x; t < n3; t += kBwdThreads) acc[t] = 0ull;
    // Scale: every per-vertex sum is bounded by (s1 - s0) * max |gP| because
    // a sample's weights are non-negative and add up to one.
    float m = 0.0f;
    for (int64_t s = s0 + threadIdx.x; s < s1; s += kBwdThreads) {
        const float *g = gP + 3 * (b * S + s);
        m = fmaxf(m, fmaxf(fabsf(g[0]), fmaxf(fabsf(g[1]), fabsf(g[2]))));
    }
    const int ks = fixed_shift(group_max<kBwdThreads>(m, red), s1 - s0);
    const int32_t *Fb = F + b * nf * 3;
    for (int64_t sb = s0; sb < s1; sb += kBwdUnroll * kBwdThreads) {
        // Issue every load of the unrolled group before the first use.
        int32_t f[kBwdUnroll];
        float w1[kBwdUnroll], w2[kBwdUnroll], g[kBwdUnroll][3];
#pragma unroll
        for (int u = 0; u < kBwdUnroll; ++u) {
            const int64_t s = sb + u * kBwdThreads + threadIdx.x;
            f[u] = -1;
            if (s < s1) {
                const int64_t k = b * S + s;
                f[u] = fidx[k];
                w1[u] = r1[k];
                w2[u] = r2[k];
                g[u][0] = gP[3 * k + 0];
                g[u][1] = gP[3 * k + 1];
                g[u][2] = gP[3 * k + 2];
            }
        }
        int32_t t[kBwdUnroll][3];
#pragma unroll
        for (int u = 0; u < kBwdUnroll; ++u) {
            const bool ok = f[u] >= 0 && f[u] < nf;
            const int32_t *tri = Fb + 3 * static_cast<int64_t>(ok ? f[u] : 0);
            t[u][0] = ok ? tri[0] : -1;
            t[u][1] = ok ? tri[1] : -1;
            t[u][2] = ok ? tri[2] : -1;
        }
#pragma unroll
        for (int u = 0; u < kBwdUnroll; ++u) {
            if (t[u][0] < 0 || t[u][0] >= nv || t[u][1] < 0 || t[u][1] >= nv || t[u][2] < 0 ||
                t[u][2] >= nv)
                continue;
            float w[3];
            bary(w1[u], w2[u], w[0], w[1], w[2]);
#pragma unroll
            for (int i = 0; i < 3; ++i) {
                const int64_t v = t[u][i];
                if (v >= v0 && v < v1) {
                    unsigned long long *a = acc + 3 * (v - v0);
#pragma unroll
                    for (int d = 0; d < 3; ++d)
                        atomicAdd(a + d, static_cast<unsigned long long>(to_fixed(w[i] * g[u][d], ks)));
                }
            }
        }
    }
    __syncthreads();
    if (nchunk == 1) {
        float *dst = gV + (b * nv + v0) * 3;
        for (int t = threadIdx.x; t < n3; t += kBwdThreads)
            dst[t] = static_cast<float>(ldexp(static_cast<double>(static_cast<long long>(acc[t])), -ks));
    } else {
        double *dst = part + ((b * nchunk + c) * nv + v0) * 3;
        for (int t = threadIdx.x; t < n3; t += kBwdThreads)
            dst[t] = ldexp(static_cast<double>(static_cast<long long>(acc[t])), -ks);
    }
}

// gV[b, e] = sum over chunks c, in order, of part[b, c, e] (e = 3 v + d).
__global__ __launch_bounds__(kThreads) void sum_chunks_kernel(int64_t B, int64_t n3, int nchunk,
                                                              const double *part, float *gV)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= B * n3) return;
    const int64_t b = k / n3, e = k - b * n3;
    const double *p = part + b * nchunk * n3 + e;
    double s = 0.0;
    int c = 0;
    // Loads of a group go out together; the adds stay in chunk order.
    for (; c + 8 <= nchunk; c += 8) {
        double v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = p[(c + i) * n3];
#pragma unroll
        for (int i = 0; i < 8; ++i) s += v[i];
    }
    for (; c < nchunk; ++c) s += p[c * n3];
    gV[k] = static_cast<float>(s);
}

struct BwdSplit {
    int nslice, nchunk;
    int64_t chunk;
};

BwdSplit split_backward(int64_t B, int64_t nv, int64_t S)
{
    BwdSplit p;
    p.nslice = static_cast<int>((nv + kVertSlice - 1) / kVertSlice);
    const int64_t groups = B * p.nslice;
    const int64_t step = static_cast<int64_t>(kBwdUnroll) * kBwdThreads;
    int64_t want = groups >= kBwdTargetGroups ? 1 : (kBwdTargetGroups + groups - 1) / groups;
    want = std::max<int64_t>(1, std::min(want, (S + step - 1) / step));
    int64_t chunk = (S + want - 1) / want;
    chunk = std::max<int64_t>(step, (chunk + step - 1) / step * step);
    p.chunk = chunk;
    p.nchunk = static_cast<int>(S > 0 ? (S + chunk - 1) / chunk : 1);
    return p;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

size_t mesh_workspace_bytes(int64_t B, int64_t nv, int64_t nf, int64_t S)
{
    const size_t cdf = static_cast<size_t>(B * nf) * 8;
    const BwdSplit p = split_backward(B, nv, S);
    const size_t part = p.nchunk > 1 ? static_cast<size_t>(B * p.nchunk * nv) * 24 : 0;
    return std::max(cdf, part);
}

hipError_t launch_mesh_choose_faces(int64_t B, int64_t nv, int64_t nf, const float *V,
                                    const int32_t *F, int64_t S, const float *u, int32_t *fidx,
                                    void *ws, hipStream_t stream)
{
    long long *cdf = static_cast<long long *>(ws);
    face_cdf_kernel<<<static_cast<uint32_t>(B), kCdfThreads, 0, stream>>>(nv, nf, V, F, cdf);
    if (S > 0)
        choose_faces_kernel<<<static_cast<uint32_t>(ceil_div(B * S, kThreads)), kThreads, 0,
                              stream>>>(B, nf, S, cdf, u, fidx);
    return hipGetLastError();
}

hipError_t launch_mesh_sample_points(int64_t B, int64_t nv, int64_t nf, const float *V,
                                     const int32_t *F, int64_t S, const int32_t *fidx,
                                     const float *r1, const float *r2, float *P,
                                     hipStream_t stream)
{
    sample_points_kernel<<<static_cast<uint32_t>(ceil_div(B * S, kThreads)), kThreads, 0,
                           stream>>>(B, nv, nf, S, V, F, fidx, r1, r2, P);
    return hipGetLastError();
}

hipError_t launch_mesh_sample_backward(int64_t B, int64_t nv, int64_t nf, const int32_t *F,
                                       int64_t S, const int32_t *fidx, const float *r1,
                                       const float *r2, const float *gP, float *gV, void *ws,
                                       hipStream_t stream)
{
    const BwdSplit p = split_backward(B, nv, S);
    double *part = static_cast<double *>(ws);
    const size_t lds = 24 * static_cast<size_t>(std::min<int64_t>(nv, kVertSlice));
    sample_backward_kernel<<<static_cast<uint32_t>(B * p.nslice * p.nchunk), kBwdThreads, lds,
                             stream>>>(nv, nf, S, p.nslice, p.nchunk, p.chunk, F, fidx, r1, r2,
                                       gP, part, gV);
    if (p.nchunk > 1)
        sum_chunks_kernel<<<static_cast<uint32_t>(ceil_div(B * 3 * nv, kThreads)), kThreads, 0,
                            stream>>>(B, 3 * nv, p.nchunk, part, gV);
    return hipGetLastError();
}

}  // namespace cdk

// Backward of barycentric interpolation onto triangle-mesh vertices, shared by
// mesh surface sampling (Kaolin Sec. 2.1) and the point-to-surface loss
// (Sec. 2.5): every sample s lies on face fidx[s] with barycentric weights
// w_s, so a vector gP[s] attached to it contributes w_{s,i} gP[s] to vertex i
// of that face:
//     gV[v] = sum over samples s whose face holds v of w_{s,v} gP[s].
//
// A workgroup owns a slice of the vertices of one item and a chunk of that
// item's samples, and adds w * gP to its vertices in LDS as 64-bit fixed-point
// integers (ds_add_u64; the scale 2^k comes from the chunk's largest |gP| so
// no sum can overflow).  Integer addition is exact, so the order in which
// lanes add does not matter and the result is bitwise reproducible; it is also
// several times faster than float LDS atomics here.  With one chunk per item
// the slice goes straight to gV; otherwise each chunk's slice goes to the
// workspace in double and sum_chunks_kernel adds the chunks in order.
// Samples whose face index is outside [0, nf), or whose face has a vertex
// outside [0, nv), contribute nothing.
#include <algorithm>

#include "cd_internal.h"
#include "mesh_common.h"

namespace cdk {
namespace {

constexpr int kThreads = 256;
constexpr int kBwdThreads = 256;
constexpr int kBwdUnroll = 2;
constexpr int kVertSlice = 2048;
// Each item's samples are split into chunks so that about one workgroup per
// CU runs (kBwdFillGroups), more where that keeps the chunks within what one
// thread holds in registers (kBwdHeld * kBwdThreads samples), up to about two
// per CU (kBwdMaxGroups); each chunk's per-vertex sums go to the workspace and
// are added in chunk order afterwards.
constexpr int64_t kBwdFillGroups = 256;
constexpr int64_t kBwdMaxGroups = 512;
constexpr int64_t kBwdHeld = 8;

// Workgroup (b, slice, chunk)'s vertices [v0, v1) of item b (n3 = 3 (v1 - v0)
// accumulators) and samples [s0, s1); workgroups run chunk-fastest.
struct Tile {
    int64_t c, b, v0, v1, s0, s1;
    int n3;
};

__device__ __forceinline__ Tile tile_of(int64_t nv, int64_t S, int nslice, int nchunk,
                                        int64_t chunk)
{
    Tile w;
    w.c = blockIdx.x % nchunk;
    const int64_t rest = blockIdx.x / nchunk;
    w.b = rest / nslice;
    w.v0 = static_cast<int64_t>(rest % nslice) * kVertSlice;
    w.v1 = std::min<int64_t>(w.v0 + kVertSlice, nv);
    w.n3 = static_cast<int>(3 * (w.v1 - w.v0));
    w.s0 = w.c * chunk;
    w.s1 = std::min<int64_t>(w.s0 + chunk, S);
    return w;
}

// Adds sample s's terms w_i * gP[s] to the vertices of face t that lie in the
// slice [v0, v1) (LDS, fixed point at scale 2^ks); a face with a vertex index
// outside [0, nv) (t = -1 for a face index out of range) adds nothing.
// kExplicit: the weights are sign * (w1, w2, w3); else bary(w1, w2).
template <bool kExplicit>
__device__ __forceinline__ void add_sample(unsigned long long *acc, const int32_t t[3], int64_t nv,
                                           int64_t v0, int64_t v1, float w1, float w2, float w3,
                                           const float g[3], float sign, int ks)
{
    if (!face_ok_nb(t, nv)) return;
    float w[3];
    if (kExplicit) {
        w[0] = sign * w1;
        w[1] = sign * w2;
        w[2] = sign * w3;
    } else {
        bary(w1, w2, w[0], w[1], w[2]);
    }
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        const int64_t v = t[i];
        if (v >= v0 && v < v1) {
            unsigned long long *a = acc + 3 * (v - v0);
#pragma unroll
            for (int d = 0; d < 3; ++d)
                atomicAdd(a + d, static_cast<unsigned long long>(to_fixed(w[i] * g[d], ks)));
        }
    }
}

// The slice's sums, scaled back: to gV when the item has one chunk, else to
// the chunk's row of the workspace (double).
__device__ __forceinline__ void write_slice(const unsigned long long *acc, int n3, int ks,
                                            int64_t b, int64_t c, int nchunk, int64_t nv,
                                            int64_t v0, double *part, float *gV)
{
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

// Workgroup (b, slice, chunk) owns vertices [v0, v1) of item b and scans the
// samples [s0, s1) of that item; it writes its slice of the per-chunk partial
// sums (or gV itself when there is one chunk).  Dynamic LDS: 24 (v1 - v0) bytes.
// kExplicit: weights from w [B, S, 3]; else from the uniforms (r1, r2).
template <bool kExplicit>
__global__ __launch_bounds__(kBwdThreads) void bary_scatter_kernel(
    int64_t nv, int64_t nf, int64_t S, int nslice, int nchunk, int64_t chunk, const int32_t *F,
    const int32_t *fidx, const float *r1, const float *r2, const float *wts, const float *gP,
    float sign, double *part, float *gV)
{
    extern __shared__ unsigned long long acc[];
    __shared__ float red[kBwdThreads / kWave];
    const Tile w = tile_of(nv, S, nslice, nchunk, chunk);
    const int64_t c = w.c, b = w.b, v0 = w.v0, v1 = w.v1, s0 = w.s0, s1 = w.s1;
    const int n3 = w.n3;
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
        float w1[kBwdUnroll], w2[kBwdUnroll], w3[kBwdUnroll], g[kBwdUnroll][3];
#pragma unroll
        for (int u = 0; u < kBwdUnroll; ++u) {
            const int64_t s = sb + u * kBwdThreads + threadIdx.x;
            f[u] = -1;
            w3[u] = 0.0f;
            if (s < s1) {
                const int64_t k = b * S + s;
                f[u] = fidx[k];
                if (kExplicit) {
                    w1[u] = wts[3 * k + 0];
                    w2[u] = wts[3 * k + 1];
                    w3[u] = wts[3 * k + 2];
                } else {
                    w1[u] = r1[k];
                    w2[u] = r2[k];
                }
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
        for (int u = 0; u < kBwdUnroll; ++u)
            add_sample<kExplicit>(acc, t[u], nv, v0, v1, w1[u], w2[u], w3[u], g[u], sign, ks);
    }
    __syncthreads();
    write_slice(acc, n3, ks, b, c, nchunk, nv, v0, part, gV);
}

// The same sums for chunks of at most kPer * kBwdThreads samples, none empty:
// a thread loads all of its samples (fidx, weights, gP) in one round and keeps
// them, so the chunk's largest |gP| needs no read of its own, and the face
// loads go out before the workgroup's maximum is formed: two dependent memory
// rounds instead of one per unrolled group plus one.  Same chunks, same shift,
// exact sums: bitwise equal to bary_scatter_kernel.
template <bool kExplicit, int kPer>
__global__ __launch_bounds__(kBwdThreads) void bary_scatter_held_kernel(
    int64_t nv, int64_t nf, int64_t S, int nslice, int nchunk, int64_t chunk, const int32_t *F,
    const int32_t *fidx, const float *r1, const float *r2, const float *wts, const float *gP,
    float sign, double *part, float *gV)
{
    extern __shared__ unsigned long long acc[];
    __shared__ float red[kBwdThreads / kWave];
    const Tile w = tile_of(nv, S, nslice, nchunk, chunk);
    const int64_t c = w.c, b = w.b, v0 = w.v0, v1 = w.v1, s0 = w.s0, s1 = w.s1;
    const int n3 = w.n3;
    // Samples past the chunk's end load its last sample (s1 > s0) and are
    // masked out of the maximum and the sums.
    int32_t f[kPer];
    float w1[kPer], w2[kPer], w3[kPer], g[kPer][3];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const int64_t k = b * S + std::min<int64_t>(s0 + u * kBwdThreads + threadIdx.x, s1 - 1);
        f[u] = fidx[k];
        if (kExplicit) {
            w1[u] = wts[3 * k + 0];
            w2[u] = wts[3 * k + 1];
            w3[u] = wts[3 * k + 2];
        } else {
            w1[u] = r1[k];
            w2[u] = r2[k];
            w3[u] = 0.0f;
        }
        g[u][0] = gP[3 * k + 0];
        g[u][1] = gP[3 * k + 1];
        g[u][2] = gP[3 * k + 2];
    }
    for (int t = threadIdx.x; t < n3; t += kBwdThreads) acc[t] = 0ull;
    float m = 0.0f;
    int32_t t[kPer][3];
    const int32_t *Fb = F + b * nf * 3;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const bool in = s0 + u * kBwdThreads + threadIdx.x < s1;
        const float mu = fmaxf(fabsf(g[u][0]), fmaxf(fabsf(g[u][1]), fabsf(g[u][2])));
        m = in ? fmaxf(m, mu) : m;
        const bool ok = in & (f[u] >= 0) & (f[u] < nf);
        const int32_t *tri = Fb + 3 * static_cast<int64_t>(ok ? f[u] : 0);
#pragma unroll
        for (int i = 0; i < 3; ++i) t[u][i] = ok ? tri[i] : -1;
    }
    const int ks = fixed_shift(group_max<kBwdThreads>(m, red), s1 - s0);
#pragma unroll
    for (int u = 0; u < kPer; ++u)
        add_sample<kExplicit>(acc, t[u], nv, v0, v1, w1[u], w2[u], w3[u], g[u], sign, ks);
    __syncthreads();
    write_slice(acc, n3, ks, b, c, nchunk, nv, v0, part, gV);
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

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct ScatterSplit {
    int nslice, nchunk;
    int64_t chunk;
};

ScatterSplit split_scatter(int64_t B, int64_t nv, int64_t S)
{
    ScatterSplit p;
    p.nslice = static_cast<int>((nv + kVertSlice - 1) / kVertSlice);
    const int64_t groups = B * p.nslice;
    const int64_t step = static_cast<int64_t>(kBwdUnroll) * kBwdThreads;
    const int64_t fill = ceil_div(kBwdFillGroups, groups), most = ceil_div(kBwdMaxGroups, groups);
    int64_t want = std::max(fill, std::min(most, ceil_div(S, kBwdHeld * kBwdThreads)));
    want = std::max<int64_t>(1, std::min(want, ceil_div(S, step)));
    int64_t chunk = (S + want - 1) / want;
    chunk = std::max<int64_t>(step, (chunk + step - 1) / step * step);
    p.chunk = chunk;
    p.nchunk = static_cast<int>(S > 0 ? (S + chunk - 1) / chunk : 1);
    return p;
}

}  // namespace

size_t bary_scatter_workspace_bytes(int64_t B, int64_t nv, int64_t S)
{
    const ScatterSplit p = split_scatter(B, nv, S);
    return p.nchunk > 1 ? static_cast<size_t>(B * p.nchunk * nv) * 24 : 0;
}

hipError_t launch_bary_scatter(int64_t B, int64_t nv, int64_t nf, const int32_t *F, int64_t S,
                               const int32_t *fidx, const float *r1, const float *r2,
                               const float *w, const float *gP, bool negate, float *gV, void *ws,
                               hipStream_t stream)
{
    const ScatterSplit p = split_scatter(B, nv, S);
    double *part = static_cast<double *>(ws);
    const size_t lds = 24 * static_cast<size_t>(std::min<int64_t>(nv, kVertSlice));
    const uint32_t grid = static_cast<uint32_t>(B * p.nslice * p.nchunk);
    const float sign = negate ? -1.0f : 1.0f;
    // Samples per thread of the held kernel (chunks are multiples of
    // kBwdUnroll * kBwdThreads = 512 samples): 2, 4 or 8, else the loop.
    const int64_t need = S > 0 ? ceil_div(p.chunk, kBwdThreads) : kBwdHeld + 1;
    const int per = need <= 2 ? 2 : need <= 4 ? 4 : need <= kBwdHeld ? 8 : 0;
    using Kernel = void (*)(int64_t, int64_t, int64_t, int, int, int64_t, const int32_t *,
                            const int32_t *, const float *, const float *, const float *,
                            const float *, float, double *, float *);
    Kernel k;
    if (w)
        k = per == 2 ? bary_scatter_held_kernel<true, 2>
          : per == 4 ? bary_scatter_held_kernel<true, 4>
          : per == 8 ? bary_scatter_held_kernel<true, 8> : bary_scatter_kernel<true>;
    else
        k = per == 2 ? bary_scatter_held_kernel<false, 2>
          : per == 4 ? bary_scatter_held_kernel<false, 4>
          : per == 8 ? bary_scatter_held_kernel<false, 8> : bary_scatter_kernel<false>;
    k<<<grid, kBwdThreads, lds, stream>>>(nv, nf, S, p.nslice, p.nchunk, p.chunk, F, fidx, r1, r2,
                                          w, gP, sign, part, gV);
    if (p.nchunk > 1)
        sum_chunks_kernel<<<static_cast<uint32_t>(ceil_div(B * 3 * nv, kThreads)), kThreads, 0,
                            stream>>>(B, 3 * nv, p.nchunk, part, gV);
    return hipGetLastError();
}

}  // namespace cdk

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
//  * the backward, gV[v] = sum of w_{s,v} gP[s], is the reproducible
//    fixed-point barycentric scatter of bary_scatter.hip.
// A face with a vertex index outside [0, nv), or a sample whose face index is
// outside [0, nf), is given area 0 / a NaN point and contributes no gradient.
#include <algorithm>

#include "cd_internal.h"
#include "mesh_common.h"

namespace cdk {
namespace {

constexpr int kCdfThreads = 1024;
constexpr int kRunRegs = 4;       // faces per thread kept in registers by face_cdf_kernel
constexpr int kThreads = 256;
constexpr int kCdfLds = 4096;      // cumulative areas staged in LDS by choose_faces_kernel

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

// kRegs > 0: each thread's run has at most kRegs faces, whose areas stay in
// registers (their loads all in flight together); kRegs = 0: they are stashed
// as float bits in the output between the passes.
template <int kRegs>
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
    // Pass 1: areas and their maximum.
    float m = 0.0f;
    float ar[kRegs > 0 ? kRegs : 1];
    if (kRegs > 0) {
        // Faces past the run's end repeat face nf - 1, and a face with a vertex
        // outside the mesh reads vertex 0 (loads only; area 0), so that no
        // branch splits the loads.
        int32_t tv[kRegs > 0 ? kRegs : 1][3];
#pragma unroll
        for (int r = 0; r < kRegs; ++r) {
            const int32_t *t = Fb + 3 * std::min<int64_t>(f0 + r, nf - 1);
#pragma unroll
            for (int c = 0; c < 3; ++c) tv[r][c] = t[c];
        }
#pragma unroll
        for (int r = 0; r < kRegs; ++r) {
            const bool ok = (f0 + r < f1) & face_ok_nb(tv[r], nv);
            int32_t tc[3];
#pragma unroll
            for (int c = 0; c < 3; ++c) tc[c] = ok ? tv[r][c] : 0;
            const float a = face_area(Vb, tc);
            ar[r] = ok ? a : 0.0f;
            m = fmaxf(m, ar[r]);
        }
    } else {
        for (int64_t f = f0; f < f1; ++f) {
            const int32_t *t = Fb + 3 * f;
            const float a = face_ok(t, nv) ? face_area(Vb, t) : 0.0f;
            out[f] = static_cast<long long>(__float_as_uint(a));
            m = fmaxf(m, a);
        }
    }
    const int k = fixed_shift(group_max<kCdfThreads>(m, red), nf);
    // Pass 2: the run's integer total, then an exact exclusive scan of the totals.
    long long own = 0;
    if (kRegs > 0) {
#pragma unroll
        for (int r = 0; r < kRegs; ++r) own += to_fixed(ar[r], k);
    } else {
        for (int64_t f = f0; f < f1; ++f) own += to_fixed(__uint_as_float(static_cast<uint32_t>(out[f])), k);
    }
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
    if (kRegs > 0) {
#pragma unroll
        for (int r = 0; r < kRegs; ++r) {
            acc += to_fixed(ar[r], k);
            if (f0 + r < f1) out[f0 + r] = acc;
        }
    } else {
        for (int64_t f = f0; f < f1; ++f) {
            acc += to_fixed(__uint_as_float(static_cast<uint32_t>(out[f])), k);
            out[f] = acc;
        }
    }
}

// The first f with c[f] > target: c[f] > c[f - 1], so face f has positive
// area.  If none (u * total rounds up to total, or u is NaN), the first f with
// c[f] == total, i.e. the last face with positive area.  c: the item's
// cumulative areas (in LDS or global memory).
__device__ __forceinline__ int64_t choose_face(const long long *c, int64_t nf, float u)
{
    const long long total = c[nf - 1];
    const double target = fmax(0.0, static_cast<double>(u) * static_cast<double>(total));
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
    return (total > 0 && lo < nf) ? lo : -1;
}

// Thread per sample.  A workgroup whose samples all belong to one item with
// at most kCdfLds faces first copies that item's cumulative areas to LDS and
// searches there (the search's dependent steps are LDS reads, not memory
// rounds); otherwise it searches global memory.
__global__ __launch_bounds__(kThreads) void choose_faces_kernel(int64_t B, int64_t nf, int64_t S,
                                                                const long long *cdf,
                                                                const float *u, int32_t *fidx)
{
    __shared__ long long sc[kCdfLds];
    const int64_t k0 = static_cast<int64_t>(blockIdx.x) * kThreads;
    const int64_t k = k0 + threadIdx.x;
    const int64_t kl = std::min(k0 + kThreads, B * S) - 1;   // the workgroup's last sample
    const int64_t b = std::min(k, kl) / S;
    const float uk = u[std::min(k, kl)];
    if (nf <= kCdfLds && k0 / S == kl / S) {
        const long long *c = cdf + b * nf;
        for (int64_t i = threadIdx.x; i < nf; i += kThreads) sc[i] = c[i];
        __syncthreads();
        if (k < B * S) fidx[k] = static_cast<int32_t>(choose_face(sc, nf, uk));
    } else if (k < B * S) {
        fidx[k] = static_cast<int32_t>(choose_face(cdf + b * nf, nf, uk));
    }
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
    // The sample's face and uniforms, then the face's vertex indices, then
    // the vertices: three memory rounds with no branch between them (an
    // invalid face or vertex index reads face / vertex 0 and yields NaN).
    const int32_t f = fidx[k];
    const float u1 = r1[k], u2 = r2[k];
    const bool fok = (f >= 0) & (f < nf);
    const int32_t *t = F + (b * nf + (fok ? f : 0)) * 3;
    int32_t tv[3];
#pragma unroll
    for (int c = 0; c < 3; ++c) tv[c] = t[c];
    const bool ok = fok & face_ok_nb(tv, nv);
    float wa, wb, wc;
    bary(u1, u2, wa, wb, wc);
    const float *Vb = V + b * nv * 3;
    float a[3], bb[3], c[3];   // all loaded before the first store (P may alias V)
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        a[d] = Vb[3 * static_cast<int64_t>(ok ? tv[0] : 0) + d];
        bb[d] = Vb[3 * static_cast<int64_t>(ok ? tv[1] : 0) + d];
        c[d] = Vb[3 * static_cast<int64_t>(ok ? tv[2] : 0) + d];
    }
#pragma unroll
    for (int d = 0; d < 3; ++d)
        P[3 * k + d] = ok ? __builtin_fmaf(wc, c[d], __builtin_fmaf(wb, bb[d], wa * a[d]))
                          : __builtin_nanf("");
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

hipError_t launch_mesh_choose_faces(int64_t B, int64_t nv, int64_t nf, const float *V,
                                    const int32_t *F, int64_t S, const float *u, int32_t *fidx,
                                    void *ws, hipStream_t stream)
{
    long long *cdf = static_cast<long long *>(ws);
    if (nf <= kCdfThreads)
        face_cdf_kernel<1><<<static_cast<uint32_t>(B), kCdfThreads, 0, stream>>>(nv, nf, V, F, cdf);
    else if (nf <= static_cast<int64_t>(kRunRegs) * kCdfThreads)
        face_cdf_kernel<kRunRegs><<<static_cast<uint32_t>(B), kCdfThreads, 0, stream>>>(nv, nf, V, F, cdf);
    else
        face_cdf_kernel<0><<<static_cast<uint32_t>(B), kCdfThreads, 0, stream>>>(nv, nf, V, F, cdf);
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

size_t mesh_workspace_bytes(int64_t B, int64_t nv, int64_t nf, int64_t S)
{
    return std::max(static_cast<size_t>(B * nf) * 8, bary_scatter_workspace_bytes(B, nv, S));
}

hipError_t launch_mesh_sample_backward(int64_t B, int64_t nv, int64_t nf, const int32_t *F,
                                       int64_t S, const int32_t *fidx, const float *r1,
                                       const float *r2, const float *gP, float *gV, void *ws,
                                       hipStream_t stream)
{
    return launch_bary_scatter(B, nv, nf, F, S, fidx, r1, r2, nullptr, gP, false, gV, ws, stream);
}

}  // namespace cdk

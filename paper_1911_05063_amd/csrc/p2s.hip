// Point-to-surface distance between point clouds and triangle meshes (Kaolin
// Sec. 2.5: the point-to-surface loss for meshes).  For every point p of item
// b: dist = min over the faces f of item b of the squared distance from p to
// the closed triangle f, fidx = the face attaining it (lowest index among
// exactly equal float32 distances).  Backward: with q the closest point and
// w its barycentric coordinates, d dist / d p = 2 (p - q) and
// d dist / d v_i = -2 w_i (p - q).
//
//  * face_record_kernel: one thread per face writes a 32-float record
//    (computed in double, stored in float32): the corner a, the dual basis
//    g0, g1 of the edges e0 = b - a, e1 = c - a in the face's plane
//    (s = (p - a).g0, t = (p - a).g1 are the projection's coordinates along
//    e0, e1), the unit normal, an inside threshold (0, or +inf for a face
//    without interior), and each edge with its direction over its squared
//    length.  A face with a vertex index out of range gets a record at which
//    every distance overflows to +inf, so it is never chosen.
//  * p2s_search_kernel: a workgroup holds 2048 points (8 per lane) in VGPRs
//    and walks a block of at most 320 faces, whose records it first copies
//    to LDS; each face's record is then read by every lane from the same LDS
//    address (a broadcast) into VGPRs, so the arithmetic has VGPR operands
//    only, which this chip can issue two at a time (SGPR operands measured
//    13% slower).  Per
//    (point, face): v = p - a; if min(s, t, 1 - s - t) >= threshold the
//    projection is inside and dist = (v.n)^2, else dist = the minimum over the
//    three edges of |v - clamp(v.e/|e|^2, 0, 1) e|^2 (the closest point of a
//    convex polygon to an outside point lies on its boundary).  Branch-free:
//    every lane evaluates the same face.
//  * Face blocks of one point group are merged through 64-bit keys
//    (float bits << 32 | face), exact and lowest-index on equal distances,
//    by p2s_merge_kernel (skipped with one block).
//  * p2s_point_grad_kernel: per point, the closest point on its face in
//    double, gP = 2 g (p - q) and the weights w; the vertex gradient is the
//    reproducible barycentric scatter of bary_scatter.hip with -gP.
#include <algorithm>
#include <cmath>

#include "cd_internal.h"
#include "mesh_common.h"

namespace cdk {
namespace {

constexpr int kRec = 32;          // floats per face record (31 used)
// Corner of a face with a vertex index out of range: every distance to such a
// record overflows to +inf (no inf - inf anywhere), so it is never chosen.
constexpr float kFar = 3.0e38f;
constexpr int kPQ = 8;            // points per lane
constexpr int kPWaves = 4;
constexpr int kPThreads = kPWaves * kWave;
constexpr int kPGroup = kPQ * kPThreads;    // points per workgroup
constexpr int kMinFB = 64;        // faces per block, at least
constexpr int kMaxFB = 320;       // faces per block, at most (records staged in 40 KB of LDS)
constexpr int64_t kTargetTiles = 2048;
constexpr int64_t kSlots = 256 * 4;   // workgroups resident at once: 256 CUs x 4
constexpr int64_t kSmallRounds = 8;   // small face blocks only for launches of 1 to 8 rounds
constexpr int kThreads = 256;

struct P2SArgs {
    const float *P;      // [B, S, 3]
    const float *rec;    // [B, nf, kRec]
    uint64_t *part;      // [B, nFB, S] keys (nFB > 1)
    float *dist;         // [B, S]
    int32_t *fidx;       // [B, S]
    int64_t S, nf;
    int nQG, nFB, FB;
    int nBig, FS;        // small blocks of FS faces follow nBig blocks of FB
    int64_t B;
};

__global__ __launch_bounds__(kThreads) void face_record_kernel(int64_t B, int64_t nv, int64_t nf,
                                                               const float *V, const int32_t *F,
                                                               float *rec)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= B * nf) return;
    const int64_t b = k / nf;
    // The three vertex indices in one load round, then the three vertices
    // (vertex 0 in place of an out-of-range index) in the next.
    const int32_t t[3] = {F[3 * k], F[3 * k + 1], F[3 * k + 2]};
    const bool ok = face_ok_nb(t, nv);
    const float *Vb = V + b * nv * 3;
    double A[3], Bv[3], C[3], e0[3], e1[3], e2[3], n[3];
    for (int i = 0; i < 3; ++i) {
        A[i] = Vb[3 * static_cast<int64_t>(ok ? t[0] : 0) + i];
        Bv[i] = Vb[3 * static_cast<int64_t>(ok ? t[1] : 0) + i];
        C[i] = Vb[3 * static_cast<int64_t>(ok ? t[2] : 0) + i];
    }
    float *r = rec + k * kRec;
    if (!ok) {
        for (int i = 0; i < kRec; ++i) r[i] = 0.0f;
        r[0] = r[1] = r[2] = kFar;
        r[12] = __builtin_inff();
        return;
    }
    for (int i = 0; i < 3; ++i) {
        e0[i] = Bv[i] - A[i];
        e1[i] = C[i] - A[i];
        e2[i] = C[i] - Bv[i];
    }
    n[0] = e0[1] * e1[2] - e0[2] * e1[1];
    n[1] = e0[2] * e1[0] - e0[0] * e1[2];
    n[2] = e0[0] * e1[1] - e0[1] * e1[0];
    const double nn = n[0] * n[0] + n[1] * n[1] + n[2] * n[2];
    // Dual basis: g0 = (e1 x n) / |n|^2, g1 = (n x e0) / |n|^2, so that
    // e0.g0 = e1.g1 = 1 and e1.g0 = e0.g1 = n.g0 = n.g1 = 0.
    double g0[3] = {0, 0, 0}, g1[3] = {0, 0, 0}, nh[3] = {0, 0, 0};
    const bool flat = !(nn > 0.0) || !std::isfinite(nn);
    // One reciprocal per denominator (double divisions are long instruction
    // sequences); the record is rounded to float32 afterwards.
    if (!flat) {
        const double rn = 1.0 / nn;
        g0[0] = (e1[1] * n[2] - e1[2] * n[1]) * rn;
        g0[1] = (e1[2] * n[0] - e1[0] * n[2]) * rn;
        g0[2] = (e1[0] * n[1] - e1[1] * n[0]) * rn;
        g1[0] = (n[1] * e0[2] - n[2] * e0[1]) * rn;
        g1[1] = (n[2] * e0[0] - n[0] * e0[2]) * rn;
        g1[2] = (n[0] * e0[1] - n[1] * e0[0]) * rn;
        const double inv = 1.0 / sqrt(nn);
        for (int i = 0; i < 3; ++i) nh[i] = n[i] * inv;
    }
    const double l0 = e0[0] * e0[0] + e0[1] * e0[1] + e0[2] * e0[2];
    const double l1 = e1[0] * e1[0] + e1[1] * e1[1] + e1[2] * e1[2];
    const double l2 = e2[0] * e2[0] + e2[1] * e2[1] + e2[2] * e2[2];
    const double r0 = l0 > 0.0 ? 1.0 / l0 : 0.0;
    const double r1 = l1 > 0.0 ? 1.0 / l1 : 0.0;
    const double r2 = l2 > 0.0 ? 1.0 / l2 : 0.0;
    for (int i = 0; i < 3; ++i) {
        r[0 + i] = static_cast<float>(A[i]);
        r[3 + i] = static_cast<float>(g0[i]);
        r[6 + i] = static_cast<float>(g1[i]);
        r[9 + i] = static_cast<float>(nh[i]);
        r[13 + i] = static_cast<float>(e0[i]);
        r[16 + i] = static_cast<float>(e0[i] * r0);
        r[19 + i] = static_cast<float>(e1[i]);
        r[22 + i] = static_cast<float>(e1[i] * r1);
        r[25 + i] = static_cast<float>(e2[i]);
        r[28 + i] = static_cast<float>(e2[i] * r2);
    }
    r[12] = flat ? __builtin_inff() : 0.0f;
    r[31] = 0.0f;
}

__device__ __forceinline__ float fmaf_(float a, float b, float c) { return __builtin_fmaf(a, b, c); }

__device__ __forceinline__ float dot3(float x, float y, float z, float a, float b, float c)
{
    return fmaf_(z, c, fmaf_(y, b, x * a));
}

// Squared distance from v (relative to the segment's origin) to the segment
// {sigma e : sigma in [0, 1]}, en = e / |e|^2.
__device__ __forceinline__ float seg2(float vx, float vy, float vz, float ex, float ey, float ez,
                                      float nx, float ny, float nz)
{
    const float sg = __builtin_amdgcn_fmed3f(dot3(vx, vy, vz, nx, ny, nz), 0.0f, 1.0f);
    const float wx = fmaf_(-sg, ex, vx), wy = fmaf_(-sg, ey, vy), wz = fmaf_(-sg, ez, vz);
    return dot3(wx, wy, wz, wx, wy, wz);
}

__global__ __launch_bounds__(kPThreads) void p2s_search_kernel(P2SArgs a)
{
    // Every (item, group) tile of the nBig large face blocks first, then those
    // of the small blocks, which the dispatcher hands out last.
    const uint32_t nbig = static_cast<uint32_t>(a.nBig);
    const uint32_t big_tiles = static_cast<uint32_t>(a.B * a.nQG) * nbig;
    uint32_t fbu, rest;
    if (blockIdx.x < big_tiles) {
        fbu = blockIdx.x % nbig;
        rest = blockIdx.x / nbig;
    } else {
        const uint32_t k = blockIdx.x - big_tiles, nsmall = static_cast<uint32_t>(a.nFB) - nbig;
        fbu = nbig + k % nsmall;
        rest = k / nsmall;
    }
    const int fb = static_cast<int>(fbu);
    const int qg = static_cast<int>(rest % static_cast<uint32_t>(a.nQG));
    const int64_t b = rest / static_cast<uint32_t>(a.nQG);
    const int64_t q0 = static_cast<int64_t>(qg) * kPGroup;

    float px[kPQ], py[kPQ], pz[kPQ], best[kPQ];
    int32_t bidx[kPQ];
#pragma unroll
    for (int k = 0; k < kPQ; ++k) {
        const int64_t q = q0 + k * kPThreads + threadIdx.x;
        const bool in = q < a.S;
        const float *p = a.P + (b * a.S + (in ? q : 0)) * 3;
        px[k] = p[0];
        py[k] = p[1];
        pz[k] = p[2];
        best[k] = __builtin_inff();
        bidx[k] = -1;
    }
    const bool large = fb < a.nBig;
    const int32_t f0 = large ? fb * a.FB : a.nBig * a.FB + (fb - a.nBig) * a.FS;
    const int32_t f1 = static_cast<int32_t>(std::min<int64_t>(f0 + (large ? a.FB : a.FS), a.nf));
    const float *rb = a.rec + b * a.nf * kRec;
    __shared__ float4 lrec[kMaxFB * (kRec / 4)];
    {
        const float4 *src4 = reinterpret_cast<const float4 *>(rb + static_cast<int64_t>(f0) * kRec);
        const int n4 = (f1 - f0) * (kRec / 4);
        for (int t = threadIdx.x; t < n4; t += kPThreads) lrec[t] = src4[t];
    }
    __syncthreads();
    for (int32_t f = f0; f < f1; ++f) {
        const float4 *r4 = lrec + (f - f0) * (kRec / 4);
        const float4 A0 = r4[0], A1 = r4[1], A2 = r4[2], A3 = r4[3], A4 = r4[4], A5 = r4[5], A6 = r4[6], A7 = r4[7];
        const float ax = A0.x, ay = A0.y, az = A0.z;
        const float g0x = A0.w, g0y = A1.x, g0z = A1.y;
        const float g1x = A1.z, g1y = A1.w, g1z = A2.x;
        const float nx = A2.y, ny = A2.z, nz = A2.w, cin = A3.x;
        const float e0x = A3.y, e0y = A3.z, e0z = A3.w, n0x = A4.x, n0y = A4.y, n0z = A4.z;
        const float e1x = A4.w, e1y = A5.x, e1z = A5.y, n1x = A5.z, n1y = A5.w, n1z = A6.x;
        const float e2x = A6.y, e2y = A6.z, e2z = A6.w, n2x = A7.x, n2y = A7.y, n2z = A7.z;
#pragma unroll
        for (int k = 0; k < kPQ; ++k) {
            const float vx = px[k] - ax, vy = py[k] - ay, vz = pz[k] - az;
            const float s = dot3(vx, vy, vz, g0x, g0y, g0z);
            const float t = dot3(vx, vy, vz, g1x, g1y, g1z);
            const float h = dot3(vx, vy, vz, nx, ny, nz);
            const float u = (1.0f - s) - t;
            const bool inside = __builtin_fminf(__builtin_fminf(s, t), u) >= cin;
            const float dab = seg2(vx, vy, vz, e0x, e0y, e0z, n0x, n0y, n0z);
            const float dca = seg2(vx, vy, vz, e1x, e1y, e1z, n1x, n1y, n1z);
            const float dbc = seg2(vx - e0x, vy - e0y, vz - e0z, e2x, e2y, e2z, n2x, n2y, n2z);
            const float edge = __builtin_fminf(__builtin_fminf(dab, dca), dbc);
            const float d = inside ? h * h : edge;
            if (d < best[k]) {
                best[k] = d;
                bidx[k] = f;
            }
        }
    }
#pragma unroll
    for (int k = 0; k < kPQ; ++k) {
        const int64_t q = q0 + k * kPThreads + threadIdx.x;
        if (q >= a.S) continue;
        if (a.nFB == 1) {
            a.dist[b * a.S + q] = best[k];
            a.fidx[b * a.S + q] = bidx[k];
        } else {
            const uint64_t key = (static_cast<uint64_t>(__float_as_uint(best[k])) << 32) |
                                 static_cast<uint32_t>(bidx[k]);
            a.part[(b * a.nFB + fb) * a.S + q] = key;
        }
    }
}

__global__ __launch_bounds__(kThreads) void p2s_merge_kernel(int64_t B, int64_t S, int nFB,
                                                             const uint64_t *part, float *dist,
                                                             int32_t *fidx)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= B * S) return;
    const int64_t b = k / S, q = k - b * S;
    const uint64_t *p = part + b * nFB * S + q;
    // Eight blocks' keys in flight at a time (indices past the last block
    // repeat it: the minimum does not change).
    uint64_t m = ~0ull;
    for (int i0 = 0; i0 < nFB; i0 += 8) {
        uint64_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = p[static_cast<int64_t>(min(i0 + u, nFB - 1)) * S];
#pragma unroll
        for (int u = 0; u < 8; ++u) m = std::min<uint64_t>(m, v[u]);
    }
    dist[k] = __uint_as_float(static_cast<uint32_t>(m >> 32));
    fidx[k] = static_cast<int32_t>(static_cast<uint32_t>(m));
}

// Closest point of the closed triangle (A, B, C) to p, in double: its
// barycentric coordinates w and the residual p - q.
__device__ void closest_point(const double p[3], const double A[3], const double Bv[3],
                              const double C[3], double w[3], double res[3])
{
    double e0[3], e1[3], v[3], n[3];
    for (int i = 0; i < 3; ++i) {
        e0[i] = Bv[i] - A[i];
        e1[i] = C[i] - A[i];
        v[i] = p[i] - A[i];
    }
    n[0] = e0[1] * e1[2] - e0[2] * e1[1];
    n[1] = e0[2] * e1[0] - e0[0] * e1[2];
    n[2] = e0[0] * e1[1] - e0[1] * e1[0];
    const double nn = n[0] * n[0] + n[1] * n[1] + n[2] * n[2];
    if (nn > 0.0) {
        // s = v.(e1 x n)/|n|^2 and t = v.(n x e0)/|n|^2, written as triple products.
        const double s = (v[0] * (e1[1] * n[2] - e1[2] * n[1]) + v[1] * (e1[2] * n[0] - e1[0] * n[2]) +
                          v[2] * (e1[0] * n[1] - e1[1] * n[0])) / nn;
        const double t = (v[0] * (n[1] * e0[2] - n[2] * e0[1]) + v[1] * (n[2] * e0[0] - n[0] * e0[2]) +
                          v[2] * (n[0] * e0[1] - n[1] * e0[0])) / nn;
        if (s >= 0.0 && t >= 0.0 && s + t <= 1.0) {
            w[0] = 1.0 - s - t;
            w[1] = s;
            w[2] = t;
            for (int i = 0; i < 3; ++i) res[i] = v[i] - s * e0[i] - t * e1[i];
            return;
        }
    }
    // On the boundary: the nearest of the three segments.
    const double *org[3] = {A, Bv, C}, *end[3] = {Bv, C, A};
    double bestd = INFINITY;
    for (int i = 0; i < 3; ++i) w[i] = res[i] = 0.0;
    for (int e = 0; e < 3; ++e) {
        double d[3], x[3];
        for (int i = 0; i < 3; ++i) {
            d[i] = end[e][i] - org[e][i];
            x[i] = p[i] - org[e][i];
        }
        const double dd = d[0] * d[0] + d[1] * d[1] + d[2] * d[2];
        double sg = dd > 0.0 ? (x[0] * d[0] + x[1] * d[1] + x[2] * d[2]) / dd : 0.0;
        sg = sg < 0.0 ? 0.0 : (sg > 1.0 ? 1.0 : sg);
        double r[3];
        for (int i = 0; i < 3; ++i) r[i] = x[i] - sg * d[i];
        const double dist = r[0] * r[0] + r[1] * r[1] + r[2] * r[2];
        if (dist < bestd) {
            bestd = dist;
            for (int i = 0; i < 3; ++i) res[i] = r[i];
            w[e] = 1.0 - sg;
            w[(e + 1) % 3] = sg;
            w[(e + 2) % 3] = 0.0;
        }
    }
}

// Per point: gP = 2 g (p - q) (to gP_out and to gp_ws for the scatter) and
// the weights w of q.  A point whose face is out of range, or has a vertex out
// of range, gets gP = 0 and weights 0.
__global__ __launch_bounds__(kThreads) void p2s_point_grad_kernel(
    int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P, const float *V,
    const int32_t *F, const int32_t *fidx, const float *g, float *gP_out, float *gp_ws, float *w_ws)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= B * S) return;
    const int64_t b = k / S;
    // The point, its factor and face, then the face's vertex indices, then the
    // vertices: three memory rounds with no branch between them (an invalid
    // face or vertex index reads face / vertex 0 and contributes nothing).
    const int32_t f = fidx[k];
    float pf[3];
#pragma unroll
    for (int i = 0; i < 3; ++i) pf[i] = P[3 * k + i];
    const float gk = g[k];
    const bool fok = (f >= 0) & (f < nf);
    const int32_t *t = F + (b * nf + (fok ? f : 0)) * 3;
    int32_t tv[3];
#pragma unroll
    for (int i = 0; i < 3; ++i) tv[i] = t[i];
    const bool ok = fok & face_ok_nb(tv, nv);
    const float *Vb = V + b * nv * 3;
    float vf[3][3];
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int i = 0; i < 3; ++i) vf[j][i] = Vb[3 * static_cast<int64_t>(ok ? tv[j] : 0) + i];
    float gp[3] = {0.0f, 0.0f, 0.0f}, wf[3] = {0.0f, 0.0f, 0.0f};
    if (ok) {
        double p[3], A[3], Bv[3], C[3], w[3], res[3];
        for (int i = 0; i < 3; ++i) {
            p[i] = pf[i];
            A[i] = vf[0][i];
            Bv[i] = vf[1][i];
            C[i] = vf[2][i];
        }
        closest_point(p, A, Bv, C, w, res);
        const double g2 = 2.0 * static_cast<double>(gk);
        for (int i = 0; i < 3; ++i) {
            gp[i] = static_cast<float>(g2 * res[i]);
            wf[i] = static_cast<float>(w[i]);
        }
    }
    for (int i = 0; i < 3; ++i) {
        if (gP_out) gP_out[3 * k + i] = gp[i];
        gp_ws[3 * k + i] = gp[i];
        w_ws[3 * k + i] = wf[i];
    }
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

}  // namespace

P2SPlan plan_p2s(int64_t B, int64_t S, int64_t nf)
{
    P2SPlan p;
    p.nQG = static_cast<int>(std::max<int64_t>(1, ceil_div(S, kPGroup)));
    const int64_t groups = B * p.nQG;
    int64_t want = groups > 0 ? ceil_div(kTargetTiles, groups) : 1;
    want = std::max<int64_t>(1, std::min(want, ceil_div(nf, kMinFB)));
    want = std::max<int64_t>(want, ceil_div(nf, kMaxFB));
    p.FB = static_cast<int>(ceil_div(nf, want));
    const int64_t blocks = ceil_div(nf, p.FB);
    p.FS = std::max(1, p.FB / 4);
    if (groups * blocks >= kSlots && groups * blocks <= kSmallRounds * kSlots) {
        // A launch of one to a few rounds: the last faces of every item go to
        // small blocks (a quarter of the size), about a quarter round of
        // resident workgroups' worth of work, dispatched last to even out the
        // end.
        const int64_t small = std::min<int64_t>(
            nf, ceil_div(ceil_div(kSlots / 4 * p.FB, std::max<int64_t>(groups, 1)), p.FS) * p.FS);
        p.nBig = static_cast<int>((nf - small) / p.FB);
        p.nFB = p.nBig + static_cast<int>(ceil_div(nf - static_cast<int64_t>(p.nBig) * p.FB, p.FS));
    } else {
        p.nBig = static_cast<int>(blocks);
        p.nFB = p.nBig;
    }
    return p;
}

size_t p2s_workspace_bytes(int64_t B, int64_t S, int64_t nv, int64_t nf)
{
    const P2SPlan p = plan_p2s(B, S, nf);
    const size_t recs = align256(static_cast<size_t>(B * nf) * kRec * 4);
    const size_t keys = p.nFB > 1 ? align256(static_cast<size_t>(B * p.nFB * S) * 8) : 0;
    const size_t per_point = align256(static_cast<size_t>(B * S) * 12);
    const size_t bwd = 2 * per_point + bary_scatter_workspace_bytes(B, nv, S);
    return std::max(recs + keys, bwd);
}

hipError_t launch_p2s_forward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                              const float *V, const int32_t *F, float *dist, int32_t *fidx,
                              void *ws, hipStream_t stream)
{
    const P2SPlan p = plan_p2s(B, S, nf);
    char *base = static_cast<char *>(ws);
    float *rec = reinterpret_cast<float *>(base);
    uint64_t *part = reinterpret_cast<uint64_t *>(base + align256(static_cast<size_t>(B * nf) * kRec * 4));
    face_record_kernel<<<static_cast<uint32_t>(ceil_div(B * nf, kThreads)), kThreads, 0, stream>>>(
        B, nv, nf, V, F, rec);
    P2SArgs a{P, rec, part, dist, fidx, S, nf, p.nQG, p.nFB, p.FB, p.nBig, p.FS, B};
    p2s_search_kernel<<<static_cast<uint32_t>(B * p.nQG * p.nFB), kPThreads, 0, stream>>>(a);
    if (p.nFB > 1)
        p2s_merge_kernel<<<static_cast<uint32_t>(ceil_div(B * S, kThreads)), kThreads, 0, stream>>>(
            B, S, p.nFB, part, dist, fidx);
    return hipGetLastError();
}

hipError_t launch_p2s_backward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                               const float *V, const int32_t *F, const int32_t *fidx,
                               const float *g, float *gP, float *gV, void *ws, hipStream_t stream)
{
    char *base = static_cast<char *>(ws);
    const size_t per_point = align256(static_cast<size_t>(B * S) * 12);
    float *gp_ws = reinterpret_cast<float *>(base);
    float *w_ws = reinterpret_cast<float *>(base + per_point);
    void *scatter_ws = base + 2 * per_point;
    if (S > 0)
        p2s_point_grad_kernel<<<static_cast<uint32_t>(ceil_div(B * S, kThreads)), kThreads, 0,
                                stream>>>(B, S, nv, nf, P, V, F, fidx, g, gP, gp_ws, w_ws);
    if (gV) {
        const hipError_t e = launch_bary_scatter(B, nv, nf, F, S, fidx, nullptr, nullptr, w_ws,
                                                 gp_ws, true, gV, scatter_ws, stream);
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

}  // namespace cdk

/*
 * mesh_oracle.c -- plain CPU oracle for differentiable mesh surface sampling.
 *
 * TEST INFRASTRUCTURE ONLY (same rules as cd_oracle.c: only the tests, the
 * smoke check and the benchmark's CPU baseline use it; no code is shared with
 * the HIP library).
 *
 * Kaolin Sec. 2.1: a polygon mesh is converted to a point cloud by sampling
 * its surface with the reparameterization trick, so that the sampled points
 * are differentiable functions of the vertex positions.  For a triangle with
 * vertices (a, b, c) and two uniform numbers r1, r2 in [0, 1):
 *     p = (1 - sqrt(r1)) a + sqrt(r1) (1 - r2) b + sqrt(r1) r2 c
 * which is uniform on the triangle; triangles are chosen with probability
 * proportional to their area (a categorical draw, not differentiated).
 *
 * Face choice: area_f = |(b - a) x (c - a)| / 2; with cdf_f = sum_{k<=f} area_k
 * and total = cdf_{nf-1}, a uniform u picks the first f with u * total < cdf_f.
 * Everything is evaluated in double from the float32 inputs.
 */
#include <math.h>
#include <stdint.h>

static void load3(const float *p, double *o)
{
    o[0] = p[0];
    o[1] = p[1];
    o[2] = p[2];
}

/* area[b, f] for every face of every item.  V [B, nv, 3], F [B, nf, 3]. */
void oracle_face_areas(int64_t B, int64_t nv, int64_t nf, const float *V, const int32_t *F,
                       double *area)
{
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t f = 0; f < nf; ++f) {
            const int32_t *t = F + (b * nf + f) * 3;
            double va[3], vb[3], vc[3];
            load3(V + (b * nv + t[0]) * 3, va);
            load3(V + (b * nv + t[1]) * 3, vb);
            load3(V + (b * nv + t[2]) * 3, vc);
            const double e1[3] = {vb[0] - va[0], vb[1] - va[1], vb[2] - va[2]};
            const double e2[3] = {vc[0] - va[0], vc[1] - va[1], vc[2] - va[2]};
            const double cx = e1[1] * e2[2] - e1[2] * e2[1];
            const double cy = e1[2] * e2[0] - e1[0] * e2[2];
            const double cz = e1[0] * e2[1] - e1[1] * e2[0];
            area[b * nf + f] = 0.5 * sqrt(cx * cx + cy * cy + cz * cz);
        }
    }
}

/* Area-weighted face choice for S uniforms per item: fidx [B, S]. */
void oracle_sample_faces(int64_t B, int64_t nv, int64_t nf, const float *V, const int32_t *F,
                         int64_t S, const float *u, double *scratch_area, int32_t *fidx)
{
    oracle_face_areas(B, nv, nf, V, F, scratch_area);
    for (int64_t b = 0; b < B; ++b) {
        const double *ar = scratch_area + b * nf;
        double total = 0.0;
        for (int64_t f = 0; f < nf; ++f) total += ar[f];
        for (int64_t s = 0; s < S; ++s) {
            const double target = (double)u[b * S + s] * total;
            double cdf = 0.0;
            int64_t pick = -1;
            for (int64_t f = 0; f < nf; ++f) {
                cdf += ar[f];
                if (target < cdf) {
                    pick = f;
                    break;
                }
            }
            if (pick < 0) { /* rounding at the top end: the last face with area */
                for (int64_t f = nf - 1; f >= 0; --f)
                    if (ar[f] > 0.0) {
                        pick = f;
                        break;
                    }
            }
            fidx[b * S + s] = (int32_t)pick;
        }
    }
}

/* Barycentric weights of the reparameterised sample. */
static void weights(double r1, double r2, double *w)
{
    const double s1 = sqrt(r1);
    w[0] = 1.0 - s1;
    w[1] = s1 * (1.0 - r2);
    w[2] = s1 * r2;
}

/* P [B, S, 3] for given faces and uniforms. */
void oracle_sample_points(int64_t B, int64_t nv, int64_t nf, const float *V, const int32_t *F,
                          int64_t S, const int32_t *fidx, const float *r1, const float *r2,
                          double *P)
{
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t s = 0; s < S; ++s) {
            const int64_t k = b * S + s;
            const int32_t *t = F + (b * nf + fidx[k]) * 3;
            double w[3];
            weights(r1[k], r2[k], w);
            for (int c = 0; c < 3; ++c) {
                P[k * 3 + c] = w[0] * V[(b * nv + t[0]) * 3 + c] +
                               w[1] * V[(b * nv + t[1]) * 3 + c] +
                               w[2] * V[(b * nv + t[2]) * 3 + c];
            }
        }
    }
}

/* gV [B, nv, 3] = d(sum gP . P) / dV: each sample adds w_i gP to its face's
 * vertex i.  Also returns, per vertex component, the sum of absolute
 * contributions (sV) and, per vertex, their number (nV). */
void oracle_sample_backward(int64_t B, int64_t nv, int64_t nf, const int32_t *F, int64_t S,
                            const int32_t *fidx, const float *r1, const float *r2,
                            const double *gP, double *gV, double *sV, int32_t *nV)
{
    for (int64_t t = 0; t < B * nv * 3; ++t) {
        gV[t] = 0.0;
        sV[t] = 0.0;
    }
    for (int64_t t = 0; t < B * nv; ++t) nV[t] = 0;
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t s = 0; s < S; ++s) {
            const int64_t k = b * S + s;
            const int32_t *tri = F + (b * nf + fidx[k]) * 3;
            double w[3];
            weights(r1[k], r2[k], w);
            for (int i = 0; i < 3; ++i) {
                const int64_t v = b * nv + tri[i];
                for (int c = 0; c < 3; ++c) {
                    const double term = w[i] * gP[k * 3 + c];
                    gV[v * 3 + c] += term;
                    sV[v * 3 + c] += fabs(term);
                }
                nV[v] += 1;
            }
        }
    }
}

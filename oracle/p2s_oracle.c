/*
 * p2s_oracle.c -- plain CPU oracle for the point-to-surface distance between
 * point clouds and triangle meshes.
 *
 * TEST INFRASTRUCTURE ONLY (same rules as cd_oracle.c: only the tests, the
 * smoke check and the benchmark's CPU baseline use it; no code is shared with
 * the HIP library).
 *
 * Kaolin Sec. 2.5 lists a point-to-surface loss for meshes beside the Chamfer
 * distance for point clouds.  For a point p and a closed triangle
 * T = {a + s (b - a) + t (c - a) : s, t >= 0, s + t <= 1} the distance is
 * min over q in T of |p - q|^2; a point's distance to a mesh is the minimum
 * over its faces (the lowest face index on exact ties), and the loss is the
 * mean over the points.
 *
 * T is convex, so the closest point q* is unique.  Either it lies in the
 * relative interior of T, where it is the orthogonal projection of p onto the
 * plane of T (and that projection is inside T), or it lies on the boundary,
 * i.e. on one of the three edges, where it is the projection of p onto the
 * edge's line clamped to the segment.  Hence
 *     dist^2 = min(plane distance if the projection is inside,
 *                  the three point-to-segment distances).
 * A zero-area triangle has no interior: the edges alone decide.
 *
 * Gradient: dist^2 = min over barycentric w in the simplex of
 * |p - sum_i w_i v_i|^2, and the minimiser w* is unique, so (envelope theorem)
 *     d dist^2 / d p   =  2 (p - q*)
 *     d dist^2 / d v_i = -2 w*_i (p - q*).
 * Everything is evaluated in double from the float32 inputs.
 */
#include <math.h>
#include <stdint.h>

static void sub3(const double *x, const double *y, double *o)
{
    o[0] = x[0] - y[0];
    o[1] = x[1] - y[1];
    o[2] = x[2] - y[2];
}

static double dot3(const double *x, const double *y)
{
    return x[0] * y[0] + x[1] * y[1] + x[2] * y[2];
}

static void cross3(const double *x, const double *y, double *o)
{
    o[0] = x[1] * y[2] - x[2] * y[1];
    o[1] = x[2] * y[0] - x[0] * y[2];
    o[2] = x[0] * y[1] - x[1] * y[0];
}

/* Squared distance from p to the segment [x, y]; *t is the parameter of the
 * closest point x + t (y - x), t in [0, 1] (0 for a zero-length segment). */
static double seg_dist2(const double *p, const double *x, const double *y, double *t)
{
    double e[3], v[3], d[3];
    sub3(y, x, e);
    sub3(p, x, v);
    const double ee = dot3(e, e);
    double s = ee > 0.0 ? dot3(v, e) / ee : 0.0;
    if (s < 0.0) s = 0.0;
    if (s > 1.0) s = 1.0;
    d[0] = v[0] - s * e[0];
    d[1] = v[1] - s * e[1];
    d[2] = v[2] - s * e[2];
    *t = s;
    return dot3(d, d);
}

/* Squared distance from p to the closed triangle (a, b, c); w receives the
 * barycentric coordinates of the closest point. */
double oracle_point_triangle(const double *p, const double *a, const double *b, const double *c,
                             double *w)
{
    double e0[3], e1[3], n[3], v[3];
    sub3(b, a, e0);
    sub3(c, a, e1);
    cross3(e0, e1, n);
    const double nn = dot3(n, n);
    if (nn > 0.0) {
        /* Projection q = p - (n.(p-a)/nn) n; its barycentric coordinates are
         * the signed areas of the sub-triangles opposite each vertex over the
         * whole area (all measured along n). */
        sub3(p, a, v);
        const double h = dot3(n, v) / nn;
        const double q[3] = {p[0] - h * n[0], p[1] - h * n[1], p[2] - h * n[2]};
        double x[3], y[3], z[3];
        sub3(c, b, x);
        sub3(q, b, y);
        cross3(x, y, z);
        const double wa = dot3(z, n) / nn;
        sub3(a, c, x);
        sub3(q, c, y);
        cross3(x, y, z);
        const double wb = dot3(z, n) / nn;
        sub3(b, a, x);
        sub3(q, a, y);
        cross3(x, y, z);
        const double wc = dot3(z, n) / nn;
        if (wa >= 0.0 && wb >= 0.0 && wc >= 0.0) {
            w[0] = wa;
            w[1] = wb;
            w[2] = wc;
            return h * h * nn;
        }
    }
    /* Boundary: the closest of the three edges ab, bc, ca (first on ties). */
    double t;
    double best = seg_dist2(p, a, b, &t);
    w[0] = 1.0 - t;
    w[1] = t;
    w[2] = 0.0;
    double d = seg_dist2(p, b, c, &t);
    if (d < best) {
        best = d;
        w[0] = 0.0;
        w[1] = 1.0 - t;
        w[2] = t;
    }
    d = seg_dist2(p, c, a, &t);
    if (d < best) {
        best = d;
        w[0] = t;
        w[1] = 0.0;
        w[2] = 1.0 - t;
    }
    return best;
}

static void vertex(const float *Vb, int32_t i, double *o)
{
    o[0] = Vb[3 * (int64_t)i + 0];
    o[1] = Vb[3 * (int64_t)i + 1];
    o[2] = Vb[3 * (int64_t)i + 2];
}

/* n independent point-triangle pairs (float32 in, double out), for pins. */
void oracle_point_triangle_batch(int64_t n, const float *p, const float *a, const float *b,
                                 const float *c, double *d2, double *w)
{
    for (int64_t k = 0; k < n; ++k) {
        double pp[3], aa[3], bb[3], cc[3];
        for (int i = 0; i < 3; ++i) {
            pp[i] = p[3 * k + i];
            aa[i] = a[3 * k + i];
            bb[i] = b[3 * k + i];
            cc[i] = c[3 * k + i];
        }
        d2[k] = oracle_point_triangle(pp, aa, bb, cc, w + 3 * k);
    }
}

/*
 * Forward: for every point p = P[b, s], dist[b, s] = min over faces f of the
 * squared distance to face f (faces in ascending order, strict <, so the
 * lowest index wins exact ties), fidx[b, s] = that face and w[b, s] the
 * barycentric coordinates of the closest point.  A mesh whose faces all have
 * an out-of-range vertex gives dist = +inf and fidx = -1.
 */
void oracle_p2s_forward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                        const float *V, const int32_t *F, double *dist, int32_t *fidx, double *w)
{
#pragma omp parallel for collapse(2) schedule(dynamic, 64)
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t s = 0; s < S; ++s) {
            const float *Vb = V + b * nv * 3;
            const int32_t *Fb = F + b * nf * 3;
            const int64_t k = b * S + s;
            double p[3] = {P[3 * k + 0], P[3 * k + 1], P[3 * k + 2]};
            double best = INFINITY, bw[3] = {0.0, 0.0, 0.0};
            int32_t arg = -1;
            for (int64_t f = 0; f < nf; ++f) {
                const int32_t *t = Fb + 3 * f;
                if (t[0] < 0 || t[0] >= nv || t[1] < 0 || t[1] >= nv || t[2] < 0 || t[2] >= nv)
                    continue;
                double a[3], bb[3], c[3], ww[3];
                vertex(Vb, t[0], a);
                vertex(Vb, t[1], bb);
                vertex(Vb, t[2], c);
                const double d = oracle_point_triangle(p, a, bb, c, ww);
                if (d < best) {
                    best = d;
                    arg = (int32_t)f;
                    bw[0] = ww[0];
                    bw[1] = ww[1];
                    bw[2] = ww[2];
                }
            }
            dist[k] = best;
            fidx[k] = arg;
            w[3 * k + 0] = bw[0];
            w[3 * k + 1] = bw[1];
            w[3 * k + 2] = bw[2];
        }
    }
}

/*
 * Backward for given face choices fidx and per-point weights g = dL/d dist:
 *   gP[b, s]    = 2 g (p - q*)
 *   gV[b, v_i] += -2 g w*_i (p - q*)   for the three vertices of the face.
 * sV receives the per-component sums of |contribution| and nV the number of
 * contributions per vertex (for tolerances).  Points whose face index is out
 * of range get gP = 0 and contribute nothing.
 */
void oracle_p2s_backward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                         const float *V, const int32_t *F, const int32_t *fidx, const double *g,
                         double *gP, double *gV, double *sV, int32_t *nV)
{
    for (int64_t i = 0; i < B * nv * 3; ++i) {
        gV[i] = 0.0;
        sV[i] = 0.0;
    }
    for (int64_t i = 0; i < B * nv; ++i) nV[i] = 0;
    for (int64_t b = 0; b < B; ++b) {
        const float *Vb = V + b * nv * 3;
        const int32_t *Fb = F + b * nf * 3;
        for (int64_t s = 0; s < S; ++s) {
            const int64_t k = b * S + s;
            const int32_t f = fidx[k];
            gP[3 * k + 0] = gP[3 * k + 1] = gP[3 * k + 2] = 0.0;
            if (f < 0 || f >= nf) continue;
            const int32_t *t = Fb + 3 * (int64_t)f;
            if (t[0] < 0 || t[0] >= nv || t[1] < 0 || t[1] >= nv || t[2] < 0 || t[2] >= nv)
                continue;
            double p[3] = {P[3 * k + 0], P[3 * k + 1], P[3 * k + 2]};
            double a[3], bb[3], c[3], w[3];
            vertex(Vb, t[0], a);
            vertex(Vb, t[1], bb);
            vertex(Vb, t[2], c);
            oracle_point_triangle(p, a, bb, c, w);
            double q[3];
            for (int i = 0; i < 3; ++i) q[i] = w[0] * a[i] + w[1] * bb[i] + w[2] * c[i];
            for (int i = 0; i < 3; ++i) gP[3 * k + i] = 2.0 * g[k] * (p[i] - q[i]);
            for (int j = 0; j < 3; ++j) {
                const int64_t v = b * nv + t[j];
                nV[v] += 1;
                for (int i = 0; i < 3; ++i) {
                    const double term = -2.0 * g[k] * w[j] * (p[i] - q[i]);
                    gV[3 * v + i] += term;
                    sV[3 * v + i] += fabs(term);
                }
            }
        }
    }
}

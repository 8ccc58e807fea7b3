/*
 * cd_oracle.c -- plain CPU oracle for the batched Chamfer distance.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the benchmark's CPU
 * baseline use it.  It shares no source with the HIP library.
 *
 * What it computes (Kaolin, Sec. 2.5: Chamfer distance for point clouds,
 * defined through the cited point-set-generation paper of Fan et al.):
 *
 *   d(p, q)        = ((p.x-q.x)^2 + (p.y-q.y)^2) + (p.z-q.z)^2   (float32)
 *   dist_xy[b,i]   = min_j d(x_i, y_j),   idx_xy[b,i] = lowest j attaining it
 *   dist_yx[b,j]   = min_i d(y_j, x_i),   idx_yx[b,j] = lowest i attaining it
 *   chamfer[b]     = w1 * mean_i dist_xy[b,i] + w2 * mean_j dist_yx[b,j]
 *   F-score@tau    = 2PR/(P+R), P = #{dist_xy < tau^2}/N, R = #{dist_yx < tau^2}/M
 *   backward       = gradient of sum_b grad_out[b] * chamfer[b] for the
 *                    nearest neighbours chosen above (a subgradient at ties)
 *
 * The nearest-neighbour decision is taken in float32, the precision the GPU
 * path computes distances in, with every operation rounded separately
 * (build with -ffp-contract=off).  A second mode evaluates the same order as
 * fma(dz,dz, fma(dy,dy, dx*dx)) with correctly rounded fmaf().  Sums, F-score
 * and gradients are evaluated in double.  All loops are the plain definition:
 * no blocking, no early exit, targets scanned in ascending index order with a
 * strict '<' so that equal distances keep the lowest index.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Squared Euclidean distance in float32, query minus target. */
static float sq_dist_f32(const float *p, const float *q, int fused)
{
    float dx = p[0] - q[0];
    float dy = p[1] - q[1];
    float dz = p[2] - q[2];
    if (fused)
        return fmaf(dz, dz, fmaf(dy, dy, dx * dx));
    float sxy = dx * dx + dy * dy;
    return sxy + dz * dz;
}

int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of later parallel loops (timing only; the results do not depend on it). */
void oracle_set_threads(int n)
{
#ifdef _OPENMP
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}

/*
 * Nearest neighbour of every query p in P[b] among the targets Q[b].
 * P: [B, NP, 3], Q: [B, NQ, 3] float32 row-major.  dist/idx: [B, NP].
 */
void oracle_nn(int64_t B, int64_t NP, int64_t NQ, const float *P, const float *Q,
               int fused, float *dist, int32_t *idx)
{
    int64_t total = B * NP;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t t = 0; t < total; ++t) {
        int64_t b = t / NP;
        const float *p = P + 3 * t;
        const float *qb = Q + 3 * b * NQ;
        float best = INFINITY;
        int64_t arg = -1;
        for (int64_t j = 0; j < NQ; ++j) {
            float d = sq_dist_f32(p, qb + 3 * j, fused);
            if (d < best) {
                best = d;
                arg = j;
            }
        }
        dist[t] = best;
        idx[t] = (int32_t)arg;
    }
}

/* chamfer[b] = w1 * (sum_i dist_xy[b,i]) / N + w2 * (sum_j dist_yx[b,j]) / M, in double. */
void oracle_chamfer(int64_t B, int64_t N, int64_t M, const float *dist_xy, const float *dist_yx,
                    double w1, double w2, double *out)
{
    for (int64_t b = 0; b < B; ++b) {
        double sx = 0.0, sy = 0.0;
        for (int64_t i = 0; i < N; ++i)
            sx += (double)dist_xy[b * N + i];
        for (int64_t j = 0; j < M; ++j)
            sy += (double)dist_yx[b * M + j];
        out[b] = w1 * (sx / (double)N) + w2 * (sy / (double)M);
    }
}

/*
 * F-score at threshold tau: a point counts as matched when its squared
 * nearest-neighbour distance is strictly below tau^2 (exact in double for a
 * float tau).  Precision over X (dist_xy), recall over Y (dist_yx).
 */
void oracle_fscore(int64_t B, int64_t N, int64_t M, const float *dist_xy, const float *dist_yx,
                   float tau, double *f, double *prec, double *rec,
                   int64_t *cnt_p, int64_t *cnt_r)
{
    double t2 = (double)tau * (double)tau;
    for (int64_t b = 0; b < B; ++b) {
        int64_t cp = 0, cr = 0;
        for (int64_t i = 0; i < N; ++i)
            cp += ((double)dist_xy[b * N + i] < t2) ? 1 : 0;
        for (int64_t j = 0; j < M; ++j)
            cr += ((double)dist_yx[b * M + j] < t2) ? 1 : 0;
        double P = (double)cp / (double)N;
        double R = (double)cr / (double)M;
        cnt_p[b] = cp;
        cnt_r[b] = cr;
        prec[b] = P;
        rec[b] = R;
        f[b] = (P + R > 0.0) ? (2.0 * P * R) / (P + R) : 0.0;
    }
}

/*
 * Gradient of L = sum_{b,i} g_xy[b,i] * dist_xy[b,i] + sum_{b,j} g_yx[b,j] * dist_yx[b,j]
 * with the nearest neighbours fixed to idx_xy / idx_yx:
 *   d dist_xy[b,i] / d x_i =  2 (x_i - y_j),   d dist_xy[b,i] / d y_j = -2 (x_i - y_j),  j = idx_xy[b,i]
 *   d dist_yx[b,j] / d y_j =  2 (y_j - x_i),   d dist_yx[b,j] / d x_i = -2 (y_j - x_i),  i = idx_yx[b,j]
 * Everything in double from the float32 inputs.  Besides gX/gY it records, per
 * output component, the sum of absolute contributions (sX/sY) and, per point,
 * the number of contributions (nX/nY); the GPU's float atomics may add the
 * same terms in any order, and these bound that reordering.
 */
void oracle_backward_pointwise(int64_t B, int64_t N, int64_t M,
                               const double *g_xy, const double *g_yx,
                               const float *X, const float *Y,
                               const int32_t *idx_xy, const int32_t *idx_yx,
                               double *gX, double *gY, double *sX, double *sY,
                               int32_t *nX, int32_t *nY)
{
    for (int64_t t = 0; t < B * N * 3; ++t) { gX[t] = 0.0; sX[t] = 0.0; }
    for (int64_t t = 0; t < B * M * 3; ++t) { gY[t] = 0.0; sY[t] = 0.0; }
    for (int64_t t = 0; t < B * N; ++t) nX[t] = 0;
    for (int64_t t = 0; t < B * M; ++t) nY[t] = 0;

    for (int64_t b = 0; b < B; ++b) {
        for (int64_t i = 0; i < N; ++i) {
            int64_t j = idx_xy[b * N + i];
            double g = g_xy[b * N + i];
            for (int c = 0; c < 3; ++c) {
                double diff = (double)X[(b * N + i) * 3 + c] - (double)Y[(b * M + j) * 3 + c];
                double term = 2.0 * g * diff;
                gX[(b * N + i) * 3 + c] += term;
                gY[(b * M + j) * 3 + c] -= term;
                sX[(b * N + i) * 3 + c] += fabs(term);
                sY[(b * M + j) * 3 + c] += fabs(term);
            }
            nX[b * N + i] += 1;
            nY[b * M + j] += 1;
        }
        for (int64_t j = 0; j < M; ++j) {
            int64_t i = idx_yx[b * M + j];
            double g = g_yx[b * M + j];
            for (int c = 0; c < 3; ++c) {
                double diff = (double)Y[(b * M + j) * 3 + c] - (double)X[(b * N + i) * 3 + c];
                double term = 2.0 * g * diff;
                gY[(b * M + j) * 3 + c] += term;
                gX[(b * N + i) * 3 + c] -= term;
                sY[(b * M + j) * 3 + c] += fabs(term);
                sX[(b * N + i) * 3 + c] += fabs(term);
            }
            nY[b * M + j] += 1;
            nX[b * N + i] += 1;
        }
    }
}

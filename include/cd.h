/*
 * cd.h -- C ABI of the MI355X (gfx950) batched Chamfer-distance library.
 *
 * Operation (Kaolin, Sec. 2.5: Chamfer distance for point clouds, defined
 * through the cited point-set-generation paper of Fan et al.).  For clouds
 * X [B,N,3] and Y [B,M,3] and the squared distance
 *     d(p,q) = ((p.x-q.x)^2 + (p.y-q.y)^2) + (p.z-q.z)^2      (float32)
 * the library computes, per item b,
 *     dist_xy[b,i] = min_j d(x_i, y_j),  idx_xy[b,i] = lowest j attaining it
 *     dist_yx[b,j] = min_i d(y_j, x_i),  idx_yx[b,j] = lowest i attaining it
 *     chamfer[b]   = w1 * mean_i dist_xy[b,i] + w2 * mean_j dist_yx[b,j]
 * the F-score at a distance threshold, and the gradient of the loss with
 * respect to both clouds.  The squared distances are evaluated in float32 as
 * fma(dz,dz, fma(dy,dy, dx*dx)) with d = query - target.
 *
 * Conventions shared by every call:
 *  - Array pointers are DEVICE memory (hipMalloc or torch tensors on the
 *    device), allocated and owned by the caller.  The library allocates no
 *    memory, keeps no pointer after a call returns and holds no mutable
 *    global state other than the thread-local error text.
 *  - Layout: X and Y are float32, row-major, contiguous [B, N, 3] / [B, M, 3]
 *    (x, y, z interleaved).  Per-point outputs are contiguous [B, N] / [B, M];
 *    per-item outputs are [B].
 *  - Every call is asynchronous on `stream` (NULL = the null stream).  CD_OK
 *    means "enqueued"; results are valid once the stream has reached them.
 *  - Arguments are checked before anything is enqueued, without touching
 *    device memory: a NULL pointer (when B > 0), B < 0, N < 1, M < 1,
 *    N or M >= 2^31 (indices are int32), B * (N + M) > 2^31 (one thread per
 *    point must fit a launch), a negative or NaN tau, or an unaligned
 *    workspace returns CD_ERR_INVALID_ARG.  B == 0 is a no-op that returns
 *    CD_OK.
 *  - Inputs must be finite and their squared distances must not overflow
 *    float32 (coordinates of magnitude at most 2^62, about 4.6e18, always
 *    satisfy this); other inputs are undefined behaviour (an overflowing
 *    distance may yield an index of -1).  Outputs must not alias inputs.
 *  - A failed launch returns CD_ERR_HIP; cd_last_error() then holds the HIP
 *    error text for the calling thread.
 */
#ifndef CD_H
#define CD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *hipStream_t;

typedef enum {
    CD_OK = 0,
    CD_ERR_INVALID_ARG = 1,
    CD_ERR_WORKSPACE = 2,
    CD_ERR_HIP = 3
} cd_status;

/* Static, human-readable name of a status code. */
const char *cd_status_string(cd_status s);

/* Detail of the last error raised on the calling thread ("" if none). */
const char *cd_last_error(void);

/* Library version as "major.minor.patch" (static string). */
const char *cd_version(void);

/*
 * Bytes of device workspace cd_forward needs for this shape (0 when B == 0):
 * one 8-byte key per point of both clouds, 8 B (N + M) rounded up to 256-byte
 * segments.  Returns 0 and sets cd_last_error() for an invalid shape.
 */
size_t cd_workspace_bytes(int64_t B, int64_t N, int64_t M);

/*
 * Nearest neighbours in both directions (Sec. 2.5: the point matching that
 * the Chamfer distance is built on).
 *   X [B,N,3], Y [B,M,3]      input clouds (device, float32)
 *   dist_xy [B,N], idx_xy [B,N]   for every x_i: min_j d(x_i,y_j) and the
 *                                 lowest j attaining it (float32 / int32)
 *   dist_yx [B,M], idx_yx [B,M]   the same for every y_j against X
 *   ws, ws_bytes               device workspace of at least
 *                              cd_workspace_bytes(B,N,M) bytes, 256-byte
 *                              aligned; its contents on entry are ignored and
 *                              on exit are unspecified.  CD_ERR_WORKSPACE if
 *                              too small.
 * Results are bitwise reproducible from run to run.
 */
cd_status cd_forward(int64_t B, int64_t N, int64_t M,
                     const float *X, const float *Y,
                     float *dist_xy, int32_t *idx_xy,
                     float *dist_yx, int32_t *idx_yx,
                     void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * cd_forward without a workspace argument, for callers that cannot allocate
 * device memory (code under graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results and checks as cd_forward
 * (the results are bitwise identical to it); the workspace is a static device
 * array of CD_FORWARD_NOALLOC_MAX_BYTES bytes inside the library, one per GPU
 * the library runs on, held until the process ends.  The call allocates
 * nothing; the first call on a device looks up that device's array address.
 * Shapes whose cd_workspace_bytes(B, N, M) exceeds the limit (about 8.4
 * million points in B (N + M)) return CD_ERR_WORKSPACE with the sizes in
 * cd_last_error(); use cd_forward for them.  Every call on one GPU shares
 * that GPU's array: calls that overlap in time on one GPU (two streams, two
 * threads) race and give undefined results; calls ordered on one stream, or
 * synchronized, are safe.
 */
#define CD_FORWARD_NOALLOC_MAX_BYTES ((size_t)64 << 20)
cd_status cd_forward_noalloc(int64_t B, int64_t N, int64_t M,
                             const float *X, const float *Y,
                             float *dist_xy, int32_t *idx_xy,
                             float *dist_yx, int32_t *idx_yx, hipStream_t stream);

/*
 * Chamfer reduction (Sec. 2.5): chamfer[b] = w1 * (sum_i dist_xy[b,i]) / N
 * + w2 * (sum_j dist_yx[b,j]) / M.  Sums are accumulated in double in a fixed
 * order and the result rounded once to float32 (bitwise reproducible).
 *   dist_xy [B,N], dist_yx [B,M]  from cd_forward;  chamfer [B] output.
 */
cd_status cd_reduce(int64_t B, int64_t N, int64_t M,
                    const float *dist_xy, const float *dist_yx,
                    float w1, float w2, float *chamfer, hipStream_t stream);

/*
 * F-score at threshold tau (a point-cloud metric beside the Chamfer distance
 * in Sec. 2.5; the paper does not define it, the standard definition is
 * used): a point is matched when its nearest-neighbour distance is strictly
 * below tau, tested exactly as dist < tau^2 on the float32 squared distance.
 *   precision[b] = #{i: dist_xy[b,i] < tau^2} / N
 *   recall[b]    = #{j: dist_yx[b,j] < tau^2} / M
 *   f[b]         = 2 P R / (P + R), or 0 when P + R == 0
 * P, R and F are computed in double and rounded to float32.  `precision` and
 * `recall` may be NULL; `f` may not.  tau < 0 or NaN is CD_ERR_INVALID_ARG.
 */
cd_status cd_fscore(int64_t B, int64_t N, int64_t M,
                    const float *dist_xy, const float *dist_yx, float tau,
                    float *f, float *precision, float *recall, hipStream_t stream);

/*
 * Chamfer reduction and F-score at several thresholds in one pass over the
 * distances (the two calls above, fused; results are bitwise identical to
 * them).  taus [ntau] is HOST memory (read during the call); chamfer [B],
 * f / precision / recall [ntau, B] are device memory (precision and recall
 * may be NULL; chamfer and f may not).  1 <= ntau <= 16, every tau >= 0 and
 * not NaN, else CD_ERR_INVALID_ARG.
 */
cd_status cd_metrics(int64_t B, int64_t N, int64_t M,
                     const float *dist_xy, const float *dist_yx, float w1, float w2,
                     const float *taus, int ntau, float *chamfer,
                     float *f, float *precision, float *recall, hipStream_t stream);

/*
 * Device workspace bytes cd_backward and cd_backward_pointwise need for these
 * sizes (0 for B == 0 or sizes cd_forward rejects): per-block bounds, and
 * per-chunk partial sums when a cloud's senders are split (at most a few
 * hundred MB), or, where the senders are first sorted by receiver slice, 4
 * bytes per point of both clouds plus each chunk's slice offsets.
 */
size_t cd_backward_workspace_bytes(int64_t B, int64_t N, int64_t M);

/*
 * Backward of sum_b grad_out[b] * chamfer[b] (the Chamfer loss used to
 * supervise networks, Sec. 2.5), for the neighbours cd_forward chose:
 *   gX[b,i] = 2 g_xy (x_i - y_{idx_xy[i]}) - sum_{j: idx_yx[j]=i} 2 g_yx (y_j - x_i)
 *   gY[b,j] = 2 g_yx (y_j - x_{idx_yx[j]}) - sum_{i: idx_xy[i]=j} 2 g_xy (x_i - y_j)
 * with g_xy = grad_out[b] * w1 / N and g_yx = grad_out[b] * w2 / M.
 *   grad_out [B]; X, Y, idx_xy, idx_yx as passed to / returned by cd_forward.
 *   gX [B,N,3], gY [B,M,3] are fully overwritten (not accumulated).
 *   ws: cd_backward_workspace_bytes(B, N, M) bytes, 256-byte aligned
 *   (CD_ERR_WORKSPACE if smaller).
 * Each term is evaluated in float32; the scatter sums are exact: every term is
 * rounded to a 64-bit fixed-point integer (grid 2^-k, with k from a bound on
 * the largest term: per block of up to 2048 receivers (fewer when the clouds
 * are small, so that more workgroups share the work) when the other cloud has at
 * most 16384 points or when the senders are sorted by receiver block first
 * (where a cloud's senders exceed 16384 points, or where repeated index scans
 * would read more than 64 MB otherwise), else per item and cloud; the grid is about 2^-61 times the number of terms times
 * that bound) and the integers are added, so the result is bitwise
 * reproducible run to run; own term + sum are added in double and rounded
 * once.  A point whose index lies
 * outside [0, M) / [0, N) contributes nothing (its own and scatter terms are
 * dropped).
 */
cd_status cd_backward(int64_t B, int64_t N, int64_t M, const float *grad_out,
                      float w1, float w2, const float *X, const float *Y,
                      const int32_t *idx_xy, const int32_t *idx_yx,
                      float *gX, float *gY, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Backward for an arbitrary loss of the nearest-neighbour distances:
 * g_xy [B,N] = dL/d dist_xy and g_yx [B,M] = dL/d dist_yx are given per point;
 * gX, gY and ws are as in cd_backward with those per-point factors.
 */
cd_status cd_backward_pointwise(int64_t B, int64_t N, int64_t M,
                                const float *g_xy, const float *g_yx,
                                const float *X, const float *Y,
                                const int32_t *idx_xy, const int32_t *idx_yx,
                                float *gX, float *gY, void *ws, size_t ws_bytes,
                                hipStream_t stream);

/*
 * Differentiable surface sampling of triangle meshes (Kaolin Sec. 2.1: mesh to
 * point-cloud conversion with the reparameterization trick), the step that
 * turns a predicted mesh into the point cloud the Chamfer loss compares.
 * Per item b: vertices V [B, nv, 3] float32, faces F [B, nf, 3] int32 (vertex
 * indices of item b), S samples.  The random numbers are inputs: u, r1, r2
 * [B, S] float32 in [0, 1).  A face with a vertex index outside [0, nv) has
 * area 0; a sample whose face index is outside [0, nf) gets a NaN point and no
 * gradient.  Checks (else CD_ERR_INVALID_ARG, nothing launched): B >= 0,
 * nv >= 1, nf >= 1, S >= 0, nv, nf, S < 2^31, B * S <= 2^31,
 * B * ceil(nv / 2048) <= 2^23.  B == 0 is a no-op; with S == 0 the forward
 * calls are no-ops and the backward writes gV = 0.
 */

/*
 * Device workspace bytes cd_mesh_sample_faces and cd_mesh_sample_backward need
 * for these sizes (the larger of the per-item cumulative face areas, 8 B nf,
 * and the backward's per-chunk vertex partial sums, at most about 48 MiB);
 * 0 for sizes the checks below reject.  One buffer serves both calls.
 */
size_t cd_mesh_workspace_bytes(int64_t B, int64_t nv, int64_t nf, int64_t S);

/*
 * Area-weighted face choice: fidx[b, s] = the first face f whose cumulative
 * area (faces 0..f) exceeds u[b, s] * total area.  Areas |(b-a) x (c-a)| / 2
 * are evaluated in float32, rounded to multiples of 2^-k (k chosen per item so
 * the total stays below 2^62, i.e. a resolution of about 2^-61 nf times the
 * largest area) and cumulated exactly in int64, so a face of zero area (or
 * with an out-of-range vertex) is never chosen.  A mesh of total area 0 gives
 * -1.  The choice is bitwise reproducible.
 * ws: cd_mesh_workspace_bytes(B, nv, nf, S) bytes, 256-byte aligned
 * (CD_ERR_WORKSPACE if smaller).
 */
cd_status cd_mesh_sample_faces(int64_t B, int64_t nv, int64_t nf, const float *V,
                               const int32_t *F, int64_t S, const float *u, int32_t *fidx,
                               void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Reparameterised samples: P[b, s] = (1 - sqrt(r1)) a + sqrt(r1) (1 - r2) b
 * + sqrt(r1) r2 c for the face fidx[b, s] = (a, b, c).  P [B, S, 3] float32.
 */
cd_status cd_mesh_sample_points(int64_t B, int64_t nv, int64_t nf, const float *V,
                                const int32_t *F, int64_t S, const int32_t *fidx,
                                const float *r1, const float *r2, float *P, hipStream_t stream);

/*
 * Backward of the samples: gV [B, nv, 3] = d(sum gP . P) / dV, i.e. each
 * sample adds its barycentric weight times gP[b, s] to each of its face's
 * three vertices.  gV is fully overwritten (vertices no sample touches get 0).
 * Each contribution w * gP is rounded from float32 to a 64-bit fixed-point
 * integer (grid 2^-k, k from the largest |gP| of a chunk of samples, about
 * 2^-61 / chunk length relative to it), summed exactly, and chunks are added
 * in double in a fixed order: the result is bitwise reproducible run to run.
 * ws: as for cd_mesh_sample_faces.
 */
cd_status cd_mesh_sample_backward(int64_t B, int64_t nv, int64_t nf, const int32_t *F,
                                  int64_t S, const int32_t *fidx, const float *r1,
                                  const float *r2, const float *gP, float *gV, void *ws,
                                  size_t ws_bytes, hipStream_t stream);

/*
 * Point-to-surface distance (Kaolin Sec. 2.5: the point-to-surface loss for
 * meshes, listed beside the Chamfer distance).  Per item b: points P [B, S, 3]
 * float32, vertices V [B, nv, 3] float32, faces F [B, nf, 3] int32.  The
 * distance of a point to a face is the squared Euclidean distance to the
 * closed triangle; the loss of an item is the mean over its points of the
 * distance to the nearest face (cd_reduce with w1 = 1, w2 = 0 computes it).
 * Faces with a vertex index outside [0, nv) are ignored.  Checks (else
 * CD_ERR_INVALID_ARG, nothing launched): B >= 0, S >= 0, nv >= 1, nf >= 1,
 * nv, nf, S < 2^31, B * S <= 2^31, B * nf <= 2^31, B * ceil(nv / 2048) <= 2^23.
 * B == 0 or S == 0 is a no-op (the backward still writes gV = 0 when S == 0).
 */

/* Device workspace bytes for cd_p2s_forward and cd_p2s_backward (one buffer
 * serves both); 0 for sizes the checks reject. */
size_t cd_p2s_workspace_bytes(int64_t B, int64_t S, int64_t nv, int64_t nf);

/*
 * dist [B, S] float32: squared distance from each point to the nearest face,
 * evaluated in float32; fidx [B, S] int32: that face, the lowest index among
 * exactly equal float32 distances; +inf and -1 when every face is ignored.
 * ws: cd_p2s_workspace_bytes(B, S, nv, nf) bytes, 256-byte aligned.
 */
cd_status cd_p2s_forward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                         const float *V, const int32_t *F, float *dist, int32_t *fidx, void *ws,
                         size_t ws_bytes, hipStream_t stream);

/*
 * Backward for the faces fidx chosen by the forward and g [B, S] = dL/d dist:
 * with q the closest point of face fidx to p (recomputed in double) and w its
 * barycentric coordinates, gP = 2 g (p - q) [B, S, 3] and
 * gV [B, nv, 3] = sum over points of -2 g w_i (p - q) on the face's vertex i
 * (exact fixed-point sums as in cd_mesh_sample_backward: bitwise
 * reproducible).  gP or gV may be NULL (not computed); both are fully
 * overwritten.  Points whose face is out of range get gP = 0.
 */
cd_status cd_p2s_backward(int64_t B, int64_t S, int64_t nv, int64_t nf, const float *P,
                          const float *V, const int32_t *F, const int32_t *fidx, const float *g,
                          float *gP, float *gV, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Approximate Earth-mover's distance between point clouds (Kaolin Sec. 2.5
 * names an approximate EMD among its point-cloud metrics, citing Fan et al.,
 * whose EMD is the optimal transport cost with Euclidean ground distance).  Per item: the
 * transport problem between X [B,N,3] and Y [B,M,3] with uniform masses 1/N,
 * 1/M and cost C_ij = |x_i - y_j|, regularised by entropy and solved with
 * log-domain Sinkhorn iterations (O(N M) work each).  Iteration t of
 * n_iters uses eps_t = eps_start (eps_end / eps_start)^(t / (n_iters - 1))
 * (eps_end if n_iters == 1) and updates
 *   f_i <- -eps_t log sum_j (1/M) exp((g_j - C_ij) / eps_t), then
 *   g_j <- -eps_t log sum_i (1/N) exp((f_i - C_ij) / eps_t).
 * The reported cost is sum_ij P_ij C_ij with P_ij = exp((f_i + g_j - C_ij) /
 * eps_end) / (N M).  Evaluated in float32 (hardware square roots and
 * exponentials); partial sums of the cost in double.  Shapes and checks as for
 * cd_forward, plus 3 B max(N, M) < 2^32 - 2^20; eps_start, eps_end > 0 and
 * finite, n_iters >= 1, else CD_ERR_INVALID_ARG.
 */

/* Device workspace bytes for cd_emd_forward and cd_emd_backward (0 for B == 0
 * or invalid sizes); one buffer serves both. */
size_t cd_emd_workspace_bytes(int64_t B, int64_t N, int64_t M);

/*
 * f [B,N], g [B,M]: the potentials, in/out.  warm_start == 0: g starts at 0
 * (f need not be initialised); otherwise the iterations start from the g
 * passed in (f is overwritten by the first update).  cost [B] float32.
 * ws: cd_emd_workspace_bytes(B, N, M) bytes, 256-byte aligned.
 */
cd_status cd_emd_forward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                         float eps_start, float eps_end, int n_iters, int warm_start, float *f,
                         float *g, float *cost, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Backward of sum_b grad_out[b] cost[b] with the plan of (f, g, eps) held
 * fixed (eps: the eps_end of the forward):
 *   gX[b,i] = grad_out[b] sum_j P_ij (x_i - y_j) / C_ij
 *   gY[b,j] = grad_out[b] sum_i P_ij (y_j - x_i) / C_ij   (terms with C_ij = 0 are 0).
 * gX, gY fully overwritten; ws as for cd_emd_forward.
 */
cd_status cd_emd_backward(int64_t B, int64_t N, int64_t M, const float *X, const float *Y,
                          const float *f, const float *g, float eps, const float *grad_out,
                          float *gX, float *gY, void *ws, size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* CD_H */

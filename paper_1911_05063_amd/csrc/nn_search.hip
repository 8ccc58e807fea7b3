// Brute-force nearest-neighbour search in both directions for the batched
// Chamfer distance (Kaolin Sec. 2.5: matching every point of one cloud to
// the nearest point of the other), hand-written for gfx950.
//
// Design (FP32 VALU, not MFMA: the contraction is only 3 deep and the
// difference-of-coordinates form is needed for accuracy on near points):
//  * One wave per work item.  A work item is (direction, batch item, block of
//    64*K queries, split of the targets).  Each lane keeps K queries in
//    registers.
//  * Targets are read with wave-uniform addresses, so they are fetched by the
//    scalar unit into SGPRs and fed to the VALU as broadcast operands: no LDS
//    traffic, no barriers, one s_load per few targets.
//  * Per pair: 3 subtractions, one multiply and two FMAs in the fixed order
//    fma(dz,dz, fma(dy,dy, dx*dx)), and half a v_min3 (two targets per min3).
//  * Deferred argmin: the inner loop tracks only the running minimum.  After
//    every sub-tile of kSubTile targets a lane notes the sub-tile if it
//    lowered the minimum strictly; at the end the noted sub-tile is rescanned
//    to find the lowest index whose distance equals the minimum.  The rescan
//    recomputes the distance with the same instructions, so equality is exact.
//  * Target splits (needed to fill 1024 SIMDs when there are few queries per
//    item) are merged with a 64-bit atomicMin on (float bits << 32 | index),
//    which orders by distance then index because distances are >= +0.
#include "cd_internal.h"

#include <algorithm>

namespace cdk {
namespace {

__device__ __forceinline__ float sq_dist(float qx, float qy, float qz, float tx, float ty,
                                         float tz)
{
    const float dx = qx - tx;
    const float dy = qy - ty;
    const float dz = qz - tz;
    return __builtin_fmaf(dz, dz, __builtin_fmaf(dy, dy, dx * dx));
}

template <int K, int SUB>
__global__ __launch_bounds__(kWave) void nn_search_kernel(NNPlan plan)
{
    static_assert(SUB % 2 == 0, "sub-tile holds target pairs");
    const uint32_t item0 = blockIdx.x;
    const bool second = item0 >= static_cast<uint32_t>(plan.d[0].items);
    const float *P = second ? plan.d[1].P : plan.d[0].P;
    const float *Q = second ? plan.d[1].Q : plan.d[0].Q;
    float *dist = second ? plan.d[1].dist : plan.d[0].dist;
    int32_t *idxo = second ? plan.d[1].idx : plan.d[0].idx;
    unsigned long long *keys = second ? plan.d[1].keys : plan.d[0].keys;
    const int NP = second ? plan.d[1].NP : plan.d[0].NP;
    const int NQ = second ? plan.d[1].NQ : plan.d[0].NQ;
    const uint32_t nqb = second ? plan.d[1].nqb : plan.d[0].nqb;
    const uint32_t nsplit = second ? plan.d[1].nsplit : plan.d[0].nsplit;
    const int chunk = second ? plan.d[1].chunk : plan.d[0].chunk;
    const uint32_t item = second ? item0 - static_cast<uint32_t>(plan.d[0].items) : item0;

    const uint32_t split = item % nsplit;
    const uint32_t rest = item / nsplit;
    const uint32_t qblk = rest % nqb;
    const uint32_t b = rest / nqb;

    const int lane = threadIdx.x;
    const float *Pb = P + static_cast<int64_t>(b) * NP * 3;
    const float *Qb = Q + static_cast<int64_t>(b) * NQ * 3;
    const int q0 = static_cast<int>(qblk) * (kWave * K);

    float qx[K], qy[K], qz[K], best[K];
    int bsub[K];
    const int t0 = static_cast<int>(split) * chunk;
    const int t1 = t0 + min(chunk, NQ - t0);
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int64_t qc = min(static_cast<int64_t>(q0) + k * kWave + lane,
                               static_cast<int64_t>(NP) - 1);
        qx[k] = Pb[3 * qc + 0];
        qy[k] = Pb[3 * qc + 1];
        qz[k] = Pb[3 * qc + 2];
        best[k] = __builtin_inff();
        bsub[k] = t0;
    }

    int j = t0;
    for (; t1 - j >= SUB; j += SUB) {
        const float *T = Qb + 3 * static_cast<int64_t>(j);
        float m[K];
#pragma unroll
        for (int jj = 0; jj < SUB; jj += 2) {
            const float ax = T[3 * jj + 0], ay = T[3 * jj + 1], az = T[3 * jj + 2];
            const float bx = T[3 * jj + 3], by = T[3 * jj + 4], bz = T[3 * jj + 5];
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const float da = sq_dist(qx[k], qy[k], qz[k], ax, ay, az);
                const float db = sq_dist(qx[k], qy[k], qz[k], bx, by, bz);
                m[k] = (jj == 0) ? fminf(da, db) : fminf(m[k], fminf(da, db));
            }
        }
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool lower = m[k] < best[k];
            best[k] = lower ? m[k] : best[k];
            bsub[k] = lower ? j : bsub[k];
        }
    }
    if (j < t1) {  // ragged last sub-tile
        float m[K];
#pragma unroll
        for (int k = 0; k < K; ++k) m[k] = __builtin_inff();
        for (int jj = j; jj < t1; ++jj) {
            const float *T = Qb + 3 * static_cast<int64_t>(jj);
            const float tx = T[0], ty = T[1], tz = T[2];
#pragma unroll
            for (int k = 0; k < K; ++k) m[k] = fminf(m[k], sq_dist(qx[k], qy[k], qz[k], tx, ty, tz));
        }
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool lower = m[k] < best[k];
            best[k] = lower ? m[k] : best[k];
            bsub[k] = lower ? j : bsub[k];
        }
    }

    // Recover the lowest index attaining the minimum inside the noted sub-tile.
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int64_t qi = static_cast<int64_t>(q0) + k * kWave + lane;
        if (qi < NP) {
            const int jb = bsub[k];
            const int je = jb + min(SUB, t1 - jb);
            int found = -1;
            for (int jj = je - 1; jj >= jb; --jj) {
                const float *T = Qb + 3 * static_cast<int64_t>(jj);
                const float d = sq_dist(qx[k], qy[k], qz[k], T[0], T[1], T[2]);
                found = (d == best[k]) ? jj : found;
            }
            const int64_t o = static_cast<int64_t>(b) * NP + qi;
            if (nsplit == 1) {
                dist[o] = best[k];
                idxo[o] = found;
            } else {
                const unsigned long long key =
                    (static_cast<unsigned long long>(__float_as_uint(best[k])) << 32) |
                    static_cast<uint32_t>(found);
                atomicMin(keys + o, key);
            }
        }
    }
}

__global__ void fill_keys_kernel(unsigned long long *keys, int64_t n)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) keys[i] = ~0ull;
}

__global__ void unpack_keys_kernel(const unsigned long long *keys, float *dist, int32_t *idx,
                                   int64_t n)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) {
        const unsigned long long key = keys[i];
        dist[i] = __uint_as_float(static_cast<uint32_t>(key >> 32));
        idx[i] = static_cast<int32_t>(static_cast<uint32_t>(key));
    }
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

WsLayout workspace_layout(int64_t B, int64_t N, int64_t M)
{
    auto up = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
    WsLayout w;
    w.keys_xy = 0;
    w.keys_yx = up(static_cast<size_t>(B * N) * 8);
    w.total = w.keys_yx + up(static_cast<size_t>(B * M) * 8);
    return w;
}

void make_plan(NNPlan &plan, int64_t B, int64_t N, int64_t M, int cu_count)
{
    const int64_t qpb = static_cast<int64_t>(kWave) * kQueriesPerLane;
    const int64_t NPs[2] = {N, M}, NQs[2] = {M, N};
    // Equal-sized work items: about 4 waves per SIMD (4 SIMDs per CU), with
    // at least 512 targets per split so the rescan stays a small fraction.
    double work = 0.0;
    for (int d = 0; d < 2; ++d) work += static_cast<double>(B) * ceil_div(NPs[d], qpb) * NQs[d];
    const double target_items = static_cast<double>(std::max(cu_count, 1)) * 16.0;
    int64_t chunk = static_cast<int64_t>(work / target_items) + 1;
    chunk = std::max<int64_t>(chunk, 512);
    for (int d = 0; d < 2; ++d) {
        NNDir &D = plan.d[d];
        D.NP = static_cast<int32_t>(NPs[d]);
        D.NQ = static_cast<int32_t>(NQs[d]);
        D.nqb = static_cast<int32_t>(ceil_div(NPs[d], qpb));
        int64_t ns = ceil_div(NQs[d], chunk);
        int64_t c = ceil_div(ceil_div(NQs[d], ns), kSubTile) * kSubTile;
        ns = ceil_div(NQs[d], c);
        D.nsplit = static_cast<int32_t>(ns);
        D.chunk = static_cast<int32_t>(c);
        D.pad = 0;
        D.items = B * D.nqb * ns;
    }
    plan.B = B;
}

hipError_t launch_forward(const NNPlan &plan, hipStream_t stream)
{
    const int64_t n[2] = {plan.B * plan.d[0].NP, plan.B * plan.d[1].NP};
    for (int d = 0; d < 2; ++d) {
        if (plan.d[d].nsplit > 1) {
            fill_keys_kernel<<<static_cast<uint32_t>(ceil_div(n[d], 256)), 256, 0, stream>>>(
                plan.d[d].keys, n[d]);
        }
    }
    const int64_t items = plan.d[0].items + plan.d[1].items;
    nn_search_kernel<kQueriesPerLane, kSubTile>
        <<<static_cast<uint32_t>(items), kWave, 0, stream>>>(plan);
    for (int d = 0; d < 2; ++d) {
        if (plan.d[d].nsplit > 1) {
            unpack_keys_kernel<<<static_cast<uint32_t>(ceil_div(n[d], 256)), 256, 0, stream>>>(
                plan.d[d].keys, plan.d[d].dist, plan.d[d].idx, n[d]);
        }
    }
    return hipGetLastError();
}

}  // namespace cdk

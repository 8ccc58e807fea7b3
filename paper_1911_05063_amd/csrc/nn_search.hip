// Brute-force nearest-neighbour search in both directions for the batched
// Chamfer distance (Kaolin Sec. 2.5: every point of one cloud is matched to
// the nearest point of the other), hand-written for gfx950.
//
// Fused symmetric search: every squared distance d(x_i, y_j) is evaluated
// once and feeds both minima, x_i's nearest y (a row of the distance matrix)
// and y_j's nearest x (a column).
//
//  * FP32 VALU, not MFMA: the contraction is only 3 deep, and the difference
//    form fma(dz,dz, fma(dy,dy, dx*dx)) with d = x - y is needed for accuracy
//    on near points (the |x|^2 + |y|^2 - 2x.y expansion cancels).
//  * Tiles: a workgroup of kWaves waves owns a query group of
//    kWaves*64*kQ x-points (kQ per lane, in registers, lane-major: lane l of
//    the group holds x-points l*kQ .. l*kQ+kQ-1) and a block of TB y-points.
//    The y-points are read with wave-uniform addresses, so the scalar unit
//    loads them into SGPRs and the VALU takes them as broadcast operands.
//  * Rows: per x-point a running minimum over the block, kept with v_min3
//    (two targets per instruction).  The argmin is deferred: a lane only
//    notes the batch of kBatch targets that last lowered its minimum strictly.
//  * Columns: per lane and target, the minimum over the lane's kQ x-points;
//    after each batch these partials are transposed through LDS so that each
//    lane reduces one target's values (half a wave each), and the lowest
//    lane holding the minimum is found.  The 4 waves combine through a 64-bit
//    LDS atomicMin on (distance bits << 32 | lane), which orders by distance
//    then lane because distances are >= +0.
//  * Target blocks: TB targets (256..512), aiming at about four rounds of
//    resident workgroups.  In a launch of one to eight rounds, the last
//    targets of every group go to small blocks (128) at the end of the grid,
//    so that the final round is filled with short tiles.  A problem too small
//    for one round gets blocks of 32..512 targets, about one round of tiles.
//  * Each tile folds its packed (distance, batch start) key per x-point and
//    (distance, lane) key per y-point into one key per point in the workspace
//    with a 64-bit global atomicMin (the arrays are filled with ~0 first), so
//    the workspace is 8 B (N + M) bytes whatever the tiling.  Distances are
//    >= +0, so the unsigned key order is distance first, then batch (lane):
//    the minimum names the first batch (lowest lane) that reaches the minimum
//    distance.  A merge kernel then recovers the exact lowest index by
//    recomputing the kBatch candidate targets of a row (8 lanes per x-point)
//    or the kQ candidate x-points of a column with the same instructions, so
//    equality is exact.
#include "cd_internal.h"

#include <algorithm>
#include <mutex>

namespace cdk {
namespace {

constexpr int kQ = 8;               // x-points per lane
constexpr int kWaves = 4;           // waves per workgroup
constexpr int kThreads = kWaves * kWave;
constexpr int kBatch = 32;          // targets per batch (row sub-tile, column batch)
constexpr int kLdsRow = kWave + 4;  // padded LDS row (floats) of the column transpose
constexpr int kMaxTB = 512;         // targets per block at most (LDS column keys)
constexpr int kMinTB = 256;         // targets per block at least
constexpr int64_t kTargetTiles = 4096;  // workgroups to aim for (4 rounds of 4 per CU on MI355X)
constexpr int64_t kSlots = 256 * 4;     // workgroups resident at once: 256 CUs x 4
constexpr int kSmallTB = 128;           // targets per block of the final, small tiles
constexpr int64_t kSmallRounds = 8;     // small tiles only for launches of 1 to 8 rounds
constexpr int64_t kSmallLaunchTiles = 1024;  // tiles to aim for below one round
constexpr int kMergeThreads = 256;
constexpr int64_t kXcds = 8;        // accelerator complex dies of an MI355X

__device__ __forceinline__ float sq_dist(float qx, float qy, float qz, float tx, float ty,
                                         float tz)
{
    const float dx = qx - tx;
    const float dy = qy - ty;
    const float dz = qz - tz;
    return __builtin_fmaf(dz, dz, __builtin_fmaf(dy, dy, dx * dx));
}

// v_min3_f32 on values that are never NaN: no canonicalisation is needed.
__device__ __forceinline__ float min3f(float a, float b, float c)
{
    float r;
    asm("v_min3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

__device__ __forceinline__ float min2f(float a, float b)
{
    float r;
    asm("v_min_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

__device__ __forceinline__ unsigned long long pack_key(float d, uint32_t low)
{
    return (static_cast<unsigned long long>(__float_as_uint(d)) << 32) | low;
}

struct KernelArgs {
    const float *X;
    const float *Y;
    unsigned long long *rowkey;  // [B, N]  min (distance, batch start) per x-point
    unsigned long long *colkey;  // [B, M]  min (distance, x lane) per y-point
    int32_t N, M, nQG, nTB, TB;
    int32_t TS, nBig;   // small blocks of TS targets follow nBig blocks of TB
    int32_t pad;
    int64_t B;
};

// One batch of kBatch targets starting at j.  FULL: the whole batch lies in
// [j, t1); otherwise the targets past t1 repeat target t1-1 (never chosen over
// it: equal distances resolve to the lower index) and write no column key.
template <bool FULL>
__device__ __forceinline__ void search_batch(const float *__restrict__ Yb, int j, int t1,
                                             const float (&qx)[kQ], const float (&qy)[kQ],
                                             const float (&qz)[kQ], float (&best)[kQ],
                                             int (&bsub)[kQ], float *lds, int lane,
                                             unsigned long long *colkeys, int t0,
                                             uint32_t lane0)
{
    float m[kQ];
    float c[kBatch];
#pragma unroll
    for (int jj = 0; jj < kBatch; jj += 2) {
        int ja = j + jj, jb = j + jj + 1;
        if (!FULL) {
            ja = min(ja, t1 - 1);
            jb = min(jb, t1 - 1);
        }
        const float *ta = Yb + 3 * static_cast<int64_t>(ja);  // 64-bit: 3*M may pass 2^31
        const float *tb = Yb + 3 * static_cast<int64_t>(jb);
        const float ax = ta[0], ay = ta[1], az = ta[2];
        const float bx = tb[0], by = tb[1], bz = tb[2];
        float da[kQ], db[kQ];
#pragma unroll
        for (int k = 0; k < kQ; ++k) {
            da[k] = sq_dist(qx[k], qy[k], qz[k], ax, ay, az);
            db[k] = sq_dist(qx[k], qy[k], qz[k], bx, by, bz);
            m[k] = (jj == 0) ? min2f(da[k], db[k]) : min3f(m[k], da[k], db[k]);
        }
        float ca = min3f(da[0], da[1], da[2]);
        float cb = min3f(db[0], db[1], db[2]);
#pragma unroll
        for (int k = 3; k + 1 < kQ; k += 2) {
            ca = min3f(ca, da[k], da[k + 1]);
            cb = min3f(cb, db[k], db[k + 1]);
        }
        if ((kQ - 3) % 2 == 1) {
            ca = min2f(ca, da[kQ - 1]);
            cb = min2f(cb, db[kQ - 1]);
        }
        c[jj] = ca;
        c[jj + 1] = cb;
    }
    // Rows: note the batch if it lowered the minimum strictly.
#pragma unroll
    for (int k = 0; k < kQ; ++k) {
        const bool lower = m[k] < best[k];
        best[k] = lower ? m[k] : best[k];
        bsub[k] = lower ? j : bsub[k];
    }

    // Columns: transpose through LDS, lds[t * kLdsRow + lane] = c[t].  LDS
    // operations of one wave execute in order, so no barrier is needed.
#pragma unroll
    for (int t = 0; t < kBatch; ++t) lds[t * kLdsRow + lane] = c[t];
    __builtin_amdgcn_wave_barrier();
    // Reducer lane r: target t = r % 32 over source lanes 32h .. 32h+31, h = r / 32.
    const int t = lane & (kBatch - 1);
    const int h = lane >> 5;
    const float4 *row = reinterpret_cast<const float4 *>(lds + t * kLdsRow + h * 32);
    float g[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float4 q = row[i];
        g[i] = min2f(min3f(q.x, q.y, q.z), q.w);
    }
    const float mn = min2f(min3f(min3f(g[0], g[1], g[2]), g[3], g[4]), min3f(g[5], g[6], g[7]));
    int fg = 7;
#pragma unroll
    for (int i = 6; i >= 0; --i) fg = (g[i] == mn) ? i : fg;
    const float4 w = row[fg];
    int fi = 3;
    fi = (w.z == mn) ? 2 : fi;
    fi = (w.y == mn) ? 1 : fi;
    fi = (w.x == mn) ? 0 : fi;
    const int first = 4 * fg + fi;  // lowest source lane (within the half) holding mn
    __builtin_amdgcn_wave_barrier();
    // Lanes r and r + 32 hold the two halves of target r: combine them.
    const auto sm = __builtin_amdgcn_permlane32_swap(__float_as_uint(mn), __float_as_uint(mn),
                                                     false, false);
    const auto sf = __builtin_amdgcn_permlane32_swap(static_cast<uint32_t>(first),
                                                     static_cast<uint32_t>(first), false, false);
    if (lane < kBatch) {
        const float m0 = __uint_as_float(sm[0]), m1 = __uint_as_float(sm[1]);
        const bool lo = m0 <= m1;
        const uint32_t src = lo ? sf[0] : 32u + sf[1];
        const int jt = j + lane;
        if (FULL || jt < t1) atomicMin(colkeys + (jt - t0), pack_key(lo ? m0 : m1, lane0 + src));
    }
}

// At most 128 VGPRs (4 waves per SIMD) and 39 KB of LDS: 4 workgroups per CU.
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 8)))
void search_kernel(KernelArgs a)
{
    __shared__ unsigned long long colkeys[kMaxTB];
    __shared__ __attribute__((aligned(16))) float ldsbuf[kWaves][kBatch * kLdsRow];
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    // The grid holds every (item, group) tile of the nBig large blocks first,
    // blockIdx.x = (b * nQG + qg) * nBig + tb, then those of the small blocks,
    // which the dispatcher hands out last and so fill the final round.
    const uint32_t nbig = static_cast<uint32_t>(a.nBig);
    const uint32_t big_tiles = static_cast<uint32_t>(a.B) * a.nQG * nbig;
    uint32_t tb, rest;
    if (blockIdx.x < big_tiles) {
        tb = blockIdx.x % nbig;
        rest = blockIdx.x / nbig;
    } else {
        const uint32_t k = blockIdx.x - big_tiles, nsmall = static_cast<uint32_t>(a.nTB) - nbig;
        tb = nbig + k % nsmall;
        rest = k / nsmall;
    }
    const uint32_t qg = rest % static_cast<uint32_t>(a.nQG);
    const uint32_t b = rest / static_cast<uint32_t>(a.nQG);
    const bool large = tb < nbig;
    const int t0 = large ? static_cast<int>(tb) * a.TB
                         : a.nBig * a.TB + static_cast<int>(tb - nbig) * a.TS;
    const int t1 = t0 + min(large ? a.TB : a.TS, a.M - t0);
    const float *Xb = a.X + static_cast<int64_t>(b) * a.N * 3;
    const float *Yb = a.Y + static_cast<int64_t>(b) * a.M * 3;

    for (int t = threadIdx.x; t < t1 - t0; t += kThreads) colkeys[t] = ~0ull;

    const uint32_t lane0 = (qg * kWaves + wave) * kWave;  // first lane of this wave in the item
    // x-point index of this lane's first x-point; below N + kThreads*kQ < 2^32.
    const uint32_t xbase = (lane0 + static_cast<uint32_t>(lane)) * kQ;
    const uint32_t nx = static_cast<uint32_t>(a.N);
    float qx[kQ], qy[kQ], qz[kQ], best[kQ];
    int bsub[kQ];
#pragma unroll
    for (int k = 0; k < kQ; ++k) {
        // x-points past N repeat x-point N-1, which has a lower index.
        const int64_t qi = min(xbase + k, nx - 1);
        qx[k] = Xb[3 * qi + 0];
        qy[k] = Xb[3 * qi + 1];
        qz[k] = Xb[3 * qi + 2];
        best[k] = __builtin_inff();
        bsub[k] = t0;
    }
    __syncthreads();

    float *lds = ldsbuf[wave];
    int j = t0;
    for (; t1 - j >= kBatch; j += kBatch)
        search_batch<true>(Yb, j, t1, qx, qy, qz, best, bsub, lds, lane, colkeys, t0, lane0);
    if (j < t1)
        search_batch<false>(Yb, j, t1, qx, qy, qz, best, bsub, lds, lane, colkeys, t0, lane0);

    // Rows: this wave's kWave*kQ keys go through its LDS buffer (free after the
    // last batch; a wave's LDS operations execute in order) so that
    // consecutive lanes update consecutive x-points: 512 contiguous bytes per
    // atomic instruction instead of a 64-byte stride.
    unsigned long long *kl = reinterpret_cast<unsigned long long *>(lds);
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int k = 0; k < kQ; ++k)
        kl[lane * kQ + k] = pack_key(best[k], static_cast<uint32_t>(bsub[k]));
    __builtin_amdgcn_wave_barrier();
    unsigned long long *rp = a.rowkey + static_cast<int64_t>(b) * a.N;
    const uint32_t wx = lane0 * kQ;
#pragma unroll
    for (int k = 0; k < kQ; ++k) {
        const uint32_t p = k * kWave + lane;
        if (wx + p < nx) atomicMin(rp + wx + p, kl[p]);
    }
    __syncthreads();
    unsigned long long *cp = a.colkey + static_cast<int64_t>(b) * a.M;
    for (int t = threadIdx.x; t < t1 - t0; t += kThreads) atomicMin(cp + t0 + t, colkeys[t]);
}

// Every key of the workspace to ~0 (no key yet), before the search folds in
// its tiles.  A kernel rather than a memset, so that callers may capture the
// forward in a graph.
constexpr int kFillThreads = 256;
constexpr int64_t kFillBlocks = 2048;

__global__ __launch_bounds__(kFillThreads) void key_fill_kernel(unsigned long long *k, int64_t n)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kFillThreads;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kFillThreads + threadIdx.x; i < n;
         i += stride)
        k[i] = ~0ull;
}

// One point's coordinates: 12-byte loads (dword-aligned vector loads).
struct P3 {
    float x, y, z;
};

// Merge blocks: per item, ceil(N / kMergeThreads) blocks of rows and then
// ceil(M / kMergeThreads) blocks of columns.  Workgroups are dispatched to
// the 8 XCDs round-robin; when B is a multiple of 8, block i runs block
// (i / 8) of the items b = i % 8 (mod 8), so that one XCD's L2 holds the
// clouds of its items the rescans read (2 items of 16384 points per XCD at
// B = 16); otherwise items follow one another.
__host__ __device__ __forceinline__ int64_t merge_blocks_per_item(int64_t N, int64_t M)
{
    return (N + kMergeThreads - 1) / kMergeThreads + (M + kMergeThreads - 1) / kMergeThreads;
}

__host__ __device__ __forceinline__ bool merge_by_xcd(int64_t B) { return B % kXcds == 0; }

// A wave of rows reads the keys of its 64 x-points (one per lane), then
// rescans their candidate batches 8 x-points at a time: 8 lanes per x-point,
// lane c taking targets c, c + 8, c + 16, c + 24 of the batch (so that one
// load instruction reads 8 consecutive targets of each of 8 batches), and the
// lowest matching index over the 8 lanes.  The rescan loads are clamped into
// the cloud instead of guarded, so that two rounds' loads are in flight
// together.  Columns likewise, 8 lanes per y-point over the kQ x-points of its
// key's lane.  The keys are read once: non-temporal loads keep them from
// evicting the coordinates that the rescans read.

__global__ __launch_bounds__(kMergeThreads) void merge_kernel(KernelArgs a, float *dxy,
                                                              int32_t *ixy, float *dyx,
                                                              int32_t *iyx)
{
    const int64_t pb = merge_blocks_per_item(a.N, a.M);
    const int64_t rb = (a.N + kMergeThreads - 1) / kMergeThreads;
    int64_t b, kb;   // item, block within the item
    if (merge_by_xcd(a.B)) {
        const int64_t j = blockIdx.x / kXcds;
        b = static_cast<int64_t>(blockIdx.x % kXcds) + kXcds * (j / pb);
        kb = j % pb;
    } else {
        b = blockIdx.x / pb;
        kb = blockIdx.x % pb;
    }
    if (b >= a.B) return;
    if (kb < rb) {
        // A block of rows of item b: whole waves, every lane of a wave here.
        const int lane = threadIdx.x % kWave;
        const int64_t ibase = kb * kMergeThreads + (threadIdx.x - lane);   // the wave's first row
        const int64_t i = ibase + lane;
        const bool mine = i < a.N;
        float val = 0.0f, px = 0.0f, py = 0.0f, pz = 0.0f;
        int js = a.M;  // candidate batch start (M: none)
        if (mine) {
            const unsigned long long key = __builtin_nontemporal_load(a.rowkey + b * a.N + i);
            val = __uint_as_float(static_cast<uint32_t>(key >> 32));
            js = static_cast<int>(static_cast<uint32_t>(key));
            js = (js < 0 || js >= a.M) ? a.M : js;  // no key: nothing to rescan
            const P3 x = reinterpret_cast<const P3 *>(a.X)[b * a.N + i];
            px = x.x;
            py = x.y;
            pz = x.z;
        }
        const P3 *Yb = reinterpret_cast<const P3 *>(a.Y + b * a.M * 3);
        const int sub = lane & 7;
        constexpr int kR = 2;  // rescan rounds whose loads are issued together
        for (int r0 = 0; r0 < 8; r0 += kR) {
            float v[kR], qx[kR], qy[kR], qz[kR];
            int je[kR], jb[kR];
            P3 ty[kR][4];
#pragma unroll
            for (int r = 0; r < kR; ++r) {
                const int src = 8 * (r0 + r) + (lane >> 3);
                v[r] = __shfl(val, src, kWave);
                const int j0 = __shfl(js, src, kWave);
                qx[r] = __shfl(px, src, kWave);
                qy[r] = __shfl(py, src, kWave);
                qz[r] = __shfl(pz, src, kWave);
                // A row past N has j0 = M: every load is target M-1 and no
                // candidate qualifies.
                je[r] = j0 + min(kBatch, a.M - j0);
                const int jl = max(je[r] - 1, 0);
                jb[r] = j0 + sub;
#pragma unroll
                for (int q = 0; q < 4; ++q) ty[r][q] = Yb[min(jb[r] + 8 * q, jl)];
            }
            int cand[kR];
#pragma unroll
            for (int r = 0; r < kR; ++r) {
                cand[r] = 0x7fffffff;
#pragma unroll
                for (int q = 3; q >= 0; --q) {
                    const float d =
                        sq_dist(qx[r], qy[r], qz[r], ty[r][q].x, ty[r][q].y, ty[r][q].z);
                    cand[r] = (jb[r] + 8 * q < je[r] && d == v[r]) ? jb[r] + 8 * q : cand[r];
                }
#pragma unroll
                for (int off = 1; off < 8; off <<= 1)
                    cand[r] = min(cand[r], __shfl_xor(cand[r], off, kWave));
            }
#pragma unroll
            for (int r = 0; r < kR; ++r) {
                const int64_t ip = ibase + 8 * (r0 + r) + (lane >> 3);
                if (sub == 0 && ip < a.N) {
                    dxy[b * a.N + ip] = v[r];
                    ixy[b * a.N + ip] = cand[r] == 0x7fffffff ? -1 : cand[r];
                }
            }
        }
    } else {
        // A block of columns of item b, rescanned like the rows: a wave takes
        // its 64 y-points' keys, then 8 y-points at a time with 8 lanes each,
        // lane c recomputing candidate i0 + c of its y-point, so that one load
        // instruction reads 8 runs of kQ consecutive x-points (coalesced); the
        // lowest matching index by a 3-step shuffle minimum.
        static_assert(kQ == 8, "one candidate x-point per lane of an 8-lane group");
        const int lane = threadIdx.x % kWave;
        const int64_t jbase = (kb - rb) * kMergeThreads + (threadIdx.x - lane);   // the wave's first column
        const int64_t jy = jbase + lane;
        const bool mine = jy < a.M;
        float val = 0.0f, yx = 0.0f, yy = 0.0f, yz = 0.0f;
        int i0 = a.N;   // first candidate (N: none)
        if (mine) {
            const unsigned long long key = __builtin_nontemporal_load(a.colkey + b * a.M + jy);
            val = __uint_as_float(static_cast<uint32_t>(key >> 32));
            const int64_t c0 = static_cast<int64_t>(static_cast<uint32_t>(key)) * kQ;
            i0 = c0 < a.N ? static_cast<int>(c0) : a.N;   // no key: nothing to rescan
            const P3 y = reinterpret_cast<const P3 *>(a.Y)[b * a.M + jy];
            yx = y.x;
            yy = y.y;
            yz = y.z;
        }
        const P3 *Xb = reinterpret_cast<const P3 *>(a.X + b * a.N * 3);
        const int sub = lane & 7;
        float v[8], qx[8], qy[8], qz[8];
        int ic[8], ie[8];
        P3 tx[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int src = 8 * r + (lane >> 3);
            v[r] = __shfl(val, src, kWave);
            const int c0 = __shfl(i0, src, kWave);
            qx[r] = __shfl(yx, src, kWave);
            qy[r] = __shfl(yy, src, kWave);
            qz[r] = __shfl(yz, src, kWave);
            // A column past M or without a key has c0 = N: the load is
            // x-point N-1 and no candidate qualifies.
            ie[r] = c0 + min(kQ, a.N - c0);
            ic[r] = c0 + sub;
            tx[r] = Xb[min(ic[r], max(ie[r] - 1, 0))];
        }
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const float d = sq_dist(tx[r].x, tx[r].y, tx[r].z, qx[r], qy[r], qz[r]);
            int cand = (ic[r] < ie[r] && d == v[r]) ? ic[r] : 0x7fffffff;
#pragma unroll
            for (int off = 1; off < 8; off <<= 1) cand = min(cand, __shfl_xor(cand, off, kWave));
            const int64_t jp = jbase + 8 * r + (lane >> 3);
            if (sub == 0 && jp < a.M) {
                dyx[b * a.M + jp] = v[r];
                iyx[b * a.M + jp] = cand == 0x7fffffff ? -1 : cand;
            }
        }
    }
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct WsOffsets {
    size_t rowkey, colkey, total;
};

WsOffsets ws_offsets(const FwdPlan &p)
{
    auto up = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
    WsOffsets w;
    w.rowkey = 0;
    w.colkey = up(static_cast<size_t>(p.B) * p.N * 8);
    w.total = w.colkey + up(static_cast<size_t>(p.B) * p.M * 8);
    return w;
}

}  // namespace

FwdPlan plan_forward(int64_t B, int64_t N, int64_t M)
{
    FwdPlan p;
    p.B = B;
    p.N = static_cast<int32_t>(N);
    p.M = static_cast<int32_t>(M);
    const int64_t per_group = static_cast<int64_t>(kThreads) * kQ;
    p.nQG = static_cast<int32_t>(ceil_div(N, per_group));
    // Split the targets until there are about kTargetTiles tiles, keeping
    // blocks between kMinTB and kMaxTB targets and a multiple of kBatch.
    const int64_t groups = std::max<int64_t>(1, B * p.nQG);
    const int64_t want_blocks = ceil_div(kTargetTiles, groups);
    int64_t TB = ceil_div(ceil_div(M, want_blocks), kBatch) * kBatch;
    TB = std::min<int64_t>(std::max<int64_t>(TB, kMinTB), kMaxTB);
    int64_t blocks = ceil_div(M, TB);
    if (groups * blocks < kSlots) {
        // Not one round even with kMinTB: smaller blocks (down to one batch)
        // until there are about one round of tiles (four waves per SIMD).
        // More and smaller tiles measured slower: per-tile set-up and key
        // updates grow faster than the parallelism helps.
        const int64_t ts = std::max<int64_t>(
            kBatch,
            ceil_div(ceil_div(M, ceil_div(kSmallLaunchTiles, groups)), kBatch) * kBatch);
        if (ts < TB) {
            TB = ts;
            blocks = ceil_div(M, TB);
        }
    }
    p.TB = static_cast<int32_t>(TB);
    p.TS = kSmallTB;
    if (TB > kSmallTB && groups * blocks >= kSlots && groups * blocks <= kSmallRounds * kSlots) {
        // A launch of one to a few rounds: the last targets of every group go
        // to small blocks, about a quarter round of resident workgroups' worth
        // of work.
        // Dispatched last, they even out the end of the launch (tiles of one
        // size finish unevenly and leave CUs idle while the final ones run).
        const int64_t small = std::min<int64_t>(
            M, ceil_div(ceil_div(kSlots / 4 * TB, groups), kSmallTB) * kSmallTB);
        p.nBig = static_cast<int32_t>((M - small) / TB);
        p.nTB = p.nBig +
                static_cast<int32_t>(ceil_div(M - static_cast<int64_t>(p.nBig) * TB, kSmallTB));
    } else {
        // Less than a round (every tile runs at once) or many rounds (the end
        // matters little, the extra row keys more): one block size.
        p.nBig = static_cast<int32_t>(blocks);
        p.nTB = p.nBig;
    }
    return p;
}

size_t forward_workspace_bytes(const FwdPlan &p) { return ws_offsets(p).total; }

int64_t forward_tiles(const FwdPlan &p) { return p.B * p.nQG * p.nTB; }

// Workspace of cd_forward_noalloc: a file-scope device array, one per GPU the
// library runs on, held until the process ends.  Host code never passes the
// array's name to a kernel (on the host it is a stand-in, not a device
// address): forward_scratch() looks up each device's address once, with that
// device current, and every use goes through that pointer.
__device__ __align__(256) unsigned long long scratch[kForwardScratchBytes / 8];

namespace {
constexpr int kMaxDevices = 256;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];
}  // namespace

hipError_t forward_scratch(hipStream_t stream, void **ptr)
{
    *ptr = nullptr;
    int dev = 0;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        int cur = 0;
        e = hipGetDevice(&cur);
        if (e != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        const hipError_t back = cur != dev ? hipSetDevice(cur) : hipSuccess;
        if (e != hipSuccess) return e;
        if (back != hipSuccess) return back;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

hipError_t launch_forward(const FwdPlan &p, const FwdArgs &f, hipStream_t stream)
{
    const WsOffsets w = ws_offsets(p);
    KernelArgs a;
    a.X = f.X;
    a.Y = f.Y;
    a.rowkey = reinterpret_cast<unsigned long long *>(static_cast<char *>(f.ws) + w.rowkey);
    a.colkey = reinterpret_cast<unsigned long long *>(static_cast<char *>(f.ws) + w.colkey);
    a.N = p.N;
    a.M = p.M;
    a.nQG = p.nQG;
    a.nTB = p.nTB;
    a.TB = p.TB;
    a.TS = p.TS;
    a.nBig = p.nBig;
    a.pad = 0;
    a.B = p.B;
    // The two key arrays and the padding between them: one fill.
    const int64_t nkeys = static_cast<int64_t>(w.total / 8);
    key_fill_kernel<<<static_cast<uint32_t>(std::min(ceil_div(nkeys, kFillThreads), kFillBlocks)),
                      kFillThreads, 0, stream>>>(a.rowkey, nkeys);
    search_kernel<<<static_cast<uint32_t>(forward_tiles(p)), kThreads, 0, stream>>>(a);
    merge_kernel<<<static_cast<uint32_t>(p.B * merge_blocks_per_item(p.N, p.M)), kMergeThreads, 0,
                   stream>>>(a, f.dist_xy, f.idx_xy, f.dist_yx, f.idx_yx);
    return hipGetLastError();
}

}  // namespace cdk

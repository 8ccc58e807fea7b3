// Backward of the Chamfer loss (Kaolin Sec. 2.5: Chamfer distance as a loss
// that supervises networks) for the neighbours the forward chose.
//
// d dist_xy[i] / d x_i = 2 (x_i - y_j) and d dist_xy[i] / d y_j = -2 (x_i - y_j)
// for j = idx_xy[i]; symmetrically for dist_yx.  So
//   gX[i] = 2 g_xy(i) (x_i - y_{idx_xy[i]}) - sum_{j: idx_yx[j] = i} 2 g_yx(j) (y_j - x_i)
//   gY[j] = 2 g_yx(j) (y_j - x_{idx_yx[j]}) - sum_{i: idx_xy[i] = j} 2 g_xy(i) (x_i - y_j)
// The first term is the point's own; the sum scatters the other cloud's
// ("senders'") terms onto their neighbours ("receivers").
//
// The scatter sums are exact and therefore bitwise reproducible: every
// contribution (a float32 product) is rounded to a 64-bit fixed-point integer
// on a grid 2^-k and the integers are added, so their order does not matter.
// k keeps every receiver's sum below 2^62 (fixed_point.h), from a bound on
// the largest term:
//  * "local" sides (senders fit one pass and one chunk): the largest term the
//    workgroup itself queued, so k is per slice of receivers and needs no
//    extra pass; the grid is about 2^-61 * (terms queued) * (largest term).
//  * other sides: bound_kernel's per-item bound, shared by all chunks: per
//    block of 1024 points of an item, the bounding box of both clouds and the
//    largest |dL/d dist|; every term component is at most 2 |g| times the
//    box's largest extent; the grid is about 2^-61 * (cloud size) times that.
// Either grid is far below the float32 rounding of the terms.
//  * scatter_kernel: a workgroup owns a slice of up to 2048 receivers (256..2048:
//    small problems take smaller slices, more workgroups) of one cloud and
//    item and a chunk of the other cloud's senders.  Per pass of 16384
//    senders it loads their neighbour indices (32 per thread in 16-byte
//    loads, all in flight at once), queues the senders that land in its
//    slice in LDS (a wave prefix sum from ballots and one LDS atomic per
//    wave), and then evaluates only the queued terms, adding them to LDS int64
//    accumulators (ds_add_u64).  With one chunk per item it then writes own +
//    scatter directly (the own terms' loads go out with the first ones, and
//    nothing waits on them before the output); otherwise the slice goes to
//    the workspace.
//  * finalize_kernel: per receiver, the chunks' integer partials summed
//    exactly, scaled back, plus the own term (in double), rounded once.
// Senders are split into chunks only on a side whose scan is much longer than
// the other's (a few receivers, many senders: one cloud much larger).
//
// Bucketed path: every slice workgroup above reads all of its item's sender
// indices, so index reads grow as (senders) x (slices), and senders beyond one
// pass need the bound pass and chunk partials.  Where a side's senders exceed
// one pass, or the scans would read more than 64 MB (B = 8 clouds of 65536
// points: 134 MB; two of 2^20: 4.3 GB), and every side has at most 1024
// slices, at most 2^21 senders and on average at most 16384 senders per
// slice:
//  * bucket_kernel: per chunk of 2048 senders, counting-sorts them by the
//    receiver slice of their neighbour (LDS histogram, prefix sum, LDS
//    cursors) and writes the chunk's entries (sender offset in the chunk,
//    receiver offset in the slice) grouped by slice, plus the chunk's slice
//    offsets;
//  * slice_kernel: per slice, reads each chunk's segment for the slice, so
//    every sender index is read once in all; the slice holds all of its
//    terms, so the shift always comes from its own largest term (no bound
//    pass, no chunk partials) and own + scatter are written directly.
// The order of entries within a segment depends on the LDS atomics, which
// does not change the exact sums.
// A point whose neighbour index lies outside the other cloud contributes
// nothing (its own term is 0 and it scatters nothing).
#include <algorithm>

#include "cd_internal.h"
#include "fixed_point.h"

namespace cdk {
namespace {

constexpr int kBlock = 512;                 // threads of a scatter workgroup
constexpr int kSliceBits = 11;
constexpr int kSlice = 1 << kSliceBits;     // receivers per workgroup, at most
constexpr int kMinSlice = 256;              // at least (small problems: more workgroups)
constexpr int64_t kCUs = 256;
constexpr int kIdx = 32;                    // sender indices per thread per pass
constexpr int64_t kPass = static_cast<int64_t>(kBlock) * kIdx;   // senders per pass
constexpr int kOwn = kSlice / kBlock;       // receivers per thread (own terms, output)
constexpr int kHold = 8;                    // queued terms per thread kept in registers
constexpr uint32_t kXcds = 8;               // accelerator complex dies of an MI355X
static_assert(kSlice % kBlock == 0, "receivers must divide evenly among the threads");
static_assert((kPass << kSliceBits) <= (int64_t{1} << 32), "queue entry must fit 32 bits");
constexpr int kBoundThreads = 1024;
constexpr int kBoundPer = 1;                // points of each cloud per thread
constexpr int kBoundBlock = kBoundThreads * kBoundPer;   // points per bound block
constexpr int kBound = 8;                   // per block: -min xyz, max xyz, max|g_xy|, max|g_yx|
constexpr int kThreads = 256;
constexpr int kBucketThreads = 256;         // threads of a bucket workgroup
constexpr int kBucketPer = 8;               // senders per thread
constexpr int kChunk = kBucketThreads * kBucketPer;   // senders per bucket chunk
constexpr int kMaxBucketSlices = 1024;      // slices per item and side (LDS histogram)
constexpr int kMaxBucketChunks = 1024;      // chunks per item and side (LDS segment table)
constexpr int64_t kMaxBucketShare = 16384;  // senders per slice on average, at most
constexpr int64_t kMinBucketScanBytes = int64_t{64} << 20;  // index bytes the slice scans would read
static_assert(kChunk == 2048 && (kChunk << kSliceBits) <= (int64_t{1} << 32),
              "bucket entry must fit 32 bits");
static_assert(kMaxBucketSlices % kBucketThreads == 0 && kMaxBucketChunks == 2 * kBlock,
              "scan layouts");

// Four consecutive int32 (a 16-byte load on dword alignment).
struct I4 {
    int32_t x, y, z, w;
};

struct BwdArgs {
    const float *gxy;   // [B] (per item) or [B, N] (pointwise)
    const float *gyx;   // [B] or [B, M]
    const float *X;
    const float *Y;
    const int32_t *idx_xy;
    const int32_t *idx_yx;
    float *gX;
    float *gY;
    float *bpart;       // [B][nblk][kBound] per-block box and |g| maxima
    int *shift;         // [B][2] fixed-point shift per item and receiving side
    long long *part;    // per-chunk partial sums (sides with more than one chunk)
    int64_t B, N, M;
    float sxy, syx;     // per-item scale (w1/N, w2/M) when not pointwise
    int nblk;           // bound blocks per item (of the larger cloud)
    int slice;          // receivers per slice (at most kSlice)
    int ns[2];          // receiving slices per item (side 0: X receives, 1: Y)
    int nc[2];          // sender chunks per item
    int local[2];       // shift from the workgroup's own terms (one chunk, one pass)
    int64_t chunk[2];   // senders per chunk (a multiple of kPass)
    int64_t poff[2];    // first partial of each side in part
    // Bucketed path: entries [side][B][nch][kChunk] and per-chunk slice offsets
    // [side][B][nch][ns + 1].
    uint32_t *entries;
    uint32_t *offs;
    int64_t ebase[2], obase[2];
    int nch[2];         // bucket chunks of kChunk senders per item
    int slice_bits;     // log2(slice)
};

// The clouds as seen from receiving side `side` of item b, with the factors
// 2 dL/d dist of senders and receivers: per point (gs, gr) if pointwise, else
// one per item (g2s, g2r).
struct Side {
    const float *R;          // receivers [n_recv, 3]
    const float *S;          // senders [n_send, 3]
    const int32_t *sidx;     // sender -> receiver
    const int32_t *ridx;     // receiver -> sender (its own neighbour)
    float *out;              // [n_recv, 3]
    const float *gs, *gr;    // [n_send], [n_recv] (pointwise)
    float g2s, g2r;          // per item (not pointwise)
    int64_t n_recv, n_send;
};

template <bool kPointwise>
__device__ __forceinline__ Side side_of(const BwdArgs &a, int side, int64_t b)
{
    Side s;
    const bool xs = side == 0;
    s.n_recv = xs ? a.N : a.M;
    s.n_send = xs ? a.M : a.N;
    s.R = (xs ? a.X : a.Y) + b * s.n_recv * 3;
    s.S = (xs ? a.Y : a.X) + b * s.n_send * 3;
    s.sidx = (xs ? a.idx_yx : a.idx_xy) + b * s.n_send;
    s.ridx = (xs ? a.idx_xy : a.idx_yx) + b * s.n_recv;
    s.out = (xs ? a.gX : a.gY) + b * s.n_recv * 3;
    if (kPointwise) {
        s.gs = (xs ? a.gyx : a.gxy) + b * s.n_send;
        s.gr = (xs ? a.gxy : a.gyx) + b * s.n_recv;
        s.g2s = s.g2r = 0.0f;
    } else {
        s.gs = s.gr = nullptr;
        const float gx = 2.0f * (a.gxy[b] * a.sxy), gy = 2.0f * (a.gyx[b] * a.syx);
        s.g2s = xs ? gy : gx;
        s.g2r = xs ? gx : gy;
    }
    return s;
}

template <bool kPointwise>
__device__ __forceinline__ float g2_send(const Side &s, int64_t j)
{
    return kPointwise ? 2.0f * s.gs[j] : s.g2s;
}

template <bool kPointwise>
__device__ __forceinline__ float g2_recv(const Side &s, int64_t i)
{
    return kPointwise ? 2.0f * s.gr[i] : s.g2r;
}

template <bool kPointwise>
__global__ __launch_bounds__(kBoundThreads) void bound_kernel(BwdArgs a)
{
    __shared__ float red[kBoundThreads / kWave][kBound];
    const int64_t b = blockIdx.x / a.nblk;
    const int64_t j0 = (blockIdx.x % a.nblk) * static_cast<int64_t>(kBoundBlock) + threadIdx.x;
    // v[0..2] = -min, v[3..5] = max of the coordinates (so all are maxima).
    float v[kBound];
#pragma unroll
    for (int c = 0; c < 6; ++c) v[c] = -__builtin_inff();
    v[6] = v[7] = 0.0f;
    if (!kPointwise) {
        v[6] = fabsf(a.gxy[b] * a.sxy);
        v[7] = fabsf(a.gyx[b] * a.syx);
    }
    // Loads from clamped indices (a point past a cloud's end repeats its last
    // point, which the maxima already hold), so that no branch splits them.
#pragma unroll
    for (int u = 0; u < kBoundPer; ++u) {
        const int64_t j = j0 + u * kBoundThreads;
        const int64_t jx = std::min<int64_t>(j, a.N - 1), jy = std::min<int64_t>(j, a.M - 1);
        const float *x = a.X + (b * a.N + jx) * 3;
        const float *y = a.Y + (b * a.M + jy) * 3;
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            v[c] = fmaxf(v[c], fmaxf(-x[c], -y[c]));
            v[3 + c] = fmaxf(v[3 + c], fmaxf(x[c], y[c]));
        }
        if (kPointwise) {
            v[6] = fmaxf(v[6], fabsf(a.gxy[b * a.N + jx]));
            v[7] = fmaxf(v[7], fabsf(a.gyx[b * a.M + jy]));
        }
    }
#pragma unroll
    for (int c = 0; c < kBound; ++c) {
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) v[c] = fmaxf(v[c], __shfl_xor(v[c], off, kWave));
    }
    if (threadIdx.x % kWave == 0) {
#pragma unroll
        for (int c = 0; c < kBound; ++c) red[threadIdx.x / kWave][c] = v[c];
    }
    __syncthreads();
    if (threadIdx.x < kBound) {
        float m = red[0][threadIdx.x];
#pragma unroll
        for (int w = 1; w < kBoundThreads / kWave; ++w) m = fmaxf(m, red[w][threadIdx.x]);
        a.bpart[blockIdx.x * kBound + threadIdx.x] = m;
    }
}

// Own term 2 g(r) (r - s) of receiver p, s its own neighbour (0 if that
// index is outside the sender cloud).
template <bool kPointwise>
__device__ __forceinline__ void own_term(const Side &s, int64_t p, float own[3])
{
    const int32_t nb = s.ridx[p];
    const bool ok = nb >= 0 && nb < s.n_send;
    const int64_t qn = ok ? nb : 0;
    const float g2 = ok ? g2_recv<kPointwise>(s, p) : 0.0f;
#pragma unroll
    for (int c = 0; c < 3; ++c) own[c] = g2 * (s.R[3 * p + c] - s.S[3 * qn + c]);
}

// The own terms of a thread's kOwn receivers (r0 + tid + k kBlock, clamped
// into the slice), loaded in two steps so that nothing waits on them before
// the output: the receivers' coordinates and neighbour indices with the
// kernel's first loads, the neighbours' coordinates once those have arrived.
// The receivers' coordinates go to the slice's copy in LDS (`rs`, 3 floats
// per receiver from r0), which the queued terms read too.  The arithmetic is
// own_term's.
template <bool kPointwise>
struct OwnTerms {
    int32_t nb[kOwn];
    float r[kOwn][3], q[kOwn][3], g[kOwn];
    int o[kOwn];   // receiver offset in the slice

    __device__ __forceinline__ void fetch(const Side &s, int64_t r0, int64_t r1, int tid)
    {
#pragma unroll
        for (int k = 0; k < kOwn; ++k) {
            const int64_t p = std::min<int64_t>(r0 + tid + k * kBlock, r1 - 1);
            o[k] = static_cast<int>(p - r0);
            nb[k] = s.ridx[p];
#pragma unroll
            for (int c = 0; c < 3; ++c) r[k][c] = s.R[3 * p + c];
            g[k] = kPointwise ? s.gr[p] : 0.0f;
        }
    }
    // Several threads may write the slice's last receiver: the same values.
    __device__ __forceinline__ void stage(float *rs) const
    {
#pragma unroll
        for (int k = 0; k < kOwn; ++k)
#pragma unroll
            for (int c = 0; c < 3; ++c) rs[3 * o[k] + c] = r[k][c];
    }
    __device__ __forceinline__ bool valid(const Side &s, int k) const
    {
        return nb[k] >= 0 && nb[k] < s.n_send;
    }
    __device__ __forceinline__ void fetch_neighbours(const Side &s)
    {
#pragma unroll
        for (int k = 0; k < kOwn; ++k) {
            const int64_t qn = valid(s, k) ? nb[k] : 0;
#pragma unroll
            for (int c = 0; c < 3; ++c) q[k][c] = s.S[3 * qn + c];
        }
    }
    __device__ __forceinline__ float g2(const Side &s, int k) const
    {
        return valid(s, k) ? (kPointwise ? 2.0f * g[k] : s.g2r) : 0.0f;
    }
    // With the receivers' coordinates from the staged copy rs.
    __device__ __forceinline__ void term(const Side &s, const float *rs, int k, float own[3]) const
    {
        const float gk = g2(s, k);
#pragma unroll
        for (int c = 0; c < 3; ++c) own[c] = gk * (rs[3 * o[k] + c] - q[k][c]);
    }
};

// Own term plus the scatter sum (double), rounded once.
__device__ __forceinline__ void write_point(const Side &s, int64_t p, const float own[3],
                                            const double scat[3])
{
#pragma unroll
    for (int c = 0; c < 3; ++c)
        s.out[3 * p + c] = static_cast<float>(static_cast<double>(own[c]) + scat[c]);
}

// Term -2 g(s) (s - r) of queue entry e (sender offset from `base` in the
// high bits, receiver offset from r0 in the low kSliceBits); ir = receiver
// offset; the receiver's coordinates from the slice's copy rs in LDS.
template <bool kPointwise>
__device__ __forceinline__ void queued_term(const Side &s, int64_t base, const float *rs,
                                            uint32_t e, float t[3], int &ir)
{
    const int64_t q = base + (e >> kSliceBits);
    ir = static_cast<int>(e & (kSlice - 1));
    const float g2 = g2_send<kPointwise>(s, q);
#pragma unroll
    for (int d = 0; d < 3; ++d) t[d] = -(g2 * (s.S[3 * q + d] - rs[3 * ir + d]));
}

__device__ __forceinline__ void add_term(unsigned long long *acc, int ir, const float t[3], int ks)
{
#pragma unroll
    for (int d = 0; d < 3; ++d)
        atomicAdd(acc + 3 * ir + d, static_cast<unsigned long long>(to_fixed(t[d], ks)));
}

__device__ __forceinline__ float max_abs3(float m, const float t[3])
{
    return fmaxf(m, fmaxf(fabsf(t[0]), fmaxf(fabsf(t[1]), fabsf(t[2]))));
}

// The terms of queue entries e0 + tid + h kBlock, h < H, with all their loads
// in flight together: an entry at or past n (n > e0) repeats entry n - 1, so
// every load is of a queued sender and no branch splits the loads.  Returns the
// largest component of the entries before n.
template <int H, bool kPointwise>
__device__ __forceinline__ float hold_terms(const Side &s, int64_t base, const float *rs,
                                            const uint32_t *queue, int e0, int n, int tid,
                                            float hold[][3], int hir[])
{
    float m = 0.0f;
#pragma unroll
    for (int h = 0; h < H; ++h) {
        const int e = e0 + tid + h * kBlock;
        queued_term<kPointwise>(s, base, rs, queue[min(e, n - 1)], hold[h], hir[h]);
    }
#pragma unroll
    for (int h = 0; h < H; ++h)
        if (e0 + tid + h * kBlock < n) m = max_abs3(m, hold[h]);
    return m;
}

// The neighbour indices of one pass of kBlock * kIdx senders from sp, avail
// of them left in the chunk: iv[4 u + k] is sender 4 (u kBlock + tid) + k,
// -1 past the end.  The first NU groups u are loaded four senders at a time
// (kFull: the whole pass lies in the chunk); a group reaching past the end
// loads the last four senders instead and picks its own; groups from NU on
// lie past the end.  NU = 0: fewer than four senders, loaded one by one.
template <int NU, bool kFull>
__device__ __forceinline__ void load_pass(const int32_t *sp, int avail, int tid,
                                          int32_t iv[kIdx])
{
    if (NU == 0) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int o = 4 * tid + k;
            const int32_t e = sp[min(o, avail - 1)];
            iv[k] = o < avail ? e : -1;
        }
    } else if (kFull) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const I4 v = *reinterpret_cast<const I4 *>(sp + 4 * (u * kBlock + tid));
            iv[4 * u] = v.x;
            iv[4 * u + 1] = v.y;
            iv[4 * u + 2] = v.z;
            iv[4 * u + 3] = v.w;
        }
    } else {
        I4 v[NU > 0 ? NU : 1];
#pragma unroll
        for (int u = 0; u < NU; ++u)
            v[u] = *reinterpret_cast<const I4 *>(sp + min(4 * (u * kBlock + tid), avail - 4));
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int o = 4 * (u * kBlock + tid);
            const int d = o - min(o, avail - 4);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int i = k + d;
                const int32_t e = i == 0 ? v[u].x : i == 1 ? v[u].y : i == 2 ? v[u].z : v[u].w;
                iv[4 * u + k] = o + k < avail ? e : -1;
            }
        }
    }
#pragma unroll
    for (int j = 4 * (NU == 0 ? 1 : NU); j < kIdx; ++j) iv[j] = -1;
}

// Exclusive prefix sum of v over the wave (lane order) and the wave's total.
__device__ __forceinline__ int wave_prefix(int v, int &total)
{
    const int lane = threadIdx.x % kWave;
    int incl = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int n = __shfl_up(incl, off, kWave);
        incl += lane >= off ? n : 0;
    }
    total = __shfl(incl, kWave - 1, kWave);
    return incl - v;
}

template <bool kPointwise>
__global__ __launch_bounds__(kBlock) void scatter_kernel(BwdArgs a)
{
    __shared__ unsigned long long acc[3 * kSlice];
    __shared__ uint32_t queue[kPass];
    __shared__ float rs[3 * kSlice];
    __shared__ float red[kBlock / kWave];
    __shared__ uint32_t qcount;
    const int tid = threadIdx.x;
    // Workgroups go to the XCDs round-robin.  With one sender chunk per side,
    // the slices of one item and side read the same sender indices and
    // coordinates, so consecutive groups are placed on one XCD (one L2);
    // chunked shapes keep the plain order, which spreads the heavier side.
    // (32-bit and branch-free: the launch has fewer than 2^32 workgroups, and
    // the decode runs before the kernel's first loads.)
    const uint32_t i = blockIdx.x, per = gridDim.x / kXcds;
    const bool remap = a.nc[0] == 1 && a.nc[1] == 1 && i < kXcds * per;
    const uint32_t wg = remap ? (i % kXcds) * per + i / kXcds : i;
    const uint32_t g0 = static_cast<uint32_t>(a.B) * static_cast<uint32_t>(a.ns[0] * a.nc[0]);
    const int side = wg < g0 ? 0 : 1;
    const uint32_t g = side == 0 ? wg : wg - g0;
    const int ns = a.ns[side], nc = a.nc[side];
    const uint32_t pi = static_cast<uint32_t>(ns * nc);
    const int64_t b = g / pi;
    const int rest = static_cast<int>(g % pi);
    const int slice = rest / nc, c = rest % nc;
    const Side s = side_of<kPointwise>(a, side, b);
    const int64_t r0 = static_cast<int64_t>(slice) * a.slice;
    const int64_t r1 = std::min<int64_t>(r0 + a.slice, s.n_recv);
    const bool local = a.local[side] != 0;

    // Own terms of this thread's receivers (used with one chunk; otherwise
    // the finalize pass adds them): independent of the scatter, so their
    // loads are issued first.
    OwnTerms<kPointwise> own;
    own.fetch(s, r0, r1, tid);

    for (int t = tid; t < 3 * (r1 - r0); t += kBlock) acc[t] = 0ull;
    if (tid == 0) qcount = 0u;
    int ks = 0;
    if (!local) {
        // Every term component is at most 2 max|g_send| times the largest
        // extent of the item's bounding box.
        const float *bp = a.bpart + b * a.nblk * kBound;
        float v[kBound];
#pragma unroll
        for (int k = 0; k < kBound; ++k) v[k] = -__builtin_inff();
        for (int64_t k = tid; k < a.nblk; k += kBlock) {
#pragma unroll
            for (int u = 0; u < kBound; ++u) v[u] = fmaxf(v[u], bp[k * kBound + u]);
        }
        float ext = 0.0f;
#pragma unroll
        for (int d = 0; d < 3; ++d) ext = fmaxf(ext, v[3 + d] + v[d]);   // max - min
        const float gs = side == 0 ? v[7] : v[6];                         // senders' |g|
        ks = fixed_shift(group_max<kBlock>(2.0f * gs * ext, red), s.n_send);
        if (slice == 0 && c == 0 && tid == 0) a.shift[b * 2 + side] = ks;
    }
    __syncthreads();

    const int64_t q0 = c * a.chunk[side];
    const int64_t q1 = std::min<int64_t>(q0 + a.chunk[side], s.n_send);
    const int32_t r0i = static_cast<int32_t>(r0);
    const uint32_t slen = static_cast<uint32_t>(r1 - r0);
    // One pass of senders from `base`: their neighbour indices, and the ones
    // landing in the slice queued in LDS; returns the queue's length.
    auto queue_pass = [&](int64_t base) -> int {
        // The pass's neighbour indices, four consecutive senders per 16-byte
        // load, all loads in flight together.  Which form runs is the same for
        // the whole workgroup, so no lane's loads wait on another's.
        int32_t iv[kIdx];
        const int32_t *sp = s.sidx + base;
        const int avail = static_cast<int>(std::min<int64_t>(q1 - base, kPass));
        if (avail == kPass)
            load_pass<kIdx / 4, true>(sp, avail, tid, iv);
        else if (avail > 4 * kBlock * (kIdx / 8))
            load_pass<kIdx / 4, false>(sp, avail, tid, iv);
        else if (avail > 4 * kBlock * (kIdx / 16))
            load_pass<kIdx / 8, false>(sp, avail, tid, iv);
        else if (avail > 4 * kBlock)
            load_pass<kIdx / 16, false>(sp, avail, tid, iv);
        else if (avail >= 4)
            load_pass<1, false>(sp, avail, tid, iv);
        else
            load_pass<0, false>(sp, avail, tid, iv);
        // Queue the senders whose neighbour lies in the slice: bit j of `hit`
        // for iv[j]; the wave's exclusive prefix of the per-lane counts from
        // one ballot per bit of the count.
        uint32_t hit = 0u;
#pragma unroll
        for (int j = 0; j < kIdx; ++j)
            hit |= (static_cast<uint32_t>(iv[j] - r0i) < slen ? 1u : 0u) << j;
        // The receivers' coordinates and own neighbour indices arrived before
        // these.  Every pass stages and fetches them (the same values): done
        // conditionally, the compiler's wait counts would assume the fetch in
        // flight and wait for it here.
        own.stage(rs);
        own.fetch_neighbours(s);
        const int cnt = __popc(hit);
        uint32_t excl = 0u, total = 0u;
#pragma unroll
        for (int k = 0; k < 6; ++k) {   // cnt <= 32
            const unsigned long long m = __ballot((cnt >> k) & 1);
            excl += __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                              __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u))
                    << k;
            total += static_cast<uint32_t>(__popcll(m)) << k;
        }
        uint32_t wbase = 0u;
        if (tid % kWave == 0 && total > 0u) wbase = atomicAdd(&qcount, total);
        uint32_t pos = __builtin_amdgcn_readfirstlane(wbase) + excl;
#pragma unroll
        for (int j = 0; j < kIdx; ++j) {
            if ((hit >> j) & 1u)
                queue[pos++] = (static_cast<uint32_t>(4 * ((j / 4) * kBlock + tid) + j % 4)
                                << kSliceBits) |
                               static_cast<uint32_t>(iv[j] - r0i);
        }
        __syncthreads();
        return static_cast<int>(qcount);
    };

    float hold[kHold][3];
    int hir[kHold];
    if (local) {
        // The only pass (no loop, so that the compiler's wait counts carry
        // nothing over from a previous pass): the shift comes from the
        // largest queued term.
        const int64_t base = q0;
        const int qlen = queue_pass(base);
        float m = 0.0f;
        if (qlen > kHold / 2 * kBlock)
            m = hold_terms<kHold, kPointwise>(s, base, rs, queue, 0, qlen, tid, hold, hir);
        else if (qlen > 0)
            m = hold_terms<kHold / 2, kPointwise>(s, base, rs, queue, 0, qlen, tid, hold, hir);
        for (int e = tid + kHold * kBlock; e < qlen; e += kBlock) {
            float t[3];
            int ir;
            queued_term<kPointwise>(s, base, rs, queue[e], t, ir);
            m = max_abs3(m, t);
        }
        ks = fixed_shift(group_max<kBlock>(m, red), qlen);
#pragma unroll
        for (int h = 0; h < kHold; ++h)
            if (tid + h * kBlock < qlen) add_term(acc, hir[h], hold[h], ks);
        for (int e = tid + kHold * kBlock; e < qlen; e += kBlock) {
            float t[3];
            int ir;
            queued_term<kPointwise>(s, base, rs, queue[e], t, ir);
            add_term(acc, ir, t, ks);
        }
        __syncthreads();   // all sums complete before the output reads them
    } else {
        for (int64_t base = q0; base < q1; base += kPass) {
            const int qlen = queue_pass(base);
            for (int e0 = 0; e0 < qlen; e0 += kHold * kBlock) {
                hold_terms<kHold, kPointwise>(s, base, rs, queue, e0, qlen, tid, hold, hir);
#pragma unroll
                for (int h = 0; h < kHold; ++h)
                    if (e0 + tid + h * kBlock < qlen) add_term(acc, hir[h], hold[h], ks);
            }
            __syncthreads();
            if (tid == 0) qcount = 0u;
            __syncthreads();
        }
    }

    if (nc == 1) {
#pragma unroll
        for (int k = 0; k < kOwn; ++k) {
            const int64_t p = r0 + tid + k * kBlock;
            if (p < r1) {
                const unsigned long long *t = acc + 3 * (p - r0);
                const double scat[3] = {
                    ldexp(static_cast<double>(static_cast<long long>(t[0])), -ks),
                    ldexp(static_cast<double>(static_cast<long long>(t[1])), -ks),
                    ldexp(static_cast<double>(static_cast<long long>(t[2])), -ks)};
                float ownk[3];
                own.term(s, rs, k, ownk);
                write_point(s, p, ownk, scat);
            }
        }
    } else {
        long long *dst = a.part + a.poff[side] + ((b * nc + c) * s.n_recv + r0) * 3;
        for (int t = tid; t < 3 * (r1 - r0); t += kBlock) dst[t] = static_cast<long long>(acc[t]);
    }
}

// Receivers of `side` (which has more than one chunk): exact sum of the
// chunks' partials, own term added, rounded once.
template <bool kPointwise>
__global__ __launch_bounds__(kThreads) void finalize_kernel(BwdArgs a, int side)
{
    const int64_t n_recv = side == 0 ? a.N : a.M;
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (k >= a.B * n_recv) return;
    const int64_t b = k / n_recv, p = k - b * n_recv;
    const Side s = side_of<kPointwise>(a, side, b);
    const int nc = a.nc[side];
    // The own term's receiver and neighbour index go out with the partials'
    // loads, its neighbour's coordinates once the partials are summed (own_term's
    // arithmetic).
    const int32_t nb = s.ridx[p];
    float r[3];
#pragma unroll
    for (int d = 0; d < 3; ++d) r[d] = s.R[3 * p + d];
    const float gr = kPointwise ? s.gr[p] : 0.0f;
    const long long *src = a.part + a.poff[side] + (b * nc * n_recv + p) * 3;
    unsigned long long sum[3] = {0ull, 0ull, 0ull};
    for (int c = 0; c < nc; ++c) {
#pragma unroll
        for (int d = 0; d < 3; ++d)
            sum[d] += static_cast<unsigned long long>(src[static_cast<int64_t>(c) * n_recv * 3 + d]);
    }
    const bool ok = nb >= 0 && nb < s.n_send;
    const int64_t qn = ok ? nb : 0;
    const float g2 = ok ? (kPointwise ? 2.0f * gr : s.g2r) : 0.0f;
    float own[3];
#pragma unroll
    for (int d = 0; d < 3; ++d) own[d] = g2 * (r[d] - s.S[3 * qn + d]);
    const int ks = a.shift[b * 2 + side];
    const double scat[3] = {ldexp(static_cast<double>(static_cast<long long>(sum[0])), -ks),
                            ldexp(static_cast<double>(static_cast<long long>(sum[1])), -ks),
                            ldexp(static_cast<double>(static_cast<long long>(sum[2])), -ks)};
    write_point(s, p, own, scat);
}

// One chunk of kChunk senders of one item and side: counting sort by receiver
// slice.  Senders whose neighbour index lies outside the receiving cloud are
// dropped.
__global__ __launch_bounds__(kBucketThreads) void bucket_kernel(BwdArgs a)
{
    constexpr int kPerThread = kMaxBucketSlices / kBucketThreads;
    __shared__ uint32_t hist[kMaxBucketSlices + 1];
    __shared__ uint32_t wtot[kBucketThreads / kWave];
    const int tid = threadIdx.x;
    // Consecutive chunks of one item and side on one XCD, like the slices that
    // read their entries (slice_kernel).
    uint32_t wg = blockIdx.x;
    const uint32_t xper = gridDim.x / kXcds;
    if (wg < kXcds * xper) wg = (wg % kXcds) * xper + wg / kXcds;
    const int64_t g0 = a.B * a.nch[0];
    const int side = static_cast<int64_t>(wg) < g0 ? 0 : 1;
    const int64_t g = side == 0 ? wg : wg - g0;
    const int nch = a.nch[side], ns = a.ns[side];
    const int64_t b = g / nch;
    const int c = static_cast<int>(g % nch);
    const bool xs = side == 0;
    const int64_t n_recv = xs ? a.N : a.M, n_send = xs ? a.M : a.N;
    const int32_t *sidx = (xs ? a.idx_yx : a.idx_xy) + b * n_send;
    const int64_t q0 = static_cast<int64_t>(c) * kChunk;
    int32_t iv[kBucketPer];
#pragma unroll
    for (int u = 0; u < kBucketPer; ++u) {
        const int64_t q = q0 + u * kBucketThreads + tid;
        const int32_t v = q < n_send ? sidx[q] : -1;
        iv[u] = (v >= 0 && v < n_recv) ? v : -1;
    }
    for (int k = tid; k <= ns; k += kBucketThreads) hist[k] = 0u;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kBucketPer; ++u)
        if (iv[u] >= 0) atomicAdd(&hist[iv[u] >> a.slice_bits], 1u);
    __syncthreads();
    // Exclusive prefix sum over the ns bins (each thread a run of consecutive
    // bins, then the waves in order); hist[ns] = the chunk's valid senders.
    const int per = (ns + kBucketThreads - 1) / kBucketThreads;
    uint32_t loc[kPerThread];
    uint32_t sum = 0u;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        const int bin = tid * per + k;
        loc[k] = (k < per && bin < ns) ? hist[bin] : 0u;
        sum += loc[k];
    }
    int total;
    const int excl = wave_prefix(static_cast<int>(sum), total);
    if (tid % kWave == 0) wtot[tid / kWave] = static_cast<uint32_t>(total);
    __syncthreads();
    uint32_t run = static_cast<uint32_t>(excl), all = 0u;
#pragma unroll
    for (int w = 0; w < kBucketThreads / kWave; ++w) {
        run += w < tid / kWave ? wtot[w] : 0u;
        all += wtot[w];
    }
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        const int bin = tid * per + k;
        if (k < per && bin < ns) {
            hist[bin] = run;
            run += loc[k];
        }
    }
    if (tid == 0) hist[ns] = all;
    __syncthreads();
    uint32_t *off = a.offs + a.obase[side] + (b * nch + c) * (ns + 1);
    for (int k = tid; k <= ns; k += kBucketThreads) off[k] = hist[k];
    __syncthreads();
    uint32_t *ent = a.entries + a.ebase[side] + (b * nch + c) * static_cast<int64_t>(kChunk);
#pragma unroll
    for (int u = 0; u < kBucketPer; ++u) {
        if (iv[u] >= 0) {
            const int sl = iv[u] >> a.slice_bits;
            const uint32_t pos = atomicAdd(&hist[sl], 1u);
            ent[pos] = (static_cast<uint32_t>(u * kBucketThreads + tid) << kSliceBits) |
                       static_cast<uint32_t>(iv[u] - (sl << a.slice_bits));
        }
    }
}

// The chunk holding flat entry e: the last c with pre[c] <= e.
__device__ __forceinline__ int chunk_of(const uint32_t *pre, int nch, int64_t e)
{
    int lo = 0, hi = nch;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (pre[mid] <= e) lo = mid; else hi = mid;
    }
    return lo;
}

// One slice of receivers of one item and side, over the entries every chunk's
// bucket holds for it.
template <bool kPointwise>
__global__ __launch_bounds__(kBlock) void slice_kernel(BwdArgs a)
{
    __shared__ unsigned long long acc[3 * kSlice];
    __shared__ uint32_t pre[kMaxBucketChunks + 1];   // entries before chunk c
    __shared__ uint32_t seg[kMaxBucketChunks];       // segment start in chunk c
    __shared__ float red[kBlock / kWave];
    __shared__ uint32_t wtot[kBlock / kWave];
    const int tid = threadIdx.x;
    // Workgroups go to the XCDs round-robin: consecutive slices of one item
    // and side are placed on one XCD, whose L2 then holds that item's clouds.
    uint32_t wg = blockIdx.x;
    const uint32_t per = gridDim.x / kXcds;
    if (wg < kXcds * per) wg = (wg % kXcds) * per + wg / kXcds;
    const int64_t g0 = a.B * a.ns[0];
    const int side = static_cast<int64_t>(wg) < g0 ? 0 : 1;
    const int64_t g = side == 0 ? wg : wg - g0;
    const int ns = a.ns[side], nch = a.nch[side];
    const int64_t b = g / ns;
    const int slice = static_cast<int>(g % ns);
    const Side s = side_of<kPointwise>(a, side, b);
    const int64_t r0 = static_cast<int64_t>(slice) * a.slice;
    const int64_t r1 = std::min<int64_t>(r0 + a.slice, s.n_recv);

    // Own terms first (their loads overlap the segment loads' round).
    float ownv[kOwn][3];
#pragma unroll
    for (int k = 0; k < kOwn; ++k)
        own_term<kPointwise>(s, std::min<int64_t>(r0 + tid + k * kBlock, r1 - 1), ownv[k]);
    // Each thread takes chunks 2 tid and 2 tid + 1: segment starts and lengths
    // (loaded for a clamped chunk, so that no branch splits the loads).
    const uint32_t *off = a.offs + a.obase[side] + b * nch * static_cast<int64_t>(ns + 1);
    uint32_t st[2], en[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int64_t c = std::min(2 * tid + k, nch - 1);
        st[k] = off[c * (ns + 1) + slice];
        en[k] = off[c * (ns + 1) + slice + 1];
    }
    for (int t = tid; t < 3 * (r1 - r0); t += kBlock) acc[t] = 0ull;
    uint32_t len[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int c = 2 * tid + k;
        len[k] = c < nch ? en[k] - st[k] : 0u;
        if (c < nch) seg[c] = st[k];
    }
    int total;
    const int excl = wave_prefix(static_cast<int>(len[0] + len[1]), total);
    if (tid % kWave == 0) wtot[tid / kWave] = static_cast<uint32_t>(total);
    __syncthreads();
    // The slice's receivers, read from the cloud (an LDS copy as in
    // scatter_kernel would leave room for one workgroup per CU instead of two).
    const float *rs = s.R + 3 * r0;
    uint32_t before = static_cast<uint32_t>(excl), all = 0u;
#pragma unroll
    for (int w = 0; w < kBlock / kWave; ++w) {
        before += w < tid / kWave ? wtot[w] : 0u;
        all += wtot[w];
    }
    if (2 * tid < nch) pre[2 * tid] = before;
    if (2 * tid + 1 < nch) pre[2 * tid + 1] = before + len[0];
    if (tid == 0) pre[nch] = all;
    __syncthreads();
    const int64_t E = all;
    const uint32_t *ent = a.entries + a.ebase[side] + b * nch * static_cast<int64_t>(kChunk);

    // Flat entry e -> its chunk (the last c with pre[c] <= e) and its term.
    auto term = [&](int64_t e, float t[3], int &ir) {
        const int lo = chunk_of(pre, nch, e);
        const uint32_t en = ent[static_cast<int64_t>(lo) * kChunk + seg[lo] + (e - pre[lo])];
        queued_term<kPointwise>(s, static_cast<int64_t>(lo) * kChunk, rs, en, t, ir);
    };
    float hold[kHold][3];
    int hir[kHold];
    float m = 0.0f;
#pragma unroll
    for (int h = 0; h < kHold; ++h) {
        const int64_t e = tid + static_cast<int64_t>(h) * kBlock;
        if (e < E) {
            term(e, hold[h], hir[h]);
            m = max_abs3(m, hold[h]);
        }
    }
    for (int64_t e = tid + static_cast<int64_t>(kHold) * kBlock; e < E; e += kBlock) {
        float t[3];
        int ir;
        term(e, t, ir);
        m = max_abs3(m, t);
    }
    const int ks = fixed_shift(group_max<kBlock>(m, red), E);
#pragma unroll
    for (int h = 0; h < kHold; ++h)
        if (tid + static_cast<int64_t>(h) * kBlock < E) add_term(acc, hir[h], hold[h], ks);
    for (int64_t e = tid + static_cast<int64_t>(kHold) * kBlock; e < E; e += kBlock) {
        float t[3];
        int ir;
        term(e, t, ir);
        add_term(acc, ir, t, ks);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kOwn; ++k) {
        const int64_t p = r0 + tid + k * kBlock;
        if (p < r1) {
            const unsigned long long *t = acc + 3 * (p - r0);
            const double scat[3] = {
                ldexp(static_cast<double>(static_cast<long long>(t[0])), -ks),
                ldexp(static_cast<double>(static_cast<long long>(t[1])), -ks),
                ldexp(static_cast<double>(static_cast<long long>(t[2])), -ks)};
            write_point(s, p, ownv[k], scat);
        }
    }
}

int64_t ceil_div(int64_t x, int64_t y) { return (x + y - 1) / y; }

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

struct BwdPlan {
    int nblk, slice, slice_bits;
    int ns[2], nc[2], local[2], nch[2];
    bool need_bound, bucketed;
    int64_t chunk[2];
    size_t bpart_bytes, shift_bytes, part_elems[2];
    size_t entry_elems[2], off_elems[2];
};

BwdPlan plan_backward(int64_t B, int64_t N, int64_t M)
{
    BwdPlan p;
    p.nblk = static_cast<int>(ceil_div(std::max(N, M), kBoundBlock));
    const int64_t n_recv[2] = {N, M}, n_send[2] = {M, N};
    int64_t rounds[2];
    // Slices of kSlice receivers, halved (down to kMinSlice) while twice the
    // workgroups still fit one per CU: every workgroup scans all senders
    // anyway, and more of them in flight shortens the few dependent memory
    // rounds that bound a small launch (more than one per CU measured slower).
    p.slice = kSlice;
    p.slice_bits = kSliceBits;
    while (p.slice > kMinSlice &&
           2 * B * (ceil_div(N, p.slice) + ceil_div(M, p.slice)) <= kCUs) {
        p.slice /= 2;
        --p.slice_bits;
    }
    bool feasible = true;
    for (int s = 0; s < 2; ++s) {
        p.ns[s] = static_cast<int>(ceil_div(n_recv[s], p.slice));
        rounds[s] = ceil_div(n_send[s], kPass);
        p.nch[s] = static_cast<int>(std::min<int64_t>(ceil_div(n_send[s], kChunk), INT32_MAX));
        if (p.ns[s] > kMaxBucketSlices || p.nch[s] > kMaxBucketChunks ||
            ceil_div(n_send[s], p.ns[s]) > kMaxBucketShare)
            feasible = false;
    }
    // The direct scan: a side whose workgroups would scan many more passes
    // than the other's splits its senders into chunks of about the other's
    // length (the long scan is what bounds the kernel's time otherwise).
    const int64_t target = std::min(rounds[0], rounds[1]);
    for (int s = 0; s < 2; ++s) {
        const int64_t want = ceil_div(rounds[s], target);
        p.chunk[s] = ceil_div(rounds[s], want) * kPass;
        p.nc[s] = static_cast<int>(ceil_div(n_send[s], p.chunk[s]));
        p.local[s] = p.nc[s] == 1 && n_send[s] <= kPass;
    }
    // Bucketing costs a launch and two dependent memory rounds.  It pays where
    // the direct scan would need the bound pass (a side's senders exceed one
    // pass) and where its repeated index scans would read much more than the
    // indices once.
    const int64_t scan_bytes =
        4 * B * (static_cast<int64_t>(p.ns[0]) * n_send[0] + static_cast<int64_t>(p.ns[1]) * n_send[1]);
    const bool direct_local = p.local[0] && p.local[1];
    p.bucketed = feasible && (!direct_local || scan_bytes >= kMinBucketScanBytes);
    for (int s = 0; s < 2; ++s) {
        p.entry_elems[s] = p.bucketed ? static_cast<size_t>(B) * p.nch[s] * kChunk : 0;
        p.off_elems[s] = p.bucketed ? static_cast<size_t>(B) * p.nch[s] * (p.ns[s] + 1) : 0;
        p.part_elems[s] = !p.bucketed && p.nc[s] > 1
                              ? static_cast<size_t>(B * p.nc[s] * n_recv[s] * 3) : 0;
    }
    p.need_bound = !p.bucketed && !direct_local;
    p.bpart_bytes = align256(static_cast<size_t>(B * p.nblk) * kBound * 4);
    p.shift_bytes = align256(static_cast<size_t>(B * 2) * 4);
    return p;
}

}  // namespace

size_t backward_workspace_bytes(int64_t B, int64_t N, int64_t M)
{
    const BwdPlan p = plan_backward(B, N, M);
    if (p.bucketed)
        return align256((p.entry_elems[0] + p.entry_elems[1]) * 4) +
               align256((p.off_elems[0] + p.off_elems[1]) * 4);
    return p.bpart_bytes + p.shift_bytes + align256((p.part_elems[0] + p.part_elems[1]) * 8);
}

hipError_t launch_backward(int64_t B, int64_t N, int64_t M, const float *g_xy,
                           const float *g_yx, bool pointwise, float sxy, float syx,
                           const float *X, const float *Y, const int32_t *idx_xy,
                           const int32_t *idx_yx, float *gX, float *gY, void *ws,
                           hipStream_t stream)
{
    const BwdPlan p = plan_backward(B, N, M);
    char *base = static_cast<char *>(ws);
    BwdArgs a{};
    a.gxy = g_xy;
    a.gyx = g_yx;
    a.X = X;
    a.Y = Y;
    a.idx_xy = idx_xy;
    a.idx_yx = idx_yx;
    a.gX = gX;
    a.gY = gY;
    a.bpart = reinterpret_cast<float *>(base);
    a.shift = reinterpret_cast<int *>(base + p.bpart_bytes);
    a.part = reinterpret_cast<long long *>(base + p.bpart_bytes + p.shift_bytes);
    a.B = B;
    a.N = N;
    a.M = M;
    a.sxy = sxy;
    a.syx = syx;
    a.nblk = p.nblk;
    a.slice = p.slice;
    for (int s = 0; s < 2; ++s) {
        a.ns[s] = p.ns[s];
        a.nc[s] = p.nc[s];
        a.local[s] = p.local[s];
        a.chunk[s] = p.chunk[s];
    }
    a.poff[0] = 0;
    a.poff[1] = static_cast<int64_t>(p.part_elems[0]);
    a.slice_bits = p.slice_bits;
    if (p.bucketed) {
        a.entries = reinterpret_cast<uint32_t *>(base);
        a.offs = reinterpret_cast<uint32_t *>(
            base + align256((p.entry_elems[0] + p.entry_elems[1]) * 4));
        a.ebase[0] = 0;
        a.ebase[1] = static_cast<int64_t>(p.entry_elems[0]);
        a.obase[0] = 0;
        a.obase[1] = static_cast<int64_t>(p.off_elems[0]);
        for (int s = 0; s < 2; ++s) a.nch[s] = p.nch[s];
        const uint32_t nb = static_cast<uint32_t>(B * (static_cast<int64_t>(p.nch[0]) + p.nch[1]));
        const uint32_t nsl = static_cast<uint32_t>(B * (static_cast<int64_t>(p.ns[0]) + p.ns[1]));
        bucket_kernel<<<nb, kBucketThreads, 0, stream>>>(a);
        if (pointwise)
            slice_kernel<true><<<nsl, kBlock, 0, stream>>>(a);
        else
            slice_kernel<false><<<nsl, kBlock, 0, stream>>>(a);
        return hipGetLastError();
    }
    const uint32_t nbound = static_cast<uint32_t>(B * p.nblk);
    const int64_t groups = B * (static_cast<int64_t>(p.ns[0]) * p.nc[0] +
                                static_cast<int64_t>(p.ns[1]) * p.nc[1]);
    if (pointwise) {
        if (p.need_bound) bound_kernel<true><<<nbound, kBoundThreads, 0, stream>>>(a);
        scatter_kernel<true><<<static_cast<uint32_t>(groups), kBlock, 0, stream>>>(a);
    } else {
        if (p.need_bound) bound_kernel<false><<<nbound, kBoundThreads, 0, stream>>>(a);
        scatter_kernel<false><<<static_cast<uint32_t>(groups), kBlock, 0, stream>>>(a);
    }
    for (int s = 0; s < 2; ++s) {
        if (p.nc[s] <= 1) continue;
        const uint32_t grid = static_cast<uint32_t>(ceil_div(B * (s == 0 ? N : M), kThreads));
        if (pointwise)
            finalize_kernel<true><<<grid, kThreads, 0, stream>>>(a, s);
        else
            finalize_kernel<false><<<grid, kThreads, 0, stream>>>(a, s);
    }
    return hipGetLastError();
}

}  // namespace cdk

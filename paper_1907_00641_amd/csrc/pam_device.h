// Device code shared by the build and filter kernels: the embedding of a
// point into the permutohedral lattice (operator E of eq. 6) in fp32 with a
// fixed operation order, barycentric weights, key hashing.
#pragma once

#include "pam_internal.h"

#include <climits>

namespace pam {

constexpr int kBlock = 256;


// ---------------------------------------------------------------------------
// Embedding: elevation, remainder-0 point, ranks (operator E)
// ---------------------------------------------------------------------------

template <int D>
struct Simplex {
    float x[D + 1];    // elevated position (fp32)
    int q[D + 1];      // remainder-0 point after the fix-up is (D+1) * q
    int rank[D + 1];   // rank of each residual (0 = largest), after the fix-up
};

// Elevation x = E p in fp32: for each coordinate an fmaf chain over the
// nonzero entries of E in ascending input index.  Returns false if a
// coordinate is not finite or exceeds 2^24 in magnitude.
template <int D>
__device__ __forceinline__ bool elevate(const float *__restrict__ p, const Elev &E, float *x)
{
#pragma clang fp contract(off)
    float pv[D];
#pragma unroll
    for (int j = 0; j < D; ++j)
        pv[j] = p[j];
    bool ok = true;
#pragma unroll
    for (int c = 0; c <= D; ++c) {
        float acc = 0.0f;
        if (c > 0)
            acc = __builtin_fmaf(E.neg[c - 1], pv[c - 1], acc);
#pragma unroll
        for (int j = c; j < D; ++j)
            acc = __builtin_fmaf(E.pos[j], pv[j], acc);
        x[c] = acc;
        ok = ok && (__builtin_fabsf(acc) <= 16777216.0f);  // false for NaN too
    }
    return ok;
}

// Returns false if the point is not finite or too far out to key.
template <int D>
__device__ __forceinline__ bool embed(const float *__restrict__ p, const Elev &E, Simplex<D> &s)
{
#pragma clang fp contract(off)
    bool ok = elevate<D>(p, E, s.x);
    float delta[D + 1];
    int sum = 0;
#pragma unroll
    for (int c = 0; c <= D; ++c) {
        float qf = __builtin_rintf(s.x[c] * E.inv);
        int q = ok ? (int)qf : 0;
        s.q[c] = q;
        sum += q;
        delta[c] = s.x[c] - (float)(q * (D + 1));
    }
#pragma unroll
    for (int c = 0; c <= D; ++c) {
        int r = 0;
#pragma unroll
        for (int c2 = 0; c2 <= D; ++c2) {
            if (c2 < c)
                r += (delta[c2] >= delta[c]) ? 1 : 0;
            else if (c2 > c)
                r += (delta[c2] > delta[c]) ? 1 : 0;
        }
        s.rank[c] = r;
    }
    // restore sum(r) = 0 by moving the |sum| most extreme coordinates by d+1
    if (sum > 0) {
#pragma unroll
        for (int c = 0; c <= D; ++c) {
            if (s.rank[c] >= D + 1 - sum) {
                s.q[c] -= 1;
                s.rank[c] += sum - (D + 1);
            } else {
                s.rank[c] += sum;
            }
        }
    } else if (sum < 0) {
#pragma unroll
        for (int c = 0; c <= D; ++c) {
            if (s.rank[c] < -sum) {
                s.q[c] += 1;
                s.rank[c] += sum + (D + 1);
            } else {
                s.rank[c] += sum;
            }
        }
    }
    return ok;
}

// Barycentric weights of the simplex vertices.  With y = (x - r)/(d+1) and
// ys[r] the y of the coordinate ranked r:
//   b_0 = 1 + ys[d] - ys[0],   b_k = ys[d-k] - ys[d+1-k]  (k >= 1).
// The residual x - r is taken from an fp64 elevation of p (the simplex
// itself comes from the fp32 decisions in embed), then the rest runs in fp32.
template <int D>
__device__ __forceinline__ void barycentric(const Simplex<D> &s, const float *__restrict__ p,
                                            const Elev &E, float *b)
{
    double pd[D];
#pragma unroll
    for (int j = 0; j < D; ++j)
        pd[j] = (double)p[j];
    float ys[D + 1];
#pragma unroll
    for (int r = 0; r <= D; ++r)
        ys[r] = 0.0f;
#pragma unroll
    for (int c = 0; c <= D; ++c) {
        double x = 0.0;
        if (c > 0)
            x = E.neg64[c - 1] * pd[c - 1];
#pragma unroll
        for (int j = c; j < D; ++j)
            x = __builtin_fma(E.pos64[j], pd[j], x);
        float y = (float)(x - (double)(s.q[c] * (D + 1))) * E.inv;
#pragma unroll
        for (int r = 0; r <= D; ++r)
            ys[r] = (s.rank[c] == r) ? y : ys[r];
    }
    b[0] = 1.0f + ys[D] - ys[0];
#pragma unroll
    for (int k = 1; k <= D; ++k)
        b[k] = ys[D - k] - ys[D + 1 - k];
}

__device__ __forceinline__ uint64_t mix64(uint64_t k)
{
    // MurmurHash3 64-bit finaliser
    k ^= k >> 33;
    k *= 0xff51afd7ed558ccdull;
    k ^= k >> 33;
    k *= 0xc4ceb9fe1a85ec53ull;
    k ^= k >> 33;
    return k;
}

// Packed key of simplex vertex k: every coordinate of vertex k is
// k + (d+1) t_c with t_c = q_c - [rank_c > d - k]; gfield carries the point
// group, already shifted into place.
template <int D>
__device__ __forceinline__ uint64_t pack_vertex(const Simplex<D> &s, int k, const KeyLayout &lay, uint64_t gfield)
{
    uint64_t key = (uint64_t)k | gfield;
#pragma unroll
    for (int c = 0; c < D; ++c) {
        int t = s.q[c] - ((s.rank[c] > D - k) ? 1 : 0);
        key |= (uint64_t)(uint32_t)(t - lay.lo[c]) << lay.shift[c];
    }
    return key;
}

// Group of point i of a batched build (binary search of the group starts),
// shifted into its key field.
__device__ __forceinline__ uint64_t group_field(const Groups64 &grp, const KeyLayout &lay, int64_t i)
{
    if (grp.G <= 1)
        return 0;
    int lo = 0, hi = grp.G;  // gstart[lo] <= i < gstart[hi]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (grp.gstart[mid] <= i)
            lo = mid;
        else
            hi = mid;
    }
    return (uint64_t)lo << lay.gshift;
}

inline unsigned blocks_for(int64_t count)
{
    return (unsigned)((count + kBlock - 1) / kBlock);
}

#define PAM_DISPATCH_D(d, CALL)                                                                   \
    switch (d) {                                                                                  \
    case 1: { constexpr int D = 1; CALL; } break;                                                 \
    case 2: { constexpr int D = 2; CALL; } break;                                                 \
    case 3: { constexpr int D = 3; CALL; } break;                                                 \
    case 4: { constexpr int D = 4; CALL; } break;                                                 \
    case 5: { constexpr int D = 5; CALL; } break;                                                 \
    case 6: { constexpr int D = 6; CALL; } break;                                                 \
    case 7: { constexpr int D = 7; CALL; } break;                                                 \
    case 8: { constexpr int D = 8; CALL; } break;                                                 \
    case 9: { constexpr int D = 9; CALL; } break;                                                 \
    case 10: { constexpr int D = 10; CALL; } break;                                               \
    case 11: { constexpr int D = 11; CALL; } break;                                               \
    case 12: { constexpr int D = 12; CALL; } break;                                               \
    case 13: { constexpr int D = 13; CALL; } break;                                               \
    case 14: { constexpr int D = 14; CALL; } break;                                               \
    case 15: { constexpr int D = 15; CALL; } break;                                               \
    case 16: { constexpr int D = 16; CALL; } break;                                               \
    default: return hipErrorInvalidValue;                                                         \
    }

}  // namespace pam

namespace pam {

// ---------------------------------------------------------------------------
// Tiles: the per-point filter kernels work on tiles of consecutive points,
// one block (one thread per point) per tile.
// ---------------------------------------------------------------------------

#ifndef PAM_TILE_POINTS
#define PAM_TILE_POINTS 512
#endif
#ifndef PAM_TILE_BIG_D
#define PAM_TILE_BIG_D 5  // largest d with PAM_TILE_POINTS-point tiles
#endif
#ifndef PAM_TILE_POINTS_HIGH_D
#define PAM_TILE_POINTS_HIGH_D 256  // tile points above PAM_TILE_BIG_D
#endif

// Tile order of the hash-table insert.  The hardware hands blocks to the 8
// XCDs in turn (block b to XCD b mod 8), each with its own L2.  Here each
// XCD takes a contiguous range of tiles instead, so that the table lines
// neighbouring tiles share stay in one L2 (the insert's probes load a slot
// before swapping it).  A bijection of [0, ntiles).  The other per-tile
// launches keep the launch order: for the resolve it sets the order of
// points within a vertex-0 bucket, which the splat's gathers follow.
#ifndef PAM_XCD_INSERT
#define PAM_XCD_INSERT 1
#endif
constexpr int kXcds = 8;

__device__ __forceinline__ int64_t xcd_tile(int64_t b, int64_t ntiles)
{
    const int64_t q = ntiles / kXcds, r = ntiles % kXcds;
    const int64_t x = b % kXcds, i = b / kXcds;
    return x * q + (x < r ? x : r) + i;
}

// this block's tile in the insert launch (blockIdx.x < ntiles)
__device__ __forceinline__ int64_t insert_tile(int64_t ntiles)
{
    return PAM_XCD_INSERT ? xcd_tile(blockIdx.x, ntiles) : (int64_t)blockIdx.x;
}

__host__ __device__ constexpr int tile_points(int d)
{
    return d <= PAM_TILE_BIG_D ? PAM_TILE_POINTS
                               : (PAM_TILE_POINTS < PAM_TILE_POINTS_HIGH_D ? PAM_TILE_POINTS : PAM_TILE_POINTS_HIGH_D);
}

// Per-tile view of the lattice.  The build writes one set of records for
// tiles of consecutive points (rowkey, lrow: the key dedup of the insert)
// and one for tiles of the simplex-sorted order (every field but rowkey),
// which the filter kernels read.  A sorted tile is cut into nwin windows of
// consecutive points.
// With nc = (points in the tile) * (d+1):
//   hdr    : nrows; flags (bit 0: the tile's vertices did not fit the LDS
//            dedup table, then only the per-point ids are valid) | nwin << 8;
//            nc; nseg
//   rowid  : nrows global vertex ids, one per distinct vertex of the tile
//   rowkey : nrows packed keys of those vertices (uint64)
//   sfirst : nwin * nrows + 1 first segment of each (window, row) pair,
//            window-major (uint16); the window-w segments of row r are
//            [sfirst[w nrows + r], sfirst[w nrows + r + 1])
//   seg    : nseg segments in (window, row) order, start | (length - 1) << 13
//            | row << 19 (uint32); a (window, row) pair's contributions are
//            cut into segments of at most kSegLen
//   order  : nseg segment indices (uint16), the work order: window by
//            window, longest first within a window (window 0's are the first
//            sfirst[nrows])
//   list   : nc entries (p << 5) | k sorted by (window, row): point p of the
//            tile contributes with its vertex k to that row (uint16); window
//            w's entries are contiguous
//   lrow   : nc rows, point-major: lrow[p * (d+1) + k] (uint16)
//   pent   : nwin * nrows + 1 first entry of each (window, row) pair in
//            list (uint16), window-major like sfirst
// Fixed-size records; offsets in bytes.
constexpr int kSegLen = 64;  // at most 64: the length field has 6 bits

__host__ __device__ constexpr uint32_t seg_encode(int start, int len, int row)
{
    return (uint32_t)start | ((uint32_t)(len - 1) << 13) | ((uint32_t)row << 19);
}
__device__ __forceinline__ void seg_decode(uint32_t sd, int &e0, int &e1, int &row)
{
    e0 = (int)(sd & 0x1fff);
    e1 = e0 + (int)((sd >> 13) & 63) + 1;
    row = (int)(sd >> 19);
}

// Points per window of a sorted tile: a (window, row) pair's contributions
// form their own segments, taken window by window.
#ifndef PAM_SPLAT_WINDOW
#define PAM_SPLAT_WINDOW 512
#endif
__host__ __device__ constexpr int splat_windows(int d)
{
    return tile_points(d) > PAM_SPLAT_WINDOW ? tile_points(d) / PAM_SPLAT_WINDOW : 1;
}

struct TileRec {
    int d, T, NC;
    size_t rowid, rowkey, sfirst, seg, order, list, lrow, pent, bytes;
    __host__ __device__ explicit TileRec(int d_) : d(d_)
    {
        T = tile_points(d_);
        NC = T * (d_ + 1);
        rowid = 16;
        rowkey = rowid + (((size_t)NC * 4 + 15) & ~(size_t)15);
        sfirst = rowkey + (size_t)NC * 8;
        seg = sfirst + (((size_t)(NC + 1) * 2 + 15) & ~(size_t)15);
        order = seg + (size_t)NC * 4;
        list = order + (((size_t)NC * 2 + 15) & ~(size_t)15);
        lrow = list + (((size_t)NC * 2 + 15) & ~(size_t)15);
        pent = lrow + (((size_t)NC * 2 + 15) & ~(size_t)15);
        bytes = (pent + (size_t)(NC + 1) * 2 + 255) & ~(size_t)255;
    }
};

constexpr uint32_t kTileOverflow = 1u;

// Per-point simplex record in sorted order: the d+1 barycentric weights
// (fp32) followed by the d+1 ranks (int8), padded to 16 bytes.
__host__ __device__ constexpr int point_bytes(int d) { return (5 * (d + 1) + 15) & ~15; }

// Runs of equal keys in consecutive lanes of a wave, for aggregating LDS
// and global atomics: the valid lanes must form a prefix of the wave.  Gives
// each valid lane the first lane of its run and the run's length.  Uses
// cross-lane operations: call in wave-uniform control flow only.
struct LaneRun {
    int lead;
    int len;
};

__device__ __forceinline__ LaneRun lane_run(uint64_t key, bool valid)
{
    const int lane = threadIdx.x & 63;
    const uint32_t lo = (uint32_t)key, hi = (uint32_t)(key >> 32);
    const uint32_t plo = __shfl_up(lo, 1), phi = __shfl_up(hi, 1);
    const bool start = valid && (lane == 0 || plo != lo || phi != hi);
    const uint64_t starts = __ballot(start);
    const uint64_t nvalid = __popcll(__ballot(valid));
    const uint64_t upto = lane == 63 ? ~0ull : ((2ull << lane) - 1);  // lanes 0..lane
    const uint64_t below = starts & upto, above = starts & ~upto;
    LaneRun r;
    r.lead = below ? 63 - __clzll(below) : lane;
    r.len = (above ? __ffsll((unsigned long long)above) - 1 : (int)nvalid) - r.lead;
    return r;
}

}  // namespace pam

namespace pam {

// Exclusive prefix sum of cnt[0..count) in LDS, in place; returns the total.
// Every thread of the block must call it; wsum is LDS scratch of
// blockDim.x / 64 + 1 ints.
__device__ __forceinline__ int block_exclusive_scan(int *cnt, int count, int *wsum)
{
    const int T = blockDim.x, t = threadIdx.x;
    const int per = (count + T - 1) / T;
    const int beg = min(t * per, count), end = min(beg + per, count);
    int s = 0;
    for (int i = beg; i < end; ++i)
        s += cnt[i];
    const int lane = t & 63, w = t >> 6;
    int x = s;
    for (int off = 1; off < 64; off <<= 1) {
        int y = __shfl_up(x, off);
        if (lane >= off)
            x += y;
    }
    if (lane == 63)
        wsum[w] = x;
    __syncthreads();
    if (t == 0) {
        int run = 0;
        for (int i = 0; i < T / 64; ++i) {
            int v = wsum[i];
            wsum[i] = run;
            run += v;
        }
        wsum[T / 64] = run;
    }
    __syncthreads();
    int excl = wsum[w] + x - s;
    for (int i = beg; i < end; ++i) {
        int v = cnt[i];
        cnt[i] = excl;
        excl += v;
    }
    const int total = wsum[T / 64];
    __syncthreads();
    return total;
}

// One pass over cnt[0..count): cnt becomes its exclusive prefix sum and
// nsg the exclusive prefix sum of ceil(cnt / len).  wsum holds
// 2 * (blockDim.x / 64 + 1) ints.  Returns the sum of ceil(cnt / len).
__device__ __forceinline__ int block_exclusive_scan_ceil(int *cnt, int *nsg, int count, int len, int *wsum)
{
    const int T = blockDim.x, t = threadIdx.x, NW = T / 64;
    const int per = (count + T - 1) / T;
    const int beg = min(t * per, count), end = min(beg + per, count);
    int s = 0, sg = 0;
    for (int i = beg; i < end; ++i) {
        const int c = cnt[i];
        s += c;
        sg += (c + len - 1) / len;
    }
    const int lane = t & 63, w = t >> 6;
    int x = s, xg = sg;
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off), yg = __shfl_up(xg, off);
        if (lane >= off) {
            x += y;
            xg += yg;
        }
    }
    if (lane == 63) {
        wsum[w] = x;
        wsum[NW + 1 + w] = xg;
    }
    __syncthreads();
    if (t == 0) {
        int run = 0, rung = 0;
        for (int i = 0; i < NW; ++i) {
            const int v = wsum[i], vg = wsum[NW + 1 + i];
            wsum[i] = run;
            wsum[NW + 1 + i] = rung;
            run += v;
            rung += vg;
        }
        wsum[NW] = run;
        wsum[2 * NW + 1] = rung;
    }
    __syncthreads();
    int excl = wsum[w] + x - s, exg = wsum[NW + 1 + w] + xg - sg;
    for (int i = beg; i < end; ++i) {
        const int c = cnt[i];
        cnt[i] = excl;
        nsg[i] = exg;
        excl += c;
        exg += (c + len - 1) / len;
    }
    const int total = wsum[2 * NW + 1];
    __syncthreads();
    return total;
}

}  // namespace pam

// HIP kernels (gfx950) of the permutohedral-lattice filter (Joutard et al.
// 2019, Section 2, eq. 6-8), for one lattice built by pam_build.hip:
//   splat      S: values times barycentric weights onto the lattice rows
//   blur       B: one lattice direction per launch, taps [1 2 1]
//   slice      Sl: weighted gather of each point's d+1 vertex rows
//   splat_bwd  S of dL/dv' and the slice-side half of eq. 8
//   slice_bwd  Sl for dL/dv (eq. 7) and the embedding gradient (eq. 8)
//
// The per-point kernels work on tiles of consecutive points of the
// simplex-sorted order the build prepared (points grouped by their vertex
// 0, so that a tile touches few lattice rows), one block per tile.  Phase A
// (one thread per point) stages the point's barycentric weights, ranks,
// vertex ids and original index in LDS.  Phase B maps a group of G lanes
// onto each point, lane l covering VEC consecutive channels of a chunk of up
// to 32 channels, so that value rows are read and written as whole (float4)
// rows at the point's original index, and the dot products of eq. 8 reduce
// inside the group with cross-lane shuffles.
//
// Splat kernels read the tile's view of the lattice prepared by the build
// (its distinct vertices as rows and its contributions sorted by row): lanes
// own whole rows and sum their contributions in registers from an LDS copy
// of the tile's values, and each row reaches the global lattice with one
// coalesced fp32 atomic per channel.  On gfx950 LDS float atomics cost about
// 3 cycles per lane, so no kernel accumulates with them.
#include "pam_device.h"

#include <type_traits>

namespace pam {

constexpr int kCH = 32;          // channels per pass over a tile

// compile-time flag for specialising a loop on a block-uniform condition
template <bool V>
using Flag = std::integral_constant<bool, V>;
template <int V>
using Int = std::integral_constant<int, V>;

template <int D>
struct Tile {
    static constexpr int T = tile_points(D);  // points (= threads) per tile
    static constexpr int NW = T / 64;         // waves per block
};

__device__ __forceinline__ void atomic_add_f32(float *p, float v)
{
    __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Cross-lane moves within rows of 16 lanes (DPP); lanes whose source lies
// outside the row read 0.
template <int CTRL>
__device__ __forceinline__ float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xb1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4e;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <- 7 - i within each 8 lanes
constexpr int kDppMirror = 0x140;     // lane i <- 15 - i within each 16 lanes
constexpr int kDppShr1 = 0x111, kDppShr2 = 0x112, kDppShr4 = 0x114, kDppShr8 = 0x118;
constexpr int kDppShl1 = 0x101;

// Orders the LDS accesses of one wave before and after it (lanes of a wave
// exchanging data through LDS).
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Sum over an aligned group of G lanes (a power of two), left in every lane
// of the group.  Call in wave-uniform control flow.
template <int G>
__device__ __forceinline__ float group_sum(float x)
{
    if constexpr (G >= 2)
        x += dpp<kDppXor1>(x);
    if constexpr (G >= 4)
        x += dpp<kDppXor2>(x);
    if constexpr (G >= 8)
        x += dpp<kDppHalfMirror>(x);
    if constexpr (G >= 16)
        x += dpp<kDppMirror>(x);
    if constexpr (G >= 32)
        x += __shfl_xor(x, 16);
    if constexpr (G >= 64)
        x += __shfl_xor(x, 32);
    return x;
}

// Inclusive prefix sum over the first N lanes of each group of G lanes
// (lane l of the group gets x_0 + ... + x_l; lanes past N are not
// meaningful).  Call in wave-uniform control flow.
template <int G, int N>
__device__ __forceinline__ float group_prefix(float x, int l)
{
    // the moves run in every lane (a lane reads its source lane's value,
    // which must be active); only the additions are selected
    if constexpr (G <= 16) {
        if constexpr (N > 1) {
            const float y = dpp<kDppShr1>(x);
            x += l >= 1 ? y : 0.0f;
        }
        if constexpr (N > 2) {
            const float y = dpp<kDppShr2>(x);
            x += l >= 2 ? y : 0.0f;
        }
        if constexpr (N > 4) {
            const float y = dpp<kDppShr4>(x);
            x += l >= 4 ? y : 0.0f;
        }
        if constexpr (N > 8) {
            const float y = dpp<kDppShr8>(x);
            x += l >= 8 ? y : 0.0f;
        }
    } else {
#pragma unroll
        for (int s = 1; s < N; s <<= 1) {
            const float y = __shfl_up(x, s, G);
            x += l >= s ? y : 0.0f;
        }
    }
    return x;
}

// Value of the next lane of the group (lanes 0 .. G-2).
template <int G>
__device__ __forceinline__ float group_next(float x)
{
    if constexpr (G <= 16)
        return dpp<kDppShl1>(x);
    else
        return __shfl_down(x, 1, G);
}

// Sums over an aligned group of G lanes (G = 2, 4 or 8) of each of the B
// values h[0 .. B) of every lane, spread over the group: afterwards lane l
// of the group holds in h[0 .. B/G) the sums of values l B/G .. l B/G +
// B/G - 1.  Each step pairs lanes that differ in one bit of l (for the top
// bit of an 8-lane group the pair is l and 7 - l, which differ in it) and
// keeps the half of the values selected by that bit.  Call in wave-uniform
// control flow.
template <int G, int B>
__device__ __forceinline__ void group_reduce_scatter(float (&h)[B], int l)
{
    static_assert(G == 2 || G == 4 || G == 8, "group of 2, 4 or 8 lanes");
    static_assert(B % G == 0, "values divide over the group");
    auto step = [&](auto ctrl, int n, bool hi) {
        constexpr int CTRL = decltype(ctrl)::value;
#pragma unroll
        for (int i = 0; i < B / 2; ++i) {
            if (i < n / 2) {
                const float keep = hi ? h[n / 2 + i] : h[i];
                const float send = hi ? h[i] : h[n / 2 + i];
                h[i] = keep + dpp<CTRL>(send);
            }
        }
    };
    int n = B;
    if constexpr (G >= 8) {
        step(std::integral_constant<int, kDppHalfMirror>{}, n, (l & 4) != 0);
        n /= 2;
    }
    if constexpr (G >= 4) {
        step(std::integral_constant<int, kDppXor2>{}, n, (l & 2) != 0);
        n /= 2;
    }
    step(std::integral_constant<int, kDppXor1>{}, n, (l & 1) != 0);
}

// Largest value over the wave (wave-uniform control flow only).
__device__ __forceinline__ int wave_max(int v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v = max(v, __shfl_xor(v, off));
    return v;
}

template <int VEC>
struct Vec {
    float v[VEC];
};

template <int VEC>
__device__ __forceinline__ Vec<VEC> load_vec(const float *__restrict__ p, bool ok)
{
    Vec<VEC> r;
    if constexpr (VEC == 4) {
        float4 x = ok ? *reinterpret_cast<const float4 *>(p) : make_float4(0.f, 0.f, 0.f, 0.f);
        r.v[0] = x.x;
        r.v[1] = x.y;
        r.v[2] = x.z;
        r.v[3] = x.w;
    } else {
        r.v[0] = ok ? *p : 0.0f;
    }
    return r;
}

template <int VEC>
__device__ __forceinline__ void store_vec(float *__restrict__ p, const Vec<VEC> &x)
{
    if constexpr (VEC == 4)
        *reinterpret_cast<float4 *>(p) = make_float4(x.v[0], x.v[1], x.v[2], x.v[3]);
    else
        *p = x.v[0];
}

// Row of original point i in the arrays of one side of the filter:
// kRowSource (val, grad_val: points [0, src_n)), kRowTarget (out, grad_out:
// points [tgt_0, n), row i - tgt_0), or -1 when the point has no row there.
// The symmetric filter has src_n = n and tgt_0 = 0 (every row is i).
constexpr int kRowNatural = -1, kRowSource = 0, kRowTarget = 1;
__device__ __forceinline__ int side_row(const FilterArgs &a, int64_t i, int side)
{
    if (side == kRowSource)
        return i < a.src_n ? (int)i : -1;
    if (side == kRowTarget)
        return i >= a.tgt_0 ? (int)(i - a.tgt_0) : -1;
    return (int)i;
}

// Phase A: one thread per point stages its barycentric weights and,
// optionally, its vertex ids, ranks and row (the original index mapped by
// side_row) in LDS (all from the build's sorted per-point records).
template <int D>
__device__ __forceinline__ void stage_points(const FilterArgs &a, int64_t base, int nt,
                                             float (*sb)[D + 1], int (*sm)[D + 1],
                                             signed char (*srank)[D + 1], int *sperm, int side = kRowNatural)
{
    constexpr int PW = point_bytes(D) / 4;
    const int t = threadIdx.x;
    if (t >= nt)
        return;
    const int64_t i = base + t;
    uint32_t w[PW];
    const uint4 *rec = reinterpret_cast<const uint4 *>(a.pts + i * (PW * 4));
#pragma unroll
    for (int u = 0; u < PW / 4; ++u) {
        const uint4 x = rec[u];
        w[4 * u] = x.x;
        w[4 * u + 1] = x.y;
        w[4 * u + 2] = x.z;
        w[4 * u + 3] = x.w;
    }
#pragma unroll
    for (int k = 0; k <= D; ++k)
        sb[t][k] = __uint_as_float(w[k]);
    if (sm) {
#pragma unroll
        for (int k = 0; k <= D; ++k)
            sm[t][k] = a.svert[i * (D + 1) + k];
    }
    if (srank) {
#pragma unroll
        for (int c = 0; c <= D; ++c)
            srank[t][c] = (signed char)((w[D + 1 + c / 4] >> (8 * (c % 4))) & 0xff);
    }
    if (sperm)
        sperm[t] = side_row(a, a.perm[i], side);
}

// Group geometry of phase B for one block (G = kCH / VEC lanes per point,
// so that a group covers kCH channels).
struct Groups {
    int G;      // lanes per point
    int l;      // lane within the group
    int first;  // first point of this lane's group in round 0
    int step;   // points per round for the whole block
    __device__ Groups(int G_, int nw)
    {
        G = G_;
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int P = 64 / G;
        l = lane & (G - 1);
        first = wave * P + lane / G;
        step = nw * P;
    }
};

// ---------------------------------------------------------------------------
// Splat (forward): L[m] += sum over the tile's points of b_k v.
//
// The build's per-tile view (TileRec) lists the tile's contributions sorted
// by row and cut into segments of at most kSegLen.  Segments are handed out
// longest first to groups of kSCH / VEC lanes (kSCH channels, VEC per
// lane).  A group sums b * x over its segment in registers, gathering each
// contribution's row of x straight from global memory (a sorted tile's rows
// are re-read d+1 times while they sit in the caches), kSplatBatch rows in
// flight at a time, and stores the sum in the segment's LDS slot; then each
// row's segment sums are added and reach the lattice with one coalesced fp32
// atomic per row and channel.  Nothing accumulates with LDS float atomics
// (on gfx950 they cost about 3 cycles per lane).
// ---------------------------------------------------------------------------

constexpr int kSCH = 32;        // channels per pass of the splat
constexpr int kSplatBatch = 8;  // contributions whose rows are requested together
constexpr int kSplatXsBytes = 16384;  // largest LDS copy of a pass's rows of x
constexpr int kXsSegCap = 768;        // segments whose tables the x-staged splat keeps in LDS

// segments whose partial sums stay in LDS
#ifndef PAM_SEG_CAP
#define PAM_SEG_CAP 192
#endif
#ifndef PAM_SEG_CAP_SMALL
#define PAM_SEG_CAP_SMALL 192
#endif
__host__ __device__ constexpr int seg_cap(int T) { return T >= 512 ? PAM_SEG_CAP : PAM_SEG_CAP_SMALL; }

#ifndef PAM_SPLAT_SPREAD
#define PAM_SPLAT_SPREAD 1  // splat threads per tile point
#endif
__host__ __device__ constexpr int splat_threads(int d) { return tile_points(d) * PAM_SPLAT_SPREAD; }

// Splat modes: x as given (forward, and the backward splat of dL/dv' in raw
// mode), or, for the normalised backward pass, x = g / z with the weight
// column taking b * gamma, or the augmented channels of the embedding
// gradient: d*C lattice channels, channel a*C + c taking f_a x_c (f the
// build's features).
constexpr int kSplatPlain = kSplatModePlain;
constexpr int kSplatNormBwd = kSplatModeNormBwd;
constexpr int kSplatAug = kSplatModeAug;

struct TileView {
    const uint32_t *hdr;
    const int32_t *rowid;
    const uint16_t *sfirst;
    const uint32_t *seg;
    const uint16_t *order;
    const uint16_t *list;
    const uint16_t *lrow;
    const uint16_t *pent;
};

template <int D>
__device__ __forceinline__ TileView tile_view(const uint8_t *tiles)
{
    const TileRec rec(D);
    const uint8_t *R = tiles + (size_t)blockIdx.x * rec.bytes;
    TileView v;
    v.hdr = reinterpret_cast<const uint32_t *>(R);
    v.rowid = reinterpret_cast<const int32_t *>(R + rec.rowid);
    v.sfirst = reinterpret_cast<const uint16_t *>(R + rec.sfirst);
    v.seg = reinterpret_cast<const uint32_t *>(R + rec.seg);
    v.order = reinterpret_cast<const uint16_t *>(R + rec.order);
    v.list = reinterpret_cast<const uint16_t *>(R + rec.list);
    v.lrow = reinterpret_cast<const uint16_t *>(R + rec.lrow);
    v.pent = reinterpret_cast<const uint16_t *>(R + rec.pent);
    return v;
}

// Block copy of `bytes` bytes (a multiple of 16 rounded up; both sides
// padded) from global to LDS in 16-byte pieces.
__device__ __forceinline__ void copy16(void *dst, const void *src, int bytes)
{
    const int n = (bytes + 15) / 16;
    for (int e = threadIdx.x; e < n; e += blockDim.x)
        reinterpret_cast<uint4 *>(dst)[e] = reinterpret_cast<const uint4 *>(src)[e];
}

// Tiles whose vertices did not fit the build's LDS table: each point adds
// its contributions to the lattice directly (one thread per point).
//   x row p is scaled by scale[p] when given; with `weights`, the weight
//   column C gets b * wcol[p] (b when wcol is null).
template <int D, bool AUG = false>
__device__ __forceinline__ void splat_direct(const FilterArgs &a, int64_t base, int nt, const float (*sb)[D + 1],
                                             const int *sperm, const float *__restrict__ x, const float *scale,
                                             bool weights, const float *wcol, float *__restrict__ L)
{
    const int C = a.c, ld = a.ld;
    for (int p = threadIdx.x; p < nt; p += blockDim.x) {
        if (sperm[p] < 0)
            continue;
        const float sc = scale ? scale[p] : 1.0f;
        const float *xr = x + (int64_t)sperm[p] * C;
        for (int k = 0; k <= D; ++k) {
            const int m = a.svert[(base + p) * (D + 1) + k];
            const float b = sb[p][k];
            float *row = L + (int64_t)m * ld;
            if constexpr (AUG) {
                const float *fr = a.feat + (int64_t)sperm[p] * D;
                for (int q = 0; q < D; ++q)
                    for (int c = 0; c < C; ++c)
                        atomic_add_f32(&row[q * C + c], b * fr[q] * xr[c]);
                continue;
            }
            for (int c = 0; c < C; ++c)
                atomic_add_f32(&row[c], b * sc * xr[c]);
            if (weights)
                atomic_add_f32(&row[C], b * (wcol ? wcol[p] : 1.0f));
        }
    }
}

constexpr int kRowPitch = kCH + 4;  // LDS pitch of a staged row (floats; spreads rows over banks)
constexpr int kSliceRows = 112;     // rows the forward slice stages
constexpr int kSliceBwdRows = 96;   // rows the backward slice stages, per lattice

// LDS copy of channels [cc, cc + kCH) of the tile's rows of L (zero beyond
// C), and of column C (the weight column) when wdst is given.
__device__ __forceinline__ void stage_rows(float *dst, float *wdst, const float *__restrict__ L,
                                           const int32_t *rowid, int nrows, int ld, int C, int cc)
{
    constexpr int Q = kCH / 4;
    for (int e = threadIdx.x; e < nrows * Q; e += blockDim.x) {
        const int r = e / Q, j = (e - r * Q) * 4;
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (cc + j < C)
            x = *reinterpret_cast<const float4 *>(L + (int64_t)rowid[r] * ld + cc + j);
        *reinterpret_cast<float4 *>(dst + r * kRowPitch + j) = x;
    }
    if (wdst) {
        for (int r = threadIdx.x; r < nrows; r += blockDim.x)
            wdst[r] = L[(int64_t)rowid[r] * ld + C];
    }
}

// VEC channels of a lattice row: the staged LDS copy (tile-local row m,
// column j of the chunk) or global memory (vertex id m, column cc + j).
template <bool STAGED, int VEC>
__device__ __forceinline__ Vec<VEC> lat_vec(const float *lds, const float *__restrict__ L, int m, int ld, int cc,
                                            int j)
{
    Vec<VEC> r;
    const float *p = STAGED ? lds + m * kRowPitch + j : L + (int64_t)m * ld + cc + j;
    if constexpr (VEC == 4) {
        const float4 x = *reinterpret_cast<const float4 *>(p);
        r.v[0] = x.x;
        r.v[1] = x.y;
        r.v[2] = x.z;
        r.v[3] = x.w;
    } else {
        r.v[0] = *p;
    }
    return r;
}

// Normalised backward prologue, per point p of the tile (a group of GL
// lanes per point): z_p = sum_k b_k Aw[m_k] and gamma_p = -<g_p, N_p> / z_p^2
// with N_p = sum_k b_k A[m_k]; leaves 1/z in sz and gamma in sgam.  When the
// tile's rows fit (`staged`), they are read from an LDS copy (rows, wrow;
// one kSCH-channel chunk at a time, the point's tile-local rows from the
// tile view), else from global memory.
template <int D, int VEC, int SCH>
__device__ __forceinline__ void norm_bwd_prologue(const FilterArgs &a, const TileView &tv, bool staged, float *rows,
                                                  float *wrow, int64_t base, int nt, const float (*sb)[D + 1],
                                                  const int *sperm, const float *__restrict__ g,
                                                  const float *__restrict__ A, float *sz, float *sgam)
{
    constexpr int GL = SCH / VEC;
    const int l = threadIdx.x & (GL - 1), q = threadIdx.x / GL, ng = blockDim.x / GL;
    const int C = a.c, ld = a.ld, nrows = (int)tv.hdr[0];
    auto chunk = [&](auto staged_flag, int cc) {
        constexpr bool S = decltype(staged_flag)::value;
        // uniform trip count for the whole block; the group reduction below
        // runs with every lane of the wave active
        for (int p0 = 0; p0 < (int)blockDim.x; p0 += ng) {
            const int p = p0 + q;
            const bool valid = p < nt && sperm[p] >= 0;
            const int pc = valid ? p : 0;
            int m[D + 1];
#pragma unroll
            for (int k = 0; k <= D; ++k)
                m[k] = S ? (int)tv.lrow[pc * (D + 1) + k] : a.svert[(base + pc) * (D + 1) + k];
            const bool on = valid && l * VEC < min(SCH, C - cc);
            const Vec<VEC> gv = load_vec<VEC>(g + (int64_t)sperm[pc] * C + cc + l * VEC, on);
            float dot = 0.0f;
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                Vec<VEC> ar;
                if (S)
                    ar = lat_vec<true, VEC>(rows, A, m[k], ld, cc, l * VEC);
                else
                    ar = load_vec<VEC>(A + (int64_t)m[k] * ld + cc + l * VEC, on);
                float dk = 0.0f;
#pragma unroll
                for (int u = 0; u < VEC; ++u)
                    dk += gv.v[u] * ar.v[u];
                dot += (valid ? sb[pc][k] : 0.0f) * dk;
            }
            dot = group_sum<GL>(dot);
            if (valid && l == 0) {
                if (cc == 0) {
                    float z = 0.0f;
#pragma unroll
                    for (int k = 0; k <= D; ++k)
                        z += sb[p][k] * (S ? wrow[m[k]] : A[(int64_t)m[k] * ld + C]);
                    sz[p] = z;
                    sgam[p] = dot;
                } else {
                    sgam[p] += dot;
                }
            }
        }
    };
    for (int cc = 0; cc < C; cc += SCH) {
        if (staged) {
            __syncthreads();  // the previous chunk's rows are consumed
            stage_rows(rows, cc == 0 ? wrow : nullptr, A, tv.rowid, nrows, ld, C, cc);
            __syncthreads();
            chunk(Flag<true>{}, cc);
        } else {
            chunk(Flag<false>{}, cc);
        }
    }
    __syncthreads();
    for (int p = threadIdx.x; p < nt; p += blockDim.x) {
        if (sperm[p] < 0) {  // no row of g: takes no part
            sz[p] = 0.0f;
            sgam[p] = 0.0f;
            continue;
        }
        const float z = sz[p];
        sz[p] = 1.0f / z;
        sgam[p] = -sgam[p] / (z * z);
    }
}

template <int D, int VEC, int MODE, int SCH, bool HA = false>
__global__ __launch_bounds__(splat_threads(D)) void k_splat(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                         const float *__restrict__ x, const float *__restrict__ A,
                                                         float *__restrict__ L, float *__restrict__ hA)
{
    static_assert(!HA || (MODE == kSplatPlain && VEC == 4), "eq. 8's term: plain mode, float4 rows");
    constexpr int T = tile_points(D);
    constexpr int NC = T * (D + 1);
    constexpr int GL = SCH / VEC;
    constexpr bool NORMB = MODE == kSplatNormBwd;
    constexpr bool AUG = MODE == kSplatAug;
    constexpr int NZ = NORMB ? T : 1;
    // XS, for tiles of 256 points (d > 5: many rows, few contributions
    // each) with passes of at most 16 channels: the pass's channels of
    // every point's row of x are copied to LDS once (thread t holds point
    // t's row), and the contributions read them there instead of gathering
    // each row d+1 times from global memory.  A row then has about one
    // segment, so segment sums go straight to the lattice (no LDS slots),
    // and the segment tables stay in LDS up to kXsSegCap segments.
    constexpr bool XS = (MODE == kSplatPlain || NORMB) && !HA && VEC == 4 && PAM_SPLAT_SPREAD == 1 && T == 256 &&
                        T * SCH * (int)sizeof(float) <= kSplatXsBytes;
    // AUG: a pass covers a chunk of SCH channels of x and every feature
    // coordinate at once (each row of x is gathered once per contribution,
    // not once per coordinate); its d * SCH sums per segment go straight to
    // the lattice like XS's.  DIRECT: no LDS slots for segment sums.
    constexpr bool DIRECT = XS || AUG;
    constexpr int SP = D + 1;  // AUG: LDS words per tile point (row of x, then its d features)
    // segment slots: narrower passes hold more segments' partial sums in
    // about the same LDS (at most 512, so that three blocks fit a CU)
    constexpr int kSegCapAll = seg_cap(T) * (kSCH / SCH) < 512 ? seg_cap(T) * (kSCH / SCH) : 512;
    constexpr int kSegCap = DIRECT ? 1 : kSegCapAll;
    constexpr int kTabCap = DIRECT ? kXsSegCap : kSegCap;  // segments whose tables are copied to LDS
    constexpr int B = AUG ? kSplatBatch / 2 : kSplatBatch;  // AUG: d accumulators per lane besides the rows
    // Per-point staging (weights, original index, and for the normalised
    // backward pass 1/z and gamma) is dead once the contributions are
    // decoded, so it shares LDS with the segment sums.
    constexpr size_t kPointBytes = sizeof(float) * T * (D + 1) + sizeof(int) * T + 2 * sizeof(float) * NZ;
    // DIRECT: per-wave scratch of the segment-sum transpose instead of slots
    constexpr int kXsWaveFloats = 64 * VEC + 64 / GL;
    constexpr size_t kSumBytes = DIRECT ? sizeof(float) * kXsWaveFloats * (splat_threads(D) / 64)
                                    : sizeof(float) * kSegCap * SCH + sizeof(float) * kSegCap;
    constexpr size_t kPoolBytes = (kPointBytes > kSumBytes ? kPointBytes : kSumBytes);
    // XS: the per-point staging lives in the LDS of the rows of x (it is
    // dead before they are copied), and the transpose scratch on its own
    constexpr size_t kXsFloats = T * SCH > (int)(kPointBytes / 4) ? T * SCH : (kPointBytes + 3) / 4;
    __shared__ __attribute__((aligned(16))) uint8_t pool[XS ? 16 : kPoolBytes];
    __shared__ __attribute__((aligned(16))) float xs[XS ? kXsFloats : 4];
    __shared__ __attribute__((aligned(16))) float xscratch[XS ? kSumBytes / 4 : 4];
    uint8_t *ppool = XS ? reinterpret_cast<uint8_t *>(xs) : pool;
    float(*sb)[D + 1] = reinterpret_cast<float(*)[D + 1]>(ppool);
    int *sperm = reinterpret_cast<int *>(ppool + sizeof(float) * T * (D + 1));
    float *sz = reinterpret_cast<float *>(ppool + sizeof(float) * T * (D + 1) + sizeof(int) * T);
    float *sgam = sz + NZ;
    float *Ps = XS ? xscratch : reinterpret_cast<float *>(pool);
    float *Pw = Ps + kSegCap * SCH;
    // one record per contribution in row order: weight (times 1/z in the
    // normalised backward pass) and the row of x; b * gamma for that pass.
    // Before the records are decoded, the normalised backward prologue keeps
    // the tile's lattice rows of A in the same LDS.
    constexpr size_t kRecBytes = DIRECT ? 16 : sizeof(int2) * NC;  // DIRECT: weights and points in recw / recp(16)
    constexpr size_t kRowsBytes = NORMB ? sizeof(float) * kSliceRows * (kRowPitch + 1) : 0;
    __shared__ __attribute__((aligned(16))) uint8_t recpool[kRecBytes > kRowsBytes ? kRecBytes : kRowsBytes];
    int2 *rec = reinterpret_cast<int2 *>(recpool);
    float *rowsA = reinterpret_cast<float *>(recpool), *wrowA = rowsA + kSliceRows * kRowPitch;
    __shared__ float recg[NORMB ? NC : 1];
    __shared__ float recw[DIRECT ? NC : 1];
    __shared__ uint8_t recp[XS ? NC : 1];
    static_assert(!XS || T <= 256, "point index in one byte");
    __shared__ uint16_t recp16[AUG ? NC : 1];
    __shared__ float spt[AUG ? T * SP : 1];
    __shared__ uint16_t lst_s[HA ? NC : 1];  // (point << 5) | k of every entry, for eq. 8's term
    __shared__ __attribute__((aligned(16))) uint32_t seg_s[kTabCap];
    __shared__ __attribute__((aligned(16))) uint16_t order_s[(kTabCap + 7) / 8 * 8];
    constexpr int kFirstCap = DIRECT ? 1 : 2 * kSegCap + 1;  // (window, row) pairs whose first segments stay in LDS
    __shared__ __attribute__((aligned(16))) uint16_t sfirst_s[(kFirstCap + 7) / 8 * 8];
    __shared__ int next_s;
    __shared__ __attribute__((aligned(16))) int32_t rowid_s[DIRECT ? kXsSegCap : 4];  // DIRECT: lattice row of each tile row

    const TileView tv = tile_view<D>(tiles);
    const int nrows = (int)tv.hdr[0], nc = (int)tv.hdr[2], nseg = (int)tv.hdr[3];
    const bool overflow = (tv.hdr[1] & kTileOverflow) != 0;
    const int nwin = (int)(tv.hdr[1] >> 8);
    const bool in_lds = nseg <= kTabCap && (DIRECT || nwin * nrows + 1 <= kFirstCap);
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const int C = a.c, ld = a.ld;
    const bool weights = !AUG && a.normalize != 0;  // weight column: b (plain) or b * gamma
    const float *scale = nullptr, *wcol = nullptr;
    // Set-up: every global load of this phase (the point's record and row,
    // the contributions this thread decodes, its 16-byte pieces of the
    // segment tables) is issued before the first wait, so that the block
    // waits for global memory once rather than once per array.
    constexpr int PW = point_bytes(D) / 4;
    constexpr int NJ = NC / T;  // contributions decoded per thread
    static_assert(kTabCap * 4 / 16 <= T && kFirstCap * 2 / 16 < T, "one table piece per thread");
    uint32_t w[PW];
    int prow = -1;
    if (t < nt) {
        const uint4 *rp = reinterpret_cast<const uint4 *>(a.pts + (base + t) * (PW * 4));
#pragma unroll
        for (int u = 0; u < PW / 4; ++u) {
            const uint4 q = rp[u];
            w[4 * u] = q.x;
            w[4 * u + 1] = q.y;
            w[4 * u + 2] = q.z;
            w[4 * u + 3] = q.w;
        }
        prow = side_row(a, a.perm[base + t], a.side);
    }
    uint32_t lst[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int e = t + j * T;
        lst[j] = (!overflow && e < nc) ? (uint32_t)tv.list[e] : 0u;
    }
    const bool tables = !overflow && in_lds;
    const int n0 = (nseg * 4 + 15) / 16, n1 = (nseg * 2 + 15) / 16, n2 = ((nwin * nrows + 1) * 2 + 15) / 16;
    const int n3 = (nrows * 4 + 15) / 16;  // every row has a segment: nrows <= nseg
    uint4 q0, q1, q2, q3;
    if (DIRECT && tables && t < n3)
        q3 = reinterpret_cast<const uint4 *>(tv.rowid)[t];
    if (tables && t < n0)
        q0 = reinterpret_cast<const uint4 *>(tv.seg)[t];
    if (tables && t < n1)
        q1 = reinterpret_cast<const uint4 *>(tv.order)[t];
    if (!DIRECT && tables && t < n2)
        q2 = reinterpret_cast<const uint4 *>(tv.sfirst)[t];
    if (t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k)
            sb[t][k] = __uint_as_float(w[k]);
        sperm[t] = prow;
    }
    if (tables) {
        if (t < n0)
            reinterpret_cast<uint4 *>(seg_s)[t] = q0;
        if (t < n1)
            reinterpret_cast<uint4 *>(order_s)[t] = q1;
        if (!DIRECT && t < n2)
            reinterpret_cast<uint4 *>(sfirst_s)[t] = q2;
        if (DIRECT && t < n3)
            reinterpret_cast<uint4 *>(rowid_s)[t] = q3;
    }
    __syncthreads();
    if constexpr (NORMB) {
        const bool staged = !overflow && nrows <= kSliceRows;
        norm_bwd_prologue<D, VEC, SCH>(a, tv, staged, rowsA, wrowA, base, nt, sb, sperm, x, A, sz, sgam);
        __syncthreads();
        scale = sz;
        wcol = sgam;
    }
    if (overflow) {
        splat_direct<D, AUG>(a, base, nt, sb, sperm, x, scale, weights, wcol, L);
        if constexpr (HA) {  // eq. 8's term of every contribution, 0 without a row of x
            for (int p = t; p < nt; p += (int)blockDim.x) {
                for (int k = 0; k <= D; ++k) {
                    float h = 0.0f;
                    if (sperm[p] >= 0) {
                        const float *xr = x + (int64_t)sperm[p] * C;
                        const float *Am = A + (int64_t)a.svert[(base + p) * (D + 1) + k] * ld;
                        for (int c = 0; c < C; ++c)
                            h += xr[c] * Am[c];
                    }
                    hA[(base + p) * (D + 1) + k] = h;
                }
            }
        }
        return;
    }
    // XS: thread t's point's row of x, channels [cc, cc + SCH) (zeros past
    // C and for points without a row), requested before the decode so that
    // the decode hides its latency, written to LDS after it
    float4 xrow[XS ? SCH / 4 : 1];
    auto load_x = [&](int cc) {
        if constexpr (XS) {
            const bool on = t < nt && prow >= 0;
#pragma unroll
            for (int q = 0; q < SCH / 4; ++q) {
                const int c = cc + 4 * q;
                xrow[q] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (on && c < C)
                    xrow[q] = *reinterpret_cast<const float4 *>(x + (int64_t)prow * C + c);
            }
        }
    };
    auto store_x = [&]() {
        if constexpr (XS) {
#pragma unroll
            for (int q = 0; q < SCH / 4; ++q)
                reinterpret_cast<float4 *>(xs + t * SCH)[q] = xrow[q];
        }
    };
    load_x(0);
    // AUG: thread t's point's features, requested before the decode and
    // written to LDS after it, next to its row of x (0 for no row: weight 0)
    float fpt[AUG ? D : 1];
    if constexpr (AUG) {
#pragma unroll
        for (int q = 0; q < D; ++q)
            fpt[q] = (t < nt && prow >= 0) ? a.feat[(int64_t)prow * D + q] : 0.0f;
    }
    // decode every contribution once (one thread each)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int e = t + j * T;
        if (e < nc) {
            const int pk = (int)lst[j];
            const int p = pk >> 5, k = pk & 31;
            const int r = sperm[p];  // -1: no row of x (weight 0, row 0 read)
            const float b = r >= 0 ? sb[p][k] : 0.0f;
            // (the fused eq. 8 term keeps -1 for "no row", to give those 0)
            if constexpr (XS) {
                recw[e] = scale ? b * scale[p] : b;
                recp[e] = (uint8_t)p;
            } else if constexpr (AUG) {
                recw[e] = b;
                recp16[e] = (uint16_t)p;
            } else {
                rec[e] = make_int2(__float_as_int(scale ? b * scale[p] : b), HA ? r : max(r, 0));
            }
            if constexpr (NORMB)
                recg[e] = b * wcol[p];
            if constexpr (HA)
                lst_s[e] = (uint16_t)pk;
        }
    }
    if constexpr (AUG) {
        if (t < nt) {
            spt[t * SP] = __int_as_float(max(prow, 0));
#pragma unroll
            for (int q = 0; q < D; ++q)
                spt[t * SP + 1 + q] = fpt[q];
        }
    }
    __syncthreads();
    constexpr int GPW = 64 / GL;  // groups per wave
    const int lane = t & 63, l = t & (GL - 1), gw = lane / GL;
    const uint32_t Cu = (uint32_t)C;
    // One pass over the tile's segments for channels [cc, cc + SCH).  IN_LDS:
    // segment table and (SUMS) partial sums in LDS (else the segment table
    // is read from the tile record and sums go straight to the lattice);
    // W: the weight column takes part.
    auto pass = [&](auto in_lds_flag, auto w_flag, int cc) {
        constexpr bool IN_LDS = decltype(in_lds_flag)::value;
        constexpr bool SUMS = IN_LDS && !XS;
        constexpr bool W = decltype(w_flag)::value;
        const int chc = min(SCH, C - cc);
        const bool lane_on = l * VEC < chc;
        const int col = min(cc + l * VEC, C - VEC);  // in bounds for every lane
        const float *xc = x + col;
        // Work is taken a wave at a time (one segment per group): the loop
        // and its exit are wave-uniform, so no cross-lane operation ever
        // runs in divergent control flow.
        for (;;) {
            int wbase = 0;
            if (lane == 0)
                wbase = atomicAdd(&next_s, GPW);
            wbase = __builtin_amdgcn_readfirstlane(wbase);
            if (wbase >= nseg)
                break;
            const int w = wbase + gw;
            if constexpr (HA) {
                // the loop's trip count is the wave's longest segment, so
                // that the group reductions of eq. 8's term run with every
                // lane active; entries past a group's segment weigh 0
                const bool gv = w < nseg;
                int sidx = 0, e0 = 0, e1 = 0, r = 0;
                if (gv) {
                    sidx = IN_LDS ? order_s[w] : tv.order[w];
                    seg_decode(IN_LDS ? seg_s[sidx] : tv.seg[sidx], e0, e1, r);
                }
                const int len = wave_max(e1 - e0);
                float4 Ar = make_float4(0.f, 0.f, 0.f, 0.f);
                if (gv && l * 4 < C)
                    Ar = *reinterpret_cast<const float4 *>(A + (int64_t)tv.rowid[r] * ld + l * 4);
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                constexpr int HB = B > GL ? B : GL;  // terms reduced per batch (padded with zeros)
                constexpr int R = HB / GL;           // terms each lane stores per batch
                for (int u = 0; u < len; u += B) {
                    int2 rr[B];
                    int pk[B];
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        const int e = max(min(e0 + u + j, e1 - 1), 0);
                        rr[j] = rec[e];
                        pk[j] = lst_s[e];
                    }
                    float bx[B];
                    float4 xv[B];
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        bx[j] = e0 + u + j < e1 ? __int_as_float(rr[j].x) : 0.0f;
                        xv[j] = *reinterpret_cast<const float4 *>(xc + (uint64_t)(uint32_t)max(rr[j].y, 0) * Cu);
                    }
                    float h[HB];
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        acc.x += bx[j] * xv[j].x;
                        acc.y += bx[j] * xv[j].y;
                        acc.z += bx[j] * xv[j].z;
                        acc.w += bx[j] * xv[j].w;
                        // a point without a row of x (the keys of the
                        // asymmetric filter's backward splat) has term 0
                        h[j] = rr[j].y >= 0 ? xv[j].x * Ar.x + xv[j].y * Ar.y + xv[j].z * Ar.z + xv[j].w * Ar.w
                                            : 0.0f;
                    }
#pragma unroll
                    for (int j = B; j < HB; ++j)
                        h[j] = 0.0f;
                    // <x_p, A_r> summed over the group: lane l keeps the
                    // terms of entries l R .. l R + R - 1 of the batch
                    group_reduce_scatter<GL, HB>(h, l);
#pragma unroll
                    for (int i = 0; i < R; ++i) {
                        const int jj = l * R + i;
                        int q = pk[0];
#pragma unroll
                        for (int j = 1; j < B; ++j)
                            q = jj == j ? pk[j] : q;
                        if (jj < B && e0 + u + jj < e1)
                            hA[(base + (q >> 5)) * (D + 1) + (q & 31)] = h[i];
                    }
                }
                if (gv) {
                    if constexpr (IN_LDS) {
                        reinterpret_cast<float4 *>(Ps + sidx * SCH)[l] = acc;
                    } else if (lane_on) {
                        float *row = L + (int64_t)tv.rowid[r] * ld + cc + l * 4;
                        atomic_add_f32(row + 0, acc.x);
                        atomic_add_f32(row + 1, acc.y);
                        atomic_add_f32(row + 2, acc.z);
                        atomic_add_f32(row + 3, acc.w);
                    }
                }
                continue;
            }
            Vec<VEC> acc;
#pragma unroll
            for (int u = 0; u < VEC; ++u)
                acc.v[u] = 0.0f;
            float accw = 0.0f;
            int xrow_id = -1;  // XS: the segment's lattice row (-1: no segment)
            if (w < nseg) {
                const int sidx = IN_LDS ? order_s[w] : tv.order[w];
                const uint32_t sd = IN_LDS ? seg_s[sidx] : tv.seg[sidx];
                int e0, e1, r;
                seg_decode(sd, e0, e1, r);
                if constexpr (XS)
                    xrow_id = IN_LDS ? rowid_s[r] : tv.rowid[r];
                for (int e = e0; e < e1; e += B) {
                    // B row requests issued together: entries past the
                    // segment's end re-read its last entry with weight 0
                    // (all reads unconditional, in stages, so that each
                    // stage's requests are in flight together)
                    int2 r[B];
#pragma unroll
                    for (int j = 0; j < B; ++j)
                        if constexpr (XS)
                            r[j] = make_int2(__float_as_int(recw[min(e + j, e1 - 1)]), (int)recp[min(e + j, e1 - 1)]);
                        else
                            r[j] = rec[min(e + j, e1 - 1)];
                    float bx[B], bw[B];
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        bx[j] = e + j < e1 ? __int_as_float(r[j].x) : 0.0f;
                        if constexpr (W)
                            bw[j] = NORMB ? (e + j < e1 ? recg[min(e + j, e1 - 1)] : 0.0f) : bx[j];
                    }
                    Vec<VEC> xv[B];
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        if constexpr (XS) {  // the point's row in LDS (lanes stay inside it: l * VEC < SCH)
                            const float4 q = reinterpret_cast<const float4 *>(xs + r[j].y * SCH)[l];
                            xv[j].v[0] = q.x;
                            xv[j].v[1] = q.y;
                            xv[j].v[2] = q.z;
                            xv[j].v[3] = q.w;
                        } else {
                            xv[j] = load_vec<VEC>(xc + (uint64_t)(uint32_t)r[j].y * Cu, true);
                        }
                    }
#pragma unroll
                    for (int j = 0; j < B; ++j) {
#pragma unroll
                        for (int u = 0; u < VEC; ++u)
                            acc.v[u] += bx[j] * xv[j].v[u];
                        if constexpr (W)
                            accw += bw[j];
                    }
                }
                if constexpr (SUMS) {
                    store_vec<VEC>(Ps + sidx * SCH + l * VEC, acc);
                    if (W && l == 0)
                        Pw[sidx] = accw;
                } else if constexpr (!XS) {
                    const int64_t row = (int64_t)tv.rowid[r] * ld;
                    if (lane_on) {
#pragma unroll
                        for (int u = 0; u < VEC; ++u)
                            atomic_add_f32(&L[row + cc + l * VEC + u], acc.v[u]);
                    }
                    if (W && l == 0)
                        atomic_add_f32(&L[row + C], accw);
                } else {
                    if (W && l == 0)
                        atomic_add_f32(&L[(int64_t)xrow_id * ld + C], accw);
                }
            }
            if constexpr (XS) {
                // The wave's segment sums reach the lattice through a
                // per-wave LDS transpose, so that each atomic instruction
                // covers whole rows (64 / SCH rows of SCH consecutive
                // channels) rather than VEC scattered floats of 64 / GL rows.
                float *wf = Ps + (t >> 6) * kXsWaveFloats;
                int *wrow = reinterpret_cast<int *>(wf + 64 * VEC);
                store_vec<VEC>(wf + gw * SCH + l * VEC, acc);
                if (l == 0)
                    wrow[gw] = xrow_id;
                wave_sync();
                const int c = lane % SCH;
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    const int g2 = i * (64 / SCH) + lane / SCH;  // group whose channel c this lane adds
                    const int row = wrow[g2];
                    if (row >= 0 && c < chc)
                        atomic_add_f32(&L[(int64_t)row * ld + cc + c], wf[g2 * SCH + c]);
                }
                wave_sync();  // the scratch is read before the next segments overwrite it
            }
        }
        __syncthreads();
        if constexpr (SUMS) {
            for (int e = t; e < nrows * SCH; e += (int)blockDim.x) {
                const int r = e / SCH, c = e - r * SCH;
                if (c >= chc)
                    continue;
                float sum = 0.0f;
                for (int w = 0; w < nwin; ++w)
                    for (int sx = sfirst_s[w * nrows + r]; sx < sfirst_s[w * nrows + r + 1]; ++sx)
                        sum += Ps[sx * SCH + c];
                atomic_add_f32(&L[(int64_t)tv.rowid[r] * ld + cc + c], sum);
            }
            if constexpr (W) {
                for (int r = t; r < nrows; r += (int)blockDim.x) {
                    float sum = 0.0f;
                    for (int w = 0; w < nwin; ++w)
                        for (int sx = sfirst_s[w * nrows + r]; sx < sfirst_s[w * nrows + r + 1]; ++sx)
                            sum += Pw[sx];
                    atomic_add_f32(&L[(int64_t)tv.rowid[r] * ld + C], sum);
                }
            }
        }
    };
    // AUG: one pass over the tile's segments for x channels [cc, cc + SCH)
    // and every feature coordinate q, lattice columns q*C + cc + c.  A
    // group accumulates d vectors per segment (b f_q x_c); each vector is
    // flushed through the wave's transpose scratch like XS's sums.
    auto pass_aug = [&](auto in_lds_flag, int cc) {
        constexpr bool IN_LDS = decltype(in_lds_flag)::value;
        const int chc = min(SCH, C - cc);
        const float *xc = x + min(cc + l * VEC, C - VEC);  // in bounds for every lane
        float *wf = Ps + (t >> 6) * kXsWaveFloats;
        int *wrow = reinterpret_cast<int *>(wf + 64 * VEC);
        const int cf = lane % SCH;  // the channel this lane flushes
        for (;;) {
            int wbase = 0;
            if (lane == 0)
                wbase = atomicAdd(&next_s, GPW);
            wbase = __builtin_amdgcn_readfirstlane(wbase);
            if (wbase >= nseg)
                break;
            const int w = wbase + gw;
            Vec<VEC> acc[D];
#pragma unroll
            for (int q = 0; q < D; ++q)
#pragma unroll
                for (int u = 0; u < VEC; ++u)
                    acc[q].v[u] = 0.0f;
            int xrow_id = -1;  // the segment's lattice row (-1: no segment)
            if (w < nseg) {
                const int sidx = IN_LDS ? order_s[w] : tv.order[w];
                const uint32_t sd = IN_LDS ? seg_s[sidx] : tv.seg[sidx];
                int e0, e1, r;
                seg_decode(sd, e0, e1, r);
                xrow_id = IN_LDS ? rowid_s[r] : tv.rowid[r];
                for (int e = e0; e < e1; e += B) {
                    // as in the other passes: B row requests together,
                    // entries past the end re-read the last with weight 0
                    int pj[B];
                    float bx[B];
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        const int ee = min(e + j, e1 - 1);
                        pj[j] = recp16[ee];
                        bx[j] = e + j < e1 ? recw[ee] : 0.0f;
                    }
                    Vec<VEC> xv[B];
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        const uint32_t xr = (uint32_t)__float_as_int(spt[pj[j] * SP]);
                        xv[j] = load_vec<VEC>(xc + (uint64_t)xr * Cu, true);
                    }
#pragma unroll
                    for (int j = 0; j < B; ++j) {
#pragma unroll
                        for (int q = 0; q < D; ++q) {
                            const float bf = bx[j] * spt[pj[j] * SP + 1 + q];
#pragma unroll
                            for (int u = 0; u < VEC; ++u)
                                acc[q].v[u] += bf * xv[j].v[u];
                        }
                    }
                }
            }
            if (l == 0)
                wrow[gw] = xrow_id;
#pragma unroll
            for (int q = 0; q < D; ++q) {
                store_vec<VEC>(wf + gw * SCH + l * VEC, acc[q]);
                wave_sync();
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    const int g2 = i * (64 / SCH) + lane / SCH;  // group whose channel cf this lane adds
                    const int row = wrow[g2];
                    if (row >= 0 && cf < chc)
                        atomic_add_f32(&L[(int64_t)row * ld + q * C + cc + cf], wf[g2 * SCH + cf]);
                }
                wave_sync();  // read before the next vector overwrites it
            }
        }
    };
    store_x();
    for (int cc = 0; cc < C; cc += SCH) {
        const bool wpass = weights && cc == 0;
        if (t == 0)
            next_s = 0;
        if (XS && cc > 0) {  // the previous pass ended with a barrier: xs is free
            load_x(cc);
            store_x();
        }
        __syncthreads();
        if constexpr (AUG) {
            if (in_lds)
                pass_aug(Flag<true>{}, cc);
            else
                pass_aug(Flag<false>{}, cc);
        } else if (in_lds) {
            if (wpass)
                pass(Flag<true>{}, Flag<true>{}, cc);
            else
                pass(Flag<true>{}, Flag<false>{}, cc);
        } else {
            if (wpass)
                pass(Flag<false>{}, Flag<true>{}, cc);
            else
                pass(Flag<false>{}, Flag<false>{}, cc);
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Blur: one direction, L'[m] = L[n-] + 2 L[m] + L[n+] (absent -> 0)
//
// A thread per (vertex, 4 channels): lattice rows are padded to ld, a
// multiple of 4 floats, and the buffers are 16-byte aligned, so every
// access is one float4 and a wave covers 16 whole 32-channel rows.  Each
// channel is computed with the same operations in the same order as a
// scalar evaluation, so results do not depend on the vector width.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float4 ld4(const float *__restrict__ p) { return *reinterpret_cast<const float4 *>(p); }

__device__ __forceinline__ float4 tap3(float4 lo, float4 mid, float4 hi, bool has_lo, bool has_hi)
{
    float4 acc = make_float4(2.0f * mid.x, 2.0f * mid.y, 2.0f * mid.z, 2.0f * mid.w);
    if (has_lo) {
        acc.x += lo.x;
        acc.y += lo.y;
        acc.z += lo.z;
        acc.w += lo.w;
    }
    if (has_hi) {
        acc.x += hi.x;
        acc.y += hi.y;
        acc.z += hi.z;
        acc.w += hi.w;
    }
    return acc;
}

__global__ __launch_bounds__(kBlock) void k_blur(const float *__restrict__ in, float *__restrict__ out,
                                                 const int32_t *__restrict__ nbr_j, int64_t M,
                                                 int32_t ld)
{
    const int q4 = ld >> 2;  // float4 per row
    const int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (e >= M * q4)
        return;
    const int64_t m = e / q4;
    const int c = (int)(e - m * q4) * 4;
    const int32_t lo = nbr_j[2 * m], hi = nbr_j[2 * m + 1];
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 a = ld4(in + m * ld + c);
    const float4 b = lo >= 0 ? ld4(in + (int64_t)lo * ld + c) : z;
    const float4 h = hi >= 0 ? ld4(in + (int64_t)hi * ld + c) : z;
    *reinterpret_cast<float4 *>(out + m * ld + c) = tap3(b, a, h, lo >= 0, hi >= 0);
}

// Two directions in one pass, out = B_jb(B_ja(in)): each output evaluates
// the three values of B_ja(in) it needs with the same operations as
// k_blur, so the result equals two separate passes bit for bit.  Worth it
// while the lattice stays in cache (the inner values are re-read).
__global__ __launch_bounds__(kBlock) void k_blur2(const float *__restrict__ in, float *__restrict__ out,
                                                  const int32_t *__restrict__ nbr_a,
                                                  const int32_t *__restrict__ nbr_b, int64_t M, int32_t ld)
{
    const int q4 = ld >> 2;
    const int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (e >= M * q4)
        return;
    const int64_t m = e / q4;
    const int c = (int)(e - m * q4) * 4;
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    const int32_t lo = nbr_b[2 * m], hi = nbr_b[2 * m + 1];
    // the (up to) three rows of the inner pass and their neighbours; every
    // load is issued before any arithmetic
    const int64_t r[3] = {lo, m, hi};
    int32_t ilo[3], ihi[3];
#pragma unroll
    for (int u = 0; u < 3; ++u) {
        const bool on = r[u] >= 0;
        ilo[u] = on ? nbr_a[2 * r[u]] : -1;
        ihi[u] = on ? nbr_a[2 * r[u] + 1] : -1;
    }
    float4 mid[3], nlo[3], nhi[3];
#pragma unroll
    for (int u = 0; u < 3; ++u) {
        mid[u] = r[u] >= 0 ? ld4(in + r[u] * ld + c) : z;
        nlo[u] = ilo[u] >= 0 ? ld4(in + (int64_t)ilo[u] * ld + c) : z;
        nhi[u] = ihi[u] >= 0 ? ld4(in + (int64_t)ihi[u] * ld + c) : z;
    }
    float4 inner[3];
#pragma unroll
    for (int u = 0; u < 3; ++u)
        inner[u] = tap3(nlo[u], mid[u], nhi[u], ilo[u] >= 0, ihi[u] >= 0);
    *reinterpret_cast<float4 *>(out + m * ld + c) = tap3(inner[0], inner[1], inner[2], lo >= 0, hi >= 0);
}

// ---------------------------------------------------------------------------
// Slice (forward): out_i = scale_i * sum_k b_k A[m_k]
//   raw: scale = 1/G_d;  normalised: scale = 1 / sum_k b_k Aw[m_k]
//
// One block per sorted tile.  Phase A (one thread per point) stages the
// point's weights, original index and tile-local rows in LDS with coalesced
// loads; in the same phase the block stages the tile's lattice rows (a
// sorted tile touches few of them) in LDS, pitch kRowPitch floats, when
// they fit.  Phase B maps a group of G lanes onto each point: the group
// gathers the point's d+1 rows (from LDS, or from global memory when the
// tile's rows were not staged) and writes the output row as whole float4
// pieces at the point's original index.  The choice between LDS and global
// rows is made once per block, outside the loops, so that the d+1 row
// reads of a point issue back to back.  Lattice rows are padded to ld (a
// multiple of 4 floats), so float4 reads that start below C stay inside
// the row; staged rows are zero beyond C.
// ---------------------------------------------------------------------------

// Phase A of the slice kernels: weights, original index, tile-local rows
// (when the tile's rows are staged) and ranks (when asked) of each point.
template <int D>
__device__ __forceinline__ void stage_slice_points(const FilterArgs &a, const TileView &tv, bool staged, int64_t base,
                                                   int nt, float (*sb)[D + 1], uint16_t (*slr)[D + 1],
                                                   signed char (*srank)[D + 1], int *sperm, int side = kRowNatural)
{
    stage_points<D>(a, base, nt, sb, nullptr, srank, sperm, side);
    const int t = threadIdx.x;
    if (staged && t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k)
            slr[t][k] = tv.lrow[t * (D + 1) + k];
    }
}

// Row index of vertex k of tile point p: tile-local when staged, else the
// global vertex id.
template <int D, bool STAGED>
__device__ __forceinline__ int point_row(const FilterArgs &a, const uint16_t (*slr)[D + 1], int64_t base, int p,
                                         int k)
{
    return STAGED ? (int)slr[p][k] : a.svert[(base + p) * (D + 1) + k];
}

// Staged rows of the slices, one pass of CH channels: pitch CH + 4 floats
// (narrow passes fit more rows in the same LDS), column CH of a row holding
// the weight column (normalised mode).  Tiles whose rows do not all fit read
// every row from global memory.
constexpr int kStageNone = 0, kStageFull = 1;

template <int CH>
__device__ __forceinline__ void stage_rows_p(float *dst, const float *__restrict__ L, const int32_t *rowid, int nst,
                                             int ld, int C, int cc, bool weights)
{
    constexpr int P = CH + 4, Q = CH / 4;
    for (int e = threadIdx.x; e < nst * Q; e += blockDim.x) {
        const int r = e / Q, j = (e - r * Q) * 4;
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (cc + j < C)
            x = *reinterpret_cast<const float4 *>(L + (int64_t)rowid[r] * ld + cc + j);
        *reinterpret_cast<float4 *>(dst + r * P + j) = x;
    }
    if (weights) {
        for (int r = threadIdx.x; r < nst; r += blockDim.x)
            dst[r * P + CH] = L[(int64_t)rowid[r] * ld + C];
    }
}

template <int VEC>
__device__ __forceinline__ Vec<VEC> vec_at(const float *p)
{
    Vec<VEC> r;
    if constexpr (VEC == 4) {
        const float4 x = *reinterpret_cast<const float4 *>(p);
        r.v[0] = x.x;
        r.v[1] = x.y;
        r.v[2] = x.z;
        r.v[3] = x.w;
    } else {
        r.v[0] = *p;
    }
    return r;
}

// VEC channels at offset j of pass cc of a point's vertex row: tile-local
// row ml (staged) or global vertex id mg.
template <int VEC, int CH, int MODE>
__device__ __forceinline__ Vec<VEC> stage_vec(const float *lds, const float *__restrict__ L, int ml, int mg, int ld,
                                              int cc, int j)
{
    if constexpr (MODE == kStageFull)
        return vec_at<VEC>(lds + ml * (CH + 4) + j);
    else
        return vec_at<VEC>(L + (int64_t)mg * ld + cc + j);
}

// Weight column of a vertex row (normalised mode), staged or global.
template <int CH, int MODE>
__device__ __forceinline__ float stage_w(const float *lds, const float *__restrict__ L, int ml, int mg, int ld, int C)
{
    if constexpr (MODE == kStageFull)
        return lds[ml * (CH + 4) + CH];
    else
        return L[(int64_t)mg * ld + C];
}

template <int D, int VEC, int CH>
__global__ __launch_bounds__(Tile<D>::T) void k_slice(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                      const float *__restrict__ A, float *__restrict__ out)
{
    constexpr int T = Tile<D>::T;
    constexpr int kFloats = kSliceRows * kRowPitch;
    constexpr int RS = kFloats / (CH + 4);  // rows the LDS holds
    __shared__ float sb[T][D + 1];
    __shared__ uint16_t slr[T][D + 1];
    __shared__ int sperm[T];
    __shared__ __attribute__((aligned(16))) float rows[kFloats];
    const TileView tv = tile_view<D>(tiles);
    const int nrows = (int)tv.hdr[0];
    const bool ovf = (tv.hdr[1] & kTileOverflow) != 0;
    const int C = a.c, ld = a.ld;
    const bool full = !ovf && nrows <= RS;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    stage_slice_points<D>(a, tv, full, base, nt, sb, slr, nullptr, sperm, kRowTarget);
    const Groups gr(CH / VEC, Tile<D>::NW);
    auto rounds = [&](auto mode_flag, int cc) {
        constexpr int MODE = decltype(mode_flag)::value;
        const bool lane_on = gr.l * VEC < min(CH, C - cc);
        if (!lane_on)
            return;
        for (int p = gr.first; p < nt; p += gr.step) {
            int ml[D + 1], mg[D + 1];
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                ml[k] = MODE != kStageNone ? (int)slr[p][k] : 0;
                mg[k] = MODE != kStageFull ? a.svert[(base + p) * (D + 1) + k] : 0;
            }
            float sc = a.E.raw_scale;
            if (a.normalize) {
                float z = 0.0f;
#pragma unroll
                for (int k = 0; k <= D; ++k)
                    z += sb[p][k] * stage_w<CH, MODE>(rows, A, ml[k], mg[k], ld, C);
                sc = 1.0f / z;
            }
            Vec<VEC> o;
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                o.v[j] = 0.0f;
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                const Vec<VEC> r = stage_vec<VEC, CH, MODE>(rows, A, ml[k], mg[k], ld, cc, gr.l * VEC);
                const float bk = sb[p][k];
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    o.v[j] += bk * r.v[j];
            }
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                o.v[j] *= sc;
            if (sperm[p] >= 0)
                store_vec<VEC>(out + (int64_t)sperm[p] * C + cc + gr.l * VEC, o);
        }
    };
    for (int cc = 0; cc < C; cc += CH) {
        if (full) {
            if (cc > 0)
                __syncthreads();
            stage_rows_p<CH>(rows, A, tv.rowid, nrows, ld, C, cc, a.normalize && cc == 0);
        }
        __syncthreads();
        if (full)
            rounds(Int<kStageFull>{}, cc);
        else
            rounds(Int<kStageNone>{}, cc);
    }
}

// ---------------------------------------------------------------------------
// Augmented-channel embedding gradient (raw mode).  With W = s_d Sl B S,
// the blurred lattices A = B S v and At = B~ S g of eq. 6-7, and the
// blurred lattices of the augmented channels L1 = B S(f (x) v) and
// L2 = B~ S(f (x) g) (d*C channels, column q*C + c), point i gets
//   df_iq = s_d [ sum_c g_ic Sl(L1)_i,qC+c + v_ic Sl(L2)_i,qC+c
//                 - f_iq sum_c (g_ic Sl(A)_ic + v_ic Sl(At)_ic) ],
// the gradient of sum_i <g_i, sum_j exp(-|f_i - f_j|^2 / 2) v_j> with each
// Gaussian sum replaced by the lattice filter.
//
// Row-major, like the splat: the tile's contributions are walked segment by
// segment (a segment: one lattice row m and a run of the points that have
// it as a vertex).  A group of GL lanes holds row m of every lattice in
// registers (VEC channels per lane and lattice) and, per contribution
// (p, k), gathers the point's rows of g and v, so that a lattice row is read
// once per segment rather than once per point.  Per contribution it forms
// the d+1 values b_k <g_p, X[m]> + b_k <v_p, Y[m]> (value 0: X, Y = A, At;
// value 1 + q: the q-th column block of L1, L2) and writes them to the
// contribution's LDS slot (no LDS atomics: each slot has one writer per
// pass); after the last pass each point adds its d+1 slots, found through a
// map from (point, vertex) to entry.
// Slots hold NVC values (all d+1 unless the tile's slots would not fit
// LDS; then the values are taken NVC at a time, g and v re-gathered per
// chunk).  Tiles whose vertices overflowed the build's table take a
// thread-per-point path from global memory.
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int slice_aug_threads(int d) { return d <= PAM_TILE_BIG_D ? 1024 : 512; }
__host__ __device__ constexpr int slice_aug_nvc(int d)
{
    // values per slot: at most about 96 KB of slots per tile
    return (d + 1) * tile_points(d) * (d + 1) * 4 <= 98304 ? d + 1 : 98304 / (tile_points(d) * (d + 1) * 4);
}
__host__ __device__ constexpr int pow2_at_least(int x) { return x <= 1 ? 1 : 2 * pow2_at_least((x + 1) / 2); }

template <int D, int VEC, int SCH>
__global__ __launch_bounds__(slice_aug_threads(D)) void k_slice_aug(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                                    const float *__restrict__ val,
                                                                    const float *__restrict__ grad,
                                                                    const float *__restrict__ A,
                                                                    const float *__restrict__ At,
                                                                    const float *__restrict__ L1,
                                                                    const float *__restrict__ L2, int32_t ldq,
                                                                    float *__restrict__ grad_feat)
{
    constexpr int T = tile_points(D);
    constexpr int NT = slice_aug_threads(D);
    constexpr int NC = T * (D + 1);
    constexpr int NV = D + 1;              // values per contribution
    constexpr int NVC = slice_aug_nvc(D);  // values per slot (per chunk)
    constexpr int GL = SCH / VEC, GPW = 64 / GL;
    constexpr int HB = pow2_at_least(NVC > GL ? NVC : GL);  // values reduced per contribution (zero padded)
    constexpr int B = 4;                                     // contributions whose rows are requested together
    constexpr int kTab = kXsSegCap;
    static_assert(NVC >= 1 && (long)NC * NVC * 4 <= 98304, "slots fit LDS");
    static_assert(GL > 8 || HB % GL == 0, "values divide over the group");
    __shared__ __attribute__((aligned(16))) float res[NC * NVC];  // before the decode: the point staging
    __shared__ int2 rec[NC];         // per entry: weight, row of g and v
    __shared__ uint16_t emap[NC];    // entry of (point p, vertex k) at p (d+1) + k
    __shared__ int sperm[T];
    __shared__ float sod[T];  // per point: sum over its vertices of value 0
    __shared__ __attribute__((aligned(16))) uint32_t seg_s[kTab];
    __shared__ __attribute__((aligned(16))) uint16_t order_s[kTab];
    __shared__ __attribute__((aligned(16))) int32_t rowid_s[kTab];
    __shared__ int next_s;
    static_assert(sizeof(float) * T * (D + 1) <= sizeof(float) * NC * NVC, "point staging fits the slots");
    float(*sb)[D + 1] = reinterpret_cast<float(*)[D + 1]>(res);

    const TileView tv = tile_view<D>(tiles);
    const int nrows = (int)tv.hdr[0], nc = (int)tv.hdr[2], nseg = (int)tv.hdr[3];
    const bool overflow = (tv.hdr[1] & kTileOverflow) != 0;
    const bool in_lds = !overflow && nseg <= kTab;
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const int C = a.c, ld = a.ld;
    const float s = a.E.raw_scale;
    stage_points<D>(a, base, nt, sb, nullptr, nullptr, sperm);  // threads t < nt
    if (in_lds) {
        for (int e = t; e < nseg; e += NT) {
            seg_s[e] = tv.seg[e];
            order_s[e] = tv.order[e];
        }
        for (int e = t; e < nrows; e += NT)
            rowid_s[e] = tv.rowid[e];
    }
    __syncthreads();
    if (overflow) {
        // a thread per point, every row read from global memory
        for (int p = t; p < nt; p += NT) {
            const int64_t row = sperm[p];
            if (row < 0)
                continue;
            float hq[D], h0 = 0.0f;
#pragma unroll
            for (int q = 0; q < D; ++q)
                hq[q] = 0.0f;
            for (int k = 0; k <= D; ++k) {
                const int64_t m = a.svert[(base + p) * (D + 1) + k];
                const float b = sb[p][k];
                for (int c = 0; c < C; ++c) {
                    const float gc = b * grad[row * C + c], vc = b * val[row * C + c];
                    h0 += gc * A[m * ld + c] + vc * At[m * ld + c];
#pragma unroll
                    for (int q = 0; q < D; ++q)
                        hq[q] += gc * L1[m * ldq + q * C + c] + vc * L2[m * ldq + q * C + c];
                }
            }
#pragma unroll
            for (int q = 0; q < D; ++q)
                grad_feat[row * D + q] = s * (hq[q] - a.feat[row * D + q] * h0);
        }
        return;
    }
    // decode every contribution once: its weight (0 for a point without a
    // row) and row; its slot is its entry
    for (int e = t; e < nc; e += NT) {
        const int pk = tv.list[e];
        const int p = pk >> 5, k = pk & 31;
        const int r = sperm[p];
        rec[e] = make_int2(__float_as_int(r >= 0 ? sb[p][k] : 0.0f), max(r, 0));
        emap[p * (D + 1) + k] = (uint16_t)e;
    }
    __syncthreads();  // the point staging is dead from here: res takes the slots
    const int lane = t & 63, l = t & (GL - 1), gw = lane / GL;
    // One pass over the tile's segments for values [v0, v0 + NVC) and value
    // channels [cc, cc + SCH); the first channel pass writes the slots, later
    // ones add to them.
    auto pass = [&](auto in_lds_flag, int v0, int cc) {
        constexpr bool IN_LDS = decltype(in_lds_flag)::value;
        const int chc = min(SCH, C - cc);
        const bool lane_on = l * VEC < chc;
        const int col = min(cc + l * VEC, C - VEC);  // in bounds for every lane
        const bool first = cc == 0;
        for (;;) {
            int wbase = 0;
            if (lane == 0)
                wbase = atomicAdd(&next_s, GPW);
            wbase = __builtin_amdgcn_readfirstlane(wbase);
            if (wbase >= nseg)
                break;
            const int w = wbase + gw;
            int e0 = 0, e1 = 0;
            int64_t m = 0;
            if (w < nseg) {
                const int sidx = IN_LDS ? order_s[w] : tv.order[w];
                int r;
                seg_decode(IN_LDS ? seg_s[sidx] : tv.seg[sidx], e0, e1, r);
                m = IN_LDS ? rowid_s[r] : tv.rowid[r];
            }
            // row m of each lattice pair, this lane's channels (0 where the
            // lane is past the chunk, for values past d, and without a segment)
            Vec<VEC> rx[NVC], ry[NVC];
#pragma unroll
            for (int i = 0; i < NVC; ++i) {
                const int vi = v0 + i;
                const bool on = w < nseg && lane_on && vi < NV;
                const float *X = vi == 0 ? A + m * ld + col : L1 + m * ldq + (vi - 1) * C + col;
                const float *Y = vi == 0 ? At + m * ld + col : L2 + m * ldq + (vi - 1) * C + col;
                rx[i] = load_vec<VEC>(on ? X : A, on);
                ry[i] = load_vec<VEC>(on ? Y : At, on);
            }
            // wave-uniform trip count (the group reductions run with every
            // lane active); entries past a group's segment weigh 0
            const int len = wave_max(e1 - e0);
            for (int u = 0; u < len; u += B) {
                int2 rj[B];
#pragma unroll
                for (int j = 0; j < B; ++j)
                    rj[j] = rec[max(min(e0 + u + j, e1 - 1), 0)];
                Vec<VEC> gq[B], vq[B];
#pragma unroll
                for (int j = 0; j < B; ++j) {
                    const uint64_t off = (uint64_t)(uint32_t)rj[j].y * (uint32_t)C + col;
                    gq[j] = load_vec<VEC>(grad + off, true);
                    vq[j] = load_vec<VEC>(val + off, true);
                }
#pragma unroll
                for (int j = 0; j < B; ++j) {
                    float h[HB];
#pragma unroll
                    for (int i = 0; i < HB; ++i) {
                        float x = 0.0f;
                        if (i < NVC) {
                            // one fused multiply-add per product
#pragma unroll
                            for (int uu = 0; uu < VEC; ++uu) {
                                x = fmaf(gq[j].v[uu], rx[i].v[uu], x);
                                x = fmaf(vq[j].v[uu], ry[i].v[uu], x);
                            }
                        }
                        h[i] = x;
                    }
                    const bool live = e0 + u + j < e1;
                    const float bx = __int_as_float(rj[j].x);
                    float *slot = res + (e0 + u + j) * NVC;
                    if constexpr (GL <= 8) {
                        // lane l keeps the sums of values l R .. l R + R - 1
                        constexpr int R = HB / GL;
                        group_reduce_scatter<GL, HB>(h, l);
#pragma unroll
                        for (int i = 0; i < R; ++i) {
                            const int vi = l * R + i;
                            if (live && vi < NVC)
                                slot[vi] = first ? bx * h[i] : slot[vi] + bx * h[i];
                        }
                    } else {
                        float mine = 0.0f;
#pragma unroll
                        for (int i = 0; i < NVC; ++i) {
                            const float y = group_sum<GL>(h[i]);
                            mine = l == i ? y : mine;
                        }
                        if (live && l < NVC)
                            slot[l] = first ? bx * mine : slot[l] + bx * mine;
                    }
                }
            }
        }
    };
    for (int v0 = 0; v0 < NV; v0 += NVC) {
        for (int cc = 0; cc < C; cc += SCH) {
            if (t == 0)
                next_s = 0;
            __syncthreads();
            if (in_lds)
                pass(Flag<true>{}, v0, cc);
            else
                pass(Flag<false>{}, v0, cc);
            __syncthreads();
        }
        // each point adds its d+1 slots: value 0 first (kept per point),
        // then df_q = s (value 1 + q - f_q value 0)
        for (int p = t; p < nt; p += NT) {
            const int64_t row = sperm[p];
            if (row < 0)
                continue;
            for (int i = 0; i < NVC && v0 + i < NV; ++i) {
                float h = 0.0f;
#pragma unroll
                for (int k = 0; k <= D; ++k)
                    h += res[emap[p * (D + 1) + k] * NVC + i];
                const int vi = v0 + i;
                if (vi == 0)
                    sod[p] = h;
                else
                    grad_feat[row * D + vi - 1] = s * (h - a.feat[row * D + vi - 1] * sod[p]);
            }
        }
        __syncthreads();  // the slots are read before the next chunk writes them
    }
}

// ---------------------------------------------------------------------------
// Backward slice: dL/dv = sc * sum_k b_k At[m_k] (eq. 7; sc = 1/G_d raw, 1
// normalised) and the embedding gradient of eq. (8).  With h_k = dL/db_k:
//   raw:        h_k = s_d (<g_i, A[m_k]> + <v_i, At[m_k]>)
//   normalised: z = sum_k b_k Aw[m_k], gamma = -sum_k b_k <g_i, A[m_k]> / z^2,
//               h_k = <g_i, A[m_k]> / z + gamma Aw[m_k] + <v_i, At[m_k]> + Atw[m_k]
// (A, Aw: the forward's blurred lattice and weight column; At, Atw: the
// reversed blur of the splat of g/z and of gamma), then
//   gx_c = (h[d - rank_c] - h[(d + 1 - rank_c) mod (d+1)]) / (d+1),
//   df_i = E^T gx.
// Phase A as in the forward slice (plus ranks); the tile's rows of At and A
// are staged when there is a single chunk of channels and they fit.  In
// phase B a group of G lanes handles a point through all its channels,
// keeping per-lane partial dot products, reduces them once, and finishes
// the point's embedding gradient itself.  Lanes past the tile's end or past
// C read clamped in-bounds data and are masked at the stores.
// ---------------------------------------------------------------------------

// Embedding gradient of one point (eq. 8) from h_k = dL/db_k, held by
// every lane of its group of G lanes: with H[r] = h[d - r] -
// h[(d + 1 - r) mod (d+1)] and gx_c = H[rank_c] / (d+1),
//   df_l = pos[l] (gx_0 + ... + gx_l) + neg[l] gx_{l+1}.
// Call in wave-uniform control flow (cross-lane steps); `valid` masks the
// stores.
template <int D, int G>
__device__ __forceinline__ void eq8_finish(const FilterArgs &a, const signed char *rank, const float *h, bool valid,
                                           float *frow, int l, float my_pos, float my_neg)
{
    float H[D + 1];
#pragma unroll
    for (int r = 0; r <= D; ++r)
        H[r] = h[D - r] - h[(D + 1 - r) % (D + 1)];
    if constexpr (D + 1 <= G) {
        // lane l <= d finishes coordinate l
        const int rl = rank[min(l, D)];
        float Hl = 0.0f;
#pragma unroll
        for (int r = 0; r <= D; ++r)
            Hl = rl == r ? H[r] : Hl;
        const float gx = l <= D ? Hl * a.E.inv : 0.0f;
        const float nxt = group_next<G>(gx);
        const float pre = group_prefix<G, D + 1>(gx, l);
        if (valid && l < D)
            frow[l] = my_pos * pre + my_neg * nxt;
    } else {
        // every lane evaluates all coordinates; the group's lanes share the
        // stores
        float gx[D + 1];
#pragma unroll
        for (int c = 0; c <= D; ++c) {
            const int rc = rank[c];
            float Hc = 0.0f;
#pragma unroll
            for (int r = 0; r <= D; ++r)
                Hc = rc == r ? H[r] : Hc;
            gx[c] = Hc * a.E.inv;
        }
        float prefix = 0.0f;
#pragma unroll
        for (int j = 0; j < D; ++j) {
            prefix += gx[j];
            if (valid && (j & (G - 1)) == l)
                frow[j] = a.E.pos[j] * prefix + a.E.neg[j] * gx[j + 1];
        }
    }
}

template <int D, int VEC, bool NORM, bool ASYM, int CH, bool HAIN>
__global__ __launch_bounds__(Tile<D>::T) void k_slice_bwd(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                          const float *__restrict__ val,
                                                          const float *__restrict__ grad,
                                                          const float *__restrict__ A,
                                                          const float *__restrict__ At,
                                                          const float *__restrict__ hA,
                                                          float *__restrict__ grad_val,
                                                          float *__restrict__ grad_feat)
{
    static_assert(!(HAIN && NORM), "the splat's <g, A_k> is taken in raw mode");
    constexpr int T = Tile<D>::T;
    constexpr int RB = kSliceBwdRows * kRowPitch / (CH + 4);  // rows the LDS holds, per lattice
    __shared__ float sb[T][D + 1];
    __shared__ uint16_t slr[T][D + 1];
    __shared__ signed char srank[T][D + 1];
    __shared__ int sperm[T];
    __shared__ __attribute__((aligned(16))) float rowsT[kSliceBwdRows * kRowPitch];
    __shared__ __attribute__((aligned(16))) float rowsA[kSliceBwdRows * kRowPitch];
    const TileView tv = tile_view<D>(tiles);
    const int nrows = (int)tv.hdr[0];
    const int C = a.c, ld = a.ld;
    // the tile's rows are staged (all C channels at once) when they fit
    const bool full = !(tv.hdr[1] & kTileOverflow) && C <= CH && nrows <= RB;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const float sc = NORM ? 1.0f : a.E.raw_scale;
    const bool want_f = grad_feat != nullptr;
    stage_slice_points<D>(a, tv, full, base, nt, sb, slr, want_f ? srank : nullptr, sperm);
    if (full) {
        stage_rows_p<CH>(rowsT, At, tv.rowid, nrows, ld, C, 0, NORM);
        if (want_f && !HAIN)
            stage_rows_p<CH>(rowsA, A, tv.rowid, nrows, ld, C, 0, NORM);
    }
    __syncthreads();
    constexpr int G = CH / VEC;
    const Groups gr(G, Tile<D>::NW);
    // eq. 8 coefficients of this lane's coordinate (lane l of a group
    // finishes coordinate l when the group has at least d+1 lanes)
    float my_pos = 0.0f, my_neg = 0.0f;
#pragma unroll
    for (int j = 0; j < D; ++j) {
        my_pos = gr.l == j ? a.E.pos[j] : my_pos;
        my_neg = gr.l == j ? a.E.neg[j] : my_neg;
    }
    auto rounds = [&](auto mode_flag, auto feat_flag) {
        constexpr int MODE = decltype(mode_flag)::value;
        constexpr bool F = decltype(feat_flag)::value;
        // The first CH channels of a round's value and gradient rows are
        // requested one round ahead, so that their latency overlaps the
        // current round's arithmetic.
        auto fetch0 = [&](int p0, Vec<VEC> &vv, Vec<VEC> &gv) {
#pragma unroll
            for (int u = 0; u < VEC; ++u)
                gv.v[u] = 0.0f;
            const int p = p0 + gr.first;
            const int64_t i = sperm[p < nt ? p : nt - 1];
            const int off = min(gr.l * VEC, C - VEC);
            if constexpr (ASYM) {  // v rows of the sources, g rows of the targets
                const int rv = side_row(a, i, kRowSource), rg = side_row(a, i, kRowTarget);
                vv = load_vec<VEC>(val + (int64_t)max(rv, 0) * C + off, rv >= 0);
                if (!HAIN)
                    gv = load_vec<VEC>(grad + (int64_t)max(rg, 0) * C + off, rg >= 0);
            } else {
                vv = load_vec<VEC>(val + i * C + off, true);
                if (!HAIN)
                    gv = load_vec<VEC>(grad + i * C + off, true);
            }
        };
        Vec<VEC> vv_next, gv_next;
        if constexpr (F)
            fetch0(0, vv_next, gv_next);
        // uniform trip count for the whole block: the group reductions run
        // with every lane of the wave active
        for (int p0 = 0; p0 < T; p0 += gr.step) {
            const int p = p0 + gr.first;
            const bool valid = p < nt;
            const int pc = valid ? p : nt - 1;
            Vec<VEC> vv0, gv0;
            if constexpr (F) {
                vv0 = vv_next;
                gv0 = gv_next;
                if (p0 + gr.step < T)
                    fetch0(p0 + gr.step, vv_next, gv_next);
            }
            int ml[D + 1], mg[D + 1];  // tile-local rows (staged) and global vertex ids
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                ml[k] = MODE != kStageNone ? (int)slr[pc][k] : 0;
                mg[k] = MODE != kStageFull ? a.svert[(base + pc) * (D + 1) + k] : 0;
            }
            const int64_t ip = sperm[pc];
            const int rv = ASYM ? side_row(a, ip, kRowSource) : (int)ip;  // row of v and dv, or -1
            const int rg = ASYM ? side_row(a, ip, kRowTarget) : (int)ip;  // row of g, or -1
            const int64_t vrow = (int64_t)max(rv, 0) * C, grow = (int64_t)max(rg, 0) * C;
            float hv[D + 1], hg[D + 1];  // raw: <v, At_k> + <g, A_k>; normalised: <v, At_k> and <g, A_k>
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                hv[k] = 0.0f;
                hg[k] = 0.0f;
            }
            // raw mode with the splat's term: <g, A_k> of this point, read
            // in the sorted order (its d+1 floats are contiguous)
            float ha[D + 1];
            if constexpr (HAIN && F) {
#pragma unroll
                for (int k = 0; k <= D; ++k)
                    ha[k] = hA[(base + pc) * (D + 1) + k];
            }
            for (int cc = 0; cc < C; cc += CH) {
                const int j0 = gr.l * VEC;
                const bool lane_on = valid && j0 < min(CH, C - cc);
                const int off = min(cc + j0, C - VEC);  // in bounds for every lane
                Vec<VEC> vv, gv;
                if constexpr (F) {
                    if (cc == 0) {
                        vv = vv0;
                        gv = gv0;
                    } else {
                        vv = load_vec<VEC>(val + vrow + off, !ASYM || rv >= 0);
                        if (!HAIN)
                            gv = load_vec<VEC>(grad + grow + off, !ASYM || rg >= 0);
                    }
                    if (!lane_on) {
#pragma unroll
                        for (int u = 0; u < VEC; ++u) {
                            vv.v[u] = 0.0f;
                            gv.v[u] = 0.0f;
                        }
                    }
                }
                Vec<VEC> o;
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    o.v[j] = 0.0f;
                // the rows of At (value gradient, <v, At_k>), then those of
                // A (<g, A_k>): d+1 rows in registers at a time
                {
                    Vec<VEC> r[D + 1];
#pragma unroll
                    for (int k = 0; k <= D; ++k)
                        r[k] = stage_vec<VEC, CH, MODE>(rowsT, At, ml[k], mg[k], ld, 0, off);
#pragma unroll
                    for (int k = 0; k <= D; ++k) {
                        const float bk = sb[pc][k];
#pragma unroll
                        for (int j = 0; j < VEC; ++j)
                            o.v[j] += bk * r[k].v[j];
                        if constexpr (F) {
                            float dv = 0.0f;
#pragma unroll
                            for (int j = 0; j < VEC; ++j)
                                dv += vv.v[j] * r[k].v[j];
                            hv[k] += dv;
                        }
                    }
                }
                if constexpr (F && !HAIN) {
                    Vec<VEC> ra[D + 1];
#pragma unroll
                    for (int k = 0; k <= D; ++k)
                        ra[k] = stage_vec<VEC, CH, MODE>(rowsA, A, ml[k], mg[k], ld, 0, off);
#pragma unroll
                    for (int k = 0; k <= D; ++k) {
                        float dg = 0.0f;
#pragma unroll
                        for (int j = 0; j < VEC; ++j)
                            dg += gv.v[j] * ra[k].v[j];
                        if constexpr (NORM)
                            hg[k] += dg;
                        else
                            hv[k] += dg;
                    }
                }
                if (grad_val && lane_on && (!ASYM || rv >= 0)) {
#pragma unroll
                    for (int j = 0; j < VEC; ++j)
                        o.v[j] *= sc;
                    store_vec<VEC>(grad_val + vrow + cc + j0, o);
                }
            }
            if constexpr (F) {
#pragma unroll
                for (int k = 0; k <= D; ++k) {
                    hv[k] = group_sum<G>(hv[k]);
                    if constexpr (NORM)
                        hg[k] = group_sum<G>(hg[k]);
                }
                float h[D + 1];
                if constexpr (NORM) {
                    float z = 0.0f, gn = 0.0f, aw[D + 1], atw[D + 1];
#pragma unroll
                    for (int k = 0; k <= D; ++k) {
                        aw[k] = stage_w<CH, MODE>(rowsA, A, ml[k], mg[k], ld, C);
                        atw[k] = stage_w<CH, MODE>(rowsT, At, ml[k], mg[k], ld, C);
                        z += sb[pc][k] * aw[k];
                        gn += sb[pc][k] * hg[k];
                    }
                    const float iz = 1.0f / z;
                    const float gam = -gn * iz * iz;
#pragma unroll
                    for (int k = 0; k <= D; ++k)
                        h[k] = hg[k] * iz + gam * aw[k] + hv[k] + atw[k];
                } else {
#pragma unroll
                    for (int k = 0; k <= D; ++k)
                        h[k] = sc * (HAIN ? hv[k] + ha[k] : hv[k]);
                }
                eq8_finish<D, G>(a, srank[pc], h, valid, grad_feat + (int64_t)sperm[pc] * D, gr.l, my_pos, my_neg);
            }
        }
    };
    if (full) {
        if (want_f)
            rounds(Int<kStageFull>{}, Flag<true>{});
        else
            rounds(Int<kStageFull>{}, Flag<false>{});
    } else {
        if (want_f)
            rounds(Int<kStageNone>{}, Flag<true>{});
        else
            rounds(Int<kStageNone>{}, Flag<false>{});
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

size_t tile_record_bytes_filter(int d) { return TileRec(d).bytes; }

bool splat_forms_eq8_term(const FilterArgs &a) { return !a.normalize && a.vec == 4 && a.c <= kSCH; }

static inline unsigned tiles_for(int d, int64_t n)
{
    const int T = tile_points(d);
    return (unsigned)((n + T - 1) / T);
}

static inline int tile_threads(int d) { return tile_points(d); }

#define PAM_DISPATCH_VEC(a, CALL)                                                                 \
    if ((a).vec == 4) {                                                                           \
        constexpr int VEC = 4;                                                                    \
        CALL;                                                                                     \
    } else {                                                                                      \
        constexpr int VEC = 1;                                                                    \
        CALL;                                                                                     \
    }

// Pass width of the splat and the slices: value rows of at most 8 or 16
// channels (float4 rows, d <= 8) take lane groups of 2 or 4 lanes instead of
// 8, so that no lane of a group idles; everything else passes over 32
// channels at a time.
#define PAM_DISPATCH_SCH(D_, VEC_, c_, CALL)                                                      \
    if constexpr ((D_) <= 8 && (VEC_) == 4) {                                                     \
        if ((c_) <= 8) {                                                                          \
            constexpr int SCH = 8;                                                                \
            CALL;                                                                                 \
        } else if ((c_) <= 16) {                                                                  \
            constexpr int SCH = 16;                                                               \
            CALL;                                                                                 \
        } else {                                                                                  \
            constexpr int SCH = kSCH;                                                             \
            CALL;                                                                                 \
        }                                                                                         \
    } else {                                                                                      \
        constexpr int SCH = kSCH;                                                                 \
        CALL;                                                                                     \
    }

hipError_t launch_splat(int d, const FilterArgs &a, const uint8_t *tiles, const float *x, const float *A,
                        int mode, float *L, float *hA, hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    if (hA && (mode != kSplatPlain || a.vec != 4 || a.normalize || a.c > kSCH))
        return hipErrorInvalidValue;  // the fused eq. 8 term: raw mode, float4 rows, one channel chunk
    const dim3 grid(tiles_for(d, a.n)), block(splat_threads(d));
    if (mode == kSplatAug) {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_splat<D, VEC, kSplatAug, SCH>),
                                                                 grid, block, 0, s, a, tiles, x, A, L, hA))));
    } else if (mode == kSplatNormBwd) {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_splat<D, VEC, kSplatNormBwd, SCH>),
                                                                 grid, block, 0, s, a, tiles, x, A, L, hA))));
    } else if (hA) {
        constexpr int VEC = 4;
        PAM_DISPATCH_D(d, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_splat<D, VEC, kSplatPlain, SCH, true>),
                                                                         grid, block, 0, s, a, tiles, x, A, L, hA)));
    } else {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_splat<D, VEC, kSplatPlain, SCH>),
                                                                 grid, block, 0, s, a, tiles, x, A, L, hA))));
    }
    return hipGetLastError();
}

hipError_t launch_blur2(const float *in, float *out, const int32_t *nbr_a, const int32_t *nbr_b, int64_t M,
                        int32_t ld, hipStream_t s)
{
    if (M <= 0)
        return hipSuccess;
    if (ld % 4 != 0)  // rows are read as float4
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_blur2, dim3(blocks_for(M * (ld / 4))), dim3(kBlock), 0, s, in, out, nbr_a, nbr_b, M, ld);
    return hipGetLastError();
}

hipError_t launch_blur(const float *in, float *out, const int32_t *nbr_j, int64_t M, int32_t ld,
                       hipStream_t s)
{
    if (M <= 0)
        return hipSuccess;
    if (ld % 4 != 0)  // rows are read as float4
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_blur, dim3(blocks_for(M * (ld / 4))), dim3(kBlock), 0, s, in, out, nbr_j, M, ld);
    return hipGetLastError();
}

hipError_t launch_slice(int d, const FilterArgs &a, const uint8_t *tiles, const float *A, float *out,
                        hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_slice<D, VEC, SCH>),
                                                             dim3(tiles_for(d, a.n)), dim3(tile_threads(d)), 0, s, a,
                                                             tiles, A, out))));
    return hipGetLastError();
}

hipError_t launch_slice_aug(int d, const FilterArgs &a, const uint8_t *tiles, const float *val, const float *grad,
                            const float *A, const float *At, const float *L1, const float *L2, int32_t ldq,
                            float *grad_feat, hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_slice_aug<D, VEC, SCH>),
                                                             dim3(tiles_for(d, a.n)), dim3(slice_aug_threads(D)), 0, s, a,
                                                             tiles, val, grad, A, At, L1, L2, ldq, grad_feat))));
    return hipGetLastError();
}

hipError_t launch_slice_bwd(int d, const FilterArgs &a, const uint8_t *tiles, const float *val, const float *grad,
                            const float *A, const float *At, const float *hA, float *grad_val, float *grad_feat,
                            hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    const dim3 grid(tiles_for(d, a.n)), block(tile_threads(d));
    if (hA && a.normalize)
        return hipErrorInvalidValue;
    if (a.src_n != a.n || a.tgt_0 != 0) {  // asymmetric filter (raw mode)
        if (hA) {
            PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_slice_bwd<D, VEC, false, true, kCH, true>), grid,
                                                                     block, 0, s, a, tiles, val, grad, A, At, hA,
                                                                     grad_val, grad_feat)));
        } else {
            PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_slice_bwd<D, VEC, false, true, kCH, false>), grid,
                                                                     block, 0, s, a, tiles, val, grad, A, At, hA,
                                                                     grad_val, grad_feat)));
        }
    } else if (a.normalize) {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_slice_bwd<D, VEC, true, false, SCH, false>),
                                                                 grid, block, 0, s, a, tiles, val, grad, A, At, hA,
                                                                 grad_val, grad_feat))));
    } else if (hA) {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_slice_bwd<D, VEC, false, false, SCH, true>),
                                                                 grid, block, 0, s, a, tiles, val, grad, A, At, hA,
                                                                 grad_val, grad_feat))));
    } else {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, PAM_DISPATCH_SCH(D, VEC, a.c, hipLaunchKernelGGL((k_slice_bwd<D, VEC, false, false, SCH, false>),
                                                                 grid, block, 0, s, a, tiles, val, grad, A, At, hA,
                                                                 grad_val, grad_feat))));
    }
    return hipGetLastError();
}

}  // namespace pam

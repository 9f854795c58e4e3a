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

namespace pam {

constexpr int kCH = 32;          // channels per pass over a tile

template <int D>
struct Tile {
    static constexpr int T = tile_points(D);  // points (= threads) per tile
    static constexpr int NW = T / 64;         // waves per block
};

__device__ __forceinline__ void atomic_add_f32(float *p, float v)
{
    __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float group_sum(float x, int G)
{
    for (int off = G >> 1; off > 0; off >>= 1)
        x += __shfl_xor(x, off);
    return x;
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

// Phase A: one thread per point stages its barycentric weights and,
// optionally, its vertex ids, ranks and original index in LDS (all from the
// build's sorted per-point records).
template <int D>
__device__ __forceinline__ void stage_points(const FilterArgs &a, int64_t base, int nt,
                                             float (*sb)[D + 1], int (*sm)[D + 1],
                                             signed char (*srank)[D + 1], int *sperm)
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
        sperm[t] = a.perm[i];
}

// Group geometry of phase B for one block.
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
// by row.  A row group of kSCH / VEC lanes owns whole rows: it sums b * v of
// the row's contributions in registers, reading v from an LDS copy of the
// tile's values, then stores the row sum in LDS; the block adds all row sums
// to the lattice with one coalesced fp32 atomic per row and channel.  No LDS
// float atomics (on gfx950 they cost about 3 cycles per lane).
// ---------------------------------------------------------------------------

constexpr int kSCH = 16;  // channels per pass of the splat

// segments whose partial sums stay in LDS
__host__ __device__ constexpr int seg_cap(int T) { return T >= 512 ? 256 : 192; }

#ifndef PAM_SPLAT_SPREAD
#define PAM_SPLAT_SPREAD 1  // splat threads per tile point
#endif
__host__ __device__ constexpr int splat_threads(int d) { return tile_points(d) * PAM_SPLAT_SPREAD; }

// Splat modes: x as given (forward, and the backward splat of dL/dv' in raw
// mode), or, for the normalised backward pass, x = g / z with the weight
// column taking b * gamma.
constexpr int kSplatPlain = 0;
constexpr int kSplatNormBwd = 1;

struct TileView {
    const uint32_t *hdr;
    const int32_t *rowid;
    const uint16_t *sfirst;
    const uint32_t *seg;
    const uint16_t *order;
    const uint16_t *list;
    const uint16_t *lrow;
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

// LDS copy of channels [cc, cc + chc) of the tile's rows of x (n x C, row
// sperm[p] for point p), pitch kSCH, zero-padded; scale[p] multiplies row p
// when given.
template <int VEC>
__device__ __forceinline__ void load_tile_chunk(float *vt, const float *__restrict__ x, const int *sperm, int nt,
                                                int C, int cc, int chc, const float *scale)
{
    constexpr int PER = kSCH / VEC;
    for (int e = threadIdx.x; e < nt * PER; e += blockDim.x) {
        const int p = e / PER, j = (e - p * PER) * VEC;
        Vec<VEC> v = load_vec<VEC>(x + (int64_t)sperm[p] * C + cc + j, j < chc);
        if (scale) {
            const float sc = scale[p];
#pragma unroll
            for (int u = 0; u < VEC; ++u)
                v.v[u] *= sc;
        }
        store_vec<VEC>(vt + p * kSCH + j, v);
    }
}

// Tiles whose vertices did not fit the build's LDS table: each point adds
// its contributions to the lattice directly (one thread per point).
//   x row p is scaled by scale[p] when given; with `weights`, the weight
//   column C gets b * wcol[p] (b when wcol is null).
template <int D>
__device__ __forceinline__ void splat_direct(const FilterArgs &a, int64_t base, int nt, const float (*sb)[D + 1],
                                             const int *sperm, const float *__restrict__ x, const float *scale,
                                             bool weights, const float *wcol, float *__restrict__ L)
{
    const int C = a.c, ld = a.ld;
    for (int p = threadIdx.x; p < nt; p += blockDim.x) {
        const float sc = scale ? scale[p] : 1.0f;
        const float *xr = x + (int64_t)sperm[p] * C;
        for (int k = 0; k <= D; ++k) {
            const int m = a.svert[(base + p) * (D + 1) + k];
            const float b = sb[p][k];
            float *row = L + (int64_t)m * ld;
            for (int c = 0; c < C; ++c)
                atomic_add_f32(&row[c], b * sc * xr[c]);
            if (weights)
                atomic_add_f32(&row[C], b * (wcol ? wcol[p] : 1.0f));
        }
    }
}

// Normalised backward prologue, per point p of the tile (a group of GL
// lanes per point): z_p = sum_k b_k Aw[m_k] and gamma_p = -<g_p, N_p> / z_p^2
// with N_p = sum_k b_k A[m_k]; leaves 1/z in sz and gamma in sgam.
template <int D, int VEC>
__device__ __forceinline__ void norm_bwd_prologue(const FilterArgs &a, int64_t base, int nt, const float (*sb)[D + 1],
                                                  const int *sperm, const float *__restrict__ g,
                                                  const float *__restrict__ A, float *sz, float *sgam)
{
    constexpr int GL = kSCH / VEC;
    const int l = threadIdx.x & (GL - 1), q = threadIdx.x / GL, ng = blockDim.x / GL;
    const int C = a.c, ld = a.ld;
    // uniform trip count for the whole block; the group reduction below
    // runs with every lane of the wave active
    for (int p0 = 0; p0 < (int)blockDim.x; p0 += ng) {
        const int p = p0 + q;
        const bool valid = p < nt;
        int m[D + 1];
        float z = 0.0f;
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            m[k] = valid ? a.svert[(base + p) * (D + 1) + k] : 0;
            z += valid ? sb[p][k] * A[(int64_t)m[k] * ld + C] : 0.0f;
        }
        float dot = 0.0f;
        const int64_t grow = (int64_t)(valid ? sperm[p] : 0) * C;
        for (int cc = 0; cc < C; cc += kSCH) {
            const bool on = valid && l * VEC < min(kSCH, C - cc);
            const Vec<VEC> gv = load_vec<VEC>(g + grow + cc + l * VEC, on);
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                const Vec<VEC> ar = load_vec<VEC>(A + (int64_t)m[k] * ld + cc + l * VEC, on);
                float dk = 0.0f;
#pragma unroll
                for (int u = 0; u < VEC; ++u)
                    dk += gv.v[u] * ar.v[u];
                dot += (valid ? sb[p][k] : 0.0f) * dk;
            }
        }
        dot = group_sum(dot, GL);
        if (valid && l == 0) {
            sz[p] = 1.0f / z;
            sgam[p] = -dot / (z * z);
        }
    }
}

// Splat of x onto L over one tile, using the build's tile view: the tile's
// contributions sorted by row, cut into segments of at most kSegLen, handed
// out longest first to groups of kSCH / VEC lanes through an LDS counter.  A
// group sums b * x over its segment in registers (x from an LDS copy of the
// tile's rows) and stores the sum in the segment's own LDS slot; then each
// row's segment sums are added and reach the lattice with one coalesced
// fp32 atomic per row and channel.  Nothing accumulates with LDS float
// atomics (on gfx950 they cost about 3 cycles per lane).
template <int D, int VEC, int MODE>
__global__ __launch_bounds__(splat_threads(D)) void k_splat(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                         const float *__restrict__ x, const float *__restrict__ A,
                                                         float *__restrict__ L)
{
    constexpr int T = tile_points(D);
    constexpr int NC = T * (D + 1);
    constexpr int GL = kSCH / VEC;
    constexpr int NZ = MODE == kSplatNormBwd ? T : 1;
    constexpr int kSegCap = seg_cap(T);
    __shared__ float sb[T][D + 1];
    __shared__ __attribute__((aligned(16))) uint16_t list_s[(NC + 7) / 8 * 8];
    __shared__ __attribute__((aligned(16))) uint32_t seg_s[kSegCap];
    __shared__ __attribute__((aligned(16))) uint16_t order_s[(kSegCap + 7) / 8 * 8];
    __shared__ __attribute__((aligned(16))) uint16_t sfirst_s[(kSegCap + 1 + 7) / 8 * 8];
    __shared__ __attribute__((aligned(16))) float vt[T * kSCH];
    __shared__ __attribute__((aligned(16))) float Ps[kSegCap * kSCH];
    __shared__ float Pw[kSegCap];
    __shared__ float sz[NZ], sgam[NZ];
    __shared__ int sperm[T];
    __shared__ int next_s;

    const TileView tv = tile_view<D>(tiles);
    const int nrows = (int)tv.hdr[0], nc = (int)tv.hdr[2], nseg = (int)tv.hdr[3];
    const bool overflow = (tv.hdr[1] & kTileOverflow) != 0;
    const bool in_lds = nseg <= kSegCap;
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const int C = a.c, ld = a.ld;
    const bool weights = a.normalize != 0;  // weight column: b (plain) or b * gamma
    const float *scale = nullptr, *wcol = nullptr;
    stage_points<D>(a, base, nt, sb, nullptr, nullptr, sperm);
    if (!overflow) {
        copy16(list_s, tv.list, nc * 2);
        if (in_lds) {
            copy16(seg_s, tv.seg, nseg * 4);
            copy16(order_s, tv.order, nseg * 2);
            copy16(sfirst_s, tv.sfirst, (nrows + 1) * 2);
        }
    }
    __syncthreads();
    if constexpr (MODE == kSplatNormBwd) {
        norm_bwd_prologue<D, VEC>(a, base, nt, sb, sperm, x, A, sz, sgam);
        __syncthreads();
        scale = sz;
        wcol = sgam;
    }
    if (overflow) {
        splat_direct<D>(a, base, nt, sb, sperm, x, scale, weights, wcol, L);
        return;
    }
    const uint16_t *order = in_lds ? order_s : tv.order;
    const uint32_t *segs = in_lds ? seg_s : tv.seg;
    constexpr int GPW = 64 / GL;  // groups per wave
    const int lane = t & 63, l = t & (GL - 1), gw = lane / GL;
    for (int cc = 0; cc < C; cc += kSCH) {
        const int chc = min(kSCH, C - cc);
        const bool lane_on = l * VEC < chc;
        const bool wpass = weights && cc == 0;
        load_tile_chunk<VEC>(vt, x, sperm, nt, C, cc, chc, scale);
        if (t == 0)
            next_s = 0;
        __syncthreads();
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
            if (w < nseg) {
                const int sidx = order[w];
                const uint32_t sd = segs[sidx];
                const int e0 = (int)(sd & 0x1fff), len = (int)((sd >> 13) & 31), r = (int)(sd >> 18);
                Vec<VEC> acc;
#pragma unroll
                for (int u = 0; u < VEC; ++u)
                    acc.v[u] = 0.0f;
                float accw = 0.0f;
                for (int e = e0; e < e0 + len; ++e) {
                    const int pk = list_s[e];
                    const int p = pk >> 5, k = pk & 31;
                    const float b = sb[p][k];
                    const Vec<VEC> xv = load_vec<VEC>(vt + p * kSCH + l * VEC, true);
#pragma unroll
                    for (int u = 0; u < VEC; ++u)
                        acc.v[u] += b * xv.v[u];
                    if (wpass)
                        accw += b * (wcol ? wcol[p] : 1.0f);
                }
                if (in_lds) {
                    store_vec<VEC>(Ps + sidx * kSCH + l * VEC, acc);
                    if (l == 0)
                        Pw[sidx] = accw;
                } else {
                    const int64_t row = (int64_t)tv.rowid[r] * ld;
                    if (lane_on) {
#pragma unroll
                        for (int u = 0; u < VEC; ++u)
                            atomic_add_f32(&L[row + cc + l * VEC + u], acc.v[u]);
                    }
                    if (wpass && l == 0)
                        atomic_add_f32(&L[row + C], accw);
                }
            }
        }
        __syncthreads();
        if (in_lds) {
            for (int e = t; e < nrows * kSCH; e += (int)blockDim.x) {
                const int r = e / kSCH, c = e - r * kSCH;
                if (c >= chc)
                    continue;
                float sum = 0.0f;
                for (int sx = sfirst_s[r]; sx < sfirst_s[r + 1]; ++sx)
                    sum += Ps[sx * kSCH + c];
                atomic_add_f32(&L[(int64_t)tv.rowid[r] * ld + cc + c], sum);
            }
            if (wpass) {
                for (int r = t; r < nrows; r += (int)blockDim.x) {
                    float sum = 0.0f;
                    for (int sx = sfirst_s[r]; sx < sfirst_s[r + 1]; ++sx)
                        sum += Pw[sx];
                    atomic_add_f32(&L[(int64_t)tv.rowid[r] * ld + C], sum);
                }
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Blur: one direction, L'[m] = L[n-] + 2 L[m] + L[n+] (absent -> 0)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_blur(const float *__restrict__ in, float *__restrict__ out,
                                                 const int32_t *__restrict__ nbr_j, int64_t M,
                                                 int32_t ld)
{
    const int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (e >= M * ld)
        return;
    const int64_t m = e / ld;
    const int c = (int)(e - m * ld);
    const int32_t lo = nbr_j[2 * m], hi = nbr_j[2 * m + 1];
    float acc = 2.0f * in[e];
    if (lo >= 0)
        acc += in[(int64_t)lo * ld + c];
    if (hi >= 0)
        acc += in[(int64_t)hi * ld + c];
    out[e] = acc;
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
// pieces at the point's original index.  Lattice rows are padded to ld (a
// multiple of 4 floats), so float4 reads that start below C stay inside
// the row.
// ---------------------------------------------------------------------------

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

template <int VEC>
__device__ __forceinline__ Vec<VEC> lds_vec(const float *p, bool ok)
{
    Vec<VEC> r;
    if constexpr (VEC == 4) {
        const float4 x = ok ? *reinterpret_cast<const float4 *>(p) : make_float4(0.f, 0.f, 0.f, 0.f);
        r.v[0] = x.x;
        r.v[1] = x.y;
        r.v[2] = x.z;
        r.v[3] = x.w;
    } else {
        r.v[0] = ok ? *p : 0.0f;
    }
    return r;
}

// Phase A of the slice kernels: weights, original index, tile-local rows
// (when the tile's rows are staged) and ranks (when asked) of each point.
template <int D>
__device__ __forceinline__ void stage_slice_points(const FilterArgs &a, const TileView &tv, bool staged, int64_t base,
                                                   int nt, float (*sb)[D + 1], uint16_t (*slr)[D + 1],
                                                   signed char (*srank)[D + 1], int *sperm)
{
    stage_points<D>(a, base, nt, sb, nullptr, srank, sperm);
    const int t = threadIdx.x;
    if (staged && t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k)
            slr[t][k] = tv.lrow[t * (D + 1) + k];
    }
}

// Row index of vertex k of tile point p: tile-local when staged, else the
// global vertex id.
template <int D>
__device__ __forceinline__ int point_row(const FilterArgs &a, bool staged, const uint16_t (*slr)[D + 1],
                                         int64_t base, int p, int k)
{
    return staged ? (int)slr[p][k] : a.svert[(base + p) * (D + 1) + k];
}

template <int D, int VEC>
__global__ __launch_bounds__(Tile<D>::T) void k_slice(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                      const float *__restrict__ A, float *__restrict__ out)
{
    constexpr int T = Tile<D>::T;
    __shared__ float sb[T][D + 1];
    __shared__ uint16_t slr[T][D + 1];
    __shared__ int sperm[T];
    __shared__ __attribute__((aligned(16))) float rows[kSliceRows * kRowPitch];
    __shared__ float wrow[kSliceRows];
    const TileView tv = tile_view<D>(tiles);
    const int nrows = (int)tv.hdr[0];
    const bool staged = !(tv.hdr[1] & kTileOverflow) && nrows <= kSliceRows;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const int C = a.c, ld = a.ld;
    stage_slice_points<D>(a, tv, staged, base, nt, sb, slr, nullptr, sperm);
    const Groups gr(a.group, Tile<D>::NW);
    for (int cc = 0; cc < C; cc += kCH) {
        if (staged) {
            if (cc > 0)
                __syncthreads();
            stage_rows(rows, (a.normalize && cc == 0) ? wrow : nullptr, A, tv.rowid, nrows, ld, C, cc);
        }
        __syncthreads();
        const bool lane_on = gr.l * VEC < min(kCH, C - cc);
        for (int p = gr.first; p < nt; p += gr.step) {
            if (!lane_on)
                continue;
            int m[D + 1];
#pragma unroll
            for (int k = 0; k <= D; ++k)
                m[k] = point_row<D>(a, staged, slr, base, p, k);
            float sc = a.E.raw_scale;
            if (a.normalize) {
                float z = 0.0f;
#pragma unroll
                for (int k = 0; k <= D; ++k)
                    z += sb[p][k] * (staged ? wrow[m[k]] : A[(int64_t)m[k] * ld + C]);
                sc = 1.0f / z;
            }
            Vec<VEC> o;
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                o.v[j] = 0.0f;
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                const Vec<VEC> r = staged ? lds_vec<VEC>(rows + m[k] * kRowPitch + gr.l * VEC, true)
                                          : load_vec<VEC>(A + (int64_t)m[k] * ld + cc + gr.l * VEC, true);
                const float bk = sb[p][k];
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    o.v[j] += bk * r.v[j];
            }
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                o.v[j] *= sc;
            store_vec<VEC>(out + (int64_t)sperm[p] * C + cc + gr.l * VEC, o);
        }
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
// the point's embedding gradient itself.
// ---------------------------------------------------------------------------

template <int D, int VEC, bool NORM>
__global__ __launch_bounds__(Tile<D>::T) void k_slice_bwd(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                          const float *__restrict__ val,
                                                          const float *__restrict__ grad,
                                                          const float *__restrict__ A,
                                                          const float *__restrict__ At,
                                                          float *__restrict__ grad_val,
                                                          float *__restrict__ grad_feat)
{
    constexpr int T = Tile<D>::T;
    constexpr int WR = NORM ? kSliceBwdRows : 1;
    __shared__ float sb[T][D + 1];
    __shared__ uint16_t slr[T][D + 1];
    __shared__ signed char srank[T][D + 1];
    __shared__ int sperm[T];
    __shared__ __attribute__((aligned(16))) float rowsT[kSliceBwdRows * kRowPitch];
    __shared__ __attribute__((aligned(16))) float rowsA[kSliceBwdRows * kRowPitch];
    __shared__ float wT[WR], wA[WR];
    const TileView tv = tile_view<D>(tiles);
    const int nrows = (int)tv.hdr[0];
    const int C = a.c, ld = a.ld;
    const bool staged = !(tv.hdr[1] & kTileOverflow) && nrows <= kSliceBwdRows && C <= kCH;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const float sc = NORM ? 1.0f : a.E.raw_scale;
    const bool want_f = grad_feat != nullptr;
    stage_slice_points<D>(a, tv, staged, base, nt, sb, slr, want_f ? srank : nullptr, sperm);
    if (staged) {
        stage_rows(rowsT, NORM ? wT : nullptr, At, tv.rowid, nrows, ld, C, 0);
        if (want_f)
            stage_rows(rowsA, NORM ? wA : nullptr, A, tv.rowid, nrows, ld, C, 0);
    }
    __syncthreads();
    const Groups gr(a.group, Tile<D>::NW);
    // uniform trip count for the whole block: the group reductions run with
    // every lane of the wave active; lanes past the tile's end are masked
    for (int p0 = 0; p0 < T; p0 += gr.step) {
        const int p = p0 + gr.first;
        const bool valid = p < nt;
        const int pc = valid ? p : nt - 1;
        int m[D + 1];
#pragma unroll
        for (int k = 0; k <= D; ++k)
            m[k] = point_row<D>(a, staged, slr, base, pc, k);
        const int64_t prow = (int64_t)sperm[pc] * C;
        float hv[D + 1], hg[D + 1];  // raw: <v, At_k> + <g, A_k>; normalised: <v, At_k> and <g, A_k>
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            hv[k] = 0.0f;
            hg[k] = 0.0f;
        }
        for (int cc = 0; cc < C; cc += kCH) {
            const bool lane_on = valid && gr.l * VEC < min(kCH, C - cc);
            const int off = cc + gr.l * VEC;
            Vec<VEC> vv, gv;
            if (want_f) {
                vv = load_vec<VEC>(val + prow + off, lane_on);
                gv = load_vec<VEC>(grad + prow + off, lane_on);
            }
            Vec<VEC> o;
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                o.v[j] = 0.0f;
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                const float bk = sb[pc][k];
                const Vec<VEC> r = staged ? lds_vec<VEC>(rowsT + m[k] * kRowPitch + gr.l * VEC, lane_on)
                                          : load_vec<VEC>(At + (int64_t)m[k] * ld + off, lane_on);
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    o.v[j] += bk * r.v[j];
                if (want_f) {
                    const Vec<VEC> ra = staged ? lds_vec<VEC>(rowsA + m[k] * kRowPitch + gr.l * VEC, lane_on)
                                               : load_vec<VEC>(A + (int64_t)m[k] * ld + off, lane_on);
                    float dv = 0.0f, dg = 0.0f;
#pragma unroll
                    for (int j = 0; j < VEC; ++j) {
                        dv += vv.v[j] * r.v[j];
                        dg += gv.v[j] * ra.v[j];
                    }
                    if constexpr (NORM) {
                        hv[k] += dv;
                        hg[k] += dg;
                    } else {
                        hv[k] += dv + dg;
                    }
                }
            }
            if (grad_val && lane_on) {
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    o.v[j] *= sc;
                store_vec<VEC>(grad_val + prow + off, o);
            }
        }
        if (!want_f)
            continue;
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            hv[k] = group_sum(hv[k], gr.G);
            if constexpr (NORM)
                hg[k] = group_sum(hg[k], gr.G);
        }
        float h[D + 1];
        if constexpr (NORM) {
            float z = 0.0f, gn = 0.0f, aw[D + 1], atw[D + 1];
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                aw[k] = staged ? wA[m[k]] : A[(int64_t)m[k] * ld + C];
                atw[k] = staged ? wT[m[k]] : At[(int64_t)m[k] * ld + C];
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
                h[k] = sc * hv[k];
        }
        float gx[D + 1];
#pragma unroll
        for (int c = 0; c <= D; ++c) {
            const int rc = srank[pc][c];
            float hp = 0.0f, hm = 0.0f;
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                hp = (k == D - rc) ? h[k] : hp;
                hm = (k == (D + 1 - rc) % (D + 1)) ? h[k] : hm;
            }
            gx[c] = (hp - hm) * a.E.inv;
        }
        // df_j = sum_c E[c][j] gx_c = pos[j] * sum_{c <= j} gx_c + neg[j] * gx_{j+1};
        // the group's lanes share the stores
        float prefix = 0.0f;
        float *frow = grad_feat + (int64_t)sperm[pc] * D;
#pragma unroll
        for (int j = 0; j < D; ++j) {
            prefix += gx[j];
            if (valid && (j & (gr.G - 1)) == gr.l)
                frow[j] = a.E.pos[j] * prefix + a.E.neg[j] * gx[j + 1];
        }
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

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

hipError_t launch_splat(int d, const FilterArgs &a, const uint8_t *tiles, const float *x, const float *A,
                        bool norm_bwd, float *L, hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    if (norm_bwd) {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_splat<D, VEC, kSplatNormBwd>),
                                                                 dim3(tiles_for(d, a.n)), dim3(splat_threads(d)), 0, s,
                                                                 a, tiles, x, A, L)));
    } else {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_splat<D, VEC, kSplatPlain>),
                                                                 dim3(tiles_for(d, a.n)), dim3(splat_threads(d)), 0, s,
                                                                 a, tiles, x, A, L)));
    }
    return hipGetLastError();
}

hipError_t launch_blur(const float *in, float *out, const int32_t *nbr_j, int64_t M, int32_t ld,
                       hipStream_t s)
{
    if (M <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_blur, dim3(blocks_for(M * ld)), dim3(kBlock), 0, s, in, out, nbr_j, M, ld);
    return hipGetLastError();
}

hipError_t launch_slice(int d, const FilterArgs &a, const uint8_t *tiles, const float *A, float *out,
                        hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_slice<D, VEC>), dim3(tiles_for(d, a.n)),
                                                             dim3(tile_threads(d)), 0, s, a, tiles, A, out)));
    return hipGetLastError();
}

hipError_t launch_slice_bwd(int d, const FilterArgs &a, const uint8_t *tiles, const float *val, const float *grad,
                            const float *A, const float *At, float *grad_val, float *grad_feat, hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    if (a.normalize) {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_slice_bwd<D, VEC, true>),
                                                                 dim3(tiles_for(d, a.n)), dim3(tile_threads(d)), 0, s,
                                                                 a, tiles, val, grad, A, At, grad_val, grad_feat)));
    } else {
        PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_slice_bwd<D, VEC, false>),
                                                                 dim3(tiles_for(d, a.n)), dim3(tile_threads(d)), 0, s,
                                                                 a, tiles, val, grad, A, At, grad_val, grad_feat)));
    }
    return hipGetLastError();
}

}  // namespace pam

// HIP kernels (gfx950) of the permutohedral-lattice filter (Joutard et al.
// 2019, Section 2, eq. 6-8), for one lattice built by pam_build.hip:
//   splat      S: values times barycentric weights onto the lattice rows
//   blur       B: one lattice direction per launch, taps [1 2 1]
//   slice      Sl: weighted gather of each point's d+1 vertex rows
//   splat_bwd  S of dL/dv' and the slice-side half of eq. 8
//   slice_bwd  Sl for dL/dv (eq. 7) and the embedding gradient (eq. 8)
//
// The per-point kernels work on tiles of consecutive points, one block per
// tile.  Phase A (one thread per point) recomputes the point's simplex and
// barycentric weights from its features and reads its vertex ids, staging
// both in LDS.  Phase B maps a group of G lanes onto each point, lane l
// covering VEC consecutive channels of a chunk of up to 32 channels, so that
// value rows are read and written as coalesced (float4) rows and the dot
// products of eq. 8 reduce inside the group with cross-lane shuffles.
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

// Phase A: one thread per point stages its barycentric weights and vertex
// ids (and optionally its ranks) in LDS.
template <int D>
__device__ __forceinline__ void stage_points(const FilterArgs &a, int64_t base, int nt,
                                             float (*sb)[D + 1], int (*sm)[D + 1],
                                             signed char (*srank)[D + 1])
{
    const int t = threadIdx.x;
    if (t >= nt)
        return;
    const int64_t i = base + t;
    Simplex<D> s;
    embed<D>(a.feat + i * D, a.E, s);
    float b[D + 1];
    barycentric<D>(s, a.feat + i * D, a.E, b);
#pragma unroll
    for (int k = 0; k <= D; ++k) {
        int m = a.vert[i * (D + 1) + k];
        // ids are never negative after a successful build; if one were, the
        // point would contribute nothing rather than index memory
        sb[t][k] = m >= 0 ? b[k] : 0.0f;
        if (sm)
            sm[t][k] = m >= 0 ? m : 0;
    }
    if (srank) {
#pragma unroll
        for (int c = 0; c <= D; ++c)
            srank[t][c] = (signed char)s.rank[c];
    }
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

constexpr int kSCH = 16;     // channels per pass of the row-owned splat
constexpr int kPRows = 512;  // rows whose sums stay in LDS (others: direct atomics)

template <int D>
__device__ __forceinline__ void tile_view(const uint8_t *tiles, const uint32_t *&hdr, const int32_t *&rowid,
                                          const uint16_t *&off, const uint16_t *&list)
{
    const TileRec rec(D);
    const uint8_t *R = tiles + (size_t)blockIdx.x * rec.bytes;
    hdr = reinterpret_cast<const uint32_t *>(R);
    rowid = reinterpret_cast<const int32_t *>(R + rec.rowid);
    off = reinterpret_cast<const uint16_t *>(R + rec.off);
    list = reinterpret_cast<const uint16_t *>(R + rec.list);
}

// LDS copy of channels [cc, cc + chc) of the tile's rows of x (n x C),
// pitch kSCH, zero-padded; scale[p] multiplies row p when given.
template <int VEC>
__device__ __forceinline__ void load_tile_chunk(float *vt, const float *__restrict__ x, int64_t base, int nt,
                                                int C, int cc, int chc, const float *scale)
{
    constexpr int PER = kSCH / VEC;
    for (int e = threadIdx.x; e < nt * PER; e += blockDim.x) {
        const int p = e / PER, j = (e - p * PER) * VEC;
        Vec<VEC> v = load_vec<VEC>(x + (base + p) * C + cc + j, j < chc);
        if (scale) {
            const float sc = scale[p];
#pragma unroll
            for (int u = 0; u < VEC; ++u)
                v.v[u] *= sc;
        }
        store_vec<VEC>(vt + p * kSCH + j, v);
    }
}

// Row sums of one channel chunk: row group q (kSCH / VEC lanes) owns rows
// q, q + ngroups, ...; sums go to P (rows < kPRows) or straight to L.
template <int D, int VEC>
__device__ __forceinline__ void row_sums(const float (*sb)[D + 1], const float *vt, const uint16_t *__restrict__ off,
                                         const uint16_t *__restrict__ list, const int32_t *__restrict__ rowid,
                                         int nrows, float *P, float *__restrict__ L, int ld, int cc, int chc)
{
    constexpr int GL = kSCH / VEC;
    const int l = threadIdx.x & (GL - 1), q = threadIdx.x / GL, ng = blockDim.x / GL;
    for (int r = q; r < nrows; r += ng) {
        const int e0 = off[r], e1 = off[r + 1];
        Vec<VEC> acc;
#pragma unroll
        for (int u = 0; u < VEC; ++u)
            acc.v[u] = 0.0f;
        for (int e = e0; e < e1; ++e) {
            const int pk = list[e];
            const int p = pk >> 5, k = pk & 31;
            const float b = sb[p][k];
            const float *src = vt + p * kSCH + l * VEC;
            if constexpr (VEC == 4) {
                const float4 x = *reinterpret_cast<const float4 *>(src);
                acc.v[0] += b * x.x;
                acc.v[1] += b * x.y;
                acc.v[2] += b * x.z;
                acc.v[3] += b * x.w;
            } else {
                acc.v[0] += b * src[0];
            }
        }
        if (r < kPRows) {
            store_vec<VEC>(P + r * kSCH + l * VEC, acc);
        } else {
#pragma unroll
            for (int u = 0; u < VEC; ++u)
                if (l * VEC + u < chc)
                    atomic_add_f32(&L[(int64_t)rowid[r] * ld + cc + l * VEC + u], acc.v[u]);
        }
    }
}

// Coalesced flush of the LDS row sums of one chunk.
__device__ __forceinline__ void flush_rows(const float *P, const int32_t *__restrict__ rowid, int nrows,
                                           float *__restrict__ L, int ld, int cc, int chc)
{
    const int np = min(nrows, kPRows);
    for (int e = threadIdx.x; e < np * kSCH; e += blockDim.x) {
        const int r = e / kSCH, c = e - r * kSCH;
        if (c < chc)
            atomic_add_f32(&L[(int64_t)rowid[r] * ld + cc + c], P[e]);
    }
}

// Weighted count column: L[rowid[r]][col] += sum over the row's entries of
// b * w[p] (w = 1 when null); one thread per row.
template <int D>
__device__ __forceinline__ void row_weight_column(const float (*sb)[D + 1], const float *w,
                                                  const uint16_t *__restrict__ off,
                                                  const uint16_t *__restrict__ list,
                                                  const int32_t *__restrict__ rowid, int nrows,
                                                  float *__restrict__ L, int ld, int col)
{
    for (int r = threadIdx.x; r < nrows; r += blockDim.x) {
        float acc = 0.0f;
        for (int e = off[r]; e < off[r + 1]; ++e) {
            const int pk = list[e];
            const int p = pk >> 5;
            acc += sb[p][pk & 31] * (w ? w[p] : 1.0f);
        }
        atomic_add_f32(&L[(int64_t)rowid[r] * ld + col], acc);
    }
}

// Tiles whose vertices did not fit the build's LDS table: every
// contribution is added to the lattice directly.
template <int D>
__device__ __forceinline__ void splat_direct(const FilterArgs &a, int64_t base, int nt, const float (*sb)[D + 1],
                                             const int (*sm)[D + 1], const float *__restrict__ x,
                                             const float *scale, const float *wcol, float *__restrict__ L)
{
    const int C = a.c, ld = a.ld;
    for (int e = threadIdx.x; e < nt * C; e += blockDim.x) {
        const int p = e / C, c = e - p * C;
        const float v = x[(base + p) * C + c] * (scale ? scale[p] : 1.0f);
#pragma unroll
        for (int k = 0; k <= D; ++k)
            atomic_add_f32(&L[(int64_t)sm[p][k] * ld + c], sb[p][k] * v);
    }
    if (a.normalize && (wcol || !scale)) {
        for (int p = threadIdx.x; p < nt; p += blockDim.x) {
#pragma unroll
            for (int k = 0; k <= D; ++k)
                atomic_add_f32(&L[(int64_t)sm[p][k] * ld + C], sb[p][k] * (wcol ? wcol[p] : 1.0f));
        }
    }
}

template <int D, int VEC>
__global__ __launch_bounds__(tile_points(D)) void k_splat(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                         const float *__restrict__ val, float *__restrict__ L)
{
    constexpr int T = tile_points(D);
    static_assert(T * (D + 1) <= (T + kPRows) * kSCH, "id scratch must fit the value tile and row sums");
    __shared__ float sb[T][D + 1];
    // value tile and row sums; an overflow tile uses the space for its ids
    __shared__ __attribute__((aligned(16))) float scratch[(T + kPRows) * kSCH];
    float *vt = scratch;
    float *P = scratch + T * kSCH;
    int(*sm)[D + 1] = reinterpret_cast<int(*)[D + 1]>(scratch);
    const uint32_t *hdr;
    const int32_t *rowid;
    const uint16_t *off, *list;
    tile_view<D>(tiles, hdr, rowid, off, list);
    const int nrows = (int)hdr[0];
    const bool overflow = (hdr[1] & kTileOverflow) != 0;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const int C = a.c, ld = a.ld;
    stage_points<D>(a, base, nt, sb, overflow ? sm : nullptr, nullptr);
    __syncthreads();
    if (overflow) {
        splat_direct<D>(a, base, nt, sb, sm, val, nullptr, nullptr, L);
        return;
    }
    if (a.normalize)
        row_weight_column<D>(sb, nullptr, off, list, rowid, nrows, L, ld, C);
    for (int cc = 0; cc < C; cc += kSCH) {
        const int chc = min(kSCH, C - cc);
        load_tile_chunk<VEC>(vt, val, base, nt, C, cc, chc, nullptr);
        __syncthreads();
        row_sums<D, VEC>(sb, vt, off, list, rowid, nrows, P, L, ld, cc, chc);
        __syncthreads();
        flush_rows(P, rowid, nrows, L, ld, cc, chc);
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
// ---------------------------------------------------------------------------

template <int D, int VEC>
__global__ __launch_bounds__(Tile<D>::T) void k_slice(FilterArgs a, const float *__restrict__ A,
                                                      float *__restrict__ out)
{
    constexpr int T = Tile<D>::T;
    __shared__ float sb[T][D + 1];
    __shared__ int sm[T][D + 1];
    __shared__ float sscale[T];
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const int C = a.c, ld = a.ld;
    stage_points<D>(a, base, nt, sb, sm, nullptr);
    if (t < nt) {
        float sc = a.E.raw_scale;
        if (a.normalize) {
            float z = 0.0f;
#pragma unroll
            for (int k = 0; k <= D; ++k)
                z += sb[t][k] * A[(int64_t)sm[t][k] * ld + C];
            sc = 1.0f / z;
        }
        sscale[t] = sc;
    }
    __syncthreads();
    const Groups gr(a.group, Tile<D>::NW);
    for (int cc = 0; cc < C; cc += kCH) {
        const int chc = min(kCH, C - cc);
        const bool lane_on = gr.l * VEC < chc;
        for (int p = gr.first; p < nt; p += gr.step) {
            if (!lane_on)
                continue;
            Vec<VEC> o;
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                o.v[j] = 0.0f;
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                const Vec<VEC> r = load_vec<VEC>(A + (int64_t)sm[p][k] * ld + cc + gr.l * VEC, true);
                const float bk = sb[p][k];
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    o.v[j] += bk * r.v[j];
            }
            const float sc = sscale[p];
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                o.v[j] *= sc;
            store_vec<VEC>(out + (base + p) * C + cc + gr.l * VEC, o);
        }
    }
}

// ---------------------------------------------------------------------------
// Backward splat of dL/dv' onto Lb, with the slice-side term of eq. (8):
//   raw:        Lb = S g;              hA[i][k] = s_d <g_i, A[m_ik]>
//   normalised: out = N/z, gt = g/z, gam = -<g, out>/z;
//               Lb = S [gt, gam];      hA[i][k] = <gt_i, A[m_ik]> + gam_i Aw[m_ik]
// hA may be null (no embedding gradient wanted): then only Lb = S g (or S gt).
// The splat is the row-owned scheme of k_splat over an LDS copy of g; the
// dot products <g_i, A[m_ik]> use a group of kSCH / VEC lanes per point,
// reading g from the same LDS copy and A from the lattice.
// ---------------------------------------------------------------------------

template <int D, int VEC>
__global__ __launch_bounds__(tile_points(D)) void k_splat_bwd(FilterArgs a, const uint8_t *__restrict__ tiles,
                                                             const float *__restrict__ grad,
                                                             const float *__restrict__ A,
                                                             float *__restrict__ Lb, float *__restrict__ hA)
{
    constexpr int T = tile_points(D);
    constexpr int GL = kSCH / VEC;
    __shared__ float sb[T][D + 1];
    __shared__ int sm[T][D + 1];
    __shared__ float sh[T][D + 1];
    __shared__ float sz[T];    // 1/z (normalised)
    __shared__ float sdot[T];  // <g, N>, then gamma
    __shared__ __attribute__((aligned(16))) float vt[T * kSCH];
    __shared__ __attribute__((aligned(16))) float P[kPRows * kSCH];
    const uint32_t *hdr;
    const int32_t *rowid;
    const uint16_t *off, *list;
    tile_view<D>(tiles, hdr, rowid, off, list);
    const int nrows = (int)hdr[0];
    const bool overflow = (hdr[1] & kTileOverflow) != 0;
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const int C = a.c, ld = a.ld;
    const bool norm = a.normalize != 0;
    const bool want_h = hA != nullptr;
#pragma unroll
    for (int k = 0; k <= D; ++k)
        sh[t][k] = 0.0f;
    sdot[t] = 0.0f;
    sz[t] = 1.0f;
    stage_points<D>(a, base, nt, sb, sm, nullptr);
    if (norm && t < nt) {
        float z = 0.0f;
#pragma unroll
        for (int k = 0; k <= D; ++k)
            z += sb[t][k] * A[(int64_t)sm[t][k] * ld + C];
        sz[t] = 1.0f / z;
    }
    __syncthreads();
    const int l = t & (GL - 1), q = t / GL, ng = T / GL;
    for (int cc = 0; cc < C; cc += kSCH) {
        const int chc = min(kSCH, C - cc);
        load_tile_chunk<VEC>(vt, grad, base, nt, C, cc, chc, nullptr);
        __syncthreads();
        if (want_h) {
            // per point: <g_p, A[m_pk]> over this chunk (and <g_p, N_p> normalised)
            for (int p = q; p < nt; p += ng) {
                const Vec<VEC> gv = load_vec<VEC>(vt + p * kSCH + l * VEC, true);
                float dn = 0.0f;
#pragma unroll
                for (int k = 0; k <= D; ++k) {
                    const Vec<VEC> ar =
                        load_vec<VEC>(A + (int64_t)sm[p][k] * ld + cc + l * VEC, l * VEC < chc);
                    float dk = 0.0f;
#pragma unroll
                    for (int u = 0; u < VEC; ++u)
                        dk += gv.v[u] * ar.v[u];
                    dk = group_sum(dk, GL);
                    dn += sb[p][k] * dk;
                    if (l == 0)
                        sh[p][k] += dk;
                }
                if (l == 0)
                    sdot[p] += dn;
            }
        }
        if (overflow) {
            __syncthreads();
            continue;
        }
        if (norm) {
            // gt = g / z: rescale the LDS copy in place
            __syncthreads();
            for (int e = t; e < nt * kSCH; e += T)
                vt[e] *= sz[e / kSCH];
            __syncthreads();
        }
        row_sums<D, VEC>(sb, vt, off, list, rowid, nrows, P, Lb, ld, cc, chc);
        __syncthreads();
        flush_rows(P, rowid, nrows, Lb, ld, cc, chc);
        __syncthreads();
    }
    if (norm && t < nt)
        sdot[t] = -sdot[t] * sz[t] * sz[t];  // gamma = -<g, N> / z^2
    __syncthreads();
    if (overflow) {
        splat_direct<D>(a, base, nt, sb, sm, grad, norm ? sz : nullptr, (norm && want_h) ? sdot : nullptr, Lb);
    } else if (norm && want_h) {
        row_weight_column<D>(sb, sdot, off, list, rowid, nrows, Lb, ld, C);
    }
    if (want_h && t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            float h = sh[t][k];
            if (norm)
                h = h * sz[t] + sdot[t] * A[(int64_t)sm[t][k] * ld + C];
            else
                h *= a.E.raw_scale;
            hA[(base + t) * (D + 1) + k] = h;
        }
    }
}

// ---------------------------------------------------------------------------
// Backward slice: dL/dv = sc * sum_k b_k At[m_k] (eq. 7; sc = 1/G_d raw, 1
// normalised) and the embedding gradient of eq. (8): with h_k = dL/db_k,
//   h_k = hA_k + sc <v_i, At[m_k]> (+ Atw[m_k] normalised),
//   gx_c = (h[d - rank_c] - h[(d + 1 - rank_c) mod (d+1)]) / (d+1),
//   df_i = E^T gx.
// ---------------------------------------------------------------------------

template <int D, int VEC>
__global__ __launch_bounds__(Tile<D>::T) void k_slice_bwd(FilterArgs a, const float *__restrict__ val,
                                                          const float *__restrict__ At,
                                                          const float *__restrict__ hA,
                                                          float *__restrict__ grad_val,
                                                          float *__restrict__ grad_feat)
{
    constexpr int T = Tile<D>::T;
    __shared__ float sb[T][D + 1];
    __shared__ int sm[T][D + 1];
    __shared__ signed char srank[T][D + 1];
    __shared__ float sh[T][D + 1];
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, a.n - base);
    const int C = a.c, ld = a.ld;
    const float sc = a.normalize ? 1.0f : a.E.raw_scale;
    const bool want_f = grad_feat != nullptr;
#pragma unroll
    for (int k = 0; k <= D; ++k)
        sh[t][k] = 0.0f;
    stage_points<D>(a, base, nt, sb, sm, want_f ? srank : nullptr);
    __syncthreads();
    const Groups gr(a.group, Tile<D>::NW);
    for (int cc = 0; cc < C; cc += kCH) {
        const int chc = min(kCH, C - cc);
        const bool lane_on = gr.l * VEC < chc;
        for (int p = gr.first; p < nt; p += gr.step) {
            Vec<VEC> vv;
            if (want_f)
                vv = load_vec<VEC>(val + (base + p) * C + cc + gr.l * VEC, lane_on);
            Vec<VEC> o;
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                o.v[j] = 0.0f;
#pragma unroll
            for (int k = 0; k <= D; ++k) {
                const Vec<VEC> r = load_vec<VEC>(At + (int64_t)sm[p][k] * ld + cc + gr.l * VEC, lane_on);
                const float bk = sb[p][k];
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    o.v[j] += bk * r.v[j];
                if (want_f) {
                    float dk = 0.0f;
#pragma unroll
                    for (int j = 0; j < VEC; ++j)
                        dk += vv.v[j] * r.v[j];
                    dk = group_sum(dk, gr.G);
                    if (gr.l == 0)
                        sh[p][k] += dk;
                }
            }
            if (grad_val && lane_on) {
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    o.v[j] *= sc;
                store_vec<VEC>(grad_val + (base + p) * C + cc + gr.l * VEC, o);
            }
        }
    }
    if (!want_f)
        return;
    __syncthreads();
    if (t >= nt)
        return;
    float h[D + 1];
#pragma unroll
    for (int k = 0; k <= D; ++k) {
        float hs = sh[t][k];
        if (a.normalize)
            hs += At[(int64_t)sm[t][k] * ld + C];
        else
            hs *= sc;
        h[k] = hA[(base + t) * (D + 1) + k] + hs;
    }
    float gx[D + 1];
#pragma unroll
    for (int c = 0; c <= D; ++c) {
        const int rc = srank[t][c];
        float hp = 0.0f, hm = 0.0f;
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            hp = (k == D - rc) ? h[k] : hp;
            hm = (k == (D + 1 - rc) % (D + 1)) ? h[k] : hm;
        }
        gx[c] = (hp - hm) * a.E.inv;
    }
    // df_j = sum_c E[c][j] gx_c = pos[j] * sum_{c <= j} gx_c + neg[j] * gx_{j+1}
    float prefix = 0.0f;
#pragma unroll
    for (int j = 0; j < D; ++j) {
        prefix += gx[j];
        grad_feat[(base + t) * D + j] = a.E.pos[j] * prefix + a.E.neg[j] * gx[j + 1];
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

static inline unsigned tiles_for(int d, int64_t n)
{
    const int T = d <= 8 ? 512 : 256;
    return (unsigned)((n + T - 1) / T);
}

static inline int tile_threads(int d) { return d <= 8 ? 512 : 256; }

#define PAM_DISPATCH_VEC(a, CALL)                                                                 \
    if ((a).vec == 4) {                                                                           \
        constexpr int VEC = 4;                                                                    \
        CALL;                                                                                     \
    } else {                                                                                      \
        constexpr int VEC = 1;                                                                    \
        CALL;                                                                                     \
    }

hipError_t launch_splat(int d, const FilterArgs &a, const uint8_t *tiles, const float *val, float *L,
                        hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_splat<D, VEC>), dim3(tiles_for(d, a.n)),
                                                             dim3(tile_threads(d)), 0, s, a, tiles, val, L)));
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

hipError_t launch_slice(int d, const FilterArgs &a, const float *A, float *out, hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_slice<D, VEC>), dim3(tiles_for(d, a.n)),
                                                             dim3(tile_threads(d)), 0, s, a, A, out)));
    return hipGetLastError();
}

hipError_t launch_splat_bwd(int d, const FilterArgs &a, const uint8_t *tiles, const float *grad, const float *A,
                            float *Lb, float *hA, hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_splat_bwd<D, VEC>), dim3(tiles_for(d, a.n)),
                                                             dim3(tile_threads(d)), 0, s, a, tiles, grad, A, Lb,
                                                             hA)));
    return hipGetLastError();
}

hipError_t launch_slice_bwd(int d, const FilterArgs &a, const float *val, const float *At,
                            const float *hA, float *grad_val, float *grad_feat, hipStream_t s)
{
    if (a.n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, PAM_DISPATCH_VEC(a, hipLaunchKernelGGL((k_slice_bwd<D, VEC>), dim3(tiles_for(d, a.n)),
                                                             dim3(tile_threads(d)), 0, s, a, val, At, hA,
                                                             grad_val, grad_feat)));
    return hipGetLastError();
}

}  // namespace pam

// HIP kernels (gfx950) of the permutohedral block's prologue (Joutard et al.
// 2019, Section 3 and the Fig. 2 caption): features are a 1x1x1 convolution
// of the input channels with a mesh of spatial coordinates appended,
// followed by a Leaky-ReLU; descriptors are a 1x1x1 convolution of the input
// channels; both are split channel-wise into groups and written in the
// grouped layout a batched lattice build takes (group g: rows g N .. g N +
// N - 1, its slice of the channels).
//
//   forward : the block's input rows are staged in LDS with coalesced
//             loads; both 1x1x1 convolutions run as 32 x 32 tiles on the
//             matrix cores.
//   backward: the pre-activations, the input gradient and the weight and
//             bias gradients (sums over all voxels of outer products) are
//             small dense contractions, run on the matrix cores per chunk of
//             voxels; the weight gradients are accumulated per block in LDS,
//             written as per-block partials and summed over the blocks in a
//             fixed order by a second kernel (deterministic).
#include "pam_internal.h"

#include <algorithm>
#include <mutex>

namespace pam {

namespace {

constexpr int kPrologueThreads = 256;
constexpr size_t kBwdLdsBudget = 150 << 10;  // LDS bytes the backward chunk size aims for
constexpr int kReduceEntries = 32;          // gradient entries per block of the reduction
constexpr int kStageBatch = 8;              // loads in flight per thread when staging rows
constexpr int kReduceThreads = 1024;

struct Sizes {
    int cin, kin, dt, ct, G, dg, cg;
    int nwf, nw;  // weight floats: wf + bf, then wv + bv
    __host__ __device__ explicit Sizes(const pam_block_desc_t &ds)
    {
        cin = ds.c_in;
        kin = cin + 3;
        dt = ds.d_tot;
        ct = ds.c_tot;
        G = ds.groups;
        dg = dt / G;
        cg = ct / G;
        nwf = dt * kin + dt;
        nw = nwf + ct * cin + ct;
    }
};

// mesh channels of voxel i (x fastest, then y, then z)
__device__ __forceinline__ void mesh_of(const pam_block_desc_t &ds, int64_t i, float m[3])
{
    const uint32_t u = (uint32_t)i, W = (uint32_t)ds.dims[0], H = (uint32_t)ds.dims[1];  // N < 2^31
    const uint32_t row = u / W, x = u - row * W, zc = row / H, y = row - zc * H;
    m[0] = (float)x * ds.mesh_scale;
    m[1] = (float)y * ds.mesh_scale;
    m[2] = (float)zc * ds.mesh_scale;
}

typedef float floatx16 __attribute__((ext_vector_type(16)));

// acc += A (32 x K) B (K x 32), K even; A(m, k) and B(k, n) read by the
// lanes as the instruction lays them out (lane l: A(l % 32, k0 + l / 32),
// B(k0 + l / 32, l % 32)).  Wave-uniform: every lane takes part.
template <class FA, class FB>
__device__ __forceinline__ void mfma_tile(floatx16 &acc, int K, const FA &A, const FB &B)
{
    const int l = threadIdx.x & 63, mn = l & 31, kh = l >> 5;
    for (int k0 = 0; k0 < K; k0 += 2)
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(A(mn, k0 + kh), B(k0 + kh, mn), acc, 0, 0, 0);
}

// row of the 32 x 32 tile held by register r of this lane (the column is
// the lane mod 32)
__device__ __forceinline__ int tile_row(int r) { return 8 * (r >> 2) + 4 * ((threadIdx.x & 63) >> 5) + (r & 3); }

// Forward, 256 voxels per block: the rows [x; mesh] are staged in LDS
// (flat coalesced copies), then
//   feat = LeakyReLU([x; mesh] wf^T + bf)  and  val = x wv^T + bv
// run as 32 x 32 tiles on the matrix cores, written straight into the
// grouped layout.
struct FwdLayout {
    int PX, PK, PV;
    size_t wf, bf, wv, bv, sxm, total;
    __host__ __device__ explicit FwdLayout(const Sizes &z)
    {
        PX = 32 * ((z.kin + 31) / 32) + 1;
        PK = z.kin | 1;
        PV = z.cin | 1;
        wf = 0;
        bf = wf + (size_t)z.dt * PK;
        wv = bf + z.dt;
        bv = wv + (size_t)z.ct * PV;
        sxm = bv + z.ct;
        total = sxm + (size_t)kPrologueThreads * PX;
    }
};

__global__ __launch_bounds__(kPrologueThreads) void k_block_fwd(pam_block_desc_t ds, int64_t n,
                                                                const float *__restrict__ x,
                                                                const float *__restrict__ wf,
                                                                const float *__restrict__ bf,
                                                                const float *__restrict__ wv,
                                                                const float *__restrict__ bv,
                                                                float *__restrict__ feat, float *__restrict__ val)
{
    extern __shared__ float sh[];
    const Sizes z(ds);
    const FwdLayout Lo(z);
    float *swf = sh + Lo.wf, *sbf = sh + Lo.bf, *swv = sh + Lo.wv, *sbv = sh + Lo.bv, *sxm = sh + Lo.sxm;
    const int t = threadIdx.x, nthr = blockDim.x, wave = t >> 6, nwaves = nthr >> 6;
    const int V = kPrologueThreads;
    const int64_t base = (int64_t)blockIdx.x * V;
    const int nv = (int)min((int64_t)V, n - base);
    for (int e = t; e < z.dt * z.kin; e += nthr)
        swf[(e / z.kin) * Lo.PK + e % z.kin] = wf[e];
    for (int e = t; e < z.ct * z.cin; e += nthr)
        swv[(e / z.cin) * Lo.PV + e % z.cin] = wv[e];
    for (int e = t; e < z.dt; e += nthr)
        sbf[e] = bf[e];
    for (int e = t; e < z.ct; e += nthr)
        sbv[e] = bv[e];
    // x rows: one flat coalesced copy, kStageBatch loads in flight per thread
    const int total = nv * z.cin;
    const float *src = x + base * z.cin;
    for (int e0 = 0; e0 < total; e0 += nthr * kStageBatch) {
        float r[kStageBatch];
#pragma unroll
        for (int u = 0; u < kStageBatch; ++u) {
            const int e = e0 + u * nthr + t;
            r[u] = e < total ? src[e] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < kStageBatch; ++u) {
            const int e = e0 + u * nthr + t;
            if (e < total) {
                const int v = e / z.cin;
                sxm[v * Lo.PX + (e - v * z.cin)] = r[u];
            }
        }
    }
    {  // mesh channels, zero padding, zero rows past the end
        float *xr = sxm + t * Lo.PX;
        if (t < nv) {
            float m[3];
            mesh_of(ds, base + t, m);
            xr[z.cin] = m[0];
            xr[z.cin + 1] = m[1];
            xr[z.cin + 2] = m[2];
            for (int c = z.kin; c < Lo.PX; ++c)
                xr[c] = 0.0f;
        } else {
            for (int c = 0; c < Lo.PX; ++c)
                xr[c] = 0.0f;
        }
    }
    __syncthreads();
    const int lane32 = t & 31;
    // features: one column tile (d_tot <= 32) per 32-voxel tile
    for (int vt = wave; vt < V / 32; vt += nwaves) {
        floatx16 acc = {0};
        mfma_tile(
            acc, (z.kin + 1) & ~1, [&](int m, int k) { return sxm[(vt * 32 + m) * Lo.PX + k]; },
            [&](int k, int o) { return (k < z.kin && o < z.dt) ? swf[o * Lo.PK + k] : 0.0f; });
        const int o = lane32;
        if (o < z.dt) {
            const int og = o / z.dg, oj = o - og * z.dg;
            const float bo = sbf[o];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int v = vt * 32 + tile_row(r);
                if (v < nv) {
                    const float a = acc[r] + bo;
                    feat[((int64_t)og * n + base + v) * z.dg + oj] = a > 0.0f ? a : ds.slope * a;
                }
            }
        }
    }
    // descriptors: (32-voxel tile, 32-channel tile)
    const int otiles = (z.ct + 31) / 32;
    for (int tt = wave; tt < (V / 32) * otiles; tt += nwaves) {
        const int vt = tt / otiles, o0 = (tt - vt * otiles) * 32;
        floatx16 acc = {0};
        mfma_tile(
            acc, (z.cin + 1) & ~1, [&](int m, int k) { return sxm[(vt * 32 + m) * Lo.PX + k]; },
            [&](int k, int o) { return (k < z.cin && o0 + o < z.ct) ? swv[(o0 + o) * Lo.PV + k] : 0.0f; });
        const int o = o0 + lane32;
        if (o < z.ct) {
            const int og = o / z.cg, oj = o - og * z.cg;
            const float bo = sbv[o];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int v = vt * 32 + tile_row(r);
                if (v < nv)
                    val[((int64_t)og * n + base + v) * z.cg + oj] = acc[r] + bo;
            }
        }
    }
}

// Backward, per chunk of V voxels (V a multiple of 32), as three small
// dense contractions on the matrix cores (v_mfma_f32_32x32x2f32, 32 x 32
// output tiles, one tile per wave at a time):
//   Z  (V x d_tot)  = [x; mesh] wf^T + bf          -> dz = grad_f * LeakyReLU'(Z)
//   dx (V x c_in)   = [dz dv] [wf[:, :c_in]; wv]
//   G  (R x (kin+1)) += [dz dv]^T [x; mesh; 1]     (R = d_tot + c_tot)
// G holds every weight and bias gradient (the last column is the bias);
// each block accumulates its chunks in LDS and writes G as one partial in
// the weight layout.  LDS pitches are odd so that the strided operand reads
// fall in distinct banks.
struct BwdLayout {
    int V, R, Kc, RT, CT, PX, PA, PK;
    size_t wf, bf, wv, sxm, sa, sp, total;  // float offsets
    __host__ __device__ BwdLayout(const Sizes &z, int V_)
    {
        V = V_;
        R = z.dt + z.ct;
        Kc = z.kin + 1;
        RT = (R + 31) / 32;
        CT = (Kc + 31) / 32;
        PX = 32 * CT + 1;
        PA = 32 * RT + 1;
        PK = z.kin | 1;
        wf = 0;
        bf = wf + (size_t)z.dt * PK;
        wv = bf + z.dt;
        sxm = wv + (size_t)z.ct * z.cin;
        sa = sxm + (size_t)V * PX;
        sp = sa + (size_t)V * PA;
        total = sp + (size_t)R * Kc;
    }
};

__global__ __launch_bounds__(kPrologueThreads) void k_block_bwd(pam_block_desc_t ds, int64_t n, int V,
                                                                const float *__restrict__ x,
                                                                const float *__restrict__ wf,
                                                                const float *__restrict__ bf,
                                                                const float *__restrict__ wv,
                                                                const float *__restrict__ gf,
                                                                const float *__restrict__ gv,
                                                                float *__restrict__ dx, float *__restrict__ part)
{
    extern __shared__ float sh[];
    const Sizes z(ds);
    const BwdLayout Lo(z, V);
    float *swf = sh + Lo.wf, *sbf = sh + Lo.bf, *swv = sh + Lo.wv;
    float *sxm = sh + Lo.sxm, *sa = sh + Lo.sa, *sp = sh + Lo.sp;
    const int t = threadIdx.x, nthr = blockDim.x;
    const int wave = t >> 6, nwaves = nthr >> 6;
    for (int e = t; e < z.dt * z.kin; e += nthr)
        swf[(e / z.kin) * Lo.PK + e % z.kin] = wf[e];
    for (int e = t; e < z.dt; e += nthr)
        sbf[e] = bf[e];
    for (int e = t; e < z.ct * z.cin; e += nthr)
        swv[e] = wv[e];
    for (int e = t; e < Lo.R * Lo.Kc; e += nthr)
        sp[e] = 0.0f;
    const int64_t nchunks = (n + V - 1) / V;
    for (int64_t ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
        const int64_t base = ch * V;
        const int nv = (int)min((int64_t)V, n - base);
        __syncthreads();  // the previous chunk is consumed
        // Stage the rows [x; mesh; 1; 0...] and [0 (dz, filled below); dv; 0...].
        // The chunk's x rows and each group's dv rows are contiguous in
        // memory: flat coalesced copies, kStageBatch loads in flight per
        // thread before their stores.
        for (int v = t >> 5; v < V; v += nthr >> 5) {  // constant columns, 32 lanes per row
            float *xr = sxm + v * Lo.PX, *ar = sa + v * Lo.PA;
            const int lane32 = t & 31;
            for (int c = z.cin + lane32; c < Lo.PX; c += 32)
                xr[c] = (v < nv && c == z.kin) ? 1.0f : 0.0f;
            if (v >= nv)
                for (int c = lane32; c < z.cin; c += 32)
                    xr[c] = 0.0f;
            for (int c = lane32; c < Lo.PA; c += 32)
                if (c < z.dt || c >= Lo.R || v >= nv)
                    ar[c] = 0.0f;
        }
        __syncthreads();  // the mesh below overwrites three of those columns
        for (int v = t; v < nv; v += nthr) {
            float m[3];
            mesh_of(ds, base + v, m);
            sxm[v * Lo.PX + z.cin] = m[0];
            sxm[v * Lo.PX + z.cin + 1] = m[1];
            sxm[v * Lo.PX + z.cin + 2] = m[2];
        }
        auto stage = [&](const float *src, int cols, float *dst, int pitch, int col0) {
            const int total = nv * cols;
            for (int e0 = 0; e0 < total; e0 += nthr * kStageBatch) {
                float r[kStageBatch];
#pragma unroll
                for (int u = 0; u < kStageBatch; ++u) {
                    const int e = e0 + u * nthr + t;
                    r[u] = e < total ? src[e] : 0.0f;
                }
#pragma unroll
                for (int u = 0; u < kStageBatch; ++u) {
                    const int e = e0 + u * nthr + t;
                    if (e < total) {
                        const int v = e / cols;
                        dst[v * pitch + col0 + (e - v * cols)] = r[u];
                    }
                }
            }
        };
        stage(x + base * z.cin, z.cin, sxm, Lo.PX, 0);
        for (int g = 0; g < z.G; ++g)
            stage(gv + ((int64_t)g * n + base) * z.cg, z.cg, sa, Lo.PA, z.dt + g * z.cg);
        __syncthreads();
        // Z = [x; mesh] wf^T over 32-voxel tiles (d_tot <= 32: one column tile)
        for (int vt = wave; vt < V / 32; vt += nwaves) {
            floatx16 acc = {0};
            mfma_tile(
                acc, (z.kin + 1) & ~1, [&](int m, int k) { return sxm[(vt * 32 + m) * Lo.PX + k]; },
                [&](int k, int o) { return (k < z.kin && o < z.dt) ? swf[o * Lo.PK + k] : 0.0f; });
            const int o = t & 31;
            const int og = o < z.dt ? o / z.dg : 0, oj = o - og * z.dg;
            const float bo = o < z.dt ? sbf[o] : 0.0f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int v = vt * 32 + tile_row(r);
                if (o < z.dt && v < nv) {
                    const float zz = acc[r] + bo;
                    const float gin = gf[((int64_t)og * n + base + v) * z.dg + oj];
                    sa[v * Lo.PA + o] = zz > 0.0f ? gin : ds.slope * gin;
                }
            }
        }
        __syncthreads();
        // dx = [dz dv] [wf[:, :c_in]; wv] over (voxel tile, input-channel tile)
        const int ctiles = (z.cin + 31) / 32;
        for (int tt = wave; tt < (V / 32) * ctiles; tt += nwaves) {
            const int vt = tt / ctiles, c0 = (tt - vt * ctiles) * 32;
            floatx16 acc = {0};
            mfma_tile(
                acc, (Lo.R + 1) & ~1, [&](int m, int k) { return sa[(vt * 32 + m) * Lo.PA + k]; },
                [&](int k, int c) {
                    const int cc = c0 + c;
                    if (cc >= z.cin || k >= Lo.R)
                        return 0.0f;
                    return k < z.dt ? swf[k * Lo.PK + cc] : swv[(k - z.dt) * z.cin + cc];
                });
            const int cc = c0 + (t & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int v = vt * 32 + tile_row(r);
                if (cc < z.cin && v < nv)
                    dx[(base + v) * z.cin + cc] = acc[r];
            }
        }
        // G += [dz dv]^T [x; mesh; 1] over (row tile, column tile)
        for (int tt = wave; tt < Lo.RT * Lo.CT; tt += nwaves) {
            const int r0 = (tt / Lo.CT) * 32, c0 = (tt % Lo.CT) * 32;
            floatx16 acc = {0};
            mfma_tile(
                acc, V, [&](int m, int v) { return sa[v * Lo.PA + r0 + m]; },
                [&](int v, int c) { return sxm[v * Lo.PX + c0 + c]; });
            const int cc = c0 + (t & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rr = r0 + tile_row(r);
                if (rr < Lo.R && cc < Lo.Kc)
                    sp[rr * Lo.Kc + cc] += acc[r];
            }
        }
    }
    __syncthreads();
    // G in the weight layout: wf (dt x kin), bf, wv (ct x cin), bv
    for (int e = t; e < z.nw; e += nthr) {
        float g;
        if (e < z.dt * z.kin) {
            const int o = e / z.kin;
            g = sp[o * Lo.Kc + (e - o * z.kin)];
        } else if (e < z.nwf) {
            g = sp[(e - z.dt * z.kin) * Lo.Kc + z.kin];
        } else if (e < z.nwf + z.ct * z.cin) {
            const int q = e - z.nwf, o = q / z.cin;
            g = sp[(z.dt + o) * Lo.Kc + (q - o * z.cin)];
        } else {
            g = sp[(z.dt + (e - z.nwf - z.ct * z.cin)) * Lo.Kc + z.kin];
        }
        part[(int64_t)blockIdx.x * z.nw + e] = g;
    }
}

// Sum of the per-block partials: a block takes kReduceEntries consecutive
// entries; thread row j (of kReduceThreads / kReduceEntries) sums partial
// blocks j, j + rows, ... (coalesced rows of entries), then the rows are
// added in a fixed order (deterministic).  Entries are scattered to the four
// gradient arrays.
__global__ __launch_bounds__(kReduceThreads) void k_block_reduce(const float *__restrict__ part, int nblocks,
                                                                 pam_block_desc_t ds, float *__restrict__ dwf,
                                                                 float *__restrict__ dbf, float *__restrict__ dwv,
                                                                 float *__restrict__ dbv)
{
    constexpr int R = kReduceThreads / kReduceEntries;
    __shared__ float rows[R][kReduceEntries];
    const Sizes z(ds);
    const int c = threadIdx.x % kReduceEntries, j = threadIdx.x / kReduceEntries;
    const int e = blockIdx.x * kReduceEntries + c;
    float acc = 0.0f;
    if (e < z.nw)
        for (int b = j; b < nblocks; b += R)
            acc += part[(int64_t)b * z.nw + e];
    rows[j][c] = acc;
    __syncthreads();
    if (j != 0 || e >= z.nw)
        return;
    acc = 0.0f;
    for (int r = 0; r < R; ++r)
        acc += rows[r][c];
    if (e < z.dt * z.kin)
        dwf[e] = acc;
    else if (e < z.nwf)
        dbf[e - z.dt * z.kin] = acc;
    else if (e < z.nwf + z.ct * z.cin)
        dwv[e - z.nwf] = acc;
    else
        dbv[e - z.nwf - z.ct * z.cin] = acc;
}

}  // namespace

size_t block_fwd_lds(const pam_block_desc_t &ds) { return FwdLayout(Sizes(ds)).total * sizeof(float); }

// voxels per chunk of the backward pass: the largest of 128, 64, 32 whose
// LDS layout fits the budget
static int block_bwd_chunk(const pam_block_desc_t &ds)
{
    const Sizes z(ds);
    for (int V = 128; V > 32; V /= 2)
        if (BwdLayout(z, V).total * sizeof(float) <= kBwdLdsBudget)
            return V;
    return 32;
}

size_t block_bwd_lds(const pam_block_desc_t &ds)
{
    return BwdLayout(Sizes(ds), block_bwd_chunk(ds)).total * sizeof(float);
}

int block_bwd_blocks(const pam_block_desc_t &ds)
{
    const int64_t n = (int64_t)ds.dims[0] * ds.dims[1] * ds.dims[2];
    const int V = block_bwd_chunk(ds);
    return (int)std::max<int64_t>(1, std::min<int64_t>((n + V - 1) / V, 1024));
}

size_t block_partials(const pam_block_desc_t &ds) { return (size_t)Sizes(ds).nw; }

hipError_t launch_block_fwd(const pam_block_desc_t &ds, const float *x, const float *wf, const float *bf,
                            const float *wv, const float *bv, float *feat, float *val, hipStream_t s)
{
    const int64_t n = (int64_t)ds.dims[0] * ds.dims[1] * ds.dims[2];
    if (n <= 0)
        return hipSuccess;
    const size_t lds = block_fwd_lds(ds);
    hipError_t e = hipFuncSetAttribute((const void *)k_block_fwd, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_block_fwd, dim3((unsigned)((n + kPrologueThreads - 1) / kPrologueThreads)),
                       dim3(kPrologueThreads), lds, s, ds, n, x, wf, bf, wv, bv, feat, val);
    return hipGetLastError();
}

hipError_t launch_block_bwd(const pam_block_desc_t &ds, const float *x, const float *wf, const float *bf,
                            const float *wv, const float *gf, const float *gv, float *dx, float *dwf, float *dbf,
                            float *dwv, float *dbv, float *part, hipStream_t s, int nblocks)
{
    const int64_t n = (int64_t)ds.dims[0] * ds.dims[1] * ds.dims[2];
    const size_t lds = block_bwd_lds(ds);
    hipError_t e = hipFuncSetAttribute((const void *)k_block_bwd, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess)
        return e;
    // the chunk loop is grid-strided, so any block count covers the volume
    const int nb = nblocks > 0 ? std::min(nblocks, block_bwd_blocks(ds)) : block_bwd_blocks(ds);
    hipLaunchKernelGGL(k_block_bwd, dim3(nb), dim3(kPrologueThreads), lds, s, ds, n, block_bwd_chunk(ds), x, wf,
                       bf, wv, gf, gv, dx, part);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    const int P = (int)block_partials(ds);
    hipLaunchKernelGGL(k_block_reduce, dim3((P + kReduceEntries - 1) / kReduceEntries), dim3(kReduceThreads), 0, s,
                       part, nb, ds, dwf, dbf, dwv, dbv);
    return hipGetLastError();
}

// Partials of the allocation-free backward pass: a fixed array in device
// memory, one copy per GPU, kept until the process ends.  In host code the
// array's name is not a device address; its address on the current device
// is taken once per device with hipGetSymbolAddress and used everywhere the
// host needs it.
static __device__ __align__(256) float scratch[kBlockScratchFloats];

hipError_t block_scratch(float **out)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static float *addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        addr[dev] = (float *)p;
    }
    *out = addr[dev];
    return hipSuccess;
}

}  // namespace pam

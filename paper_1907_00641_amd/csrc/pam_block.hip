// HIP kernels (gfx950) of the permutohedral block's prologue (Joutard et al.
// 2019, Section 3 and the Fig. 2 caption): features are a 1x1x1 convolution
// of the input channels with a mesh of spatial coordinates appended,
// followed by a Leaky-ReLU; descriptors are a 1x1x1 convolution of the input
// channels; both are split channel-wise into groups and written in the
// grouped layout a batched lattice build takes (group g: rows g N .. g N +
// N - 1, its slice of the channels).
//
//   forward : one thread per voxel; the block's input rows are staged in LDS
//             with coalesced loads, the weights sit in LDS and are read as
//             broadcasts.
//   backward: one thread per voxel for the input gradient; the weight and
//             bias gradients (sums over all voxels of outer products) are
//             accumulated per block in LDS, one entry per thread slot,
//             written as per-block partials and summed over the blocks in a
//             fixed order by a second kernel (deterministic).
#include "pam_internal.h"

#include <algorithm>

namespace pam {

namespace {

constexpr int kPrologueThreads = 256;
constexpr size_t kBwdLdsBudget = 96 << 10;  // LDS bytes the backward chunk size aims for
constexpr int kReduceEntries = 32;          // gradient entries per block of the reduction
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

// weights into LDS: wf (dt x kin), bf (dt), wv (ct x cin), bv (ct)
__device__ void load_weights(const Sizes &z, const float *wf, const float *bf, const float *wv, const float *bv,
                             float *s)
{
    for (int e = threadIdx.x; e < z.nw; e += blockDim.x) {
        float w;
        if (e < z.dt * z.kin)
            w = wf[e];
        else if (e < z.nwf)
            w = bf[e - z.dt * z.kin];
        else if (e < z.nwf + z.ct * z.cin)
            w = wv[e - z.nwf];
        else
            w = bv ? bv[e - z.nwf - z.ct * z.cin] : 0.0f;
        s[e] = w;
    }
}

// mesh channels of voxel i (x fastest, then y, then z)
__device__ __forceinline__ void mesh_of(const pam_block_desc_t &ds, int64_t i, float m[3])
{
    const int64_t W = ds.dims[0], H = ds.dims[1];
    m[0] = (float)(i % W) * ds.mesh_scale;
    m[1] = (float)((i / W) % H) * ds.mesh_scale;
    m[2] = (float)(i / (W * H)) * ds.mesh_scale;
}

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
    const int pitch = z.cin | 1;  // odd pitch: rows of consecutive voxels start in different banks
    float *sw = sh, *sx = sh + z.nw;
    load_weights(z, wf, bf, wv, bv, sw);
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * kPrologueThreads;
    const int nt = (int)min((int64_t)kPrologueThreads, n - base);
    for (int e = t; e < nt * z.cin; e += kPrologueThreads) {
        const int p = e / z.cin, c = e - p * z.cin;
        sx[p * pitch + c] = x[base * z.cin + e];
    }
    __syncthreads();
    if (t >= nt)
        return;
    const int64_t i = base + t;
    float m[3];
    mesh_of(ds, i, m);
    const float *xr = sx + t * pitch;
    for (int o = 0; o < z.dt; ++o) {
        const float *w = sw + o * z.kin;
        float acc = sw[z.dt * z.kin + o];
        for (int k = 0; k < z.cin; ++k)
            acc += w[k] * xr[k];
        acc += w[z.cin] * m[0] + w[z.cin + 1] * m[1] + w[z.cin + 2] * m[2];
        const float f = acc > 0.0f ? acc : ds.slope * acc;
        const int g = o / z.dg;
        feat[((int64_t)g * n + i) * z.dg + (o - g * z.dg)] = f;
    }
    for (int o = 0; o < z.ct; ++o) {
        const float *w = sw + z.nwf + o * z.cin;
        float acc = sw[z.nwf + z.ct * z.cin + o];
        for (int k = 0; k < z.cin; ++k)
            acc += w[k] * xr[k];
        const int g = o / z.cg;
        val[((int64_t)g * n + i) * z.cg + (o - g * z.cg)] = acc;
    }
}

// Backward.  Per chunk of V voxels (V <= blockDim, one thread each): the
// pre-activations are recomputed, dz = grad_f * LeakyReLU' and the input
// gradient formed, and [x; mesh], dz and dv staged in LDS; then every
// thread adds the chunk's contribution to its entries of the block's
// partial weight gradients (LDS, entry e owned by thread e mod blockDim).
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
    const int P = z.nw;  // gradient entries, laid out like the weights
    float *sw = sh;
    float *sp = sw + z.nw;                         // partial gradients
    float *sxm = sp + P;           // V x kin
    float *sdz = sxm + V * z.kin;  // V x dt
    float *sdv = sdz + V * z.dt;   // V x ct
    load_weights(z, wf, bf, wv, nullptr, sw);
    const int t = threadIdx.x;
    for (int e = t; e < P; e += blockDim.x)
        sp[e] = 0.0f;
    const int64_t nchunks = (n + V - 1) / V;
    for (int64_t ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
        const int64_t base = ch * V;
        const int nv = (int)min((int64_t)V, n - base);
        __syncthreads();  // the previous chunk's LDS tiles are consumed
        if (t < V) {
            float *xm = sxm + t * z.kin, *dz = sdz + t * z.dt, *dv = sdv + t * z.ct;
            if (t < nv) {
                const int64_t i = base + t;
                for (int k = 0; k < z.cin; ++k)
                    xm[k] = x[i * z.cin + k];
                mesh_of(ds, i, xm + z.cin);
                for (int o = 0; o < z.dt; ++o) {
                    const float *w = sw + o * z.kin;
                    float acc = sw[z.dt * z.kin + o];
                    for (int k = 0; k < z.kin; ++k)
                        acc += w[k] * xm[k];
                    const int g = o / z.dg;
                    const float g_in = gf[((int64_t)g * n + i) * z.dg + (o - g * z.dg)];
                    dz[o] = acc > 0.0f ? g_in : ds.slope * g_in;
                }
                for (int o = 0; o < z.ct; ++o) {
                    const int g = o / z.cg;
                    dv[o] = gv[((int64_t)g * n + i) * z.cg + (o - g * z.cg)];
                }
                for (int k = 0; k < z.cin; ++k) {
                    float acc = 0.0f;
                    for (int o = 0; o < z.dt; ++o)
                        acc += sw[o * z.kin + k] * dz[o];
                    for (int o = 0; o < z.ct; ++o)
                        acc += sw[z.nwf + o * z.cin + k] * dv[o];
                    dx[i * z.cin + k] = acc;
                }
            } else {  // past the end: zero rows add nothing
                for (int k = 0; k < z.kin; ++k)
                    xm[k] = 0.0f;
                for (int o = 0; o < z.dt; ++o)
                    dz[o] = 0.0f;
                for (int o = 0; o < z.ct; ++o)
                    dv[o] = 0.0f;
            }
        }
        __syncthreads();
        for (int e = t; e < P; e += blockDim.x) {
            float acc = 0.0f;
            if (e < z.dt * z.kin) {
                const int o = e / z.kin, k = e - o * z.kin;
                for (int v = 0; v < V; ++v)
                    acc += sdz[v * z.dt + o] * sxm[v * z.kin + k];
            } else if (e < z.nwf) {
                const int o = e - z.dt * z.kin;
                for (int v = 0; v < V; ++v)
                    acc += sdz[v * z.dt + o];
            } else if (e < z.nwf + z.ct * z.cin) {
                const int o = (e - z.nwf) / z.cin, k = (e - z.nwf) - o * z.cin;
                for (int v = 0; v < V; ++v)
                    acc += sdv[v * z.ct + o] * sxm[v * z.kin + k];
            } else {
                const int o = e - z.nwf - z.ct * z.cin;
                for (int v = 0; v < V; ++v)
                    acc += sdv[v * z.ct + o];
            }
            sp[e] += acc;
        }
    }
    __syncthreads();
    for (int e = t; e < P; e += blockDim.x)
        part[(int64_t)blockIdx.x * P + e] = sp[e];
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

size_t block_fwd_lds(const pam_block_desc_t &ds)
{
    const Sizes z(ds);
    return sizeof(float) * ((size_t)z.nw + (size_t)kPrologueThreads * (z.cin | 1));
}

// voxels per chunk of the backward pass: a whole block's worth when the
// tiles fit the LDS budget, else 64
static int block_bwd_chunk(const pam_block_desc_t &ds)
{
    const Sizes z(ds);
    const size_t per = sizeof(float) * (z.kin + z.dt + z.ct), fixed = sizeof(float) * 2 * (size_t)z.nw;
    return fixed + per * kPrologueThreads <= kBwdLdsBudget ? kPrologueThreads : 64;
}

size_t block_bwd_lds(const pam_block_desc_t &ds)
{
    const Sizes z(ds);
    return sizeof(float) * (2 * (size_t)z.nw + (size_t)block_bwd_chunk(ds) * (z.kin + z.dt + z.ct));
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
                            float *dwv, float *dbv, float *part, hipStream_t s)
{
    const int64_t n = (int64_t)ds.dims[0] * ds.dims[1] * ds.dims[2];
    const size_t lds = block_bwd_lds(ds);
    hipError_t e = hipFuncSetAttribute((const void *)k_block_bwd, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess)
        return e;
    const int nb = block_bwd_blocks(ds);
    hipLaunchKernelGGL(k_block_bwd, dim3(nb), dim3(kPrologueThreads), lds, s, ds, n, block_bwd_chunk(ds), x, wf,
                       bf, wv, gf, gv, dx, part);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    const int P = (int)block_partials(ds);
    hipLaunchKernelGGL(k_block_reduce, dim3((P + kReduceEntries - 1) / kReduceEntries), dim3(kReduceThreads), 0, s,
                       part, nb, ds, dwf, dbf, dwv, dbv);
    return hipGetLastError();
}

}  // namespace pam

// Measurement utility (not part of the filter): a copy of fp32 rows whose
// read and write positions follow a permutation or the identity.  Timed by
// the benchmark to measure what HBM delivers for the per-point kernels'
// access pattern: value rows of C floats read or written at the original
// index of points taken in the simplex-sorted order, i.e. at random rows.
#include "pam_device.h"

namespace pam {

// Thread per 16-byte piece; a row of row4 pieces is read from source row
// (mode & 1 ? perm[i] : i) and written to destination row
// (mode & 2 ? perm[i] : i).  Rows outside [0, n) are skipped.
__global__ __launch_bounds__(kBlock) void k_copy_rows(const float4 *__restrict__ src, float4 *__restrict__ dst,
                                                      const int32_t *__restrict__ perm, int64_t n, int row4,
                                                      int mode)
{
    const int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (e >= n * row4)
        return;
    const int64_t i = e / row4;
    const int l = (int)(e - i * row4);
    const int64_t p = (mode & 3) ? (int64_t)perm[i] : i;
    if (p < 0 || p >= n)
        return;
    const int64_t r = (mode & 1) ? p : i, w = (mode & 2) ? p : i;
    dst[w * row4 + l] = src[r * row4 + l];
}

hipError_t launch_copy_rows(const float *src, float *dst, const int32_t *perm, int64_t n, int32_t row_floats,
                            int32_t mode, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    const int row4 = row_floats / 4;
    hipLaunchKernelGGL(k_copy_rows, dim3(blocks_for(n * row4)), dim3(kBlock), 0, s,
                       reinterpret_cast<const float4 *>(src), reinterpret_cast<float4 *>(dst), perm, n, row4, mode);
    return hipGetLastError();
}

}  // namespace pam

/*
 * pam_probe.h -- measurement utility of the MI355X permutohedral-lattice
 * filter library (libpam_lattice.so), kept apart from the filter's own ABI
 * in pam_lattice.h.  It is not part of the filter: the benchmark times it to
 * measure the HBM ceilings of the access patterns the filter kernels use
 * (rows copied in order and through a permutation).  Conventions (device
 * pointers, streams, status codes, pam_last_error) as in pam_lattice.h.
 */
#ifndef PAM_PROBE_H
#define PAM_PROBE_H

#include "pam_lattice.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Measurement utility, not part of the filter: copies n rows of row_floats
 * fp32 values from src to dst (device pointers, 16-byte aligned, not
 * overlapping; row_floats a positive multiple of 4).  Row i is read from
 * source row perm[i] when bit 0 of mode is set, else i, and written to
 * destination row perm[i] when bit 1 is set, else i; perm (device, n int32)
 * is read only when mode is not 0, and entries outside [0, n) skip their row.
 * The benchmark times it to measure the HBM ceiling of sequential and
 * random-row access.  Asynchronous; argument errors return
 * PAM_ERR_INVALID_ARGUMENT before anything is enqueued.
 */
pam_status_t pam_probe_copy_rows(const float *src, float *dst, const int32_t *perm, int64_t n,
                                 int32_t row_floats, int32_t mode, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PAM_PROBE_H */

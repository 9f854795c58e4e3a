// Internal declarations shared by the kernels (pam_build.hip,
// pam_filter.hip) and the C ABI (pam_abi.cpp) of the permutohedral-lattice
// filter library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/pam_lattice.h"
#include "../../include/pam_probe.h"

namespace pam {

constexpr int kMaxD = PAM_MAX_D;
constexpr uint64_t kEmptyKey = ~0ull;  // hash slot sentinel; packed keys use <= 63 bits

// device-side status bits (Ctl::flags)
constexpr uint32_t kFlagTableFull = 1u;  // insertion probed the whole table (the host adds: load > cap / 2)
constexpr uint32_t kFlagKeyRange = 2u;   // keys need more than 63 bits
constexpr uint32_t kFlagBadFeature = 4u; // non-finite feature or |x| > 2^24
constexpr uint32_t kFlagLayoutMiss = 8u; // a key does not fit the fixed layout of the fast insert

// fp32 entries of the embedding matrix E = alpha * Q, (d+1) x d.  Every
// entry above the diagonal band of column j equals pos[j]; the single
// negative entry of column j (row j+1) is neg[j].  inv = fp32(1/(d+1)).
struct Elev {
    float pos[kMaxD];
    float neg[kMaxD];
    float inv;
    float raw_scale;  // fp32(1/G_d)
    // the same entries in fp64: the barycentric weights are taken from an
    // fp64 elevation, so that their accuracy does not degrade with |x|
    double pos64[kMaxD];
    double neg64[kMaxD];
};

// Packing of a vertex key into 63 bits.  Vertex k of a simplex has every
// coordinate equal to k + (d+1) t_c; the key stores k in the low kbits bits
// and, for each stored coordinate c < d, t_c - lo[c] in bits[c] bits at
// shift[c]; the point group (batched builds) takes gbits bits at gshift.
struct KeyLayout {
    int32_t lo[kMaxD];
    int32_t shift[kMaxD];
    int32_t bits[kMaxD];
    int32_t kbits;
    int32_t gshift;
    int32_t gbits;
    int32_t total_bits;
};

// Point groups of a batched build: points [gstart[g], gstart[g+1]) form
// group g (device array of G+1 entries; G = 1 and gstart = null for one
// group).
struct Groups64 {
    const int64_t *gstart;
    int32_t G;
};

// Small device-resident control block of a lattice handle.
struct Ctl {
    int32_t qmin[kMaxD];  // range of the rounded remainder-0 quotients
    int32_t qmax[kMaxD];
    KeyLayout lay;
    uint32_t flags;  // kFlag* bits
    uint32_t count;  // keys inserted into the hash table
    uint32_t nvert;  // ids handed out by compaction
    uint32_t pad;
};

enum KernelKind : int32_t {
    kKRange = 0,
    kKLayout,
    kKFill,
    kKInsert,
    kKCompact,
    kKResolve,
    kKScan,
    kKScatter,
    kKTiles,
    kKSplat,
    kKBlur,
    kKSlice,
    kKSplatBwd,
    kKSliceBwd,
    kKSplatAug,
    kKSliceAug,
    kKNumKinds
};

const char *kernel_name(int32_t kind);

// launch parameters shared by the filter kernels, which work in the
// simplex-sorted point order
struct FilterArgs {
    const uint8_t *pts;    // per sorted point: barycentric weights and ranks
    const int32_t *svert;  // per sorted point: its d+1 vertex ids
    const int32_t *perm;   // per sorted point: its index in the caller's arrays
    int64_t n;
    int32_t c;       // value channels
    int32_t ld;      // lattice row stride: c (+1 weight column when normalised),
                     // rounded up to a multiple of 4 floats
    int32_t normalize;
    int32_t vec;     // channels per lane access: 4 (float4) or 1
    const float *feat;  // the build's n x d features (augmented-channel passes)
    // Asymmetric filter: original points [0, src_n) carry the values (rows of
    // val and grad_val), points [tgt_0, n) are read out (row i - tgt_0 of out
    // and grad_out).  The symmetric filter has src_n = n, tgt_0 = 0.
    int64_t src_n;
    int64_t tgt_0;
    int32_t side;    // the splat's input rows: 0 = val (sources), 1 = grad_out (targets)
    Elev E;
};

// Bytes of a per-tile record as each kernel translation unit lays it out;
// the host checks that they agree with its own layout (a library linked
// from objects compiled against different headers would index the tile
// buffers with one size and allocate them with another).
size_t tile_record_bytes_build(int d);
size_t tile_record_bytes_filter(int d);

// ---- launchers (pam_build.hip, pam_filter.hip); all return the hipError_t of the launch
// the range pass writes per-block partials: kRangeBlocks * (2d + 1) ints
// (at most kRangePartInts); it also clears the hash table (cap slots)
constexpr int kRangeBlocks = 2048;
constexpr int64_t kRangePartInts = (int64_t)kRangeBlocks * (2 * kMaxD + 1);
// measurement utility (pam_probe.hip)
hipError_t launch_copy_rows(const float *src, float *dst, const int32_t *perm, int64_t n, int32_t row_floats,
                            int32_t mode, hipStream_t s);
hipError_t launch_range(int d, const float *feat, int64_t n, const Elev &E, int32_t *part, uint64_t *tkeys,
                        uint64_t cap, hipStream_t s);
hipError_t launch_layout(int d, int64_t n, int gbits, Ctl *ctl, const int32_t *part, hipStream_t s);
hipError_t launch_fill_f32(float *p, float value, int64_t count, hipStream_t s);
// fixed: null to take the key layout the range pass computed (ctl->lay);
// else a fixed layout (fixed_layout) that the insert checks every key
// against (kFlagLayoutMiss) and writes to ctl->lay; it also flags
// non-finite features.  The fixed layout needs a table cleared and the
// control block's flags and counters zeroed (the previous build's tiles
// launch leaves them so).
hipError_t launch_insert_tiles(int d, const float *feat, int64_t n, const Elev &E, const Groups64 &grp, Ctl *ctl,
                               const KeyLayout *fixed, uint64_t *tkeys, uint64_t cap, uint8_t *tiles,
                               hipStream_t s);
// A key layout that needs no range pass: every stored coordinate's quotient
// in [-2^(b-1), 2^(b-1)) with b bits, b = (63 - bits of k - gbits) / d;
// false when b < 6 (then the range pass always runs).
bool fixed_layout(int d, int gbits, KeyLayout *lay);
// also zeroes bucket[0..M)
hipError_t launch_compact(const uint64_t *tkeys, int32_t *tids, uint64_t *vkeys, int32_t *bucket, uint64_t cap,
                          Ctl *ctl, hipStream_t s);
hipError_t launch_resolve(int d, const float *feat, int64_t n, const Elev &E, const Groups64 &grp, const Ctl *ctl,
                          const uint64_t *tkeys, const int32_t *tids, uint64_t cap, uint8_t *tiles,
                          int32_t *vert, int32_t *bucket, int32_t *pos0, const uint64_t *vkeys, int64_t M,
                          int32_t *nbr, hipStream_t s);
// ints of scratch launch_exclusive_scan needs for `count` elements
int64_t scan_scratch_ints(int64_t count);
hipError_t launch_exclusive_scan(int32_t *x, int64_t count, int32_t *sums, hipStream_t s);
// ids from the tiles of consecutive points (ntiles, as the resolve left
// them), or from vert (natural order) for tiles that overflowed
hipError_t launch_scatter(int d, const float *feat, int64_t n, const Elev &E, const uint8_t *ntiles,
                          const int32_t *vert, const int32_t *start, const int32_t *pos0, int32_t *perm,
                          uint8_t *psort, int32_t *svert, hipStream_t s);
// also clears the first zelems floats (a multiple of 4) of z0 and z1, and,
// with tkeys, the next build's hash table (cap slots) and the flags and
// counters of ctl
hipError_t launch_sorted_tiles(int d, const int32_t *svert, int64_t n, uint8_t *tiles, float *z0, float *z1,
                               int64_t zelems, uint64_t *tkeys, uint64_t cap, Ctl *ctl, hipStream_t s);
// x onto L.  mode: kSplatModePlain (forward, or backward raw),
// kSplatModeNormBwd (x / z and the weight column b * gamma, with A the
// forward lattice), kSplatModeAug (d*C channels f_q x_c, a.ld wide).
// hA (plain mode, raw, c <= 32, float4 rows; else null): per sorted point
// and vertex k, <x_p, A[m_pk]> (the slice-side term of eq. 8), n x (d+1).
constexpr int kSplatModePlain = 0, kSplatModeNormBwd = 1, kSplatModeAug = 2;
// whether the backward splat of these arguments can form eq. 8's term (hA)
bool splat_forms_eq8_term(const FilterArgs &a);
hipError_t launch_splat(int d, const FilterArgs &a, const uint8_t *tiles, const float *x, const float *A,
                        int mode, float *L, float *hA, hipStream_t s);
hipError_t launch_blur(const float *in, float *out, const int32_t *nbr_j, int64_t M, int32_t ld,
                       hipStream_t s);
// two directions, a then b, in one pass (same result as two passes)
hipError_t launch_blur2(const float *in, float *out, const int32_t *nbr_a, const int32_t *nbr_b, int64_t M,
                        int32_t ld, hipStream_t s);
hipError_t launch_slice(int d, const FilterArgs &a, const uint8_t *tiles, const float *A, float *out,
                        hipStream_t s);
// hA: the backward splat's <g_p, A[m_pk]> (raw mode); then grad is not read
// for eq. 8 (null: formed here from grad and A)
hipError_t launch_slice_bwd(int d, const FilterArgs &a, const uint8_t *tiles, const float *val, const float *grad,
                            const float *A, const float *At, const float *hA, float *grad_val, float *grad_feat,
                            hipStream_t s);
// augmented-channel embedding gradient from A, At (a.ld wide) and the
// augmented lattices L1, L2 (ldq wide)
hipError_t launch_slice_aug(int d, const FilterArgs &a, const uint8_t *tiles, const float *val, const float *grad,
                            const float *A, const float *At, const float *L1, const float *L2, int32_t ldq,
                            float *grad_feat, hipStream_t s);
// per-point vertex ids and weights from the sorted records, in the caller's order
hipError_t launch_export_points(int d, const uint8_t *pts, const int32_t *svert, const int32_t *perm, int64_t n,
                                int32_t *vert, float *bary, hipStream_t s);
hipError_t launch_unpack_keys(int d, const uint64_t *vkeys, int64_t M, const Ctl *ctl,
                              int32_t *keys, hipStream_t s);
hipError_t launch_vertex_groups(const uint64_t *vkeys, int64_t M, const Ctl *ctl, int32_t *vgroup, hipStream_t s);

// permutohedral block prologue (pam_block.hip)
size_t block_fwd_lds(const pam_block_desc_t &ds);
size_t block_bwd_lds(const pam_block_desc_t &ds);
int block_bwd_blocks(const pam_block_desc_t &ds);
size_t block_partials(const pam_block_desc_t &ds);
hipError_t launch_block_fwd(const pam_block_desc_t &ds, const float *x, const float *wf, const float *bf,
                            const float *wv, const float *bv, float *feat, float *val, hipStream_t s);
// nblocks > 0 caps the backward pass's block count (and with it the
// partials it writes: nblocks * block_partials floats)
hipError_t launch_block_bwd(const pam_block_desc_t &ds, const float *x, const float *wf, const float *bf,
                            const float *wv, const float *gf, const float *gv, float *dx, float *dwf, float *dbf,
                            float *dwv, float *dbv, float *part, hipStream_t s, int nblocks = 0);
// fixed device array for the partials of pam_block_bwd_noalloc (floats)
constexpr size_t kBlockScratchFloats = (size_t)1 << 20;
// its address on the current device (taken once per device)
hipError_t block_scratch(float **out);

}  // namespace pam

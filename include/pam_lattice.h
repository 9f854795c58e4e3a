/*
 * pam_lattice.h -- C ABI of the MI355X (gfx950) permutohedral-lattice filter
 * behind the Permutohedral Attention Module (PAM; Joutard et al., 2019).
 *
 * The operation (paper, Section 2 "Permutohedral Attention Module"): given
 * feature/descriptor pairs (f_i, v_i), i < n, with f_i in R^d and v_i in R^C,
 * compute v'_i = sum_j K(f_i, f_j) v_j (eq. 4-5) in O(n) with the
 * permutohedral lattice: embed the features (operator E), splat the values
 * onto the enclosing simplices (S), blur along each of the d+1 lattice
 * directions in turn (B), slice back (Sl) -- eq. 6.  The kernel K is read as
 * exp(-|f_i - f_j|^2 / 2).  The backward pass gives the value gradient with
 * the same filter, blur directions reversed (eq. 7), and the feature
 * gradient from the blurred lattices of v and dL/dv' combined through the
 * embedding matrix and the per-point permutation (eq. 8).
 *
 * Conventions shared by every entry point:
 *   - Array pointers are DEVICE pointers unless stated otherwise; arrays are
 *     row-major, contiguous, fp32, 4-byte aligned.  The caller owns them.
 *   - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *     Work is enqueued on that stream; calls return before it finishes,
 *     except where a call says it synchronises.
 *   - No exception crosses the ABI.  Argument errors are detected on the host
 *     before anything is enqueued, and leave outputs untouched.  Errors of
 *     earlier asynchronous work surface as PAM_ERR_DEVICE on a later call.
 *     pam_last_error() gives a thread-local text for the last failure.
 *   - A handle is used from one host thread and one stream at a time.
 *     Separate handles are independent.
 *   - Logging: the environment variable PAM_LOG_LEVEL (read once) set to 1
 *     prints one line per build and filter call on stderr (sizes, vertex
 *     count, flags); 2 also prints every failure with its message.
 *   - PAM_FUSE_EQ8=1 in the environment (read at every pam_filter_bwd call;
 *     raw mode, c <= 32, 16-byte aligned rows of a multiple of 4 channels):
 *     the splat of grad_out also forms the slice-side term of eq. 8, so the
 *     backward slice does not read grad_out again.  Same results up to fp32
 *     summation order; off by default (slower overall on MI355X).
 */
#ifndef PAM_LATTICE_H
#define PAM_LATTICE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pam_lattice_s *pam_lattice_t; /* opaque; owns its device buffers */

typedef enum {
    PAM_OK = 0,
    PAM_ERR_INVALID_ARGUMENT = 1, /* null pointer, size out of range, unknown flag */
    PAM_ERR_OUT_OF_MEMORY = 2,    /* a device allocation failed */
    PAM_ERR_CAPACITY = 3,         /* lattice needs more than half the hash table, regrowth disabled */
    PAM_ERR_KEY_RANGE = 4,        /* a feature is not finite, or the lattice keys
                                     do not fit the 63-bit packed key */
    PAM_ERR_STATE = 5,            /* bwd without a matching fwd on this lattice */
    PAM_ERR_DEVICE = 6            /* a HIP runtime call or kernel failed */
} pam_status_t;

/* flags for pam_filter_fwd / pam_filter_bwd */
#define PAM_NORMALIZE 1u /* divide by the filtered constant-1 channel */
#define PAM_EGRAD_AUGMENTED 2u /* pam_filter_bwd: grad_feat by augmented channels (raw mode only) */

#define PAM_MAX_D 16
#define PAM_MAX_C 1024
#define PAM_MAX_GROUPS 65536

/*
 * Build (or rebuild) the sparse lattice of the features: operator E of eq. 6
 * plus the vertex set it touches (Section 2, Fig. 1 caption: the features
 * are embedded in a hyperplane of R^{d+1} partitioned into simplices).
 *   feat : n x d fp32 features (device).  Borrowed: pam_filter_bwd with
 *          PAM_EGRAD_AUGMENTED re-reads it, so it must stay valid and
 *          unchanged until the next build on the handle or its destruction.
 *          The other calls read only what the build derived from it.
 *   n    : number of points, 0 <= n, n * (d+1) < 2^31.
 *   d    : feature dimension, 1 <= d <= PAM_MAX_D.
 *   lat  : *lat == NULL creates a handle on the current HIP device; otherwise
 *          the handle is rebuilt in place, reusing its buffers (grown when
 *          needed) and sizing the hash table from the previous vertex count.
 * Synchronises the stream after each insert attempt, to read back the vertex
 * count: once normally; once more when a rebuild's keys do not fit the fixed
 * key layout it tries first (it then measures their range), and after each
 * regrowth of the hash table.  Invalidates the forward state kept for
 * pam_filter_bwd.
 */
pam_status_t pam_lattice_build(const float *feat, int64_t n, int32_t d, void *stream,
                               pam_lattice_t *lat);

/*
 * Batched build: the points form `groups` independent point sets, filtered
 * in one launch sequence as if each had its own lattice (Section 3: the
 * permutohedral block splits features and values into two groups and runs
 * the module on each; a batch of volumes is the same case).  The group id
 * is a field of every vertex key, so no vertex, blur link or contribution
 * crosses groups.  fwd/bwd then take the n x c values of all groups
 * together.
 *   group_start : host array of groups + 1 offsets, group_start[0] = 0,
 *                 nondecreasing, group_start[groups] = n; points
 *                 [group_start[g], group_start[g+1]) form group g (empty
 *                 groups allowed).  Read during the call only.
 *   groups      : 1 <= groups <= PAM_MAX_GROUPS (groups = 1 is
 *                 pam_lattice_build; group_start may then be NULL).
 * Other arguments, buffers and errors as pam_lattice_build; the group field
 * counts towards the 63 key bits (PAM_ERR_KEY_RANGE when they run out).
 */
pam_status_t pam_lattice_build_groups(const float *feat, int64_t n, int32_t d, const int64_t *group_start,
                                      int32_t groups, void *stream, pam_lattice_t *lat);

/*
 * Forward filter, eq. 6: out = Sl(B(S(E(f), val)), E(f)).
 *   val   : n x c fp32 values (device); out : n x c fp32 (device); they must
 *           not overlap.  1 <= c <= PAM_MAX_C.
 *   flags : 0 = raw mode, out approximates sum_j exp(-|f_i-f_j|^2/2) v_j
 *           (the lattice result times the constant 1/G_d);
 *           PAM_NORMALIZE = the lattice result divided by the same filter of
 *           a constant 1 (normalised non-local means).
 * Keeps the blurred lattice in the handle for pam_filter_bwd.  Asynchronous.
 */
pam_status_t pam_filter_fwd(pam_lattice_t lat, const float *val, int32_t c, uint32_t flags,
                            float *out, void *stream);

/*
 * Backward filter for L with upstream gradient grad_out = dL/dv'.
 *   grad_val  = dL/dv, eq. 7: the same filter applied to grad_out with the
 *               blur directions in reverse order;  n x c fp32, or NULL to skip.
 *   grad_feat = dL/df, eq. 8: for point i, the blurred lattices of val
 *               (forward order) and grad_out (reverse order) read at its
 *               simplex vertices, contracted with grad_out_i and val_i, turned
 *               into a gradient of the elevated position through the
 *               permutation found by E, and mapped back by E^T; n x d fp32,
 *               or NULL to skip.  The simplex of each point is held fixed
 *               (one-sided at simplex boundaries).
 *   val, grad_out : n x c fp32 inputs; val must be the values of the last
 *               pam_filter_fwd call.
 *   flags : as for pam_filter_fwd, plus PAM_EGRAD_AUGMENTED (raw mode only;
 *           with PAM_NORMALIZE the call fails with PAM_ERR_INVALID_ARGUMENT):
 *           grad_feat is then the gradient of the exact Gaussian sum that
 *           the filter approximates (eq. 4-5), written with filters of the
 *           augmented channels f (x) val and f (x) grad_out, each filter
 *           replaced by the lattice one W = Sl B S / G_d (forward blur order)
 *           or its transpose (reverse order):
 *             dL/df_i = sum_c g_ic [W(f (x) v)_ic - f_i (W v)_ic]
 *                     + v_ic [W^T(f (x) g)_ic - f_i (W^T g)_ic],
 *           with g = grad_out, v = val.  It filters 2 d c extra channels
 *           and reads feat (the build's borrowed features).  grad_val is
 *           eq. 7 either way.  Scratch: three M x 4*ceil(d c / 4) fp32
 *           lattices, kept in the handle.
 * Requires a previous pam_filter_fwd on this build with the same c and the
 * same PAM_NORMALIZE bit (PAM_ERR_STATE otherwise).  Outputs must not overlap
 * inputs.  Asynchronous.
 */
pam_status_t pam_filter_bwd(pam_lattice_t lat, const float *val, const float *grad_out,
                            int32_t c, uint32_t flags, float *grad_val, float *grad_feat,
                            void *stream);

/*
 * Asymmetric filter (queries attend to keys; the paper's closing section
 * names asymmetric attention as future work):
 *   out_i = sum_j K(q_i, k_j) v_j,  K(a, b) = exp(-|a - b|^2 / 2),
 * approximated as s_d Sl_q(B(S_k(v))): the values are splatted at the key
 * embeddings only and sliced at the query embeddings only.  The lattice is
 * built by pam_lattice_build (or _groups) over the n points [keys; queries]:
 * points [0, n_keys) are the keys, points [n_keys, n) the queries, so the
 * vertex set holds the simplices of both and the blur reaches every vertex
 * a query reads.  With the queries equal to the keys this is the symmetric
 * filter.  Raw mode only (PAM_NORMALIZE and PAM_EGRAD_AUGMENTED:
 * PAM_ERR_INVALID_ARGUMENT).
 *   n_keys  : 0 <= n_keys <= n.
 *   val     : n_keys x c fp32 values of the keys (device).
 *   out     : (n - n_keys) x c fp32 (device), row i for query n_keys + i.
 * Keeps the blurred lattice for pam_filter_bwd_asym.  Asynchronous.
 */
pam_status_t pam_filter_fwd_asym(pam_lattice_t lat, int64_t n_keys, const float *val, int32_t c, uint32_t flags,
                                 float *out, void *stream);

/*
 * Backward pass of pam_filter_fwd_asym (eq. 7 and 8 with the splat at the
 * keys and the slice at the queries):
 *   grad_out  : (n - n_keys) x c fp32, dL/dout of the queries.
 *   grad_val  : n_keys x c fp32, dL/dv = s_d Sl_k(B~(S_q(grad_out))), or NULL.
 *   grad_feat : n x d fp32, or NULL: rows [0, n_keys) get the splat-side term
 *               of eq. 8 (<v_j, B~ S_q g> at the key's vertices), rows
 *               [n_keys, n) the slice-side term (<g_i, B S_k v> at the
 *               query's vertices).
 * Requires a previous pam_filter_fwd_asym on this build with the same n_keys
 * and c (PAM_ERR_STATE otherwise).  Outputs must not overlap inputs.
 * Asynchronous.
 */
pam_status_t pam_filter_bwd_asym(pam_lattice_t lat, int64_t n_keys, const float *val, const float *grad_out,
                                 int32_t c, uint32_t flags, float *grad_val, float *grad_feat, void *stream);

/*
 * Permutohedral block prologue (Section 3 and the Fig. 2 caption): the
 * feature extractor is a 1x1x1 convolution of the input channels with a
 * mesh of spatial coordinates appended, followed by a Leaky-ReLU; the
 * descriptor extractor is a 1x1x1 convolution of the input channels; both
 * are split channel-wise into `groups` and the module runs on each group
 * independently.  Outputs are written in the grouped layout that
 * pam_lattice_build_groups (group_start = {0, N, 2N, ...}) and the filter
 * calls take.
 *   x    : N x c_in fp32, voxel i = x + W (y + H z) (x fastest), N = W H D.
 *   wf   : d_tot x (c_in + 3) fp32, input columns: the c_in channels, then
 *          the mesh channels mesh_scale * (x, y, z); bf : d_tot fp32.
 *   wv   : c_tot x c_in fp32; bv : c_tot fp32.
 *   feat : (groups N) x (d_tot / groups): row g N + i holds
 *          LeakyReLU(wf [x_i; mesh_i] + bf) channels [g d_g, (g+1) d_g).
 *   val  : (groups N) x (c_tot / groups), likewise for wv x_i + bv.
 * Limits: 1 <= c_in <= 64; 1 <= groups <= 8 dividing d_tot and c_tot;
 * d_tot <= 32 with d_tot / groups <= PAM_MAX_D; c_tot <= 128; W, H, D >= 1
 * and N (d_tot + c_tot) < 2^31.  All pointers device, caller-owned;
 * asynchronous; argument errors leave outputs untouched.
 */
typedef struct {
    int32_t c_in;
    int32_t d_tot;
    int32_t c_tot;
    int32_t groups;
    int32_t dims[3]; /* W, H, D */
    float mesh_scale;
    float slope;     /* Leaky-ReLU slope for negative inputs */
} pam_block_desc_t;

pam_status_t pam_block_fwd(const pam_block_desc_t *desc, const float *x, const float *wf, const float *bf,
                           const float *wv, const float *bv, float *feat, float *val, void *stream);

/* Bytes of device workspace pam_block_bwd needs for `desc` (0 on invalid
 * arguments). */
size_t pam_block_bwd_workspace(const pam_block_desc_t *desc);

/*
 * Backward pass of pam_block_fwd for upstream gradients grad_feat, grad_val
 * in the grouped layout (what pam_filter_bwd's grad_feat / grad_val return
 * for a batched build over the block's groups).  Outputs (device,
 * caller-owned, each written in full): grad_x (N x c_in), grad_wf, grad_bf,
 * grad_wv, grad_bv (the weights' shapes).  The weight gradients are summed
 * over the voxels in a fixed order (deterministic).  workspace: device
 * buffer of pam_block_bwd_workspace(desc) bytes, owned by the caller and
 * overwritten.  Asynchronous.
 */
pam_status_t pam_block_bwd(const pam_block_desc_t *desc, const float *x, const float *wf, const float *bf,
                           const float *wv, const float *grad_feat, const float *grad_val, float *grad_x,
                           float *grad_wf, float *grad_bf, float *grad_wv, float *grad_bv, void *workspace,
                           void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * backward pass as pam_block_bwd without a workspace argument.  The
 * per-block partial weight gradients go to a fixed device array of 2^20
 * floats (4 MiB) that the library holds on each GPU it runs on until the
 * process ends; the call uses min(the usual block count, 2^20 / P) blocks,
 * P = d_tot (c_in + 4) + c_tot (c_in + 1) partial floats per block (every
 * descriptor within the limits above fits; a larger P is refused with
 * PAM_ERR_CAPACITY).  Allocates nothing (no hipMalloc, hipFree or
 * allocating library call).  All calls on one GPU share that array: calls
 * that overlap in time on one GPU (concurrent streams or threads) race and
 * must be serialised by the caller.  Results equal pam_block_bwd's up to
 * fp32 summation order (the block count may differ).  Other arguments,
 * outputs and errors as pam_block_bwd.
 */
pam_status_t pam_block_bwd_noalloc(const pam_block_desc_t *desc, const float *x, const float *wf, const float *bf,
                                   const float *wv, const float *grad_feat, const float *grad_val, float *grad_x,
                                   float *grad_wf, float *grad_bf, float *grad_wv, float *grad_bv, void *stream);

/* Vertex count M and hash-table capacity of the last build.  Either output
 * pointer (host) may be NULL.  Does not synchronise. */
pam_status_t pam_lattice_stats(pam_lattice_t lat, int64_t *num_vertices, int64_t *table_capacity);

/*
 * Copy the lattice to HOST buffers (for tests).  Synchronises.  Any pointer
 * may be NULL to skip it.
 *   keys : M x d int32, the d stored coordinates of every vertex (the last
 *          coordinate is minus their sum), in vertex-id order;
 *   vert : n x (d+1) int32, the vertex id of each point's simplex vertex k,
 *          where vertex k has every coordinate congruent to k mod d+1;
 *   bary : n x (d+1) fp32 barycentric weights, same order;
 *          vert and bary are copied from the per-point records the filter
 *          kernels read (in their sorted order), mapped back to the
 *          caller's point order;
 *   nbr  : M x (d+1) x 2 int32, for vertex m and direction j the ids of
 *          key_m - u_j and key_m + u_j (u_j = (d+1) e_j - 1), -1 if absent.
 * Vertex ids are implementation-defined (not ordered).
 */
pam_status_t pam_lattice_export(pam_lattice_t lat, int32_t *keys, int32_t *vert, float *bary,
                                int32_t *nbr);

/*
 * Group id of every vertex of a batched build, in id order (host array of
 * num_vertices int32; all 0 after pam_lattice_build).  Synchronises.
 */
pam_status_t pam_lattice_export_groups(pam_lattice_t lat, int32_t *vgroup);

/*
 * Sizing control for the next build (tests of the regrowth path and callers
 * who know their lattice size).  table_capacity > 0 sets the hash-table
 * capacity of the next build (rounded up to a power of two, at least 64);
 * 0 keeps the automatic sizing.  A build whose vertex count exceeds half
 * the capacity (or that fills the table) grows the table 4x and retries;
 * allow_regrow = 0 makes it fail with PAM_ERR_CAPACITY instead.
 */
pam_status_t pam_lattice_set_capacity(pam_lattice_t lat, int64_t table_capacity,
                                      int32_t allow_regrow);

/*
 * Per-kernel timing with HIP events recorded on the caller's stream around
 * every kernel launch of this handle.  enable = 1 starts (and clears) the
 * record, 0 stops it.  Recording adds event overhead between launches.
 */
pam_status_t pam_timing_enable(pam_lattice_t lat, int32_t enable);

/* Kernel kinds for pam_timing_read; pam_kernel_name gives their names. */
int32_t pam_kernel_count(void);
const char *pam_kernel_name(int32_t kind);

/*
 * Synchronise and return, for one kernel kind, the number of recorded
 * launches and their summed duration in milliseconds (host pointers).
 */
pam_status_t pam_timing_read(pam_lattice_t lat, int32_t kind, int64_t *launches,
                             double *total_ms);

/* Free the handle and its device buffers (synchronises its last stream).
 * NULL is ignored. */
void pam_lattice_destroy(pam_lattice_t lat);

const char *pam_status_string(pam_status_t s);
const char *pam_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PAM_LATTICE_H */

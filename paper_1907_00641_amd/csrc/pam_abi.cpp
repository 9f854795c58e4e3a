// C ABI of the permutohedral-lattice filter library: argument validation,
// handle and buffer management, launch sequencing and per-kernel timing.
// The kernels live in pam_build.hip and pam_filter.hip.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <initializer_list>
#include <string>
#include <vector>

#include "pam_device.h"

using namespace pam;

namespace {

thread_local std::string g_last_error;

// Logging to stderr, by the environment variable PAM_LOG_LEVEL (read once):
// 0 or unset = silent, 1 = one line per build and filter call, 2 = also
// every failure with its message.
int log_level()
{
    static const int level = [] {
        const char *v = getenv("PAM_LOG_LEVEL");
        return v ? atoi(v) : 0;
    }();
    return level;
}

// PAM_FUSE_EQ8 (read at every backward call): 1 = the backward splat forms
// eq. 8's slice-side term
bool fuse_eq8()
{
    const char *v = getenv("PAM_FUSE_EQ8");
    return v && atoi(v) != 0;
}

void log_line(int level, const char *fmt, ...)
{
    if (log_level() < level)
        return;
    va_list ap;
    va_start(ap, fmt);
    fputs("[pam] ", stderr);
    vfprintf(stderr, fmt, ap);
    fputc('\n', stderr);
    va_end(ap);
}

pam_status_t fail(pam_status_t s, const std::string &msg)
{
    g_last_error = msg;
    log_line(2, "error %d: %s", (int)s, msg.c_str());
    return s;
}

pam_status_t hip_fail(hipError_t e, const char *what)
{
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return e == hipErrorOutOfMemory ? PAM_ERR_OUT_OF_MEMORY : PAM_ERR_DEVICE;
}

#define PAM_HIP(call, what)                                                                       \
    do {                                                                                          \
        hipError_t e_ = (call);                                                                   \
        if (e_ != hipSuccess)                                                                     \
            return hip_fail(e_, what);                                                            \
    } while (0)

struct TimingRec {
    int32_t kind;
    hipEvent_t start, stop;
};

// Device buffer that only grows.
struct DevBuf {
    void *ptr = nullptr;
    size_t bytes = 0;
};

}  // namespace

struct pam_lattice_s {
    int device = 0;
    hipStream_t stream = nullptr;  // stream of the last call
    int32_t d = 0;
    int64_t n = 0;
    const float *feat = nullptr;
    Elev E{};
    bool built = false;

    Ctl *ctl = nullptr;       // device control block
    Ctl *ctl_host = nullptr;  // pinned host copy
    DevBuf tkeys, tids, vkeys, nbr, vert, lat[4];
    DevBuf aug[3];          // augmented-channel lattices of the embedding gradient
    DevBuf part;            // per-block quotient ranges of the range pass
    DevBuf gstart;          // group starts of a batched build (G + 1 int64)
    int32_t groups = 1;
    int32_t gbits = 0;
    DevBuf ntiles;          // tiles of consecutive points: key dedup of the insert
    DevBuf bucket, scan;    // points per vertex 0, then bucket starts; scan scratch
    DevBuf pos0;            // per point: position within its bucket
    DevBuf perm, pts, svert, tiles;  // the simplex-sorted order and its tile view
    DevBuf hA;              // backward splat's <g_p, A[m_pk]> per sorted point and vertex (raw mode)
    uint64_t cap = 0;         // hash-table capacity of the last build
    uint64_t clean_cap = 0;   // table emptied and control counters zeroed for this capacity (0: not known)
    int64_t M = 0;
    int64_t prev_M = -1;

    int64_t cap_request = 0;
    bool allow_regrow = true;

    // Lattice buffers known to hold zeros in their first zeroed[b] floats
    // (cleared by the build for the next filter calls, which then skip
    // their clearing launch); last_ld is the row stride of the last filter
    // call, the one the build clears for.
    int64_t zeroed[4] = {0, 0, 0, 0};
    int32_t last_ld = 0;

    bool fwd_valid = false;
    int32_t fwd_c = 0;
    uint32_t fwd_flags = 0;
    int fwd_A = 0;  // lattice buffer holding the forward's blurred lattice
    int64_t fwd_src = 0, fwd_tgt = 0;  // source count and first target of the forward call

    bool timing = false;
    std::vector<TimingRec> pending;
    std::vector<hipEvent_t> event_pool;
    double t_sum[kKNumKinds] = {};
    int64_t t_count[kKNumKinds] = {};
};

namespace {

struct DeviceGuard {
    int prev = -1;
    bool switched = false;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) {
            switched = hipSetDevice(dev) == hipSuccess;
        }
    }
    ~DeviceGuard()
    {
        if (switched)
            (void)hipSetDevice(prev);
    }
};

pam_status_t ensure(DevBuf &b, size_t bytes, const char *what)
{
    if (bytes <= b.bytes)
        return PAM_OK;
    if (b.ptr) {
        PAM_HIP(hipFree(b.ptr), what);
        b.ptr = nullptr;
        b.bytes = 0;
    }
    size_t alloc = std::max<size_t>(bytes, 256);
    hipError_t e = hipMalloc(&b.ptr, alloc);
    if (e != hipSuccess) {
        b.ptr = nullptr;
        return hip_fail(e, what);
    }
    b.bytes = alloc;
    return PAM_OK;
}

hipEvent_t take_event(pam_lattice_s *h)
{
    if (!h->event_pool.empty()) {
        hipEvent_t e = h->event_pool.back();
        h->event_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess)
        return nullptr;
    return e;
}

// Records HIP events around one launch when timing is enabled.
struct Timed {
    pam_lattice_s *h;
    int32_t kind;
    hipEvent_t a = nullptr, b = nullptr;
    Timed(pam_lattice_s *h_, int32_t kind_) : h(h_), kind(kind_)
    {
        if (h->timing) {
            a = take_event(h);
            b = take_event(h);
            if (a && b)
                (void)hipEventRecord(a, h->stream);
        }
    }
    ~Timed()
    {
        if (h->timing && a && b) {
            (void)hipEventRecord(b, h->stream);
            h->pending.push_back({kind, a, b});
        }
    }
};

#define PAM_LAUNCH(h, kind, call, what)                                                           \
    do {                                                                                          \
        hipError_t e_;                                                                            \
        {                                                                                         \
            Timed t_(h, kind);                                                                    \
            e_ = (call);                                                                          \
        }                                                                                         \
        if (e_ != hipSuccess)                                                                     \
            return hip_fail(e_, what);                                                            \
    } while (0)

void drain_timing(pam_lattice_s *h)
{
    for (auto &r : h->pending) {
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, r.start, r.stop) == hipSuccess) {
            h->t_sum[r.kind] += ms;
            h->t_count[r.kind] += 1;
        }
        h->event_pool.push_back(r.start);
        h->event_pool.push_back(r.stop);
    }
    h->pending.clear();
}

// fp32 entries of E = alpha Q: alpha = (d+1) sqrt(2/3); column j of Q has
// 1/sqrt((j+1)(j+2)) on rows 0..j and -(j+1)/sqrt((j+1)(j+2)) on row j+1.
Elev make_elev(int d)
{
    Elev E{};
    const double alpha = (double)(d + 1) * sqrt(2.0 / 3.0);
    for (int j = 0; j < d; ++j) {
        double nrm = sqrt((double)(j + 1) * (double)(j + 2));
        E.pos64[j] = alpha * (1.0 / nrm);
        E.neg64[j] = alpha * (-(double)(j + 1) / nrm);
        E.pos[j] = (float)E.pos64[j];
        E.neg[j] = (float)E.neg64[j];
    }
    E.inv = (float)(1.0 / (double)(d + 1));
    // 1/G_d, G_d = 4^{d+1} (3/(4 pi))^{d/2} / sqrt(d+1): lattice kernel mass
    // over the mass of exp(-|x|^2/2)
    double G = pow(4.0, d + 1) * pow(3.0 / (4.0 * M_PI), 0.5 * d) / sqrt((double)(d + 1));
    E.raw_scale = (float)(1.0 / G);
    return E;
}

uint64_t next_pow2(uint64_t v)
{
    uint64_t p = 1;
    while (p < v)
        p <<= 1;
    return p;
}

bool overlaps(const void *a, size_t abytes, const void *b, size_t bbytes)
{
    const char *pa = (const char *)a, *pb = (const char *)b;
    return pa < pb + bbytes && pb < pa + abytes;
}

pam_status_t check_sticky_error()
{
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return hip_fail(e, "earlier asynchronous work");
    return PAM_OK;
}

Groups64 groups_of(const pam_lattice_s *h)
{
    Groups64 g;
    g.gstart = h->groups > 1 ? (const int64_t *)h->gstart.ptr : nullptr;
    g.G = h->groups;
    return g;
}

// One insertion attempt at capacity h->cap.  Returns the device flags.
// allow_fixed: the keys may be packed with the fixed layout (no range pass)
// when the table is known empty at this capacity; a key that does not fit
// it sets kFlagLayoutMiss and the caller retries without.
pam_status_t insert_pass(pam_lattice_s *h, bool allow_fixed, uint32_t *flags_out)
{
    hipStream_t s = h->stream;
    pam_status_t st;
    const void *tk = h->tkeys.ptr;
    if ((st = ensure(h->tkeys, h->cap * sizeof(uint64_t), "hash table keys")) != PAM_OK)
        return st;
    if ((st = ensure(h->tids, h->cap * sizeof(int32_t), "hash table ids")) != PAM_OK)
        return st;
    KeyLayout fixed{};
    const bool fast = allow_fixed && h->clean_cap == h->cap && h->tkeys.ptr == tk &&
                      fixed_layout(h->d, h->gbits, &fixed);
    h->clean_cap = 0;  // the insert fills the table
    if (!fast) {
        if ((st = ensure(h->part, (size_t)kRangePartInts * sizeof(int32_t), "range partials")) != PAM_OK)
            return st;
        PAM_LAUNCH(h, kKRange,
                   launch_range(h->d, h->feat, h->n, h->E, (int32_t *)h->part.ptr, (uint64_t *)h->tkeys.ptr, h->cap,
                                s),
                   "range");
        PAM_LAUNCH(h, kKLayout, launch_layout(h->d, h->n, h->gbits, h->ctl, (const int32_t *)h->part.ptr, s),
                   "layout");
    }
    const TileRec rec(h->d);
    const int64_t ntiles = (h->n + rec.T - 1) / rec.T;
    if ((st = ensure(h->ntiles, (size_t)ntiles * rec.bytes, "per-tile key dedup")) != PAM_OK)
        return st;
    PAM_LAUNCH(h, kKInsert,
               launch_insert_tiles(h->d, h->feat, h->n, h->E, groups_of(h), h->ctl, fast ? &fixed : nullptr,
                                   (uint64_t *)h->tkeys.ptr, h->cap, (uint8_t *)h->ntiles.ptr, s),
               "insert");
    PAM_HIP(hipMemcpyAsync(h->ctl_host, h->ctl, sizeof(Ctl), hipMemcpyDeviceToHost, s), "readback");
    PAM_HIP(hipStreamSynchronize(s), "build synchronise");
    *flags_out = h->ctl_host->flags;
    // load factor above one half: regrow as for a full table
    if ((uint64_t)h->ctl_host->count > h->cap / 2)
        *flags_out |= kFlagTableFull;
    return PAM_OK;
}

}  // namespace

extern "C" {

const char *pam_status_string(pam_status_t s)
{
    switch (s) {
    case PAM_OK: return "ok";
    case PAM_ERR_INVALID_ARGUMENT: return "invalid argument";
    case PAM_ERR_OUT_OF_MEMORY: return "out of device memory";
    case PAM_ERR_CAPACITY: return "hash table capacity exceeded";
    case PAM_ERR_KEY_RANGE: return "feature out of the representable lattice key range";
    case PAM_ERR_STATE: return "no matching forward pass";
    case PAM_ERR_DEVICE: return "HIP device error";
    }
    return "unknown status";
}

const char *pam_last_error(void) { return g_last_error.c_str(); }

int32_t pam_kernel_count(void) { return kKNumKinds; }

const char *pam_kernel_name(int32_t kind) { return kernel_name(kind); }

static pam_status_t ensure_lattice_buffers(pam_lattice_s *h, int64_t elems);

static pam_status_t build_impl(const float *feat, int64_t n, int32_t d, const int64_t *group_start, int32_t groups,
                               void *stream, pam_lattice_t *lat)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    if (d < 1 || d > PAM_MAX_D)
        return fail(PAM_ERR_INVALID_ARGUMENT, "d must be in [1, 16]");
    if (n < 0 || n * (int64_t)(d + 1) >= ((int64_t)1 << 31))
        return fail(PAM_ERR_INVALID_ARGUMENT, "n must satisfy 0 <= n and n*(d+1) < 2^31");
    if (n > 0 && !feat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "feat is NULL");
    if (groups < 1 || groups > PAM_MAX_GROUPS)
        return fail(PAM_ERR_INVALID_ARGUMENT, "groups must be in [1, 65536]");
    if (tile_record_bytes_build(d) != TileRec(d).bytes || tile_record_bytes_filter(d) != TileRec(d).bytes)
        return fail(PAM_ERR_DEVICE, "library linked from objects built against different tile layouts");
    if (groups > 1) {
        if (!group_start)
            return fail(PAM_ERR_INVALID_ARGUMENT, "group_start is NULL");
        if (group_start[0] != 0 || group_start[groups] != n)
            return fail(PAM_ERR_INVALID_ARGUMENT, "group_start must run from 0 to n");
        for (int32_t g = 0; g < groups; ++g)
            if (group_start[g + 1] < group_start[g])
                return fail(PAM_ERR_INVALID_ARGUMENT, "group_start must be nondecreasing");
    }

    pam_lattice_s *h = *lat;
    bool created = false;
    if (!h) {
        h = new (std::nothrow) pam_lattice_s();
        if (!h)
            return fail(PAM_ERR_OUT_OF_MEMORY, "host allocation of the handle");
        if (hipGetDevice(&h->device) != hipSuccess) {
            delete h;
            return fail(PAM_ERR_DEVICE, "no HIP device");
        }
        hipError_t e = hipMalloc((void **)&h->ctl, sizeof(Ctl));
        if (e == hipSuccess)
            e = hipHostMalloc((void **)&h->ctl_host, sizeof(Ctl), hipHostMallocDefault);
        if (e != hipSuccess) {
            pam_status_t st = hip_fail(e, "control block");
            if (h->ctl)
                (void)hipFree(h->ctl);
            delete h;
            return st;
        }
        created = true;
    }
    DeviceGuard guard(h->device);
    if (!created) {
        pam_status_t st = check_sticky_error();
        if (st != PAM_OK)
            return st;
    }
    h->stream = (hipStream_t)stream;
    h->built = false;
    h->fwd_valid = false;
    h->d = d;
    h->n = n;
    h->feat = feat;
    h->E = make_elev(d);
    h->groups = groups;
    h->gbits = 0;
    while ((1 << h->gbits) < groups)
        ++h->gbits;
    if (created)
        *lat = h;
    if (n == 0) {
        h->M = 0;
        h->built = true;
        return PAM_OK;
    }

    pam_status_t st;
    if ((st = ensure(h->vert, (size_t)n * (d + 1) * sizeof(int32_t), "per-point vertex ids")) != PAM_OK)
        return st;
    if (groups > 1) {
        if ((st = ensure(h->gstart, (size_t)(groups + 1) * sizeof(int64_t), "group starts")) != PAM_OK)
            return st;
        PAM_HIP(hipMemcpyAsync(h->gstart.ptr, group_start, (size_t)(groups + 1) * sizeof(int64_t),
                               hipMemcpyHostToDevice, h->stream),
                "group starts upload");
    }

    if (h->cap_request > 0) {
        h->cap = next_pow2(std::max<int64_t>(h->cap_request, 64));
        h->cap_request = 0;
    } else if (h->prev_M >= 0) {
        h->cap = next_pow2(std::max<int64_t>(4 * h->prev_M, 1024));
    } else {
        int64_t guess = std::min<int64_t>(std::max<int64_t>(n * (d + 1) / 4, 1024), (int64_t)1 << 24);
        h->cap = next_pow2((uint64_t)guess);
    }

    bool allow_fixed = true;
    for (;;) {
        uint32_t flags = 0;
        if ((st = insert_pass(h, allow_fixed, &flags)) != PAM_OK)
            return st;
        if (flags & kFlagBadFeature)
            return fail(PAM_ERR_KEY_RANGE, "a feature is not finite or its elevation exceeds 2^24");
        if (flags & kFlagKeyRange)
            return fail(PAM_ERR_KEY_RANGE, "lattice keys need more than 63 bits");
        if (flags & kFlagLayoutMiss) {  // keys outside the fixed layout: lay them out from their range
            allow_fixed = false;
            continue;
        }
        if (!(flags & kFlagTableFull))
            break;
        if (!h->allow_regrow)
            return fail(PAM_ERR_CAPACITY, "hash table full (regrowth disabled)");
        if (h->cap >= ((uint64_t)1 << 34))
            return fail(PAM_ERR_CAPACITY, "hash table cannot grow further");
        h->cap *= 4;
    }

    const int64_t M = h->ctl_host->count;
    hipStream_t s = h->stream;
    const TileRec rec(d);
    const int64_t ntiles = (n + rec.T - 1) / rec.T;
    const size_t M1 = (size_t)std::max<int64_t>(M, 1);
    if ((st = ensure(h->vkeys, M1 * sizeof(uint64_t), "vertex keys")) != PAM_OK ||
        (st = ensure(h->nbr, M1 * (d + 1) * 2 * sizeof(int32_t), "neighbour table")) != PAM_OK ||
        (st = ensure(h->bucket, M1 * sizeof(int32_t), "vertex-0 buckets")) != PAM_OK ||
        (st = ensure(h->scan, (size_t)scan_scratch_ints(M) * sizeof(int32_t), "scan scratch")) != PAM_OK ||
        (st = ensure(h->pos0, (size_t)n * sizeof(int32_t), "bucket positions")) != PAM_OK ||
        (st = ensure(h->perm, (size_t)n * sizeof(int32_t), "sorted order")) != PAM_OK ||
        (st = ensure(h->pts, (size_t)n * point_bytes(d), "sorted point records")) != PAM_OK ||
        (st = ensure(h->svert, (size_t)n * (d + 1) * sizeof(int32_t), "sorted vertex ids")) != PAM_OK ||
        (st = ensure(h->tiles, (size_t)ntiles * rec.bytes, "per-tile lattice view")) != PAM_OK)
        return st;
    PAM_LAUNCH(h, kKCompact,
               launch_compact((const uint64_t *)h->tkeys.ptr, (int32_t *)h->tids.ptr,
                              (uint64_t *)h->vkeys.ptr, (int32_t *)h->bucket.ptr, h->cap, h->ctl, s),
               "compact");
    PAM_LAUNCH(h, kKResolve,
               launch_resolve(d, feat, n, h->E, groups_of(h), h->ctl, (const uint64_t *)h->tkeys.ptr,
                              (const int32_t *)h->tids.ptr,
                              h->cap, (uint8_t *)h->ntiles.ptr, (int32_t *)h->vert.ptr,
                              (int32_t *)h->bucket.ptr, (int32_t *)h->pos0.ptr, (const uint64_t *)h->vkeys.ptr, M,
                              (int32_t *)h->nbr.ptr, s),
               "resolve");
    PAM_LAUNCH(h, kKScan, launch_exclusive_scan((int32_t *)h->bucket.ptr, M, (int32_t *)h->scan.ptr, s), "scan");
    PAM_LAUNCH(h, kKScatter,
               launch_scatter(d, feat, n, h->E, (const uint8_t *)h->ntiles.ptr, (const int32_t *)h->vert.ptr,
                              (const int32_t *)h->bucket.ptr, (const int32_t *)h->pos0.ptr, (int32_t *)h->perm.ptr,
                              (uint8_t *)h->pts.ptr, (int32_t *)h->svert.ptr, s),
               "scatter");
    // the tiles launch also clears the splat targets of the next forward
    // and backward calls (buffers 0 and 2) for the last row stride used
    int64_t zelems = 0;
    h->zeroed[0] = h->zeroed[2] = 0;
    if (h->last_ld > 0) {
        zelems = M * h->last_ld;
        if ((st = ensure_lattice_buffers(h, zelems)) != PAM_OK)
            return st;
    }
    PAM_LAUNCH(h, kKTiles,
               launch_sorted_tiles(d, (const int32_t *)h->svert.ptr, n, (uint8_t *)h->tiles.ptr,
                                   (float *)h->lat[0].ptr, (float *)h->lat[2].ptr, zelems, (uint64_t *)h->tkeys.ptr,
                                   h->cap, h->ctl, s),
               "tiles");
    h->zeroed[0] = h->zeroed[2] = zelems;
    h->clean_cap = h->cap;  // the tiles launch emptied the table for the next build
    h->M = M;
    h->prev_M = M;
    h->built = true;
    log_line(1, "build n=%lld d=%d groups=%d M=%lld table=%llu", (long long)n, d, h->groups, (long long)M,
             (unsigned long long)h->cap);
    return PAM_OK;
}

pam_status_t pam_lattice_build(const float *feat, int64_t n, int32_t d, void *stream, pam_lattice_t *lat)
{
    return build_impl(feat, n, d, nullptr, 1, stream, lat);
}

pam_status_t pam_lattice_build_groups(const float *feat, int64_t n, int32_t d, const int64_t *group_start,
                                      int32_t groups, void *stream, pam_lattice_t *lat)
{
    return build_impl(feat, n, d, group_start, groups, stream, lat);
}

static pam_status_t check_filter_args(pam_lattice_s *h, const float *val, int32_t c, uint32_t flags,
                                      uint32_t allowed = PAM_NORMALIZE)
{
    if (!h)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    if (!h->built)
        return fail(PAM_ERR_STATE, "lattice not built");
    if (c < 1 || c > PAM_MAX_C)
        return fail(PAM_ERR_INVALID_ARGUMENT, "c must be in [1, 1024]");
    if (flags & ~allowed)
        return fail(PAM_ERR_INVALID_ARGUMENT, "unknown flag bits");
    if ((flags & PAM_EGRAD_AUGMENTED) && (flags & PAM_NORMALIZE))
        return fail(PAM_ERR_INVALID_ARGUMENT, "PAM_EGRAD_AUGMENTED needs raw mode (no PAM_NORMALIZE)");
    (void)val;  // the callers check the arrays against their row counts
    return PAM_OK;
}

static pam_status_t ensure_lattice_buffers(pam_lattice_s *h, int64_t elems)
{
    for (int b = 0; b < 4; ++b) {
        void *before = h->lat[b].ptr;
        pam_status_t st = ensure(h->lat[b], (size_t)std::max<int64_t>(elems, 1) * sizeof(float), "lattice buffer");
        if (h->lat[b].ptr != before)
            h->zeroed[b] = 0;  // a new allocation holds no known zeros
        if (st != PAM_OK)
            return st;
    }
    return PAM_OK;
}

// Lattice row stride for c channels (plus the weight column when
// normalised), padded to 4 floats so rows can be read as float4.
static int32_t lattice_ld(int32_t c, uint32_t flags)
{
    int32_t w = c + ((flags & PAM_NORMALIZE) ? 1 : 0);
    return (w + 3) & ~3;
}

// rows: the n x c arrays of the call; float4 access needs c % 4 == 0 and
// 16-byte aligned rows.
static FilterArgs filter_args(pam_lattice_s *h, int32_t c, uint32_t flags,
                              std::initializer_list<const void *> rows)
{
    FilterArgs a{};
    a.pts = (const uint8_t *)h->pts.ptr;
    a.svert = (const int32_t *)h->svert.ptr;
    a.perm = (const int32_t *)h->perm.ptr;
    a.n = h->n;
    a.c = c;
    a.normalize = (flags & PAM_NORMALIZE) ? 1 : 0;
    a.ld = lattice_ld(c, flags);
    bool v4 = (c % 4) == 0;
    for (const void *p : rows)
        v4 = v4 && (((uintptr_t)p) % 16 == 0);
    a.vec = v4 ? 4 : 1;
    a.feat = h->feat;
    a.src_n = h->n;
    a.tgt_0 = 0;
    a.side = 0;
    a.E = h->E;
    return a;
}

// d+1 blur passes from buffer `src`, directions ascending (forward, B) or
// descending (backward, the reversed blur); returns the buffer index holding
// the result.  While the lattice is cache-sized, directions are fused in
// pairs (one launch per pair, same result as separate passes).
constexpr int64_t kBlurFuseBytes = (int64_t)32 << 20;

static pam_status_t blur_all(pam_lattice_s *h, DevBuf *buf, int src, int other, int32_t ld, bool reverse,
                             int *result)
{
    const int d = h->d;
    const int64_t M = h->M;
    const bool fuse = M * ld * (int64_t)sizeof(float) <= kBlurFuseBytes;
    auto nbr = [&](int t) {
        const int j = reverse ? d - t : t;
        return (const int32_t *)h->nbr.ptr + (int64_t)j * M * 2;
    };
    int cur = src, nxt = other;
    for (int t = 0; t <= d;) {
        if (fuse && t + 1 <= d) {
            PAM_LAUNCH(h, kKBlur,
                       launch_blur2((const float *)buf[cur].ptr, (float *)buf[nxt].ptr, nbr(t), nbr(t + 1), M, ld,
                                    h->stream),
                       "blur");
            t += 2;
        } else {
            PAM_LAUNCH(h, kKBlur,
                       launch_blur((const float *)buf[cur].ptr, (float *)buf[nxt].ptr, nbr(t), M, ld, h->stream),
                       "blur");
            t += 1;
        }
        std::swap(cur, nxt);
    }
    *result = cur;
    return PAM_OK;
}

// Forward filter with sources [0, src_n) (rows of val) and targets
// [tgt_0, n) (rows of out); the symmetric call has src_n = n, tgt_0 = 0.
static pam_status_t filter_fwd(pam_lattice_s *h, int64_t src_n, int64_t tgt_0, const float *val, int32_t c,
                               uint32_t flags, float *out, void *stream)
{
    pam_status_t st = check_filter_args(h, val, c, flags);
    if (st != PAM_OK)
        return st;
    const int64_t nv = src_n, no = h->n - tgt_0;
    if (nv > 0 && !val)
        return fail(PAM_ERR_INVALID_ARGUMENT, "val is NULL");
    if (no > 0 && !out)
        return fail(PAM_ERR_INVALID_ARGUMENT, "out is NULL");
    if (nv > 0 && no > 0 && overlaps(val, (size_t)nv * c * sizeof(float), out, (size_t)no * c * sizeof(float)))
        return fail(PAM_ERR_INVALID_ARGUMENT, "out overlaps val");
    DeviceGuard guard(h->device);
    if ((st = check_sticky_error()) != PAM_OK)
        return st;
    h->stream = (hipStream_t)stream;
    h->fwd_valid = false;
    if (h->n == 0 || no == 0) {
        h->fwd_valid = true;
        h->fwd_c = c;
        h->fwd_flags = flags;
        h->fwd_src = src_n;
        h->fwd_tgt = tgt_0;
        h->fwd_A = -1;  // nothing filtered
        return PAM_OK;
    }
    FilterArgs a = filter_args(h, c, flags, {val, out});
    a.src_n = src_n;
    a.tgt_0 = tgt_0;
    a.side = 0;
    const int64_t elems = h->M * a.ld;
    if ((st = ensure_lattice_buffers(h, elems)) != PAM_OK)
        return st;
    if (h->zeroed[0] < elems)
        PAM_LAUNCH(h, kKFill, launch_fill_f32((float *)h->lat[0].ptr, 0.0f, elems, h->stream), "lattice clear");
    h->zeroed[0] = h->zeroed[1] = 0;  // the splat and the blur write them
    h->last_ld = a.ld;
    if (nv > 0)
        PAM_LAUNCH(h, kKSplat,
                   launch_splat(h->d, a, (const uint8_t *)h->tiles.ptr, val, nullptr, kSplatModePlain,
                                (float *)h->lat[0].ptr, nullptr, h->stream),
                   "splat");
    int A = 0;
    if ((st = blur_all(h, h->lat, 0, 1, a.ld, false, &A)) != PAM_OK)
        return st;
    PAM_LAUNCH(h, kKSlice,
               launch_slice(h->d, a, (const uint8_t *)h->tiles.ptr, (const float *)h->lat[A].ptr, out, h->stream),
               "slice");
    h->fwd_valid = true;
    h->fwd_c = c;
    h->fwd_flags = flags;
    h->fwd_src = src_n;
    h->fwd_tgt = tgt_0;
    h->fwd_A = A;
    log_line(1, "fwd n=%lld c=%d flags=%u sources=%lld targets=%lld", (long long)h->n, c, flags, (long long)src_n,
             (long long)(h->n - tgt_0));
    return PAM_OK;
}

pam_status_t pam_filter_fwd(pam_lattice_t lat, const float *val, int32_t c, uint32_t flags, float *out,
                            void *stream)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    return filter_fwd(lat, lat->n, 0, val, c, flags, out, stream);
}

pam_status_t pam_filter_fwd_asym(pam_lattice_t lat, int64_t n_keys, const float *val, int32_t c, uint32_t flags,
                                 float *out, void *stream)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    if (flags & PAM_NORMALIZE)
        return fail(PAM_ERR_INVALID_ARGUMENT, "the asymmetric filter is raw mode only");
    if (lat->built && (n_keys < 0 || n_keys > lat->n))
        return fail(PAM_ERR_INVALID_ARGUMENT, "n_keys must be in [0, n]");
    return filter_fwd(lat, n_keys, n_keys, val, c, flags, out, stream);
}

static pam_status_t filter_bwd(pam_lattice_s *h, int64_t src_n, int64_t tgt_0, const float *val,
                               const float *grad_out, int32_t c, uint32_t flags, float *grad_val, float *grad_feat,
                               void *stream)
{
    pam_status_t st = check_filter_args(h, val, c, flags, PAM_NORMALIZE | PAM_EGRAD_AUGMENTED);
    if (st != PAM_OK)
        return st;
    const int64_t nv = src_n, no = h->n - tgt_0;
    if (nv > 0 && !val)
        return fail(PAM_ERR_INVALID_ARGUMENT, "val is NULL");
    if (no > 0 && !grad_out)
        return fail(PAM_ERR_INVALID_ARGUMENT, "grad_out is NULL");
    const bool aug = (flags & PAM_EGRAD_AUGMENTED) != 0;
    const bool asym = src_n != h->n || tgt_0 != 0;
    if (aug && asym)
        return fail(PAM_ERR_INVALID_ARGUMENT, "PAM_EGRAD_AUGMENTED is not available for the asymmetric filter");
    flags &= PAM_NORMALIZE;
    if (!h->fwd_valid || h->fwd_c != c || h->fwd_flags != flags || h->fwd_src != src_n || h->fwd_tgt != tgt_0)
        return fail(PAM_ERR_STATE, "pam_filter_bwd needs a pam_filter_fwd with the same c, flags and points");
    const size_t vbytes = (size_t)nv * c * sizeof(float), gbytes = (size_t)no * c * sizeof(float);
    const size_t fbytes = (size_t)h->n * h->d * sizeof(float);
    if (h->n > 0) {
        if (grad_val && nv > 0 && (overlaps(grad_val, vbytes, val, vbytes) || overlaps(grad_val, vbytes, grad_out, gbytes)))
            return fail(PAM_ERR_INVALID_ARGUMENT, "grad_val overlaps an input");
        if (grad_feat && (overlaps(grad_feat, fbytes, val, vbytes) ||
                          overlaps(grad_feat, fbytes, grad_out, gbytes) ||
                          overlaps(grad_feat, fbytes, h->feat, fbytes) ||
                          (grad_val && overlaps(grad_feat, fbytes, grad_val, vbytes))))
            return fail(PAM_ERR_INVALID_ARGUMENT, "grad_feat overlaps another array");
    }
    DeviceGuard guard(h->device);
    if ((st = check_sticky_error()) != PAM_OK)
        return st;
    h->stream = (hipStream_t)stream;
    if (h->n == 0 || (!grad_val && !grad_feat))
        return PAM_OK;
    if (nv == 0 || no == 0) {  // no source reaches a target: both gradients vanish
        if (grad_val && nv > 0)
            PAM_LAUNCH(h, kKFill, launch_fill_f32(grad_val, 0.0f, nv * c, h->stream), "gradient clear");
        if (grad_feat)
            PAM_LAUNCH(h, kKFill, launch_fill_f32(grad_feat, 0.0f, h->n * h->d, h->stream), "gradient clear");
        return PAM_OK;
    }
    FilterArgs a = filter_args(h, c, flags, {val, grad_out, grad_val});
    a.src_n = src_n;
    a.tgt_0 = tgt_0;
    a.side = 1;  // the backward splat takes the rows of grad_out
    const int64_t elems = h->M * a.ld;
    const int b0 = 2, b1 = 3;
    const float *A = (const float *)h->lat[h->fwd_A].ptr;
    // normalised: the backward splat takes g / z (and b * gamma in the
    // weight column, which only the embedding gradient reads)
    const bool norm_bwd = a.normalize != 0;
    if (h->zeroed[b0] < elems)
        PAM_LAUNCH(h, kKFill, launch_fill_f32((float *)h->lat[b0].ptr, 0.0f, elems, h->stream), "lattice clear");
    h->zeroed[b0] = h->zeroed[b1] = 0;  // the splat and the blur write them
    float *eq8_feat = aug ? nullptr : grad_feat;
    // PAM_FUSE_EQ8=1 in the environment (raw mode, float4 rows of at most
    // 32 channels): the splat of grad_out also forms eq. 8's <g, A_k>, so
    // that the backward slice does not re-read grad_out.  Off by default:
    // the splat then holds two blocks per CU instead of three and the step
    // is slower overall.
    float *hA = nullptr;
    if (eq8_feat && fuse_eq8() && splat_forms_eq8_term(a)) {
        if ((st = ensure(h->hA, (size_t)h->n * (h->d + 1) * sizeof(float), "eq. 8 splat term")) != PAM_OK)
            return st;
        hA = (float *)h->hA.ptr;
    }
    PAM_LAUNCH(h, kKSplatBwd,
               launch_splat(h->d, a, (const uint8_t *)h->tiles.ptr, grad_out, A,
                            norm_bwd ? kSplatModeNormBwd : kSplatModePlain, (float *)h->lat[b0].ptr, hA, h->stream),
               "splat_bwd");
    int At = b0;
    if ((st = blur_all(h, h->lat, b0, b1, a.ld, true, &At)) != PAM_OK)
        return st;
    if (grad_val || eq8_feat)
        PAM_LAUNCH(h, kKSliceBwd,
                   launch_slice_bwd(h->d, a, (const uint8_t *)h->tiles.ptr, val, grad_out, A,
                                    (const float *)h->lat[At].ptr, hA, grad_val, eq8_feat, h->stream),
                   "slice_bwd");
    log_line(1, "bwd n=%lld c=%d flags=%u%s grad_val=%s grad_feat=%s", (long long)h->n, c, flags,
             aug ? " augmented" : "", grad_val ? "yes" : "no", grad_feat ? "yes" : "no");
    if (!aug || !grad_feat)
        return PAM_OK;
    // augmented channels f (x) val (forward blur order) and f (x) grad_out
    // (reverse order), then the gradient from all four lattices
    FilterArgs q = a;
    q.side = 0;
    q.ld = (int32_t)(((int64_t)h->d * c + 3) & ~(int64_t)3);
    const int64_t qelems = h->M * q.ld;
    for (int b = 0; b < 3; ++b)
        if ((st = ensure(h->aug[b], (size_t)std::max<int64_t>(qelems, 1) * sizeof(float), "augmented lattice")) !=
            PAM_OK)
            return st;
    PAM_LAUNCH(h, kKFill, launch_fill_f32((float *)h->aug[0].ptr, 0.0f, qelems, h->stream), "lattice clear");
    PAM_LAUNCH(h, kKSplatAug,
               launch_splat(h->d, q, (const uint8_t *)h->tiles.ptr, val, nullptr, kSplatModeAug,
                            (float *)h->aug[0].ptr, nullptr, h->stream),
               "splat_aug");
    int L1 = 0;
    if ((st = blur_all(h, h->aug, 0, 1, q.ld, false, &L1)) != PAM_OK)
        return st;
    PAM_LAUNCH(h, kKFill, launch_fill_f32((float *)h->aug[2].ptr, 0.0f, qelems, h->stream), "lattice clear");
    PAM_LAUNCH(h, kKSplatAug,
               launch_splat(h->d, q, (const uint8_t *)h->tiles.ptr, grad_out, nullptr, kSplatModeAug,
                            (float *)h->aug[2].ptr, nullptr, h->stream),
               "splat_aug");
    int L2 = 2;
    if ((st = blur_all(h, h->aug, 2, 1 - L1, q.ld, true, &L2)) != PAM_OK)
        return st;
    PAM_LAUNCH(h, kKSliceAug,
               launch_slice_aug(h->d, a, (const uint8_t *)h->tiles.ptr, val, grad_out, A, (const float *)h->lat[At].ptr,
                                (const float *)h->aug[L1].ptr, (const float *)h->aug[L2].ptr, q.ld, grad_feat,
                                h->stream),
               "slice_aug");
    return PAM_OK;
}

pam_status_t pam_filter_bwd(pam_lattice_t lat, const float *val, const float *grad_out, int32_t c,
                            uint32_t flags, float *grad_val, float *grad_feat, void *stream)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    return filter_bwd(lat, lat->n, 0, val, grad_out, c, flags, grad_val, grad_feat, stream);
}

pam_status_t pam_filter_bwd_asym(pam_lattice_t lat, int64_t n_keys, const float *val, const float *grad_out,
                                 int32_t c, uint32_t flags, float *grad_val, float *grad_feat, void *stream)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    if (flags & PAM_NORMALIZE)
        return fail(PAM_ERR_INVALID_ARGUMENT, "the asymmetric filter is raw mode only");
    if (lat->built && (n_keys < 0 || n_keys > lat->n))
        return fail(PAM_ERR_INVALID_ARGUMENT, "n_keys must be in [0, n]");
    return filter_bwd(lat, n_keys, n_keys, val, grad_out, c, flags, grad_val, grad_feat, stream);
}

// ---- permutohedral block prologue

static pam_status_t check_block(const pam_block_desc_t *ds)
{
    if (!ds)
        return fail(PAM_ERR_INVALID_ARGUMENT, "desc is NULL");
    if (ds->c_in < 1 || ds->c_in > 64)
        return fail(PAM_ERR_INVALID_ARGUMENT, "c_in must be in [1, 64]");
    if (ds->groups < 1 || ds->groups > 8 || ds->d_tot < ds->groups || ds->c_tot < ds->groups ||
        ds->d_tot % ds->groups || ds->c_tot % ds->groups)
        return fail(PAM_ERR_INVALID_ARGUMENT, "groups must be in [1, 8] and divide d_tot and c_tot");
    if (ds->d_tot > 32 || ds->d_tot / ds->groups > PAM_MAX_D || ds->c_tot > 128)
        return fail(PAM_ERR_INVALID_ARGUMENT, "d_tot <= 32, d_tot / groups <= 16 and c_tot <= 128 required");
    if (ds->dims[0] < 1 || ds->dims[1] < 1 || ds->dims[2] < 1)
        return fail(PAM_ERR_INVALID_ARGUMENT, "dims must be positive");
    const int64_t n = (int64_t)ds->dims[0] * ds->dims[1] * ds->dims[2];
    if (n * (ds->d_tot + ds->c_tot + ds->c_in) >= ((int64_t)1 << 31))
        return fail(PAM_ERR_INVALID_ARGUMENT, "volume too large");
    return PAM_OK;
}

pam_status_t pam_block_fwd(const pam_block_desc_t *desc, const float *x, const float *wf, const float *bf,
                           const float *wv, const float *bv, float *feat, float *val, void *stream)
{
    pam_status_t st = check_block(desc);
    if (st != PAM_OK)
        return st;
    if (!x || !wf || !bf || !wv || !bv || !feat || !val)
        return fail(PAM_ERR_INVALID_ARGUMENT, "a pointer is NULL");
    const int64_t n = (int64_t)desc->dims[0] * desc->dims[1] * desc->dims[2];
    const size_t xb = (size_t)n * desc->c_in * 4, fb = (size_t)n * desc->d_tot * 4, vb = (size_t)n * desc->c_tot * 4;
    if (overlaps(feat, fb, val, vb) || overlaps(feat, fb, x, xb) || overlaps(val, vb, x, xb))
        return fail(PAM_ERR_INVALID_ARGUMENT, "outputs overlap");
    if ((st = check_sticky_error()) != PAM_OK)
        return st;
    PAM_HIP(launch_block_fwd(*desc, x, wf, bf, wv, bv, feat, val, (hipStream_t)stream), "block forward");
    return PAM_OK;
}

size_t pam_block_bwd_workspace(const pam_block_desc_t *desc)
{
    if (check_block(desc) != PAM_OK)
        return 0;
    return (size_t)block_bwd_blocks(*desc) * block_partials(*desc) * sizeof(float);
}

pam_status_t pam_block_bwd(const pam_block_desc_t *desc, const float *x, const float *wf, const float *bf,
                           const float *wv, const float *grad_feat, const float *grad_val, float *grad_x,
                           float *grad_wf, float *grad_bf, float *grad_wv, float *grad_bv, void *workspace,
                           void *stream)
{
    pam_status_t st = check_block(desc);
    if (st != PAM_OK)
        return st;
    if (!x || !wf || !bf || !wv || !grad_feat || !grad_val || !grad_x || !grad_wf || !grad_bf || !grad_wv ||
        !grad_bv || !workspace)
        return fail(PAM_ERR_INVALID_ARGUMENT, "a pointer is NULL");
    const int64_t n = (int64_t)desc->dims[0] * desc->dims[1] * desc->dims[2];
    const size_t xb = (size_t)n * desc->c_in * 4, fb = (size_t)n * desc->d_tot * 4, vb = (size_t)n * desc->c_tot * 4;
    if (overlaps(grad_x, xb, x, xb) || overlaps(grad_x, xb, grad_feat, fb) || overlaps(grad_x, xb, grad_val, vb))
        return fail(PAM_ERR_INVALID_ARGUMENT, "grad_x overlaps an input");
    if ((st = check_sticky_error()) != PAM_OK)
        return st;
    PAM_HIP(launch_block_bwd(*desc, x, wf, bf, wv, grad_feat, grad_val, grad_x, grad_wf, grad_bf, grad_wv, grad_bv,
                             (float *)workspace, (hipStream_t)stream),
            "block backward");
    return PAM_OK;
}

pam_status_t pam_block_bwd_noalloc(const pam_block_desc_t *desc, const float *x, const float *wf, const float *bf,
                                   const float *wv, const float *grad_feat, const float *grad_val, float *grad_x,
                                   float *grad_wf, float *grad_bf, float *grad_wv, float *grad_bv, void *stream)
{
    pam_status_t st = check_block(desc);
    if (st != PAM_OK)
        return st;
    if (!x || !wf || !bf || !wv || !grad_feat || !grad_val || !grad_x || !grad_wf || !grad_bf || !grad_wv ||
        !grad_bv)
        return fail(PAM_ERR_INVALID_ARGUMENT, "a pointer is NULL");
    const int64_t n = (int64_t)desc->dims[0] * desc->dims[1] * desc->dims[2];
    const size_t xb = (size_t)n * desc->c_in * 4, fb = (size_t)n * desc->d_tot * 4, vb = (size_t)n * desc->c_tot * 4;
    if (overlaps(grad_x, xb, x, xb) || overlaps(grad_x, xb, grad_feat, fb) || overlaps(grad_x, xb, grad_val, vb))
        return fail(PAM_ERR_INVALID_ARGUMENT, "grad_x overlaps an input");
    // one row of partials per block: as many blocks as the fixed array holds
    const size_t per_block = block_partials(*desc);
    if (per_block > kBlockScratchFloats)
        return fail(PAM_ERR_CAPACITY, "the weight gradients exceed the fixed scratch array (2^20 floats per block)");
    if ((st = check_sticky_error()) != PAM_OK)
        return st;
    float *part = nullptr;
    PAM_HIP(block_scratch(&part), "scratch address");
    const int nb = (int)std::min<size_t>(kBlockScratchFloats / per_block, (size_t)block_bwd_blocks(*desc));
    PAM_HIP(launch_block_bwd(*desc, x, wf, bf, wv, grad_feat, grad_val, grad_x, grad_wf, grad_bf, grad_wv, grad_bv,
                             part, (hipStream_t)stream, nb),
            "block backward");
    return PAM_OK;
}

pam_status_t pam_probe_copy_rows(const float *src, float *dst, const int32_t *perm, int64_t n,
                                 int32_t row_floats, int32_t mode, void *stream)
{
    if (n < 0 || row_floats <= 0 || row_floats % 4 != 0 || mode < 0 || mode > 3)
        return fail(PAM_ERR_INVALID_ARGUMENT, "n >= 0, row_floats a positive multiple of 4, mode in [0, 3]");
    if (n > 0 && (!src || !dst || (mode && !perm)))
        return fail(PAM_ERR_INVALID_ARGUMENT, "NULL pointer");
    if (((uintptr_t)src | (uintptr_t)dst) % 16 != 0)
        return fail(PAM_ERR_INVALID_ARGUMENT, "src and dst must be 16-byte aligned");
    if (n > 0 && overlaps(src, (size_t)n * row_floats * sizeof(float), dst, (size_t)n * row_floats * sizeof(float)))
        return fail(PAM_ERR_INVALID_ARGUMENT, "src and dst overlap");
    pam_status_t st = check_sticky_error();
    if (st != PAM_OK)
        return st;
    PAM_HIP(launch_copy_rows(src, dst, perm, n, row_floats, mode, (hipStream_t)stream), "probe copy");
    return PAM_OK;
}

pam_status_t pam_lattice_stats(pam_lattice_t lat, int64_t *num_vertices, int64_t *table_capacity)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    if (!lat->built)
        return fail(PAM_ERR_STATE, "lattice not built");
    if (num_vertices)
        *num_vertices = lat->M;
    if (table_capacity)
        *table_capacity = (int64_t)lat->cap;
    return PAM_OK;
}

pam_status_t pam_lattice_export(pam_lattice_t lat, int32_t *keys, int32_t *vert, float *bary, int32_t *nbr)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    pam_lattice_s *h = lat;
    if (!h->built)
        return fail(PAM_ERR_STATE, "lattice not built");
    DeviceGuard guard(h->device);
    hipStream_t s = h->stream;
    const int d = h->d;
    const int64_t M = h->M, n = h->n;
    PAM_HIP(hipStreamSynchronize(s), "export synchronise");
    if (keys && M > 0) {
        int32_t *tmp = nullptr;
        PAM_HIP(hipMalloc((void **)&tmp, (size_t)M * d * sizeof(int32_t)), "export keys");
        hipError_t e = launch_unpack_keys(d, (const uint64_t *)h->vkeys.ptr, M, h->ctl, tmp, s);
        if (e == hipSuccess)
            e = hipMemcpyAsync(keys, tmp, (size_t)M * d * sizeof(int32_t), hipMemcpyDeviceToHost, s);
        if (e == hipSuccess)
            e = hipStreamSynchronize(s);
        (void)hipFree(tmp);
        if (e != hipSuccess)
            return hip_fail(e, "export keys");
    }
    if ((vert || bary) && n > 0) {
        // from the sorted per-point records the filter kernels read
        const size_t ib = (size_t)n * (d + 1) * sizeof(int32_t), fb = (size_t)n * (d + 1) * sizeof(float);
        void *tmp = nullptr;
        PAM_HIP(hipMalloc(&tmp, ib + fb), "export points");
        int32_t *tv = (int32_t *)tmp;
        float *tb = (float *)((char *)tmp + ib);
        hipError_t e = launch_export_points(d, (const uint8_t *)h->pts.ptr, (const int32_t *)h->svert.ptr,
                                            (const int32_t *)h->perm.ptr, n, tv, tb, s);
        if (e == hipSuccess && vert)
            e = hipMemcpyAsync(vert, tv, ib, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess && bary)
            e = hipMemcpyAsync(bary, tb, fb, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess)
            e = hipStreamSynchronize(s);
        (void)hipFree(tmp);
        if (e != hipSuccess)
            return hip_fail(e, "export points");
    }
    if (nbr && M > 0) {
        std::vector<int32_t> dm((size_t)M * (d + 1) * 2);
        PAM_HIP(hipMemcpy(dm.data(), h->nbr.ptr, dm.size() * sizeof(int32_t), hipMemcpyDeviceToHost),
                "export nbr");
        for (int64_t m = 0; m < M; ++m)
            for (int j = 0; j <= d; ++j)
                for (int sg = 0; sg < 2; ++sg)
                    nbr[(m * (d + 1) + j) * 2 + sg] = dm[((size_t)j * M + m) * 2 + sg];
    }
    return PAM_OK;
}

pam_status_t pam_lattice_export_groups(pam_lattice_t lat, int32_t *vgroup)
{
    if (!lat || !vgroup)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat or vgroup is NULL");
    pam_lattice_s *h = lat;
    if (!h->built)
        return fail(PAM_ERR_STATE, "lattice not built");
    if (h->M == 0)
        return PAM_OK;
    DeviceGuard guard(h->device);
    hipStream_t s = h->stream;
    int32_t *tmp = nullptr;
    PAM_HIP(hipMalloc((void **)&tmp, (size_t)h->M * sizeof(int32_t)), "export groups");
    hipError_t e = launch_vertex_groups((const uint64_t *)h->vkeys.ptr, h->M, h->ctl, tmp, s);
    if (e == hipSuccess)
        e = hipMemcpyAsync(vgroup, tmp, (size_t)h->M * sizeof(int32_t), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess)
        e = hipStreamSynchronize(s);
    (void)hipFree(tmp);
    if (e != hipSuccess)
        return hip_fail(e, "export groups");
    return PAM_OK;
}

pam_status_t pam_lattice_set_capacity(pam_lattice_t lat, int64_t table_capacity, int32_t allow_regrow)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    if (table_capacity < 0 || table_capacity > ((int64_t)1 << 34))
        return fail(PAM_ERR_INVALID_ARGUMENT, "table_capacity out of range");
    lat->cap_request = table_capacity;
    lat->allow_regrow = allow_regrow != 0;
    return PAM_OK;
}

pam_status_t pam_timing_enable(pam_lattice_t lat, int32_t enable)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    DeviceGuard guard(lat->device);
    if (enable) {
        PAM_HIP(hipStreamSynchronize(lat->stream), "timing synchronise");
        drain_timing(lat);
        for (int k = 0; k < kKNumKinds; ++k) {
            lat->t_sum[k] = 0.0;
            lat->t_count[k] = 0;
        }
    }
    lat->timing = enable != 0;
    return PAM_OK;
}

pam_status_t pam_timing_read(pam_lattice_t lat, int32_t kind, int64_t *launches, double *total_ms)
{
    if (!lat)
        return fail(PAM_ERR_INVALID_ARGUMENT, "lat is NULL");
    if (kind < 0 || kind >= kKNumKinds)
        return fail(PAM_ERR_INVALID_ARGUMENT, "unknown kernel kind");
    DeviceGuard guard(lat->device);
    PAM_HIP(hipStreamSynchronize(lat->stream), "timing synchronise");
    drain_timing(lat);
    if (launches)
        *launches = lat->t_count[kind];
    if (total_ms)
        *total_ms = lat->t_sum[kind];
    return PAM_OK;
}

void pam_lattice_destroy(pam_lattice_t lat)
{
    if (!lat)
        return;
    {
        DeviceGuard guard(lat->device);
        (void)hipStreamSynchronize(lat->stream);
        drain_timing(lat);
        for (hipEvent_t e : lat->event_pool)
            (void)hipEventDestroy(e);
        DevBuf *bufs[] = {&lat->tkeys, &lat->tids,   &lat->vkeys,  &lat->nbr,    &lat->vert,
                          &lat->ntiles, &lat->bucket, &lat->scan,   &lat->pos0,   &lat->perm,
                          &lat->pts,    &lat->svert,  &lat->tiles,  &lat->lat[0], &lat->lat[1],
                          &lat->lat[2], &lat->lat[3], &lat->part, &lat->gstart, &lat->aug[0],
                          &lat->aug[1], &lat->aug[2], &lat->hA};
        for (DevBuf *b : bufs)
            if (b->ptr)
                (void)hipFree(b->ptr);
        if (lat->ctl)
            (void)hipFree(lat->ctl);
        if (lat->ctl_host)
            (void)hipHostFree(lat->ctl_host);
    }
    delete lat;
}

}  // extern "C"

namespace pam {

const char *kernel_name(int32_t kind)
{
    static const char *names[kKNumKinds] = {"range",   "layout",  "fill",       "insert",    "compact",
                                            "resolve", "scan",    "scatter",    "tiles",     "splat",
                                            "blur",    "slice",   "splat_bwd",  "slice_bwd", "splat_aug",
                                            "slice_aug"};
    if (kind < 0 || kind >= kKNumKinds)
        return "unknown";
    return names[kind];
}

}  // namespace pam

// HIP kernels (gfx950) that build the sparse permutohedral lattice of a
// point set (Joutard et al. 2019, Section 2: operator E of eq. 6 and the
// vertex set its simplices touch), and the simplex-sorted point order the
// filter kernels work in:
//   range      per point: rounded remainder-0 quotients -> per-coordinate
//              min/max (sizes the packed key)
//   layout     one thread: bit layout of the 63-bit packed key
//   insert     per tile of consecutive points: the tile's distinct vertex
//              keys into an open-addressing hash table
//   compact    per table slot: dense vertex ids
//   resolve    per point: the d+1 vertex ids; points counted per vertex 0
//   scan       exclusive prefix sum of those counts
//   scatter    per point: barycentric weights, ranks and ids written to the
//              point's place in the order sorted by vertex 0
//   tiles      per tile of the sorted order: distinct vertices as rows,
//              contributions sorted by row, segments, work order
//   neighbours per vertex and direction: ids of key -/+ u_j (extra blocks
//              of the resolve launch)
#include "pam_device.h"

#include <algorithm>

namespace pam {

// Per block: the min and max of the rounded quotients of its points, to
// part[c * kRangeBlocks + block] and part[(D + c) * kRangeBlocks + block],
// and whether one of them is not finite or too large, to
// part[2D * kRangeBlocks + block]; k_layout reduces the blocks.  The grid
// also clears the hash table for the insert.
constexpr int kRangeUnroll = 4;

template <int D>
__global__ __launch_bounds__(kBlock) void k_range(const float *__restrict__ feat, int64_t n, Elev E,
                                                  int32_t *__restrict__ part, uint64_t *__restrict__ tkeys,
                                                  uint64_t cap)
{
    for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < cap; i += (uint64_t)gridDim.x * kBlock)
        tkeys[i] = kEmptyKey;
    __shared__ int smin[kBlock / 64][D];
    __shared__ int smax[kBlock / 64][D];
    int qmin[D], qmax[D];
#pragma unroll
    for (int c = 0; c < D; ++c) {
        qmin[c] = INT_MAX;
        qmax[c] = INT_MIN;
    }
    bool bad = false;
    // kRangeUnroll points per thread and trip, their features requested
    // together before any is elevated
    constexpr int U = kRangeUnroll;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i0 = (int64_t)blockIdx.x * kBlock + threadIdx.x; i0 < n; i0 += U * stride) {
        float pl[U][D];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = i0 + u * stride;
#pragma unroll
            for (int j = 0; j < D; ++j)
                pl[u][j] = i < n ? feat[i * D + j] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (i0 + u * stride >= n)
                break;
            float x[D + 1];
            const bool ok = elevate<D>(pl[u], E, x);
            bad |= !ok;
            // rounded quotients before the remainder-0 fix-up; the fix-up and
            // the vertex offsets move them by at most -2..+1
#pragma unroll
            for (int c = 0; c < D; ++c) {
                const int q = ok ? (int)__builtin_rintf(x[c] * E.inv) : 0;
                qmin[c] = min(qmin[c], q);
                qmax[c] = max(qmax[c], q);
            }
        }
    }
#pragma unroll
    for (int c = 0; c < D; ++c) {
        for (int off = 32; off > 0; off >>= 1) {
            qmin[c] = min(qmin[c], __shfl_xor(qmin[c], off));
            qmax[c] = max(qmax[c], __shfl_xor(qmax[c], off));
        }
    }
    int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) {
#pragma unroll
        for (int c = 0; c < D; ++c) {
            smin[wave][c] = qmin[c];
            smax[wave][c] = qmax[c];
        }
    }
    __shared__ int bad_s;
    if (threadIdx.x == 0)
        bad_s = 0;
    __syncthreads();
    if (__ballot(bad) != 0 && lane == 0)
        bad_s = 1;
    __syncthreads();
    if (threadIdx.x == 0)
        part[2 * D * kRangeBlocks + blockIdx.x] = bad_s;
    if (threadIdx.x < D) {
        int c = threadIdx.x, lo = INT_MAX, hi = INT_MIN;
        for (int w = 0; w < kBlock / 64; ++w) {
            lo = min(lo, smin[w][c]);
            hi = max(hi, smax[w][c]);
        }
        part[c * kRangeBlocks + blockIdx.x] = lo;
        part[(D + c) * kRangeBlocks + blockIdx.x] = hi;
    }
}

// One block of 1024 threads: reduces the per-block ranges of k_range (all
// 2d+1 partial rows requested at once), resets the control block, and one
// thread lays out the packed key.
constexpr int kLayoutThreads = 1024;
static_assert(kRangeBlocks == 2 * kLayoutThreads, "two partials per layout thread");

template <int D>
__global__ __launch_bounds__(kLayoutThreads) void k_layout(Ctl *ctl, const int32_t *__restrict__ part, int nblocks,
                                                           int gbits)
{
    constexpr int d = D;
    constexpr int NW = kLayoutThreads / 64;
    __shared__ int sred[2 * D + 1][NW];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const bool on0 = t < nblocks, on1 = t + kLayoutThreads < nblocks;
    int v[2 * D + 1];
#pragma unroll
    for (int r = 0; r <= 2 * D; ++r) {
        const int id = r < D ? INT_MAX : (r < 2 * D ? INT_MIN : 0);
        const int a = on0 ? part[r * kRangeBlocks + t] : id;
        const int b = on1 ? part[r * kRangeBlocks + t + kLayoutThreads] : id;
        v[r] = r < D ? min(a, b) : (r < 2 * D ? max(a, b) : (a | b));
    }
#pragma unroll
    for (int r = 0; r <= 2 * D; ++r) {
        for (int off = 32; off > 0; off >>= 1) {
            const int o = __shfl_xor(v[r], off);
            v[r] = r < D ? min(v[r], o) : (r < 2 * D ? max(v[r], o) : (v[r] | o));
        }
        if (lane == 0)
            sred[r][wave] = v[r];
    }
    __syncthreads();
    if (t != 0)
        return;
    int bad = 0;
    for (int w = 0; w < NW; ++w)
        bad |= sred[2 * D][w];
    ctl->flags = bad ? kFlagBadFeature : 0u;
    ctl->count = 0;
    ctl->nvert = 0;
    ctl->pad = 0;
    for (int c = 0; c < d; ++c) {
        int lo = INT_MAX, hi = INT_MIN;
        for (int w = 0; w < NW; ++w) {
            lo = min(lo, sred[c][w]);
            hi = max(hi, sred[D + c][w]);
        }
        ctl->qmin[c] = lo;
        ctl->qmax[c] = hi;
    }
    KeyLayout &lay = ctl->lay;
    int kbits = 32 - __clz(d);  // bits for 0..d
    int shift = kbits;
    bool fits = true;
    for (int c = 0; c < d; ++c) {
        // vertex quotients lie in [qmin - 2, qmax + 1]; a neighbour outside
        // that range cannot be a vertex and packs as absent
        int64_t lo = (int64_t)ctl->qmin[c] - 2;
        int64_t width = (int64_t)ctl->qmax[c] - (int64_t)ctl->qmin[c] + 4;
        int bits = 64 - __clzll((unsigned long long)(width - 1));
        lay.lo[c] = (int32_t)lo;
        lay.shift[c] = shift;
        lay.bits[c] = bits;
        shift += bits;
        if (bits > 31 || shift > 63)
            fits = false;
    }
    lay.kbits = kbits;
    lay.gshift = shift;
    lay.gbits = gbits;
    shift += gbits;
    if (shift > 63)
        fits = false;
    lay.total_bits = shift;
    if (!fits)
        ctl->flags |= kFlagKeyRange;
}

__global__ void k_fill_f32(float *p, float value, int64_t count)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
}

// Insert key into the open-addressing table (linear probing).  Plain loads
// may see a stale empty slot; the compare-and-swap decides.  Keys are only
// ever written once (empty -> key), so a stale read is either empty or the
// final key.  Most keys of a tile are already in the table (the tiles
// around it share them), and the plain load finds those in the caches,
// where a compare-and-swap would go to the L2 every time.  Counts new keys
// in `added`; sets `full` if the whole table was probed.  Returns the key's
// slot (all ones when the table is full).
__device__ __forceinline__ uint64_t table_insert(uint64_t *tkeys, uint64_t mask, uint64_t key, uint32_t &added,
                                                 bool &full)
{
    uint64_t h = mix64(key) & mask;
    for (uint64_t probe = 0; probe <= mask; ++probe) {
        const uint64_t cur = tkeys[h];
        if (cur == key)
            return h;
        if (cur == kEmptyKey) {
            const uint64_t prev = atomicCAS((unsigned long long *)&tkeys[h], (unsigned long long)kEmptyKey,
                                            (unsigned long long)key);
            if (prev == kEmptyKey) {
                ++added;
                return h;
            }
            if (prev == key)
                return h;
        }
        h = (h + 1) & mask;
    }
    full = true;
    return ~0ull;
}

// Dense ids for the occupied slots: each block counts its PER * kBlock
// slots, scans the counts, and takes its id range with one update of a
// single counter (updates of one address serialise, so large tables take
// more slots per block).  Also clears the per-vertex bucket counters.
constexpr uint64_t kCompactWideCap = 1ull << 20;  // tables from this size take 16 slots per thread, else 4

template <int PER>
__global__ __launch_bounds__(kBlock) void k_compact(const uint64_t *__restrict__ tkeys, int32_t *tids,
                                                    uint64_t *vkeys, int32_t *__restrict__ bucket, uint64_t cap,
                                                    Ctl *ctl)
{
    constexpr int kCompactPer = PER;
    __shared__ int cs[kBlock];
    __shared__ int wsum[kBlock / 64 + 1];
    __shared__ uint32_t base_s;
    const uint64_t b0 = (uint64_t)blockIdx.x * kBlock * kCompactPer + threadIdx.x;
    int c = 0;
#pragma unroll
    for (int j = 0; j < kCompactPer; ++j) {
        const uint64_t s = b0 + (uint64_t)j * kBlock;
        c += (s < cap && tkeys[s] != kEmptyKey) ? 1 : 0;
    }
    cs[threadIdx.x] = c;
    __syncthreads();
    const int total = block_exclusive_scan(cs, kBlock, wsum);
    if (threadIdx.x == 0)
        base_s = total ? atomicAdd(&ctl->nvert, (uint32_t)total) : 0u;
    __syncthreads();
    uint32_t id = base_s + (uint32_t)cs[threadIdx.x];
#pragma unroll
    for (int j = 0; j < kCompactPer; ++j) {
        const uint64_t s = b0 + (uint64_t)j * kBlock;
        if (s < cap) {
            const uint64_t key = tkeys[s];
            if (key != kEmptyKey) {
                tids[s] = (int32_t)id;
                vkeys[id] = key;
                bucket[id] = 0;  // vertex-0 counts of k_resolve start at zero
                ++id;
            }
        }
    }
}

__device__ __forceinline__ int32_t probe_id(const uint64_t *__restrict__ tkeys,
                                            const int32_t *__restrict__ tids, uint64_t mask,
                                            uint64_t key)
{
    uint64_t h = mix64(key) & mask;
    for (uint64_t probe = 0; probe <= mask; ++probe) {
        uint64_t cur = tkeys[h];
        if (cur == key)
            return tids[h];
        if (cur == kEmptyKey)
            return -1;
        h = (h + 1) & mask;
    }
    return -1;
}

__device__ __forceinline__ void unpack_key(uint64_t key, int d, const KeyLayout &lay, int *coord)
{
    int k = (int)(key & ((1ull << lay.kbits) - 1));
    for (int c = 0; c < d; ++c) {
        int t = (int)((key >> lay.shift[c]) & ((1ull << lay.bits[c]) - 1)) + lay.lo[c];
        coord[c] = k + (d + 1) * t;
    }
}

// Pack explicit coordinates (all congruent mod d+1); false if outside the
// layout's range (such a vertex cannot be in the table).
__device__ __forceinline__ bool pack_coords(const int *coord, int d, const KeyLayout &lay,
                                            uint64_t *out)
{
    int k = ((coord[0] % (d + 1)) + (d + 1)) % (d + 1);
    uint64_t key = (uint64_t)k;
    for (int c = 0; c < d; ++c) {
        int t = (coord[c] - k) / (d + 1);
        int64_t off = (int64_t)t - lay.lo[c];
        if (off < 0 || off >= (1ll << lay.bits[c]))
            return false;
        key |= (uint64_t)off << lay.shift[c];
    }
    *out = key;
    return true;
}

// One entry of the neighbour table, item e = j * M + m: the ids of key_m
// -/+ u_j (-1 if absent).  nbr is direction-major:
// nbr[(j * M + m) * 2 + 0] = id(key_m - u_j), nbr[(j * M + m) * 2 + 1] = id(key_m + u_j).
__device__ __forceinline__ void neighbour_item(int d, const uint64_t *__restrict__ vkeys, int64_t M,
                                               const KeyLayout &lay, const uint64_t *__restrict__ tkeys,
                                               const int32_t *__restrict__ tids, uint64_t mask,
                                               int32_t *__restrict__ nbr, int64_t e)
{
    int64_t m = e % M;
    int j = (int)(e / M);
    int base[kMaxD], nb[kMaxD];
    const uint64_t key_m = vkeys[m];
    const uint64_t gfield = lay.gbits ? key_m & (((1ull << lay.gbits) - 1) << lay.gshift) : 0;
    unpack_key(key_m, d, lay, base);
    // both keys first, then both probes side by side: their first slots,
    // then their ids, are requested together
    uint64_t key[2] = {0, 0};
    bool ok[2];
    for (int sgn = 0; sgn < 2; ++sgn) {
        int step = sgn ? 1 : -1;
        for (int c = 0; c < d; ++c)
            nb[c] = base[c] + step * ((c == j) ? d : -1);
        ok[sgn] = pack_coords(nb, d, lay, &key[sgn]);
        key[sgn] |= gfield;
    }
    uint64_t h[2], cur[2];
    for (int sgn = 0; sgn < 2; ++sgn) {
        h[sgn] = mix64(key[sgn]) & mask;
        cur[sgn] = ok[sgn] ? tkeys[h[sgn]] : kEmptyKey;
    }
    int64_t slot[2];
    for (int sgn = 0; sgn < 2; ++sgn) {
        slot[sgn] = -1;
        for (uint64_t probe = 0; ok[sgn] && probe <= mask; ++probe) {
            if (cur[sgn] == key[sgn]) {
                slot[sgn] = (int64_t)h[sgn];
                break;
            }
            if (cur[sgn] == kEmptyKey)
                break;
            h[sgn] = (h[sgn] + 1) & mask;
            cur[sgn] = tkeys[h[sgn]];
        }
    }
    const int32_t id0 = slot[0] >= 0 ? tids[slot[0]] : -1;
    const int32_t id1 = slot[1] >= 0 ? tids[slot[1]] : -1;
    reinterpret_cast<int2 *>(nbr)[j * M + m] = make_int2(id0, id1);
}

__global__ void k_vertex_groups(const uint64_t *__restrict__ vkeys, int64_t M, const Ctl *ctl, int32_t *vgroup)
{
    const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (m >= M)
        return;
    const KeyLayout &lay = ctl->lay;
    vgroup[m] = lay.gbits ? (int32_t)((vkeys[m] >> lay.gshift) & ((1ull << lay.gbits) - 1)) : 0;
}

__global__ void k_unpack_keys(int d, const uint64_t *__restrict__ vkeys, int64_t M, const Ctl *ctl,
                              int32_t *keys)
{
    int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (m >= M)
        return;
    int coord[kMaxD];
    unpack_key(vkeys[m], d, ctl->lay, coord);
    for (int c = 0; c < d; ++c)
        keys[m * d + c] = coord[c];
}

// Per sorted position s: the point's vertex ids and barycentric weights as
// the filter kernels read them (the sorted records), written back at the
// point's original index perm[s].
__global__ void k_export_points(int d, const uint8_t *__restrict__ pts, const int32_t *__restrict__ svert,
                                const int32_t *__restrict__ perm, int64_t n, int32_t *vert, float *bary)
{
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= n)
        return;
    const int64_t i = perm[s];
    const float *w = reinterpret_cast<const float *>(pts + s * point_bytes(d));
    for (int k = 0; k <= d; ++k) {
        bary[i * (d + 1) + k] = w[k];
        vert[i * (d + 1) + k] = svert[s * (d + 1) + k];
    }
}


// The lattice's vertex set, built a tile of consecutive points at a time:
// the d+1 vertex keys of every point are deduplicated in an LDS hash
// (64-bit compare-and-swap), and only the tile's distinct keys are inserted
// into the global table.  The tile's record keeps the distinct keys and each
// point's local row, so that k_resolve attaches global ids with one table
// lookup per distinct key.
// LDS hash of a tile: 2048 slots while a tile has at most 3072
// contributions (d <= 5 at 512 points), else 4096.
__host__ __device__ constexpr int tile_hash_bits(int d) { return tile_points(d) * (d + 1) <= 3072 ? 11 : 12; }
constexpr int kTileProbe = 64;

template <int D>
__global__ __launch_bounds__(tile_points(D)) void k_insert_tiles(const float *__restrict__ feat, int64_t n, Elev E,
                                                                 Groups64 grp, Ctl *ctl, KeyLayout fixed,
                                                                 int use_fixed, uint64_t *tkeys, uint64_t mask,
                                                                 uint8_t *__restrict__ tiles)
{
    constexpr int T = tile_points(D);
    constexpr int kTileHashBits = tile_hash_bits(D);
    constexpr int kTileHash = 1 << kTileHashBits;
    __shared__ uint64_t hkey[kTileHash];
    __shared__ int16_t hrow[kTileHash];
    __shared__ uint64_t rkey[kTileHash];  // distinct keys, row order
    __shared__ int nrows_s, overflow_s, full_s, miss_s;
    __shared__ uint32_t added_s;
    if (!use_fixed && (ctl->flags & (kFlagKeyRange | kFlagBadFeature)))
        return;
    const KeyLayout lay = use_fixed ? fixed : ctl->lay;
    if (use_fixed && blockIdx.x == 0 && threadIdx.x == 0)
        ctl->lay = fixed;  // for the later kernels of the build (identical in every block)
    const TileRec rec(D);
    const int t = threadIdx.x;
    const int64_t tile = insert_tile((n + T - 1) / T);
    const int64_t base = tile * T;
    const int nt = (int)min((int64_t)T, n - base);
    const int nc = nt * (D + 1);
    uint8_t *R = tiles + (size_t)tile * rec.bytes;
    uint32_t *hdr = reinterpret_cast<uint32_t *>(R);
    uint64_t *rowkey = reinterpret_cast<uint64_t *>(R + rec.rowkey);
    uint16_t *lrow = reinterpret_cast<uint16_t *>(R + rec.lrow);
    for (int e = t; e < kTileHash; e += T)
        hkey[e] = kEmptyKey;
    if (t == 0) {
        nrows_s = 0;
        overflow_s = 0;
        added_s = 0;
        full_s = 0;
        miss_s = 0;
    }
    __syncthreads();
    // Neighbouring points often share vertices: only the first lane of a
    // run of equal keys in a wave probes the LDS table, the others take its
    // slot.  The loop over k is wave-uniform (cross-lane operations).
    const int lane = t & 63;
    const bool valid = t < nt;
    uint64_t key[D + 1];
    int slot[D + 1];
    Simplex<D> s;
    uint64_t gfield = 0;
    if (valid) {
        const bool ok = embed<D>(feat + (base + t) * D, E, s);
        gfield = group_field(grp, lay, base + t);
        if (use_fixed) {
            // every vertex quotient of the point is q_c or q_c - 1: both must
            // fit the fixed layout's field (else the build takes the range pass)
            bool fits = ok;
#pragma unroll
            for (int c = 0; c < D; ++c)
                fits = fits && s.q[c] - 1 - lay.lo[c] >= 0 && s.q[c] - lay.lo[c] < (1 << lay.bits[c]);
            if (!ok)
                atomicOr(&ctl->flags, kFlagBadFeature);
            if (!fits)
                miss_s = 1;
        }
    }
#pragma unroll
    for (int k = 0; k <= D; ++k) {
        key[k] = valid ? pack_vertex<D>(s, k, lay, gfield) : kEmptyKey;
        const LaneRun run = lane_run(key[k], valid);
        int found = -1;
        if (valid && run.lead == lane) {
            uint32_t h = (uint32_t)(mix64(key[k]) >> (64 - kTileHashBits));
            for (int probe = 0; probe < kTileProbe; ++probe) {
                const uint64_t prev = atomicCAS((unsigned long long *)&hkey[h], (unsigned long long)kEmptyKey,
                                                (unsigned long long)key[k]);
                if (prev == kEmptyKey) {
                    const int r = atomicAdd(&nrows_s, 1);
                    hrow[h] = r;
                    rkey[r] = key[k];
                    found = (int)h;
                    break;
                }
                if (prev == key[k]) {
                    found = (int)h;
                    break;
                }
                h = (h + 1) & (kTileHash - 1);
            }
        }
        found = __shfl(found, run.lead);
        slot[k] = found;
        if (valid && found < 0)
            overflow_s = 1;
    }
    __syncthreads();
    if (miss_s) {  // block-uniform: the keys are not valid in this layout
        if (t == 0)
            atomicOr(&ctl->flags, kFlagLayoutMiss);
        return;
    }
    uint32_t added = 0;
    bool full = false;
    if (overflow_s) {
        // no room to deduplicate: every key of the tile goes to the table
        if (t < nt) {
#pragma unroll
            for (int k = 0; k <= D; ++k)
                table_insert(tkeys, mask, key[k], added, full);
        }
    } else {
        // each distinct key's slot goes to the tile record (its rowid field,
        // unused by tiles of consecutive points) so that k_resolve reads the
        // key's id without probing; -1 when the slot does not fit an int32
        int32_t *rslot = reinterpret_cast<int32_t *>(R + rec.rowid);
        for (int r = t; r < nrows_s; r += T) {
            const uint64_t h = table_insert(tkeys, mask, rkey[r], added, full);
            rowkey[r] = rkey[r];
            rslot[r] = h <= 0x7fffffffull ? (int32_t)h : -1;
        }
        if (t < nt) {
#pragma unroll
            for (int k = 0; k <= D; ++k)
                lrow[t * (D + 1) + k] = (uint16_t)hrow[slot[k]];
        }
    }
    if (added)
        atomicAdd(&added_s, added);
    if (full)
        full_s = 1;
    __syncthreads();
    if (t == 0) {
        // the count's result is not needed here (the host compares the
        // final count with the load limit), so the add does not return
        if (added_s)
            atomicAdd(&ctl->count, added_s);
        if (full_s)
            atomicOr(&ctl->flags, kFlagTableFull);
        hdr[0] = overflow_s ? 0u : (uint32_t)nrows_s;
        hdr[1] = overflow_s ? kTileOverflow : 0u;
        hdr[2] = (uint32_t)nc;
        hdr[3] = 0;
    }
}

// Per tile of consecutive points: the global id of each distinct key of the
// tile, one table lookup each, written over the key's slot in the tile's
// record (tiles that overflowed their LDS table look up every point's keys
// and write the points' ids in natural order instead), and each point's
// position among the points that share its vertex 0.
// The grid's blocks past the last tile fill the neighbour table (one item
// per thread), which needs only the compacted vertex keys and the table.
template <int D>
__global__ __launch_bounds__(tile_points(D)) void k_resolve(const float *__restrict__ feat, int64_t n, Elev E,
                                                            Groups64 grp, const Ctl *ctl,
                                                            const uint64_t *__restrict__ tkeys,
                                                            const int32_t *__restrict__ tids, uint64_t mask,
                                                            uint8_t *__restrict__ tiles,
                                                            int32_t *__restrict__ vert, int32_t *__restrict__ bucket,
                                                            int32_t *__restrict__ pos0,
                                                            const uint64_t *__restrict__ vkeys, int64_t M,
                                                            int32_t *__restrict__ nbr)
{
    constexpr int T = tile_points(D);
    constexpr int NC = T * (D + 1);
    constexpr int J = (1 << tile_hash_bits(D)) / T;  // rows per thread at most (a tile's rows fit the insert's LDS table)
    __shared__ int rid[NC];
    __shared__ int cnt0[NC];  // per row: the tile's points with it as vertex 0, then their bucket base
    const int64_t ntiles = (n + T - 1) / T;
    if ((int64_t)blockIdx.x >= ntiles) {  // block-uniform
        const int64_t e = ((int64_t)blockIdx.x - ntiles) * T + threadIdx.x;
        if (e < M * (D + 1))
            neighbour_item(D, vkeys, M, ctl->lay, tkeys, tids, mask, nbr, e);
        return;
    }
    const TileRec rec(D);
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, n - base);
    uint8_t *R = tiles + (size_t)blockIdx.x * rec.bytes;
    const uint32_t *hdr = reinterpret_cast<const uint32_t *>(R);
    const uint64_t *rowkey = reinterpret_cast<const uint64_t *>(R + rec.rowkey);
    const uint16_t *lrow = reinterpret_cast<const uint16_t *>(R + rec.lrow);
    const bool overflow = (hdr[1] & kTileOverflow) != 0;
    const int nrows = (int)hdr[0];
    if (!overflow) {
        // the insert's slot of each distinct key (or -1) becomes the key's id,
        // in place: the scatter reads the points' ids from this record
        // (a thread's rows are requested together: slots, then ids)
        int32_t *rslot = reinterpret_cast<int32_t *>(R + rec.rowid);
        int32_t hs[J], ids[J];
#pragma unroll
        for (int j = 0; j < J; ++j)
            hs[j] = t + j * T < nrows ? rslot[t + j * T] : -1;
#pragma unroll
        for (int j = 0; j < J; ++j)
            ids[j] = hs[j] >= 0 ? tids[hs[j]] : -1;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int r = t + j * T;
            if (r < nrows) {
                const int32_t id = hs[j] >= 0 ? ids[j] : probe_id(tkeys, tids, mask, rowkey[r]);
                rid[r] = id;
                rslot[r] = id;
                cnt0[r] = 0;
            }
        }
    }
    __syncthreads();
    // Bucket positions: the tile's points are counted per vertex-0 row in
    // LDS (one atomic per run of equal rows in a wave), then each row takes
    // its range of its bucket with one global atomic.
    const int lane = t & 63;
    const bool counted = !overflow && t < nt;
    const int r0 = counted ? (int)lrow[t * (D + 1)] : 0;
    const LaneRun run = lane_run((uint64_t)(uint32_t)r0, counted);
    int lpos = 0;
    if (counted && run.lead == lane)
        lpos = atomicAdd(&cnt0[r0], run.len);
    lpos = __shfl(lpos, run.lead) + (lane - run.lead);
    __syncthreads();
    if (!overflow) {
        int got[J];
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int r = t + j * T;
            const int c = r < nrows ? cnt0[r] : 0;
            got[j] = c > 0 ? atomicAdd(&bucket[max(rid[r], 0)], c) : 0;
        }
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int r = t + j * T;
            if (r < nrows && cnt0[r] > 0)
                cnt0[r] = got[j];
        }
    }
    __syncthreads();
    if (t >= nt)
        return;
    const int64_t i = base + t;
    if (overflow) {
        // no per-tile rows: every key is looked up, and the ids go to the
        // natural-order array the scatter reads for such tiles
        const KeyLayout lay = ctl->lay;
        Simplex<D> s;
        embed<D>(feat + i * D, E, s);
        int ids[D + 1];
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            ids[k] = probe_id(tkeys, tids, mask, pack_vertex<D>(s, k, lay, group_field(grp, lay, i)));
            vert[i * (D + 1) + k] = ids[k];
        }
        pos0[i] = atomicAdd(&bucket[max(ids[0], 0)], 1);
    } else {
        pos0[i] = cnt0[r0] + lpos;
    }
}

// Exclusive prefix sum of an int array of any length: per-block scans of
// kBlock * kScanPer elements, a scan of the block totals (one block, in
// chunks with a running carry), and a final add.
constexpr int kScanPer = 8;  // elements per thread
constexpr int kScanChunk = 4096;
constexpr int64_t kScanOneBlock = 24576;  // up to here one block scans the array

// One block: exclusive scan of x[0..count), count <= kScanOneBlock.  Each
// thread holds kScanOneBlock / 1024 consecutive elements in registers (read
// and written as int4), the threads' sums are scanned across the wave with
// shuffles and across the block's 16 waves in LDS.
__global__ __launch_bounds__(1024) void k_scan_lds(int32_t *__restrict__ x, int count)
{
    constexpr int PER = (int)(kScanOneBlock / 1024);
    static_assert(PER % 4 == 0 && PER * 1024 == kScanOneBlock, "int4 pieces per thread");
    constexpr int NW = 1024 / 64;
    __shared__ int wsum[NW];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int b0 = t * PER;
    int v[PER];
#pragma unroll
    for (int q = 0; q < PER / 4; ++q) {
        const int e = b0 + 4 * q;
        int4 z = make_int4(0, 0, 0, 0);
        if (e + 3 < count) {
            z = *reinterpret_cast<const int4 *>(x + e);
        } else {
            z.x = e < count ? x[e] : 0;
            z.y = e + 1 < count ? x[e + 1] : 0;
            z.z = e + 2 < count ? x[e + 2] : 0;
        }
        v[4 * q] = z.x;
        v[4 * q + 1] = z.y;
        v[4 * q + 2] = z.z;
        v[4 * q + 3] = z.w;
    }
    int s = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i)
        s += v[i];
    int incl = s;  // inclusive scan of the thread sums over the wave
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (lane >= off)
            incl += y;
    }
    if (lane == 63)
        wsum[w] = incl;
    __syncthreads();
    if (t == 0) {
        int run = 0;
        for (int i = 0; i < NW; ++i) {
            const int u = wsum[i];
            wsum[i] = run;
            run += u;
        }
    }
    __syncthreads();
    int run = wsum[w] + incl - s;  // exclusive prefix of this thread's first element
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int u = v[i];
        v[i] = run;
        run += u;
    }
#pragma unroll
    for (int q = 0; q < PER / 4; ++q) {
        const int e = b0 + 4 * q;
        if (e + 3 < count) {
            *reinterpret_cast<int4 *>(x + e) = make_int4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
        } else {
            if (e < count)
                x[e] = v[4 * q];
            if (e + 1 < count)
                x[e + 1] = v[4 * q + 1];
            if (e + 2 < count)
                x[e + 2] = v[4 * q + 2];
        }
    }
}

__global__ __launch_bounds__(kBlock) void k_scan_blocks(int32_t *__restrict__ x, int64_t count,
                                                        int32_t *__restrict__ sums)
{
    __shared__ int cs[kBlock * kScanPer];
    __shared__ int wsum[kBlock / 64 + 1];
    const int64_t b0 = (int64_t)blockIdx.x * kBlock * kScanPer;
    for (int e = threadIdx.x; e < kBlock * kScanPer; e += kBlock)
        cs[e] = (b0 + e < count) ? x[b0 + e] : 0;
    __syncthreads();
    const int total = block_exclusive_scan(cs, kBlock * kScanPer, wsum);
    for (int e = threadIdx.x; e < kBlock * kScanPer; e += kBlock)
        if (b0 + e < count)
            x[b0 + e] = cs[e];
    if (threadIdx.x == 0)
        sums[blockIdx.x] = total;
}

// One block: in-place exclusive scan of sums[0..nblocks) in chunks with a
// running carry (the block totals of k_scan_blocks, or a short array).
__global__ __launch_bounds__(1024) void k_scan_sums(int32_t *__restrict__ sums, int64_t nblocks)
{
    __shared__ int cs[kScanChunk];
    __shared__ int wsum[1024 / 64 + 1];
    int carry = 0;
    for (int64_t c0 = 0; c0 < nblocks; c0 += kScanChunk) {
        for (int e = threadIdx.x; e < kScanChunk; e += 1024)
            cs[e] = (c0 + e < nblocks) ? sums[c0 + e] : 0;
        __syncthreads();
        const int total = block_exclusive_scan(cs, kScanChunk, wsum);
        for (int e = threadIdx.x; e < kScanChunk; e += 1024)
            if (c0 + e < nblocks)
                sums[c0 + e] = cs[e] + carry;
        carry += total;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kBlock) void k_scan_add(int32_t *__restrict__ x, int64_t count,
                                                     const int32_t *__restrict__ sums)
{
    const int64_t b0 = (int64_t)blockIdx.x * kBlock * kScanPer;
    const int add = sums[blockIdx.x];
    for (int e = threadIdx.x; e < kBlock * kScanPer; e += kBlock)
        if (b0 + e < count)
            x[b0 + e] += add;
}

// Every point to its place in the simplex-sorted order: points are grouped
// by their vertex 0 (bucket starts from the scan), within a group in the
// order in which they took their positions.  The point's record there holds
// its barycentric weights and ranks (recomputed from its features), next to
// its d+1 vertex ids and its original index.  A vertex id that is missing
// (never after a successful build) becomes vertex 0 with weight 0.
template <int D>
__global__ __launch_bounds__(kBlock) void k_scatter(const float *__restrict__ feat, int64_t n, Elev E,
                                                    const uint8_t *__restrict__ ntiles,
                                                    const int32_t *__restrict__ vert,
                                                    const int32_t *__restrict__ start,
                                                    const int32_t *__restrict__ pos0, int32_t *__restrict__ perm,
                                                    uint8_t *__restrict__ psort, int32_t *__restrict__ svert)
{
    constexpr int PW = point_bytes(D) / 4;
    constexpr int T = tile_points(D);
    static_assert(T % kBlock == 0, "a block's points lie in one tile");
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n)
        return;
    // the point's ids: its local rows in its tile of consecutive points and
    // the tile's row ids (written by the resolve), or the natural-order ids
    // of a tile that overflowed its LDS table
    const TileRec rec(D);
    const int64_t tile = i / T;
    const int p = (int)(i - tile * T);
    const uint8_t *R = ntiles + (size_t)tile * rec.bytes;
    const bool overflow = (reinterpret_cast<const uint32_t *>(R)[1] & kTileOverflow) != 0;
    int ids[D + 1];
    if (!overflow) {
        const uint16_t *lrow = reinterpret_cast<const uint16_t *>(R + rec.lrow) + p * (D + 1);
        const int32_t *rid = reinterpret_cast<const int32_t *>(R + rec.rowid);
        int lr[D + 1];
#pragma unroll
        for (int k = 0; k <= D; ++k)
            lr[k] = lrow[k];
#pragma unroll
        for (int k = 0; k <= D; ++k)
            ids[k] = rid[lr[k]];
    } else {
#pragma unroll
        for (int k = 0; k <= D; ++k)
            ids[k] = vert[i * (D + 1) + k];
    }
    const int64_t dst = (int64_t)start[max(ids[0], 0)] + pos0[i];
    Simplex<D> s;
    embed<D>(feat + i * D, E, s);
    float b[D + 1];
    barycentric<D>(s, feat + i * D, E, b);
    uint32_t w[PW];
#pragma unroll
    for (int u = 0; u < PW; ++u)
        w[u] = 0u;
#pragma unroll
    for (int k = 0; k <= D; ++k)
        w[k] = __float_as_uint(ids[k] >= 0 ? b[k] : 0.0f);
#pragma unroll
    for (int c = 0; c <= D; ++c)
        w[D + 1 + c / 4] |= (uint32_t)(s.rank[c] & 0xff) << (8 * (c % 4));
    uint4 *prec = reinterpret_cast<uint4 *>(psort + dst * (PW * 4));
#pragma unroll
    for (int u = 0; u < PW / 4; ++u)
        prec[u] = make_uint4(w[4 * u], w[4 * u + 1], w[4 * u + 2], w[4 * u + 3]);
    if constexpr ((D + 1) % 2 == 0) {
#pragma unroll
        for (int k = 0; k <= D; k += 2)
            reinterpret_cast<int2 *>(svert + dst * (D + 1))[k / 2] = make_int2(max(ids[k], 0), max(ids[k + 1], 0));
    } else {
#pragma unroll
        for (int k = 0; k <= D; ++k)
            svert[dst * (D + 1) + k] = max(ids[k], 0);
    }
    perm[dst] = (int32_t)i;
}

// Per tile of the sorted order: the tile's distinct vertex ids become dense
// rows (LDS hash, integer compare-and-swap); the tile's (point, vertex)
// contributions are counting-sorted by (window, row) (integer LDS atomics
// give each its position within its pair); each pair's contributions are
// cut into segments of at most kSegLen, and the segments are
// counting-sorted window by window and by length, longest first, the order
// in which the splat hands them out.
// The grid's blocks past the last tile clear the first `zelems` floats of
// z0 and z1 (a multiple of 4; the lattice buffers the next filter calls
// splat into), so that those calls need no clearing launch of their own,
// and, with tkeys, empty the hash table's cap slots and zero the control
// block's flags and counters for the next build's insert.
template <int D>
__global__ __launch_bounds__(tile_points(D)) void k_sorted_tiles(const int32_t *__restrict__ svert, int64_t n,
                                                                 uint8_t *__restrict__ tiles, float *__restrict__ z0,
                                                                 float *__restrict__ z1, int64_t zelems,
                                                                 uint64_t *__restrict__ tkeys, uint64_t cap, Ctl *ctl)
{
    constexpr int T = tile_points(D);
    constexpr int NC = T * (D + 1);
    static_assert(NC < (1 << 13), "segment start and row must fit their 13-bit fields");
    const int64_t ntiles = (n + T - 1) / T;
    if ((int64_t)blockIdx.x >= ntiles) {  // block-uniform
        const int64_t e = ((int64_t)blockIdx.x - ntiles) * T + threadIdx.x;  // 16-byte piece
        if (4 * e < zelems) {
            const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
            reinterpret_cast<float4 *>(z0)[e] = z;
            reinterpret_cast<float4 *>(z1)[e] = z;
        }
        if (tkeys) {
            if ((uint64_t)(2 * e) < cap)  // cap is a power of two >= 64: whole pieces
                reinterpret_cast<ulonglong2 *>(tkeys)[e] = make_ulonglong2(kEmptyKey, kEmptyKey);
            if (e == 0) {
                ctl->flags = 0;
                ctl->count = 0;
                ctl->nvert = 0;
            }
        }
        return;
    }
    constexpr int kTileHashBits = tile_hash_bits(D);
    constexpr int kTileHash = 1 << kTileHashBits;
    __shared__ int hkey[kTileHash];
    __shared__ int16_t hrow[kTileHash];
    constexpr int kWin = splat_windows(D);  // point windows per tile
    constexpr int kWinPts = T / kWin;
    static_assert(kWin == 1 || kWinPts >= 64, "a wave must not span two windows");
    __shared__ int cnt[kTileHash + 1];  // per (window, row): count, then first entry
    __shared__ int nsg[kTileHash + 1];  // per (window, row): segment count, then first segment
    __shared__ int hist[kWin * (kSegLen + 1)];
    __shared__ int wsum[2 * (T / 64 + 1)];
    __shared__ int nrows_s, overflow_s;
    const TileRec rec(D);
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, n - base);
    const int nc = nt * (D + 1);
    uint8_t *R = tiles + (size_t)blockIdx.x * rec.bytes;
    uint32_t *hdr = reinterpret_cast<uint32_t *>(R);
    int32_t *rowid = reinterpret_cast<int32_t *>(R + rec.rowid);
    uint16_t *sfirst = reinterpret_cast<uint16_t *>(R + rec.sfirst);
    uint32_t *seg = reinterpret_cast<uint32_t *>(R + rec.seg);
    uint16_t *order = reinterpret_cast<uint16_t *>(R + rec.order);
    uint16_t *list = reinterpret_cast<uint16_t *>(R + rec.list);
    uint16_t *lrow = reinterpret_cast<uint16_t *>(R + rec.lrow);
    uint16_t *pent = reinterpret_cast<uint16_t *>(R + rec.pent);
    for (int e = t; e < kTileHash; e += T)
        hkey[e] = -1;
    for (int e = t; e <= kTileHash; e += T) {
        cnt[e] = 0;
        nsg[e] = 0;
    }
    for (int e = t; e < kWin * (kSegLen + 1); e += T)
        hist[e] = 0;
    if (t == 0) {
        nrows_s = 0;
        overflow_s = 0;
    }
    __syncthreads();
    // Sorted points share vertices in long runs: only the first lane of a
    // run of equal ids in a wave probes the LDS table (and later counts the
    // whole run), the others take its results.  The loops over k are
    // wave-uniform (cross-lane operations).
    const int lane = t & 63;
    const bool valid = t < nt;
    int slot[D + 1];
    LaneRun run[D + 1];
#pragma unroll
    for (int k = 0; k <= D; ++k) {
        const int m = valid ? svert[(base + t) * (D + 1) + k] : 0;  // >= 0
        run[k] = lane_run((uint64_t)(uint32_t)m, valid);
        int found = -1;
        if (valid && run[k].lead == lane) {
            uint32_t h = ((uint32_t)m * 2654435761u) >> (32 - kTileHashBits);
            for (int probe = 0; probe < kTileProbe; ++probe) {
                const int prev = atomicCAS(&hkey[h], -1, m);
                if (prev == -1) {
                    const int r = atomicAdd(&nrows_s, 1);
                    hrow[h] = r;
                    rowid[r] = m;
                    found = (int)h;
                    break;
                }
                if (prev == m) {
                    found = (int)h;
                    break;
                }
                h = (h + 1) & (kTileHash - 1);
            }
        }
        found = __shfl(found, run[k].lead);
        slot[k] = found;
        if (valid && found < 0)
            overflow_s = 1;
    }
    __syncthreads();
    // a tile whose (window, row) pairs do not fit the counters or the record
    // takes the overflow path too
    if (kWin > 1 && t == 0 && !(nrows_s * kWin <= kTileHash && nrows_s * kWin <= NC))
        overflow_s = 1;
    __syncthreads();
    if (overflow_s) {
        if (t == 0) {
            hdr[0] = 0;
            hdr[1] = kTileOverflow;
            hdr[2] = (uint32_t)nc;
            hdr[3] = 0;
        }
        return;
    }
    // Contributions are counting-sorted by (point window, row): a row's
    // contributions from one window of consecutive points form their own
    // segments, and window w's entries and segments are contiguous.
    const int nrows = nrows_s;
    const int nwin = kWin;
    const int nq = nrows * nwin;
    const int win = nwin > 1 ? t / kWinPts : 0;
    int q[D + 1], pos[D + 1];
#pragma unroll
    for (int k = 0; k <= D; ++k) {
        const int row = valid ? hrow[slot[k]] : 0;
        q[k] = win * nrows + row;
        int b = 0;
        if (valid && run[k].lead == lane)
            b = atomicAdd(&cnt[q[k]], run[k].len);
        pos[k] = __shfl(b, run[k].lead) + (lane - run[k].lead);
        if (valid)
            lrow[t * (D + 1) + k] = (uint16_t)row;
    }
    __syncthreads();
    // cnt[q]: first entry of pair q; nsg[q]: its first segment
    const int nseg = block_exclusive_scan_ceil(cnt, nsg, nq, kSegLen, wsum);
    if (t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k)
            list[cnt[q[k]] + pos[k]] = (uint16_t)((t << 5) | k);
    }
    // segments in (window, row) order, and a histogram of (window, length)
    for (int qq = t; qq < nq; qq += T) {
        const int e0 = cnt[qq], e1 = (qq + 1 < nq) ? cnt[qq + 1] : nc;
        const int w = qq / nrows, r = qq - w * nrows;
        sfirst[qq] = (uint16_t)nsg[qq];
        pent[qq] = (uint16_t)e0;
        for (int j = 0, e = e0; e < e1; ++j, e += kSegLen) {
            const int len = min(kSegLen, e1 - e);
            seg[nsg[qq] + j] = seg_encode(e, len, r);
            atomicAdd(&hist[w * (kSegLen + 1) + kSegLen - len], 1);  // longest first within a window
        }
    }
    __syncthreads();
    if (t < 64) {
        // bucket starts (then used as cursors): an exclusive scan of the
        // histogram by the first wave, each lane over NBL consecutive buckets
        constexpr int NB = kWin * (kSegLen + 1), NBL = (NB + 63) / 64;
        int v[NBL], sum = 0;
#pragma unroll
        for (int i = 0; i < NBL; ++i) {
            const int b = t * NBL + i;
            v[i] = b < NB ? hist[b] : 0;
            sum += v[i];
        }
        int incl = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(incl, off);
            if (t >= off)
                incl += y;
        }
        int run = incl - sum;
#pragma unroll
        for (int i = 0; i < NBL; ++i) {
            const int b = t * NBL + i;
            if (b < NB)
                hist[b] = run;
            run += v[i];
        }
    }
    if (t == 0) {
        sfirst[nq] = (uint16_t)nseg;
        pent[nq] = (uint16_t)nc;
        hdr[0] = (uint32_t)nrows;
        hdr[1] = (uint32_t)nwin << 8;
        hdr[2] = (uint32_t)nc;
        hdr[3] = (uint32_t)nseg;
    }
    __syncthreads();
    // work order: windows in turn, longest segments first within a window
    for (int qq = t; qq < nq; qq += T) {
        const int e0 = cnt[qq], e1 = (qq + 1 < nq) ? cnt[qq + 1] : nc;
        const int w = qq / nrows;
        for (int j = 0, e = e0; e < e1; ++j, e += kSegLen) {
            const int len = min(kSegLen, e1 - e);
            order[atomicAdd(&hist[w * (kSegLen + 1) + kSegLen - len], 1)] = (uint16_t)(nsg[qq] + j);
        }
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

static unsigned range_blocks(int64_t n)
{
    const unsigned grid = blocks_for(n);
    return grid > kRangeBlocks ? kRangeBlocks : (grid == 0 ? 1 : grid);
}

size_t tile_record_bytes_build(int d) { return TileRec(d).bytes; }

hipError_t launch_range(int d, const float *feat, int64_t n, const Elev &E, int32_t *part, uint64_t *tkeys,
                        uint64_t cap, hipStream_t s)
{
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_range<D>, dim3(range_blocks(n)), dim3(kBlock), 0, s, feat, n, E, part,
                                         tkeys, cap));
    return hipGetLastError();
}

hipError_t launch_layout(int d, int64_t n, int gbits, Ctl *ctl, const int32_t *part, hipStream_t s)
{
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_layout<D>, dim3(1), dim3(kLayoutThreads), 0, s, ctl, part,
                                         (int)range_blocks(n), gbits));
    return hipGetLastError();
}

hipError_t launch_fill_f32(float *p, float value, int64_t count, hipStream_t s)
{
    if (count <= 0)
        return hipSuccess;
    unsigned grid = blocks_for(count);
    grid = grid > 4096 ? 4096 : grid;
    hipLaunchKernelGGL(k_fill_f32, dim3(grid), dim3(kBlock), 0, s, p, value, count);
    return hipGetLastError();
}

hipError_t launch_insert_tiles(int d, const float *feat, int64_t n, const Elev &E, const Groups64 &grp, Ctl *ctl,
                               const KeyLayout *fixed, uint64_t *tkeys, uint64_t cap, uint8_t *tiles,
                               hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    const unsigned grid = (unsigned)((n + tile_points(d) - 1) / tile_points(d));
    const KeyLayout lay = fixed ? *fixed : KeyLayout{};
    const int use_fixed = fixed ? 1 : 0;
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_insert_tiles<D>, dim3(grid), dim3(tile_points(d)), 0, s, feat, n, E, grp,
                                         ctl, lay, use_fixed, tkeys, cap - 1, tiles));
    return hipGetLastError();
}

bool fixed_layout(int d, int gbits, KeyLayout *lay)
{
    if (d < 1 || d > kMaxD)
        return false;
    int kbits = 0;
    while ((1 << kbits) <= d)
        ++kbits;  // bits for 0..d
    const int bits = (63 - kbits - gbits) / d;
    if (bits < 6)
        return false;
    KeyLayout L{};
    int shift = kbits;
    for (int c = 0; c < d; ++c) {
        L.lo[c] = -(1 << (bits - 1));
        L.bits[c] = bits;
        L.shift[c] = shift;
        shift += bits;
    }
    L.kbits = kbits;
    L.gshift = shift;
    L.gbits = gbits;
    L.total_bits = shift + gbits;
    *lay = L;
    return true;
}

hipError_t launch_resolve(int d, const float *feat, int64_t n, const Elev &E, const Groups64 &grp, const Ctl *ctl,
                          const uint64_t *tkeys, const int32_t *tids, uint64_t cap, uint8_t *tiles,
                          int32_t *vert, int32_t *bucket, int32_t *pos0, const uint64_t *vkeys, int64_t M,
                          int32_t *nbr, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    const int T = tile_points(d);
    const int64_t grid = (n + T - 1) / T + (M * (d + 1) + T - 1) / T;
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_resolve<D>, dim3((unsigned)grid), dim3(T), 0, s, feat, n, E, grp, ctl,
                                         tkeys, tids, cap - 1, tiles, vert, bucket, pos0, vkeys, M, nbr));
    return hipGetLastError();
}

int64_t scan_scratch_ints(int64_t count)
{
    const int64_t per = (int64_t)kBlock * kScanPer;
    return count <= 0 ? 1 : (count + per - 1) / per;
}

hipError_t launch_exclusive_scan(int32_t *x, int64_t count, int32_t *sums, hipStream_t s)
{
    if (count <= 0)
        return hipSuccess;
    if (count <= kScanOneBlock) {
        hipLaunchKernelGGL(k_scan_lds, dim3(1), dim3(1024), 0, s, x, (int)count);
        return hipGetLastError();
    }
    const int64_t nb = scan_scratch_ints(count);
    hipLaunchKernelGGL(k_scan_blocks, dim3((unsigned)nb), dim3(kBlock), 0, s, x, count, sums);
    hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(1024), 0, s, sums, nb);
    hipLaunchKernelGGL(k_scan_add, dim3((unsigned)nb), dim3(kBlock), 0, s, x, count, sums);
    return hipGetLastError();
}

hipError_t launch_scatter(int d, const float *feat, int64_t n, const Elev &E, const uint8_t *ntiles,
                          const int32_t *vert, const int32_t *start, const int32_t *pos0, int32_t *perm,
                          uint8_t *psort, int32_t *svert, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_scatter<D>, dim3(blocks_for(n)), dim3(kBlock), 0, s, feat, n, E, ntiles,
                                         vert, start, pos0, perm, psort, svert));
    return hipGetLastError();
}

hipError_t launch_sorted_tiles(int d, const int32_t *svert, int64_t n, uint8_t *tiles, float *z0, float *z1,
                               int64_t zelems, uint64_t *tkeys, uint64_t cap, Ctl *ctl, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    if (zelems % 4 != 0 || (zelems > 0 && (!z0 || !z1)))
        return hipErrorInvalidValue;
    if (tkeys && (cap < 2 || (cap & (cap - 1)) != 0 || !ctl))
        return hipErrorInvalidValue;
    const int T = tile_points(d);
    const int64_t pieces = std::max<int64_t>(zelems / 4, tkeys ? (int64_t)(cap / 2) : 0);
    const int64_t grid = (n + T - 1) / T + std::max<int64_t>((pieces + T - 1) / T, tkeys ? 1 : 0);
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_sorted_tiles<D>, dim3((unsigned)grid), dim3(T), 0, s, svert, n, tiles, z0,
                                         z1, zelems, tkeys, cap, ctl));
    return hipGetLastError();
}

hipError_t launch_compact(const uint64_t *tkeys, int32_t *tids, uint64_t *vkeys, int32_t *bucket, uint64_t cap,
                          Ctl *ctl, hipStream_t s)
{
    if (cap >= kCompactWideCap) {
        const uint64_t per_block = (uint64_t)kBlock * 16;
        hipLaunchKernelGGL(k_compact<16>, dim3((unsigned)((cap + per_block - 1) / per_block)), dim3(kBlock), 0, s,
                           tkeys, tids, vkeys, bucket, cap, ctl);
    } else {
        const uint64_t per_block = (uint64_t)kBlock * 4;
        hipLaunchKernelGGL(k_compact<4>, dim3((unsigned)((cap + per_block - 1) / per_block)), dim3(kBlock), 0, s,
                           tkeys, tids, vkeys, bucket, cap, ctl);
    }
    return hipGetLastError();
}


hipError_t launch_export_points(int d, const uint8_t *pts, const int32_t *svert, const int32_t *perm, int64_t n,
                                int32_t *vert, float *bary, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_export_points, dim3(blocks_for(n)), dim3(kBlock), 0, s, d, pts, svert, perm, n, vert, bary);
    return hipGetLastError();
}

hipError_t launch_vertex_groups(const uint64_t *vkeys, int64_t M, const Ctl *ctl, int32_t *vgroup, hipStream_t s)
{
    if (M <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_vertex_groups, dim3(blocks_for(M)), dim3(kBlock), 0, s, vkeys, M, ctl, vgroup);
    return hipGetLastError();
}

hipError_t launch_unpack_keys(int d, const uint64_t *vkeys, int64_t M, const Ctl *ctl, int32_t *keys,
                              hipStream_t s)
{
    if (M <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_unpack_keys, dim3(blocks_for(M)), dim3(kBlock), 0, s, d, vkeys, M, ctl, keys);
    return hipGetLastError();
}



}  // namespace pam

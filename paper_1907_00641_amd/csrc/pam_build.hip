// HIP kernels (gfx950) that build the sparse permutohedral lattice of a
// point set (Joutard et al. 2019, Section 2: operator E of eq. 6 and the
// vertex set its simplices touch):
//   range      per point: rounded remainder-0 quotients -> per-coordinate
//              min/max (sizes the packed key)
//   layout     one thread: bit layout of the 63-bit packed key
//   insert     per point: the d+1 simplex vertex keys into an open-addressing
//              hash table (read before compare-and-swap)
//   compact    per table slot: dense vertex ids, wave-aggregated counter
//   lookup     per point: the d+1 vertex ids
//   neighbours per vertex and direction: ids of key -/+ u_j
#include "pam_device.h"

namespace pam {

__global__ void k_init_ctl(Ctl *ctl)
{
    int t = threadIdx.x;
    if (t < kMaxD) {
        ctl->qmin[t] = INT_MAX;
        ctl->qmax[t] = INT_MIN;
    }
    if (t == 0) {
        ctl->flags = 0;
        ctl->count = 0;
        ctl->nvert = 0;
        ctl->pad = 0;
    }
}

template <int D>
__global__ __launch_bounds__(kBlock) void k_range(const float *__restrict__ feat, int64_t n, Elev E,
                                                  Ctl *ctl)
{
    __shared__ int smin[kBlock / 64][D];
    __shared__ int smax[kBlock / 64][D];
    int qmin[D], qmax[D];
#pragma unroll
    for (int c = 0; c < D; ++c) {
        qmin[c] = INT_MAX;
        qmax[c] = INT_MIN;
    }
    bool bad = false;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kBlock) {
        float x[D + 1];
        const bool ok = elevate<D>(feat + i * D, E, x);
        bad |= !ok;
        // rounded quotients before the remainder-0 fix-up; the fix-up and the
        // vertex offsets move them by at most -2..+1
#pragma unroll
        for (int c = 0; c < D; ++c) {
            const int q = ok ? (int)__builtin_rintf(x[c] * E.inv) : 0;
            qmin[c] = min(qmin[c], q);
            qmax[c] = max(qmax[c], q);
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
    if (__ballot(bad) != 0 && lane == 0)
        atomicOr(&ctl->flags, kFlagBadFeature);
    __syncthreads();
    if (threadIdx.x < D) {
        int c = threadIdx.x, lo = INT_MAX, hi = INT_MIN;
        for (int w = 0; w < kBlock / 64; ++w) {
            lo = min(lo, smin[w][c]);
            hi = max(hi, smax[w][c]);
        }
        if (lo != INT_MAX) {
            atomicMin(&ctl->qmin[c], lo);
            atomicMax(&ctl->qmax[c], hi);
        }
    }
}

__global__ void k_layout(int d, Ctl *ctl)
{
    if (threadIdx.x != 0 || blockIdx.x != 0)
        return;
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
    lay.total_bits = shift;
    if (!fits)
        atomicOr(&ctl->flags, kFlagKeyRange);
}

__global__ void k_fill_u64(uint64_t *p, uint64_t value, int64_t count)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
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
// final key.  Counts new keys in `added`; sets `full` if the whole table
// was probed.
__device__ __forceinline__ void table_insert(uint64_t *tkeys, uint64_t mask, uint64_t key, uint32_t &added,
                                             bool &full)
{
    uint64_t h = mix64(key) & mask;
    for (uint64_t probe = 0; probe <= mask; ++probe) {
        const uint64_t cur = tkeys[h];
        if (cur == key)
            return;
        if (cur == kEmptyKey) {
            const uint64_t prev = atomicCAS((unsigned long long *)&tkeys[h], (unsigned long long)kEmptyKey,
                                            (unsigned long long)key);
            if (prev == kEmptyKey) {
                ++added;
                return;
            }
            if (prev == key)
                return;
        }
        h = (h + 1) & mask;
    }
    full = true;
}

// Dense ids for the occupied slots: each block counts its slots, scans the
// counts, and takes its id range with one counter update.
constexpr int kCompactPer = 16;  // slots per thread

__global__ __launch_bounds__(kBlock) void k_compact(const uint64_t *__restrict__ tkeys, int32_t *tids,
                                                    uint64_t *vkeys, uint64_t cap, Ctl *ctl)
{
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

// nbr is direction-major: nbr[(j * M + m) * 2 + 0] = id(key_m - u_j),
// nbr[(j * M + m) * 2 + 1] = id(key_m + u_j).
__global__ __launch_bounds__(kBlock) void k_neighbours(int d, const uint64_t *__restrict__ vkeys,
                                                       int64_t M, const Ctl *ctl,
                                                       const uint64_t *__restrict__ tkeys,
                                                       const int32_t *__restrict__ tids,
                                                       uint64_t mask, int32_t *__restrict__ nbr)
{
    int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (e >= M * (d + 1))
        return;
    int64_t m = e % M;
    int j = (int)(e / M);
    const KeyLayout &lay = ctl->lay;
    int base[kMaxD], nb[kMaxD];
    unpack_key(vkeys[m], d, lay, base);
    for (int sgn = 0; sgn < 2; ++sgn) {
        int step = sgn ? 1 : -1;
        for (int c = 0; c < d; ++c)
            nb[c] = base[c] + step * ((c == j) ? d : -1);
        uint64_t key;
        int32_t id = -1;
        if (pack_coords(nb, d, lay, &key))
            id = probe_id(tkeys, tids, mask, key);
        nbr[(j * M + m) * 2 + sgn] = id;
    }
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

template <int D>
__global__ void k_export_bary(const float *__restrict__ feat, int64_t n, Elev E, float *bary)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n)
        return;
    Simplex<D> s;
    embed<D>(feat + i * D, E, s);
    float b[D + 1];
    barycentric<D>(s, feat + i * D, E, b);
    for (int k = 0; k <= D; ++k)
        bary[i * (D + 1) + k] = b[k];
}


// The lattice's vertex set, built a tile of points at a time.  Per tile:
// the d+1 vertex keys of every point are deduplicated in an LDS hash
// (64-bit compare-and-swap); only the tile's distinct keys are inserted into
// the global table.  The distinct vertices become the tile's rows, and the
// tile's (point, vertex) contributions are counting-sorted by row (integer
// LDS atomics give each contribution its position within its row); rows are
// cut into segments of at most kSegLen contributions, and the segments are
// counting-sorted by length, longest first, the order in which the splat
// hands them out.  Global ids are attached after compaction by k_resolve.
constexpr int kTileHashBits = 12;
constexpr int kTileHash = 1 << kTileHashBits;
constexpr int kTileProbe = 64;

template <int D>
__global__ __launch_bounds__(tile_points(D)) void k_tile_keys(const float *__restrict__ feat, int64_t n, Elev E,
                                                              Ctl *ctl, uint64_t *tkeys, uint64_t mask,
                                                              uint32_t max_load, uint8_t *__restrict__ tiles)
{
    constexpr int T = tile_points(D);
    constexpr int NC = T * (D + 1);
    static_assert(NC < (1 << 13), "segment start and row must fit their fields");
    __shared__ uint64_t hkey[kTileHash];
    __shared__ int hrow[kTileHash];
    __shared__ uint64_t rkey[NC];  // distinct keys, row order
    __shared__ int cnt[NC + 1];    // per row: count, then first entry
    __shared__ int nsg[NC + 1];    // per row: segment count, then first segment
    __shared__ int hist[kSegLen + 1];
    __shared__ int wsum[T / 64 + 1];
    __shared__ int nrows_s, overflow_s;
    __shared__ uint32_t added_s;
    __shared__ int full_s;
    if (ctl->flags & (kFlagKeyRange | kFlagBadFeature))
        return;
    const KeyLayout lay = ctl->lay;
    const TileRec rec(D);
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, n - base);
    const int nc = nt * (D + 1);
    uint8_t *R = tiles + (size_t)blockIdx.x * rec.bytes;
    uint32_t *hdr = reinterpret_cast<uint32_t *>(R);
    uint64_t *rowkey = reinterpret_cast<uint64_t *>(R + rec.rowkey);
    uint16_t *sfirst = reinterpret_cast<uint16_t *>(R + rec.sfirst);
    uint32_t *seg = reinterpret_cast<uint32_t *>(R + rec.seg);
    uint16_t *order = reinterpret_cast<uint16_t *>(R + rec.order);
    uint16_t *list = reinterpret_cast<uint16_t *>(R + rec.list);
    uint16_t *lrow = reinterpret_cast<uint16_t *>(R + rec.lrow);
    for (int e = t; e < kTileHash; e += T)
        hkey[e] = kEmptyKey;
    for (int e = t; e <= NC; e += T) {
        cnt[e] = 0;
        nsg[e] = 0;
    }
    if (t <= kSegLen)
        hist[t] = 0;
    if (t == 0) {
        nrows_s = 0;
        overflow_s = 0;
        added_s = 0;
        full_s = 0;
    }
    __syncthreads();
    uint64_t key[D + 1];
    int slot[D + 1];
    if (t < nt) {
        Simplex<D> s;
        embed<D>(feat + (base + t) * D, E, s);
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            key[k] = pack_vertex<D>(s, k, lay);
            uint32_t h = (uint32_t)(mix64(key[k]) >> (64 - kTileHashBits));
            int found = -1;
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
            slot[k] = found;
            if (found < 0)
                overflow_s = 1;
        }
    }
    __syncthreads();
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
        for (int r = t; r < nrows_s; r += T)
            table_insert(tkeys, mask, rkey[r], added, full);
    }
    if (added)
        atomicAdd(&added_s, added);
    if (full)
        full_s = 1;
    __syncthreads();
    if (t == 0) {
        if (added_s && atomicAdd(&ctl->count, added_s) + added_s > max_load)
            full_s = 1;
        if (full_s)
            atomicOr(&ctl->flags, kFlagTableFull);
    }
    if (overflow_s) {
        if (t == 0) {
            hdr[0] = 0;
            hdr[1] = kTileOverflow;
            hdr[2] = (uint32_t)nc;
            hdr[3] = 0;
        }
        return;
    }
    const int nrows = nrows_s;
    int row[D + 1], pos[D + 1];
    if (t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            row[k] = hrow[slot[k]];
            pos[k] = atomicAdd(&cnt[row[k]], 1);
            lrow[t * (D + 1) + k] = (uint16_t)row[k];
        }
    }
    for (int r = t; r < nrows; r += T)
        rowkey[r] = rkey[r];
    __syncthreads();
    for (int r = t; r < nrows; r += T)
        nsg[r] = (cnt[r] + kSegLen - 1) / kSegLen;
    __syncthreads();
    block_exclusive_scan(cnt, nrows, wsum);                   // cnt[r]: first entry of row r
    const int nseg = block_exclusive_scan(nsg, nrows, wsum);  // nsg[r]: first segment of row r
    if (t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k)
            list[cnt[row[k]] + pos[k]] = (uint16_t)((t << 5) | k);
    }
    // segments in row order, and a histogram of their lengths
    for (int r = t; r < nrows; r += T) {
        const int e0 = cnt[r], e1 = (r + 1 < nrows) ? cnt[r + 1] : nc;
        sfirst[r] = (uint16_t)nsg[r];
        for (int j = 0, e = e0; e < e1; ++j, e += kSegLen) {
            const int len = min(kSegLen, e1 - e);
            seg[nsg[r] + j] = (uint32_t)e | ((uint32_t)len << 13) | ((uint32_t)r << 18);
            atomicAdd(&hist[kSegLen - len], 1);  // bucket 0 = longest
        }
    }
    __syncthreads();
    if (t == 0) {
        int run = 0;  // bucket starts, then used as cursors
        for (int b = 0; b <= kSegLen; ++b) {
            const int v = hist[b];
            hist[b] = run;
            run += v;
        }
        sfirst[nrows] = (uint16_t)nseg;
        hdr[0] = (uint32_t)nrows;
        hdr[1] = 0;
        hdr[2] = (uint32_t)nc;
        hdr[3] = (uint32_t)nseg;
    }
    __syncthreads();
    // work order: longest segments first
    for (int r = t; r < nrows; r += T) {
        const int e0 = cnt[r], e1 = (r + 1 < nrows) ? cnt[r + 1] : nc;
        for (int j = 0, e = e0; e < e1; ++j, e += kSegLen) {
            const int len = min(kSegLen, e1 - e);
            order[atomicAdd(&hist[kSegLen - len], 1)] = (uint16_t)(nsg[r] + j);
        }
    }
}

// Global ids for the tile's rows (one table lookup per distinct vertex),
// then the per-point vertex ids.  Tiles that overflowed their LDS table look
// up every key of every point.
template <int D>
__global__ __launch_bounds__(tile_points(D)) void k_resolve(const float *__restrict__ feat, int64_t n, Elev E,
                                                            const Ctl *ctl, const uint64_t *__restrict__ tkeys,
                                                            const int32_t *__restrict__ tids, uint64_t mask,
                                                            uint8_t *__restrict__ tiles, int32_t *__restrict__ vert)
{
    constexpr int T = tile_points(D);
    constexpr int NC = T * (D + 1);
    __shared__ int rid[NC];
    const TileRec rec(D);
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * T;
    const int nt = (int)min((int64_t)T, n - base);
    uint8_t *R = tiles + (size_t)blockIdx.x * rec.bytes;
    const uint32_t *hdr = reinterpret_cast<const uint32_t *>(R);
    int32_t *rowid = reinterpret_cast<int32_t *>(R + rec.rowid);
    const uint64_t *rowkey = reinterpret_cast<const uint64_t *>(R + rec.rowkey);
    const uint16_t *lrow = reinterpret_cast<const uint16_t *>(R + rec.lrow);
    const int nrows = (int)hdr[0], nc = (int)hdr[2];
    if (hdr[1] & kTileOverflow) {
        if (t < nt) {
            const KeyLayout lay = ctl->lay;
            Simplex<D> s;
            embed<D>(feat + (base + t) * D, E, s);
#pragma unroll
            for (int k = 0; k <= D; ++k)
                vert[(base + t) * (D + 1) + k] = probe_id(tkeys, tids, mask, pack_vertex<D>(s, k, lay));
        }
        return;
    }
    for (int r = t; r < nrows; r += T) {
        const int32_t id = probe_id(tkeys, tids, mask, rowkey[r]);
        rowid[r] = id;
        rid[r] = id;
    }
    __syncthreads();
    int32_t *v = vert + base * (D + 1);
    for (int e = t; e < nc; e += T)
        v[e] = rid[lrow[e]];
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

hipError_t launch_init_ctl(Ctl *ctl, hipStream_t s)
{
    hipLaunchKernelGGL(k_init_ctl, dim3(1), dim3(64), 0, s, ctl);
    return hipGetLastError();
}

hipError_t launch_range(int d, const float *feat, int64_t n, const Elev &E, Ctl *ctl, hipStream_t s)
{
    unsigned grid = blocks_for(n);
    grid = grid > 2048 ? 2048 : (grid == 0 ? 1 : grid);
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_range<D>, dim3(grid), dim3(kBlock), 0, s, feat, n, E, ctl));
    return hipGetLastError();
}

hipError_t launch_layout(int d, Ctl *ctl, hipStream_t s)
{
    hipLaunchKernelGGL(k_layout, dim3(1), dim3(64), 0, s, d, ctl);
    return hipGetLastError();
}

hipError_t launch_fill_u64(uint64_t *p, uint64_t value, int64_t count, hipStream_t s)
{
    if (count <= 0)
        return hipSuccess;
    unsigned grid = blocks_for(count);
    grid = grid > 4096 ? 4096 : grid;
    hipLaunchKernelGGL(k_fill_u64, dim3(grid), dim3(kBlock), 0, s, p, value, count);
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

hipError_t launch_tile_keys(int d, const float *feat, int64_t n, const Elev &E, Ctl *ctl, uint64_t *tkeys,
                            uint64_t cap, uint32_t max_load, uint8_t *tiles, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    const unsigned grid = (unsigned)((n + tile_points(d) - 1) / tile_points(d));
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_tile_keys<D>, dim3(grid), dim3(tile_points(d)), 0, s, feat, n, E, ctl,
                                         tkeys, cap - 1, max_load, tiles));
    return hipGetLastError();
}

hipError_t launch_resolve(int d, const float *feat, int64_t n, const Elev &E, const Ctl *ctl,
                          const uint64_t *tkeys, const int32_t *tids, uint64_t cap, uint8_t *tiles, int32_t *vert,
                          hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    const unsigned grid = (unsigned)((n + tile_points(d) - 1) / tile_points(d));
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_resolve<D>, dim3(grid), dim3(tile_points(d)), 0, s, feat, n, E, ctl,
                                         tkeys, tids, cap - 1, tiles, vert));
    return hipGetLastError();
}

hipError_t launch_compact(const uint64_t *tkeys, int32_t *tids, uint64_t *vkeys, uint64_t cap,
                          Ctl *ctl, hipStream_t s)
{
    const uint64_t per_block = (uint64_t)kBlock * kCompactPer;
    hipLaunchKernelGGL(k_compact, dim3((unsigned)((cap + per_block - 1) / per_block)), dim3(kBlock), 0, s, tkeys,
                       tids, vkeys, cap, ctl);
    return hipGetLastError();
}

hipError_t launch_neighbours(int d, const uint64_t *vkeys, int64_t M, const Ctl *ctl,
                             const uint64_t *tkeys, const int32_t *tids, uint64_t cap,
                             int32_t *nbr, hipStream_t s)
{
    if (M <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_neighbours, dim3(blocks_for(M * (d + 1))), dim3(kBlock), 0, s, d, vkeys, M,
                       ctl, tkeys, tids, cap - 1, nbr);
    return hipGetLastError();
}

hipError_t launch_export_bary(int d, const float *feat, int64_t n, const Elev &E, float *bary,
                              hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_export_bary<D>, dim3(blocks_for(n)), dim3(kBlock), 0, s, feat,
                                         n, E, bary));
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

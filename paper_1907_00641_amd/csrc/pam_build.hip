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
        Simplex<D> s;
        bad |= !embed<D>(feat + i * D, E, s);
        // rounded quotients before the fix-up; the fix-up and the vertex
        // offsets move them by at most -2..+1
#pragma unroll
        for (int c = 0; c < D; ++c) {
            int q = (int)__builtin_rintf(s.x[c] * E.inv);
            q = __builtin_fabsf(s.x[c]) <= 16777216.0f ? q : 0;
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

template <int D>
__global__ __launch_bounds__(kBlock) void k_insert(const float *__restrict__ feat, int64_t n, Elev E,
                                                   Ctl *ctl, uint64_t *tkeys, uint64_t mask,
                                                   uint32_t max_load)
{
    if (ctl->flags & (kFlagKeyRange | kFlagBadFeature))
        return;
    int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n)
        return;
    const KeyLayout lay = ctl->lay;
    Simplex<D> s;
    embed<D>(feat + i * D, E, s);
    for (int k = 0; k <= D; ++k) {
        uint64_t key = pack_vertex<D>(s, k, lay);
        uint64_t h = mix64(key) & mask;
        bool done = false;
        for (uint64_t probe = 0; probe <= mask; ++probe) {
            uint64_t cur = __hip_atomic_load(&tkeys[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (cur == key) {
                done = true;
                break;
            }
            if (cur == kEmptyKey) {
                uint64_t prev = atomicCAS((unsigned long long *)&tkeys[h], (unsigned long long)kEmptyKey,
                                          (unsigned long long)key);
                if (prev == kEmptyKey) {
                    if (atomicAdd(&ctl->count, 1u) >= max_load)
                        atomicOr(&ctl->flags, kFlagTableFull);
                    done = true;
                    break;
                }
                if (prev == key) {
                    done = true;
                    break;
                }
            }
            h = (h + 1) & mask;
        }
        if (!done) {
            atomicOr(&ctl->flags, kFlagTableFull);
            return;
        }
    }
}

// Dense ids for the occupied slots: one counter update per wave.
__global__ __launch_bounds__(kBlock) void k_compact(const uint64_t *__restrict__ tkeys, int32_t *tids,
                                                    uint64_t *vkeys, uint64_t cap, Ctl *ctl)
{
    uint64_t s = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    uint64_t key = s < cap ? tkeys[s] : kEmptyKey;
    bool occ = key != kEmptyKey;
    unsigned long long ballot = __ballot(occ);
    if (ballot == 0)
        return;
    int lane = threadIdx.x & 63;
    int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(ballot >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)ballot, 0));
    int leader = __ffsll((long long)ballot) - 1;
    uint32_t base = 0;
    if (lane == leader)
        base = atomicAdd(&ctl->nvert, (uint32_t)__popcll(ballot));
    base = __builtin_amdgcn_readlane(base, leader);  // leader is wave-uniform
    if (occ) {
        uint32_t id = base + (uint32_t)below;
        tids[s] = (int32_t)id;
        vkeys[id] = key;
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

template <int D>
__global__ __launch_bounds__(kBlock) void k_lookup(const float *__restrict__ feat, int64_t n, Elev E,
                                                   const Ctl *ctl, const uint64_t *__restrict__ tkeys,
                                                   const int32_t *__restrict__ tids, uint64_t mask,
                                                   int32_t *__restrict__ vert)
{
    int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n)
        return;
    const KeyLayout lay = ctl->lay;
    Simplex<D> s;
    embed<D>(feat + i * D, E, s);
#pragma unroll
    for (int k = 0; k <= D; ++k)
        vert[i * (D + 1) + k] = probe_id(tkeys, tids, mask, pack_vertex<D>(s, k, lay));
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


// Per-tile view of the lattice for the splat kernel (layout in TileRec):
// the tile's distinct vertices become dense rows (LDS hash, compare-and-swap
// on integer keys); the tile's (point, vertex) contributions are
// counting-sorted by row (integer LDS atomics give each contribution its
// position within its row); rows are cut into segments of at most kSegLen
// contributions, and the segments are counting-sorted by length, longest
// first, which is the order in which the splat hands them out.
constexpr int kTileHashBits = 12;
constexpr int kTileHash = 1 << kTileHashBits;
constexpr int kTileProbe = 64;

template <int D>
__global__ __launch_bounds__(tile_points(D)) void k_tiles(const int32_t *__restrict__ vert, int64_t n,
                                                          uint8_t *__restrict__ tiles)
{
    constexpr int T = tile_points(D);
    constexpr int NC = T * (D + 1);
    static_assert(NC < (1 << 13), "segment start and row must fit their fields");
    __shared__ int hkey[kTileHash];
    __shared__ int hrow[kTileHash];
    __shared__ int cnt[NC + 1];   // per row: count, then first entry
    __shared__ int nsg[NC + 1];   // per row: segment count, then first segment
    __shared__ int hist[kSegLen + 1];
    __shared__ int wsum[T / 64 + 1];
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
    for (int e = t; e < kTileHash; e += T)
        hkey[e] = -1;
    for (int e = t; e <= NC; e += T) {
        cnt[e] = 0;
        nsg[e] = 0;
    }
    if (t <= kSegLen)
        hist[t] = 0;
    if (t == 0) {
        nrows_s = 0;
        overflow_s = 0;
    }
    __syncthreads();
    int slot[D + 1];
    if (t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            const int m = vert[(base + t) * (D + 1) + k];
            uint32_t h = ((uint32_t)m * 2654435761u) >> (32 - kTileHashBits);
            int found = -1;
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
            slot[k] = found;
            if (found < 0)
                overflow_s = 1;
        }
    }
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
    int row[D + 1], pos[D + 1];
    if (t < nt) {
#pragma unroll
        for (int k = 0; k <= D; ++k) {
            row[k] = hrow[slot[k]];
            pos[k] = atomicAdd(&cnt[row[k]], 1);
        }
    }
    __syncthreads();
    const int nrows = nrows_s;
    for (int r = t; r < nrows; r += T)
        nsg[r] = (cnt[r] + kSegLen - 1) / kSegLen;
    __syncthreads();
    block_exclusive_scan(cnt, nrows, wsum);           // cnt[r]: first entry of row r
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

hipError_t launch_insert(int d, const float *feat, int64_t n, const Elev &E, Ctl *ctl,
                         uint64_t *tkeys, uint64_t cap, uint32_t max_load, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_insert<D>, dim3(blocks_for(n)), dim3(kBlock), 0, s, feat, n,
                                         E, ctl, tkeys, cap - 1, max_load));
    return hipGetLastError();
}

hipError_t launch_compact(const uint64_t *tkeys, int32_t *tids, uint64_t *vkeys, uint64_t cap,
                          Ctl *ctl, hipStream_t s)
{
    hipLaunchKernelGGL(k_compact, dim3(blocks_for((int64_t)cap)), dim3(kBlock), 0, s, tkeys, tids,
                       vkeys, cap, ctl);
    return hipGetLastError();
}

hipError_t launch_lookup(int d, const float *feat, int64_t n, const Elev &E, const Ctl *ctl,
                         const uint64_t *tkeys, const int32_t *tids, uint64_t cap, int32_t *vert,
                         hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_lookup<D>, dim3(blocks_for(n)), dim3(kBlock), 0, s, feat, n,
                                         E, ctl, tkeys, tids, cap - 1, vert));
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

hipError_t launch_tiles(int d, const int32_t *vert, int64_t n, uint8_t *tiles, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    const unsigned grid = (unsigned)((n + tile_points(d) - 1) / tile_points(d));
    PAM_DISPATCH_D(d, hipLaunchKernelGGL(k_tiles<D>, dim3(grid), dim3(tile_points(d)), 0, s, vert, n, tiles));
    return hipGetLastError();
}

}  // namespace pam

// Stable counting sort of each (batch, head, round) segment by bucket, then
// position (Reformer, Sec. 2 "LSH attention": the permutation i -> s_i;
// App. A: one permutation s^(r) per round), and the row gather into sorted
// order.
//
// A segment of L positions is cut into tiles of kTile positions.
//   1. hist:    per (tile, round) bucket counts, LDS atomics.
//   2. scan:    exclusive scan of the counts in (bucket, tile) order gives
//               every (bucket, tile) pair its first output slot, and the
//               bucket start offsets.
//   3. scatter: each wave ranks its quarter of a tile in position order; the
//               rank of a position among equal buckets of its 64-lane group
//               comes from ballots over the bucket bits (peer mask + popcount),
//               so equal keys keep their position order (stable).
#include "common.h"
#include "launch.h"

#include <mutex>

namespace lsh {
namespace {

constexpr int kTile = 4096;
constexpr int kSortWaves = 4;
constexpr int kPerWave = kTile / kSortWaves;
constexpr int kHistLdsInts = 8192;

__device__ __forceinline__ int clamp_bucket(int b, int n_b) { return min(max(b, 0), n_b - 1); }

// A tile is one workgroup (one per CU at the usual sizes), so it runs 16
// waves to keep enough loads in flight.
constexpr int kHistThreads = 1024;

__global__ __launch_bounds__(kHistThreads) void sort_hist_kernel(const int32_t* __restrict__ buckets, int L,
                                                        int n_r, int n_b, int rounds_per_group,
                                                        int n_tiles, int32_t* __restrict__ counts) {
    extern __shared__ int hist[];
    const int tile = blockIdx.x;
    const int64_t bh = blockIdx.y;
    const int r0 = blockIdx.z * rounds_per_group;
    const int nr = min(rounds_per_group, n_r - r0);
    for (int i = threadIdx.x; i < nr * n_b; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    const int p0 = tile * kTile, p1 = min(L, p0 + kTile);
    for (int p = p0 + threadIdx.x; p < p1; p += blockDim.x) {
        const int32_t* row = buckets + (bh * L + p) * n_r + r0;
        for (int r = 0; r < nr; ++r) atomicAdd(&hist[r * n_b + clamp_bucket(row[r], n_b)], 1);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nr * n_b; i += blockDim.x) {
        const int r = r0 + i / n_b, b = i % n_b;
        counts[((bh * n_r + r) * n_b + b) * n_tiles + tile] = hist[i];
    }
}

// Each thread owns a contiguous run of the segment's (bucket, tile) counts
// and holds it in registers (16-byte loads, all in flight together), so the
// scan costs one round trip to memory instead of one per count.
constexpr int kScanPerThread = 64;  // counts per thread held in registers

__global__ __launch_bounds__(256) void sort_scan_kernel(int32_t* __restrict__ counts, int L,
                                                        int n_b, int n_tiles,
                                                        int32_t* __restrict__ bucket_start) {
    __shared__ int part[256];
    const int64_t seg = blockIdx.x;
    const int64_t E = (int64_t)n_b * n_tiles;
    int32_t* c = counts + seg * E;
    int32_t* bs = bucket_start + seg * (n_b + 1);
    const int64_t per = (E + 255) / 256;
    const int64_t lo = min(E, threadIdx.x * per), hi = min(E, lo + per);
    int s = 0;
    if (per <= kScanPerThread && (E & 3) == 0 && (per & 3) == 0) {
        int v[kScanPerThread];
#pragma unroll
        for (int k = 0; k < kScanPerThread; k += 4) {
            const int64_t e = lo + k;
            int4 x = make_int4(0, 0, 0, 0);
            if (k < per && e < hi) x = *reinterpret_cast<const int4*>(c + e);
            v[k] = x.x;
            v[k + 1] = x.y;
            v[k + 2] = x.z;
            v[k + 3] = x.w;
        }
#pragma unroll
        for (int k = 0; k < kScanPerThread; ++k) s += v[k];
        part[threadIdx.x] = s;
        __syncthreads();
        for (int o = 1; o < 256; o <<= 1) {
            const int x = (int)threadIdx.x >= o ? part[threadIdx.x - o] : 0;
            __syncthreads();
            part[threadIdx.x] += x;
            __syncthreads();
        }
        int run = part[threadIdx.x] - s;
        // (bucket, tile) of element lo, stepped along the run: a bucket's
        // start is the exclusive prefix at its tile 0
        int bucket = (int)(lo / n_tiles), t = (int)(lo % n_tiles);
#pragma unroll
        for (int k = 0; k < kScanPerThread; k += 4) {
            const int64_t e = lo + k;
            if (k < per && e < hi) {
                int4 x;
                x.x = run;
                x.y = run + v[k];
                x.z = x.y + v[k + 1];
                x.w = x.z + v[k + 2];
                *reinterpret_cast<int4*>(c + e) = x;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (t == 0) bs[bucket] = u == 0 ? x.x : (u == 1 ? x.y : (u == 2 ? x.z : x.w));
                    if (++t == n_tiles) {
                        t = 0;
                        ++bucket;
                    }
                }
                run = x.w + v[k + 3];
            }
        }
    } else {
        for (int64_t e = lo; e < hi; ++e) s += c[e];
        part[threadIdx.x] = s;
        __syncthreads();
        // Hillis-Steele inclusive scan over 256 partial sums.
        for (int o = 1; o < 256; o <<= 1) {
            const int x = (int)threadIdx.x >= o ? part[threadIdx.x - o] : 0;
            __syncthreads();
            part[threadIdx.x] += x;
            __syncthreads();
        }
        int run = part[threadIdx.x] - s;
        int bucket = (int)(lo / n_tiles), t = (int)(lo % n_tiles);
        for (int64_t e = lo; e < hi; ++e) {
            const int v = c[e];
            c[e] = run;
            if (t == 0) bs[bucket] = run;
            if (++t == n_tiles) {
                t = 0;
                ++bucket;
            }
            run += v;
        }
    }
    if (threadIdx.x == 0) bs[n_b] = L;
}

__global__ __launch_bounds__(256) void sort_scatter_kernel(const int32_t* __restrict__ buckets,
                                                           const int32_t* __restrict__ offsets,
                                                           int L, int n_r, int n_b, int n_bits,
                                                           int n_tiles, int32_t* __restrict__ perm,
                                                           int32_t* __restrict__ undo) {
    extern __shared__ int base[];  // [kSortWaves][n_b]
    // Workgroup b of the launch runs on XCD b % 8 (round-robin dispatch).
    // Each XCD is given a contiguous run of (segment, tile) items, so the
    // tiles of a segment write their scattered 4-byte slots into the same
    // XCD's L2, which merges them into whole lines before they reach HBM,
    // and the rounds of one (batch, head) read its bucket ids through one L2.
    const int64_t nblk = (int64_t)gridDim.x * gridDim.y;
    const int64_t bid = blockIdx.x + (int64_t)blockIdx.y * gridDim.x;
    const int64_t item = nblk % 8 == 0 ? (bid % 8) * (nblk / 8) + bid / 8 : bid;
    const int tile = (int)(item % gridDim.x);
    const int64_t seg = item / gridDim.x;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int* wbase = base + wave * n_b;

    for (int i = threadIdx.x; i < kSortWaves * n_b; i += blockDim.x) base[i] = 0;
    const int p0 = tile * kTile + wave * kPerWave;
    const int p1 = min(L, p0 + kPerWave);
    // this lane's ids, all loads in flight at once (kPerWave / 64 per lane);
    // positions past the segment load a valid id that is never used, so the
    // loads are unconditional and not each followed by its own wait
    constexpr int kIter = kPerWave / 64;
    int ids[kIter];
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
        const int pos = min(max(p0 + 64 * it + lane, 0), max(p1 - 1, 0));
        ids[it] = buckets[(bh * L + pos) * n_r + r];
    }
#pragma unroll
    for (int it = 0; it < kIter; ++it) ids[it] = clamp_bucket(ids[it], n_b);
    __syncthreads();
#pragma unroll
    for (int it = 0; it < kIter; ++it)
        if (p0 + 64 * it + lane < p1) atomicAdd(&wbase[ids[it]], 1);
    __syncthreads();
    // Per-wave starting slot of every bucket: the tile's offset plus the counts
    // of the earlier waves of this tile.
    for (int b = threadIdx.x; b < n_b; b += blockDim.x) {
        int off = offsets[(seg * n_b + b) * n_tiles + tile];
        for (int w = 0; w < kSortWaves; ++w) {
            const int cnt = base[w * n_b + b];
            base[w * n_b + b] = off;
            off += cnt;
        }
    }
    __syncthreads();

    int32_t* pseg = perm + seg * L;
    int32_t* useg = undo + seg * L;
    const uint64_t lt_mask = (1ull << lane) - 1ull;
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
        const int pos = p0 + 64 * it + lane;
        const bool active = pos < p1;
        const int b = ids[it];
        uint64_t peers = __ballot(active);
        for (int bit = 0; bit < n_bits; ++bit) {
            const bool set = (b >> bit) & 1;
            const uint64_t m = __ballot(set && active);
            peers &= set ? m : ~m;
        }
        const int before = __popcll(peers & lt_mask);
        const int start = wbase[b];
        if (active) {
            const int slot = start + before;
            pseg[slot] = pos;
            useg[pos] = slot;
            if ((peers >> lane) == 1ull) wbase[b] = start + __popcll(peers);
        }
    }
}

// dst[seg][s] = src[bh][perm[seg][s]] for rows of `row_bytes`, 16 B per thread.
__global__ __launch_bounds__(256) void gather_kernel(const char* __restrict__ src,
                                                     const int32_t* __restrict__ perm, int L,
                                                     int n_r, int parts, int64_t total,
                                                     char* __restrict__ dst) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        const int part = (int)(idx % parts);
        const int64_t out_row = idx / parts;  // (seg, s)
        const int64_t seg = out_row / L;
        const int64_t bh = seg / n_r;
        const int64_t in_row = bh * L + min(max(perm[out_row], 0), L - 1);
        *reinterpret_cast<u32x4*>(dst + (out_row * parts + part) * 16) =
            *reinterpret_cast<const u32x4*>(src + (in_row * parts + part) * 16);
    }
}

}  // namespace

int sort_tile_positions(int L) { return kTile; }

// Scratch of lsh_sort_permute_static: a fixed device array in this code
// object, so that call allocates nothing.  Host code never passes `scratch`
// itself to a kernel (on the host it names a stand-in, not device memory):
// its device address is looked up once per device with that device current,
// and that address is what the kernels receive.
static __device__ __align__(256) char scratch[kSortScratchBytes];

namespace {
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t sort_static_scratch(void** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

size_t sort_workspace_bytes(int64_t BH, int L, int n_rounds, int n_buckets) {
    const int64_t n_tiles = (L + kTile - 1) / kTile;
    return align256((size_t)(BH * n_rounds * n_buckets * n_tiles) * sizeof(int32_t));
}

hipError_t launch_sort(int64_t BH, int L, int n_rounds, int n_buckets, const int32_t* buckets,
                       int32_t* perm, int32_t* undo, int32_t* bucket_start, void* workspace,
                       hipStream_t stream) {
    if (BH == 0 || L == 0) return hipSuccess;
    const int n_tiles = (L + kTile - 1) / kTile;
    int32_t* counts = static_cast<int32_t*>(workspace);
    const int rpg = std::max(1, std::min(n_rounds, kHistLdsInts / n_buckets));
    const int groups = (n_rounds + rpg - 1) / rpg;
    int n_bits = 0;
    while ((1 << n_bits) < n_buckets) ++n_bits;

    sort_hist_kernel<<<dim3(n_tiles, (unsigned)BH, groups), kHistThreads, rpg * n_buckets * sizeof(int), stream>>>(
        buckets, L, n_rounds, n_buckets, rpg, n_tiles, counts);
    sort_scan_kernel<<<(unsigned)(BH * n_rounds), 256, 0, stream>>>(counts, L, n_buckets, n_tiles,
                                                                    bucket_start);
    sort_scatter_kernel<<<dim3(n_tiles, (unsigned)(BH * n_rounds)), 256,
                          kSortWaves * n_buckets * sizeof(int), stream>>>(
        buckets, counts, L, n_rounds, n_buckets, n_bits, n_tiles, perm, undo);
    return hipGetLastError();
}

hipError_t launch_gather(int64_t BH, int L, int n_rounds, bool f32, const void* src,
                         const int32_t* perm, void* dst, hipStream_t stream) {
    const int parts = (f32 ? 4 : 2) * kHeadDim / 16;
    const int64_t total = BH * n_rounds * (int64_t)L * parts;
    if (total == 0) return hipSuccess;
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
    gather_kernel<<<(unsigned)blocks, 256, 0, stream>>>(static_cast<const char*>(src), perm, L,
                                                         n_rounds, parts, total,
                                                         static_cast<char*>(dst));
    return hipGetLastError();
}

}  // namespace lsh

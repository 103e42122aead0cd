// Stable counting sort of each (batch, head, round) segment by bucket, then
// position (Reformer, Sec. 2 "LSH attention": the permutation i -> s_i;
// App. A: one permutation s^(r) per round), and the row gather into sorted
// order.
//
// A segment of L positions is cut into tiles of kTile positions.
//   1. hist:    per (tile, round) bucket counts, LDS atomics; stored
//               [segment][tile][bucket].  With a workspace it also writes
//               the ids once more, one round after another as 16-bit values
//               ([segment][position]), so that the scatter reads them
//               coalesced instead of one 4-byte word in every n_r.
//   2. scan:    exclusive scan of the counts in (bucket, tile) order gives
//               every (bucket, tile) pair its first output slot, and the
//               bucket start offsets.
//   3. scatter: each of eight waves ranks its eighth of a tile in position
//               order; the rank of a position among equal buckets of its
//               64-lane group is the count of lower lanes with the same
//               bucket (their lane mask from an LDS table on the id's low
//               bits and one ballot per high bit), so equal keys keep their
//               position order (stable).  undo is written in position
//               order; perm is first put in the tile's sorted order in LDS
//               and written from there, run by run.
#include "common.h"
#include "launch.h"

#include <mutex>

namespace lsh {
namespace {

constexpr int kTile = 4096;
constexpr int kSortWaves = 8;
constexpr int kPerWave = kTile / kSortWaves;
constexpr int kHistLdsInts = 8192;

__device__ __forceinline__ int clamp_bucket(int b, int n_b) { return min(max(b, 0), n_b - 1); }

// A tile is one workgroup (one per CU at the usual sizes), so it runs 16
// waves to keep enough loads in flight.
constexpr int kHistThreads = 1024;

constexpr int kHistRows = kTile / kHistThreads;  // positions per thread

// LDS of the histogram: the counts of its rounds (rounded up to 16 bytes),
// then, when it writes the 16-bit id copy, the tile's ids of those rounds.
__host__ __device__ inline int hist_words(int rounds, int n_b) { return (rounds * n_b + 3) & ~3; }
size_t hist_lds_bytes(int rounds, int n_b, bool ids16) {
    return (size_t)hist_words(rounds, n_b) * sizeof(int) + (ids16 ? (size_t)rounds * kTile * sizeof(uint16_t) : 0);
}
constexpr int kHistMaxRounds = 16;

__global__ __launch_bounds__(kHistThreads) void sort_hist_kernel(const int32_t* __restrict__ buckets, int L,
                                                        int n_r, int n_b, int rounds_per_group,
                                                        int n_tiles, int32_t* __restrict__ counts,
                                                        uint16_t* __restrict__ ids16) {
    extern __shared__ int hist[];
    const int tile = blockIdx.x;
    const int64_t bh = blockIdx.y;
    const int r0 = blockIdx.z * rounds_per_group;
    const int nr = min(rounds_per_group, n_r - r0);
    for (int i = threadIdx.x; i < nr * n_b; i += blockDim.x) hist[i] = 0;
    const int p0 = tile * kTile, p1 = min(L, p0 + kTile);
    // every id of the thread's positions loaded before the first atomic
    // (16-byte loads when a position's ids of this group are aligned)
    int ids[kHistRows][kHistMaxRounds];
    const bool vec = (n_r % 4) == 0 && (r0 % 4) == 0;
#pragma unroll
    for (int k = 0; k < kHistRows; ++k) {
        const int p = min(p0 + (int)threadIdx.x + kHistThreads * k, p1 - 1);  // past the tile: reloads a valid row
        const int32_t* row = buckets + (bh * L + p) * n_r + r0;
        if (vec) {
#pragma unroll
            for (int c4 = 0; c4 < kHistMaxRounds / 4; ++c4)
                if (4 * c4 < nr) {
                    const int4 x = *reinterpret_cast<const int4*>(row + 4 * c4);
                    ids[k][4 * c4] = x.x;
                    ids[k][4 * c4 + 1] = x.y;
                    ids[k][4 * c4 + 2] = x.z;
                    ids[k][4 * c4 + 3] = x.w;
                }
        } else {
#pragma unroll
            for (int r = 0; r < kHistMaxRounds; ++r)
                if (r < nr) ids[k][r] = row[r];
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kHistRows; ++k)
        if (p0 + (int)threadIdx.x + kHistThreads * k < p1) {
#pragma unroll
            for (int r = 0; r < kHistMaxRounds; ++r)
                if (r < nr) atomicAdd(&hist[r * n_b + clamp_bucket(ids[k][r], n_b)], 1);
        }
    // The ids again, one round after another as 16-bit values, for the
    // scatter's coalesced reads: transposed in LDS, then written 16 bytes
    // per lane.
    uint16_t* t16 = reinterpret_cast<uint16_t*>(hist + hist_words(rounds_per_group, n_b));
    if (ids16) {
#pragma unroll
        for (int k = 0; k < kHistRows; ++k) {
            const int u = (int)threadIdx.x + kHistThreads * k;
#pragma unroll
            for (int r = 0; r < kHistMaxRounds; ++r)
                if (r < nr) t16[r * kTile + u] = (uint16_t)clamp_bucket(ids[k][r], n_b);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nr * n_b; i += blockDim.x) {
        const int r = r0 + i / n_b, b = i % n_b;
        counts[((bh * n_r + r) * n_tiles + tile) * n_b + b] = hist[i];
    }
    if (ids16) {
        constexpr int kPieces = kTile / 8;  // 16-byte pieces of a round's row
        const bool aligned = (L % 8) == 0;
        for (int i = threadIdx.x; i < nr * kPieces; i += blockDim.x) {
            const int r = i / kPieces, u = 8 * (i % kPieces);
            uint16_t* dst = ids16 + (bh * n_r + r0 + r) * L + p0 + u;
            if (aligned && p0 + u + 8 <= p1) {
                *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(t16 + r * kTile + u);
            } else {
                for (int e = 0; e < 8 && p0 + u + e < p1; ++e) dst[e] = t16[r * kTile + u + e];
            }
        }
    }
}

// Counts of a segment are [tile][bucket]; the scan replaces every count by
// its first output slot in (bucket, tile) order and writes the bucket start
// offsets.  Up to 16 tiles (L <= 65536) and 1024 buckets: one thread per
// bucket holds its counts for every tile in registers (all loads in flight
// together), the threads' sums are scanned across each wave with shuffles
// and across the waves in LDS, so the scan costs one round trip to memory.
constexpr int kScanTiles = 16;
constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void sort_scan_kernel(int32_t* __restrict__ counts, int L, int n_b,
                                                                 int n_tiles, int32_t* __restrict__ bucket_start) {
    __shared__ int wsum[kScanThreads / 64];
    const int64_t seg = blockIdx.x;
    int32_t* c = counts + seg * (int64_t)n_b * n_tiles;
    int32_t* bs = bucket_start + seg * (n_b + 1);
    const int b = threadIdx.x, lane = b & 63, wave = b >> 6;
    const bool owner = b < n_b;
    const int bl = min(b, n_b - 1);
    int v[kScanTiles];
#pragma unroll
    for (int t = 0; t < kScanTiles; ++t) v[t] = c[(int64_t)min(t, n_tiles - 1) * n_b + bl];
    int sum = 0;
#pragma unroll
    for (int t = 0; t < kScanTiles; ++t) {
        if (t >= n_tiles || !owner) v[t] = 0;
        sum += v[t];
    }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int run = incl - sum;
    for (int w = 0; w < wave; ++w) run += wsum[w];
    if (owner) {
        bs[b] = run;
#pragma unroll
        for (int t = 0; t < kScanTiles; ++t)
            if (t < n_tiles) {
                c[(int64_t)t * n_b + b] = run;
                run += v[t];
            }
    }
    if (b == 0) bs[n_b] = L;
}

// The same for any number of tiles and buckets: each of 256 threads owns a
// run of consecutive buckets and walks their tiles twice.
__global__ __launch_bounds__(256) void sort_scan_any_kernel(int32_t* __restrict__ counts, int L, int n_b,
                                                            int n_tiles, int32_t* __restrict__ bucket_start) {
    __shared__ int part[256];
    const int64_t seg = blockIdx.x;
    int32_t* c = counts + seg * (int64_t)n_b * n_tiles;
    int32_t* bs = bucket_start + seg * (n_b + 1);
    const int per = (n_b + 255) / 256;
    const int b0 = min(n_b, (int)threadIdx.x * per), b1 = min(n_b, b0 + per);
    int s = 0;
    for (int b = b0; b < b1; ++b)
        for (int t = 0; t < n_tiles; ++t) s += c[(int64_t)t * n_b + b];
    // exclusive prefix of the threads' sums
    part[threadIdx.x] = s;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {
        const int x = (int)threadIdx.x >= o ? part[threadIdx.x - o] : 0;
        __syncthreads();
        part[threadIdx.x] += x;
        __syncthreads();
    }
    int run = part[threadIdx.x] - s;
    for (int b = b0; b < b1; ++b) {
        bs[b] = run;
        for (int t = 0; t < n_tiles; ++t) {
            const int x = c[(int64_t)t * n_b + b];
            c[(int64_t)t * n_b + b] = run;
            run += x;
        }
    }
    if (threadIdx.x == 0) bs[n_b] = L;
}

// LDS of the scatter: per-wave next local slot of every bucket as 16-bit
// fields [kSortWaves][n_b rounded up to even] (slots in a tile stay below
// 2^16), the tile's (first global slot - first local slot) of every bucket,
// the tile in sorted order [kTile], and per wave a table of lane masks by the
// low bits of the id, whose first words hold the waves' sums of the bucket
// scan before the ranking starts.  At 1024 buckets this is 40 KB, four
// workgroups per CU.
constexpr int kScatterBucketsPerThread = 2;  // one 32-bit word of 16-bit fields; n_b <= 2 * kSortWaves * 64
__host__ __device__ inline int even_buckets(int n_b) { return (n_b + 1) & ~1; }
constexpr int kLowBits = 6;  // id bits resolved through the mask table; the rest by ballots
size_t scatter_lds_bytes(int n_b) {
    return (size_t)kSortWaves * even_buckets(n_b) * sizeof(uint16_t) + even_buckets(n_b) * sizeof(int) +
           kTile * sizeof(uint32_t) + kSortWaves * (1 << kLowBits) * sizeof(uint64_t);
}

template <bool IDS16>
__global__ __launch_bounds__(kSortWaves * 64) void sort_scatter_kernel(const int32_t* __restrict__ buckets,
                                                           const uint16_t* __restrict__ ids16,
                                                           const int32_t* __restrict__ offsets,
                                                           int L, int n_r, int n_b,
                                                           int n_tiles, int32_t* __restrict__ perm,
                                                           int32_t* __restrict__ undo) {
    extern __shared__ int smem[];
    const int half = even_buckets(n_b) / 2;  // 32-bit words per wave's row
    uint32_t* base = reinterpret_cast<uint32_t*>(smem);  // [kSortWaves][half], two 16-bit fields each
    int* delta = smem + kSortWaves * half;                // [2 * half]
    uint32_t* staged = reinterpret_cast<uint32_t*>(delta + 2 * half);  // [kTile]: bucket << 16 | position in tile
    // [kSortWaves][2^kLowBits] lane masks (8-byte aligned: every part above
    // is a multiple of 8 bytes); until the ranking, its first words are the
    // waves' sums of the bucket scan [kSortWaves]
    uint64_t* masks = reinterpret_cast<uint64_t*>(staged + kTile);
    int* wsum = reinterpret_cast<int*>(masks);
    // Workgroup b of the launch runs on XCD b % 8 (round-robin dispatch).
    // Each XCD is given a contiguous run of (segment, tile) items, so the
    // tiles of a segment write their perm runs into the same XCD's L2, which
    // merges them into whole lines before they reach HBM, and the rounds of
    // one (batch, head) read its bucket ids through one L2.
    const int64_t nblk = (int64_t)gridDim.x * gridDim.y;
    const int64_t bid = blockIdx.x + (int64_t)blockIdx.y * gridDim.x;
    const int64_t item = nblk % 8 == 0 ? (bid % 8) * (nblk / 8) + bid / 8 : bid;
    const int tile = (int)(item % gridDim.x);
    const int64_t seg = item / gridDim.x;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t* wrow = base + wave * half;
    uint16_t* wslot = reinterpret_cast<uint16_t*>(wrow);
    uint64_t* wmask = masks + wave * (1 << kLowBits);

    for (int i = threadIdx.x; i < kSortWaves * half; i += blockDim.x) base[i] = 0;
    const int t0 = tile * kTile;
    const int n_tile = min(kTile, L - t0);
    const int p0 = t0 + wave * kPerWave;
    const int p1 = min(L, p0 + kPerWave);
    // this lane's ids, all loads in flight at once (kPerWave / 64 per lane);
    // positions past the segment load a valid id that is never used, so the
    // loads are unconditional and not each followed by its own wait
    constexpr int kIter = kPerWave / 64;
    int ids[kIter];
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
        const int pos = min(max(p0 + 64 * it + lane, 0), max(p1 - 1, 0));
        ids[it] = IDS16 ? (int)ids16[seg * L + pos] : buckets[(bh * L + pos) * n_r + r];
    }
    // the tile's first global slot of this thread's two buckets, loaded
    // with the ids
    const int b0 = (int)threadIdx.x * kScatterBucketsPerThread;
    int goff[kScatterBucketsPerThread];
#pragma unroll
    for (int k = 0; k < kScatterBucketsPerThread; ++k)
        goff[k] = offsets[(seg * n_tiles + tile) * n_b + min(b0 + k, n_b - 1)];
#pragma unroll
    for (int it = 0; it < kIter; ++it) ids[it] = clamp_bucket(ids[it], n_b);
    __syncthreads();
    // per-wave counts (a wave holds at most kPerWave < 2^16 of a bucket)
#pragma unroll
    for (int it = 0; it < kIter; ++it)
        if (p0 + 64 * it + lane < p1) atomicAdd(&wrow[ids[it] >> 1], 1u << ((ids[it] & 1) << 4));
    __syncthreads();
    // The tile's count of the thread's two buckets (one word of every
    // wave's row), whose exclusive scan over the workgroup (thread order is
    // bucket order) is each bucket's first slot in the tile's own sorted
    // order; then every wave's first local slot of the two buckets: that
    // plus the counts of the earlier waves of this tile.
    const bool owner = b0 < n_b;
    uint32_t word[kSortWaves];
    uint32_t c_lo = 0, c_hi = 0;
#pragma unroll
    for (int w = 0; w < kSortWaves; ++w) {
        word[w] = owner ? base[w * half + threadIdx.x] : 0u;
        c_lo += word[w] & 0xFFFFu;
        c_hi += word[w] >> 16;
    }
    const int tot = (int)(c_lo + c_hi);
    int incl = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int local = incl - tot;
    for (int w = 0; w < wave; ++w) local += wsum[w];
    if (owner) {
        uint32_t run_lo = (uint32_t)local, run_hi = (uint32_t)local + c_lo;
        delta[b0] = goff[0] - (int)run_lo;
        delta[b0 + 1] = goff[1] - (int)run_hi;
#pragma unroll
        for (int w = 0; w < kSortWaves; ++w) {
            base[w * half + threadIdx.x] = run_lo | (run_hi << 16);
            run_lo += word[w] & 0xFFFFu;
            run_hi += word[w] >> 16;
        }
    }
    __syncthreads();
    // the wave's mask table, cleared now that no wave reads the scan sums
    // (the wave's own LDS operations run in order, so no barrier follows)
    if (lane < (1 << kLowBits)) wmask[lane] = 0;

    // Rank of a position among the equal buckets of its 64-lane group: the
    // lanes holding the same bucket are those agreeing with it on every bit
    // of the id (ids are below n_b <= 1024): on the low kLowBits bits, the
    // lanes that set their bit in the wave's mask entry of those bits (an
    // LDS atomic or, read back and cleared by the same wave, whose LDS
    // operations run in order), on each higher bit, the lanes whose ballot
    // of that bit agrees; the rank counts those below the lane, so equal
    // keys keep their position order.  The highest lane of each bucket moves the bucket's
    // next slot on (the wave's LDS operations run in order).  undo is
    // written here, in position order; perm goes to the tile's sorted copy
    // in LDS first.
    int32_t* pseg = perm + seg * L;
    int32_t* useg = undo + seg * L;
    constexpr int kIdBits = 10;  // ids below n_b <= 1024
#pragma unroll
    for (int it = 0; it < kIter; ++it) {
        const int pos = p0 + 64 * it + lane;
        const bool active = pos < p1;
        const int b = ids[it];
        const int start = wslot[b];
        const int d = delta[b];
        uint64_t* entry = wmask + (b & ((1 << kLowBits) - 1));
        if (active) atomicOr(reinterpret_cast<unsigned long long*>(entry), 1ull << lane);
        const uint64_t same_low = *entry;  // after every lane's or
        *entry = 0;                        // after every lane's read
        // lanes differing from this one in a higher bit: for every bit, the
        // ballot of the bit xor this lane's bit spread over the word
        uint32_t diff_lo = 0, diff_hi = 0;
#pragma unroll
        for (int bit = kLowBits; bit < kIdBits; ++bit) {
            const uint32_t spread = (uint32_t)__builtin_amdgcn_sbfe(b, bit, 1);  // 0 or all ones
            const uint64_t ones = __ballot(spread != 0u);
            diff_lo |= (uint32_t)ones ^ spread;
            diff_hi |= (uint32_t)(ones >> 32) ^ spread;
        }
        const uint64_t peers = same_low & ~(((uint64_t)diff_hi << 32) | diff_lo);
        const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(peers >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)peers, 0u));
        if (active) {
            const int slot = start + before;  // in the tile's sorted order
            staged[min(slot, kTile - 1)] = ((uint32_t)b << 16) | (uint32_t)(pos - t0);
            useg[pos] = slot + d;
            if ((peers >> lane) == 1ull) wslot[b] = (uint16_t)(start + __popcll(peers));
        }
    }
    __syncthreads();
    // The tile in sorted order: consecutive entries of one bucket go to
    // consecutive slots, so each wave's stores cover a few runs of whole
    // words instead of one scattered word per lane.
    constexpr int kOut = kTile / (kSortWaves * 64);
    uint32_t e[kOut];
#pragma unroll
    for (int k = 0; k < kOut; ++k) e[k] = staged[threadIdx.x + k * kSortWaves * 64];
#pragma unroll
    for (int k = 0; k < kOut; ++k) {
        const int j = threadIdx.x + k * kSortWaves * 64;
        if (j < n_tile) pseg[min(max(delta[e[k] >> 16] + j, 0), L - 1)] = t0 + (int)(e[k] & 0xFFFFu);
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

size_t sort_counts_bytes(int64_t BH, int L, int n_rounds, int n_buckets) {
    const int64_t n_tiles = (L + kTile - 1) / kTile;
    return align256((size_t)(BH * n_rounds * n_buckets * n_tiles) * sizeof(int32_t));
}
size_t sort_workspace_bytes(int64_t BH, int L, int n_rounds, int n_buckets) {
    return sort_counts_bytes(BH, L, n_rounds, n_buckets) + align256((size_t)BH * n_rounds * L * sizeof(uint16_t));
}

hipError_t launch_sort(int64_t BH, int L, int n_rounds, int n_buckets, const int32_t* buckets,
                       int32_t* perm, int32_t* undo, int32_t* bucket_start, void* workspace,
                       bool round_major_ids, hipStream_t stream) {
    if (BH == 0 || L == 0) return hipSuccess;
    const int n_tiles = (L + kTile - 1) / kTile;
    int32_t* counts = static_cast<int32_t*>(workspace);
    uint16_t* ids16 = round_major_ids ? reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) +
                                                                     sort_counts_bytes(BH, L, n_rounds, n_buckets))
                                      : nullptr;
    const int rpg = std::max(1, std::min(n_rounds, kHistLdsInts / n_buckets));
    const int groups = (n_rounds + rpg - 1) / rpg;

    const size_t hist_lds = hist_lds_bytes(rpg, n_buckets, ids16 != nullptr);
    if (hist_lds > 65536)
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&sort_hist_kernel),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)hist_lds);
    sort_hist_kernel<<<dim3(n_tiles, (unsigned)BH, groups), kHistThreads, hist_lds, stream>>>(
        buckets, L, n_rounds, n_buckets, rpg, n_tiles, counts, ids16);
    if (n_tiles <= kScanTiles && n_buckets <= kScanThreads)
        sort_scan_kernel<<<(unsigned)(BH * n_rounds), kScanThreads, 0, stream>>>(counts, L, n_buckets, n_tiles,
                                                                                 bucket_start);
    else
        sort_scan_any_kernel<<<(unsigned)(BH * n_rounds), 256, 0, stream>>>(counts, L, n_buckets, n_tiles,
                                                                            bucket_start);
    const dim3 grid(n_tiles, (unsigned)(BH * n_rounds));
    if (ids16)
        sort_scatter_kernel<true><<<grid, kSortWaves * 64, scatter_lds_bytes(n_buckets), stream>>>(
            buckets, ids16, counts, L, n_rounds, n_buckets, n_tiles, perm, undo);
    else
        sort_scatter_kernel<false><<<grid, kSortWaves * 64, scatter_lds_bytes(n_buckets), stream>>>(
            buckets, ids16, counts, L, n_rounds, n_buckets, n_tiles, perm, undo);
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

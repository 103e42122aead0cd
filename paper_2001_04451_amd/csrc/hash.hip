// Angular LSH: h(x) = argmax([xR; -xR]) for every query and round
// (Reformer, Sec. 2 "Locality sensitive hashing"; one R per round as in
// eq. union-pairs).
//
// Design (gfx950):
//  * The projections xR are a dense [rows x 64] * [64 x n_b/2] contraction per
//    round, run on the bf16 matrix cores.  R (fp32) is split exactly into
//    bf16 planes R = R_hi + R_mid + res with |res| <= 2^-16 |R|; bf16 x bf16
//    products are exact in fp32, so the screened projection differs from the
//    exact one by a bounded amount (residual, fp32 accumulation, and the
//    index bits packed into the low mantissa).
//  * Each lane keeps the two largest |projection| keys it has seen; the
//    argmax index inside a 32-column tile rides in the low mantissa bits of
//    the key, so one and-or, one max and one median-of-three per projection
//    suffice, and the tile of the best key is noted once per tile.
//  * If the gap between the best and second-best key cannot rule out an
//    exchange under the error bound, the row-round is appended to a list and
//    recomputed afterwards in fp64 by a second kernel (same products and
//    summation order as a plain loop), so the ids always equal the exact
//    argmax.
#include "common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr int kHashWaves = 4;
constexpr int kRB = 2;  // 32-row blocks per wave: each staged R tile feeds 2 * 8 MFMAs
constexpr uint32_t kKeyMask = 0x7FFFFFF0u;  // |value| with 4 index bits
constexpr int kHashRowsPerBlock = 32 * kRB * kHashWaves;
constexpr int kColStride = 72;                      // bf16 per staged R column (64 + pad)
constexpr int kTilesPerStage = 2;                   // 64 R columns per LDS stage
constexpr int kMaxColsPerLane = 8;                  // exact path: n_b/2 <= 512

// One R column per block of 64 lanes (lane = t): bf16 planes hi/mid and an
// fp32 copy, all [n_r][half_pad][64] (column contiguous, zero padded), and
// the column's 2-norm.
__global__ __launch_bounds__(64) void prep_r_cols_kernel(const float* __restrict__ R, int half,
                                                         int half_pad, uint16_t* __restrict__ r_hi,
                                                         uint16_t* __restrict__ r_mid,
                                                         float* __restrict__ r_t,
                                                         float* __restrict__ col_norm) {
    const int c = blockIdx.x, r = blockIdx.y, t = threadIdx.x;
    const float x = c < half ? R[((size_t)r * kHeadDim + t) * half + c] : 0.f;
    const uint32_t hi = f32_to_bf16_bits(x);
    const float res = x - bf16_bits_to_f32(hi);  // exact (Sterbenz)
    const uint32_t mid = f32_to_bf16_bits(res);
    const size_t o = ((size_t)r * half_pad + c) * kHeadDim + t;
    r_hi[o] = (uint16_t)hi;
    r_mid[o] = (uint16_t)mid;
    r_t[o] = x;
    float ss = x * x;
    for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
    if (t == 0) col_norm[(size_t)r * half_pad + c] = sqrtf(ss);
}

// Largest column norm of each round; also clears the round's refinement counter.
__global__ __launch_bounds__(256) void prep_r_max_kernel(const float* __restrict__ col_norm,
                                                         int half_pad,
                                                         float* __restrict__ col_norm_max,
                                                         int* __restrict__ refine_count) {
    __shared__ float red[256];
    const int r = blockIdx.x;
    float mx = 0.f;
    for (int c = threadIdx.x; c < half_pad; c += blockDim.x)
        mx = fmaxf(mx, col_norm[(size_t)r * half_pad + c]);
    red[threadIdx.x] = mx;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        col_norm_max[r] = red[0];
        refine_count[r] = 0;
    }
}

template <bool F32>
__device__ __forceinline__ float q_value(const void* q, int64_t row, int k) {
    if constexpr (F32) {
        return static_cast<const float*>(q)[row * kHeadDim + k];
    } else {
        return bf16_bits_to_f32(static_cast<const uint16_t*>(q)[row * kHeadDim + k]);
    }
}

// Exact argmax of [xR; -xR] for the listed row-rounds of one round.  The
// round's R (fp32, [d][n_b/2], at most 128 KB) is staged in LDS once per
// block; each wave settles one row-round at a time.  Column c's projection
// is the left-to-right sum over t of the exact products q_t * R_tc in fp64
// (the order of a plain loop), and ties go to the first index of [xR; -xR].
constexpr int kRefineThreads = 512;

template <bool F32>
__global__ __launch_bounds__(kRefineThreads) void hash_refine_kernel(const void* __restrict__ q,
                                                          const float* __restrict__ R, int half,
                                                          int n_r, int64_t list_stride,
                                                          const int* __restrict__ lists,
                                                          const int* __restrict__ counts,
                                                          int32_t* __restrict__ buckets) {
    extern __shared__ float Rs[];  // [64][half]
    const int r = blockIdx.y;
    const int n = counts[r];
    constexpr int kWavesPerBlock = kRefineThreads / 64;
    if (n == 0 || (int)blockIdx.x * kWavesPerBlock >= n) return;  // uniform per block
    // stage the round's R: 16-byte pieces, eight loads in flight per thread
    const f32x4* Rr = reinterpret_cast<const f32x4*>(R + (size_t)r * kHeadDim * half);
    f32x4* Rs4 = reinterpret_cast<f32x4*>(Rs);
    const int n4 = kHeadDim * half / 4;
    for (int i0 = threadIdx.x; i0 < n4; i0 += 8 * blockDim.x) {
        f32x4 tmp[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * blockDim.x;
            if (i < n4) tmp[u] = Rr[i];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * blockDim.x;
            if (i < n4) Rs4[i] = tmp[u];
        }
    }
    __syncthreads();
    const int* list = lists + list_stride * r;
    const int lane = lane_id();
    const int waves = gridDim.x * kWavesPerBlock;
    for (int e = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6); e < n; e += waves) {
        const int64_t row = list[e];
        const float qv = q_value<F32>(q, row, lane);
        double p[kMaxColsPerLane];
#pragma unroll
        for (int k = 0; k < kMaxColsPerLane; ++k) p[k] = 0.0;
        // q_t reaches every lane through a scalar register (readlane), and the
        // fully unrolled sum lets the LDS reads run ahead of the fp64 adds.
#pragma unroll
        for (int t = 0; t < kHeadDim; ++t) {
            const double qt = (double)__builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, qv), t));
#pragma unroll
            for (int k = 0; k < kMaxColsPerLane; ++k) {
                const int c = lane + 64 * k;
                if (c < half) p[k] = __dadd_rn(p[k], __dmul_rn(qt, (double)Rs[t * half + c]));
            }
        }
        double bv = -__builtin_inf();
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int k = 0; k < kMaxColsPerLane; ++k) {
            const int c = lane + 64 * k;
            if (c < half) {
                if (p[k] > bv || (p[k] == bv && c < bi)) { bv = p[k]; bi = c; }
                const double m = -p[k];
                if (m > bv || (m == bv && half + c < bi)) { bv = m; bi = half + c; }
            }
        }
        for (int o = 32; o >= 1; o >>= 1) {
            const double ov = __shfl_xor(bv, o);
            const int oi = __shfl_xor(bi, o);
            if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
        }
        if (lane == 0) buckets[row * n_r + r] = bi;
    }
}

struct Tile {
    f32x16 acc[kRB];
};

template <bool F32>
__device__ __forceinline__ void tile_mfma(Tile& T, const uint16_t (*st)[kColStride],
                                          const uint16_t (*st_mid)[kColStride], int col, int h,
                                          const bf16x8 (&qa)[kRB][4], const bf16x8 (&qm)[kRB][4]) {
    bf16x8 ahi[4], amid[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        ahi[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(&st[col][32 * h + 8 * s]));
        amid[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(&st_mid[col][32 * h + 8 * s]));
    }
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) T.acc[rb] = f32x16{};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) T.acc[rb] = mfma32x32x16(ahi[s], qa[rb][s], T.acc[rb]);
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) T.acc[rb] = mfma32x32x16(amid[s], qa[rb][s], T.acc[rb]);
        if constexpr (F32) {
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb) T.acc[rb] = mfma32x32x16(ahi[s], qm[rb][s], T.acc[rb]);
        }
    }
}

// Keys are |projection| bit patterns (non-negative floats order like their
// bits as unsigned integers) with the low 4 mantissa bits replaced by the
// register index j inside the tile: one and-or, one unsigned median-of-three
// and one unsigned max per projection.  The tile holding the best key is
// recorded when the running best changes during the tile.
__device__ __forceinline__ void tile_epilogue(const Tile& T, int tile, uint32_t (&best)[kRB],
                                              uint32_t (&second)[kRB], int (&best_tile)[kRB]) {
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
        uint32_t b = best[rb], sc = second[rb];
        const uint32_t b0 = b;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const uint32_t key = (__float_as_uint(T.acc[rb][j]) & kKeyMask) | (uint32_t)j;
            sc = max(min(key, b), min(max(key, b), sc));  // median of three
            b = max(key, b);
        }
        best_tile[rb] = b != b0 ? tile : best_tile[rb];
        best[rb] = b;
        second[rb] = sc;
    }
}

template <bool F32>
__global__ __launch_bounds__(256, 2) void hash_kernel(
    const void* __restrict__ q, int64_t rows, int n_r, int half, int half_pad,
    const uint16_t* __restrict__ r_hi, const uint16_t* __restrict__ r_mid,
    const float* __restrict__ r_t, const float* __restrict__ col_norm_max, float err_sum,
    float err_pack, int32_t* __restrict__ buckets, int* __restrict__ refine_lists,
    int* __restrict__ refine_counts) {
    // [buf][plane][column][k]
    __shared__ __attribute__((aligned(16))) uint16_t stage[2][2][kTilesPerStage * 32][kColStride];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6, h = lane >> 5, n = lane & 31;
    const int64_t row0 = (int64_t)blockIdx.x * kHashRowsPerBlock + wave * (32 * kRB);

    // Queries as the B operand: lane holds row (n) and k = 32h + 8s + e, s = 0..3.
    bf16x8 qa[kRB][4];
    bf16x8 qm[kRB][4];  // fp32 input: second bf16 plane of q
    float qn[kRB];
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
        const int64_t row = row0 + rb * 32 + n;
        const bool valid = row < rows;
        float ss = 0.f;
        if constexpr (F32) {
            const float* src = static_cast<const float*>(q) + row * kHeadDim + 32 * h;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                f32x4 x0 = valid ? *reinterpret_cast<const f32x4*>(src + 8 * s) : f32x4{0, 0, 0, 0};
                f32x4 x1 = valid ? *reinterpret_cast<const f32x4*>(src + 8 * s + 4) : f32x4{0, 0, 0, 0};
                float xs[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
                u32x4 hi, mid;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t h0 = f32_to_bf16_bits(xs[2 * e]), h1 = f32_to_bf16_bits(xs[2 * e + 1]);
                    const uint32_t m0 = f32_to_bf16_bits(xs[2 * e] - bf16_bits_to_f32(h0));
                    const uint32_t m1 = f32_to_bf16_bits(xs[2 * e + 1] - bf16_bits_to_f32(h1));
                    hi[e] = h0 | (h1 << 16);
                    mid[e] = m0 | (m1 << 16);
                    ss = fmaf(xs[2 * e], xs[2 * e], ss);
                    ss = fmaf(xs[2 * e + 1], xs[2 * e + 1], ss);
                }
                qa[rb][s] = as_bf16x8(hi);
                qm[rb][s] = as_bf16x8(mid);
            }
        } else {
            const uint16_t* src = static_cast<const uint16_t*>(q) + row * kHeadDim + 32 * h;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const u32x4 raw = valid ? *reinterpret_cast<const u32x4*>(src + 8 * s) : u32x4{0, 0, 0, 0};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float a = __uint_as_float(raw[e] << 16), b = __uint_as_float(raw[e] & 0xFFFF0000u);
                    ss = fmaf(a, a, ss);
                    ss = fmaf(b, b, ss);
                }
                qa[rb][s] = as_bf16x8(raw);
                qm[rb][s] = as_bf16x8(u32x4{0, 0, 0, 0});
            }
        }
        ss += __shfl_xor(ss, 32);
        qn[rb] = sqrtf(ss);
    }

    const int n_tiles = half_pad / 32;
    const int cols_per_stage = kTilesPerStage * 32;
    const int n_stages = (half_pad + cols_per_stage - 1) / cols_per_stage;
    constexpr int kLoads = 2 * kTilesPerStage * 32 * 8 / 256;  // 16-byte pieces per thread

    for (int r = 0; r < n_r; ++r) {
        const uint16_t* hi_r = r_hi + (size_t)r * half_pad * kHeadDim;
        const uint16_t* mid_r = r_mid + (size_t)r * half_pad * kHeadDim;
        uint32_t best[kRB], second[kRB];
        int best_tile[kRB];
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
            best[rb] = second[rb] = 0u;
            best_tile[rb] = 0;
        }

        u32x4 pre[kLoads];
        auto gload = [&](int st) {
#pragma unroll
            for (int i = 0; i < kLoads; ++i) {
                const int idx = tid + 256 * i;
                const int plane = idx / (cols_per_stage * 8);
                const int col = (idx >> 3) % cols_per_stage, part = idx & 7;
                const int gcol = st * cols_per_stage + col;
                const uint16_t* base = plane ? mid_r : hi_r;
                pre[i] = gcol < half_pad
                             ? *reinterpret_cast<const u32x4*>(base + (size_t)gcol * kHeadDim + part * 8)
                             : u32x4{0, 0, 0, 0};
            }
        };
        auto lstore = [&](int buf) {
#pragma unroll
            for (int i = 0; i < kLoads; ++i) {
                const int idx = tid + 256 * i;
                const int plane = idx / (cols_per_stage * 8);
                const int col = (idx >> 3) % cols_per_stage, part = idx & 7;
                *reinterpret_cast<u32x4*>(&stage[buf][plane][col][part * 8]) = pre[i];
            }
        };

        gload(0);
        lstore(0);
        __syncthreads();
        for (int st = 0; st < n_stages; ++st) {
            if (st + 1 < n_stages) gload(st + 1);
            const int buf = st & 1;
            const int t0 = st * kTilesPerStage;
            const int nt = min(kTilesPerStage, n_tiles - t0);
            // The second tile's MFMAs are issued before the first tile's
            // epilogue, so the matrix core and the vector ALUs overlap inside
            // the wave; the two waves sharing a SIMD overlap the rest.
            static_assert(kTilesPerStage == 2, "pipeline written for two tiles per stage");
            Tile ta, tb;
            tile_mfma<F32>(ta, stage[buf][0], stage[buf][1], n, h, qa, qm);
            if (nt > 1) tile_mfma<F32>(tb, stage[buf][0], stage[buf][1], 32 + n, h, qa, qm);
            tile_epilogue(ta, t0, best, second, best_tile);
            if (nt > 1) tile_epilogue(tb, t0 + 1, best, second, best_tile);
            if (st + 1 < n_stages) lstore((st + 1) & 1);
            __syncthreads();
        }

        // Round epilogue: merge the two lane halves (different columns of the
        // same row), decide, and queue close calls for the exact pass.
        const float cn = col_norm_max[r];
        const float* r_t_round = r_t + (size_t)r * half_pad * kHeadDim;
        int* list = refine_lists + rows * r;
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
            const int64_t row = row0 + rb * 32 + n;
            const bool valid = row < rows;
            const uint32_t bp = __shfl_xor(best[rb], 32), sp = __shfl_xor(second[rb], 32);
            const int tp = __shfl_xor(best_tile[rb], 32);
            const bool mine = best[rb] > bp || (best[rb] == bp && h == 0);
            const uint32_t bk = mine ? best[rb] : bp;
            const float b1 = __uint_as_float(bk);
            const float s1 = __uint_as_float(max(min(best[rb], bp), max(second[rb], sp)));
            const int hw = mine ? h : (h ^ 1);
            const int tw = mine ? best_tile[rb] : tp;
            const uint32_t j = bk & 15u;
            const int col = tw * 32 + 8 * (int)(j >> 2) + 4 * hw + (int)(j & 3u);
            // Every screened key is within eps = err_sum*|q|*max|R_c| + err_pack*key
            // of its exact |projection|; an exchange of winners needs a gap <= 2 eps.
            const float thr = 2.04f * (err_sum * qn[rb] * cn + err_pack * b1);
            const bool flag = !(b1 - s1 > thr) || col >= half;
            // Sign of the winning projection.  When the row is not flagged its
            // magnitude exceeds the error bound, so fp32 gets the sign right.
            const int colc = col < half ? col : 0;
            const f32x4* rt = reinterpret_cast<const f32x4*>(r_t_round + (size_t)colc * kHeadDim + 32 * h);
            float part = 0.f;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const f32x4 ra = rt[2 * s], rb4 = rt[2 * s + 1];
                const float rv[8] = {ra[0], ra[1], ra[2], ra[3], rb4[0], rb4[1], rb4[2], rb4[3]};
                const u32x4 w = __builtin_bit_cast(u32x4, qa[rb][s]);
                const u32x4 m = __builtin_bit_cast(u32x4, qm[rb][s]);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float lo = __uint_as_float(w[e] << 16) + __uint_as_float(m[e] << 16);
                    const float hi = __uint_as_float(w[e] & 0xFFFF0000u) + __uint_as_float(m[e] & 0xFFFF0000u);
                    part = fmaf(lo, rv[2 * e], part);
                    part = fmaf(hi, rv[2 * e + 1], part);
                }
            }
            const float p = part + __shfl_xor(part, 32);
            const bool queue = flag && valid && h == 0;
            if (valid && h == 0 && !flag) buckets[row * n_r + r] = p > 0.f ? col : half + col;
            // wave-aggregated append to this round's refinement list
            const uint64_t qmask = __ballot(queue);
            if (qmask) {
                const int leader = __ffsll((unsigned long long)qmask) - 1;
                int slot0 = 0;
                if (lane == leader) slot0 = atomicAdd(&refine_counts[r], __popcll(qmask));
                slot0 = __shfl(slot0, leader);
                if (queue) list[slot0 + __popcll(qmask & ((1ull << lane) - 1ull))] = (int)row;
            }
        }
    }
}

struct HashWs {
    uint16_t* r_hi;
    uint16_t* r_mid;
    float* r_t;
    float* col_norm;
    float* col_norm_max;
    int* count;
    int* list;
    size_t bytes;
};

HashWs carve(void* base, int64_t rows, int n_rounds, int half_pad) {
    const size_t per = (size_t)n_rounds * half_pad * kHeadDim;
    char* p = static_cast<char*>(base);
    HashWs w{};
    size_t off = 0;
    w.r_hi = reinterpret_cast<uint16_t*>(p + off);
    off += align256(per * 2);
    w.r_mid = reinterpret_cast<uint16_t*>(p + off);
    off += align256(per * 2);
    w.r_t = reinterpret_cast<float*>(p + off);
    off += align256(per * 4);
    w.col_norm = reinterpret_cast<float*>(p + off);
    off += align256((size_t)n_rounds * half_pad * 4);
    w.col_norm_max = reinterpret_cast<float*>(p + off);
    off += align256((size_t)n_rounds * 4);
    w.count = reinterpret_cast<int*>(p + off);
    off += align256((size_t)n_rounds * 4);
    w.list = reinterpret_cast<int*>(p + off);
    off += align256((size_t)rows * n_rounds * 4);
    w.bytes = off;
    return w;
}

}  // namespace

size_t hash_workspace_bytes(int64_t rows, int n_rounds, int n_buckets) {
    const int half_pad = (n_buckets / 2 + 31) / 32 * 32;
    return carve(nullptr, rows, n_rounds, half_pad).bytes;
}

hipError_t launch_hash(const void* q, bool f32, int64_t rows, int n_rounds, int n_buckets,
                       const float* R, int32_t* buckets, void* workspace, hipStream_t stream) {
    const int half = n_buckets / 2;
    const int half_pad = (half + 31) / 32 * 32;
    const HashWs w = carve(workspace, rows, n_rounds, half_pad);

    prep_r_cols_kernel<<<dim3(half_pad, n_rounds), 64, 0, stream>>>(R, half, half_pad, w.r_hi,
                                                                     w.r_mid, w.r_t, w.col_norm);
    prep_r_max_kernel<<<n_rounds, 256, 0, stream>>>(w.col_norm, half_pad, w.col_norm_max, w.count);
    if (rows == 0) return hipGetLastError();

    // Error bound of a screened key against the exact |projection| p_c:
    //  * the dropped bf16 plane(s), <= 2^-16 sum_t |q_t R_tc| each;
    //  * fp32 accumulation of the exact bf16 products, <= one ulp of the
    //    partial sum (<= 2^-23 sum_t |q_t R_tc|) per addition;
    //  * the 4 index bits written over the low mantissa, < 2^-19 |key|.
    // sum_t |q_t R_tc| <= |q| |R_c| (Cauchy-Schwarz) <= |q| max_c |R_c|.
    const double adds = f32 ? 3 * kHeadDim : 2 * kHeadDim;
    const double resid = f32 ? 3.1 * 0x1p-16 : 0x1p-16;
    const float err_sum = (float)((resid + adds * 0x1p-23) * 1.01);
    const float err_pack = (float)0x1p-19;

    const unsigned grid = (unsigned)((rows + kHashRowsPerBlock - 1) / kHashRowsPerBlock);
    const size_t refine_lds = (size_t)kHeadDim * half * sizeof(float);
    // Refinement blocks per round: one 128 KB-LDS block per CU over all rounds
    // (a typical list holds well under 1% of the rows; longer ones are strided).
    const unsigned refine_blocks =
        (unsigned)std::max<int64_t>(1, std::min<int64_t>((256 + n_rounds - 1) / n_rounds, rows / 1024));
    if (f32) {
        hash_kernel<true><<<grid, 256, 0, stream>>>(q, rows, n_rounds, half, half_pad, w.r_hi,
                                                     w.r_mid, w.r_t, w.col_norm_max, err_sum,
                                                     err_pack, buckets, w.list, w.count);
        hipFuncSetAttribute(reinterpret_cast<const void*>(&hash_refine_kernel<true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)refine_lds);
        hash_refine_kernel<true><<<dim3(refine_blocks, n_rounds), kRefineThreads, refine_lds, stream>>>(
            q, R, half, n_rounds, rows, w.list, w.count, buckets);
    } else {
        hash_kernel<false><<<grid, 256, 0, stream>>>(q, rows, n_rounds, half, half_pad, w.r_hi,
                                                      w.r_mid, w.r_t, w.col_norm_max, err_sum,
                                                      err_pack, buckets, w.list, w.count);
        hipFuncSetAttribute(reinterpret_cast<const void*>(&hash_refine_kernel<false>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)refine_lds);
        hash_refine_kernel<false><<<dim3(refine_blocks, n_rounds), kRefineThreads, refine_lds, stream>>>(
            q, R, half, n_rounds, rows, w.list, w.count, buckets);
    }
    return hipGetLastError();
}

}  // namespace lsh

// Angular LSH: h(x) = argmax([xR; -xR]) for every query and round
// (Reformer, Sec. 2 "Locality sensitive hashing"; one R per round as in
// eq. union-pairs).
//
// Design (gfx950):
//  * The projections xR are a dense [rows x 64] * [64 x n_b/2] contraction per
//    round, run on the matrix cores with 16-bit operands and fp32
//    accumulation.  For bf16 input, q and each round of R are scaled by
//    powers of two (which leaves every argmax unchanged) and R is split into
//    binary16 planes R = R_hi + R_mid + res, |R_hi - R| <= 2^-12 |R|;
//    the scaled bf16 q is exact in binary16.  For fp32 input, q and R are
//    split into bf16 planes instead.  16-bit products are exact in fp32, so
//    a screened projection differs from the exact one by a bounded amount
//    (residual, fp32 accumulation, and the index bits packed into the low
//    mantissa).
//  * R streams through LDS by direct global-to-LDS copies, 256 columns per
//    stage, while each wave's products for the next tile are interleaved
//    with the vector epilogue of the current one (one in-order instruction
//    stream keeps both the matrix core and the vector ALUs busy).
//  * Each lane keeps the two largest |projection| keys it has seen; the
//    index inside a 32-column tile rides in the low bits of the key, so an
//    and-or per projection and a max3, a med3 and a max per two suffice, and
//    the tile of the best key is noted once per tile.  A row's ids for all
//    rounds are written together at the end.
//  * If the gap between the best and second-best key cannot rule out an
//    exchange under the error bound, the row-round is appended to a list and
//    recomputed afterwards over both planes, and what that leaves open in
//    fp64 by a last kernel (same products and summation order as a plain
//    loop), so the ids always equal the exact argmax.
#include "common.h"
#include "launch.h"

#include <type_traits>

namespace lsh {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kRB = 2;  // 32-row blocks per wave: each staged R tile feeds 2 * 8 MFMAs

// Largest |R| of each 1/kScaleParts of each round (block (part, r)): the
// fp16 planes' scale is taken from these partial maxima.
constexpr int kScaleParts = 32;

__global__ __launch_bounds__(256) void prep_r_part_kernel(const float* __restrict__ R, int half,
                                                          float* __restrict__ r_part) {
    __shared__ float red[4];
    const int part = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
    const int n = kHeadDim * half;
    const int per = (n + kScaleParts - 1) / kScaleParts;
    const int lo = part * per, hi = min(n, lo + per);
    const float* Rr = R + (size_t)r * n;
    float m = 0.f;
    for (int i = lo + tid; i < hi; i += 256) m = fmaxf(m, fabsf(Rr[i]));
    m = wave_max(m);
    if ((tid & 63) == 0) red[tid >> 6] = m;
    __syncthreads();
    if (tid == 0) r_part[r * kScaleParts + part] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// The exponent sr with max |R| * 2^sr in [2^14, 2^15) (0 when the round is
// zero or not finite): a positive scale of a whole round leaves every
// argmax unchanged.
__device__ __forceinline__ int round_scale_exp(const float* __restrict__ part) {
    float m = 0.f;
    for (int i = 0; i < kScaleParts; ++i) m = fmaxf(m, part[i]);
    // m in [2^e, 2^(e+1)) (frexp: m = f 2^k with f in [0.5, 1), e = k - 1)
    int k = 0;
    (void)frexpf(m, &k);
    return (m > 0.f && m <= 3.4e38f) ? 14 - (k - 1) : 0;
}

// x * 2^e for |e| up to 254, in two exact steps.
__device__ __forceinline__ double ldexp2(double x, int e) {
    const int a = e / 2;
    return x * __builtin_bit_cast(double, (uint64_t)(1023 + a) << 52) *
           __builtin_bit_cast(double, (uint64_t)(1023 + e - a) << 52);
}

// Nearest binary16 of x (|x| < 2^15 here), or 0 below fp16's normal range:
// the planes hold no subnormal, whatever the matrix cores do with them.
__device__ __forceinline__ uint32_t f16_normal_bits(double x) {
    const _Float16 h = fabs(x) < 0x1p-14 ? (_Float16)0.f : (_Float16)(float)x;
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// One R column per block of 64 lanes (lane = t): two 16-bit planes hi/mid,
// [n_r][half_pad][64] (column contiguous, zero padded), and three 2-norms of
// the column, [3][n_r][half_pad]: |R_c|, |R_c - hi_c|, |R_c - hi_c - mid_c|.
//  * F16 (bf16 input): binary16 planes of R_c * 2^sr[r] (sr from the
//    round's partial maxima, also written to r_exp); the norms are of the
//    scaled column, formed in fp64 from exact residuals.
//  * bf16 planes (fp32 input): R = hi + mid + res with each step exact.
template <bool F16>
__global__ __launch_bounds__(64) void prep_r_cols_kernel(const float* __restrict__ R, int half,
                                                         int half_pad, const float* __restrict__ r_part,
                                                         int* __restrict__ r_exp,
                                                         uint16_t* __restrict__ r_hi,
                                                         uint16_t* __restrict__ r_mid,
                                                         float* __restrict__ col_norm) {
    const int c = blockIdx.x, r = blockIdx.y, t = threadIdx.x;
    const int n_r = gridDim.y;
    const float x = c < half ? R[((size_t)r * kHeadDim + t) * half + c] : 0.f;
    uint32_t hi, mid;
    float n0, n1, n2;
    if constexpr (F16) {
        const int sr = round_scale_exp(r_part + r * kScaleParts);
        if (c == 0 && t == 0) r_exp[r] = sr;
        const double xs = ldexp2((double)x, sr);
        hi = f16_normal_bits(xs);
        const double res = xs - (double)f16_bits_to_f32(hi);  // exact in fp64
        mid = f16_normal_bits(res);
        const double res2 = res - (double)f16_bits_to_f32(mid);  // exact
        double s0 = xs * xs, s1 = res * res, s2 = res2 * res2;
        for (int off = 32; off >= 1; off >>= 1) {
            s0 += __shfl_xor(s0, off);
            s1 += __shfl_xor(s1, off);
            s2 += __shfl_xor(s2, off);
        }
        // rounded up to fp32 (the bounds that use them are upper bounds)
        n0 = (float)sqrt(s0) * (1.f + 0x1p-22f);
        n1 = (float)sqrt(s1) * (1.f + 0x1p-22f);
        n2 = (float)sqrt(s2) * (1.f + 0x1p-22f);
    } else {
        hi = f32_to_bf16_bits(x);
        const float res = x - bf16_bits_to_f32(hi);  // exact (Sterbenz)
        mid = f32_to_bf16_bits(res);
        const float res2 = res - bf16_bits_to_f32(mid);  // exact
        float s0 = x * x, s1 = res * res, s2 = res2 * res2;
        for (int off = 32; off >= 1; off >>= 1) {
            s0 += __shfl_xor(s0, off);
            s1 += __shfl_xor(s1, off);
            s2 += __shfl_xor(s2, off);
        }
        n0 = sqrtf(s0);
        n1 = sqrtf(s1);
        n2 = sqrtf(s2);
    }
    const size_t o = ((size_t)r * half_pad + c) * kHeadDim + t;
    r_hi[o] = (uint16_t)hi;
    r_mid[o] = (uint16_t)mid;
    if (t == 0) {
        const size_t plane = (size_t)n_r * half_pad, k = (size_t)r * half_pad + c;
        col_norm[k] = n0;
        col_norm[plane + k] = n1;
        col_norm[2 * plane + k] = n2;
    }
}

// Largest of each column norm per round (block (r, which)); block (0, 0)
// also clears the n_clear list counters.
__global__ __launch_bounds__(256) void prep_r_max_kernel(const float* __restrict__ col_norm, int n_r,
                                                         int half_pad, float* __restrict__ norm_max,
                                                         int* __restrict__ counts, int n_clear) {
    __shared__ float red[256];
    const int r = blockIdx.x, which = blockIdx.y;
    if (r == 0 && which == 0)
        for (int i = threadIdx.x; i < n_clear; i += blockDim.x) counts[i] = 0;
    const float* cn = col_norm + ((size_t)which * n_r + r) * half_pad;
    float mx = 0.f;
    for (int c = threadIdx.x; c < half_pad; c += blockDim.x) mx = fmaxf(mx, cn[c]);
    red[threadIdx.x] = mx;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    if (threadIdx.x == 0) norm_max[which * n_r + r] = red[0];
}

template <bool F32>
__device__ __forceinline__ float q_value(const void* q, int64_t row, int k) {
    if constexpr (F32) {
        return static_cast<const float*>(q)[row * kHeadDim + k];
    } else {
        return bf16_bits_to_f32(static_cast<const uint16_t*>(q)[row * kHeadDim + k]);
    }
}

// Exact argmax of [xR; -xR] for the listed row-rounds of one round.  A
// block takes the list in groups of 64 entries, one per lane of every wave,
// in two passes:
//  1. each wave forms the fp32 projections of its 32 columns for all 64
//     entries (lane = entry): R's values are the same for every lane, so they
//     are scalar loads (R[t][c0 .. c0+31] is contiguous), fetched one t ahead,
//     and nothing is staged.  The fp32
//     value is within eps = (64 * 2^-24 * 1.01 + 2^-46) * |q| * max_c |R_c|
//     of the fp64 one, so only a column whose fp32 magnitude is within 2 eps
//     of the entry's largest can hold the fp64 argmax;
//  2. for those candidates, the projection as the oracle forms it: the
//     left-to-right sum over t of the exact products q_t * R_tc in fp64, one
//     lane per (entry, candidate), sixteen candidate lanes per entry.  Ties go
//     to the first index of [xR; -xR].
// An entry with more than sixteen candidates (q = 0 makes every column one),
// or none (a non-finite q), takes the plain fp64 pass over every column,
// one wave per entry.
constexpr int kRefineThreads = 1024;
constexpr int kRefineWaves = kRefineThreads / 64;
constexpr int kRefineGroup = 64;     // entries per pass
constexpr int kRefineCand = 16;      // candidate lanes per entry
constexpr int kRefineCols = 32;      // columns per wave in pass 1
static_assert(kRefineWaves * kRefineCols >= 512, "pass 1 covers n_b / 2 <= 512 columns");
static_assert(kRefineWaves * 64 == kRefineGroup * kRefineCand, "pass 2 lanes");

__device__ __forceinline__ void better(double v, int i, double& bv, int& bi) {
    if (v > bv || (v == bv && i < bi)) {
        bv = v;
        bi = i;
    }
}

struct RefineShared {
    float qs[kRefineGroup][kHeadDim + 1];  // the group's q rows
    float qn[kRefineGroup];                // and their norms
    float mx[kRefineWaves][kRefineGroup];  // per wave: largest |fp32 projection| of each entry
    int cnt[kRefineGroup];                 // candidates found per entry
    int cand[kRefineGroup][kRefineCand];   // their columns
};

template <bool F32>
__global__ __launch_bounds__(kRefineThreads, 1) void hash_refine_kernel(const void* __restrict__ q,
                                                          const float* __restrict__ R, int half,
                                                          int n_r, int64_t list_stride,
                                                          const int* __restrict__ lists,
                                                          const int* __restrict__ counts,
                                                          const float* __restrict__ col_norm_max,
                                                          const int* __restrict__ r_exp,
                                                          int32_t* __restrict__ buckets) {
    __shared__ RefineShared S;
    const int r = blockIdx.y;
    const int n = counts[r];
    const int groups = (n + kRefineGroup - 1) / kRefineGroup;
    if ((int)blockIdx.x >= groups) return;  // uniform per block
    const int* list = lists + list_stride * r;
    const float* Rr = R + (size_t)r * kHeadDim * half;  // [t][half]
    const int lane = lane_id();
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // max_c |R_c| of the round as given (the planes' norms are of R * 2^r_exp)
    const float cn = r_exp ? ldexpf(col_norm_max[r], -r_exp[r]) : col_norm_max[r];
    const int c0 = wave * kRefineCols;  // this wave's columns in pass 1
    const int ncols = max(0, min(kRefineCols, half - c0));

    for (int g = blockIdx.x; g < groups; g += gridDim.x) {
        if (wave == 0) {
            // the group's q rows, one per lane, into LDS
            const int64_t row = list[min(g * kRefineGroup + lane, n - 1)];
            float qr[kHeadDim];
            if constexpr (F32) {
                const f32x4* src = reinterpret_cast<const f32x4*>(static_cast<const float*>(q) + row * kHeadDim);
#pragma unroll
                for (int t4 = 0; t4 < kHeadDim / 4; ++t4) {
                    const f32x4 x = src[t4];
#pragma unroll
                    for (int e2 = 0; e2 < 4; ++e2) qr[4 * t4 + e2] = x[e2];
                }
            } else {
                const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(q) + row * kHeadDim);
#pragma unroll
                for (int t8 = 0; t8 < kHeadDim / 8; ++t8) {
                    const u32x4 x = src[t8];
#pragma unroll
                    for (int e2 = 0; e2 < 4; ++e2) {
                        qr[8 * t8 + 2 * e2] = __uint_as_float(x[e2] << 16);
                        qr[8 * t8 + 2 * e2 + 1] = __uint_as_float(x[e2] & 0xFFFF0000u);
                    }
                }
            }
            float ss = 0.f;
#pragma unroll
            for (int t = 0; t < kHeadDim; ++t) {
                ss = fmaf(qr[t], qr[t], ss);
                S.qs[lane][t] = qr[t];
            }
            S.qn[lane] = sqrtf(ss);
            S.cnt[lane] = 0;
        }
        __syncthreads();

        // pass 1: fp32 projections of columns c0 .. c0+ncols-1 for the
        // lane's entry; the next t's R values and q value are loaded before
        // the current t's products
        float p[kRefineCols];
#pragma unroll
        for (int j = 0; j < kRefineCols; ++j) p[j] = 0.f;
        auto pass1 = [&](auto full_tag) {
            constexpr bool FULL = decltype(full_tag)::value;  // ncols == kRefineCols
            const int last = ncols - 1;
            auto col = [&](int j) { return FULL ? j : min(j, last); };
            float rc[kRefineCols], qt = S.qs[lane][0];
#pragma unroll
            for (int j = 0; j < kRefineCols; ++j) rc[j] = Rr[c0 + col(j)];
            for (int t = 0; t < kHeadDim; ++t) {
                const int tn = min(t + 1, kHeadDim - 1);
                float rn[kRefineCols];
                const float* rt = Rr + (size_t)tn * half + c0;
#pragma unroll
                for (int j = 0; j < kRefineCols; ++j) rn[j] = rt[col(j)];
                const float qn = S.qs[lane][tn];
#pragma unroll
                for (int j = 0; j < kRefineCols; ++j) p[j] = fmaf(qt, rc[j], p[j]);
#pragma unroll
                for (int j = 0; j < kRefineCols; ++j) rc[j] = rn[j];
                qt = qn;
            }
        };
        if (ncols == kRefineCols)
            pass1(std::true_type{});
        else if (ncols > 0)
            pass1(std::false_type{});
        float mxl = 0.f;
#pragma unroll
        for (int j = 0; j < kRefineCols; ++j)
            if (j < ncols) mxl = fmaxf(mxl, fabsf(p[j]));
        S.mx[wave][lane] = mxl;
        __syncthreads();
        float mx = 0.f;
#pragma unroll
        for (int w = 0; w < kRefineWaves; ++w) mx = fmaxf(mx, S.mx[w][lane]);
        const float eps = (float)((64.0 * 0x1p-24 * 1.01 + 0x1p-46) * 1.01) * S.qn[lane] * cn;
        const float cut = mx - 2.f * eps;
#pragma unroll
        for (int j = 0; j < kRefineCols; ++j)
            if (j < ncols && fabsf(p[j]) >= cut) {
                const int k = atomicAdd(&S.cnt[lane], 1);
                if (k < kRefineCand) S.cand[lane][k] = c0 + j;
            }
        __syncthreads();

        // pass 2: lane = (entry i, candidate k), four entries per wave
        {
            const int i = wave * (kRefineGroup / kRefineWaves) + lane / kRefineCand;
            const int k = lane % kRefineCand;
            const int ci = S.cnt[i];
            double bv = -__builtin_inf();
            int bi = 0x7FFFFFFF;
            if (ci >= 1 && ci <= kRefineCand && k < ci) {
                const int c = S.cand[i][k];
                // q_t * R_tc is exact in fp64 (at most 48 significant bits), so
                // whether the compiler fuses the multiply into the add or not,
                // the sum rounds exactly as the plain loop does.
                // R's column in runs of 16 values, all of a run's loads in flight together
                double acc = 0.0;
                for (int t0 = 0; t0 < kHeadDim; t0 += 16) {
                    float rcol[16];
#pragma unroll
                    for (int u = 0; u < 16; ++u) rcol[u] = Rr[(size_t)(t0 + u) * half + c];
#pragma unroll
                    for (int u = 0; u < 16; ++u)
                        acc = __dadd_rn(acc, __dmul_rn((double)S.qs[i][t0 + u], (double)rcol[u]));
                }
                better(acc, c, bv, bi);
                better(-acc, half + c, bv, bi);
            }
#pragma unroll
            for (int o = 1; o < kRefineCand; o <<= 1) {
                const double ov = __shfl_xor(bv, o);
                const int oi = __shfl_xor(bi, o);
                better(ov, oi, bv, bi);
            }
            const int ei = g * kRefineGroup + i;
            if (k == 0 && ei < n && ci >= 1 && ci <= kRefineCand) buckets[(int64_t)list[ei] * n_r + r] = bi;
        }

        // entries with too many candidates: every column in fp64, one wave each
        for (int i = wave; i < kRefineGroup; i += kRefineWaves) {
            const int ei = g * kRefineGroup + i;
            const int ci = S.cnt[i];
            if (ei >= n || (ci >= 1 && ci <= kRefineCand)) continue;  // uniform per wave
            double bv = -__builtin_inf();
            int bi = 0x7FFFFFFF;
            for (int c = lane; c < half; c += 64) {
                double acc = 0.0;
                for (int t = 0; t < kHeadDim; ++t)
                    acc = __dadd_rn(acc, __dmul_rn((double)S.qs[i][t], (double)Rr[(size_t)t * half + c]));
                better(acc, c, bv, bi);
                better(-acc, half + c, bv, bi);
            }
            for (int o = 32; o >= 1; o >>= 1) {
                const double ov = __shfl_xor(bv, o);
                const int oi = __shfl_xor(bi, o);
                better(ov, oi, bv, bi);
            }
            if (lane == 0) buckets[(int64_t)list[ei] * n_r + r] = bi;
        }
        __syncthreads();  // the group's LDS is reused by the next one
    }
}

// R streams through LDS in stages of ST tiles (32 ST columns) of one round,
// NP planes, double-buffered: 2 x NP x 32 ST x 128 B, at most 128 KB (one
// plane with ST = 16, two with ST = 8).  ST is the round's tile count
// rounded up to a power of two, capped there, so small rounds compute no
// idle tiles and large ones few barriers.  A stage is copied straight from
// global memory into LDS (buffer loads to LDS, no registers in between)
// while the previous one is consumed, so there is one barrier per stage.  A
// 16-byte piece p of column c sits at slot p ^ stage_swz(c) of the column's
// 128 bytes: the 16 columns read together by one operand load then hit
// distinct banks.
template <int NP, int ST>
struct Stage {
    static constexpr int kCols = 32 * ST;
    static constexpr size_t kBytes = 2ull * NP * kCols * 128;  // both buffers
    static __device__ __forceinline__ uint32_t offset(int buf, int plane, int col) {
        return (uint32_t)(((buf * NP + plane) * kCols + col) * 128);
    }
};

__device__ __forceinline__ int stage_swz(int c) { return (c ^ (c >> 3)) & 7; }

// LDS past the stage buffers: each wave's winners [64 rows][rounds] as
// 16-bit ids.  The stage area is at least as large as the screen's final
// list gathering needs, [rounds][64 WAVES] rows and two counters per round.
__host__ __device__ constexpr size_t hash_win_offset(size_t stage_bytes, int waves, int rounds) {
    const size_t lists = (size_t)rounds * (64 * waves + 2) * 4;
    return ((stage_bytes > lists ? stage_bytes : lists) + 15) / 16 * 16;
}

// The screen's open row-rounds go to kSegs segments per round (workgroup b
// appends to segment b % kSegs), so each list counter sees few atomics.
constexpr int kSegs = 64;

// The screen: waves per SIMD it is built for (three workgroups of four waves
// on a CU, registers and LDS permitting), and its largest stage.
constexpr int kScreenOcc = 3;
constexpr int kScreenMaxTiles = 4;

// Passes of the main kernel.
enum : int {
    kScreen = 0,  // bf16 input: R's hi plane only, every row and round
    kExact = 1,   // both planes (three products for fp32 input), every row and round
    kListed = 2,  // bf16 input: both planes, the rows the screen left open in one round
};

struct Tile {
    f32x16 acc[kRB];
};

// Keys order projections by |projection| truncated to a few bits less than
// fp32's 24 (non-negative floats order like their bit patterns), with an
// index in the bits the truncation frees:
//  * fp32 input: the bit pattern rotated left by one (sign in bit 0,
//    |projection| in bits 5..31, the register j of the tile in bits 1..4):
//    one rotate and one and-or per projection, and the key also carries the
//    winner's sign.  The winner's tile is noted after every tile.
//  * bf16 input: |projection| in bits 6..30 and 16 (t % 4) + j in bits
//    0..5 (tile t of the round), one and-or; the winner's group of four
//    tiles is noted after every fourth tile, and its sign is recomputed once
//    per row and round.
// Keys of tiles past the round are masked to their index, near zero.
template <bool F32, int ST>
constexpr int kKeyTiles = F32 ? 1 : (ST < 4 ? ST : 4);  // tiles sharing one index field

template <bool F32>
__device__ __forceinline__ uint32_t proj_key(float x, int idx, bool live) {
    const uint32_t u = __float_as_uint(x);
    if constexpr (F32) {
        return (__builtin_amdgcn_alignbit(u, u, 31) & (live ? 0xFFFFFFE1u : 0u)) | ((uint32_t)idx << 1);
    } else {
        return (u & (live ? 0x7FFFFFC0u : 0u)) | (uint32_t)idx;
    }
}
template <bool F32>
__device__ __forceinline__ uint32_t key_index(uint32_t key) {
    return F32 ? (key >> 1) & 15u : key & 63u;
}
template <bool F32>
__device__ __forceinline__ float key_magnitude(uint32_t key) {
    return __uint_as_float(F32 ? (key >> 1) & 0x7FFFFFF0u : key & 0x7FFFFFC0u);
}

// Running best b and second best sc (b >= sc) after two more keys: the
// largest of {b, k1, k2} is the new best, the middle one is the largest of
// the rest of those three, and sc joins the rest.  One max3, one med3 and
// one max per two projections.
// (max3 as inline assembly: left to itself the compiler shares max(b, k1)
// with the median and spends a fourth instruction.)
__device__ __forceinline__ void key_update2(uint32_t k1, uint32_t k2, uint32_t& b, uint32_t& sc) {
    const uint32_t mid = max(min(b, k1), min(max(b, k1), k2));  // median of three
    uint32_t top;
    asm("v_max3_u32 %0, %1, %2, %3" : "=v"(top) : "v"(b), "v"(k1), "v"(k2));
    b = top;
    sc = max(sc, mid);
}

// Lane offsets of the NP-plane operand pieces of tiles 0 and 1 inside a
// stage buffer: piece i is k-step i / NP of plane i % NP.  Column 32 t + n
// of tile t sits at 4096 t + 128 n with its pieces in swizzled slots, and
// stage_swz(32 t + n) = stage_swz(n) ^ 4 (t % 2): even tiles share tile 0's
// slot pattern, odd ones tile 1's.
template <int NP, int ST>
__device__ __forceinline__ void piece_offsets(uint32_t (&off)[2][8], int n, int h) {
#pragma unroll
    for (int par = 0; par < 2; ++par)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int s = NP == 2 ? i >> 1 : i;
            const int plane = NP == 2 ? (i & 1) : 0;
            off[par][i] = (uint32_t)(plane * Stage<NP, ST>::kCols * 128 + (32 * par + n) * 128 +
                                     (((4 * h + s) ^ stage_swz(32 * par + n)) << 4));
        }
}

// Products of 16-bit operand words: bf16 planes for fp32 input, binary16
// planes (of scaled q and R) for bf16 input.
template <bool F32>
__device__ __forceinline__ f32x16 mfma_op(u32x4 a, u32x4 b, f32x16 c) {
    if constexpr (F32)
        return mfma32x32x16(as_bf16x8(a), as_bf16x8(b), c);
    else
        return mfma32x32x16(as_f16x8(a), as_f16x8(b), c);
}

// One step of the tile pipeline, in eight slices.  Slice i issues (MF) the
// products of the tile held in `op` into `nxt` for operand piece i (both
// planes; for fp32 input the hi plane also meets q's second plane) or, with
// one plane, for piece i / 2 on even slices; refills that piece with the same
// piece of tile TP (PREF) of the stage at `sb`; and runs one eighth of the
// epilogue of the previous tile `cur`, tile TC of the stage (EPI).  A wave
// issues in order, so this interleaving is what lets the vector ALUs work
// while the matrix core runs; the scheduling barriers keep the compiler from
// regrouping the slices.  Tile numbers are compile-time constants, so the
// operand addresses are a lane offset plus an immediate and the key indices
// are inline constants.
template <bool F32, int NP, int G, bool MF, int TP, int TC>
__device__ __forceinline__ void tile_step(Tile& nxt, u32x4 (&op)[8], const char* __restrict__ sb,
                                          const uint32_t (&poff)[2][8], const u32x4 (&qa)[kRB][4],
                                          const u32x4 (&qm)[kRB][4], const Tile& cur, bool live,
                                          uint32_t (&best)[kRB], uint32_t (&second)[kRB]) {
    static_assert(kRB == 2, "slices written for two row blocks");
    constexpr bool PREF = TP >= 0, EPI = TC >= 0;
    constexpr int idx0 = EPI ? 16 * (TC % G) : 0;
    uint32_t b[kRB] = {best[0], best[1]}, sc[kRB] = {second[0], second[1]};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_barrier(0);
        if (MF && (NP == 2 || (i & 1) == 0)) {
            const int pi = NP == 2 ? i : i >> 1;  // operand piece
            const int s = i >> 1;  // k-step
            const bool hi_plane = NP == 1 || (i & 1) == 0;
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb)
                nxt.acc[rb] = mfma_op<F32>(op[pi], qa[rb][s], pi == 0 ? f32x16{} : nxt.acc[rb]);
            if constexpr (F32) {
                if (hi_plane) {
#pragma unroll
                    for (int rb = 0; rb < kRB; ++rb) nxt.acc[rb] = mfma_op<F32>(op[pi], qm[rb][s], nxt.acc[rb]);
                }
            }
            if constexpr (PREF)
                op[pi] = *reinterpret_cast<const u32x4*>(sb + poff[TP & 1][pi] + (TP & ~1) * 4096);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (EPI) {
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb)
                key_update2(proj_key<F32>(cur.acc[rb][2 * i], idx0 + 2 * i, live),
                            proj_key<F32>(cur.acc[rb][2 * i + 1], idx0 + 2 * i + 1, live), b[rb], sc[rb]);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (EPI) {
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
            best[rb] = b[rb];
            second[rb] = sc[rb];
        }
    }
}

// Source offsets of 1 KB runs of 8 columns (c0 .. c0+7, c0 a multiple of
// 8, stage-local): lane = 8 cl + slot fetches the piece that belongs at LDS
// slot `slot` of column c0 + cl, piece slot ^ stage_swz(c0 + cl).  As
// stage_swz(c0 + cl) = cl ^ (c0 / 8 % 8), the lane's byte offset in the run
// is run_lane_offset(lane) ^ (16 * (c0 / 8 % 8)): one xor per run.
__device__ __forceinline__ uint32_t run_lane_offset(int lane) {
    const int cl = lane >> 3, slot = lane & 7;
    return (uint32_t)(cl * 128 + ((slot ^ cl) << 4));
}

// Raw buffer over one R plane (word 3 of the descriptor: raw, untyped
// 32-bit data as on other CDNA parts); loads past num_records return 0.
constexpr int kRawBufferWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t plane_buffer(const uint16_t* plane, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(plane), 0, (int)bytes, kRawBufferWord3);
}

// One run straight into LDS: a buffer load with the run's column in the
// scalar offset and the lane's piece in the vector offset (no 64-bit vector
// addresses to keep).
__device__ __forceinline__ void copy_run(__amdgpu_buffer_rsrc_t plane, int64_t col0, uint32_t lane_off, int c0,
                                         char* lds_dst) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(plane, (__attribute__((address_space(3))) void*)lds_dst, 16,
                                             lane_off ^ (uint32_t)(((c0 >> 3) & 7) << 4), (uint32_t)(col0 * 128),
                                             0, 0);
}

// Copy global stage g (round g / spr, columns (g % spr) * 32 ST ...) of NP
// planes into buffer buf.  Each wave moves whole 1 KB runs of 8 columns of
// one plane; a run past the round copies the round's first columns instead
// (any valid address: never read).
template <int WAVES, int NP, int ST>
__device__ __forceinline__ void load_stage(char* smem, int buf, int g, int spr, int half_pad,
                                           __amdgpu_buffer_rsrc_t r_hi, __amdgpu_buffer_rsrc_t r_mid, int wave,
                                           uint32_t lane_off) {
    constexpr int kCols = Stage<NP, ST>::kCols;
    constexpr int kRuns = NP * kCols / 8;  // 1 KB runs per stage
    const int r = g / spr, st = g % spr;
#pragma unroll
    for (int i = 0; i < (kRuns + WAVES - 1) / WAVES; ++i) {
        const int run = wave + i * WAVES;  // uniform per wave
        if (kRuns % WAVES == 0 || run < kRuns) {
            const int plane = run / (kCols / 8);
            const int c0 = (run % (kCols / 8)) * 8;
            const int gc0 = st * kCols + c0;
            copy_run(plane ? r_mid : r_hi, (int64_t)r * half_pad + (gc0 < half_pad ? gc0 : 0), lane_off, c0,
                     smem + Stage<NP, ST>::offset(buf, plane, c0));
        }
    }
}

// This lane half's 32 k-values of q . R_col for one binary16 plane: 16 pair
// products in four short chains (fp32 sums of exact products).
__device__ __forceinline__ float dot_planes(const u32x4 (&qa4)[4], const u32x4 (&rv)[4]) {
    typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
    float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t qw = qa4[s4][e], rw = rv[s4][e];
            part[e] = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, qw), __builtin_bit_cast(f16x2, rw), part[e],
                                             false);
        }
    }
    return (part[0] + part[1]) + (part[2] + part[3]);
}

// The tile pipeline of one stage of ST tiles: step T issues tile T's
// products (into ta for even T, tb for odd), prefetches tile T + 1's
// operands and runs the epilogue of tile T - 1; a last step runs tile
// ST - 1's epilogue alone.  ge(t) is called after tile t's epilogue.
template <bool F32, int NP, int ST, int T, class GE>
__device__ __forceinline__ void stage_pipe(Tile& ta, Tile& tb, u32x4 (&op)[8], const char* __restrict__ sb,
                                           const uint32_t (&poff)[2][8], const u32x4 (&qa)[kRB][4],
                                           const u32x4 (&qm)[kRB][4], int nt, uint32_t (&best)[kRB],
                                           uint32_t (&second)[kRB], GE& ge) {
    if constexpr (T < ST) {
        Tile& nxt = T % 2 == 0 ? ta : tb;
        Tile& cur = T % 2 == 0 ? tb : ta;
        tile_step<F32, NP, kKeyTiles<F32, ST>, true, (T + 1 < ST ? T + 1 : -1), T - 1>(
            nxt, op, sb, poff, qa, qm, cur, T - 1 < nt, best, second);
        if constexpr (T >= 1) ge(T - 1);
        stage_pipe<F32, NP, ST, T + 1>(ta, tb, op, sb, poff, qa, qm, nt, best, second, ge);
    } else {
        Tile& cur = (ST - 1) % 2 == 0 ? ta : tb;
        tile_step<F32, NP, kKeyTiles<F32, ST>, false, -1, ST - 1>(cur, op, sb, poff, qa, qm, cur, ST - 1 < nt, best,
                                                                  second);
        ge(ST - 1);
    }
}

// Winner of a row-round as kept in LDS until the row's ids are written:
// the bucket id, or kUnsettled when a later pass must decide.
constexpr uint16_t kUnsettled = 0xFFFFu;

// The main kernel, one of three passes (MODE).  A wave owns 64 rows (two
// 32-row blocks) and sweeps every staged tile once for them.
//  * kScreen and kExact take rows blockIdx.x * 64 * WAVES + ... and all
//    rounds; kListed takes, for round blockIdx.z, the rows the screen left
//    open in that round (its segments one after another), in chunks of
//    64 * WAVES, workgroup blockIdx.x taking every gridDim.x-th chunk.
//  * Every screened projection is within
//        eps = |q| * (res_max[r] + err_acc * max_c |R_c|)
//    of the exact one (res_max: largest 2-norm of R's columns less the
//    planes used, none for fp32 input, whose planes' residual is inside
//    err_acc), and a key's magnitude is low by at most err_pack of it.  For
//    bf16 input the best key's column w is then recomputed, by the screen
//    over the hi plane (within |q| (|R_w - hi_w| + err_acc max_c |R_c|)),
//    by the listed pass over both planes (within eps2, from res_max2 and
//    err_acc2), and the row-round is settled when that value's magnitude
//    less its bound exceeds the second key plus eps; for fp32 input when the
//    best and second keys are more than 2 eps apart.
//    A settled id goes to buckets.  Otherwise the row is appended to the round's list: the
//    screen's lists are segmented, [round][kSegs][seg_cap] with counts
//    [round][kSegs]; the exact passes' are [round][rows] with one count per
//    round (few rows reach them).
template <bool F32, int MODE, int WAVES, int ST>
__global__ __launch_bounds__(WAVES * 64, (MODE == kScreen ? kScreenOcc : 1)) void hash_kernel(
    const void* __restrict__ q, int64_t rows, int n_r, int half, int half_pad,
    const uint16_t* __restrict__ r_hi, const uint16_t* __restrict__ r_mid,
    const float* __restrict__ col_norm_max, const float* __restrict__ res_max, float err_acc,
    const float* __restrict__ res_max2, float err_acc2, float err_pack, const float* __restrict__ col_res,
    int32_t* __restrict__ buckets, const int* __restrict__ list_in,
    const int* __restrict__ count_in, int* __restrict__ list_out, int* __restrict__ count_out,
    int64_t seg_cap) {
    static_assert(!F32 || MODE == kExact, "fp32 input takes the exact pass only");
    constexpr int NP = MODE == kScreen ? 1 : 2;
    constexpr int kWaveRows = 64;
    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63, h = lane >> 5, n = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t run_off = run_lane_offset(lane);
    const uint32_t plane_bytes = (uint32_t)((size_t)n_r * half_pad * kHeadDim * 2);
    const __amdgpu_buffer_rsrc_t rs_hi = plane_buffer(r_hi, plane_bytes), rs_mid = plane_buffer(r_mid, plane_bytes);
    using SG = Stage<NP, ST>;
    const int tpr = half_pad / 32;            // tiles per round
    const int spr = (tpr + ST - 1) / ST;      // stages per round
    const int r_lo = MODE == kListed ? (int)blockIdx.z : 0;
    const int r_end = MODE == kListed ? r_lo + 1 : n_r;
    const int nrb = r_end - r_lo;  // rounds of this block
    // kListed: the round's open rows, segment after segment; lane s holds
    // the end of segment s in that sequence (kSegs is the wave width)
    int64_t listed = 0;
    int seg_end = 0;
    if constexpr (MODE == kListed) {
        static_assert(kSegs == 64, "one segment per lane");
        int incl = count_in[(int64_t)r_lo * kSegs + lane];
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(incl, o);
            if (lane >= o) incl += y;
        }
        seg_end = incl;
        listed = __shfl(incl, 63);
    }
    // kListed: the workgroups take the round's chunks of 64 * WAVES rows in
    // turn; the other passes take one chunk each.
    for (int64_t chunk = blockIdx.x;; chunk += gridDim.x) {
    if (MODE == kListed && chunk * (WAVES * kWaveRows) >= listed) break;  // uniform per block
    const int64_t slot0 = chunk * (WAVES * kWaveRows) + wave * kWaveRows;
    // the row of lane n of row block rb (lane half h keeps row block h's
    // results at the end)
    auto row_of = [&](int rb, bool& valid) -> int64_t {
        const int64_t k = slot0 + rb * 32 + n;
        if constexpr (MODE == kListed) {
            valid = k < listed;
            // segment of entry k: the first s with seg_end[s] > k (binary
            // search over the lanes; every lane takes part in the shuffles)
            const int kk = (int)min(k, max(listed - 1, (int64_t)0));
            int sg = 0;
#pragma unroll
            for (int step = 32; step >= 1; step >>= 1)
                if (__shfl(seg_end, sg + step - 1) <= kk) sg += step;
            sg = min(sg, 63);
            const int before = __shfl(seg_end, max(sg - 1, 0));
            const int64_t at = ((int64_t)r_lo * kSegs + sg) * seg_cap + (kk - (sg > 0 ? before : 0));
            return valid ? list_in[at] : 0;
        } else {
            valid = k < rows;
            return valid ? k : 0;
        }
    };
    // this wave's winners: [row in wave][round of the block]
    uint16_t* win = reinterpret_cast<uint16_t*>(smem + hash_win_offset(SG::kBytes, WAVES, nrb)) +
                    (size_t)wave * kWaveRows * nrb;

    load_stage<WAVES, NP, ST>(smem, 0, r_lo * spr, spr, half_pad, rs_hi, rs_mid, wave, run_off);

    // Queries as the B operand: lane holds row (n) and k = 32h + 8s + e, s = 0..3.
    u32x4 qa[kRB][4];
    u32x4 qm[kRB][4];  // fp32 input: second bf16 plane of q
    float qn[kRB];
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
        bool valid;
        const int64_t row = row_of(rb, valid);
        float ss = 0.f;
        if constexpr (F32) {
            const float* src = static_cast<const float*>(q) + row * kHeadDim + 32 * h;
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                f32x4 x0 = valid ? *reinterpret_cast<const f32x4*>(src + 8 * s4) : f32x4{0, 0, 0, 0};
                f32x4 x1 = valid ? *reinterpret_cast<const f32x4*>(src + 8 * s4 + 4) : f32x4{0, 0, 0, 0};
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
                qa[rb][s4] = hi;
                qm[rb][s4] = mid;
            }
        } else {
            // The row times 2^sq, with its largest |q_t| brought into
            // [2^14, 2^15): exact in fp32, and in binary16 for every value
            // from fp16's smallest normal 2^-14 up (bf16 has 8 significant
            // bits); smaller values are dropped, |delta q| <= 8 * 2^-14.
            const uint16_t* src = static_cast<const uint16_t*>(q) + row * kHeadDim + 32 * h;
            u32x4 raw[4];
            float mx = 0.f;
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                raw[s4] = valid ? *reinterpret_cast<const u32x4*>(src + 8 * s4) : u32x4{0, 0, 0, 0};
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    mx = fmaxf(mx, fmaxf(fabsf(__uint_as_float(raw[s4][e] << 16)),
                                         fabsf(__uint_as_float(raw[s4][e] & 0xFFFF0000u))));
            }
            mx = max_xor32(mx);
            int k = 0;
            (void)frexpf(mx, &k);
            const int sq = (mx > 0.f && mx <= 3.4e38f) ? 14 - (k - 1) : 0;
            const float f1 = __uint_as_float((uint32_t)(127 + sq / 2) << 23);
            const float f2 = __uint_as_float((uint32_t)(127 + sq - sq / 2) << 23);
            auto to_f16 = [&](float x) {
                const float xs = x * f1 * f2;
                ss = fmaf(xs, xs, ss);
                return fabsf(xs) < 0x1p-14f ? 0.f : xs;
            };
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                u32x4 w;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    w[e] = pack_f16x2(to_f16(__uint_as_float(raw[s4][e] << 16)),
                                      to_f16(__uint_as_float(raw[s4][e] & 0xFFFF0000u)));
                qa[rb][s4] = w;
                qm[rb][s4] = u32x4{0, 0, 0, 0};
            }
        }
        ss = sum_xor32(ss);
        qn[rb] = sqrtf(ss);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    uint32_t poff[2][8];
    piece_offsets<NP, ST>(poff, n, h);
    constexpr int G = kKeyTiles<F32, ST>;
    // best and second key, the best key before the current group of G
    // tiles, and the group the best key came from
    uint32_t best[kRB], second[kRB], grp_start[kRB];
    int best_grp[kRB];
    const int g_end = r_end * spr;
    for (int g = r_lo * spr; g < g_end; ++g) {
        const int r = g / spr, st = g % spr, buf = (g - r_lo * spr) & 1;
        if (st == 0) {
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb) {
                best[rb] = second[rb] = grp_start[rb] = 0u;
                best_grp[rb] = 0;
            }
        }
        // the next stage lands in the other buffer while this one computes
        if (g + 1 < g_end)
            load_stage<WAVES, NP, ST>(smem, buf ^ 1, g + 1, spr, half_pad, rs_hi, rs_mid, wave, run_off);
        const char* sb = smem + SG::offset(buf, 0, 0);
        const int nt = min(ST, tpr - st * ST);
        const int t0 = st * ST;
        // after the epilogue of stage tile tc: note the group if it ends there
        // (stages start on group boundaries: G divides ST)
        auto group_end = [&](int tc) {
            if ((tc + 1) % G == 0) {
#pragma unroll
                for (int rb = 0; rb < kRB; ++rb) {
                    best_grp[rb] = best[rb] != grp_start[rb] ? (t0 + tc) / G : best_grp[rb];
                    grp_start[rb] = best[rb];
                }
            }
        };
        // Every stage runs all ST tiles; tiles past the round (a last,
        // partial stage) compute on stale LDS and their keys are masked to
        // (near) zero, so they can only win when every key is tiny, and such
        // a row is left to the exact passes.
        {
            Tile ta, tb;
            u32x4 op[8];
#pragma unroll
            for (int i = 0; i < 4 * NP; ++i) op[i] = *reinterpret_cast<const u32x4*>(sb + poff[0][i]);
            stage_pipe<F32, NP, ST, 0>(ta, tb, op, sb, poff, qa, qm, nt, best, second, group_end);
        }

        if (st == spr - 1) {
            // Round epilogue: merge the two lane halves (different columns of
            // the same row) and decide; lane half h keeps row block h's result.
            const float cn = col_norm_max[r];
            const float res = F32 ? 0.f : res_max[r];
            uint32_t bk[kRB], sk[kRB];
            int col[kRB];
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb) {
                const uint32_t bb = best[rb], ss2 = second[rb];
                const uint32_t bp = xor32(bb), sp = xor32(ss2);
                const int tp = (int)xor32((uint32_t)best_grp[rb]);
                const bool mine = bb > bp || (bb == bp && h == 0);
                bk[rb] = mine ? bb : bp;
                sk[rb] = max(min(bb, bp), max(ss2, sp));
                const int hw = mine ? h : (h ^ 1);
                const int gw = mine ? best_grp[rb] : tp;
                const uint32_t idx = key_index<F32>(bk[rb]), j = idx & 15u;
                const int tw = gw * G + (int)(idx >> 4);  // tile of the round
                col[rb] = tw * 32 + 8 * (int)(j >> 2) + 4 * hw + (int)(j & 3u);
            }
            if constexpr (F32) {
                // Every screened key is within eps of its exact |projection|;
                // an exchange of winners needs a gap <= 2 eps.  When the gap is
                // larger the winner's magnitude exceeds eps, so the screened
                // sign (bit 0 of the key) is the exact one.
#pragma unroll
                for (int rb = 0; rb < kRB; ++rb) {
                    const float b1 = key_magnitude<F32>(bk[rb]), s1 = key_magnitude<F32>(sk[rb]);
                    const float thr = 2.04f * (qn[rb] * (res + err_acc * cn) + err_pack * b1);
                    const bool flag = !(b1 - s1 > thr) || col[rb] >= half;
                    const int id = (bk[rb] & 1u) ? half + col[rb] : col[rb];
                    if (rb == h) win[(rb * 32 + n) * nrb + (r - r_lo)] = flag ? kUnsettled : (uint16_t)id;
                }
            } else {
                // x = q_row . R_col of the best key's column (fp32 sums of
                // the exact products; each lane half adds its 32 k-values).
                // Every other column's exact |projection| is at most the
                // second key (raised by the truncated bits) plus the pass's
                // eps, so the winner is certain when |x| less x's own error
                // bound exceeds that, and its sign is x's.  A flagged winner
                // may sit past the round; any valid column stands in.
                //  * The screen takes x over the hi plane alone: within
                //    eps_w = |q| (|R_w - hi_w| + err_acc max_c |R_c|) for the
                //    winner's column w.  Rows it leaves open go to the listed
                //    pass, which costs less than the mid plane's loads here.
                //  * The listed pass takes x over both planes, within eps2.
                // The pieces come from global memory (the planes are small
                // and stay in the caches).
                constexpr bool kHiOnly = MODE == kScreen;
                u32x4 hv[kRB][4], mv[kRB][4];
                // Lane half h keeps only row block h's decision, so it needs
                // only that winner's residual: one gather (a 4-byte gather
                // costs the address unit as much as a 16-byte one), issued
                // first, with the planes' (left to itself the compiler issues
                // it after the first block's products and waits on it).
                float res_own = 0.f;
                if constexpr (kHiOnly)
                    res_own = col_res[(size_t)r * half_pad + min(h ? col[1] : col[0], half_pad - 1)];
#pragma unroll
                for (int rb = 0; rb < kRB; ++rb) {
                    const int cc = min(col[rb], half_pad - 1);
                    const size_t o = ((size_t)r * half_pad + cc) * kHeadDim + 32 * h;
                    const u32x4* ph = reinterpret_cast<const u32x4*>(r_hi + o);
                    const u32x4* pm = reinterpret_cast<const u32x4*>(r_mid + o);
#pragma unroll
                    for (int s4 = 0; s4 < 4; ++s4) {
                        hv[rb][s4] = ph[s4];
                        if constexpr (!kHiOnly) mv[rb][s4] = pm[s4];
                    }
                }
                if constexpr (kHiOnly) asm volatile("" : "+v"(res_own));
#pragma unroll
                for (int rb = 0; rb < kRB; ++rb) {
                    float half_x = dot_planes(qa[rb], hv[rb]);
                    if constexpr (!kHiOnly) half_x += dot_planes(qa[rb], mv[rb]);
                    const float x = sum_xor32(half_x);
                    const float s1 = key_magnitude<F32>(sk[rb]);
                    const float eps = 1.02f * qn[rb] * (res + err_acc * cn);
                    const float eps_x = kHiOnly ? 1.02f * qn[rb] * (res_own + err_acc * cn)  // kept for rb == h
                                                : 1.02f * qn[rb] * (res_max2[r] + err_acc2 * cn);
                    const bool flag = !(fabsf(x) - eps_x > s1 * (1.f + 2.f * err_pack) + eps) || col[rb] >= half;
                    const int id = x < 0.f ? half + col[rb] : col[rb];
                    if (rb == h) win[(rb * 32 + n) * nrb + (r - r_lo)] = flag ? kUnsettled : (uint16_t)id;
                }
            }
        }
        // the next stage has landed and every wave is done with this buffer
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    }

    // Write each row's ids and queue the row-rounds left open.
    bool valid;
    const int64_t row = row_of(h, valid);
    const uint16_t* w = win + (h * 32 + n) * nrb;
    if constexpr (MODE == kScreen) {
        // Gather the block's open rows per round in LDS (the stage buffers
        // are free now), then reserve room in this block's segment with one
        // atomic per round and copy them out.
        int* lq = reinterpret_cast<int*>(smem);            // [nrb][WAVES * 64]
        int* lcnt = lq + nrb * WAVES * kWaveRows;          // [nrb]
        int* lbase = lcnt + nrb;                           // [nrb]
        if (tid < nrb) lcnt[tid] = 0;
        __syncthreads();
        for (int rr = 0; rr < nrb; ++rr) {
            const uint16_t id = w[rr];
            const bool queue = valid && id == kUnsettled;
            if (valid) buckets[row * n_r + r_lo + rr] = id == kUnsettled ? 0 : (int32_t)id;
            const uint64_t qmask = __ballot(queue);
            if (qmask) {
                const int leader = __ffsll((unsigned long long)qmask) - 1;
                int lslot = 0;
                if (lane == leader) lslot = atomicAdd(&lcnt[rr], __popcll(qmask));
                lslot = __shfl(lslot, leader);
                if (queue) lq[rr * WAVES * kWaveRows + lslot + __popcll(qmask & ((1ull << lane) - 1ull))] = (int)row;
            }
        }
        __syncthreads();
        const int64_t seg = blockIdx.x % kSegs;
        if (tid < nrb) lbase[tid] = lcnt[tid] > 0 ? atomicAdd(&count_out[(int64_t)(r_lo + tid) * kSegs + seg], lcnt[tid]) : 0;
        __syncthreads();
        for (int rr = 0; rr < nrb; ++rr) {
            int* dst = list_out + ((int64_t)(r_lo + rr) * kSegs + seg) * seg_cap + lbase[rr];
            for (int i = tid; i < lcnt[rr]; i += WAVES * 64) dst[i] = lq[rr * WAVES * kWaveRows + i];
        }
    } else {
        for (int rr = 0; rr < nrb; ++rr) {
            const int r = r_lo + rr;
            const uint16_t id = w[rr];
            const bool queue = valid && id == kUnsettled;
            if (valid) buckets[row * n_r + r] = id == kUnsettled ? 0 : (int32_t)id;
            // wave-aggregated append to this round's list
            const uint64_t qmask = __ballot(queue);
            if (qmask) {
                int* list = list_out + rows * r;
                const int leader = __ffsll((unsigned long long)qmask) - 1;
                int lslot = 0;
                if (lane == leader) lslot = atomicAdd(&count_out[r], __popcll(qmask));
                lslot = __shfl(lslot, leader);
                if (queue) list[lslot + __popcll(qmask & ((1ull << lane) - 1ull))] = (int)row;
            }
        }
    }
    if (MODE != kListed) break;
    __syncthreads();  // the next chunk restages R over the buffers just read
    }
}

struct HashWs {
    uint16_t* r_hi;
    uint16_t* r_mid;
    float* col_norm;  // [3][n_r][half_pad]: |R_c|, |R_c - hi_c|, |R_c - hi_c - mid_c|
    float* norm_max;  // [3][n_r]: the largest of each
    int* r_exp;       // [n_r]: binary16 planes hold R * 2^r_exp (bf16 input)
    float* r_part;    // [n_r][kScaleParts]: partial maxima of |R|
    int* count;       // [n_r][kSegs] rows left open by the screen, then [n_r] by the exact passes
    int* list1;       // [n_r][kSegs][seg_cap]
    int* list2;       // [n_r][rows]
    int64_t seg_cap;
    size_t bytes;
};

constexpr int kHashWaves = 4;
constexpr int64_t kRowsPerBlock = kHashWaves * 64;

HashWs carve(void* base, int64_t rows, int n_rounds, int half_pad) {
    const size_t per = (size_t)n_rounds * half_pad * kHeadDim;
    const int64_t blocks = (rows + kRowsPerBlock - 1) / kRowsPerBlock;
    char* p = static_cast<char*>(base);
    HashWs w{};
    w.seg_cap = (blocks + kSegs - 1) / kSegs * kRowsPerBlock;
    size_t off = 0;
    w.r_hi = reinterpret_cast<uint16_t*>(p + off);
    off += align256(per * 2);
    w.r_mid = reinterpret_cast<uint16_t*>(p + off);
    off += align256(per * 2);
    w.col_norm = reinterpret_cast<float*>(p + off);
    off += align256((size_t)3 * n_rounds * half_pad * 4);
    w.norm_max = reinterpret_cast<float*>(p + off);
    off += align256((size_t)3 * n_rounds * 4);
    w.r_exp = reinterpret_cast<int*>(p + off);
    off += align256((size_t)n_rounds * 4);
    w.r_part = reinterpret_cast<float*>(p + off);
    off += align256((size_t)n_rounds * kScaleParts * 4);
    w.count = reinterpret_cast<int*>(p + off);
    off += align256((size_t)n_rounds * (kSegs + 1) * 4);
    w.list1 = reinterpret_cast<int*>(p + off);
    off += align256((size_t)n_rounds * kSegs * w.seg_cap * 4);
    w.list2 = reinterpret_cast<int*>(p + off);
    off += align256((size_t)n_rounds * rows * 4);
    w.bytes = off;
    return w;
}

// Arguments of one pass of hash_kernel.
struct PassArgs {
    const void* q;
    int64_t rows;
    int n_r, half, half_pad;
    const uint16_t *r_hi, *r_mid;
    const float *cn_max, *res;
    float err_acc;
    const float* res2;
    float err_acc2, err_pack;
    const float* col_res;
    int32_t* buckets;
    const int *list_in, *count_in;
    int *list_out, *count_out;
    int64_t seg_cap;
};

template <bool F32, int MODE, int WAVES, int ST>
void launch_pass_st(const PassArgs& a, dim3 grid, int rounds, hipStream_t stream) {
    constexpr int NP = MODE == kScreen ? 1 : 2;
    const size_t lds = hash_win_offset(Stage<NP, ST>::kBytes, WAVES, rounds) + (size_t)WAVES * 64 * rounds * 2;
    auto* k = &hash_kernel<F32, MODE, WAVES, ST>;
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    k<<<grid, WAVES * 64, lds, stream>>>(a.q, a.rows, a.n_r, a.half, a.half_pad, a.r_hi, a.r_mid, a.cn_max, a.res,
                                         a.err_acc, a.res2, a.err_acc2, a.err_pack, a.col_res, a.buckets, a.list_in,
                                         a.count_in, a.list_out, a.count_out, a.seg_cap);
}

// Tiles per stage: the round's tile count rounded up to a power of two, at
// most kScreenMaxTiles for the screen (one plane), 8 for the fp32 pass (two
// planes) and 2 for the listed pass (two planes: 240 registers, two waves a
// SIMD; four tiles take 337, one wave a SIMD, and were slower).
template <bool F32, int MODE, int WAVES>
void launch_pass(const PassArgs& a, dim3 grid, int rounds, hipStream_t stream) {
    constexpr int kMax = MODE == kScreen ? kScreenMaxTiles : (MODE == kListed ? 2 : 8);
    const int tpr = a.half_pad / 32;
    if (tpr <= 1)
        launch_pass_st<F32, MODE, WAVES, 1>(a, grid, rounds, stream);
    else if (tpr <= 2 || kMax == 2)
        launch_pass_st<F32, MODE, WAVES, 2>(a, grid, rounds, stream);
    else if (tpr <= 4 || kMax == 4) {
        if constexpr (kMax >= 4) launch_pass_st<F32, MODE, WAVES, 4>(a, grid, rounds, stream);
    }
    else if (tpr <= 8 || kMax == 8) {
        if constexpr (kMax >= 8) launch_pass_st<F32, MODE, WAVES, 8>(a, grid, rounds, stream);
    } else {
        if constexpr (kMax >= 16) launch_pass_st<F32, MODE, WAVES, 16>(a, grid, rounds, stream);
    }
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
    const float* cn_max = w.norm_max;                       // max |R_c|
    const float* res1_max = w.norm_max + n_rounds;          // max |R_c - hi_c|
    const float* res2_max = w.norm_max + 2 * n_rounds;      // max |R_c - hi_c - mid_c|
    int* count1 = w.count;                                  // [n_r][kSegs]: left open by the screen
    int* count2 = w.count + (size_t)n_rounds * kSegs;       // [n_r]: left to the fp64 refinement

    if (f32) {
        prep_r_cols_kernel<false><<<dim3(half_pad, n_rounds), 64, 0, stream>>>(
            R, half, half_pad, nullptr, nullptr, w.r_hi, w.r_mid, w.col_norm);
    } else {
        prep_r_part_kernel<<<dim3(kScaleParts, n_rounds), 256, 0, stream>>>(R, half, w.r_part);
        prep_r_cols_kernel<true><<<dim3(half_pad, n_rounds), 64, 0, stream>>>(
            R, half, half_pad, w.r_part, w.r_exp, w.r_hi, w.r_mid, w.col_norm);
    }
    prep_r_max_kernel<<<dim3(n_rounds, 3), 256, 0, stream>>>(w.col_norm, n_rounds, half_pad, w.norm_max,
                                                             w.count, n_rounds * (kSegs + 1));
    if (rows == 0) return hipGetLastError();

    // Error of a screened key against the exact |projection| p_c, beyond the
    // planes' residual q . (R_c - planes) <= |q| |R_c - planes|:
    //  * fp32 accumulation of the exact 16-bit products, <= one ulp of the
    //    partial sum (<= 2^-23 sum_t |q_t R_tc|) per addition;
    //  * for bf16 input, the scaled q's values below 2^-14 that binary16
    //    drops: |delta q| <= 8 * 2^-14 <= 2^-25 |q| (|q| >= 2^14 scaled);
    //  * for fp32 input, q's own residual after two bf16 planes and R's
    //    after two (<= 3.1 * 2^-16 sum_t |q_t R_tc| together);
    //  * the index bits written over the low mantissa, < 2^-19 |key| for
    //    fp32 input (4 bits), < 2^-17 |key| for bf16 input (6 bits).
    // sum_t |q_t R_tc| <= |q| |R_c| (Cauchy-Schwarz) <= |q| max_c |R_c|.
    const float err_pack = f32 ? (float)0x1p-19 : (float)0x1p-17;
    const float acc1 = (float)((kHeadDim * 0x1p-23 + 0x1p-25) * 1.01);
    const float acc2 = (float)((2 * kHeadDim * 0x1p-23 + 0x1p-25) * 1.01);
    const float acc_f32 = (float)((3.1 * 0x1p-16 + 3 * kHeadDim * 0x1p-23) * 1.01);

    constexpr int kWaves = kHashWaves;
    const unsigned grid = (unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock);
    // Refinement blocks per round: a typical list holds well under 1% of the
    // rows, a few groups of 64 per round; longer lists are strided.
    const unsigned refine_blocks =
        (unsigned)std::max<int64_t>(1, std::min<int64_t>(256, (rows + kRefineGroup - 1) / kRefineGroup));
    if (f32) {
        launch_pass<true, kExact, kWaves>(
            PassArgs{q, rows, n_rounds, half, half_pad, w.r_hi, w.r_mid, cn_max, nullptr, acc_f32, nullptr, 0.f,
                     err_pack, nullptr, buckets, nullptr, nullptr, w.list2, count2, 0},
            dim3(grid), n_rounds, stream);
        hash_refine_kernel<true><<<dim3(refine_blocks, n_rounds), kRefineThreads, 0, stream>>>(
            q, R, half, n_rounds, rows, w.list2, count2, cn_max, nullptr, buckets);
    } else {
        // screen with R's hi plane; the rows it leaves open get both planes;
        // what those leave open gets the fp64 refinement
        launch_pass<false, kScreen, kWaves>(
            PassArgs{q, rows, n_rounds, half, half_pad, w.r_hi, w.r_mid, cn_max, res1_max, acc1, res2_max, acc2,
                     err_pack, w.col_norm + (size_t)n_rounds * half_pad, buckets, nullptr, nullptr, w.list1, count1,
                     w.seg_cap},
            dim3(grid), n_rounds, stream);
        // Four waves a workgroup.  Deciding from the hi plane alone, the
        // screen leaves about 1.5% of row-rounds open on Gaussian data:
        // 128 workgroups per round cover 128 * 256 open rows, 3.1% of 1M
        // rows; longer lists loop.
        constexpr int kListedWaves = 4;
        const int64_t listed_rows = kListedWaves * 64;
        const unsigned per_round = (unsigned)std::min<int64_t>(128, (rows + listed_rows - 1) / listed_rows);
        launch_pass<false, kListed, kListedWaves>(
            PassArgs{q, rows, n_rounds, half, half_pad, w.r_hi, w.r_mid, cn_max, res2_max, acc2, res2_max, acc2,
                     err_pack, nullptr, buckets, w.list1, count1, w.list2, count2, w.seg_cap},
            dim3(per_round, 1, n_rounds), 1, stream);
        hash_refine_kernel<false><<<dim3(refine_blocks, n_rounds), kRefineThreads, 0, stream>>>(
            q, R, half, n_rounds, rows, w.list2, count2, cn_max, w.r_exp, buckets);
    }
    return hipGetLastError();
}

}  // namespace lsh

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
//    argmax index rides in the low mantissa bits of the key, so one
//    bit-insert, one max and one median-of-three per projection suffice.
//  * If the gap between the best and second-best key cannot rule out an
//    exchange under the error bound, the row-round is recomputed exactly in
//    fp64 (same product and summation order as a plain loop), so the ids
//    always equal the exact argmax.
#include "common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr int kHashWaves = 4;
constexpr int kHashRowsPerBlock = 64 * kHashWaves;  // each wave: two 32-row blocks
constexpr int kColStride = 72;                      // bf16 per staged R column (64 + pad)
constexpr int kMaxColsPerLane = 16;                 // exact path: n_b/2 <= 1024

// R [n_r][64][half] fp32 -> bf16 planes hi/mid and an fp32 copy, all
// [n_r][half_pad][64] (one R column contiguous), zero-padded to half_pad
// columns, plus the largest column 2-norm of each round.
__global__ __launch_bounds__(256) void prep_r_kernel(const float* __restrict__ R, int half,
                                                     int half_pad, uint16_t* __restrict__ r_hi,
                                                     uint16_t* __restrict__ r_mid,
                                                     float* __restrict__ r_t,
                                                     float* __restrict__ col_norm_max) {
    const int r = blockIdx.x;
    __shared__ float red[256];
    float mx = 0.f;
    for (int c = threadIdx.x; c < half_pad; c += blockDim.x) {
        float ss = 0.f;
        for (int t = 0; t < kHeadDim; ++t) {
            const float x = c < half ? R[((size_t)r * kHeadDim + t) * half + c] : 0.f;
            const uint32_t hi = f32_to_bf16_bits(x);
            const float res = x - bf16_bits_to_f32(hi);  // exact (Sterbenz)
            const uint32_t mid = f32_to_bf16_bits(res);
            const size_t o = ((size_t)r * half_pad + c) * kHeadDim + t;
            r_hi[o] = (uint16_t)hi;
            r_mid[o] = (uint16_t)mid;
            r_t[o] = x;
            ss = fmaf(x, x, ss);
        }
        mx = fmaxf(mx, sqrtf(ss));
    }
    red[threadIdx.x] = mx;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    if (threadIdx.x == 0) col_norm_max[r] = red[0];
}

template <bool F32>
__device__ __forceinline__ float q_value(const void* q, int64_t row, int k) {
    if constexpr (F32) {
        return static_cast<const float*>(q)[row * kHeadDim + k];
    } else {
        return bf16_bits_to_f32(static_cast<const uint16_t*>(q)[row * kHeadDim + k]);
    }
}

// Exact argmax of [xR; -xR] for one row-round, computed by the whole wave in
// fp64: column c's projection is the left-to-right sum over t of the exact
// products q_t * R_tc.  Ties go to the first index.  Returns the bucket.
template <bool F32>
__device__ int exact_bucket(const void* q, int64_t row, const float* __restrict__ r_t_round,
                            int half) {
    const int lane = lane_id();
    const float qv = q_value<F32>(q, row, lane);
    double p[kMaxColsPerLane];
#pragma unroll
    for (int k = 0; k < kMaxColsPerLane; ++k) p[k] = 0.0;
    for (int t = 0; t < kHeadDim; ++t) {
        const double qt = (double)__shfl(qv, t);
#pragma unroll
        for (int k = 0; k < kMaxColsPerLane; ++k) {
            const int c = lane + 64 * k;
            if (c < half) p[k] = __dadd_rn(p[k], __dmul_rn(qt, (double)r_t_round[(size_t)c * kHeadDim + t]));
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
    return bi;
}

template <bool F32>
__global__ __launch_bounds__(256, 2) void hash_kernel(
    const void* __restrict__ q, int64_t rows, int n_r, int half, int half_pad,
    const uint16_t* __restrict__ r_hi, const uint16_t* __restrict__ r_mid,
    const float* __restrict__ r_t, const float* __restrict__ col_norm_max, float thr_coef,
    int idx_bits, int32_t* __restrict__ buckets) {
    __shared__ __attribute__((aligned(16))) uint16_t stage[2][2][64][kColStride];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6, h = lane >> 5, n = lane & 31;
    const int64_t row0 = (int64_t)blockIdx.x * kHashRowsPerBlock + wave * 64;

    // Queries as the B operand: lane holds row (n) and k = 32h + 8s + e, s = 0..3.
    bf16x8 qa[2][4];
    bf16x8 qm[2][4];  // fp32 input: second bf16 plane of q
    float qn[2];
    bool valid[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
        const int64_t row = row0 + rb * 32 + n;
        valid[rb] = row < rows;
        float ss = 0.f;
        if constexpr (F32) {
            const float* src = static_cast<const float*>(q) + row * kHeadDim + 32 * h;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                f32x4 x0 = valid[rb] ? *reinterpret_cast<const f32x4*>(src + 8 * s) : f32x4{0, 0, 0, 0};
                f32x4 x1 = valid[rb] ? *reinterpret_cast<const f32x4*>(src + 8 * s + 4) : f32x4{0, 0, 0, 0};
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
                const u32x4 raw = valid[rb] ? *reinterpret_cast<const u32x4*>(src + 8 * s) : u32x4{0, 0, 0, 0};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float a = __uint_as_float(raw[e] << 16), b = __uint_as_float(raw[e] & 0xFFFF0000u);
                    ss = fmaf(a, a, ss);
                    ss = fmaf(b, b, ss);
                }
                qa[rb][s] = as_bf16x8(raw);
            }
        }
        ss += __shfl_xor(ss, 32);
        qn[rb] = sqrtf(ss);
    }

    const uint32_t idx_mask = (1u << idx_bits) - 1u;
    const int n_tiles = half_pad / 32;
    const int n_stages = (n_tiles + 1) / 2;

    for (int r = 0; r < n_r; ++r) {
        const uint16_t* hi_r = r_hi + (size_t)r * half_pad * kHeadDim;
        const uint16_t* mid_r = r_mid + (size_t)r * half_pad * kHeadDim;
        float best[2] = {0.f, 0.f}, second[2] = {0.f, 0.f};

        // Stage loader: 2 planes x 64 columns x 128 B = 1024 x 16 B per stage.
        u32x4 pre[4];
        auto gload = [&](int st) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int idx = tid + 256 * i;
                const int plane = idx >> 9, col = (idx >> 3) & 63, part = idx & 7;
                const int gcol = st * 64 + col;
                const uint16_t* base = plane ? mid_r : hi_r;
                pre[i] = gcol < half_pad
                             ? *reinterpret_cast<const u32x4*>(base + (size_t)gcol * kHeadDim + part * 8)
                             : u32x4{0, 0, 0, 0};
            }
        };
        auto lstore = [&](int buf) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int idx = tid + 256 * i;
                const int plane = idx >> 9, col = (idx >> 3) & 63, part = idx & 7;
                *reinterpret_cast<u32x4*>(&stage[buf][plane][col][part * 8]) = pre[i];
            }
        };

        gload(0);
        lstore(0);
        __syncthreads();
        for (int st = 0; st < n_stages; ++st) {
            if (st + 1 < n_stages) gload(st + 1);
            const int buf = st & 1;
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) {
                const int tile = st * 2 + tt;
                if (tile < n_tiles) {
                    bf16x8 ahi[4], amid[4];
#pragma unroll
                    for (int s = 0; s < 4; ++s) {
                        ahi[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(&stage[buf][0][tt * 32 + n][32 * h + 8 * s]));
                        amid[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(&stage[buf][1][tt * 32 + n][32 * h + 8 * s]));
                    }
                    const uint32_t ubase = (uint32_t)tile << 4;
#pragma unroll
                    for (int rb = 0; rb < 2; ++rb) {
                        f32x16 acc = {};
#pragma unroll
                        for (int s = 0; s < 4; ++s) {
                            acc = mfma32x32x16(ahi[s], qa[rb][s], acc);
                            acc = mfma32x32x16(amid[s], qa[rb][s], acc);
                            if constexpr (F32) acc = mfma32x32x16(ahi[s], qm[rb][s], acc);
                        }
                        float b = best[rb], sc = second[rb];
#pragma unroll
                        for (int j = 0; j < 16; ++j) {
                            const float key = fabsf(__uint_as_float((__float_as_uint(acc[j]) & ~idx_mask) | (ubase | (uint32_t)j)));
                            sc = __builtin_amdgcn_fmed3f(key, b, sc);
                            b = fmaxf(key, b);
                        }
                        best[rb] = b;
                        second[rb] = sc;
                    }
                }
            }
            if (st + 1 < n_stages) lstore((st + 1) & 1);
            __syncthreads();
        }

        // Round epilogue: merge the two lane halves (different columns of the
        // same row), decide, and settle close calls exactly.
        const float cn = col_norm_max[r];
        const float* r_t_round = r_t + (size_t)r * half_pad * kHeadDim;
        bool flag[2];
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
            const int64_t row = row0 + rb * 32 + n;
            const float bp = __shfl_xor(best[rb], 32), sp = __shfl_xor(second[rb], 32);
            const bool mine = best[rb] > bp || (best[rb] == bp && h == 0);
            const float b1 = mine ? best[rb] : bp;
            const float s1 = fmaxf(fminf(best[rb], bp), fmaxf(second[rb], sp));
            const int hw = mine ? h : (h ^ 1);
            const uint32_t u = __float_as_uint(b1) & idx_mask;
            const int col = (int)(u >> 4) * 32 + 8 * (int)((u & 15u) >> 2) + 4 * hw + (int)(u & 3u);
            const float thr = thr_coef * qn[rb] * cn;
            flag[rb] = !(b1 - s1 > thr) || col >= half;
            // Sign of the winning projection.  When the row is not flagged its
            // magnitude exceeds the error bound, so fp32 gets the sign right.
            const int colc = col < half ? col : 0;
            const float* rt = r_t_round + (size_t)colc * kHeadDim + 32 * h;
            float part = 0.f;
            if (valid[rb]) {
                for (int k = 0; k < 32; ++k) part = fmaf(q_value<F32>(q, row, 32 * h + k), rt[k], part);
            }
            const float p = part + __shfl_xor(part, 32);
            if (valid[rb] && h == 0 && !flag[rb]) buckets[row * n_r + r] = p > 0.f ? col : half + col;
        }
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
            uint64_t fl = __ballot(flag[rb] && valid[rb] && h == 0);
            while (fl) {
                const int src = __ffsll((unsigned long long)fl) - 1;
                fl &= fl - 1;
                const int64_t frow = row0 + rb * 32 + src;
                const int bkt = exact_bucket<F32>(q, frow, r_t_round, half);
                if (lane == 0) buckets[frow * n_r + r] = bkt;
            }
        }
    }
}

int ceil_log2(int x) {
    int b = 0;
    while ((1 << b) < x) ++b;
    return b;
}

}  // namespace

size_t hash_workspace_bytes(int n_rounds, int n_buckets) {
    const size_t half_pad = (size_t)((n_buckets / 2 + 31) / 32) * 32;
    const size_t per = (size_t)n_rounds * half_pad * kHeadDim;
    return align256(per * 2) * 2 + align256(per * 4) + align256((size_t)n_rounds * 4);
}

hipError_t launch_hash(const void* q, bool f32, int64_t rows, int n_rounds, int n_buckets,
                       const float* R, int32_t* buckets, void* workspace, hipStream_t stream) {
    const int half = n_buckets / 2;
    const int half_pad = (half + 31) / 32 * 32;
    const size_t per = (size_t)n_rounds * half_pad * kHeadDim;
    char* ws = static_cast<char*>(workspace);
    uint16_t* r_hi = reinterpret_cast<uint16_t*>(ws);
    uint16_t* r_mid = reinterpret_cast<uint16_t*>(ws + align256(per * 2));
    float* r_t = reinterpret_cast<float*>(ws + 2 * align256(per * 2));
    float* cnm = reinterpret_cast<float*>(ws + 2 * align256(per * 2) + align256(per * 4));

    prep_r_kernel<<<n_rounds, 256, 0, stream>>>(R, half, half_pad, r_hi, r_mid, r_t, cnm);
    if (rows == 0) return hipGetLastError();

    const int n_tiles = half_pad / 32;
    const int idx_bits = 4 + ceil_log2(n_tiles);
    // Error bound of a screened projection, as a multiple of |q| * max_c |R_c|:
    // plane residual(s), fp32 accumulation (2^-22 per addition, a 4x margin
    // over round-to-nearest), and the index bits packed into the mantissa.
    const double acc_terms = f32 ? 3 * kHeadDim : 2 * kHeadDim;
    const double resid = f32 ? 3.1 * 0x1p-16 : 0x1p-16;
    const double eps = resid + acc_terms * 0x1p-22 + std::ldexp(1.0, idx_bits - 23);
    const float thr_coef = (float)(2.0 * eps * 1.02);

    const unsigned grid = (unsigned)((rows + kHashRowsPerBlock - 1) / kHashRowsPerBlock);
    if (f32)
        hash_kernel<true><<<grid, 256, 0, stream>>>(q, rows, n_rounds, half, half_pad, r_hi, r_mid,
                                                     r_t, cnm, thr_coef, idx_bits, buckets);
    else
        hash_kernel<false><<<grid, 256, 0, stream>>>(q, rows, n_rounds, half, half_pad, r_hi, r_mid,
                                                      r_t, cnm, thr_coef, idx_bits, buckets);
    return hipGetLastError();
}

}  // namespace lsh

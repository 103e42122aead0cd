// Device helpers shared by the LSH attention kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lsh {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kHeadDim = 64;  // d_k handled by every kernel
constexpr int kChunk = 64;    // m handled by every kernel
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// Round to nearest, ties to even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    bf16x2_t v;
    v[0] = (__bf16)lo;
    v[1] = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

// Round to nearest, ties to even, into IEEE binary16 (lo in bits 0..15).
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
    f16x2_t v;
    v[0] = (_Float16)lo;
    v[1] = (_Float16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t bits16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float x) {
    return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ f16x8 as_f16x8(u32x4 v) { return __builtin_bit_cast(f16x8, v); }

// D = A(32x16) * B(16x32) + C on the matrix cores, fp32 accumulate.
// Lane l holds A row (l % 32), B column (l % 32), and 8 k-values each; the
// same lane/slot pairs meet in the product, so any consistent k order works.
// C: lane l, register j holds row 8*(j/4) + 4*(l/32) + (j%4), column l % 32.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// The same shape with IEEE binary16 operands.
__device__ __forceinline__ f32x16 mfma32x32x16(f16x8 a, f16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

// Exchanges between the 16-lane rows of a wave with gfx950's row swaps:
// VALU operations, without the LDS round trip of __shfl_xor.  pair16(x)
// gives, in some order, x of lane l and of lane l ^ 16; pair32 likewise for
// l ^ 32.  (permlane16_swap(a, b) trades the odd rows of a with the even
// rows of b, permlane32_swap(a, b) the upper half of a with the lower half
// of b; with a = b = x each lane ends up holding both values.)
struct LanePair {
    uint32_t a, b;
};
__device__ __forceinline__ LanePair pair16(uint32_t x) {
    const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    return {p[0], p[1]};
}
__device__ __forceinline__ LanePair pair32(uint32_t x) {
    const auto p = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return {p[0], p[1]};
}
// x of lane l ^ 16 and of lane l ^ 32 (the partner's value is the first of
// the pair in the upper row or half, the second in the lower).
__device__ __forceinline__ uint32_t xor16(uint32_t x) {
    const LanePair p = pair16(x);
    return (threadIdx.x & 16) ? p.a : p.b;
}
__device__ __forceinline__ uint32_t xor32(uint32_t x) {
    const LanePair p = pair32(x);
    return (threadIdx.x & 32) ? p.a : p.b;
}
// x[l] + x[l ^ 16] and x[l] + x[l ^ 32] (the same value in both lanes of a
// pair, as the additions commute); likewise the maxima.
__device__ __forceinline__ float sum_xor16(float x) {
    const LanePair p = pair16(__float_as_uint(x));
    return __uint_as_float(p.a) + __uint_as_float(p.b);
}
__device__ __forceinline__ float sum_xor32(float x) {
    const LanePair p = pair32(__float_as_uint(x));
    return __uint_as_float(p.a) + __uint_as_float(p.b);
}
__device__ __forceinline__ float max_xor16(float x) {
    const LanePair p = pair16(__float_as_uint(x));
    return fmaxf(__uint_as_float(p.a), __uint_as_float(p.b));
}
__device__ __forceinline__ float max_xor32(float x) {
    const LanePair p = pair32(__float_as_uint(x));
    return fmaxf(__uint_as_float(p.a), __uint_as_float(p.b));
}

// Sum / max over each aligned group of eight lanes with DPP moves (no LDS
// round trip): lanes i ^ 1, then i ^ 2 (quad permutes), then the mirrored
// lane 7 - i of the group, which after the first two steps holds the same
// value as lane i ^ 4.  Every lane of a group ends with the same value, the
// one the xor butterfly gives.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141; // lane 7 - i within each group of eight
__device__ __forceinline__ float group8_sum(float x) {
    x += dpp_f32<kDppXor1>(x);
    x += dpp_f32<kDppXor2>(x);
    return x + dpp_f32<kDppHalfMirror>(x);
}
__device__ __forceinline__ float group8_max(float x) {
    x = fmaxf(x, dpp_f32<kDppXor1>(x));
    x = fmaxf(x, dpp_f32<kDppXor2>(x));
    return fmaxf(x, dpp_f32<kDppHalfMirror>(x));
}

__device__ __forceinline__ float wave_max(float x) {
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}

}  // namespace lsh

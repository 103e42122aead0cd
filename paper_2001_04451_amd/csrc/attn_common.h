// Device helpers shared by the chunked-attention kernels (forward and
// backward): swizzled LDS row tiles, the key-row permutation that lets an
// S^T accumulator be reused as a matrix-core operand, and the packed bucket
// signatures behind N_ij.
#pragma once

#include "common.h"

namespace lsh {

// Rows of 64 bf16 values (128 B) are staged in LDS as 8 pieces of 16 B with
// piece p of row r stored at slot p ^ (r & 7) ^ (((r >> 3) & 1) << k), where
// layout K picks k: K = 0, k = 2, for reads of rows kappa(0..7), rows
// r..r+7 and the two lane halves 8 rows apart (32-row operands); K = 1,
// k = 1, for the same piece of sixteen consecutive rows read by the sixteen
// lanes of a 16-row operand.  Measured with SQ_LDS_BANK_CONFLICT on the
// forward kernel (the hardware's grouping of a 16-byte read's lanes is not
// documented): 6.4 M conflict cycles per call under K = 1, 31 M under K = 0
// and under p ^ ((r ^ (r >> 3)) & 7), 28 M under p ^ ((r >> 1) & 7), 145 M
// under p ^ ((r >> 2) & 7) and with no swizzle.
template <int K = 0>
__device__ __forceinline__ int swz(int row, int piece) {
    return piece ^ (row & 7) ^ (((row >> 3) & 1) << (K == 0 ? 2 : 1));
}

template <int K = 0>
__device__ __forceinline__ uint32_t row_piece_offset(int row, int piece) {
    return (uint32_t)row * 128u + (uint32_t)swz<K>(row, piece) * 16u;
}

template <int K = 0>
__device__ __forceinline__ u32x4 lds_piece(const char* base, int row, int piece) {
    return *reinterpret_cast<const u32x4*>(base + row_piece_offset<K>(row, piece));
}

__device__ __forceinline__ void lds_store_piece(char* base, int row, int piece, u32x4 v) {
    *reinterpret_cast<u32x4*>(base + row_piece_offset(row, piece)) = v;
}

__device__ __forceinline__ uint32_t lds_elem(const char* base, int row, int d) {
    return *reinterpret_cast<const uint16_t*>(base + row_piece_offset(row, d >> 3) + (d & 7) * 2);
}

// The A operand of a 32-row tile (lane l, row l%32) holds tile row kappa(l%32)
// so that accumulator register j of lane l corresponds to tile row
// 16*(j/8) + 8*(l/32) + (j%8): registers 8u..8u+7 are then exactly the
// k-slots of the 16-row block u in the B-operand layout of the next product.
__device__ __forceinline__ int kappa(int m) {
    return 16 * (m >> 4) + 8 * ((m >> 2) & 1) + 4 * ((m >> 3) & 1) + (m & 3);
}

// Operand with rows along the lane (row r0 + lane%32, k = 32h + 8s + e).
__device__ __forceinline__ bf16x8 row_operand(const char* base, int row, int h, int s) {
    return as_bf16x8(lds_piece(base, row, 4 * h + s));
}

// Transposed operand: lane holds column d (fixed) of the 8 rows r0 .. r0+7.
__device__ __forceinline__ bf16x8 col_operand(const char* base, int r0, int d) {
    u32x4 v;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2)
        v[e2] = lds_elem(base, r0 + 2 * e2, d) | (lds_elem(base, r0 + 2 * e2 + 1, d) << 16);
    return as_bf16x8(v);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
constexpr bf16x2 kOnes = {(__bf16)1.0f, (__bf16)1.0f};
constexpr bf16x4 kOnes4 = {(__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f};

__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16x16x16(bf16x4 a, bf16x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// Copy 16 (4) bytes per lane from global memory to LDS at lds_base + 16
// (4) * lane; lds_base is uniform over the wave.  Written as inline assembly
// so that the compiler does not order every later LDS read of the step
// behind these copies (it cannot tell the slot being filled from the slots
// being read); the kernel waits for them itself before each barrier.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    // the same address in every lane; readfirstlane puts it in a scalar register
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p);
}
__device__ __forceinline__ void copy16_to_lds(const void* src, const void* lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds_addr(lds_base))
                 : "memory", "m0");
}

__device__ __forceinline__ void copy4_to_lds(const void* src, const void* lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(src), "s"(lds_addr(lds_base))
                 : "memory", "m0");
}

// V^T operand of a 16x16x16 product for keys r0 .. r0+15 and dims d0 .. d0+15:
// lane l needs V[r0 + 4(l/16) + k][d0 + l%16] for k = 0..3.  The transposing
// read gives lane i of each 16-lane group element i%4 of the 8-byte runs read
// by lanes 4k + i/4, so lane i reads row r0 + 4(l/16) + i/4, dims
// d0 + 4(i%4) .. +3: vt_offset is that byte offset (r0 a multiple of 16, so
// the swizzle depends on the lane only).
template <int K = 0>
__device__ __forceinline__ uint32_t vt_offset(int r0, int d0, int lane) {
    const int i = lane & 15;
    const int row = r0 + 4 * (lane >> 4) + (i >> 2);
    const int d = d0 + 4 * (i & 3);
    return row_piece_offset<K>(row, d >> 3) + (uint32_t)((d & 4) << 1);
}
__device__ __forceinline__ bf16x4 vt_read(const char* p) {
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const i16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(__attribute__((address_space(3))) char*)p);
    return __builtin_bit_cast(bf16x4, x);
}

// Bucket signature word w of a token: its ids in rounds 2w and 2w+1 (10 bits
// each) at bit offsets w and w+11.  Adding sig_add(w) to (a ^ b) carries into
// guard bit w+10 (w+21) exactly when the first (second) ids differ; the guard
// bits of different words are distinct, so the number of rounds in which two
// tokens differ is the popcount of the OR over w of
// ((a_w ^ b_w) + sig_add(w)) & sig_guard(w).
__device__ __forceinline__ constexpr uint32_t sig_add(int w) {
    return (0x3FFu << w) | (0x3FFu << (w + 11));
}
__device__ __forceinline__ constexpr uint32_t sig_guard(int w) {
    return (1u << (w + 10)) | (1u << (w + 21));
}

// Words per token for NW signature words (NW = 0 for one round, whose id still
// sits in word 0), and the round-r id of a token from its words.
__host__ __device__ constexpr int sig_stride(int nw) { return nw <= 1 ? 1 : (nw <= 2 ? 2 : (nw <= 4 ? 4 : 8)); }
__device__ __forceinline__ uint32_t sig_round_id(const uint32_t* words, int r) {
    return (words[r >> 1] >> ((r >> 1) + 11 * (r & 1))) & 0x3FFu;
}

// (a & b) | c as one v_and_or_b32: left to itself the compiler regroups the
// OR chain over the signature words into separate ANDs and three-way ORs.
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t b, uint32_t c) {
    uint32_t d;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "s"(b), "v"(c));
    return d;
}

}  // namespace lsh

// Undo the per-round sort and combine the rounds (Reformer App. A):
//   z_i = log sum_r exp z_r(i),   o_i = sum_r exp(z_r(i) - z_i) o_r(i).
// The scatter back to position order is done as a gather through `undo`, so
// every write is a contiguous output row.  For bf16 calls the per-round rows
// are fp16 scaled by 2^-e (e one byte per row); 2^e is folded into the
// round's weight.
#include "common.h"
#include "launch.h"

#include <type_traits>

namespace lsh {
namespace {

constexpr int kMaxRounds = 16;

// Eight lanes share a row.  Lane p of the group first handles round p (and
// p + 8 when n_r > 8): its slot from undo, its log-partition z_r, and after
// a max / sum across the group (shuffles) its weight exp(z_r - z), formed as
// exp(z_r - max_r z_r) / sum so that it is exact at any magnitude of z.  Then
// every lane takes 8 of the row's 64 values (16 bytes of fp16, two float4
// of fp32) from all rounds, with the slots and weights of the other rounds
// read from their lanes.  The code is straight-line for every n_r: rounds
// past n_r read a valid slot and get weight 0, so each lane's loads are all
// in flight together.  The per-round rows are read once each and marked
// non-temporal, so they stream past the L2 instead of evicting the
// log-partition lines, which serve 32 gathers each.  The weighted sum is
// formed in fp32.  NRL is n_r rounded up to a power of two.
template <bool F32, int NRL>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ o_rounds,
                                                      const uint8_t* __restrict__ o_exp,
                                                      const float* __restrict__ lse_rounds,
                                                      const int32_t* __restrict__ undo,
                                                      void* __restrict__ out,
                                                      float* __restrict__ lse_total, int64_t rows,
                                                      int L, int n_r) {
    // Rows from the last to the first: the attention kernel writes the
    // per-round rows segment after segment, so the last (batch, head) slices'
    // rows are the ones most likely still in the Infinity Cache when the
    // combine starts (at L = 64K, 16 heads, 8 rounds: 0.290 -> 0.276 ms;
    // unchanged at L = 32K, 64 slices, 4 rounds).
    const int64_t row = ((int64_t)(gridDim.x - 1 - blockIdx.x) * blockDim.x + threadIdx.x) >> 3;
    const int part = threadIdx.x & 7;
    // Rows past the end leave as whole 8-lane groups; every shuffle below
    // stays inside a group.
    if (row >= rows) return;
    const int64_t bh = row / L;
    const int64_t i = row % L;
    const int64_t seg0 = bh * n_r;
    const int lane = threadIdx.x & 63, group0 = lane & ~7;
    constexpr int RPL = NRL > 8 ? 2 : 1;  // rounds per lane

    // this lane's rounds: part and part + 8
    int u[RPL];
    bool live[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
        const int r = part + 8 * k;
        live[k] = r < n_r;
        u[k] = min(max(undo[(seg0 + min(r, n_r - 1)) * L + i], 0), L - 1);
    }
    // every round's slot in every lane of the group (rounds n_r .. NRL-1
    // read round n_r - 1's row, with weight 0 below); the rows' loads are
    // issued here, alongside the log-partitions', not after the weights
    constexpr int NR = NRL;
    int64_t sl[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) sl[r] = (seg0 + min(r, n_r - 1)) * L + __shfl(u[r >> 3], group0 + (r & 7));
    constexpr int kPieces = F32 ? 2 : 1;  // 16-byte pieces of a lane's 8 values
    u32x4 o[NR][kPieces];
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int pc = 0; pc < kPieces; ++pc)
            o[r][pc] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
                static_cast<const char*>(o_rounds) + (sl[r] * kHeadDim + part * 8) * (F32 ? 4 : 2) + 16 * pc));
    float zr[RPL];
    uint32_t ex[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
        const int64_t at = (seg0 + min(part + 8 * k, n_r - 1)) * L + u[k];
        zr[k] = lse_rounds[at];
        ex[k] = F32 ? 0u : min((uint32_t)o_exp[at], 126u);
    }
    float zmax = -__builtin_inff();
#pragma unroll
    for (int k = 0; k < RPL; ++k)
        if (live[k]) zmax = fmaxf(zmax, zr[k]);
    zmax = group8_max(zmax);
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < RPL; ++k) sum += live[k] ? expf(zr[k] - zmax) : 0.f;
    sum = group8_sum(sum);
    const float z = zmax + logf(sum);
    // weights relative to the largest round, not to z: a token alone in its
    // buckets has z_r near -self_mask, where one fp32 spacing of z is 2^-7,
    // and exp(z_r - z) would carry that rounding into every weight
    const float inv_sum = 1.f / sum;
    float wk[RPL];
#pragma unroll
    for (int k = 0; k < RPL; ++k)  // times 2^e, the scale of the stored row
        wk[k] = live[k] ? expf(zr[k] - zmax) * inv_sum * __uint_as_float((127u + ex[k]) << 23) : 0.f;
    float w[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) w[r] = __shfl(wk[r >> 3], group0 + (r & 7));

    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if constexpr (F32) {
#pragma unroll
        for (int r = 0; r < NR; ++r)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = fmaf(w[r], __uint_as_float(o[r][e >> 2][e & 3]), acc[e]);
        float* dst = static_cast<float*>(out) + row * kHeadDim + part * 8;
        *reinterpret_cast<f32x4*>(dst) = f32x4{acc[0], acc[1], acc[2], acc[3]};
        *reinterpret_cast<f32x4*>(dst + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
    } else {
#pragma unroll
        for (int r = 0; r < NR; ++r)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc[2 * e] = fmaf(w[r], f16_bits_to_f32(o[r][0][e] & 0xFFFFu), acc[2 * e]);
                acc[2 * e + 1] = fmaf(w[r], f16_bits_to_f32(o[r][0][e] >> 16), acc[2 * e + 1]);
            }
        u32x4 packed;
#pragma unroll
        for (int e = 0; e < 4; ++e) packed[e] = pack_bf16x2(acc[2 * e], acc[2 * e + 1]);
        *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(out) + row * kHeadDim + part * 8) = packed;
    }
    if (lse_total && part == 0) lse_total[row] = z;
}

}  // namespace

hipError_t launch_combine(int64_t BH, int L, int n_rounds, bool f32, const void* o_rounds,
                          const uint8_t* o_exp, const float* lse_rounds, const int32_t* undo, void* out,
                          float* lse_total, hipStream_t stream) {
    const int64_t rows = BH * L;
    if (rows == 0) return hipSuccess;
    const unsigned grid = (unsigned)((rows * 8 + 255) / 256);
    if (n_rounds > kMaxRounds) return hipErrorInvalidValue;
    auto go = [&](auto f32_tag, auto nrl_tag) {
        combine_kernel<decltype(f32_tag)::value, decltype(nrl_tag)::value><<<grid, 256, 0, stream>>>(
            o_rounds, o_exp, lse_rounds, undo, out, lse_total, rows, L, n_rounds);
    };
    auto by_rounds = [&](auto f32_tag) {
        if (n_rounds <= 1) go(f32_tag, std::integral_constant<int, 1>{});
        else if (n_rounds <= 2) go(f32_tag, std::integral_constant<int, 2>{});
        else if (n_rounds <= 4) go(f32_tag, std::integral_constant<int, 4>{});
        else if (n_rounds <= 8) go(f32_tag, std::integral_constant<int, 8>{});
        else go(f32_tag, std::integral_constant<int, 16>{});
    };
    if (f32)
        by_rounds(std::true_type{});
    else
        by_rounds(std::false_type{});
    return hipGetLastError();
}

}  // namespace lsh

// Undo the per-round sort and combine the rounds (Reformer App. A):
//   z_i = log sum_r exp z_r(i),   o_i = sum_r exp(z_r(i) - z_i) o_r(i).
// The scatter back to position order is done as a gather through `undo`, so
// every write is a contiguous output row.
#include "common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr int kMaxRounds = 16;

// Eight lanes share a row (8 of its 64 values each, 16 bytes of bf16 or two
// float4 of fp32).  All loads of a row are issued before they are used
// (slots, then the log-partitions, then the rows), so each lane keeps up to
// 16 independent requests in flight instead of walking a dependent chain per
// round.  The weighted sum is formed in fp32.  The per-round rows are read
// once each and marked non-temporal, so they stream past the L2 instead of
// evicting the log-partition lines, which serve 32 gathers each.
template <bool F32>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ o_rounds,
                                                      const float* __restrict__ lse_rounds,
                                                      const int32_t* __restrict__ undo,
                                                      void* __restrict__ out,
                                                      float* __restrict__ lse_total, int64_t rows,
                                                      int L, int n_r) {
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 3;
    const int part = threadIdx.x & 7;
    if (row >= rows) return;
    const int64_t bh = row / L;
    const int64_t i = row % L;
    const int64_t seg0 = bh * n_r;

    int64_t base[kMaxRounds];
    float z_r[kMaxRounds];
#pragma unroll
    for (int r = 0; r < kMaxRounds; ++r)
        if (r < n_r) base[r] = (seg0 + r) * L + min(max(undo[(seg0 + r) * L + i], 0), L - 1);
    float zmax = -__builtin_inff();
#pragma unroll
    for (int r = 0; r < kMaxRounds; ++r)
        if (r < n_r) {
            z_r[r] = lse_rounds[base[r]];
            zmax = fmaxf(zmax, z_r[r]);
        }
    float sum = 0.f;
#pragma unroll
    for (int r = 0; r < kMaxRounds; ++r)
        if (r < n_r) sum += expf(z_r[r] - zmax);
    const float z = zmax + logf(sum);
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if constexpr (F32) {
        const float* src = static_cast<const float*>(o_rounds);
        f32x4 o[kMaxRounds][2];
#pragma unroll
        for (int r = 0; r < kMaxRounds; ++r)
            if (r < n_r) {
                o[r][0] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src + base[r] * kHeadDim + part * 8));
                o[r][1] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src + base[r] * kHeadDim + part * 8 + 4));
            }
#pragma unroll
        for (int r = 0; r < kMaxRounds; ++r)
            if (r < n_r) {
                const float w = expf(z_r[r] - z);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[e] = fmaf(w, o[r][e >> 2][e & 3], acc[e]);
            }
        float* dst = static_cast<float*>(out) + row * kHeadDim + part * 8;
        *reinterpret_cast<f32x4*>(dst) = f32x4{acc[0], acc[1], acc[2], acc[3]};
        *reinterpret_cast<f32x4*>(dst + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
    } else {
        const uint16_t* src = static_cast<const uint16_t*>(o_rounds);
        u32x4 o[kMaxRounds];
#pragma unroll
        for (int r = 0; r < kMaxRounds; ++r)
            if (r < n_r) o[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + base[r] * kHeadDim + part * 8));
#pragma unroll
        for (int r = 0; r < kMaxRounds; ++r)
            if (r < n_r) {
                const float w = expf(z_r[r] - z);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[2 * e] = fmaf(w, bf16_bits_to_f32(o[r][e] & 0xFFFFu), acc[2 * e]);
                    acc[2 * e + 1] = fmaf(w, __uint_as_float(o[r][e] & 0xFFFF0000u), acc[2 * e + 1]);
                }
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
                          const float* lse_rounds, const int32_t* undo, void* out,
                          float* lse_total, hipStream_t stream) {
    const int64_t rows = BH * L;
    if (rows == 0) return hipSuccess;
    const unsigned grid = (unsigned)((rows * 8 + 255) / 256);
    if (f32)
        combine_kernel<true><<<grid, 256, 0, stream>>>(o_rounds, lse_rounds, undo, out, lse_total,
                                                       rows, L, n_rounds);
    else
        combine_kernel<false><<<grid, 256, 0, stream>>>(o_rounds, lse_rounds, undo, out, lse_total,
                                                        rows, L, n_rounds);
    return hipGetLastError();
}

}  // namespace lsh

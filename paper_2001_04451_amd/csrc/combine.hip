// Undo the per-round sort and combine the rounds (Reformer App. A):
//   z_i = log sum_r exp z_r(i),   o_i = sum_r exp(z_r(i) - z_i) o_r(i).
// The scatter back to position order is done as a gather through `undo`, so
// every write is a contiguous output row.  Sixteen lanes share a row (one
// float4 of the 64 values each); the per-round log-partitions are read once
// per lane group and stay in L1 for the three passes.
#include "common.h"
#include "launch.h"

namespace lsh {
namespace {

template <bool F32_OUT>
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ o_rounds,
                                                      const float* __restrict__ lse_rounds,
                                                      const int32_t* __restrict__ undo,
                                                      void* __restrict__ out,
                                                      float* __restrict__ lse_total, int64_t rows,
                                                      int L, int n_r) {
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
    const int part = threadIdx.x & 15;
    if (row >= rows) return;
    const int64_t bh = row / L;
    const int64_t i = row % L;
    const int64_t seg0 = bh * n_r;

    float zmax = -__builtin_inff();
    for (int r = 0; r < n_r; ++r) {
        const int64_t s = min(max(undo[(seg0 + r) * L + i], 0), L - 1);
        zmax = fmaxf(zmax, lse_rounds[(seg0 + r) * L + s]);
    }
    float sum = 0.f;
    for (int r = 0; r < n_r; ++r) {
        const int64_t s = min(max(undo[(seg0 + r) * L + i], 0), L - 1);
        sum += expf(lse_rounds[(seg0 + r) * L + s] - zmax);
    }
    const float z = zmax + logf(sum);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int r = 0; r < n_r; ++r) {
        const int64_t s = min(max(undo[(seg0 + r) * L + i], 0), L - 1);
        const float w = expf(lse_rounds[(seg0 + r) * L + s] - z);
        const f32x4 o = *reinterpret_cast<const f32x4*>(o_rounds + ((seg0 + r) * L + s) * kHeadDim + part * 4);
        acc[0] = fmaf(w, o[0], acc[0]);
        acc[1] = fmaf(w, o[1], acc[1]);
        acc[2] = fmaf(w, o[2], acc[2]);
        acc[3] = fmaf(w, o[3], acc[3]);
    }
    if constexpr (F32_OUT) {
        *reinterpret_cast<f32x4*>(static_cast<float*>(out) + row * kHeadDim + part * 4) = acc;
    } else {
        uint2 packed = make_uint2(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]));
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(out) + row * kHeadDim + part * 4) = packed;
    }
    if (lse_total && part == 0) lse_total[row] = z;
}

}  // namespace

hipError_t launch_combine(int64_t BH, int L, int n_rounds, bool f32_out, const float* o_rounds,
                          const float* lse_rounds, const int32_t* undo, void* out,
                          float* lse_total, hipStream_t stream) {
    const int64_t rows = BH * L;
    if (rows == 0) return hipSuccess;
    const unsigned grid = (unsigned)((rows * 16 + 255) / 256);
    if (f32_out)
        combine_kernel<true><<<grid, 256, 0, stream>>>(o_rounds, lse_rounds, undo, out, lse_total,
                                                       rows, L, n_rounds);
    else
        combine_kernel<false><<<grid, 256, 0, stream>>>(o_rounds, lse_rounds, undo, out, lse_total,
                                                        rows, L, n_rounds);
    return hipGetLastError();
}

}  // namespace lsh

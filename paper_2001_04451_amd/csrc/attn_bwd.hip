// Backward of chunked LSH attention (placeholder until the kernels land).
#include "common.h"
#include "launch.h"

namespace lsh {

size_t bwd_workspace_bytes(int64_t BH, int L, int n_rounds) {
    const size_t rr = (size_t)BH * n_rounds * L;
    return align256(rr * kHeadDim * sizeof(float)) * 3 + align256((size_t)BH * L * sizeof(float));
}

hipError_t launch_attn_bwd(int64_t, int, int, int, bool, float, float, const void*, const void*,
                           const void*, const void*, const float*, const int32_t*,
                           const int32_t*, const int32_t*, const int32_t*, float*, float*, void*,
                           hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace lsh

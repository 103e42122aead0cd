// Kernel launchers behind the C ABI.  Arguments are already validated by the
// caller (lsh_api.cpp); every launcher only enqueues work on `stream` and
// returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

struct lsh_config;  // include/lsh.h

namespace lsh {

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

constexpr int kHeadDimHost = 64;  // d_k the kernels are specialised for
constexpr int kChunkHost = 64;    // chunk length m the kernels are specialised for

// ---- hashing ----
size_t hash_workspace_bytes(int64_t rows, int n_rounds, int n_buckets);
hipError_t launch_hash(const void* q, bool f32, int64_t rows, int n_rounds, int n_buckets,
                       const float* R, int32_t* buckets, void* workspace, hipStream_t stream);

// ---- counting sort and row gather ----
int sort_tile_positions(int L);
// Workspace of launch_sort: the per-tile bucket counts, plus, when
// round_major_ids is set, a 16-bit copy of the ids in [segment][position]
// order (sort_workspace_bytes covers both, sort_counts_bytes the counts).
size_t sort_counts_bytes(int64_t BH, int L, int n_rounds, int n_buckets);
size_t sort_workspace_bytes(int64_t BH, int L, int n_rounds, int n_buckets);
hipError_t launch_sort(int64_t BH, int L, int n_rounds, int n_buckets, const int32_t* buckets,
                       int32_t* perm, int32_t* undo, int32_t* bucket_start, void* workspace,
                       bool round_major_ids, hipStream_t stream);
// The fixed scratch array of lsh_sort_permute_static (sort.hip): its size,
// and its device address on the current device (looked up on the first call
// on each device).
constexpr size_t kSortScratchBytes = (size_t)16 << 20;
constexpr int kMaxDevices = 64;
hipError_t sort_static_scratch(void** ptr);
hipError_t launch_gather(int64_t BH, int L, int n_rounds, bool f32, const void* src,
                         const int32_t* perm, void* dst, hipStream_t stream);

// ---- chunked attention, forward ----
size_t attn_fwd_workspace_bytes(int64_t BH, int L, int n_rounds, bool f32);
hipError_t launch_attn_fwd(int64_t BH, int L, int n_rounds, int n_buckets, int chunk, int after,
                           bool across, bool causal, float scale, float self_mask, bool f32,
                           const void* q, const void* v, const int32_t* buckets,
                           const int32_t* perm, const int32_t* undo,
                           const int32_t* bucket_start, void* o_rounds, uint8_t* o_exp,
                           float* lse_rounds, void* workspace, hipStream_t stream);

// ---- round combination ----
hipError_t launch_combine(int64_t BH, int L, int n_rounds, bool f32, const void* o_rounds,
                          const uint8_t* o_exp, const float* lse_rounds, const int32_t* undo, void* out,
                          float* lse_total, hipStream_t stream);

// ---- backward ----
size_t bwd_workspace_bytes(int64_t BH, int L, int n_rounds);
hipError_t launch_attn_bwd(int64_t BH, int L, int n_rounds, int n_buckets, bool causal,
                           float scale, float self_mask, const void* q, const void* v,
                           const void* out, const void* dout, const float* lse_total,
                           const int32_t* buckets, const int32_t* perm, const int32_t* undo,
                           const int32_t* bucket_start, float* dq, float* dv, void* workspace,
                           hipStream_t stream);

// ---- full (dense) shared-QK attention, forward ----
size_t dense_workspace_bytes(int64_t BH, int L);
hipError_t launch_dense_fwd(int64_t BH, int L, bool causal, float scale, float self_mask,
                            const void* q, const void* v, void* out, float* lse, void* workspace,
                            hipStream_t stream);

// ---- reversible block: LayerNorm and the dense products ----
// LSH_OK when lsh_attention_fwd takes this configuration and dtype (its
// checks, without any HIP call); otherwise the status it would return.
int attention_fwd_supported(const ::lsh_config* cfg, int dtype);
// fp32 rows [rows][D] -> bf16 rows, D a multiple of 128 up to 4096.
hipError_t launch_layer_norm(const float* x, const float* g, const float* b, uint16_t* out, int64_t rows, int D,
                             float eps, hipStream_t stream);
// C = A W^T (A: [M][K] bf16 rows, or with a_heads the [B][H][L][64] layout
// with K = 64 H, M = B L; W [N][K] bf16; N a multiple of 128, K of 64), then:
enum : int {
    kLinearResid = 0,     // out_f32 = resid + sign (C + bias)   (resid may be null)
    kLinearReluBf16 = 1,  // out_bf16 = bf16(relu(C + bias))      [M][N]
    kLinearHeads = 2      // out_bf16 = bf16(C + bias) in the [B][H][L][64] layout (N = 64 H)
};
hipError_t launch_linear(const uint16_t* a, bool a_heads, int L, int H, const uint16_t* w, int64_t M, int N, int K,
                         const float* bias, int out_kind, const float* resid, float sign, float* out_f32,
                         uint16_t* out_bf16, hipStream_t stream);

}  // namespace lsh

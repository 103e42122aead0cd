// The C ABI of liblsh (declared in include/lsh.h): argument validation,
// workspace carving and kernel launches.  Validation runs before any HIP
// call, so every LSH_ERR_INVALID / LSH_ERR_UNSUPPORTED path works without a
// GPU.
#include "lsh.h"

#include <cmath>

#include "launch.h"

namespace {

constexpr int64_t kMaxElems = (int64_t)1 << 31;

// Smallest self_mask the kernels accept.  They give a token's own key weight
// zero whenever it has another target, and treat a row whose total
// log-partition is below -self_mask/2 as its own only target; both are exact
// in fp32 while self_mask > 2*scale*|q_i| + log(n_rounds) + 17 for every row,
// which at this minimum holds for scale*|q_i| up to about 4,990.
constexpr float kMinSelfMask = 1e4f;

bool finitef(float x) { return std::isfinite(x); }

// Shape checks shared by every entry point.
int check_config(const lsh_config* cfg) {
    if (!cfg) return LSH_ERR_INVALID;
    if (cfg->B < 1 || cfg->H < 1 || cfg->L < 1 || cfg->d < 1) return LSH_ERR_INVALID;
    if (cfg->n_buckets < 2 || (cfg->n_buckets % 2) != 0) return LSH_ERR_INVALID;
    if (cfg->n_rounds < 1 || cfg->chunk < 1) return LSH_ERR_INVALID;
    if (!finitef(cfg->scale) || !finitef(cfg->self_mask)) return LSH_ERR_INVALID;
    if (cfg->chunks_after < 0) return LSH_ERR_INVALID;
    return LSH_OK;
}

int check_dtype(int dtype) {
    return (dtype == LSH_F32 || dtype == LSH_BF16) ? LSH_OK : LSH_ERR_INVALID;
}

// What the kernels are specialised for (the chunk length is checked by the
// entry points that use it, see check_chunk).
int check_supported(const lsh_config* cfg) {
    if (cfg->d != lsh::kHeadDimHost) return LSH_ERR_UNSUPPORTED;
    if (cfg->n_buckets > 1024 || cfg->n_rounds > 16) return LSH_ERR_UNSUPPORTED;
    const int64_t rr = (int64_t)cfg->B * cfg->H * cfg->L * cfg->n_rounds;
    if (rr >= kMaxElems || rr * cfg->d >= ((int64_t)1 << 40)) return LSH_ERR_UNSUPPORTED;
    if ((int64_t)cfg->B * cfg->H * cfg->n_rounds >= 65536) return LSH_ERR_UNSUPPORTED;
    return LSH_OK;
}

int64_t bh_of(const lsh_config* cfg) { return (int64_t)cfg->B * cfg->H; }

// The attention entry points need self_mask >= kMinSelfMask.
int check_self_mask(const lsh_config* cfg) {
    return cfg->self_mask >= kMinSelfMask ? LSH_OK : LSH_ERR_UNSUPPORTED;
}

// What the chunked-attention kernels take: the forward chunks of 64 or 128
// and a look-ahead of at most one chunk, attention across buckets on the fp32
// forward; the backward only the paper's own window (chunks of 64, no
// look-ahead, bucket-restricted targets).
int check_chunk(const lsh_config* cfg, int dtype, bool backward) {
    if (cfg->chunks_after > 1) return LSH_ERR_UNSUPPORTED;
    if (backward)
        return cfg->chunk == lsh::kChunkHost && cfg->chunks_after == 0 && !cfg->attend_across
                   ? LSH_OK
                   : LSH_ERR_UNSUPPORTED;
    if (cfg->chunk != 64 && cfg->chunk != 128) return LSH_ERR_UNSUPPORTED;
    if (dtype == LSH_BF16 && cfg->attend_across) return LSH_ERR_UNSUPPORTED;
    return LSH_OK;
}

// The dense baseline reads only the shape, the mask flag and the scales.
int check_dense_config(const lsh_config* cfg) {
    if (!cfg) return LSH_ERR_INVALID;
    if (cfg->B < 1 || cfg->H < 1 || cfg->L < 1 || cfg->d < 1) return LSH_ERR_INVALID;
    if (!finitef(cfg->scale) || !finitef(cfg->self_mask)) return LSH_ERR_INVALID;
    return LSH_OK;
}

int check_dense_supported(const lsh_config* cfg, int dtype) {
    if (dtype != LSH_BF16 || cfg->d != lsh::kHeadDimHost) return LSH_ERR_UNSUPPORTED;
    if (check_self_mask(cfg) != LSH_OK) return LSH_ERR_UNSUPPORTED;
    const int64_t BH = (int64_t)cfg->B * cfg->H;
    if (BH >= 65536 || BH * cfg->L >= kMaxElems) return LSH_ERR_UNSUPPORTED;
    return LSH_OK;
}

// The kernels move rows in 16-byte pieces.
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
template <typename... P>
bool all_aligned(P... p) {
    return (aligned16(p) && ...);
}

int status_of(hipError_t e) { return e == hipSuccess ? LSH_OK : LSH_ERR_HIP; }

// bytes of one o_rounds value: fp32 for fp32 calls, fp16 for bf16 calls
size_t elem_bytes(lsh_dtype dtype) { return dtype == LSH_F32 ? 4 : 2; }

// o_rounds, then o_exp (bf16 calls only), then lse_rounds (fp32), each
// 256-byte aligned
size_t rounds_bytes(const lsh_config* cfg, lsh_dtype dtype) {
    const size_t rr = (size_t)bh_of(cfg) * cfg->n_rounds * cfg->L;
    return lsh::align256(rr * cfg->d * elem_bytes(dtype));
}
size_t exp_bytes(const lsh_config* cfg, lsh_dtype dtype) {
    return dtype == LSH_F32 ? 0 : lsh::align256((size_t)bh_of(cfg) * cfg->n_rounds * cfg->L);
}
size_t fwd_rounds_bytes(const lsh_config* cfg, lsh_dtype dtype) {
    const size_t rr = (size_t)bh_of(cfg) * cfg->n_rounds * cfg->L;
    return rounds_bytes(cfg, dtype) + exp_bytes(cfg, dtype) + lsh::align256(rr * sizeof(float));
}

#define LSH_TRY(expr)              \
    do {                           \
        const int _st = (expr);    \
        if (_st != LSH_OK) return _st; \
    } while (0)

}  // namespace

namespace lsh {
int attention_fwd_supported(const lsh_config* cfg, int dtype) {
    LSH_TRY(check_config(cfg));
    LSH_TRY(check_dtype(dtype));
    LSH_TRY(check_supported(cfg));
    LSH_TRY(check_chunk(cfg, dtype, false));
    return check_self_mask(cfg);
}
}  // namespace lsh

extern "C" {

const char* lsh_status_string(int status) {
    switch (status) {
        case LSH_OK: return "ok";
        case LSH_ERR_INVALID: return "invalid argument";
        case LSH_ERR_UNSUPPORTED: return "unsupported configuration";
        case LSH_ERR_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

size_t lsh_workspace_bytes(const lsh_config* cfg, lsh_dtype dtype, int op) {
    if (op == LSH_OP_DENSE_FWD) {
        if (check_dense_config(cfg) != LSH_OK || check_dtype(dtype) != LSH_OK) return 0;
        return lsh::dense_workspace_bytes(bh_of(cfg), cfg->L);
    }
    if (check_config(cfg) != LSH_OK || check_dtype(dtype) != LSH_OK) return 0;
    const int64_t BH = bh_of(cfg);
    const size_t hash = lsh::hash_workspace_bytes(BH * cfg->L, cfg->n_rounds, cfg->n_buckets);
    const size_t sort = lsh::sort_workspace_bytes(BH, cfg->L, cfg->n_rounds, cfg->n_buckets);
    switch (op) {
        case LSH_OP_HASH: return hash;
        case LSH_OP_SORT: return sort;
        case LSH_OP_ATTN_FWD: return lsh::attn_fwd_workspace_bytes(BH, cfg->L, cfg->n_rounds, dtype == LSH_F32);
        case LSH_OP_COMBINE: return 0;
        case LSH_OP_ATTN_BWD: return lsh::bwd_workspace_bytes(BH, cfg->L, cfg->n_rounds);
        case LSH_OP_FORWARD: {
            const size_t attn = lsh::attn_fwd_workspace_bytes(BH, cfg->L, cfg->n_rounds, dtype == LSH_F32);
            const size_t scratch = hash > sort ? hash : sort;
            return fwd_rounds_bytes(cfg, dtype) + (scratch > attn ? scratch : attn);
        }
        default: return 0;
    }
}

int lsh_hash(const lsh_config* cfg, lsh_dtype dtype, const void* q, const float* R,
             int32_t* buckets, void* workspace, size_t workspace_bytes, void* stream) {
    LSH_TRY(check_config(cfg));
    LSH_TRY(check_dtype(dtype));
    if (!q || !R || !buckets || !workspace) return LSH_ERR_INVALID;
    if (!all_aligned(q, R, workspace)) return LSH_ERR_INVALID;
    if (workspace_bytes < lsh::hash_workspace_bytes(bh_of(cfg) * cfg->L, cfg->n_rounds, cfg->n_buckets))
        return LSH_ERR_INVALID;
    LSH_TRY(check_supported(cfg));
    const hipStream_t st = static_cast<hipStream_t>(stream);
    const bool f32 = dtype == LSH_F32;
    if (!cfg->r_per_head) {
        const int64_t rows = bh_of(cfg) * cfg->L;
        return status_of(lsh::launch_hash(q, f32, rows, cfg->n_rounds, cfg->n_buckets, R, buckets,
                                          workspace, st));
    }
    // one R per head: every (batch, head) slice is hashed with its head's R,
    // slice by slice (the slices share nothing, and each pass needs one R)
    const size_t r_set = (size_t)cfg->n_rounds * cfg->d * (cfg->n_buckets / 2);
    const size_t row_bytes = (size_t)cfg->d * elem_bytes(dtype);
    for (int64_t bh = 0; bh < bh_of(cfg); ++bh) {
        const int64_t row0 = bh * cfg->L;
        LSH_TRY(status_of(lsh::launch_hash(static_cast<const char*>(q) + row0 * row_bytes, f32, cfg->L,
                                           cfg->n_rounds, cfg->n_buckets, R + (bh % cfg->H) * r_set,
                                           buckets + row0 * cfg->n_rounds, workspace, st)));
    }
    return LSH_OK;
}

int lsh_sort_permute(const lsh_config* cfg, const int32_t* buckets, int32_t* perm, int32_t* undo,
                     int32_t* bucket_start, void* workspace, size_t workspace_bytes,
                     void* stream) {
    LSH_TRY(check_config(cfg));
    if (!buckets || !perm || !undo || !bucket_start || !workspace) return LSH_ERR_INVALID;
    if (workspace_bytes <
        lsh::sort_workspace_bytes(bh_of(cfg), cfg->L, cfg->n_rounds, cfg->n_buckets))
        return LSH_ERR_INVALID;
    LSH_TRY(check_supported(cfg));
    return status_of(lsh::launch_sort(bh_of(cfg), cfg->L, cfg->n_rounds, cfg->n_buckets, buckets,
                                      perm, undo, bucket_start, workspace, true,
                                      static_cast<hipStream_t>(stream)));
}

int lsh_sort_permute_static(const lsh_config* cfg, const int32_t* buckets, int32_t* perm,
                            int32_t* undo, int32_t* bucket_start, void* stream) {
    LSH_TRY(check_config(cfg));
    if (!buckets || !perm || !undo || !bucket_start) return LSH_ERR_INVALID;
    LSH_TRY(check_supported(cfg));
    if (lsh::sort_counts_bytes(bh_of(cfg), cfg->L, cfg->n_rounds, cfg->n_buckets) > lsh::kSortScratchBytes)
        return LSH_ERR_UNSUPPORTED;
    void* scratch = nullptr;
    LSH_TRY(status_of(lsh::sort_static_scratch(&scratch)));
    // the counts are written in full by every call: nothing needs clearing;
    // the scatter reads the ids where they are (no 16-bit copy in scratch)
    return status_of(lsh::launch_sort(bh_of(cfg), cfg->L, cfg->n_rounds, cfg->n_buckets, buckets,
                                      perm, undo, bucket_start, scratch, false,
                                      static_cast<hipStream_t>(stream)));
}

int lsh_gather_rows(const lsh_config* cfg, lsh_dtype dtype, const void* src, const int32_t* perm,
                    void* dst, void* stream) {
    LSH_TRY(check_config(cfg));
    LSH_TRY(check_dtype(dtype));
    if (!src || !perm || !dst) return LSH_ERR_INVALID;
    if (!all_aligned(src, dst)) return LSH_ERR_INVALID;
    LSH_TRY(check_supported(cfg));
    return status_of(lsh::launch_gather(bh_of(cfg), cfg->L, cfg->n_rounds, dtype == LSH_F32, src,
                                        perm, dst, static_cast<hipStream_t>(stream)));
}

int lsh_chunk_attn_fwd(const lsh_config* cfg, lsh_dtype dtype, const void* q, const void* v,
                       const int32_t* buckets, const int32_t* perm, const int32_t* undo,
                       const int32_t* bucket_start, void* o_rounds, uint8_t* o_exp,
                       float* lse_rounds, void* workspace, size_t workspace_bytes, void* stream) {
    LSH_TRY(check_config(cfg));
    LSH_TRY(check_dtype(dtype));
    if (!q || !v || !buckets || !perm || !bucket_start || !o_rounds || !lse_rounds)
        return LSH_ERR_INVALID;
    if (cfg->attend_across && !undo) return LSH_ERR_INVALID;
    if (dtype == LSH_BF16 && !o_exp) return LSH_ERR_INVALID;
    if (!all_aligned(q, v, o_rounds)) return LSH_ERR_INVALID;
    const size_t need = lsh_workspace_bytes(cfg, dtype, LSH_OP_ATTN_FWD);
    if (need > 0 && (!workspace || workspace_bytes < need || !all_aligned(workspace)))
        return LSH_ERR_INVALID;
    LSH_TRY(check_supported(cfg));
    LSH_TRY(check_chunk(cfg, dtype, false));
    LSH_TRY(check_self_mask(cfg));
    return status_of(lsh::launch_attn_fwd(bh_of(cfg), cfg->L, cfg->n_rounds, cfg->n_buckets, cfg->chunk,
                                          cfg->chunks_after, cfg->attend_across != 0,
                                          cfg->causal != 0, cfg->scale, cfg->self_mask,
                                          dtype == LSH_F32, q, v, buckets, perm, undo, bucket_start,
                                          o_rounds, o_exp, lse_rounds, workspace,
                                          static_cast<hipStream_t>(stream)));
}

int lsh_combine_rounds(const lsh_config* cfg, lsh_dtype dtype, const void* o_rounds,
                       const uint8_t* o_exp, const float* lse_rounds, const int32_t* undo,
                       void* out, float* lse_total, void* stream) {
    LSH_TRY(check_config(cfg));
    LSH_TRY(check_dtype(dtype));
    if (!o_rounds || !lse_rounds || !undo || !out) return LSH_ERR_INVALID;
    if (dtype == LSH_BF16 && !o_exp) return LSH_ERR_INVALID;
    if (!all_aligned(o_rounds, out)) return LSH_ERR_INVALID;
    LSH_TRY(check_supported(cfg));
    return status_of(lsh::launch_combine(bh_of(cfg), cfg->L, cfg->n_rounds, dtype == LSH_F32,
                                         o_rounds, o_exp, lse_rounds, undo, out, lse_total,
                                         static_cast<hipStream_t>(stream)));
}

int lsh_attention_fwd(const lsh_config* cfg, lsh_dtype dtype, const void* q, const void* v,
                      const float* R, void* out, float* lse_total, int32_t* buckets,
                      int32_t* perm, int32_t* undo, int32_t* bucket_start, void* workspace,
                      size_t workspace_bytes, void* stream) {
    LSH_TRY(check_config(cfg));
    LSH_TRY(check_dtype(dtype));
    if (!q || !v || !R || !out || !buckets || !perm || !undo || !bucket_start || !workspace)
        return LSH_ERR_INVALID;
    if (workspace_bytes < lsh_workspace_bytes(cfg, dtype, LSH_OP_FORWARD)) return LSH_ERR_INVALID;
    LSH_TRY(check_supported(cfg));
    LSH_TRY(check_chunk(cfg, dtype, false));
    LSH_TRY(check_self_mask(cfg));
    char* ws = static_cast<char*>(workspace);
    void* o_rounds = ws;
    uint8_t* o_exp = dtype == LSH_F32 ? nullptr : reinterpret_cast<uint8_t*>(ws + rounds_bytes(cfg, dtype));
    float* lse_rounds =
        reinterpret_cast<float*>(ws + rounds_bytes(cfg, dtype) + exp_bytes(cfg, dtype));
    void* scratch = ws + fwd_rounds_bytes(cfg, dtype);
    const size_t scratch_bytes = workspace_bytes - fwd_rounds_bytes(cfg, dtype);
    LSH_TRY(lsh_hash(cfg, dtype, q, R, buckets, scratch, scratch_bytes, stream));
    LSH_TRY(lsh_sort_permute(cfg, buckets, perm, undo, bucket_start, scratch, scratch_bytes, stream));
    LSH_TRY(lsh_chunk_attn_fwd(cfg, dtype, q, v, buckets, perm, undo, bucket_start, o_rounds,
                               o_exp, lse_rounds, scratch, scratch_bytes, stream));
    return lsh_combine_rounds(cfg, dtype, o_rounds, o_exp, lse_rounds, undo, out, lse_total, stream);
}

int lsh_chunk_attn_bwd(const lsh_config* cfg, lsh_dtype dtype, const void* q, const void* v,
                       const void* out, const void* dout, const float* lse_total,
                       const int32_t* buckets, const int32_t* perm, const int32_t* undo,
                       const int32_t* bucket_start, float* dq, float* dv, void* workspace,
                       size_t workspace_bytes, void* stream) {
    LSH_TRY(check_config(cfg));
    LSH_TRY(check_dtype(dtype));
    if (!q || !v || !out || !dout || !lse_total || !buckets || !perm || !undo || !bucket_start ||
        !dq || !dv || !workspace)
        return LSH_ERR_INVALID;
    if (!all_aligned(q, v, out, dout, dq, dv, workspace)) return LSH_ERR_INVALID;
    if (workspace_bytes < lsh::bwd_workspace_bytes(bh_of(cfg), cfg->L, cfg->n_rounds))
        return LSH_ERR_INVALID;
    LSH_TRY(check_supported(cfg));
    LSH_TRY(check_chunk(cfg, dtype, true));
    LSH_TRY(check_self_mask(cfg));
    if (dtype != LSH_BF16) return LSH_ERR_UNSUPPORTED;
    return status_of(lsh::launch_attn_bwd(bh_of(cfg), cfg->L, cfg->n_rounds, cfg->n_buckets,
                                          cfg->causal != 0, cfg->scale, cfg->self_mask, q, v, out,
                                          dout, lse_total, buckets, perm, undo, bucket_start, dq,
                                          dv, workspace, static_cast<hipStream_t>(stream)));
}

int lsh_dense_attn_fwd(const lsh_config* cfg, lsh_dtype dtype, const void* q, const void* v,
                       void* out, float* lse, void* workspace, size_t workspace_bytes,
                       void* stream) {
    LSH_TRY(check_dense_config(cfg));
    LSH_TRY(check_dtype(dtype));
    if (!q || !v || !out || !workspace) return LSH_ERR_INVALID;
    if (!all_aligned(q, v, out, workspace)) return LSH_ERR_INVALID;
    if (workspace_bytes < lsh::dense_workspace_bytes(bh_of(cfg), cfg->L)) return LSH_ERR_INVALID;
    LSH_TRY(check_dense_supported(cfg, dtype));
    return status_of(lsh::launch_dense_fwd(bh_of(cfg), cfg->L, cfg->causal != 0, cfg->scale,
                                           cfg->self_mask, q, v, out, lse, workspace,
                                           static_cast<hipStream_t>(stream)));
}

}  // extern "C"

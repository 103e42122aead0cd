// The C ABI of the reversible block (declared in include/lsh_block.h):
// validation, workspace carving, and the chain LayerNorm -> products -> LSH
// attention -> product for F, LayerNorm -> product -> product per row chunk
// for G (Reformer Sec. 3).  Validation runs before any HIP call.
#include "lsh_block.h"

#include <cmath>

#include "launch.h"

namespace {

constexpr int64_t kMaxOffsetElems = ((int64_t)1 << 31) - 64;  // buffer offsets stay below 2^32 bytes

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
template <typename... P>
bool all_aligned(P... p) {
    return (aligned16(p) && ...);
}

int status_of(hipError_t e) { return e == hipSuccess ? LSH_OK : LSH_ERR_HIP; }

#define LSH_TRY(expr)                  \
    do {                               \
        const int _st = (expr);        \
        if (_st != LSH_OK) return _st; \
    } while (0)

int64_t rows_of(const lsh_block_config* c) { return (int64_t)c->attn.B * c->attn.L; }
int d_model(const lsh_block_config* c) { return 64 * c->attn.H; }
int64_t ff_rows(const lsh_block_config* c) {
    const int64_t M = rows_of(c);
    return c->ff_chunk > 0 && c->ff_chunk < M ? c->ff_chunk : M;
}

int check_block(const lsh_block_config* c) {
    if (!c) return LSH_ERR_INVALID;
    if (lsh_workspace_bytes(&c->attn, LSH_BF16, LSH_OP_FORWARD) == 0) return LSH_ERR_INVALID;
    if (c->d_ff < 1 || !std::isfinite(c->ln_eps) || c->ln_eps < 0.f) return LSH_ERR_INVALID;
    LSH_TRY(lsh::attention_fwd_supported(&c->attn, LSH_BF16));
    const int D = d_model(c);
    if (D % 128 != 0 || D > 4096 || c->d_ff % 128 != 0) return LSH_ERR_UNSUPPORTED;
    const int64_t wide = D > c->d_ff ? D : c->d_ff;
    if (rows_of(c) * wide >= kMaxOffsetElems) return LSH_ERR_UNSUPPORTED;
    return LSH_OK;
}

int check_weights(const lsh_block_weights* w, bool attn, bool ff) {
    if (!w) return LSH_ERR_INVALID;
    if (attn && (!w->ln1_g || !w->ln1_b || !w->w_qk || !w->w_v || !w->w_o || !w->R)) return LSH_ERR_INVALID;
    if (ff && (!w->ln2_g || !w->ln2_b || !w->w1 || !w->b1 || !w->w2 || !w->b2)) return LSH_ERR_INVALID;
    if (attn && !all_aligned(w->ln1_g, w->ln1_b, w->w_qk, w->w_v, w->w_o, w->R)) return LSH_ERR_INVALID;
    if (ff && !all_aligned(w->ln2_g, w->ln2_b, w->w1, w->b1, w->w2, w->b2)) return LSH_ERR_INVALID;
    return LSH_OK;
}

// F's workspace: the normalised rows, q, v and the attention's output (bf16,
// [B][H][L][64]), the total log-partition, the ids and permutations, and the
// LSH forward's own workspace; each 256-byte aligned.
struct AttnWs {
    uint16_t *ln, *q, *v, *ao;
    float* lse;
    int32_t *buckets, *perm, *undo, *bstart;
    void* fwd;
    size_t fwd_bytes, bytes;
};

AttnWs carve_attn(const lsh_block_config* c, void* base) {
    using lsh::align256;
    const lsh_config& a = c->attn;
    const size_t M = (size_t)rows_of(c), D = (size_t)d_model(c);
    const size_t BHL = (size_t)a.B * a.H * a.L;
    char* p = static_cast<char*>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char* r = p ? p + off : nullptr;
        off += align256(bytes);
        return r;
    };
    AttnWs w{};
    w.ln = reinterpret_cast<uint16_t*>(take(M * D * 2));
    w.q = reinterpret_cast<uint16_t*>(take(M * D * 2));
    w.v = reinterpret_cast<uint16_t*>(take(M * D * 2));
    w.ao = reinterpret_cast<uint16_t*>(take(M * D * 2));
    w.lse = reinterpret_cast<float*>(take(BHL * 4));
    w.buckets = reinterpret_cast<int32_t*>(take(BHL * a.n_rounds * 4));
    w.perm = reinterpret_cast<int32_t*>(take(BHL * a.n_rounds * 4));
    w.undo = reinterpret_cast<int32_t*>(take(BHL * a.n_rounds * 4));
    w.bstart = reinterpret_cast<int32_t*>(take((size_t)a.B * a.H * a.n_rounds * (a.n_buckets + 1) * 4));
    w.fwd_bytes = lsh_workspace_bytes(&a, LSH_BF16, LSH_OP_FORWARD);
    w.fwd = take(w.fwd_bytes);
    w.bytes = off;
    return w;
}

// G's workspace: one chunk's normalised rows and hidden layer (bf16).
struct FfWs {
    uint16_t *ln, *h;
    size_t bytes;
};

FfWs carve_ff(const lsh_block_config* c, void* base) {
    using lsh::align256;
    const size_t R = (size_t)ff_rows(c);
    char* p = static_cast<char*>(base);
    FfWs w{};
    w.ln = reinterpret_cast<uint16_t*>(p);
    const size_t ln_bytes = align256(R * d_model(c) * 2);
    w.h = p ? reinterpret_cast<uint16_t*>(p + ln_bytes) : nullptr;
    w.bytes = ln_bytes + align256(R * (size_t)c->d_ff * 2);
    return w;
}

size_t ws_need(const lsh_block_config* c, int op) {
    const size_t a = carve_attn(c, nullptr).bytes, f = carve_ff(c, nullptr).bytes;
    switch (op) {
        case LSH_BLOCK_OP_ATTN: return a;
        case LSH_BLOCK_OP_FF: return f;
        case LSH_BLOCK_OP_BLOCK: return a > f ? a : f;
        default: return 0;
    }
}

int check_ws(const lsh_block_config* c, int op, const void* ws, size_t bytes) {
    if (!ws || !aligned16(ws) || bytes < ws_need(c, op)) return LSH_ERR_INVALID;
    return LSH_OK;
}

// out = resid + sign F(x); arguments already checked.
int run_attention(const lsh_block_config* c, const lsh_block_weights* w, const float* x, const float* resid,
                  float* out, float sign, void* ws, hipStream_t st) {
    const AttnWs a = carve_attn(c, ws);
    const int64_t M = rows_of(c);
    const int D = d_model(c);
    LSH_TRY(status_of(lsh::launch_layer_norm(x, w->ln1_g, w->ln1_b, a.ln, M, D, c->ln_eps, st)));
    const auto* wqk = static_cast<const uint16_t*>(w->w_qk);
    const auto* wv = static_cast<const uint16_t*>(w->w_v);
    LSH_TRY(status_of(lsh::launch_linear(a.ln, false, c->attn.L, c->attn.H, wqk, M, D, D, nullptr,
                                         lsh::kLinearHeads, nullptr, 0.f, nullptr, a.q, st)));
    LSH_TRY(status_of(lsh::launch_linear(a.ln, false, c->attn.L, c->attn.H, wv, M, D, D, nullptr,
                                         lsh::kLinearHeads, nullptr, 0.f, nullptr, a.v, st)));
    LSH_TRY(lsh_attention_fwd(&c->attn, LSH_BF16, a.q, a.v, w->R, a.ao, a.lse, a.buckets, a.perm, a.undo,
                              a.bstart, a.fwd, a.fwd_bytes, st));
    return status_of(lsh::launch_linear(a.ao, true, c->attn.L, c->attn.H, static_cast<const uint16_t*>(w->w_o),
                                        M, D, D, nullptr, lsh::kLinearResid, resid, sign, out, nullptr, st));
}

// out = resid + sign G(x), chunk by chunk of rows.
int run_feed_forward(const lsh_block_config* c, const lsh_block_weights* w, const float* x, const float* resid,
                     float* out, float sign, void* ws, hipStream_t st) {
    const FfWs f = carve_ff(c, ws);
    const int64_t M = rows_of(c), R = ff_rows(c);
    const int D = d_model(c);
    for (int64_t s = 0; s < M; s += R) {
        const int64_t rows = M - s < R ? M - s : R;
        LSH_TRY(status_of(lsh::launch_layer_norm(x + s * D, w->ln2_g, w->ln2_b, f.ln, rows, D, c->ln_eps, st)));
        LSH_TRY(status_of(lsh::launch_linear(f.ln, false, 0, 0, static_cast<const uint16_t*>(w->w1), rows,
                                             c->d_ff, D, w->b1, lsh::kLinearReluBf16, nullptr, 0.f, nullptr,
                                             f.h, st)));
        LSH_TRY(status_of(lsh::launch_linear(f.h, false, 0, 0, static_cast<const uint16_t*>(w->w2), rows, D,
                                             c->d_ff, w->b2, lsh::kLinearResid, resid ? resid + s * D : nullptr,
                                             sign, out + s * D, nullptr, st)));
    }
    return LSH_OK;
}

}  // namespace

extern "C" {

size_t lsh_block_workspace_bytes(const lsh_block_config* cfg, int op) {
    if (check_block(cfg) == LSH_ERR_INVALID) return 0;
    return ws_need(cfg, op);
}

int lsh_rev_attention(const lsh_block_config* cfg, const lsh_block_weights* w, const float* x,
                      const float* resid, float* out, float sign, void* workspace, size_t workspace_bytes,
                      void* stream) {
    LSH_TRY(check_block(cfg));
    LSH_TRY(check_weights(w, true, false));
    if (!x || !out || !all_aligned(x, out) || (resid && !aligned16(resid)) || !std::isfinite(sign))
        return LSH_ERR_INVALID;
    LSH_TRY(check_ws(cfg, LSH_BLOCK_OP_ATTN, workspace, workspace_bytes));
    return run_attention(cfg, w, x, resid, out, sign, workspace, static_cast<hipStream_t>(stream));
}

int lsh_rev_feed_forward(const lsh_block_config* cfg, const lsh_block_weights* w, const float* x,
                         const float* resid, float* out, float sign, void* workspace, size_t workspace_bytes,
                         void* stream) {
    LSH_TRY(check_block(cfg));
    LSH_TRY(check_weights(w, false, true));
    if (!x || !out || !all_aligned(x, out) || (resid && !aligned16(resid)) || !std::isfinite(sign))
        return LSH_ERR_INVALID;
    LSH_TRY(check_ws(cfg, LSH_BLOCK_OP_FF, workspace, workspace_bytes));
    return run_feed_forward(cfg, w, x, resid, out, sign, workspace, static_cast<hipStream_t>(stream));
}

int lsh_rev_block_fwd(const lsh_block_config* cfg, const lsh_block_weights* w, const float* x1, const float* x2,
                      float* y1, float* y2, void* workspace, size_t workspace_bytes, void* stream) {
    LSH_TRY(check_block(cfg));
    LSH_TRY(check_weights(w, true, true));
    if (!x1 || !x2 || !y1 || !y2 || !all_aligned(x1, x2, y1, y2)) return LSH_ERR_INVALID;
    LSH_TRY(check_ws(cfg, LSH_BLOCK_OP_BLOCK, workspace, workspace_bytes));
    const hipStream_t st = static_cast<hipStream_t>(stream);
    LSH_TRY(run_attention(cfg, w, x2, x1, y1, 1.f, workspace, st));
    return run_feed_forward(cfg, w, y1, x2, y2, 1.f, workspace, st);
}

int lsh_rev_block_inv(const lsh_block_config* cfg, const lsh_block_weights* w, const float* y1, const float* y2,
                      float* x1, float* x2, void* workspace, size_t workspace_bytes, void* stream) {
    LSH_TRY(check_block(cfg));
    LSH_TRY(check_weights(w, true, true));
    if (!x1 || !x2 || !y1 || !y2 || !all_aligned(x1, x2, y1, y2)) return LSH_ERR_INVALID;
    LSH_TRY(check_ws(cfg, LSH_BLOCK_OP_BLOCK, workspace, workspace_bytes));
    const hipStream_t st = static_cast<hipStream_t>(stream);
    LSH_TRY(run_feed_forward(cfg, w, y1, y2, x2, -1.f, workspace, st));
    return run_attention(cfg, w, x2, y1, x1, -1.f, workspace, st);
}

int lsh_linear_bf16(int64_t M, int32_t N, int32_t K, const void* a, const void* w, const float* bias,
                    const float* resid, float sign, float* out_f32, void* out_bf16, void* stream) {
    if (M < 0 || N < 1 || K < 1 || !a || !w || (!out_f32 && !out_bf16) || !std::isfinite(sign))
        return LSH_ERR_INVALID;
    if (!all_aligned(a, w) || (bias && !aligned16(bias)) || (resid && !aligned16(resid)) ||
        (out_f32 && !aligned16(out_f32)) || (out_bf16 && !aligned16(out_bf16)))
        return LSH_ERR_INVALID;
    if (N % 128 != 0 || K % 64 != 0) return LSH_ERR_UNSUPPORTED;
    if (M * (N > K ? N : K) >= kMaxOffsetElems) return LSH_ERR_UNSUPPORTED;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    if (out_f32)
        return status_of(lsh::launch_linear(static_cast<const uint16_t*>(a), false, 0, 0,
                                            static_cast<const uint16_t*>(w), M, N, K, bias, lsh::kLinearResid,
                                            resid, sign, out_f32, nullptr, st));
    return status_of(lsh::launch_linear(static_cast<const uint16_t*>(a), false, 0, 0, static_cast<const uint16_t*>(w),
                                        M, N, K, bias, lsh::kLinearReluBf16, nullptr, 0.f, nullptr,
                                        static_cast<uint16_t*>(out_bf16), st));
}

}  // extern "C"

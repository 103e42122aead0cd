/*
 * liblsh, reversible block: the RevNet block of the Reformer around LSH
 * attention (Kitaev, Kaiser and Levskaya, "Reformer: The Efficient
 * Transformer", Sec. 3, "RevNets", "Reversible Transformer", "Chunking").
 *
 *   forward:  y1 = x1 + F(x2),   y2 = x2 + G(y1)
 *   inverse:  x2 = y2 - G(y1),   x1 = y1 - F(x2)
 *
 * F is the attention layer and G the feed-forward layer, each with its
 * LayerNorm inside the residual branch:
 *   F(x) = concat_h( LSHAttention(q_h, v_h) ) W_o^T,
 *          q = LN1(x) W_qk^T, v = LN1(x) W_v^T split into H heads of 64
 *          (shared-QK: the keys are the normalised queries, Sec. 2);
 *   G(x) = relu( LN2(x) W1^T + b1 ) W2^T + b2, computed on chunks of
 *          ff_chunk rows one after another (the result does not depend on
 *          the chunk size; only the scratch memory does).
 * Every product takes bf16 operands and accumulates in fp32: the normalised
 * rows, q and v, the attention output and the hidden layer are rounded to
 * bf16 where they enter a product.  The residual streams x1, x2, y1, y2 are
 * fp32.  The activation (ReLU) is a reading: the paper does not name it.
 *
 * Conventions are those of lsh.h (device pointers, caller-owned memory and
 * workspace, asynchronous calls on `stream`, lsh_status results, INVALID and
 * UNSUPPORTED returned before any HIP call).  Additionally:
 *   x1, x2, y1, y2, out, resid   [B][L][d_model] fp32, d_model = 64 * attn.H
 *   w_qk, w_v     [64 H][d_model]  bf16 (out x in, as a linear layer's weight)
 *   w_o           [d_model][64 H]  bf16
 *   w1 [d_ff][d_model], w2 [d_model][d_ff]  bf16;  b1 [d_ff], b2 [d_model] fp32
 *   ln*_g, ln*_b  [d_model] fp32;  R as in lsh.h
 * Every tensor must be 16-byte aligned.  Outputs must not alias inputs.
 * Supported: the attention configurations of lsh_attention_fwd in bf16,
 * d_model = 64 H a multiple of 128 and at most 4096, d_ff a multiple of 128,
 * B*L*max(d_model, d_ff) < 2^31 (LSH_ERR_UNSUPPORTED otherwise).
 */
#ifndef LSH_BLOCK_H
#define LSH_BLOCK_H

#include "lsh.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lsh_block_config {
    lsh_config attn;  /* the attention's configuration: B, H, L, d = 64, hashing and chunking */
    int32_t d_ff;     /* feed-forward width */
    int32_t ff_chunk; /* rows of the feed-forward per chunk; <= 0: all B*L rows at once */
    float ln_eps;     /* LayerNorm epsilon (added to the variance) */
} lsh_block_config;

typedef struct lsh_block_weights {
    const float *ln1_g, *ln1_b;
    const void *w_qk, *w_v, *w_o;
    const float *R;
    const float *ln2_g, *ln2_b;
    const void *w1;
    const float *b1;
    const void *w2;
    const float *b2;
} lsh_block_weights;

typedef enum lsh_block_op {
    LSH_BLOCK_OP_ATTN = 0,  /* lsh_rev_attention */
    LSH_BLOCK_OP_FF = 1,    /* lsh_rev_feed_forward */
    LSH_BLOCK_OP_BLOCK = 2  /* lsh_rev_block_fwd and lsh_rev_block_inv */
} lsh_block_op;

/* Workspace bytes an entry point needs (0 for an invalid configuration). */
size_t lsh_block_workspace_bytes(const lsh_block_config *cfg, int op);

/* out = resid + sign * F(x)   (Sec. 3, "Reversible Transformer": F is the
 * attention layer with its LayerNorm inside).  resid may be NULL (then 0);
 * sign is +1 for the forward residual and -1 for the inverse. */
int lsh_rev_attention(const lsh_block_config *cfg, const lsh_block_weights *w, const float *x,
                      const float *resid, float *out, float sign, void *workspace,
                      size_t workspace_bytes, void *stream);

/* out = resid + sign * G(x), G the feed-forward layer run on chunks of
 * cfg->ff_chunk rows (Sec. 3, "Chunking").  resid may be NULL. */
int lsh_rev_feed_forward(const lsh_block_config *cfg, const lsh_block_weights *w, const float *x,
                         const float *resid, float *out, float sign, void *workspace,
                         size_t workspace_bytes, void *stream);

/* (y1, y2) = (x1 + F(x2), x2 + G(y1))   (Sec. 3, "RevNets"). */
int lsh_rev_block_fwd(const lsh_block_config *cfg, const lsh_block_weights *w, const float *x1,
                      const float *x2, float *y1, float *y2, void *workspace,
                      size_t workspace_bytes, void *stream);

/* (x1, x2) from (y1, y2): x2 = y2 - G(y1), then x1 = y1 - F(x2)
 * (Sec. 3, eq. reverse-ff).  Reproduces x1, x2 up to the rounding of the
 * fp32 residual additions whenever F(x2) is evaluated on the same bf16
 * operands as in the forward. */
int lsh_rev_block_inv(const lsh_block_config *cfg, const lsh_block_weights *w, const float *y1,
                      const float *y2, float *x1, float *x2, void *workspace,
                      size_t workspace_bytes, void *stream);

/* The block's product, exposed for tests: for a [M][K] bf16, w [N][K] bf16
 * (N a multiple of 128, K of 64), out_f32 = resid + sign * (a w^T + bias)
 * when out_f32 is given, else out_bf16 = bf16(relu(a w^T + bias)).  bias and
 * resid may be NULL. */
int lsh_linear_bf16(int64_t M, int32_t N, int32_t K, const void *a, const void *w,
                    const float *bias, const float *resid, float sign, float *out_f32,
                    void *out_bf16, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LSH_BLOCK_H */

/*
 * liblsh: Reformer LSH attention on one MI355X (gfx950).
 *
 * C ABI over hand-written HIP kernels.  The operation is the LSH attention of
 * Kitaev, Kaiser and Levskaya, "Reformer: The Efficient Transformer" (ICLR
 * 2020): shared-QK angular hashing, a per-round sort by (bucket, position),
 * chunked attention of every chunk of m sorted queries to its own and the
 * previous chunk, and a log-sum-exp weighted combination of the rounds.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * Pointers.  Every tensor argument is a DEVICE pointer to contiguous,
 *   row-major memory that the caller allocated and owns; the library never
 *   allocates, frees or synchronises.  Inputs are only read.  Outputs must
 *   not alias inputs or each other.  q, v, R, dout, the row outputs and the
 *   workspace must be 16-byte aligned (LSH_ERR_INVALID otherwise).
 * Layouts.  "BH" is B*H flattened, batch-major.
 *   q, v, dout        [B][H][L][d]        dtype of the call (fp32 or bf16)
 *   R                 [n_rounds][d][n_buckets/2]   fp32
 *   buckets           [B][H][L][n_rounds] int32    (a token's ids adjacent)
 *   perm, undo        [B][H][n_rounds][L] int32    perm: sorted slot -> position,
 *                                                   undo: position -> sorted slot
 *   bucket_start      [B][H][n_rounds][n_buckets+1] int32: first sorted slot of
 *                     each bucket, last entry = L
 *   o_rounds          [B][H][n_rounds][L][d] sorted-slot order: fp32 for fp32
 *                     calls; for bf16 calls IEEE fp16, each row scaled by
 *                     2^-o_exp[row] (11 significant bits, so that the combined
 *                     output is rounded to bf16 only once)
 *   o_exp             [B][H][n_rounds][L]    uint8, sorted-slot order (bf16 calls
 *                     only): 0 unless a row's largest magnitude reaches 2^15
 *   lse_rounds        [B][H][n_rounds][L]    fp32, sorted-slot order
 *   out               [B][H][L][d]        dtype of the call
 *   lse_total         [B][H][L]           fp32
 *   dq, dv            [B][H][L][d]        fp32
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  Calls
 *   only enqueue work and return; results are ready when the stream is.
 * Workspace.  Entry points that need scratch memory take a device buffer of
 *   at least lsh_workspace_bytes(cfg, dtype, op) bytes, 256-byte aligned.
 * Errors.  Every entry point returns an lsh_status.  LSH_ERR_INVALID and
 *   LSH_ERR_UNSUPPORTED are returned before any HIP call is made, so they can
 *   be tested without a GPU; LSH_ERR_HIP reports a failed launch.  No C++
 *   exception crosses this interface.  The library keeps no mutable global
 *   state (apart from lsh_sort_permute_static's fixed scratch array), so
 *   calls on different streams may run concurrently.
 * self_mask.  The attention entry points (lsh_chunk_attn_fwd and _bwd,
 *   lsh_attention_fwd, lsh_dense_attn_fwd) return LSH_ERR_UNSUPPORTED for
 *   self_mask < 1e4.  The kernels give a token's own key weight zero whenever
 *   the token has another target, and treat a token whose total
 *   log-partition is below -self_mask/2 as its own only target; both are
 *   exact in fp32 while self_mask > 2*scale*|q_i| + log(n_rounds) + 17 for
 *   every row (App. A sets the self mask to 1e5).
 * Supported on the GPU: d = 64; on the forward (both dtypes) chunk = 64 or
 *   128 (the length of the paper's usual configuration, Sec. 5) and
 *   chunks_after <= 1; attend_across on the fp32 forward only; the backward
 *   takes chunk = 64 without look-ahead or attend_across (LSH_ERR_UNSUPPORTED
 *   otherwise; entry points that do not use the chunk ignore it);
 *   r_per_head everywhere; 2 <= n_buckets <= 1024 (even), 1 <= n_rounds <= 16,
 *   B*H*L*n_rounds < 2^31.  L need not be a multiple of
 *   the chunk: the last chunk then holds the L mod m remaining sorted slots
 *   (the paper is silent; read as padding with tokens that are no one's
 *   target).
 */
#ifndef LSH_H
#define LSH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lsh_status {
    LSH_OK = 0,
    LSH_ERR_INVALID = -1,     /* NULL pointer, bad size, bad workspace */
    LSH_ERR_UNSUPPORTED = -2, /* valid, but not a shape the kernels handle */
    LSH_ERR_HIP = -3          /* a HIP launch or runtime call failed */
} lsh_status;

typedef enum lsh_dtype {
    LSH_F32 = 0,  /* IEEE binary32 */
    LSH_BF16 = 1  /* bfloat16; arithmetic accumulates in fp32 */
} lsh_dtype;

/* Which call a workspace is sized for. */
typedef enum lsh_op {
    LSH_OP_HASH = 0,
    LSH_OP_SORT = 1,
    LSH_OP_ATTN_FWD = 2,
    LSH_OP_COMBINE = 3,
    LSH_OP_ATTN_BWD = 4,
    LSH_OP_FORWARD = 5, /* lsh_attention_fwd: all four forward calls */
    LSH_OP_DENSE_FWD = 6 /* lsh_dense_attn_fwd */
} lsh_op;

/* Problem description (Sec. 2 of the paper: one shared Q=K tensor and V of
 * shape [batch, length, d_model] split into heads; b = n_buckets hash
 * buckets from a random R of shape [d_k, b/2]; n_rounds hash functions;
 * chunks of m sorted positions; optional causal masking). */
typedef struct lsh_config {
    int32_t B, H, L, d;
    int32_t n_buckets; /* b: even, >= 2 */
    int32_t n_rounds;  /* number of hash functions, >= 1 */
    int32_t chunk;     /* m: chunk length in sorted slots (the last chunk may be partial) */
    int32_t causal;    /* nonzero: a position never attends to a later one */
    float scale;       /* logit scale, 1/sqrt(d_k) in eq. attn */
    float self_mask;   /* mask value for j == i, 1e5 in App. A */
    /* Variants the paper does not spell out (0 = the paper's method): */
    int32_t chunks_after;  /* look-ahead: the window of chunk c is chunks c-1 .. c+after
                              (one chunk closes the non-causal gap in Sec. 2's claim that
                              buckets smaller than m lie inside the window) */
    int32_t attend_across; /* nonzero: every key of the window is a target, not only the
                              query's bucket; N_ij counts the rounds in which j falls in
                              i's window (App. A with P^(r)_i read as the window) */
    int32_t r_per_head;    /* nonzero: R holds one [n_rounds][d][n_buckets/2] set per head,
                              [H][n_rounds][d][n_buckets/2] */
} lsh_config;

/* Human-readable name of a status code (static storage). */
const char *lsh_status_string(int status);

/* Bytes of workspace `op` needs for this configuration (0 if none). */
size_t lsh_workspace_bytes(const lsh_config *cfg, lsh_dtype dtype, int op);

/* Angular LSH of every query in every round (Sec. 2, "Locality sensitive
 * hashing": h(x) = argmax([xR; -xR]), one R per round as in eq.
 * union-pairs).  R is shared by every batch entry and head, or with
 * r_per_head one set per head, [H][n_rounds][d][n_buckets/2] (each (batch,
 * head) slice is then hashed in its own pass).  The hash is of
 * the stored q (the normalised key has the same hash).  Ties in the argmax
 * resolve to the first index of [xR; -xR].  The ids equal those of the exact
 * argmax: projections are screened with bf16 matrix cores under a
 * guaranteed error bound, and every row-round the bound cannot settle is
 * recomputed in fp64.
 *   q        [B][H][L][d] (dtype), R [n_rounds][d][n_buckets/2] fp32
 *   buckets  [B][H][L][n_rounds] int32 (written)
 *   workspace >= lsh_workspace_bytes(cfg, dtype, LSH_OP_HASH) */
int lsh_hash(const lsh_config *cfg, lsh_dtype dtype, const void *q, const float *R,
             int32_t *buckets, void *workspace, size_t workspace_bytes, void *stream);

/* Stable sort of every (batch, head, round) segment by bucket, then by
 * position (Sec. 2, "LSH attention": the permutation i -> s_i; App. A:
 * s^(r) per round), as a counting sort.
 *   buckets       [B][H][L][n_rounds] int32, ids in [0, n_buckets)
 *   perm, undo    [B][H][n_rounds][L] int32 (written)
 *   bucket_start  [B][H][n_rounds][n_buckets+1] int32 (written)
 *   workspace >= lsh_workspace_bytes(cfg, dtype, LSH_OP_SORT)
 * Ids outside [0, n_buckets) give unspecified (but in-bounds) results. */
int lsh_sort_permute(const lsh_config *cfg, const int32_t *buckets, int32_t *perm,
                     int32_t *undo, int32_t *bucket_start, void *workspace,
                     size_t workspace_bytes, void *stream);

/* lsh_sort_permute without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops).
 * Its scratch (per-tile bucket counts, 4 * B*H*n_rounds*n_buckets*ceil(L/4096)
 * bytes) is a fixed 16 MiB device array inside the library, one per GPU,
 * held until the process ends; its address is looked up on the first call
 * on each device (the current device).  The call allocates nothing.
 * Configurations whose counts exceed 16 MiB return LSH_ERR_UNSUPPORTED.
 * Every call on a GPU shares that GPU's array: calls that may overlap on one
 * GPU (other streams, other host threads) race and must be serialised by the
 * caller.  Each call writes every count it reads, so no state carries over
 * from the previous call.  Arguments and results as lsh_sort_permute. */
int lsh_sort_permute_static(const lsh_config *cfg, const int32_t *buckets, int32_t *perm,
                            int32_t *undo, int32_t *bucket_start, void *stream);

/* Gather rows into sorted order (the "chunks of m consecutive queries after
 * sorting" of Sec. 2): dst[b][h][r][s] = src[b][h][perm[b][h][r][s]].
 * lsh_chunk_attn_fwd performs this gather itself while staging its chunks;
 * this call exists for callers that want the sorted copies.
 *   src  [B][H][L][d] (dtype), dst [B][H][n_rounds][L][d] (dtype, written) */
int lsh_gather_rows(const lsh_config *cfg, lsh_dtype dtype, const void *src,
                    const int32_t *perm, void *dst, void *stream);

/* One round of chunked LSH attention for every sorted query, all rounds at
 * once (App. A: o^(r)_i and z(i, P^(r)_i)).  The query at sorted slot s, in
 * chunk c = floor(s/m), attends to the keys at slots of chunks c-1 and c
 * (the set P~ of Sec. 2; chunk 0 has no previous chunk), with keys
 * k_j = q_j/|q_j| and logits scale*q_i.k_j - m^(r)_ij, where m^(r)_ij is
 * infinite for keys of another bucket and for later positions under causal
 * masking, self_mask for j == i, and log N_ij otherwise (N_ij: number of
 * rounds in which j shares i's bucket).
 *   q, v          [B][H][L][d] (dtype), in original position order
 *   buckets, perm, bucket_start: as written by lsh_hash / lsh_sort_permute
 *   undo          as written by lsh_sort_permute; read only with attend_across
 *                 (where it must not be NULL; it may be NULL otherwise)
 *   o_rounds      [B][H][n_rounds][L][d] (written, sorted order): each round's
 *                 output, accumulated and normalised in fp32, stored as fp32
 *                 (fp32 calls) or as fp16 scaled by 2^-o_exp (bf16 calls)
 *   o_exp         [B][H][n_rounds][L] uint8 (written; bf16 calls, where it must
 *                 not be NULL; ignored and may be NULL for fp32 calls)
 *   lse_rounds    [B][H][n_rounds][L] fp32 (written, sorted order)
 *   workspace     >= lsh_workspace_bytes(cfg, dtype, LSH_OP_ATTN_FWD) bytes
 *                 (per-token key scales and packed bucket ids for bf16 calls;
 *                 0 bytes, and workspace may be NULL, for fp32 calls) */
int lsh_chunk_attn_fwd(const lsh_config *cfg, lsh_dtype dtype, const void *q, const void *v,
                       const int32_t *buckets, const int32_t *perm, const int32_t *undo,
                       const int32_t *bucket_start, void *o_rounds, uint8_t *o_exp,
                       float *lse_rounds, void *workspace, size_t workspace_bytes,
                       void *stream);

/* Undo the sort and combine the rounds (App. A):
 *   z_i = log sum_r exp z_r(i),  out_i = sum_r exp(z_r(i) - z_i) o_r(i).
 *   o_rounds, o_exp, lse_rounds: as written by lsh_chunk_attn_fwd (o_exp
 *                 required for bf16 calls); the weighted sum is formed in fp32
 *   undo          [B][H][n_rounds][L] int32
 *   out           [B][H][L][d] (dtype, written)
 *   lse_total     [B][H][L] fp32 (written; may be NULL) */
int lsh_combine_rounds(const lsh_config *cfg, lsh_dtype dtype, const void *o_rounds,
                       const uint8_t *o_exp, const float *lse_rounds, const int32_t *undo,
                       void *out, float *lse_total, void *stream);

/* The whole forward: lsh_hash, lsh_sort_permute, lsh_chunk_attn_fwd and
 * lsh_combine_rounds in sequence on one stream.  buckets, perm, undo and
 * bucket_start are outputs because the backward needs them; o_rounds, o_exp
 * and lse_rounds live in the workspace.
 *   workspace >= lsh_workspace_bytes(cfg, dtype, LSH_OP_FORWARD) */
int lsh_attention_fwd(const lsh_config *cfg, lsh_dtype dtype, const void *q, const void *v,
                      const float *R, void *out, float *lse_total, int32_t *buckets,
                      int32_t *perm, int32_t *undo, int32_t *bucket_start, void *workspace,
                      size_t workspace_bytes, void *stream);

/* Gradients of the combined output with respect to q (through both the
 * query role and the key role, including k = q/|q|) and v, with the buckets
 * held fixed (argmax has zero gradient almost everywhere).  Logits are
 * recomputed from q, perm and lse_total, as the paper recomputes attention
 * in the backward pass of memory-efficient attention (Sec. 2).  The paper
 * does not state the LSH backward; this is the exact derivative of the
 * forward above.
 *   q, v, out, dout  [B][H][L][d] (dtype); out as written by the forward
 *   lse_total        [B][H][L] fp32 from the forward
 *   buckets, perm, undo, bucket_start: from the forward
 *   dq, dv           [B][H][L][d] fp32 (overwritten)
 *   workspace >= lsh_workspace_bytes(cfg, dtype, LSH_OP_ATTN_BWD)
 * bf16 only on the GPU. */
int lsh_chunk_attn_bwd(const lsh_config *cfg, lsh_dtype dtype, const void *q, const void *v,
                       const void *out, const void *dout, const float *lse_total,
                       const int32_t *buckets, const int32_t *perm, const int32_t *undo,
                       const int32_t *bucket_start, float *dq, float *dv, void *workspace,
                       size_t workspace_bytes, void *stream);

/* Full shared-QK attention, the memory-efficient baseline of Sec. 2: every
 * query's softmax over all keys computed without materialising QK^T.  Keys
 * are k_j = q_j/|q_j| (a zero row gives k = 0), the logit of query i and
 * key j is scale*q_i.k_j, self_mask is subtracted for j == i (App. A), and
 * under causal masking no key later than i counts (Sec. 2, "Causal masking
 * for shared-QK attention").  This is what the LSH forward approximates; with
 * one bucket, one round and a chunk covering the sequence the two coincide.
 * It is the baseline of the paper's speed-versus-length comparison (Sec. 5).
 *   q, v      [B][H][L][d] bf16, position order
 *   out       [B][H][L][d] bf16 (written); accumulated in fp32
 *   lse       [B][H][L] fp32 log-partition (written; may be NULL)
 *   workspace >= lsh_workspace_bytes(cfg, dtype, LSH_OP_DENSE_FWD): per-row
 *             key scales
 * Only B, H, L, d, causal, scale and self_mask of cfg are read; the hashing
 * fields are ignored (n_buckets, n_rounds and chunk are not validated).
 * bf16 only, d = 64, B*H < 65536 and B*H*L < 2^31 on the GPU (otherwise
 * LSH_ERR_UNSUPPORTED). */
int lsh_dense_attn_fwd(const lsh_config *cfg, lsh_dtype dtype, const void *q, const void *v,
                       void *out, float *lse, void *workspace, size_t workspace_bytes,
                       void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LSH_H */

/*
 * Reference CPU implementation of Reformer LSH attention
 * (Kitaev, Kaiser, Levskaya, "Reformer: The Efficient Transformer", ICLR 2020).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the oracle that the GPU path is
 * checked against.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark may load it; the GPU library never links, calls or
 * includes anything from here, and this file includes nothing from it.
 *
 * Everything is computed in double precision with plain loops, in the order
 * the paper states the method.  Inputs arrive as doubles (bf16 and fp32
 * tensors convert to double exactly).  OpenMP splits independent rows,
 * segments or (batch, head) slices; no loop is blocked or reordered.
 *
 * Layouts (row-major, "BH" = batch * heads flattened):
 *   q, v, dout, out, dq, dv : [BH][L][d]
 *   R                       : [n_rounds][d][n_buckets/2]
 *   buckets, near_tie       : [BH][L][n_rounds]   (one token's ids adjacent)
 *   perm, undo              : [BH][n_rounds][L]   perm: sorted slot -> position,
 *                                                  undo: position -> sorted slot
 *   o_rounds                : [BH][n_rounds][L][d] (sorted-slot order)
 *   lse_rounds              : [BH][n_rounds][L]    (sorted-slot order)
 *   lse_total               : [BH][L]
 *
 * Readings of points the paper leaves open (each also listed in the design
 * notes of the repository):
 *   - the hash is taken of the stored query q (k = q/|q| has the same hash in
 *     exact arithmetic); argmax ties go to the first index of [qR; -qR];
 *   - logits are scale * q_i.k_j with scale = 1/sqrt(d_k) (Sec. 2, eq. attn),
 *     and the App. A mask term is subtracted after scaling;
 *   - mask precedence is: other bucket -> excluded; causal future -> excluded;
 *     self -> self_mask (1e5); otherwise log N_ij; N_ij counts the rounds in
 *     which j shares i's bucket, whether or not j falls in i's window;
 *   - the window has no wrap-around: chunk 0 looks back at nothing;
 *   - when m does not divide L the last chunk holds the L mod m remaining
 *     slots (as if the sequence were padded with tokens that are no one's
 *     target);
 *   - a zero query gives k = 0;
 *   - variants the paper does not spell out, each off by default: a
 *     look-ahead of `after` chunks (the window of chunk c is chunks
 *     c-1 .. c+after; the paper's P~ is after = 0), attending across buckets
 *     (the target set of round r is the window itself instead of the bucket
 *     within it, so App. A applies with P^(r)_i read as P~^(r)_i and N_ij
 *     counts the rounds in which j falls in i's window), and one R per head
 *     (R holds H_R sets [n_rounds][d][n_buckets/2]; a row of head h uses set
 *     h mod H_R).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define REF_OK 0
#define REF_ERR_INVALID -1
#define REF_ERR_NOMEM -4

/* Number of threads the parallel loops below use (reporting only). */
int lsh_ref_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

static double dot(const double *a, const double *b, int64_t d)
{
    double s = 0.0;
    for (int64_t t = 0; t < d; ++t) s += a[t] * b[t];
    return s;
}

/* |q_j| for every row: the key of row j is q_j / |q_j| (Sec. 2, "LSH
 * attention": keys are set to the normalised queries so h(k_j) = h(q_j)). */
static void row_norms(int64_t rows, int64_t d, const double *q, double *norm)
{
#pragma omp parallel for schedule(static)
    for (int64_t row = 0; row < rows; ++row)
        norm[row] = sqrt(dot(q + row * d, q + row * d, d));
}

/* Angular LSH (Sec. 2, "Locality sensitive hashing"): with a random R of
 * shape [d_k, b/2], h(x) = argmax([xR; -xR]).  One R per round (Sec. 2,
 * "Multi-round LSH attention", eq. union-pairs).  H_R = 1: one R shared by
 * every batch entry and head; H_R = H: one R per head, a row of slice bh
 * (bh = b*H + h) using set bh mod H_R.  near_tie marks row-rounds whose two
 * largest entries of [xR; -xR] differ by less than 1e-6 of the largest (or
 * are equal). */
int lsh_ref_hash(int64_t BH, int64_t L, int64_t d, int64_t n_buckets,
                 int64_t n_rounds, int64_t H_R, const double *q, const double *R,
                 int32_t *buckets, uint8_t *near_tie)
{
    if (BH < 0 || L < 0 || d < 1 || n_buckets < 2 || n_buckets % 2 ||
        n_rounds < 1 || H_R < 1 || !q || !R || !buckets)
        return REF_ERR_INVALID;
    const int64_t half = n_buckets / 2;
    const int64_t rows = BH * L;
    int err = 0;
#pragma omp parallel
    {
        double *vals = (double *)malloc((size_t)n_buckets * sizeof(double));
        if (!vals) {
#pragma omp atomic write
            err = 1;
        }
#pragma omp for schedule(static)
        for (int64_t row = 0; row < rows; ++row) {
            if (!vals) continue;
            const double *x = q + row * d;
            const double *Rh = R + ((row / (L > 0 ? L : 1)) % H_R) * n_rounds * d * half;
            for (int64_t r = 0; r < n_rounds; ++r) {
                const double *Rr = Rh + r * d * half;
                /* [xR; -xR] */
                for (int64_t c = 0; c < half; ++c) {
                    double p = 0.0;
                    for (int64_t t = 0; t < d; ++t) p += x[t] * Rr[t * half + c];
                    vals[c] = p;
                    vals[half + c] = -p;
                }
                int64_t best = 0;
                for (int64_t c = 1; c < n_buckets; ++c)
                    if (vals[c] > vals[best]) best = c;
                double second = -INFINITY;
                for (int64_t c = 0; c < n_buckets; ++c)
                    if (c != best && vals[c] > second) second = vals[c];
                buckets[row * n_rounds + r] = (int32_t)best;
                if (near_tie)
                    near_tie[row * n_rounds + r] =
                        (uint8_t)((vals[best] - second) < 1e-6 * fabs(vals[best]) ||
                                  vals[best] == second);
            }
        }
        free(vals);
    }
    return err ? REF_ERR_NOMEM : REF_OK;
}

typedef struct {
    int32_t bucket;
    int32_t pos;
} ref_item;

static int cmp_item(const void *a, const void *b)
{
    const ref_item *x = (const ref_item *)a, *y = (const ref_item *)b;
    if (x->bucket != y->bucket) return x->bucket < y->bucket ? -1 : 1;
    return (x->pos > y->pos) - (x->pos < y->pos);
}

/* Sort by bucket and, inside a bucket, by sequence position (Sec. 2, "LSH
 * attention"), separately for every round (App. A, s^(r)).  The key
 * (bucket, position) is unique, so the order is unique. */
int lsh_ref_sort_permute(int64_t BH, int64_t L, int64_t n_rounds,
                         const int32_t *buckets, int32_t *perm, int32_t *undo)
{
    if (BH < 0 || L < 0 || n_rounds < 1 || !buckets || !perm || !undo)
        return REF_ERR_INVALID;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t seg = 0; seg < BH * n_rounds; ++seg) {
        const int64_t bh = seg / n_rounds, r = seg % n_rounds;
        ref_item *items = (ref_item *)malloc((size_t)(L > 0 ? L : 1) * sizeof(ref_item));
        if (!items) {
#pragma omp atomic write
            err = 1;
            continue;
        }
        for (int64_t i = 0; i < L; ++i) {
            items[i].bucket = buckets[(bh * L + i) * n_rounds + r];
            items[i].pos = (int32_t)i;
        }
        qsort(items, (size_t)L, sizeof(ref_item), cmp_item);
        int32_t *p = perm + (bh * n_rounds + r) * L;
        int32_t *u = undo + (bh * n_rounds + r) * L;
        for (int64_t s = 0; s < L; ++s) {
            p[s] = items[s].pos;
            u[items[s].pos] = (int32_t)s;
        }
        free(items);
    }
    return err ? REF_ERR_NOMEM : REF_OK;
}

/* N_ij of App. A: the number of rounds in which j lands in i's bucket. */
static int64_t n_shared(const int32_t *buckets, int64_t base, int64_t i,
                        int64_t j, int64_t n_rounds)
{
    int64_t n = 0;
    for (int64_t r = 0; r < n_rounds; ++r)
        n += buckets[(base + i) * n_rounds + r] == buckets[(base + j) * n_rounds + r];
    return n;
}

/* Attending across buckets: the number of rounds in which key j lies in
 * query i's window, chunks floor(s_i/m) - 1 .. floor(s_i/m) + after of that
 * round's sorted order (undo: position -> slot, [n_rounds][L] of the
 * slice). */
static int64_t n_window(const int32_t *undo, int64_t L, int64_t i, int64_t j,
                        int64_t n_rounds, int64_t chunk, int64_t after)
{
    int64_t n = 0;
    for (int64_t r = 0; r < n_rounds; ++r) {
        const int64_t ci = undo[r * L + i] / chunk, cj = undo[r * L + j] / chunk;
        n += cj >= ci - 1 && cj <= ci + after;
    }
    return n;
}

/* Mask term m^(r)_ij of App. A for query i and key j in round r.  Returns 0
 * when j is not a target at all (other bucket, or the future under causal
 * masking, Sec. 2 "Causal masking for shared-QK attention"); otherwise sets
 * *M to 1e5 for j == i and to log N_ij for every other target.  Across
 * buckets (undo non-NULL) no key of the window is dropped for its bucket
 * and N_ij counts window memberships. */
static int mask_term(const int32_t *buckets, const int32_t *undo, int64_t L,
                     int64_t chunk, int64_t after, int64_t base, int64_t i,
                     int64_t j, int64_t r, int64_t n_rounds, int causal,
                     double self_mask, double *M)
{
    if (!undo && buckets[(base + j) * n_rounds + r] != buckets[(base + i) * n_rounds + r])
        return 0;
    if (causal && j > i) return 0;
    if (j == i)
        *M = self_mask;
    else if (undo)
        *M = log((double)n_window(undo, L, i, j, n_rounds, chunk, after));
    else
        *M = log((double)n_shared(buckets, base, i, j, n_rounds));
    return 1;
}

/* undo[slice][r][perm[slice][r][s]] = s, for the across-buckets counts. */
static int32_t *undo_of(int64_t BH, int64_t n_rounds, int64_t L, const int32_t *perm)
{
    int32_t *u = (int32_t *)malloc((size_t)(BH * n_rounds * L > 0 ? BH * n_rounds * L : 1) *
                                   sizeof(int32_t));
    if (!u) return NULL;
    for (int64_t seg = 0; seg < BH * n_rounds; ++seg)
        for (int64_t s = 0; s < L; ++s) u[seg * L + perm[seg * L + s]] = (int32_t)s;
    return u;
}

/* One round of chunked LSH attention for every query (App. A, o^(r)_i and
 * z(i, P^(r)_i)).  The query at sorted slot s, in chunk c = floor(s/m),
 * looks at the keys whose slots lie in chunks c-1 .. c+after (the set P~ of
 * Sec. 2 for after = 0), with logits a_ij = scale * q_i.k_j - m^(r)_ij. */
int lsh_ref_chunk_attn_fwd(int64_t BH, int64_t L, int64_t d, int64_t n_rounds,
                           int64_t chunk, int64_t after, int across, int causal,
                           double scale, double self_mask, const double *q,
                           const double *v, const int32_t *buckets,
                           const int32_t *perm, double *o_rounds,
                           double *lse_rounds)
{
    if (BH < 0 || L < 0 || d < 1 || n_rounds < 1 || chunk < 1 || after < 0 ||
        !q || !v || !buckets || !perm || !o_rounds ||
        !lse_rounds)
        return REF_ERR_INVALID;
    double *norm = (double *)malloc((size_t)(BH * L > 0 ? BH * L : 1) * sizeof(double));
    if (!norm) return REF_ERR_NOMEM;
    int32_t *undo = across ? undo_of(BH, n_rounds, L, perm) : NULL;
    if (across && !undo) {
        free(norm);
        return REF_ERR_NOMEM;
    }
    row_norms(BH * L, d, q, norm);
    const int64_t span = (2 + after) * chunk; /* keys in a window */
    int err = 0;
#pragma omp parallel
    {
        double *a = (double *)malloc((size_t)span * sizeof(double));
        int64_t *tgt = (int64_t *)malloc((size_t)span * sizeof(int64_t));
        if (!a || !tgt) {
#pragma omp atomic write
            err = 1;
        }
#pragma omp for schedule(static)
        for (int64_t idx = 0; idx < BH * n_rounds * L; ++idx) {
            if (!a || !tgt) continue;
            const int64_t bh = idx / (n_rounds * L);
            const int64_t r = (idx / L) % n_rounds;
            const int64_t s = idx % L;
            const int64_t base = bh * L;
            const int32_t *p = perm + (bh * n_rounds + r) * L;
            const int64_t i = p[s];
            const int64_t c = s / chunk;
            const int64_t t_lo = (c - 1) * chunk < 0 ? 0 : (c - 1) * chunk;
            const int64_t t_hi = (c + 1 + after) * chunk < L ? (c + 1 + after) * chunk : L;
            const double *qi = q + (base + i) * d;
            const int32_t *u = undo ? undo + bh * n_rounds * L : NULL;
            int64_t n = 0;
            double amax = -INFINITY;
            for (int64_t t = t_lo; t < t_hi; ++t) {
                const int64_t j = p[t];
                double M;
                if (!mask_term(buckets, u, L, chunk, after, base, i, j, r, n_rounds, causal,
                               self_mask, &M))
                    continue;
                const double nj = norm[base + j];
                const double qk = nj > 0.0 ? dot(qi, q + (base + j) * d, d) / nj : 0.0;
                a[n] = scale * qk - M;
                tgt[n] = j;
                if (a[n] > amax) amax = a[n];
                ++n;
            }
            /* j = i is always a target, so n >= 1 and z is finite. */
            double sum = 0.0;
            for (int64_t e = 0; e < n; ++e) sum += exp(a[e] - amax);
            const double z = amax + log(sum);
            double *o = o_rounds + ((bh * n_rounds + r) * L + s) * d;
            for (int64_t t = 0; t < d; ++t) o[t] = 0.0;
            for (int64_t e = 0; e < n; ++e) {
                const double w = exp(a[e] - z);
                const double *vj = v + (base + tgt[e]) * d;
                for (int64_t t = 0; t < d; ++t) o[t] += w * vj[t];
            }
            lse_rounds[(bh * n_rounds + r) * L + s] = z;
        }
        free(a);
        free(tgt);
    }
    free(norm);
    free(undo);
    return err ? REF_ERR_NOMEM : REF_OK;
}

/* Full shared-QK attention, the memory-efficient baseline of Sec. 2 ("the
 * attention can be computed for each query separately"): for query i of the
 * (batch, head) slice starting at row `base`, the softmax over all keys
 * k_j = q_j/|q_j| of a_ij = scale * q_i.k_j, with self_mask subtracted for
 * j == i and, under causal masking, no j later than i (Sec. 2, "Causal
 * masking for shared-QK attention").  The LSH forward approximates exactly
 * this; it is the speed baseline of the paper's speed-versus-length
 * comparison (Sec. 5).  a: scratch of L doubles. */
static void dense_row(int64_t L, int64_t d, int causal, double scale, double self_mask,
                      const double *q, const double *v, const double *norm, int64_t base,
                      int64_t i, double *a, double *o, double *z_out)
{
    const int64_t n = causal ? i + 1 : L; /* keys 0 .. n-1 */
    const double *qi = q + (base + i) * d;
    double amax = -INFINITY;
    for (int64_t j = 0; j < n; ++j) {
        const double nj = norm[base + j];
        const double qk = nj > 0.0 ? dot(qi, q + (base + j) * d, d) / nj : 0.0;
        a[j] = scale * qk - (j == i ? self_mask : 0.0);
        if (a[j] > amax) amax = a[j];
    }
    /* j = i is always a key, so n >= 1 and z is finite. */
    double sum = 0.0;
    for (int64_t j = 0; j < n; ++j) sum += exp(a[j] - amax);
    const double z = amax + log(sum);
    for (int64_t t = 0; t < d; ++t) o[t] = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        const double w = exp(a[j] - z);
        const double *vj = v + (base + j) * d;
        for (int64_t t = 0; t < d; ++t) o[t] += w * vj[t];
    }
    *z_out = z;
}

/* Dense attention for `n_sel` selected rows (sel: flat row index bh*L + i
 * into [BH][L]); out [n_sel][d], lse [n_sel].  All rows when sel is NULL
 * (then n_sel must be BH*L and out is [BH][L][d]). */
int lsh_ref_dense_attn_fwd(int64_t BH, int64_t L, int64_t d, int causal,
                           double scale, double self_mask, const double *q,
                           const double *v, int64_t n_sel, const int64_t *sel,
                           double *out, double *lse)
{
    if (BH < 0 || L < 0 || d < 1 || !q || !v || !out || !lse || n_sel < 0)
        return REF_ERR_INVALID;
    if (!sel && n_sel != BH * L) return REF_ERR_INVALID;
    for (int64_t k = 0; sel && k < n_sel; ++k)
        if (sel[k] < 0 || sel[k] >= BH * L) return REF_ERR_INVALID;
    double *norm = (double *)malloc((size_t)(BH * L > 0 ? BH * L : 1) * sizeof(double));
    if (!norm) return REF_ERR_NOMEM;
    row_norms(BH * L, d, q, norm);
    int err = 0;
#pragma omp parallel
    {
        double *a = (double *)malloc((size_t)(L > 0 ? L : 1) * sizeof(double));
        if (!a) {
#pragma omp atomic write
            err = 1;
        }
#pragma omp for schedule(static)
        for (int64_t k = 0; k < n_sel; ++k) {
            if (!a) continue;
            const int64_t row = sel ? sel[k] : k;
            dense_row(L, d, causal, scale, self_mask, q, v, norm, (row / L) * L, row % L, a,
                      out + k * d, lse + k);
        }
        free(a);
    }
    free(norm);
    return err ? REF_ERR_NOMEM : REF_OK;
}

/* Undo the sort and combine the rounds (App. A):
 *   z(i, P_i) = log sum_r exp z(i, P^(r)_i),
 *   o_i = sum_r exp(z(i, P^(r)_i) - z(i, P_i)) o^(r)_i. */
int lsh_ref_combine_rounds(int64_t BH, int64_t L, int64_t d, int64_t n_rounds,
                           const double *o_rounds, const double *lse_rounds,
                           const int32_t *undo, double *out, double *lse_total)
{
    if (BH < 0 || L < 0 || d < 1 || n_rounds < 1 || !o_rounds || !lse_rounds ||
        !undo || !out)
        return REF_ERR_INVALID;
#pragma omp parallel for schedule(static)
    for (int64_t row = 0; row < BH * L; ++row) {
        const int64_t bh = row / L, i = row % L;
        double zmax = -INFINITY;
        for (int64_t r = 0; r < n_rounds; ++r) {
            const int64_t s = undo[(bh * n_rounds + r) * L + i];
            const double zr = lse_rounds[(bh * n_rounds + r) * L + s];
            if (zr > zmax) zmax = zr;
        }
        double sum = 0.0;
        for (int64_t r = 0; r < n_rounds; ++r) {
            const int64_t s = undo[(bh * n_rounds + r) * L + i];
            sum += exp(lse_rounds[(bh * n_rounds + r) * L + s] - zmax);
        }
        const double z = zmax + log(sum);
        double *o = out + row * d;
        for (int64_t t = 0; t < d; ++t) o[t] = 0.0;
        for (int64_t r = 0; r < n_rounds; ++r) {
            const int64_t s = undo[(bh * n_rounds + r) * L + i];
            const double w = exp(lse_rounds[(bh * n_rounds + r) * L + s] - z);
            const double *orow = o_rounds + ((bh * n_rounds + r) * L + s) * d;
            for (int64_t t = 0; t < d; ++t) o[t] += w * orow[t];
        }
        if (lse_total) lse_total[row] = z;
    }
    return REF_OK;
}

/* Gradient of the combined output with respect to q and v, buckets held
 * fixed.  The combined output is one softmax over every (round, key) entry
 * (r, j) of query i with logit a^(r)_ij (App. A), so with
 * P = exp(a - z(i, P_i)) and D_i = dO_i . o_i:
 *   dv_j    += P dO_i
 *   dA       = P (dO_i . v_j - D_i)
 *   dq_i    += scale dA k_j            (query role)
 *   dk_j    += scale dA q_i            (key role)
 * and the key role flows back through k_j = q_j/|q_j|:
 *   dq_j    += (dk_j - (dk_j . k_j) k_j) / |q_j|.
 * The logits are recomputed from q, as the paper does for memory-efficient
 * attention (Sec. 2, "Memory-efficient attention"). */
int lsh_ref_chunk_attn_bwd(int64_t BH, int64_t L, int64_t d, int64_t n_rounds,
                           int64_t chunk, int64_t after, int across, int causal,
                           double scale, double self_mask, const double *q,
                           const double *v, const double *out,
                           const double *dout, const double *lse_total,
                           const int32_t *buckets, const int32_t *perm,
                           double *dq, double *dv)
{
    if (BH < 0 || L < 0 || d < 1 || n_rounds < 1 || chunk < 1 || after < 0 ||
        !q || !v || !out || !dout || !lse_total ||
        !buckets || !perm || !dq || !dv)
        return REF_ERR_INVALID;
    int32_t *undo = across ? undo_of(BH, n_rounds, L, perm) : NULL;
    if (across && !undo) return REF_ERR_NOMEM;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t bh = 0; bh < BH; ++bh) {
        const int64_t base = bh * L;
        double *norm = (double *)malloc((size_t)(L > 0 ? L : 1) * sizeof(double));
        double *dk = (double *)calloc((size_t)(L * d > 0 ? L * d : 1), sizeof(double));
        double *kj = (double *)malloc((size_t)d * sizeof(double));
        if (!norm || !dk || !kj) {
#pragma omp atomic write
            err = 1;
            free(norm);
            free(dk);
            free(kj);
            continue;
        }
        row_norms(L, d, q + base * d, norm);
        for (int64_t e = 0; e < L * d; ++e) {
            dq[base * d + e] = 0.0;
            dv[base * d + e] = 0.0;
        }
        for (int64_t r = 0; r < n_rounds; ++r) {
            const int32_t *p = perm + (bh * n_rounds + r) * L;
            for (int64_t s = 0; s < L; ++s) {
                const int64_t i = p[s];
                const int64_t c = s / chunk;
                const int64_t t_lo = (c - 1) * chunk < 0 ? 0 : (c - 1) * chunk;
                const int64_t t_hi = (c + 1 + after) * chunk < L ? (c + 1 + after) * chunk : L;
                const double *qi = q + (base + i) * d;
                const double *dOi = dout + (base + i) * d;
                const double Di = dot(dOi, out + (base + i) * d, d);
                const double zi = lse_total[base + i];
                const int32_t *u = undo ? undo + bh * n_rounds * L : NULL;
                for (int64_t t = t_lo; t < t_hi; ++t) {
                    const int64_t j = p[t];
                    double M;
                    if (!mask_term(buckets, u, L, chunk, after, base, i, j, r, n_rounds, causal,
                                   self_mask, &M))
                        continue;
                    const double nj = norm[j];
                    for (int64_t u = 0; u < d; ++u)
                        kj[u] = nj > 0.0 ? q[(base + j) * d + u] / nj : 0.0;
                    const double a = scale * dot(qi, kj, d) - M;
                    const double P = exp(a - zi);
                    const double *vj = v + (base + j) * d;
                    const double dA = P * (dot(dOi, vj, d) - Di);
                    for (int64_t u = 0; u < d; ++u) {
                        dv[(base + j) * d + u] += P * dOi[u];
                        dq[(base + i) * d + u] += scale * dA * kj[u];
                        dk[j * d + u] += scale * dA * qi[u];
                    }
                }
            }
        }
        for (int64_t j = 0; j < L; ++j) {
            const double nj = norm[j];
            if (!(nj > 0.0)) continue;
            for (int64_t u = 0; u < d; ++u) kj[u] = q[(base + j) * d + u] / nj;
            const double proj = dot(dk + j * d, kj, d);
            for (int64_t u = 0; u < d; ++u)
                dq[(base + j) * d + u] += (dk[j * d + u] - proj * kj[u]) / nj;
        }
        free(norm);
        free(dk);
        free(kj);
    }
    free(undo);
    return err ? REF_ERR_NOMEM : REF_OK;
}

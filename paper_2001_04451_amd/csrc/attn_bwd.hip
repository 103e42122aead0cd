// Backward of chunked LSH attention (gradients with respect to q and v,
// buckets held fixed).  The paper gives no LSH backward; it recomputes
// attention in the backward pass of its memory-efficient attention (Sec. 2),
// and this follows that: the logits of every round are recomputed from q,
// perm and the forward's total log-partition z_i, with
//   P = exp(a - z_i),  dA = P (dO_i . v_j - D_i),  D_i = dO_i . o_i,
//   dv_j += P dO_i,  dq_i += scale dA k_j,  dk_j += scale dA q_i,
// and dk flows back through k_j = q_j/|q_j|:
//   dq_j += (dk_j - (dk_j . k_j) k_j) / |q_j|.
//
// Kernels (gfx950):
//  * bwd_prep:   one record per token: its packed bucket ids, its key scale
//                scale*log2(e)/|q|, its log-partition in log2 units and
//                D = dO . o.
//  * bwd_strip:  twelve waves walk a strip of chunks of one (batch, head,
//                round) segment: eight own key blocks (pass 1 and the
//                finishing below), four form dQ (pass 2).  Step c takes the queries of chunk c
//                against the 128 keys of chunks c-1 and c (their whole
//                window), so every (query, key) pair of the round is met in
//                exactly one step, and the keys of chunk c meet their last
//                queries in step c+1.  The rows sit in LDS rings (q rows and
//                records: four slots, v: three, dO: two), and chunk c+1 is
//                gathered into the free slots (through perm, straight from
//                global memory into LDS) while step c computes.  A step runs
//                the finishing of chunk c-2's key blocks and pass 1 of step c
//                on the key waves while the dQ waves run pass 2 of step c-1,
//                with dA'^T and dQ double-buffered, so it needs a single
//                barrier.
//                Pass 1, lanes on keys: each wave owns one 16-key block of
//                one chunk for the two steps in which that chunk is in the
//                window.  Per 16x16 tile S = Q K^T and dP = dO V^T on the
//                matrix cores, then P, dA and dA' = dA * scale/|q_j| per
//                element; P (as bf16 hi + lo, so dv keeps fp32 accuracy) and
//                dA are already the B operands of dV^T += dO^T P and
//                dK^T += Q^T dA, and dA' goes to LDS transposed.
//                Pass 2, lanes on queries: dQ^T += K^T dA'^T over the window,
//                with dA'^T read back through the LDS transpose read; dQ goes
//                to LDS for the step that finishes those tokens as keys.
//                The step after a key block's chunk leaves the window, its
//                owner adds dk through the normalisation Jacobian to dQ (the
//                same 16 tokens) and writes the round's partials of dq and dv, in
//                sorted-slot order (whole contiguous rows; scattering them to
//                position order here costs more than gathering them below),
//                as fp16 rows scaled by 2^-e (e = 0 unless a row's largest
//                magnitude reaches 2^15; one byte per row).
//  * bwd_reduce: per position, the sum over rounds, each round's partial
//                gathered through undo; plus dO for a token that was its own
//                only target in every round (its weights are then 1/n_rounds
//                on each round's self entry).
// Every (query, key) pair of a round is computed once, by one lane, and every
// sum has a fixed order: no atomics, and the results are deterministic.
#include "attn_common.h"
#include "launch.h"

#include <type_traits>

namespace lsh {
namespace {

constexpr int kMaskedIndex = 32;  // table index of a masked-out pair
constexpr int kKeyWaves = 8;                      // waves owning key blocks (passes 1 and the finishing)
constexpr int kBwdThreads = (kKeyWaves + 4) * 64;  // plus four dQ waves (pass 2)

// Per-token record: signature words [0, SW), then the key scale, the total
// log-partition in log2 units and D, in the last three words.
template <int NW>
struct BwdRec {
    static constexpr int SW = sig_stride(NW);
    static constexpr int RW = SW + 3 <= 4 ? 4 : (SW + 3 <= 8 ? 8 : 12);
};

// LDS of one workgroup.  Step c reads the q rows and records of chunks
// c-2 .. c (the finishing of chunk c-2, the dQ of chunk c-1, the pairs of
// step c) and gathers chunk c+1: a four-slot ring; v rows are read for
// chunks c-1 and c (three slots), dO rows for chunk c (two slots).  dA'^T
// and dQ are double-buffered by the parity of their chunk, and the query
// fields (interval, log-partition, D, signature words) kept for three
// chunks, so that a step needs one barrier.  Beyond four signature words
// (more than eight rounds) the signature words are read from the records.
template <int NW>
struct BwdShared {
    static constexpr int kQSlots = 4, kVSlots = 3, kDSlots = 2;
    static constexpr int kQsigWords = NW >= 1 && NW <= 4 ? NW : 1;
    char Qs[kQSlots * kChunk * 128];  // q rows (swizzled)
    char Vs[kVSlots * kChunk * 128];  // v rows
    char Ds[kDSlots * kChunk * 128];  // dO rows
    char Ts[2][2 * kChunk * 128];     // dA'^T: 128 window keys x 64 queries (bf16), by step parity
    float X[2][kChunk * kHeadDim];    // dQ of a chunk's tokens, [token][dim] (see xoff), by chunk parity
    uint32_t rec[kQSlots * kChunk][BwdRec<NW>::RW];
    // per chunk (three chunks: c-1, c and the one set up for c+1), per
    // query: its key interval in window rows (lo | hi << 16, both in
    // 0 .. 127), its log-partition (log2 units) and D, and its signature
    // words, laid out so that a lane reads its four queries' fields as
    // 16-byte runs
    uint32_t lohi[3][kChunk];
    float2 zd[3][kChunk];
    uint32_t qsig[3][kQsigWords][kChunk];
    float tab[kMaskedIndex + 1];      // -log2 N by mismatch count; -inf = masked
};
static_assert(sizeof(BwdShared<4>) <= 160 * 1024 && sizeof(BwdShared<8>) <= 160 * 1024, "LDS");

// Row i of chunk `chunk` in a ring of SLOTS chunk slots.
template <int SLOTS>
__device__ __forceinline__ int slot_row(int chunk, int i) {
    return ((chunk % SLOTS + SLOTS) % SLOTS) * kChunk + i;
}

// Float offset of dims 4cb .. 4cb+3 of token t in a dQ buffer: rows of 64
// floats, their 16-byte groups xor-swizzled by the row so that the 16 tokens
// a lane group touches fall in different banks.
__device__ __forceinline__ int xoff(int t, int cb) { return t * kHeadDim + ((cb ^ (t & 7)) << 2); }

template <int NW, bool CAUSAL>
__global__ __launch_bounds__(kBwdThreads, 1) void bwd_strip_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const uint32_t* __restrict__ rec,
    const int32_t* __restrict__ perm, uint16_t* __restrict__ part_q, uint16_t* __restrict__ part_v,
    uint8_t* __restrict__ part_e, int L, int n_r, float scale, int chunks_per_strip) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    using Shared = BwdShared<NW>;
    Shared& S = *reinterpret_cast<Shared*>(smem);
    constexpr int SW = BwdRec<NW>::SW, RW = BwdRec<NW>::RW;
    constexpr bool kWaveSig = NW >= 1 && NW <= 4;  // per-wave signature copies
    auto ring_row = [](int chunk, int i) { return slot_row<Shared::kQSlots>(chunk, i); };
    auto ringv_row = [](int chunk, int i) { return slot_row<Shared::kVSlots>(chunk, i); };
    auto ring2_row = [](int chunk, int i) { return slot_row<Shared::kDSlots>(chunk, i); };

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 15, g = lane >> 4;
    const int64_t seg = blockIdx.y;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int n_chunks = (L + kChunk - 1) / kChunk;
    const int c0 = blockIdx.x * chunks_per_strip;
    const int c1 = min(n_chunks, c0 + chunks_per_strip);
    const int32_t* pseg = perm + seg * L;
    const int64_t rowbase = bh * L;
    const float scale_log2e = scale * kLog2e;
    if (tid <= kMaskedIndex) S.tab[tid] = tid < n_r ? -__log2f((float)(n_r - tid)) : -__builtin_inff();

    // Position of slot `lane` of chunk cc (any valid row for slots outside the
    // sequence: they are never a valid key or query, and write nothing).
    auto chunk_pos = [&](int cc) -> int {
        const int slot = cc * kChunk + lane;
        return cc >= 0 && slot < L ? pseg[slot] : 0;
    };
    // Gather chunk cc into its ring slots (dQ waves only, so that the key
    // waves issue no global loads): dQ wave w copies q, v and dO rows
    // 16w .. 16w+15 (each lane the 16-byte piece that belongs at its LDS
    // slot), and dQ wave 0 also the whole chunk's records, which it then
    // reads to set up the chunk's query fields (set_queries).
    const int dw = wave - kKeyWaves;  // dQ wave index (0..3 on the dQ waves)
    auto stage = [&](int cc, int pos_raw) {
        const int pos_lane = min(max(pos_raw, 0), L - 1);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int r0 = 16 * dw + 8 * h;
            const int row = r0 + (lane >> 3);
            const int p = __shfl(pos_lane, row);
            const int64_t off = (rowbase + p) * kHeadDim + swz(row, lane & 7) * 8;
            copy16_to_lds(q + off, S.Qs + ring_row(cc, r0) * 128);
            copy16_to_lds(v + off, S.Vs + ringv_row(cc, r0) * 128);
            copy16_to_lds(dout + off, S.Ds + ring2_row(cc, r0) * 128);
        }
        constexpr int U = RW / 4;  // 16-byte units per record
        if (dw == 0) {
#pragma unroll
            for (int k = 0; k < U; ++k) {
                const int u = 64 * k + lane, rr = u / U;
                const int pr = __shfl(pos_lane, rr);
                copy16_to_lds(rec + (rowbase + pr) * RW + 4 * (u % U), &S.rec[ring_row(cc, 0)][0] + 256 * k);
            }
        }
    };
    // The query fields of chunk cc (dQ wave 0, lane = query, once the records of
    // chunks cc-1 and cc are in LDS): each query's key interval [lo, hi] in
    // window rows (0..63: chunk cc-1, 64..127: chunk cc) from the bucket
    // boundaries of the window, its log-partition and D, its signature words.
    auto set_queries = [&](int cc) {
        const uint32_t kA = sig_round_id(&S.rec[ring_row(cc - 1, lane)][0], r);
        const uint32_t kB = sig_round_id(&S.rec[ring_row(cc, lane)][0], r);
        const uint32_t prevA = __shfl_up(kA, 1);
        const uint32_t lastA = __shfl(kA, 63);
        const uint32_t prevB0 = __shfl_up(kB, 1);
        const uint32_t prevB = lane == 0 ? lastA : prevB0;
        const uint64_t bA = __ballot(lane == 0 || kA != prevA);
        const uint64_t bB = __ballot(kB != prevB);
        const uint64_t upto = bB & (~0ull >> (63 - lane));
        const int lo_w = upto ? 127 - __clzll(upto) : 63 - __clzll(bA);
        int lo_q = max(lo_w, (1 - cc) * kChunk);  // no slot before 0
        int hi_q;
        if constexpr (CAUSAL) {
            hi_q = kChunk + lane - 1;
        } else {
            const uint64_t after = lane < 63 ? bB & (~0ull << (lane + 1)) : 0ull;
            hi_q = after ? 62 + __ffsll((long long)after) : 127;
        }
        hi_q = min(hi_q, L - 1 - (cc - 1) * kChunk);  // no slot past the sequence
        if (cc * kChunk + lane >= L) {                // no query here
            lo_q = 1;
            hi_q = 0;
        }
        const int buf = cc % 3;
        S.lohi[buf][lane] = (uint32_t)lo_q | ((uint32_t)hi_q << 16);
        const uint32_t* qrec = &S.rec[ring_row(cc, lane)][0];
        S.zd[buf][lane] = make_float2(__uint_as_float(qrec[RW - 2]), __uint_as_float(qrec[RW - 1]));
        if constexpr (kWaveSig) {
#pragma unroll
            for (int w = 0; w < NW; ++w) S.qsig[buf][w][lane] = qrec[w];
        }
    };
    // whether the query of this lane, in the step of chunk cc, reaches window
    // block kw
    auto reaches = [&](int cc, int kw) {
        const uint32_t lh = S.lohi[cc % 3][lane];
        const int lo = (int)(lh & 0xFFFFu), hi = (int)(lh >> 16);
        return lo <= hi && lo <= 16 * kw + 15 && hi >= 16 * kw;
    };

    const bool key_wave = wave < kKeyWaves;
    int pf_pos = 0;
    if (!key_wave) {
        stage(c0 - 1, chunk_pos(c0 - 1));
        stage(c0, chunk_pos(c0));
        pf_pos = chunk_pos(c0 + 1);
    }
    __builtin_amdgcn_s_waitcnt(0);
    if (dw == 0) set_queries(c0);
    __syncthreads();

    // This wave's key block: block b of every chunk of parity cp, held for
    // the two steps in which the chunk is in the window and finished at the
    // start of the step after (when its tokens' dQ is complete).
    const int b = wave & 3, cp = wave >> 2;
    f32x4 accK[4] = {f32x4{}, f32x4{}, f32x4{}, f32x4{}};  // dK^T by 16-dim blocks
    f32x4 accV[4] = {f32x4{}, f32x4{}, f32x4{}, f32x4{}};  // dV^T

    // Step c: (A) the key waves of chunk c's parity finish their key block of
    // chunk c-2; (B) the dQ waves form dQ of chunk c-1's queries from the
    // dA'^T of step c-1; (C) the key waves take the pairs of chunk c's
    // queries with the keys of chunks c-1 and c.
    for (int c = c0; c <= c1 + 1; ++c) {
        int pf_next = 0;
        if (!key_wave) {
            if (c + 1 <= c1) stage(c + 1, pf_pos);
            pf_next = chunk_pos(c + 2);
        }

        // ---- (A) key block of chunk c-2: its tokens are done as keys (steps
        // c-2, c-1) and as queries (dQ from step c-1) ----
        if (key_wave && (c & 1) == cp) {
            const int kc = c - 2;
            const int t_i = 16 * b + n;
            const int slot = kc * kChunk + t_i;
            if (kc >= c0 && slot < L) {  // chunk c0-1 belongs to the previous strip
                const int tr = ring_row(kc, t_i);
                const float cf = __uint_as_float(S.rec[tr][RW - 3]);
                const float inv = cf * (1.f / scale_log2e);  // 1/|q|, 0 for a zero row
                const float* Xk = S.X[kc & 1];
                f32x4 qv[4], xq[4];
                float kd = 0.f;
#pragma unroll
                for (int bd = 0; bd < 4; ++bd) {
                    const uint2 w2 = *reinterpret_cast<const uint2*>(
                        S.Qs + row_piece_offset(tr, 2 * bd + (g >> 1)) + 8 * (g & 1));
                    qv[bd] = f32x4{__uint_as_float(w2.x << 16), __uint_as_float(w2.x & 0xFFFF0000u),
                                   __uint_as_float(w2.y << 16), __uint_as_float(w2.y & 0xFFFF0000u)};
                    xq[bd] = *reinterpret_cast<const f32x4*>(&Xk[xoff(t_i, 4 * bd + g)]);
#pragma unroll
                    for (int j = 0; j < 4; ++j) kd = fmaf(accK[bd][j], qv[bd][j], kd);
                }
                kd = sum_xor32(sum_xor16(kd));
                const float proj = scale * kd * inv;  // dk . k
                f32x4 a[4];
                float mq = 0.f, mv = 0.f;
#pragma unroll
                for (int bd = 0; bd < 4; ++bd)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        a[bd][j] = kLn2 * xq[bd][j] + (scale * accK[bd][j] - proj * qv[bd][j] * inv) * inv;
                        mq = fmaxf(mq, fabsf(a[bd][j]));
                        mv = fmaxf(mv, fabsf(accV[bd][j]));
                    }
                mq = max_xor32(max_xor16(mq));
                mv = max_xor32(max_xor16(mv));
                // 2^(E-127) <= max < 2^(E-126): e = max(0, E - 141) puts the
                // scaled row below 2^15, inside fp16's range
                const int eq = max(0, (int)((__float_as_uint(mq) >> 23) & 0xFFu) - 141);
                const int ev = max(0, (int)((__float_as_uint(mv) >> 23) & 0xFFu) - 141);
                const float sq = __uint_as_float((uint32_t)(127 - eq) << 23);
                const float sv = __uint_as_float((uint32_t)(127 - ev) << 23);
                const int64_t prow = seg * L + slot;  // sorted order
                uint16_t* dqrow = part_q + prow * kHeadDim;
                uint16_t* dvrow = part_v + prow * kHeadDim;
#pragma unroll
                for (int bd = 0; bd < 4; ++bd) {
                    *reinterpret_cast<uint2*>(dqrow + 16 * bd + 4 * g) =
                        make_uint2(pack_f16x2(a[bd][0] * sq, a[bd][1] * sq), pack_f16x2(a[bd][2] * sq, a[bd][3] * sq));
                    *reinterpret_cast<uint2*>(dvrow + 16 * bd + 4 * g) =
                        make_uint2(pack_f16x2(accV[bd][0] * sv, accV[bd][1] * sv),
                                   pack_f16x2(accV[bd][2] * sv, accV[bd][3] * sv));
                }
                if (g == 0) reinterpret_cast<uint16_t*>(part_e)[prow] = (uint16_t)(eq | (ev << 8));
            }
#pragma unroll
            for (int bd = 0; bd < 4; ++bd) {
                accK[bd] = f32x4{};
                accV[bd] = f32x4{};
            }
        }

        // ---- (B) dQ of query block qb of chunk c-1 over the window of
        // step c-1 (keys of chunks c-2 and c-1) ----
        if (!key_wave && c - 1 >= c0 && c - 1 < c1) {
            const int qb = wave - kKeyWaves;
            const char* Tp = S.Ts[(c - 1) & 1];
            f32x4 dq4[4] = {f32x4{}, f32x4{}, f32x4{}, f32x4{}};
#pragma unroll
            for (int kw2 = 0; kw2 < 8; ++kw2) {
                const uint64_t reach = __ballot(reaches(c - 1, kw2));
                if (((reach >> (16 * qb)) & 0xFFFFull) == 0) continue;
                const bf16x4 bT = vt_read(Tp + vt_offset(16 * kw2, 16 * qb, lane));
                const int kbase = ring_row(c - 2 + (kw2 >> 2), 16 * (kw2 & 3));
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    dq4[i] = mfma16x16x16(vt_read(S.Qs + vt_offset(kbase, 16 * i, lane)), bT, dq4[i]);
            }
            float* Xq = S.X[(c - 1) & 1];
#pragma unroll
            for (int i = 0; i < 4; ++i) *reinterpret_cast<f32x4*>(&Xq[xoff(16 * qb + n, 4 * i + g)]) = dq4[i];
        }

        // ---- (C) step c ----
        if (key_wave && c <= c1) {
            // pass 1: this wave's key block against the 64 queries
            const int k_chunk = (c & 1) == cp ? c : c - 1;  // the chunk of this wave's parity
            const int kw = (k_chunk == c ? 4 : 0) + b;      // its window block
            if (!(k_chunk == c && c == c1)) {               // chunk c1 belongs to the next strip
                // queries that reach this key block (one bit per query)
                const uint64_t qmask = __ballot(reaches(c, kw));
                const int krow = ring_row(k_chunk, 16 * b + n);
                const int krow_v = ringv_row(k_chunk, 16 * b + n);
                const int key_w = 16 * kw + n;
                const uint32_t* krec = &S.rec[krow][0];
                const float cf_k = __uint_as_float(krec[RW - 3]);
                uint32_t ks[NW > 0 ? NW : 1];
#pragma unroll
                for (int w = 0; w < (NW > 0 ? NW : 1); ++w) ks[w] = krec[w];
                const bf16x8 bk0 = as_bf16x8(lds_piece(S.Qs, krow, g));
                const bf16x8 bk1 = as_bf16x8(lds_piece(S.Qs, krow, 4 + g));
                const bf16x8 bv0 = as_bf16x8(lds_piece(S.Vs, krow_v, g));
                const bf16x8 bv1 = as_bf16x8(lds_piece(S.Vs, krow_v, 4 + g));
                char* Tc = S.Ts[c & 1];
#pragma unroll
                for (int qb = 0; qb < 4; ++qb) {
                    if (((qmask >> (16 * qb)) & 0xFFFFull) == 0) continue;
                    const int qrow = ring_row(c, 16 * qb + n);
                    const int drow = ring2_row(c, 16 * qb + n);
                    f32x4 sacc = mfma16x16x32(as_bf16x8(lds_piece(S.Qs, qrow, g)), bk0, f32x4{});
                    sacc = mfma16x16x32(as_bf16x8(lds_piece(S.Qs, qrow, 4 + g)), bk1, sacc);
                    f32x4 dpacc = mfma16x16x32(as_bf16x8(lds_piece(S.Ds, drow, g)), bv0, f32x4{});
                    dpacc = mfma16x16x32(as_bf16x8(lds_piece(S.Ds, drow, 4 + g)), bv1, dpacc);
                    // lane holds queries 16qb + 4g + j (j = 0..3) against key n
                    // the lane's four queries: intervals, log-partitions, D and
                    // signature words, one 16-byte read per field (lane groups
                    // read consecutive runs, so these reads do not conflict)
                    const int q0 = 16 * qb + 4 * g;
                    const int qbuf = c % 3;
                    const u32x4 lh4 = *reinterpret_cast<const u32x4*>(&S.lohi[qbuf][q0]);
                    const f32x4 zd01 = *reinterpret_cast<const f32x4*>(&S.zd[qbuf][q0]);
                    const f32x4 zd23 = *reinterpret_cast<const f32x4*>(&S.zd[qbuf][q0 + 2]);
                    u32x4 qs4[NW > 0 ? NW : 1];
                    if constexpr (NW > 0) {
#pragma unroll
                        for (int w = 0; w < NW; ++w) {
                            if constexpr (kWaveSig) {
                                qs4[w] = *reinterpret_cast<const u32x4*>(&S.qsig[qbuf][w][q0]);
                            } else {
#pragma unroll
                                for (int j = 0; j < 4; ++j) qs4[w][j] = S.rec[ring_row(c, q0 + j)][w];
                            }
                        }
                    }
                    const int lo_a[4] = {(int)(lh4[0] & 0xFFFFu), (int)(lh4[1] & 0xFFFFu), (int)(lh4[2] & 0xFFFFu),
                                         (int)(lh4[3] & 0xFFFFu)};
                    const int hi_a[4] = {(int)(lh4[0] >> 16), (int)(lh4[1] >> 16), (int)(lh4[2] >> 16),
                                         (int)(lh4[3] >> 16)};
                    const float z2_a[4] = {zd01[0], zd01[2], zd23[0], zd23[2]};
                    const float D_a[4] = {zd01[1], zd01[3], zd23[1], zd23[3]};
                    float p[4], da[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        bool valid = lo_a[j] <= key_w && key_w <= hi_a[j];
                        if constexpr (!CAUSAL) valid = valid && key_w != kChunk + q0 + j;
                        uint32_t t = valid ? 0u : ~0u;
                        if constexpr (NW > 0) {
#pragma unroll
                            for (int w = 0; w < NW; ++w)
                                t = and_or((qs4[w][j] ^ ks[w]) + sig_add(w), sig_guard(w), t);
                        }
                        p[j] = __builtin_amdgcn_exp2f(fmaf(sacc[j], cf_k, S.tab[__popc(t)] - z2_a[j]));
                        da[j] = p[j] * (dpacc[j] - D_a[j]);
                    }
                    // P as bf16 hi + lo planes, dA and dA' = dA * scale*log2(e)/|q_j|
                    uint32_t ph[2], pl[2], dab[2], dpb[2];
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2) {
                        ph[h2] = pack_bf16x2(p[2 * h2], p[2 * h2 + 1]);
                        pl[h2] = pack_bf16x2(p[2 * h2] - __uint_as_float(ph[h2] << 16),
                                             p[2 * h2 + 1] - __uint_as_float(ph[h2] & 0xFFFF0000u));
                        dab[h2] = pack_bf16x2(da[2 * h2], da[2 * h2 + 1]);
                        dpb[h2] = pack_bf16x2(da[2 * h2] * cf_k, da[2 * h2 + 1] * cf_k);
                    }
                    const bf16x4 Bph = __builtin_bit_cast(bf16x4, make_uint2(ph[0], ph[1]));
                    const bf16x4 Bpl = __builtin_bit_cast(bf16x4, make_uint2(pl[0], pl[1]));
                    const bf16x4 Bda = __builtin_bit_cast(bf16x4, make_uint2(dab[0], dab[1]));
                    // dA'^T row key_w, queries q0 .. q0+3
                    *reinterpret_cast<uint2*>(Tc + row_piece_offset(key_w, 2 * qb + (g >> 1)) + 8 * (g & 1)) =
                        make_uint2(dpb[0], dpb[1]);
                    const int dbase = ring2_row(c, 16 * qb), qbase = ring_row(c, 16 * qb);
#pragma unroll
                    for (int bd = 0; bd < 4; ++bd) {
                        const bf16x4 dOt = vt_read(S.Ds + vt_offset(dbase, 16 * bd, lane));
                        accV[bd] = mfma16x16x16(dOt, Bph, accV[bd]);
                        accV[bd] = mfma16x16x16(dOt, Bpl, accV[bd]);
                        accK[bd] = mfma16x16x16(vt_read(S.Qs + vt_offset(qbase, 16 * bd, lane)), Bda, accK[bd]);
                    }
                }
            }
        }
        pf_pos = pf_next;
        __builtin_amdgcn_s_waitcnt(0);  // this wave's copies of chunk c+1 have landed
        if (dw == 0 && c + 1 <= c1) set_queries(c + 1);
        __syncthreads();                // ... and every wave is done with step c
    }
}

// Per-token record (see BwdRec): eight lanes per token, one 16-byte piece of
// the q, out and dout rows each; lane p writes record words p (and p + 8).
template <int NW>
__global__ __launch_bounds__(256) void bwd_prep_kernel(const uint16_t* __restrict__ q,
                                                       const uint16_t* __restrict__ out,
                                                       const uint16_t* __restrict__ dout,
                                                       const float* __restrict__ lse_total,
                                                       const int32_t* __restrict__ buckets,
                                                       int64_t rows, int n_r, float scale_log2e,
                                                       uint32_t* __restrict__ rec) {
    constexpr int SW = BwdRec<NW>::SW, RW = BwdRec<NW>::RW;
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 3;
    const int part = threadIdx.x & 7;
    if (row >= rows) return;  // whole groups of eight lanes leave together
    const u32x4 x = *reinterpret_cast<const u32x4*>(q + row * kHeadDim + part * 8);
    const u32x4 o = *reinterpret_cast<const u32x4*>(out + row * kHeadDim + part * 8);
    const u32x4 gd = *reinterpret_cast<const u32x4*>(dout + row * kHeadDim + part * 8);
    float ss = 0.f, D = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(x[e] << 16), hi = __uint_as_float(x[e] & 0xFFFF0000u);
        ss = fmaf(lo, lo, fmaf(hi, hi, ss));
        D = fmaf(__uint_as_float(o[e] << 16), __uint_as_float(gd[e] << 16), D);
        D = fmaf(__uint_as_float(o[e] & 0xFFFF0000u), __uint_as_float(gd[e] & 0xFFFF0000u), D);
    }
    ss = group8_sum(ss);
    D = group8_sum(D);
    const int32_t* brow = buckets + row * n_r;
#pragma unroll
    for (int w = part; w < RW; w += 8) {
        uint32_t word = 0;
        if (w < SW) {
            const uint32_t id0 = 2 * w < n_r ? (uint32_t)brow[2 * w] & 0x3FFu : 0u;
            const uint32_t id1 = 2 * w + 1 < n_r ? (uint32_t)brow[2 * w + 1] & 0x3FFu : 0u;
            word = (id0 << w) | (id1 << (w + 11));
        } else if (w == RW - 3) {
            const float nn = sqrtf(ss);
            word = __float_as_uint(nn > 0.f ? scale_log2e / nn : 0.f);
        } else if (w == RW - 2) {
            word = __float_as_uint(lse_total[row] * kLog2e);
        } else if (w == RW - 1) {
            word = __float_as_uint(D);
        }
        rec[row * RW + w] = word;
    }
}


// dq, dv of a position: the sum of its per-round partials (each at the
// token's slot undo[i] of its round, fixed round order, each fp16 row times
// 2^e), plus dO for a token whose only target in every round was itself.
// Sixteen lanes take kReduceRows adjacent positions (two up to four rounds,
// where the registers allow it at full occupancy; else one), four values of
// each row per lane, with every load of those rows in flight together.
// NRL: n_r rounded up to a power of two; rounds past n_r read round 0 with
// weight 0, so the loads are unconditional.
template <int NRL>
constexpr int reduce_rows() { return NRL <= 4 ? 2 : 1; }

template <int NRL>
__global__ __launch_bounds__(256) void bwd_reduce_kernel(
    const uint16_t* __restrict__ dout, const float* __restrict__ lse_total,
    const uint16_t* __restrict__ part_q, const uint16_t* __restrict__ part_v,
    const uint8_t* __restrict__ part_e, const int32_t* __restrict__ undo, int64_t rows, int L,
    int n_r, float self_mask, float* __restrict__ dq, float* __restrict__ dv) {
    constexpr int kReduceRows = reduce_rows<NRL>();
    const int64_t row0 = (((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4) * kReduceRows;
    const int part = threadIdx.x & 15;
    if (row0 >= rows) return;  // whole 16-lane groups leave together
    int64_t sbase[kReduceRows][NRL];
    int slot[kReduceRows][NRL];
    float z[kReduceRows];
#pragma unroll
    for (int k = 0; k < kReduceRows; ++k) {
        const int64_t row = min(row0 + k, rows - 1);  // past the end: a valid row, never stored
        const int64_t bh = row / L, i = row % L;
        z[k] = lse_total[row];
#pragma unroll
        for (int rr = 0; rr < NRL; ++rr) {
            sbase[k][rr] = (bh * n_r + (rr < n_r ? rr : 0)) * L;
            slot[k][rr] = undo[sbase[k][rr] + i];
        }
    }
    uint2 xq[kReduceRows][NRL], xv[kReduceRows][NRL];
    uint32_t eq[kReduceRows][NRL], ev[kReduceRows][NRL];
#pragma unroll
    for (int k = 0; k < kReduceRows; ++k)
#pragma unroll
        for (int rr = 0; rr < NRL; ++rr) {
            const int64_t prow = sbase[k][rr] + min(max(slot[k][rr], 0), L - 1);
            xq[k][rr] = *reinterpret_cast<const uint2*>(part_q + prow * kHeadDim + part * 4);
            xv[k][rr] = *reinterpret_cast<const uint2*>(part_v + prow * kHeadDim + part * 4);
            const uint32_t e2 = reinterpret_cast<const uint16_t*>(part_e)[prow];
            eq[k][rr] = e2 & 0xFFu;
            ev[k][rr] = e2 >> 8;
        }
#pragma unroll
    for (int k = 0; k < kReduceRows; ++k) {
        const int64_t row = row0 + k;
        f32x4 aq = {0, 0, 0, 0}, av = {0, 0, 0, 0};
#pragma unroll
        for (int rr = 0; rr < NRL; ++rr) {
            const float wq = rr < n_r ? __uint_as_float((127u + min(eq[k][rr], 126u)) << 23) : 0.f;
            const float wv = rr < n_r ? __uint_as_float((127u + min(ev[k][rr], 126u)) << 23) : 0.f;
            aq[0] = fmaf(wq, f16_bits_to_f32(xq[k][rr].x & 0xFFFFu), aq[0]);
            aq[1] = fmaf(wq, f16_bits_to_f32(xq[k][rr].x >> 16), aq[1]);
            aq[2] = fmaf(wq, f16_bits_to_f32(xq[k][rr].y & 0xFFFFu), aq[2]);
            aq[3] = fmaf(wq, f16_bits_to_f32(xq[k][rr].y >> 16), aq[3]);
            av[0] = fmaf(wv, f16_bits_to_f32(xv[k][rr].x & 0xFFFFu), av[0]);
            av[1] = fmaf(wv, f16_bits_to_f32(xv[k][rr].x >> 16), av[1]);
            av[2] = fmaf(wv, f16_bits_to_f32(xv[k][rr].y & 0xFFFFu), av[2]);
            av[3] = fmaf(wv, f16_bits_to_f32(xv[k][rr].y >> 16), av[3]);
        }
        if (row < rows) {
            if (z[k] < -0.5f * self_mask) {
                const uint2 g = *reinterpret_cast<const uint2*>(dout + row * kHeadDim + part * 4);
                av[0] += bf16_bits_to_f32(g.x & 0xFFFF);
                av[1] += bf16_bits_to_f32(g.x >> 16);
                av[2] += bf16_bits_to_f32(g.y & 0xFFFF);
                av[3] += bf16_bits_to_f32(g.y >> 16);
            }
            *reinterpret_cast<f32x4*>(dq + row * kHeadDim + part * 4) = aq;
            *reinterpret_cast<f32x4*>(dv + row * kHeadDim + part * 4) = av;
        }
    }
}

int rec_words(int n_rounds) {
    const int nw = n_rounds == 1 ? 0 : (n_rounds + 1) / 2;
    const int sw = sig_stride(nw);
    return sw + 3 <= 4 ? 4 : (sw + 3 <= 8 ? 8 : 12);
}

struct BwdWs {
    uint16_t* part_q;  // per round: dq through the query role plus the key role's dk through k = q/|q|
    uint16_t* part_v;
    uint8_t* part_e;   // exponents: [round-rows] pairs, dq's byte then dv's
    uint32_t* rec;
    size_t bytes;
};

BwdWs carve(void* base, int64_t BH, int L, int n_rounds) {
    const size_t rr = (size_t)BH * n_rounds * L;
    char* p = static_cast<char*>(base);
    BwdWs w{};
    size_t off = 0;
    w.part_q = reinterpret_cast<uint16_t*>(p + off);
    off += align256(rr * kHeadDim * 2);
    w.part_v = reinterpret_cast<uint16_t*>(p + off);
    off += align256(rr * kHeadDim * 2);
    w.part_e = reinterpret_cast<uint8_t*>(p + off);
    off += align256(rr * 2);
    w.rec = reinterpret_cast<uint32_t*>(p + off);
    off += align256((size_t)BH * L * 4 * rec_words(n_rounds));
    w.bytes = off;
    return w;
}

template <int NW>
hipError_t launch_nw(bool causal, int64_t BH, int L, int n_rounds, float scale, const uint16_t* q,
                     const uint16_t* v, const uint16_t* out, const uint16_t* dout,
                     const float* lse_total, const int32_t* buckets, const int32_t* perm,
                     const BwdWs& w, hipStream_t stream) {
    const int64_t rows = BH * L;
    bwd_prep_kernel<NW><<<(unsigned)((rows * 8 + 255) / 256), 256, 0, stream>>>(
        q, out, dout, lse_total, buckets, rows, n_rounds, scale * kLog2e, w.rec);
    // Strips of chunks: long enough that the first window and the pair that
    // the previous strip also computes are a small overhead, short enough to
    // give every CU several workgroups in turn (one fits at a time).
    const int64_t n_chunks = (L + kChunk - 1) / kChunk, segs = BH * n_rounds;
    const int cps = (int)std::max<int64_t>(1, std::min<int64_t>(32, n_chunks * segs / 2048));
    const dim3 grid((unsigned)((n_chunks + cps - 1) / cps), (unsigned)segs);
    auto go = [&](auto causal_tag) {
        constexpr bool C = decltype(causal_tag)::value;
        const size_t lds = sizeof(BwdShared<NW>);
        hipFuncSetAttribute(reinterpret_cast<const void*>(&bwd_strip_kernel<NW, C>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        bwd_strip_kernel<NW, C><<<grid, kBwdThreads, lds, stream>>>(
            q, v, dout, w.rec, perm, w.part_q, w.part_v, w.part_e, L, n_rounds, scale, cps);
    };
    if (causal)
        go(std::true_type{});
    else
        go(std::false_type{});
    return hipGetLastError();
}

}  // namespace

size_t bwd_workspace_bytes(int64_t BH, int L, int n_rounds) {
    return carve(nullptr, BH, L, n_rounds).bytes;
}

hipError_t launch_attn_bwd(int64_t BH, int L, int n_rounds, int n_buckets, bool causal,
                           float scale, float self_mask, const void* q_, const void* v_,
                           const void* out_, const void* dout_, const float* lse_total,
                           const int32_t* buckets, const int32_t* perm, const int32_t* undo,
                           const int32_t* bucket_start, float* dq, float* dv, void* workspace,
                           hipStream_t stream) {
    const int64_t rows = BH * L;
    if (rows == 0) return hipSuccess;
    const BwdWs w = carve(workspace, BH, L, n_rounds);
    const uint16_t* q = static_cast<const uint16_t*>(q_);
    const uint16_t* v = static_cast<const uint16_t*>(v_);
    const uint16_t* out = static_cast<const uint16_t*>(out_);
    const uint16_t* dout = static_cast<const uint16_t*>(dout_);
    const int nw = n_rounds == 1 ? 0 : (n_rounds + 1) / 2;
    hipError_t e;
#define LSH_BWD_CASE(W)                                                                             \
    case W:                                                                                         \
        e = launch_nw<W>(causal, BH, L, n_rounds, scale, q, v, out, dout, lse_total, buckets, perm, \
                         w, stream);                                                                \
        break;
    switch (nw) {
        LSH_BWD_CASE(0)
        LSH_BWD_CASE(1)
        LSH_BWD_CASE(2)
        LSH_BWD_CASE(3)
        LSH_BWD_CASE(4)
        LSH_BWD_CASE(5)
        LSH_BWD_CASE(6)
        LSH_BWD_CASE(7)
        LSH_BWD_CASE(8)
        default:
            return hipErrorInvalidValue;
    }
#undef LSH_BWD_CASE
    if (e != hipSuccess) return e;
    auto reduce = [&](auto nrl) {
        constexpr int kRows = reduce_rows<decltype(nrl)::value>();
        const unsigned row_grid = (unsigned)(((rows + kRows - 1) / kRows * 16 + 255) / 256);
        bwd_reduce_kernel<decltype(nrl)::value><<<row_grid, 256, 0, stream>>>(
            dout, lse_total, w.part_q, w.part_v, w.part_e, undo, rows, L, n_rounds, self_mask, dq, dv);
    };
    if (n_rounds <= 1) reduce(std::integral_constant<int, 1>{});
    else if (n_rounds <= 2) reduce(std::integral_constant<int, 2>{});
    else if (n_rounds <= 4) reduce(std::integral_constant<int, 4>{});
    else if (n_rounds <= 8) reduce(std::integral_constant<int, 8>{});
    else reduce(std::integral_constant<int, 16>{});
    return hipGetLastError();
}

}  // namespace lsh

// Chunked LSH attention, forward, all rounds (Reformer Sec. 2 "LSH
// attention" and App. A).
//
// For the query at sorted slot s of round r (chunk c = s/64) the candidate
// keys are the 128 slots of chunks c-1 and c.  Because slots are sorted by
// (bucket, position), the keys sharing the query's bucket form one slot
// interval, and under causal masking "j earlier than i" inside a bucket is
// "slot before s".  So the bucket and causal masks are an interval test
// [lo, hi] per query, with the self key handled apart: with any other target
// its weight exp(-1e5) vanishes in fp32 and fp64 alike, and without one the
// output is v_i and the log-partition is scale*|q_i| - 1e5.
//
// Logits are kept in log2 units: x = (q_i.q_j) * scale*log2(e)/|q_j| - log2 N_ij.
//
// bf16 path (gfx950 matrix cores).  A workgroup of four waves walks a strip
// of chunks of one segment, one chunk per step.  The rows of chunks c-1, c
// and the incoming c+1 sit in an LDS ring of three 64-row slots: q and v rows
// as XOR-swizzled 128-byte rows, the signature words and the key scales.  The
// slot that chunk c+1 lands in held chunk c-2, which step c never reads, so
// the next chunk is gathered (through perm) straight from global memory into
// LDS while step c computes (global_load_lds: no registers, no vector
// instructions), and one barrier per step suffices.
//
// Each wave takes 16 queries of the chunk against their 128-key window as
// eight 16x16 tiles: S^T = K Q^T on mfma_f32_16x16x32_bf16 (lane l holds keys
// 4(l/16)..+3 of query l%16), masks and softmax on those four accumulators,
// then O^T = V^T P^T on mfma_f32_16x16x16_bf16 with the accumulators packed
// as the B operand as they are, and the V^T operand read from the v rows by
// the LDS transpose read.  Tiles with no valid key for the wave's queries are
// skipped.  A query's interval comes from the window's bucket boundaries: a
// 128-bit mask (two ballots) of the slots whose round-r bucket differs from
// the previous slot's; lo is the last boundary at or before the query.
//
// Per score element the VALU work is what bounds this kernel, so it is kept
// to a few instructions: the interval mask is one bit of a per-lane word, the
// count of rounds in which i and j differ is one popcount over the guard bits
// of the packed bucket signatures (all words merged, see sig_add), and the
// mask and log2 N_ij come together from one 33-entry LDS table indexed by that
// popcount (index 32 = masked).  The softmax needs no running maximum when
// the wave's logit bound B_i = scale*log2(e)*|q_i| is moderate: every logit
// lies in [-B_i - log2 n_r, B_i], so for B_i <= 60 exp2(x) itself neither
// overflows nor underflows; waves with a larger bound fall back to the online
// maximum.  The row sum l_i adds the fp32 weights, so the log-partition is
// exact to fp32.  P V takes the weights rounded to bf16, and the output is
// normalised by the sum of those same rounded weights (one more matrix
// product with an all-ones operand), so the weights applied to the values
// sum to one: a query with a single target returns that value unchanged and
// the weight rounding only moves the output by a fraction of the spread of
// its values.
//
// Each round's output row is stored as fp16 (11 significant bits, the same
// bytes as bf16) scaled by 2^-e, with e = 0 unless the row's largest
// magnitude reaches 2^15 (then e brings it below 2^15); e goes to a byte per
// row.  With 11 bits the only rounding of bf16 size left on the way to the
// combined output is the output's own.
#include "attn_common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr float kFastBound = 60.f;  // largest B_i handled without a running maximum
constexpr int kSwz = 1;             // LDS row layout (attn_common.h): 16-row operand reads
constexpr int kMaskedIndex = 32;    // table index of a masked-out key


template <bool B>
struct BoolTag {
    static constexpr bool value = B;
};

// Shape of the bf16 kernel for chunks of M sorted slots and a look-ahead of
// AFTER chunks: 16 queries per wave; the window is chunks c-1 .. c+AFTER;
// the ring holds the window and the chunk being gathered.
template <int M, int AFTER>
struct FwdGeom {
    static constexpr int kWaves = M / 16;
    static constexpr int kThreads = 64 * kWaves;
    static constexpr int kWinChunks = 2 + AFTER;
    static constexpr int kWinKeys = kWinChunks * M;
    static constexpr int kGroups = kWinKeys / 64;  // 64-slot groups of the window
    static constexpr int kTiles = kWinKeys / 16;
    static constexpr int kTilesPerChunk = M / 16;
    static constexpr int kSlots = kWinChunks + 1;
    static constexpr int kRows = kSlots * M;
    static constexpr int kPosRegs = M / 64;        // slot positions a lane holds per chunk
    // workgroups per CU the LDS allows (and that the kernel is built for)
    static constexpr int kOcc = M == 64 ? (AFTER == 0 ? 3 : 2) : 1;
};

template <int NW>
struct FwdSig {
    static constexpr int stride = NW <= 1 ? 1 : (NW <= 2 ? 2 : (NW <= 4 ? 4 : 8));  // words per token
    // Per-token record gathered with every staged row: the signature words,
    // zeros, and the key scale in the last word; 16, 32 or 64 bytes.
    static constexpr int rec_words = stride + 1 <= 4 ? 4 : (stride + 1 <= 8 ? 8 : 16);
};

template <int NW, int M, int AFTER>
struct FwdShared {
    static constexpr int kRows = FwdGeom<M, AFTER>::kRows;
    char Qs[kRows * 128];  // q rows, 16-byte pieces at swizzled slots (see swz)
    char Vs[kRows * 128];  // v rows, same layout
    uint32_t sig[kRows][FwdSig<NW>::stride];  // bucket signature words
    float cf[kRows];                          // scale*log2(e)/|q_row| (0 for a zero row)
    float tab[kMaskedIndex + 1];              // -log2 N by mismatch count; -inf = masked
};

template <int NW, class SH>
__device__ __forceinline__ void read_sig(const SH& S, int row, uint32_t (&out)[NW > 0 ? NW : 1]) {
    if constexpr (NW <= 1) {
        out[0] = S.sig[row][0];
    } else if constexpr (NW == 2) {
        const uint2 w = *reinterpret_cast<const uint2*>(&S.sig[row][0]);
        out[0] = w.x;
        out[1] = w.y;
    } else {
#pragma unroll
        for (int w4 = 0; w4 < (NW + 3) / 4; ++w4) {
            const u32x4 w = *reinterpret_cast<const u32x4*>(&S.sig[row][4 * w4]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (4 * w4 + e < NW) out[4 * w4 + e] = w[e];
        }
    }
}

template <int NW, bool CAUSAL, int M, int AFTER>
__global__ __launch_bounds__((FwdGeom<M, AFTER>::kThreads), (FwdGeom<M, AFTER>::kOcc)) void attn_fwd_bf16_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v, const uint32_t* __restrict__ rec,
    const int32_t* __restrict__ perm, uint16_t* __restrict__ o_rounds,
    uint8_t* __restrict__ o_exp, float* __restrict__ lse_rounds, int L, int n_r, float scale,
    float self_mask, int chunks_per_strip) {
    using G = FwdGeom<M, AFTER>;
    using Shared = FwdShared<NW, M, AFTER>;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    Shared& S = *reinterpret_cast<Shared*>(smem);
    constexpr int SW = FwdSig<NW>::stride, RW = FwdSig<NW>::rec_words;
    auto ring_row = [](int chunk, int i) { return ((chunk % G::kSlots + G::kSlots) % G::kSlots) * M + i; };

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 15, g = lane >> 4;  // query (and key row) of the lane, key group
    const int64_t seg = blockIdx.y;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int n_chunks = (L + M - 1) / M;  // the last may be partial
    const int c0 = blockIdx.x * chunks_per_strip;
    const int c1 = min(n_chunks, c0 + chunks_per_strip);
    const float scale_log2e = scale * kLog2e;
    const int32_t* pseg = perm + seg * L;
    const int64_t rowbase = bh * L;
    const int rw = r >> 1, rsh = (r >> 1) + 11 * (r & 1);  // field r of a signature
    if (tid <= kMaskedIndex) S.tab[tid] = tid < n_r ? -__log2f((float)(n_r - tid)) : -__builtin_inff();

    // Positions of slots 64p + lane of chunk cc, as stored (clamped where
    // they are used); for a slot outside the sequence (before chunk 0, or
    // past L) any valid row: such slots are never a valid key (see lo and hi
    // below) and their queries store nothing.
    struct Pos {
        int p[G::kPosRegs];
    };
    auto chunk_pos = [&](int cc) -> Pos {
        Pos x;
#pragma unroll
        for (int k = 0; k < G::kPosRegs; ++k) {
            const int slot = cc * M + 64 * k + lane;
            x.p[k] = cc >= 0 && slot < L ? pseg[slot] : 0;
        }
        return x;
    };
    // Gather chunk cc into its ring slot: wave w copies q and v rows
    // 16w .. 16w+15 (each lane the piece that belongs at its LDS slot), and
    // the signature words and key scales are split over the waves.
    auto stage = [&](int cc, Pos pos_raw) {
        int pos_lane[G::kPosRegs];
#pragma unroll
        for (int k = 0; k < G::kPosRegs; ++k) pos_lane[k] = min(max(pos_raw.p[k], 0), L - 1);
        // position of chunk row `row` (uniform choice of register per wave)
        auto pos_of = [&](int row) {
            int p = __shfl(pos_lane[0], row & 63);
#pragma unroll
            for (int k = 1; k < G::kPosRegs; ++k)
                if ((row >> 6) == k) p = __shfl(pos_lane[k], row & 63);
            return p;
        };
        const int slot0 = ring_row(cc, 0);
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int row = 16 * wave + 8 * k + (lane >> 3);
            const int p = pos_of(row);
            const int64_t off = (rowbase + p) * kHeadDim + swz<kSwz>(row, lane & 7) * 8;
            copy16_to_lds(q + off, S.Qs + (slot0 + 16 * wave + 8 * k) * 128);
            copy16_to_lds(v + off, S.Vs + (slot0 + 16 * wave + 8 * k) * 128);
        }
        if constexpr (SW >= 4) {
            constexpr int U = SW / 4;  // 16-byte units per row
#pragma unroll
            for (int k = 0; k < M * U / 64; ++k)
                if (wave == k) {
                    const int u = 64 * k + lane, row = u / U;
                    const int p = pos_of(row);
                    copy16_to_lds(rec + (rowbase + p) * RW + 4 * (u % U), &S.sig[slot0][0] + 256 * k);
                }
        } else {
#pragma unroll
            for (int k = 0; k < M * SW / 64; ++k)
                if (wave == k) {
                    const int u = 64 * k + lane, row = u / SW;
                    const int p = pos_of(row);
                    copy4_to_lds(rec + (rowbase + p) * RW + (u % SW), &S.sig[slot0][0] + 64 * k);
                }
        }
#pragma unroll
        for (int k = 0; k < G::kPosRegs; ++k)
            if (wave == G::kWaves - 1 - k)
                copy4_to_lds(rec + (rowbase + pos_lane[k]) * RW + (RW - 1), &S.cf[slot0 + 64 * k]);
    };

#pragma unroll
    for (int k = -1; k <= AFTER; ++k) stage(c0 + k, chunk_pos(c0 + k));
    Pos pf_pos = chunk_pos(c0 + AFTER + 1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // A chunk's output rows are stored at the start of the next step: the
    // wait before each barrier (for the staging copies, counted together with
    // stores) then finds them long completed.
    uint2 out_pend[4] = {};
    float lse_pend = 0.f;
    uint32_t exp_pend = 0;
    int64_t row_pend = -1;
    auto flush = [&]() {
        if (row_pend >= 0) {
            uint16_t* orow = o_rounds + row_pend * kHeadDim + 4 * g;
#pragma unroll
            for (int b = 0; b < 4; ++b) *reinterpret_cast<uint2*>(orow + 16 * b) = out_pend[b];
            if (g == 0) {
                lse_rounds[row_pend] = lse_pend;
                o_exp[row_pend] = (uint8_t)exp_pend;
            }
        }
    };

    for (int c = c0; c < c1; ++c) {
        if (c + 1 < c1) stage(c + AFTER + 1, pf_pos);
        const Pos pf_next = chunk_pos(c + AFTER + 2);
        flush();

        // ---- this wave's 16 queries of chunk c ----
        const int u = 16 * wave + n;  // query row inside the chunk
        const int s_q = c * M + u;
        const int rq = ring_row(c, u);
        uint32_t qsig[NW > 0 ? NW : 1];
        read_sig<NW>(S, rq, qsig);
        const bf16x8 qb0 = as_bf16x8(lds_piece<kSwz>(S.Qs, rq, g));
        const bf16x8 qb1 = as_bf16x8(lds_piece<kSwz>(S.Qs, rq, 4 + g));
        const float cfq = S.cf[rq];
        // B_i (to within an ulp: it picks the fast path, with a wide margin,
        // and gives a lone query's log-partition)
        const float bound = cfq > 0.f ? scale_log2e * scale_log2e * __builtin_amdgcn_rcpf(cfq) : 0.f;
        const bool fast = __ballot(!(bound <= kFastBound)) == 0;

        // Bucket boundaries of the window (window slot w = slot (c-1)M + w):
        // bit l of bnd[gi] is set when window slot 64 gi + l starts a new
        // round-r bucket (window slot 0 always does).
        uint64_t bnd[G::kGroups];
        {
            uint32_t last = 0;
#pragma unroll
            for (int gi = 0; gi < G::kGroups; ++gi) {
                const int wc = (64 * gi) / M, wrow = (64 * gi) % M + lane;
                const uint32_t id = (S.sig[ring_row(c - 1 + wc, wrow)][rw] >> rsh) & 0x3FFu;
                const uint32_t up = __shfl_up(id, 1);
                const uint32_t prev = lane == 0 ? last : up;
                bnd[gi] = __ballot((gi == 0 && lane == 0) || id != prev);
                last = __shfl(id, 63);
            }
        }
        // the query's key interval [lo_w, hi_w] in window slots: the last
        // boundary at or before its own slot M + u, and (without causal
        // masking) the slot before the next boundary; its group gq is
        // uniform over the wave
        const int qs = M + u, gq = qs >> 6, bq = qs & 63;
        int lo_w = 0;
#pragma unroll
        for (int gi = 0; gi < G::kGroups; ++gi) {
            const uint64_t mm = gi < gq ? bnd[gi] : (gi == gq ? bnd[gi] & (~0ull >> (63 - bq)) : 0ull);
            if (mm) lo_w = 64 * gi + 63 - __clzll(mm);
        }
        int hi_w;
        if constexpr (CAUSAL) {
            hi_w = qs - 1;
        } else {
            hi_w = G::kWinKeys - 1;
#pragma unroll
            for (int gi = G::kGroups - 1; gi >= 0; --gi) {
                const uint64_t mm = gi > gq ? bnd[gi]
                                            : (gi == gq && bq < 63 ? bnd[gi] & (~0ull << (bq + 1)) : 0ull);
                if (mm) hi_w = 64 * gi + __ffsll((long long)mm) - 2;
            }
        }
        // no slot before 0 and no key past the sequence
        lo_w = max(lo_w, (1 - c) * M);
        hi_w = min(hi_w, L - 1 - (c - 1) * M);
        // valid keys of this lane's query as a window mask (vm[gi]: window
        // slots 64 gi .. 64 gi + 63), then per lane group the complement
        // shifted so that bit 16(kt%2) + j of nv[kt/2] is set when tile key
        // 4g + j of tile kt is masked out
        uint64_t vm[G::kGroups];
#pragma unroll
        for (int gi = 0; gi < G::kGroups; ++gi) {
            const int lg = lo_w - 64 * gi, hg = hi_w - 64 * gi;
            vm[gi] = (hg < 0 || lg > 63) ? 0ull
                                         : ((lg <= 0 ? ~0ull : ~0ull << lg) & (hg >= 63 ? ~0ull : ~0ull >> (63 - hg)));
        }
        if constexpr (!CAUSAL) {  // the query itself
#pragma unroll
            for (int gi = 0; gi < G::kGroups; ++gi)
                if (gi == gq) vm[gi] &= ~(1ull << bq);
        }
        uint32_t nv[2 * G::kGroups];
        bool act[G::kTiles];
#pragma unroll
        for (int gi = 0; gi < G::kGroups; ++gi) {
            const uint64_t sh = ~vm[gi] >> (4 * g);
            nv[2 * gi] = (uint32_t)sh;
            nv[2 * gi + 1] = (uint32_t)(sh >> 32);
#pragma unroll
            for (int k = 0; k < 4; ++k) act[4 * gi + k] = __ballot(((vm[gi] >> (16 * k)) & 0xFFFFu) != 0) != 0;
        }

        // Per-lane LDS offsets of the window chunks' first rows (tile kt adds
        // a constant number of rows): K operand pieces g and 4+g, the V^T
        // operands of the four 16-dim blocks, the signature row.
        uint32_t kofs[G::kWinChunks][2], vofs[G::kWinChunks][4];
        int srow[G::kWinChunks];
#pragma unroll
        for (int ch = 0; ch < G::kWinChunks; ++ch) {
            const int base = ring_row(c - 1 + ch, 0);
            kofs[ch][0] = row_piece_offset<kSwz>(base + n, g);
            kofs[ch][1] = row_piece_offset<kSwz>(base + n, 4 + g);
#pragma unroll
            for (int b = 0; b < 4; ++b) vofs[ch][b] = vt_offset<kSwz>(base, 16 * b, lane);
            srow[ch] = base + 4 * g;
        }

        auto attend = [&](auto fast_tag) {
            constexpr bool FAST = decltype(fast_tag)::value;
            float m = -__builtin_inff(), lsum = 0.f;
            // oacc[0..3]: O^T by 16-dim blocks; oacc[4]: the sum of the bf16
            // weights (every register of a lane holds its query's sum)
            f32x4 oacc[5] = {f32x4{}, f32x4{}, f32x4{}, f32x4{}, f32x4{}};
#pragma unroll
            for (int kt = 0; kt < G::kTiles; ++kt) {
                if (!act[kt]) continue;
                // window chunk of the tile and its first row in that chunk
                const int ch = kt / G::kTilesPerChunk, roff = 16 * (kt % G::kTilesPerChunk);
                f32x4 acc = mfma16x16x32(as_bf16x8(*reinterpret_cast<const u32x4*>(S.Qs + kofs[ch][0] + roff * 128)),
                                         qb0, f32x4{});
                acc = mfma16x16x32(as_bf16x8(*reinterpret_cast<const u32x4*>(S.Qs + kofs[ch][1] + roff * 128)), qb1,
                                   acc);
                const int kbase = srow[ch] + roff;
                const f32x4 cfk = *reinterpret_cast<const f32x4*>(&S.cf[kbase]);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int bit = 16 * (kt & 1) + j;  // of nv[kt / 2]; -1 when masked
                    uint32_t t = (uint32_t)((int32_t)(nv[kt >> 1] << (31 - bit)) >> 31);
                    if constexpr (NW > 0) {
                        uint32_t ksig[NW];
                        read_sig<NW>(S, kbase + j, ksig);
#pragma unroll
                        for (int w = 0; w < NW; ++w) t = and_or((qsig[w] ^ ksig[w]) + sig_add(w), sig_guard(w), t);
                    }
                    acc[j] = fmaf(acc[j], cfk[j], S.tab[__popc(t)]);
                }
                float off = 0.f;
                if constexpr (!FAST) {  // online maximum over the four lane groups of a query
                    float mt = fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3]));
                    mt = max_xor32(max_xor16(mt));
                    const float m_new = fmaxf(m, mt);
                    off = m_new > -__builtin_inff() ? m_new : 0.f;
                    const float corr = __builtin_amdgcn_exp2f(m - off);
                    lsum *= corr;
#pragma unroll
                    for (int b = 0; b < 5; ++b) oacc[b] *= corr;
                    m = m_new;
                }
                uint32_t pw[2];
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) {
                    const float pa = __builtin_amdgcn_exp2f(FAST ? acc[2 * h2] : acc[2 * h2] - off);
                    const float pb = __builtin_amdgcn_exp2f(FAST ? acc[2 * h2 + 1] : acc[2 * h2 + 1] - off);
                    pw[h2] = pack_bf16x2(pa, pb);
                    // the row sum takes the fp32 weights, so z_r is exact to fp32 (the
                    // backward renormalises with it); P V takes them rounded to bf16
                    lsum += pa;
                    lsum += pb;
                }
                const bf16x4 pk = __builtin_bit_cast(bf16x4, make_uint2(pw[0], pw[1]));
#pragma unroll
                for (int b = 0; b < 4; ++b) oacc[b] = mfma16x16x16(vt_read(S.Vs + vofs[ch][b] + roff * 128), pk, oacc[b]);
                oacc[4] = mfma16x16x16(kOnes4, pk, oacc[4]);
            }
            lsum = sum_xor32(sum_xor16(lsum));
            const bool alone = !(lsum > 0.f);  // only itself left as a target
            if (__ballot(alone) != 0) {
                // The output of a lone query is v_i: one more P V step on the
                // diagonal tile with P = 1 at (i, i) for those queries and 0
                // elsewhere adds exactly v_i to their (zero) accumulators.
                // Query n's own key is key n of that tile (rows 16w .. 16w+15
                // of chunk c), held by lane group n / 4 as its element n % 4.
                const bool mine = alone && g == (n >> 2);
                const uint32_t one = (n & 1) ? 0x3F800000u : 0x3F80u;  // bf16 1.0 in its half
                const uint2 w2 = make_uint2(mine && (n & 2) == 0 ? one : 0u, mine && (n & 2) != 0 ? one : 0u);
                const bf16x4 pk = __builtin_bit_cast(bf16x4, w2);
#pragma unroll
                for (int b = 0; b < 4; ++b) oacc[b] = mfma16x16x16(vt_read(S.Vs + vofs[1][b] + 16 * wave * 128), pk, oacc[b]);
            }
            const float mref = FAST ? 0.f : m;
            // normalised by the sum of the bf16 weights P V used (1/l to
            // within 1 ulp); a lone query divides its exact v_i by 1.  The
            // largest magnitude is taken before normalising (one multiply
            // less per element): scaling by inv > 0 keeps the maximum's place.
            const float inv = alone ? 1.f : __builtin_amdgcn_rcpf(oacc[4][0]);
            float amax = 0.f;
#pragma unroll
            for (int b = 0; b < 4; ++b)
#pragma unroll
                for (int e = 0; e < 4; ++e) amax = fmaxf(amax, fabsf(oacc[b][e]));
            amax = max_xor32(max_xor16(amax));
            amax *= inv;
            // 2^(E-127) <= amax < 2^(E-126): e = max(0, E - 141) puts the
            // scaled row below 2^15, inside fp16's range
            const int ex = max(0, (int)((__float_as_uint(amax) >> 23) & 0xFFu) - 141);
            const float fac = inv * __uint_as_float((uint32_t)(127 - ex) << 23);
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                out_pend[b].x = pack_f16x2(oacc[b][0] * fac, oacc[b][1] * fac);
                out_pend[b].y = pack_f16x2(oacc[b][2] * fac, oacc[b][3] * fac);
            }
            exp_pend = (uint32_t)ex;
            // z = scale*|q_i| - self_mask when the token is its own only target
            lse_pend = alone ? bound * kLn2 - self_mask : (mref + __log2f(lsum)) * kLn2;
            row_pend = s_q < L ? seg * L + s_q : -1;
        };
        if (fast)
            attend(BoolTag<true>{});
        else
            attend(BoolTag<false>{});

        pf_pos = pf_next;
        __builtin_amdgcn_s_waitcnt(0);  // this wave's copies of the next chunk have landed
        __syncthreads();                // ... and every wave is done with chunk c-1
    }
    flush();
}

// fp32 path: one workgroup per chunk of M sorted slots (M = 64, or 128, the
// chunk length of the paper's usual configuration), one lane per query in
// each of KS waves, exact fp32 arithmetic on the VALU with an online softmax
// over the query's keys.  Wave s takes every KS-th key of the query's range;
// the KS partial softmaxes (max, sum, weighted row) are merged at the end.  The window is chunks c-1 .. c+after; it is walked one chunk at a
// time (the query's own chunk first), each staged in LDS.  Two variants the
// paper does not spell out: a look-ahead of `after` chunks, and attending
// across buckets (every key of the window is a target, and N_ij counts the
// rounds in which j falls in i's window, from undo).
template <int M, int KS>
__global__ __launch_bounds__(M * KS) void attn_fwd_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ v, const int32_t* __restrict__ buckets,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ undo,
    const int32_t* __restrict__ bstart, float* __restrict__ o_rounds,
    float* __restrict__ lse_rounds, int L, int n_r, int n_b, int causal, int after, int across,
    float scale, float self_mask) {
    // rows padded to 68 floats: 16-byte aligned for the broadcast reads of
    // the key loop
    constexpr int kRow = kHeadDim + 4;
    __shared__ __attribute__((aligned(16))) float Ks[M][kRow];
    __shared__ __attribute__((aligned(16))) float Vs2[M][kRow];
    __shared__ float inv[M];
    __shared__ int spos[M];
    // waves 1 .. KS-1: their partial (max, sum, row) per query
    __shared__ float part[KS > 1 ? KS - 1 : 1][KS > 1 ? M : 1][kHeadDim + 2];
    static_assert(M % kHeadDim == 0 && M * KS <= 256, "whole waves of queries per key split");

    constexpr int NT = M * KS;
    const int tid = threadIdx.x;
    const int t = tid % M;       // the query's slot in the chunk
    const int ks = tid / M;      // the key split
    const int64_t seg = blockIdx.y;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int c = blockIdx.x;
    const int s_q = c * M + t;
    const bool has_q = s_q < L;  // a slot past L (a partial last chunk) has no query
    const int32_t* pseg = perm + seg * L;
    const int i_q = pseg[min(s_q, L - 1)];
    const int32_t* bi = buckets + (bh * L + i_q) * n_r;
    const int beta = min(max(bi[r], 0), n_b - 1);
    const int32_t* bs = bstart + seg * (n_b + 1);
    const int w_lo = max(0, (c - 1) * M), w_hi = min(L, (c + 1 + after) * M) - 1;  // window slots
    // the query's keys: its bucket's slots inside the window, or the whole
    // window across buckets.  No key later than the query under causal
    // masking: inside one bucket slot order is position order, so that is
    // the slot bound s_q - 1; across buckets it is a test of positions.
    const int lo = across ? w_lo : max(bs[beta], w_lo);
    const int hi = across ? w_hi : (causal ? s_q - 1 : min(bs[beta + 1] - 1, w_hi));
    const bool pos_causal = across && causal;
    // across buckets: the query's chunk in every round
    int ci[16];
    if (across)
        for (int rr = 0; rr < n_r; ++rr) ci[rr] = undo[(bh * n_r + rr) * L + i_q] / M;

    float qi[kHeadDim];
    float m = -__builtin_inff(), l = 0.f;
    float o[kHeadDim];
    for (int u = 0; u < kHeadDim; ++u) o[u] = 0.f;
    const int n_win = 2 + after;
    for (int piece = 0; piece < n_win; ++piece) {
        // chunk c first (it holds the queries), then c-1, c+1, ...
        const int k = piece == 0 ? c : (piece == 1 ? c - 1 : c + piece - 1);
        const int slot0 = k * M;
        __syncthreads();  // the previous piece is no longer read
        // positions first, then thread tid copies dim tid % 64 of row
        // tid / 64 of each group of NT / 64 rows, from clamped addresses
        if (ks == 0) {
            const int slot = slot0 + t;
            const int pos = min(max(pseg[min(max(slot, 0), L - 1)], 0), L - 1);
            spos[t] = slot >= 0 && slot < L ? pos : -1;
        }
        __syncthreads();
        constexpr int kRowsPerPass = NT / kHeadDim;
        const int dcol = tid % kHeadDim, rsub = tid / kHeadDim;
#pragma unroll 8
        for (int rho0 = 0; rho0 < M; rho0 += kRowsPerPass) {
            const int rho = rho0 + rsub;
            const int pos = spos[rho];
            const int64_t src = (bh * L + max(pos, 0)) * kHeadDim + dcol;
            const float kq = q[src], kv = v[src];
            Ks[rho][dcol] = pos >= 0 ? kq : 0.f;
            Vs2[rho][dcol] = pos >= 0 ? kv : 0.f;
        }
        __syncthreads();
        if (ks == 0) {
            float ss = 0.f;
            for (int u = 0; u < kHeadDim; ++u) ss = fmaf(Ks[t][u], Ks[t][u], ss);
            inv[t] = ss > 0.f ? 1.f / sqrtf(ss) : 0.f;
        }
        if (piece == 0)
            for (int u = 0; u < kHeadDim; ++u) qi[u] = Ks[t][u];
        __syncthreads();
        if (!has_q) continue;
        const int t_lo = max(lo, slot0), t_hi = min(hi, slot0 + M - 1);
        for (int tk = t_lo + ks; tk <= t_hi; tk += KS) {
            if (tk == s_q) continue;
            const int rho = tk - slot0;
            if (pos_causal && spos[rho] > i_q) continue;
            // four independent chains: one wave per chunk leaves nothing
            // else to hide a 64-long chain of dependent FMAs
            const f32x4* kr = reinterpret_cast<const f32x4*>(&Ks[rho][0]);
            float d[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int u4 = 0; u4 < kHeadDim / 4; ++u4) {
                const f32x4 kk = kr[u4];
#pragma unroll
                for (int e = 0; e < 4; ++e) d[e] = fmaf(qi[4 * u4 + e], kk[e], d[e]);
            }
            const float dot = (d[0] + d[1]) + (d[2] + d[3]);
            float a = scale * (dot * inv[rho]);
            if (n_r > 1) {
                int nn = 0;
                if (across) {
                    for (int rr = 0; rr < n_r; ++rr) {
                        const int cj = undo[(bh * n_r + rr) * L + spos[rho]] / M;
                        nn += cj >= ci[rr] - 1 && cj <= ci[rr] + after;
                    }
                } else {
                    const int32_t* bj = buckets + (bh * L + spos[rho]) * n_r;
                    for (int rr = 0; rr < n_r; ++rr) nn += bi[rr] == bj[rr];
                }
                a -= logf((float)nn);
            }
            const float mn = fmaxf(m, a);
            const float corr = expf(m - mn);
            const float p = expf(a - mn);
            l = l * corr + p;
            const f32x4* vr = reinterpret_cast<const f32x4*>(&Vs2[rho][0]);
#pragma unroll
            for (int u4 = 0; u4 < kHeadDim / 4; ++u4) {
                const f32x4 vv = vr[u4];
#pragma unroll
                for (int e = 0; e < 4; ++e) o[4 * u4 + e] = fmaf(o[4 * u4 + e], corr, p * vv[e]);
            }
            m = mn;
        }
    }
    if constexpr (KS > 1) {
        // merge the splits' partial softmaxes into wave 0 (a split that saw
        // no key has m = -inf and l = 0, and weighs nothing)
        if (ks > 0) {
            float* pp = part[ks - 1][t];
            pp[0] = m;
            pp[1] = l;
            for (int u = 0; u < kHeadDim; ++u) pp[2 + u] = o[u];
        }
        __syncthreads();
        if (ks > 0) return;
        float mm = m;
        for (int k = 0; k < KS - 1; ++k) mm = fmaxf(mm, part[k][t][0]);
        if (mm > -__builtin_inff()) {
            const float c0 = expf(m - mm);
            l *= c0;
            for (int u = 0; u < kHeadDim; ++u) o[u] *= c0;
            for (int k = 0; k < KS - 1; ++k) {
                const float* pp = part[k][t];
                const float ck = expf(pp[0] - mm);
                l = fmaf(pp[1], ck, l);
                for (int u = 0; u < kHeadDim; ++u) o[u] = fmaf(pp[2 + u], ck, o[u]);
            }
            m = mm;
        }
    }
    if (!has_q) return;
    float* orow = o_rounds + (seg * L + s_q) * kHeadDim;
    if (l > 0.f) {
        const float il = 1.f / l;
#pragma unroll
        for (int u4 = 0; u4 < kHeadDim / 4; ++u4)
            reinterpret_cast<f32x4*>(orow)[u4] =
                f32x4{o[4 * u4] * il, o[4 * u4 + 1] * il, o[4 * u4 + 2] * il, o[4 * u4 + 3] * il};
        lse_rounds[seg * L + s_q] = m + logf(l);
    } else {
        // only itself left as a target: v_i, log-partition scale*|q_i| - self_mask
        float ss = 0.f;
        for (int u = 0; u < kHeadDim; ++u) ss = fmaf(qi[u], qi[u], ss);
        const int64_t src = (bh * L + i_q) * kHeadDim;
        for (int u = 0; u < kHeadDim; ++u) orow[u] = v[src + u];
        lse_rounds[seg * L + s_q] = scale * sqrtf(ss) - self_mask;
    }
}

// Per-token record that the chunk kernel gathers with every staged row, made
// once instead of once per round: the bucket signature words (see sig_add)
// and the key scale scale*log2(e)/|q| (0 for a zero row) in the last word.
// Eight lanes per token, one 16-byte piece of the q row each; lane p writes
// record words p (and p + 8).
template <int NW>
__global__ __launch_bounds__(256) void attn_prep_kernel(const uint16_t* __restrict__ q,
                                                        const int32_t* __restrict__ buckets,
                                                        int64_t rows, int n_r, float scale_log2e,
                                                        uint32_t* __restrict__ rec) {
    constexpr int SW = FwdSig<NW>::stride, RW = FwdSig<NW>::rec_words;
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 3;
    const int part = threadIdx.x & 7;
    if (row >= rows) return;  // whole groups of eight lanes leave together
    const u32x4 x = *reinterpret_cast<const u32x4*>(q + row * kHeadDim + part * 8);
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(x[e] << 16), hi = __uint_as_float(x[e] & 0xFFFF0000u);
        ss = fmaf(lo, lo, fmaf(hi, hi, ss));
    }
    ss += __shfl_xor(ss, 1);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 4);
    const int32_t* brow = buckets + row * n_r;
#pragma unroll
    for (int w = part; w < RW; w += 8) {
        uint32_t word = 0;
        if (w < SW) {
            const uint32_t id0 = 2 * w < n_r ? (uint32_t)brow[2 * w] & 0x3FFu : 0u;
            const uint32_t id1 = 2 * w + 1 < n_r ? (uint32_t)brow[2 * w + 1] & 0x3FFu : 0u;
            word = (id0 << w) | (id1 << (w + 11));
        } else if (w == RW - 1) {
            const float nn = sqrtf(ss);
            word = __float_as_uint(nn > 0.f ? scale_log2e / nn : 0.f);
        }
        rec[row * RW + w] = word;
    }
}


template <int NW, int M, int AFTER>
void launch_kernel(bool causal, dim3 grid, const uint16_t* q, const uint16_t* v, const uint32_t* rec,
                   const int32_t* perm, uint16_t* o, uint8_t* o_exp, float* lse, int L, int n_r,
                   float scale, float self_mask, int cps, hipStream_t stream) {
    constexpr int kThreads = FwdGeom<M, AFTER>::kThreads;
    const size_t lds = sizeof(FwdShared<NW, M, AFTER>);
    auto go = [&](auto kernel) {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
        kernel<<<grid, kThreads, lds, stream>>>(q, v, rec, perm, o, o_exp, lse, L, n_r, scale, self_mask, cps);
    };
    if (causal)
        go(&attn_fwd_bf16_kernel<NW, true, M, AFTER>);
    else
        go(&attn_fwd_bf16_kernel<NW, false, M, AFTER>);
}

template <int NW>
hipError_t launch_bf16(bool causal, int M, int after, const uint16_t* q, const uint16_t* v,
                       const int32_t* buckets, const int32_t* perm, uint16_t* o, uint8_t* o_exp,
                       float* lse, int64_t BH, int L, int n_r, float scale, float self_mask,
                       void* workspace, hipStream_t stream) {
    const int64_t rows = BH * L;
    uint32_t* rec = static_cast<uint32_t*>(workspace);
    attn_prep_kernel<NW><<<(unsigned)((rows * 8 + 255) / 256), 256, 0, stream>>>(
        q, buckets, rows, n_r, scale * kLog2e, rec);
    // Strips of chunks: long enough that staging the strip's first window is
    // a small overhead, short enough to give the chip several rounds of
    // workgroups (kOcc fit on a CU at once).
    const int64_t n_chunks = (L + M - 1) / M, segs = BH * n_r;
    const int occ = M == 64 ? (after == 0 ? 3 : 2) : 1;
    const int cps = (int)std::max<int64_t>(1, std::min<int64_t>(16, n_chunks * segs / (1024 * occ)));
    const dim3 grid((unsigned)((n_chunks + cps - 1) / cps), (unsigned)segs);
    if (M == 64 && after == 0)
        launch_kernel<NW, 64, 0>(causal, grid, q, v, rec, perm, o, o_exp, lse, L, n_r, scale, self_mask, cps, stream);
    else if (M == 64)
        launch_kernel<NW, 64, 1>(causal, grid, q, v, rec, perm, o, o_exp, lse, L, n_r, scale, self_mask, cps, stream);
    else if (after == 0)
        launch_kernel<NW, 128, 0>(causal, grid, q, v, rec, perm, o, o_exp, lse, L, n_r, scale, self_mask, cps, stream);
    else
        launch_kernel<NW, 128, 1>(causal, grid, q, v, rec, perm, o, o_exp, lse, L, n_r, scale, self_mask, cps, stream);
    return hipGetLastError();
}

int sig_words(int n_rounds) {
    const int nw = n_rounds == 1 ? 0 : (n_rounds + 1) / 2;
    return nw <= 1 ? 1 : (nw <= 2 ? 2 : (nw <= 4 ? 4 : 8));
}

}  // namespace

size_t attn_fwd_workspace_bytes(int64_t BH, int L, int n_rounds, bool f32) {
    if (f32) return 0;
    const size_t rows = (size_t)BH * L;
    const int sw = sig_words(n_rounds);
    const size_t rec_words = sw + 1 <= 4 ? 4 : (sw + 1 <= 8 ? 8 : 16);
    return align256(rows * 4 * rec_words);
}

hipError_t launch_attn_fwd(int64_t BH, int L, int n_rounds, int n_buckets, int chunk, int after,
                           bool across, bool causal, float scale, float self_mask, bool f32,
                           const void* q, const void* v, const int32_t* buckets,
                           const int32_t* perm, const int32_t* undo,
                           const int32_t* bucket_start, void* o_rounds, uint8_t* o_exp,
                           float* lse_rounds, void* workspace, hipStream_t stream) {
    if (BH == 0 || L == 0) return hipSuccess;
    const unsigned segs = (unsigned)(BH * n_rounds);
    if (f32) {
        const dim3 grid((unsigned)((L + chunk - 1) / chunk), segs);
        if (chunk == 128)
            attn_fwd_f32_kernel<128, 2><<<grid, 256, 0, stream>>>(
                static_cast<const float*>(q), static_cast<const float*>(v), buckets, perm, undo,
                bucket_start, static_cast<float*>(o_rounds), lse_rounds, L, n_rounds, n_buckets,
                causal ? 1 : 0, after, across ? 1 : 0, scale, self_mask);
        else
            attn_fwd_f32_kernel<64, 4><<<grid, 256, 0, stream>>>(
                static_cast<const float*>(q), static_cast<const float*>(v), buckets, perm, undo,
                bucket_start, static_cast<float*>(o_rounds), lse_rounds, L, n_rounds, n_buckets,
                causal ? 1 : 0, after, across ? 1 : 0, scale, self_mask);
        return hipGetLastError();
    }
    const uint16_t* qb = static_cast<const uint16_t*>(q);
    const uint16_t* vb = static_cast<const uint16_t*>(v);
    uint16_t* ob = static_cast<uint16_t*>(o_rounds);
    const int nw = n_rounds == 1 ? 0 : (n_rounds + 1) / 2;
#define LSH_FWD_CASE(W)                                                                              \
    case W:                                                                                          \
        return launch_bf16<W>(causal, chunk, after, qb, vb, buckets, perm, ob, o_exp, lse_rounds, BH, L, \
                              n_rounds, scale, self_mask, workspace, stream);
    switch (nw) {
        LSH_FWD_CASE(0)
        LSH_FWD_CASE(1)
        LSH_FWD_CASE(2)
        LSH_FWD_CASE(3)
        LSH_FWD_CASE(4)
        LSH_FWD_CASE(5)
        LSH_FWD_CASE(6)
        LSH_FWD_CASE(7)
        LSH_FWD_CASE(8)
        default:
            return hipErrorInvalidValue;
    }
#undef LSH_FWD_CASE
}

}  // namespace lsh

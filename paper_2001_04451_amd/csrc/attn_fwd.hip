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
// bf16 path (gfx950 matrix cores).  A workgroup walks a strip of chunk
// pairs of one segment.  The rows of the three live chunks (c0-1, c0, c0+1)
// sit in an LDS ring of three 64-row slots (chunk c in slot (c+3) % 3): the
// query/key rows as XOR-swizzled 128-byte rows, V transposed (row d holds the
// 192 ring keys) so that the V^T operand is one 16-byte read.  Moving to the
// next pair only brings in two new chunks; their loads are issued before the
// current pair computes and land in LDS after it.  Each wave takes 32
// queries against their 128-key window as four 32x32 tiles:
// S^T = K Q^T on mfma_f32_32x32x16_bf16, masks and softmax on the
// accumulators, then O^T = V^T P^T with the accumulators reused as the B
// operand (the K rows are loaded in a permuted order; see kappa).  Tiles with
// no valid key for the wave's queries are skipped.
//
// Per score element the VALU work is what bounds this kernel, so it is kept
// to a few instructions: the interval mask is one bit of a per-lane word, the
// count of rounds in which i and j differ is one popcount over the guard bits
// of the packed bucket signatures (all words merged, see sig_word), and the
// mask and log2 N_ij come together from one 33-entry LDS table indexed by that
// popcount (index 32 = masked).  The softmax needs no running maximum when
// the wave's logit bound B_i = scale*log2(e)*|q_i| is moderate: every logit
// lies in [-B_i - log2 n_r, B_i], so for B_i <= 60 exp2(x) itself neither
// overflows nor underflows; waves with a larger bound fall back to the online
// maximum.  The row sum l_i adds the bf16-rounded weights that enter P V.
#include "attn_common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr int kRing = 192;  // three chunk slots of 64 rows
constexpr int kMaxBucketsStaged = 1024;
constexpr float kFastBound = 60.f;  // largest B_i handled without a running maximum
constexpr int kMaskedIndex = 32;    // table index of a masked-out key

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
constexpr bf16x2 kOnes = {(__bf16)1.0f, (__bf16)1.0f};

template <bool B>
struct BoolTag {
    static constexpr bool value = B;
};

__device__ __forceinline__ int ring_row(int chunk, int i) { return ((chunk + 3) % 3) * kChunk + i; }

// Bucket signature word w of a token: its ids in rounds 2w and 2w+1 (10 bits
// each) at bit offsets w and w+11.  Adding sig_add(w) to (a ^ b) carries into
// guard bit w+10 (w+21) exactly when the first (second) ids differ; the guard
// bits of different words are distinct, so the number of rounds in which two
// tokens differ is the popcount of the OR over w of
// ((a_w ^ b_w) + sig_add(w)) & sig_guard(w).
__device__ __forceinline__ constexpr uint32_t sig_add(int w) {
    return (0x3FFu << w) | (0x3FFu << (w + 11));
}
__device__ __forceinline__ constexpr uint32_t sig_guard(int w) {
    return (1u << (w + 10)) | (1u << (w + 21));
}

// (a & b) | c as one v_and_or_b32: left to itself the compiler regroups the
// OR chain over the signature words into separate ANDs and three-way ORs.
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t b, uint32_t c) {
    uint32_t d;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "s"(b), "v"(c));
    return d;
}

template <int NW>
struct FwdSig {
    static constexpr int stride = NW <= 1 ? 1 : (NW <= 2 ? 2 : (NW <= 4 ? 4 : 8));  // words per token
    // Per-token record gathered with every staged row: the signature words,
    // zeros, and the key scale in the last word; 16, 32 or 64 bytes, so one
    // record is one aligned run of 16-byte pieces.
    static constexpr int rec_words = stride + 1 <= 4 ? 4 : (stride + 1 <= 8 ? 8 : 16);
    static constexpr int pieces = rec_words / 4;
    static constexpr int aux_per_thread = (4 * pieces + 7) / 8;  // pieces a thread loads per quad
};

template <int NW>
struct FwdShared {
    char Qs[kRing * 128];           // query/key rows (swizzled)
    char Vt[kHeadDim * kRing * 2];  // V^T: row d, 16-byte blocks of 8 keys (swizzled)
    float cf[kRing];                // scale*log2(e)/|q_row| (0 for a zero row)
    uint32_t sig[kRing][FwdSig<NW>::stride];  // bucket signature words (0 outside the sequence)
    int bstart[kMaxBucketsStaged + 1];  // the segment's bucket starts
    float tab[kMaskedIndex + 1];        // -log2 N by mismatch count; -inf = masked
};

// Byte offset of keys k..k+3 (k % 4 == 0) in row d of V^T.  Block b of row d
// sits at b ^ vt_swz(d): the 16 rows read together land in distinct banks.
__device__ __forceinline__ int vt_swz(int d) { return (d + (d >> 3)) & 7; }
__device__ __forceinline__ uint32_t vt_offset(int d, int k) {
    return (uint32_t)d * (kRing * 2) + (uint32_t)(((k >> 3) ^ vt_swz(d)) << 4) + (uint32_t)((k & 4) << 1);
}

// Four consecutive rows of a batch, as loaded by one thread: 16-byte piece
// `part` of each q and v row, and the record pieces k = part (+8) of the
// quad (row k / pieces, piece k % pieces).
template <int NW>
struct RowQuad {
    u32x4 q[4], v[4];
    u32x4 aux[FwdSig<NW>::aux_per_thread];
};

template <int NW>
__device__ __forceinline__ void load_quad(RowQuad<NW>& R, const uint16_t* __restrict__ q,
                                          const uint16_t* __restrict__ v,
                                          const u32x4* __restrict__ rec, int64_t bh, int L,
                                          const int (&pos)[4], int part) {
    constexpr int PP = FwdSig<NW>::pieces;
    const u32x4 zero = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const bool ok = pos[i] >= 0;
        const int64_t grow = bh * L + (ok ? pos[i] : 0);
        R.q[i] = ok ? *reinterpret_cast<const u32x4*>(q + grow * kHeadDim + part * 8) : zero;
        R.v[i] = ok ? *reinterpret_cast<const u32x4*>(v + grow * kHeadDim + part * 8) : zero;
    }
#pragma unroll
    for (int a = 0; a < FwdSig<NW>::aux_per_thread; ++a) {
        const int k = part + 8 * a;
        const int i = k / PP;  // row of the quad (k < 4 * PP)
        const bool ok = k < 4 * PP && pos[i < 4 ? i : 0] >= 0;
        const int64_t grow = bh * L + (ok ? pos[i] : 0);
        R.aux[a] = ok ? rec[grow * PP + k % PP] : zero;
    }
}

// Store a quad at ring rows rr0 .. rr0+3 (Q rows, V transposed, signature
// words and key scales).
template <int NW>
__device__ __forceinline__ void store_quad(FwdShared<NW>& S, const RowQuad<NW>& R, int rr0, int part) {
    constexpr int SW = FwdSig<NW>::stride;
    constexpr int PP = FwdSig<NW>::pieces;
#pragma unroll
    for (int i = 0; i < 4; ++i) lds_store_piece(S.Qs, rr0 + i, part, R.q[i]);
    // V^T: dword e of a piece holds d = 8*part + 2e (low half) and 2e+1 (high)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t a0 = R.v[0][e], a1 = R.v[1][e], a2 = R.v[2][e], a3 = R.v[3][e];
        uint2 lo, hi;
        lo.x = (a0 & 0xFFFFu) | (a1 << 16);
        lo.y = (a2 & 0xFFFFu) | (a3 << 16);
        hi.x = (a0 >> 16) | (a1 & 0xFFFF0000u);
        hi.y = (a2 >> 16) | (a3 & 0xFFFF0000u);
        const int d = 8 * part + 2 * e;
        *reinterpret_cast<uint2*>(S.Vt + vt_offset(d, rr0)) = lo;
        *reinterpret_cast<uint2*>(S.Vt + vt_offset(d + 1, rr0)) = hi;
    }
    // record piece pc of row i: signature words 4pc..4pc+3 (those below SW),
    // the key scale in word 3 of the last piece
#pragma unroll
    for (int a = 0; a < FwdSig<NW>::aux_per_thread; ++a) {
        const int k = part + 8 * a;
        if (k < 4 * PP) {
            const int i = k / PP, pc = k % PP;
            uint32_t* dst = &S.sig[rr0 + i][0];
            if constexpr (SW >= 4) {
                if (4 * pc < SW) *reinterpret_cast<u32x4*>(dst + 4 * pc) = R.aux[a];
            } else if constexpr (SW == 2) {
                *reinterpret_cast<uint2*>(dst) = make_uint2(R.aux[a][0], R.aux[a][1]);
            } else {
                dst[0] = R.aux[a][0];
            }
            if (pc == PP - 1) S.cf[rr0 + i] = __uint_as_float(R.aux[a][3]);
        }
    }
}

template <int NW>
__device__ __forceinline__ void read_sig(const FwdShared<NW>& S, int row, uint32_t (&out)[NW > 0 ? NW : 1]) {
    if constexpr (NW <= 1) {
        out[0] = S.sig[row][0];
    } else if constexpr (NW == 2) {
        const uint2 w = *reinterpret_cast<const uint2*>(&S.sig[row][0]);
        out[0] = w.x;
        out[1] = w.y;
    } else if constexpr (NW > 2) {
#pragma unroll
        for (int w4 = 0; w4 < (NW + 3) / 4; ++w4) {
            const u32x4 w = *reinterpret_cast<const u32x4*>(&S.sig[row][4 * w4]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (4 * w4 + e < NW) out[4 * w4 + e] = w[e];
        }
    }
}

// Slots of the quads that thread `tid` loads for the batch of chunks
// c_first .. c_first + n_chunks_batch - 1 (four consecutive rows per group of
// eight threads); -1 outside the sequence or past the strip.
__device__ __forceinline__ void quad_positions(const int32_t* __restrict__ pseg, int c_first,
                                               int n_chunks_batch, bool live, int n_chunks, int L,
                                               int tid, int (&pos)[4]) {
    const int g = tid >> 3;
    const int chunk = c_first + (4 * g) / kChunk;
    const bool ok = live && g < n_chunks_batch * (kChunk / 4) && chunk >= 0 && chunk < n_chunks;
    int4 p4 = make_int4(-1, -1, -1, -1);
    if (ok) p4 = *reinterpret_cast<const int4*>(pseg + (int64_t)c_first * kChunk + 4 * g);
    pos[0] = ok ? min(max(p4.x, 0), L - 1) : -1;
    pos[1] = ok ? min(max(p4.y, 0), L - 1) : -1;
    pos[2] = ok ? min(max(p4.z, 0), L - 1) : -1;
    pos[3] = ok ? min(max(p4.w, 0), L - 1) : -1;
}

template <int NW, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v,
    const u32x4* __restrict__ rec, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ bstart, uint16_t* __restrict__ o_rounds,
    float* __restrict__ lse_rounds, int L, int n_r, int n_b, float scale, float self_mask,
    int pairs_per_strip) {
    __shared__ __attribute__((aligned(16))) FwdShared<NW> S;

    const int tid = threadIdx.x;
    const int64_t seg = blockIdx.y;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int n_chunks = L / kChunk;
    const int n_pairs = (n_chunks + 1) / 2;
    const int p0 = blockIdx.x * pairs_per_strip;
    const int p1 = min(n_pairs, p0 + pairs_per_strip);
    const float scale_log2e = scale * kLog2e;
    const int32_t* pseg = perm + seg * L;
    const int part = tid & 7;
    const int qrow = 4 * (tid >> 3);  // first row of this thread's quad in a batch
    for (int b = tid; b <= n_b; b += 256) S.bstart[b] = bstart[seg * (n_b + 1) + b];
    if (tid <= kMaskedIndex)
        S.tab[tid] = tid < n_r ? -__log2f((float)(n_r - tid)) : -__builtin_inff();

    // ---- stage the first window: chunk 2p0-1, then chunks 2p0 and 2p0+1 ----
    {
        int pos[4];
        RowQuad<NW> R;
        quad_positions(pseg, 2 * p0 - 1, 1, true, n_chunks, L, tid, pos);
        load_quad<NW>(R, q, v, rec, bh, L, pos, part);
        if (qrow < kChunk) store_quad<NW>(S, R, ring_row(2 * p0 - 1, qrow), part);
        quad_positions(pseg, 2 * p0, 2, true, n_chunks, L, tid, pos);
        load_quad<NW>(R, q, v, rec, bh, L, pos, part);
        store_quad<NW>(S, R, ring_row(2 * p0 + qrow / kChunk, qrow % kChunk), part);
    }
    __syncthreads();

    const int lane = tid & 63, wave = tid >> 6, h = lane >> 5, n = lane & 31;
    const int cw = wave >> 1, qh = wave & 1;

    int pf_pos[4];
    quad_positions(pseg, 2 * (p0 + 1), 2, p0 + 1 < p1, n_chunks, L, tid, pf_pos);

    for (int p = p0; p < p1; ++p) {
        const bool more = p + 1 < p1;
        // the next pair's new chunks load during this pair's compute
        RowQuad<NW> pf;
        load_quad<NW>(pf, q, v, rec, bh, L, pf_pos, part);
        int pf_pos2[4];
        quad_positions(pseg, 2 * (p + 2), 2, p + 2 < p1, n_chunks, L, tid, pf_pos2);

        // ---- compute: per key tile, S^T, masks, softmax, P V ----
        const int cq = 2 * p + cw;  // this wave's query chunk
        if (cq < n_chunks) {
            const int rq = ring_row(cq, qh * 32 + n);
            const int s_q = cq * kChunk + qh * 32 + n;
            uint32_t qsig[NW > 0 ? NW : 1];
            read_sig<NW>(S, rq, qsig);
            // the query's bucket in this round: field r of its signature
            const int beta = min((int)((qsig[r >> 1] >> ((r >> 1) + 11 * (r & 1))) & 0x3FFu), n_b - 1);
            const int wlo = max(0, (cq - 1) * kChunk);
            const int lo = max(S.bstart[beta], wlo);
            const int hi = CAUSAL ? s_q - 1 : min(S.bstart[beta + 1], (cq + 1) * kChunk) - 1;
            bf16x8 qb[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) qb[s] = row_operand(S.Qs, rq, h, s);
            const float cfq = S.cf[rq];
            const float bound = cfq > 0.f ? scale_log2e * scale_log2e / cfq : 0.f;  // B_i
            const bool fast = __ballot(!(bound <= kFastBound)) == 0;
            bool act[4];
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                const int tb = (cq - 1) * kChunk + kt * 32;
                act[kt] = __ballot(lo <= hi && lo <= tb + 31 && hi >= tb) != 0;
            }
            // FAST: every logit of the wave lies in [-B_i - log2 n_r, B_i] with
            // B_i <= 60, so exp2 of the logit itself is a normal fp32 (and
            // bf16) number: no running maximum and no offset are needed.
            auto attend = [&](auto fast_tag) {
            constexpr bool FAST = decltype(fast_tag)::value;
            float m = -__builtin_inff(), lsum = 0.f;
            f32x16 oacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                if (!act[kt]) continue;
                const int kr0 = ring_row(cq - 1 + (kt >> 1), (kt & 1) * 32);
                f32x16 acc = {};
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    acc = mfma32x32x16(row_operand(S.Qs, kr0 + kappa(n), h, s), qb[s], acc);
                // masked keys of this lane's query: bit k of minv <-> tile key 8h + k
                const int tb = (cq - 1) * kChunk + kt * 32;
                const int lo_t = max(lo - tb, 0), hi_t = min(hi - tb, 31);
                uint32_t valid = lo_t <= hi_t ? (0xFFFFFFFFu >> (31 - hi_t)) & (0xFFFFFFFFu << lo_t) : 0u;
                if constexpr (!CAUSAL) {
                    const int self_t = s_q - tb;
                    if (self_t >= 0 && self_t < 32) valid &= ~(1u << self_t);
                }
                const uint32_t minv = ~valid >> (8 * h);
#pragma unroll
                for (int run = 0; run < 2; ++run) {
                    const int kbase = kr0 + 16 * run + 8 * h;
                    const f32x4 c0 = *reinterpret_cast<const f32x4*>(&S.cf[kbase]);
                    const f32x4 c1 = *reinterpret_cast<const f32x4*>(&S.cf[kbase + 4]);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int j = 8 * run + e;
                        uint32_t t = (uint32_t)((int32_t)(minv << (31 - (16 * run + e))) >> 31);
                        if constexpr (NW > 0) {
                            uint32_t ksig[NW];
                            read_sig<NW>(S, kbase + e, ksig);
#pragma unroll
                            for (int w = 0; w < NW; ++w) t = and_or(((qsig[w] ^ ksig[w]) + sig_add(w)), sig_guard(w), t);
                        }
                        const float cfk = e < 4 ? c0[e] : c1[e - 4];
                        acc[j] = fmaf(acc[j], cfk, S.tab[__popc(t)]);
                    }
                }
                float off = 0.f;
                if constexpr (!FAST) {  // online maximum (both lane halves share the row max)
                    float mt = acc[0];
#pragma unroll
                    for (int j = 1; j < 16; ++j) mt = fmaxf(mt, acc[j]);
                    mt = fmaxf(mt, __shfl_xor(mt, 32));
                    const float m_new = fmaxf(m, mt);
                    off = m_new > -__builtin_inff() ? m_new : 0.f;
                    const float corr = __builtin_amdgcn_exp2f(m - off);
                    lsum *= corr;
#pragma unroll
                    for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                        for (int k = 0; k < 16; ++k) oacc[dt][k] *= corr;
                    m = m_new;
                }
                u32x4 pk[2];
#pragma unroll
                for (int ku = 0; ku < 2; ++ku)
#pragma unroll
                    for (int e2 = 0; e2 < 4; ++e2) {
                        const int j = 8 * ku + 2 * e2;
                        const float pa = __builtin_amdgcn_exp2f(FAST ? acc[j] : acc[j] - off);
                        const float pb2 = __builtin_amdgcn_exp2f(FAST ? acc[j + 1] : acc[j + 1] - off);
                        const uint32_t w2 = pack_bf16x2(pa, pb2);
                        pk[ku][e2] = w2;
                        // the row sum takes the bf16 weights that enter P V
                        lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w2), kOnes, lsum, false);
                    }
#pragma unroll
                for (int ku = 0; ku < 2; ++ku) {
                    const int kb = kr0 + 16 * ku + 8 * h;
#pragma unroll
                    for (int dt = 0; dt < 2; ++dt) {
                        const int d = 32 * dt + n;
                        const u32x4 va = *reinterpret_cast<const u32x4*>(S.Vt + vt_offset(d, kb));
                        oacc[dt] = mfma32x32x16(as_bf16x8(va), as_bf16x8(pk[ku]), oacc[dt]);
                    }
                }
            }
            lsum += __shfl_xor(lsum, 32);
            const bool alone = !(lsum > 0.f);  // only itself left as a target
            if (__ballot(alone) != 0) {
                // The output of a lone query is v_i: one more P V step on the
                // diagonal tile with P = 1 at (i, i) for those queries and 0
                // elsewhere adds exactly v_i to their (zero) accumulators.
                // Query n's own key is key n of that tile, held by the lane
                // half (n / 8) % 2 at element n % 8 of key group n / 16.
                const bool mine = alone && h == ((n >> 3) & 1);
                const uint32_t one = (n & 1) ? 0x3F800000u : 0x3F80u;  // bf16 1.0 in its half
                const int kr_diag = ring_row(cq, qh * 32);
#pragma unroll
                for (int ku = 0; ku < 2; ++ku) {
                    u32x4 pk;
#pragma unroll
                    for (int w = 0; w < 4; ++w) pk[w] = (mine && (n >> 4) == ku && ((n & 7) >> 1) == w) ? one : 0u;
                    const int kb = kr_diag + 16 * ku + 8 * h;
#pragma unroll
                    for (int dt = 0; dt < 2; ++dt) {
                        const u32x4 va = *reinterpret_cast<const u32x4*>(S.Vt + vt_offset(32 * dt + n, kb));
                        oacc[dt] = mfma32x32x16(as_bf16x8(va), as_bf16x8(pk), oacc[dt]);
                    }
                }
            }
            const float mref = FAST ? 0.f : m;
            uint16_t* orow = o_rounds + (seg * L + s_q) * kHeadDim;
            // 1/l to within 1 ulp; the result is rounded to bf16.  A lone
            // query divides its exact v_i by 1.
            const float inv = alone ? 1.f : __builtin_amdgcn_rcpf(lsum);
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int d0 = 32 * dt + 8 * i + 4 * h;
                    uint2 o;
                    o.x = pack_bf16x2(oacc[dt][4 * i] * inv, oacc[dt][4 * i + 1] * inv);
                    o.y = pack_bf16x2(oacc[dt][4 * i + 2] * inv, oacc[dt][4 * i + 3] * inv);
                    *reinterpret_cast<uint2*>(orow + d0) = o;
                }
            if (h == 0) {
                // z = scale*|q_i| - self_mask when the token is its own only target
                lse_rounds[seg * L + s_q] = alone ? bound * kLn2 - self_mask : (mref + __log2f(lsum)) * kLn2;
            }
            };
            if (fast)
                attend(BoolTag<true>{});
            else
                attend(BoolTag<false>{});
        }

        __syncthreads();  // every wave is done with the slots of chunks 2p-1 and 2p
        if (more) store_quad<NW>(S, pf, ring_row(2 * p + 2 + qrow / kChunk, qrow % kChunk), part);
#pragma unroll
        for (int i = 0; i < 4; ++i) pf_pos[i] = pf_pos2[i];
        __syncthreads();
    }
}

// fp32 path: one wave per chunk, one lane per query, exact fp32 arithmetic
// on the VALU with an online softmax over the query's key interval.
__global__ __launch_bounds__(64) void attn_fwd_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ v, const int32_t* __restrict__ buckets,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ bstart,
    float* __restrict__ o_rounds, float* __restrict__ lse_rounds, int L, int n_r, int n_b,
    int causal, float scale, float self_mask) {
    __shared__ float Ks[128][kHeadDim + 1];
    __shared__ float Vs2[128][kHeadDim + 1];
    __shared__ float inv[128];
    __shared__ int spos[128];

    const int t = threadIdx.x;
    const int64_t seg = blockIdx.y;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int c = blockIdx.x;
    const int slot0 = (c - 1) * kChunk;
    for (int rho = 0; rho < 128; ++rho) {
        const int slot = slot0 + rho;
        const bool ok = slot >= 0;
        const int pos = ok ? min(max(perm[seg * L + slot], 0), L - 1) : 0;
        Ks[rho][t] = ok ? q[(bh * L + pos) * kHeadDim + t] : 0.f;
        Vs2[rho][t] = ok ? v[(bh * L + pos) * kHeadDim + t] : 0.f;
        if (t == 0) spos[rho] = ok ? pos : -1;
    }
    __syncthreads();
    for (int rr = t; rr < 128; rr += 64) {
        float ss = 0.f;
        for (int u = 0; u < kHeadDim; ++u) ss = fmaf(Ks[rr][u], Ks[rr][u], ss);
        inv[rr] = ss > 0.f ? 1.f / sqrtf(ss) : 0.f;
    }
    __syncthreads();

    const int rq = 64 + t;
    const int s_q = c * kChunk + t;
    const int i_q = spos[rq];
    const int32_t* bi = buckets + (bh * L + i_q) * n_r;
    const int beta = min(max(bi[r], 0), n_b - 1);
    const int32_t* bs = bstart + seg * (n_b + 1);
    const int lo = max(bs[beta], max(0, slot0));
    const int hi = causal ? s_q - 1 : min(bs[beta + 1], (c + 1) * kChunk) - 1;

    float qi[kHeadDim];
    for (int u = 0; u < kHeadDim; ++u) qi[u] = Ks[rq][u];
    float m = -__builtin_inff(), l = 0.f;
    float o[kHeadDim];
    for (int u = 0; u < kHeadDim; ++u) o[u] = 0.f;
    for (int tk = lo; tk <= hi; ++tk) {
        if (tk == s_q) continue;
        const int rho = tk - slot0;
        float dot = 0.f;
        for (int u = 0; u < kHeadDim; ++u) dot = fmaf(qi[u], Ks[rho][u], dot);
        float a = scale * (dot * inv[rho]);
        if (n_r > 1) {
            const int32_t* bj = buckets + (bh * L + spos[rho]) * n_r;
            int nn = 0;
            for (int rr = 0; rr < n_r; ++rr) nn += bi[rr] == bj[rr];
            a -= logf((float)nn);
        }
        const float mn = fmaxf(m, a);
        const float corr = expf(m - mn);
        const float p = expf(a - mn);
        l = l * corr + p;
        for (int u = 0; u < kHeadDim; ++u) o[u] = fmaf(o[u], corr, p * Vs2[rho][u]);
        m = mn;
    }
    float* orow = o_rounds + (seg * L + s_q) * kHeadDim;
    if (l > 0.f) {
        const float il = 1.f / l;
        for (int u = 0; u < kHeadDim; ++u) orow[u] = o[u] * il;
        lse_rounds[seg * L + s_q] = m + logf(l);
    } else {
        float ss = 0.f;
        for (int u = 0; u < kHeadDim; ++u) ss = fmaf(qi[u], qi[u], ss);
        for (int u = 0; u < kHeadDim; ++u) orow[u] = Vs2[rq][u];
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

template <int NW>
hipError_t launch_bf16(dim3 grid, bool causal, const uint16_t* q, const uint16_t* v,
                       const int32_t* buckets, const int32_t* perm, const int32_t* bs, uint16_t* o,
                       float* lse, int64_t BH, int L, int n_r, int n_b, float scale, float self_mask,
                       int pps, void* workspace, hipStream_t stream) {
    const int64_t rows = BH * L;
    u32x4* rec = static_cast<u32x4*>(workspace);
    attn_prep_kernel<NW><<<(unsigned)((rows * 8 + 255) / 256), 256, 0, stream>>>(
        q, buckets, rows, n_r, scale * kLog2e, reinterpret_cast<uint32_t*>(rec));
    if (causal)
        attn_fwd_bf16_kernel<NW, true><<<grid, 256, 0, stream>>>(q, v, rec, perm, bs, o, lse, L, n_r,
                                                                 n_b, scale, self_mask, pps);
    else
        attn_fwd_bf16_kernel<NW, false><<<grid, 256, 0, stream>>>(q, v, rec, perm, bs, o, lse, L, n_r,
                                                                  n_b, scale, self_mask, pps);
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

hipError_t launch_attn_fwd(int64_t BH, int L, int n_rounds, int n_buckets, bool causal,
                           float scale, float self_mask, bool f32, const void* q, const void* v,
                           const int32_t* buckets, const int32_t* perm,
                           const int32_t* bucket_start, void* o_rounds, float* lse_rounds,
                           void* workspace, hipStream_t stream) {
    if (BH == 0 || L == 0) return hipSuccess;
    const unsigned segs = (unsigned)(BH * n_rounds);
    if (f32) {
        attn_fwd_f32_kernel<<<dim3(L / kChunk, segs), 64, 0, stream>>>(
            static_cast<const float*>(q), static_cast<const float*>(v), buckets, perm, bucket_start,
            static_cast<float*>(o_rounds), lse_rounds, L, n_rounds, n_buckets, causal ? 1 : 0, scale,
            self_mask);
        return hipGetLastError();
    }
    // Strips of chunk pairs: long enough to reuse the shared chunk between
    // neighbouring pairs and to hide the next pair's loads, short enough to
    // leave several workgroups per CU for the whole chip.
    const int64_t n_pairs = (L / kChunk + 1) / 2;
    const int pps = (int)std::max<int64_t>(1, std::min<int64_t>(16, n_pairs * segs / 3072));
    const dim3 grid((unsigned)((n_pairs + pps - 1) / pps), segs);
    const uint16_t* qb = static_cast<const uint16_t*>(q);
    const uint16_t* vb = static_cast<const uint16_t*>(v);
    uint16_t* ob = static_cast<uint16_t*>(o_rounds);
    const int nw = n_rounds == 1 ? 0 : (n_rounds + 1) / 2;
#define LSH_FWD_CASE(W)                                                                         \
    case W:                                                                                     \
        return launch_bf16<W>(grid, causal, qb, vb, buckets, perm, bucket_start, ob, lse_rounds, \
                              BH, L, n_rounds, n_buckets, scale, self_mask, pps, workspace, stream);
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

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
// Logits are kept in log2 units: x = (q_i.q_j) * scale*log2(e)/|q_j| - log2 N_ij,
// with N_ij from packed bucket signatures (attn_common.h).
//
// bf16 path (gfx950 matrix cores).  A workgroup walks a strip of chunk
// pairs of one segment.  The rows of the three live chunks (c0-1, c0, c0+1)
// sit in an LDS ring of three 64-row slots (chunk c in slot (c+3) % 3),
// gathered through perm into XOR-swizzled 128-byte rows; moving to the next
// pair only brings in two new chunks, and their loads are issued while the
// current pair computes (perm first, the rows after the first half of the
// compute) so that their latency hides behind it.  Each wave takes 32
// queries against their 128-key window as four 32x32 tiles:
// S^T = K Q^T on mfma_f32_32x32x16_bf16, masks and softmax on the
// accumulators, then O^T = V^T P^T with the accumulators reused as the B
// operand (the K rows are loaded in a permuted order; see kappa).  Tiles with
// no valid key for the wave's queries are skipped.
#include "attn_common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr int kRing = 192;  // three chunk slots of 64 rows
constexpr int kMaxBucketsStaged = 1024;

__device__ __forceinline__ int ring_row(int chunk, int i) { return ((chunk + 3) % 3) * kChunk + i; }

template <int NW>
struct FwdSig {
    static constexpr int stride = NW == 0 ? 1 : (NW <= 1 ? 1 : (NW <= 2 ? 2 : (NW <= 4 ? 4 : 8)));
};

template <int NW>
struct FwdShared {
    char Qs[kRing * 128];
    char Vs[kRing * 128];
    float cf[kRing];     // scale*log2(e)/|q_row| (0 for a zero row)
    int beta[kRing];     // the row's bucket in this round (-1 outside the sequence)
    uint32_t sig[kRing][FwdSig<NW>::stride];
    int bstart[kMaxBucketsStaged + 1];  // the segment's bucket starts
};

// One row of a chunk, as loaded by its eight threads (one 16-byte piece each).
template <int NW>
struct RowLoad {
    u32x4 q, v;
    int beta;
    uint32_t sig;
    bool ok;
};

template <int NW>
__device__ __forceinline__ void load_piece(RowLoad<NW>& R, const uint16_t* __restrict__ q,
                                           const uint16_t* __restrict__ v,
                                           const int32_t* __restrict__ buckets, int64_t bh, int L,
                                           int n_r, int n_b, int r, int pos, int part) {
    R.ok = pos >= 0;
    const int64_t grow = bh * L + (R.ok ? pos : 0);
    const u32x4 zero = {0, 0, 0, 0};
    R.q = R.ok ? *reinterpret_cast<const u32x4*>(q + grow * kHeadDim + part * 8) : zero;
    R.v = R.ok ? *reinterpret_cast<const u32x4*>(v + grow * kHeadDim + part * 8) : zero;
    const int32_t* brow = buckets + grow * n_r;
    R.beta = (R.ok && part == 0) ? min(max(brow[r], 0), n_b - 1) : -1;
    R.sig = 0;
    if constexpr (NW > 0) {
        if (R.ok && part < NW) {
            R.sig = (uint32_t)brow[2 * part];
            if (2 * part + 1 < n_r) R.sig |= (uint32_t)brow[2 * part + 1] << 11;
        }
    }
}

// Store one loaded piece; the eight threads of the row reduce |q|^2 together.
template <int NW>
__device__ __forceinline__ void store_piece(FwdShared<NW>& S, const RowLoad<NW>& R, int lrow,
                                            int part, float scale_log2e) {
    lds_store_piece(S.Qs, lrow, part, R.q);
    lds_store_piece(S.Vs, lrow, part, R.v);
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float a = __uint_as_float(R.q[e] << 16), b = __uint_as_float(R.q[e] & 0xFFFF0000u);
        ss = fmaf(a, a, fmaf(b, b, ss));
    }
    ss += __shfl_xor(ss, 1);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 4);
    if (part == 0) {
        const float nn = sqrtf(ss);
        S.cf[lrow] = nn > 0.f ? scale_log2e / nn : 0.f;
        S.beta[lrow] = R.beta;
    }
    if constexpr (NW > 0) {
        if (part < FwdSig<NW>::stride) S.sig[lrow][part] = part < NW ? R.sig : 0u;
    }
}

template <int NW>
__device__ __forceinline__ void read_sig(const FwdShared<NW>& S, int row, uint32_t (&out)[NW > 0 ? NW : 1]) {
    if constexpr (NW == 1) {
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

template <int NW, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v,
    const int32_t* __restrict__ buckets, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ bstart, float* __restrict__ o_rounds,
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
    for (int b = tid; b <= n_b; b += 256) S.bstart[b] = bstart[seg * (n_b + 1) + b];

    // ---- stage the first window: chunks 2p0-1 .. 2p0+1 ----
#pragma unroll
    for (int i = 0; i < 6; ++i) {
        const int rr = (tid >> 3) + 32 * i;  // 0..191 over the three chunks
        const int chunk = 2 * p0 - 1 + rr / kChunk;
        const int slot = chunk * kChunk + rr % kChunk;
        const int pos = (slot >= 0 && slot < L) ? min(max(pseg[slot], 0), L - 1) : -1;
        RowLoad<NW> R;
        load_piece<NW>(R, q, v, buckets, bh, L, n_r, n_b, r, pos, part);
        store_piece<NW>(S, R, ring_row(chunk, rr % kChunk), part, scale_log2e);
    }
    __syncthreads();

    const int lane = tid & 63, wave = tid >> 6, h = lane >> 5, n = lane & 31;
    const int cw = wave >> 1, qh = wave & 1;

    // positions of the next pair's two new chunks (prefetch, step 1)
    int pf_pos[4];
    auto load_pos = [&](int pn, int (&pos)[4]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int rr = (tid >> 3) + 32 * i;  // 0..127 over chunks 2pn, 2pn+1
            const int slot = 2 * pn * kChunk + rr;
            pos[i] = (pn < p1 && slot < L) ? min(max(pseg[slot], 0), L - 1) : -1;
        }
    };
    load_pos(p0 + 1, pf_pos);

    for (int p = p0; p < p1; ++p) {
        const bool more = p + 1 < p1;
        // prefetch, step 2: the rows of the next pair's new chunks, in flight
        // during this pair's compute; step 1 for the pair after that
        RowLoad<NW> pf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            load_piece<NW>(pf[i], q, v, buckets, bh, L, n_r, n_b, r, pf_pos[i], part);
        int pf_pos2[4];
        load_pos(p + 2, pf_pos2);

        // ---- compute: per key tile, S^T, masks, online softmax, P V ----
        const int cq = 2 * p + cw;  // this wave's query chunk
        const bool active = cq < n_chunks;
        if (active) {
            const int rq = ring_row(cq, qh * 32 + n);
            const int s_q = cq * kChunk + qh * 32 + n;
            const int beta = max(S.beta[rq], 0);
            const int wlo = max(0, (cq - 1) * kChunk);
            const int lo = max(S.bstart[beta], wlo);
            const int hi = CAUSAL ? s_q - 1 : min(S.bstart[beta + 1], (cq + 1) * kChunk) - 1;
            bf16x8 qb[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) qb[s] = row_operand(S.Qs, rq, h, s);
            uint32_t qsig[NW > 0 ? NW : 1];
            read_sig<NW>(S, rq, qsig);
            bool act[4];
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                const int tb = (cq - 1) * kChunk + kt * 32;
                act[kt] = __ballot(lo <= hi && lo <= tb + 31 && hi >= tb) != 0;
            }
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
                const int tb = (cq - 1) * kChunk + kt * 32;
                const int lo_t = lo - tb, hi_t = hi - tb, self_t = s_q - tb;
                float mt = -__builtin_inff();
#pragma unroll
                for (int run = 0; run < 2; ++run) {
                    const int kbase = kr0 + 16 * run + 8 * h;
                    const f32x4 c0 = *reinterpret_cast<const f32x4*>(&S.cf[kbase]);
                    const f32x4 c1 = *reinterpret_cast<const f32x4*>(&S.cf[kbase + 4]);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int j = 8 * run + e;
                        const int kk = 16 * run + 8 * h + e;
                        bool valid = kk >= lo_t && kk <= hi_t;
                        if constexpr (!CAUSAL) valid = valid && kk != self_t;
                        float nlog2 = 0.f;
                        if constexpr (NW > 0) {
                            uint32_t ksig[NW];
                            read_sig<NW>(S, kbase + e, ksig);
                            int nm = 0;
#pragma unroll
                            for (int w = 0; w < NW; ++w) nm += sig_mismatches(qsig[w], ksig[w]);
                            nlog2 = __log2f((float)(n_r - nm));
                        }
                        const float cfk = e < 4 ? c0[e] : c1[e - 4];
                        acc[j] = valid ? fmaf(acc[j], cfk, -nlog2) : -__builtin_inff();
                        mt = fmaxf(mt, acc[j]);
                    }
                }
                // online softmax over the tiles (both lane halves share the row max)
                mt = fmaxf(mt, __shfl_xor(mt, 32));
                const float m_new = fmaxf(m, mt);
                const float msub = m_new > -__builtin_inff() ? m_new : 0.f;
                const float corr = __builtin_amdgcn_exp2f(m - msub);
                lsum *= corr;
#pragma unroll
                for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                    for (int k = 0; k < 16; ++k) oacc[dt][k] *= corr;
                m = m_new;
                u32x4 pk[2];
#pragma unroll
                for (int ku = 0; ku < 2; ++ku)
#pragma unroll
                    for (int e2 = 0; e2 < 4; ++e2) {
                        const int j = 8 * ku + 2 * e2;
                        const float pa = __builtin_amdgcn_exp2f(acc[j] - msub);
                        const float pb2 = __builtin_amdgcn_exp2f(acc[j + 1] - msub);
                        lsum += pa + pb2;
                        pk[ku][e2] = pack_bf16x2(pa, pb2);
                    }
#pragma unroll
                for (int ku = 0; ku < 2; ++ku)
#pragma unroll
                    for (int dt = 0; dt < 2; ++dt)
                        oacc[dt] = mfma32x32x16(col_operand(S.Vs, kr0 + 16 * ku + 8 * h, 32 * dt + n),
                                                as_bf16x8(pk[ku]), oacc[dt]);
            }
            lsum += __shfl_xor(lsum, 32);
            const bool alone = !(m > -__builtin_inff());  // only itself left as a target
            float* orow = o_rounds + (seg * L + s_q) * kHeadDim;
            const float inv = alone ? 0.f : 1.f / lsum;
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int d0 = 32 * dt + 8 * i + 4 * h;
                    f32x4 o;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        o[e] = alone ? bf16_bits_to_f32(lds_elem(S.Vs, rq, d0 + e)) : oacc[dt][4 * i + e] * inv;
                    *reinterpret_cast<f32x4*>(orow + d0) = o;
                }
            if (h == 0) {
                // z = scale*|q_i| - self_mask when the token is its own only target
                const float cfq = S.cf[rq];
                const float qnorm = cfq > 0.f ? scale_log2e / cfq : 0.f;
                lse_rounds[seg * L + s_q] = alone ? scale * qnorm - self_mask : (m + __log2f(lsum)) * kLn2;
            }
        }

        __syncthreads();  // every wave is done with the slots of chunks 2p-1 and 2p
        if (more) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rr = (tid >> 3) + 32 * i;
                store_piece<NW>(S, pf[i], ring_row(2 * p + 2 + rr / kChunk, rr % kChunk), part, scale_log2e);
            }
        }
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

template <int NW>
hipError_t launch_bf16(dim3 grid, bool causal, const uint16_t* q, const uint16_t* v,
                       const int32_t* buckets, const int32_t* perm, const int32_t* bs, float* o,
                       float* lse, int L, int n_r, int n_b, float scale, float self_mask, int pps,
                       hipStream_t stream) {
    if (causal)
        attn_fwd_bf16_kernel<NW, true><<<grid, 256, 0, stream>>>(q, v, buckets, perm, bs, o, lse, L,
                                                                 n_r, n_b, scale, self_mask, pps);
    else
        attn_fwd_bf16_kernel<NW, false><<<grid, 256, 0, stream>>>(q, v, buckets, perm, bs, o, lse, L,
                                                                  n_r, n_b, scale, self_mask, pps);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_fwd(int64_t BH, int L, int n_rounds, int n_buckets, bool causal,
                           float scale, float self_mask, bool f32, const void* q, const void* v,
                           const int32_t* buckets, const int32_t* perm,
                           const int32_t* bucket_start, float* o_rounds, float* lse_rounds,
                           hipStream_t stream) {
    if (BH == 0 || L == 0) return hipSuccess;
    const unsigned segs = (unsigned)(BH * n_rounds);
    if (f32) {
        attn_fwd_f32_kernel<<<dim3(L / kChunk, segs), 64, 0, stream>>>(
            static_cast<const float*>(q), static_cast<const float*>(v), buckets, perm, bucket_start,
            o_rounds, lse_rounds, L, n_rounds, n_buckets, causal ? 1 : 0, scale, self_mask);
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
    const int nw = n_rounds == 1 ? 0 : (n_rounds + 1) / 2;
#define LSH_FWD_CASE(W)                                                                         \
    case W:                                                                                     \
        return launch_bf16<W>(grid, causal, qb, vb, buckets, perm, bucket_start, o_rounds,      \
                              lse_rounds, L, n_rounds, n_buckets, scale, self_mask, pps, stream);
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

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
// N_ij (the number of rounds in which j shares i's bucket) comes from packed
// bucket signatures, two 10-bit ids per word with guard bits:
//   nonzero fields of (a ^ b) = popcount(((a ^ b) + 0x1FFBFF) & 0x200400).
//
// bf16 path (gfx950 matrix cores): one workgroup stages the rows of chunks
// c0-1 .. c0+1 (gathered through perm) in LDS; each wave takes 32 queries
// against the 128-key window as four 32x32 tiles: S^T = K Q^T on
// mfma_f32_32x32x16_bf16, masks/softmax on the accumulators, then
// O^T = V^T P^T reusing the accumulators as the B operand (the K rows are
// loaded in a permuted order so that no shuffle is needed).  Tiles without
// any valid key for the wave's queries are skipped entirely.
#include "common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr int kRows = 192;  // LDS rows: chunks c0-1, c0, c0+1
constexpr int kQStride = 72;
constexpr int kVStride = 68;
constexpr uint32_t kSigAdd = 0x3FFu | (0x3FFu << 11);
constexpr uint32_t kSigGuard = (1u << 10) | (1u << 21);

// A-operand row m of a key tile holds key kappa(m), which puts key
// 16*(j/8) + 8*(l/32) + (j%8) in accumulator register j of lane l.
__device__ __forceinline__ int kappa(int m) {
    return 16 * (m >> 4) + 8 * ((m >> 2) & 1) + 4 * ((m >> 3) & 1) + (m & 3);
}

template <int NW, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v,
    const int32_t* __restrict__ buckets, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ bstart, float* __restrict__ o_rounds,
    float* __restrict__ lse_rounds, int L, int n_r, int n_b, float scale, float self_mask) {
    constexpr int SIGS = NW == 0 ? 1 : (NW <= 4 ? 4 : 8);
    __shared__ __attribute__((aligned(16))) uint16_t Qs[kRows][kQStride];
    __shared__ __attribute__((aligned(16))) uint16_t Vs[kRows][kVStride];
    __shared__ __attribute__((aligned(16))) float cf[kRows];
    __shared__ float nrm[kRows];
    __shared__ int sbeta[kRows];
    __shared__ __attribute__((aligned(16))) uint32_t sig[kRows][SIGS];

    const int tid = threadIdx.x;
    const int64_t seg = blockIdx.y;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int pair = blockIdx.x;
    const int slot0 = (2 * pair - 1) * kChunk;
    const float scale_log2e = scale * kLog2e;

    // ---- stage rows [slot0, slot0 + 192) gathered through perm ----
#pragma unroll
    for (int i = 0; i < 6; ++i) {
        const int idx = tid + 256 * i;
        const int rho = idx >> 3, part = idx & 7;
        const int slot = slot0 + rho;
        const bool ok = slot >= 0 && slot < L;
        const int pos = ok ? min(max(perm[seg * L + slot], 0), L - 1) : 0;
        const int64_t grow = bh * L + pos;
        const u32x4 qq = ok ? *reinterpret_cast<const u32x4*>(q + grow * kHeadDim + part * 8) : u32x4{0, 0, 0, 0};
        const u32x4 vv = ok ? *reinterpret_cast<const u32x4*>(v + grow * kHeadDim + part * 8) : u32x4{0, 0, 0, 0};
        *reinterpret_cast<u32x4*>(&Qs[rho][part * 8]) = qq;
        uint32_t* vdst = reinterpret_cast<uint32_t*>(&Vs[rho][part * 8]);
        *reinterpret_cast<uint2*>(vdst) = make_uint2(vv[0], vv[1]);
        *reinterpret_cast<uint2*>(vdst + 2) = make_uint2(vv[2], vv[3]);
        float ss = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = __uint_as_float(qq[e] << 16), b = __uint_as_float(qq[e] & 0xFFFF0000u);
            ss = fmaf(a, a, fmaf(b, b, ss));
        }
        ss += __shfl_xor(ss, 1);
        ss += __shfl_xor(ss, 2);
        ss += __shfl_xor(ss, 4);
        const int32_t* brow = buckets + grow * n_r;
        if (part == 0) {
            const float nn = sqrtf(ss);
            nrm[rho] = nn;
            cf[rho] = nn > 0.f ? scale_log2e / nn : 0.f;
            sbeta[rho] = ok ? min(max(brow[r], 0), n_b - 1) : -1;
        }
        if constexpr (NW > 0) {
            if (part < NW) {
                const int ra = 2 * part, rb = 2 * part + 1;
                uint32_t w = 0;
                if (ok) {
                    w = (uint32_t)brow[ra];
                    if (rb < n_r) w |= (uint32_t)brow[rb] << 11;
                }
                sig[rho][part] = w;
            }
        }
    }
    __syncthreads();

    // ---- per wave: 32 queries against the 128-key window ----
    const int lane = tid & 63, wave = tid >> 6, h = lane >> 5, n = lane & 31;
    const int cw = wave >> 1, qh = wave & 1;
    const int c = 2 * pair + cw;
    if (c >= L / kChunk) return;  // no barrier follows
    const int kb = cw * kChunk;                  // LDS row of the first window key
    const int rq = kb + kChunk + qh * 32 + n;    // LDS row of this lane's query
    const int s_q = c * kChunk + qh * 32 + n;    // its sorted slot
    const int wlo = max(0, (c - 1) * kChunk);
    const int32_t* bs = bstart + seg * (n_b + 1);
    const int beta = sbeta[rq];
    const int lo = max(bs[beta], wlo);
    const int hi = CAUSAL ? s_q - 1 : min(bs[beta + 1], (c + 1) * kChunk) - 1;

    bf16x8 qb[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) qb[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(&Qs[rq][32 * h + 8 * s]));
    uint32_t qsig[NW > 0 ? NW : 1];
#pragma unroll
    for (int w = 0; w < NW; ++w) qsig[w] = sig[rq][w];

    bool act[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        const int tb = (c - 1) * kChunk + kt * 32;
        act[kt] = __ballot(lo <= hi && lo <= tb + 31 && hi >= tb) != 0;
    }

    f32x16 acc[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        acc[kt] = f32x16{};
        if (act[kt]) {
            const int arow = kb + kt * 32 + kappa(n);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4*>(&Qs[arow][32 * h + 8 * s]));
                acc[kt] = mfma32x32x16(a, qb[s], acc[kt]);
            }
        }
    }

    // pass 1: masked logits (log2 units) and the row maximum.  The lane's 16
    // keys of a tile are two runs of 8 consecutive rows, so their per-key
    // factors and signatures come in as 16-byte LDS reads.
    float mrow = -__builtin_inff();
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        if (!act[kt]) continue;
        const int tb = (c - 1) * kChunk + kt * 32;
        const int lo_t = lo - tb, hi_t = hi - tb, self_t = s_q - tb;  // bounds in tile coordinates
#pragma unroll
        for (int run = 0; run < 2; ++run) {
            const int kbase = kb + kt * 32 + 16 * run + 8 * h;  // LDS row of the run's first key
            const f32x4 c0 = *reinterpret_cast<const f32x4*>(&cf[kbase]);
            const f32x4 c1 = *reinterpret_cast<const f32x4*>(&cf[kbase + 4]);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int j = 8 * run + e;
                const int kk = 16 * run + 8 * h + e;  // key index inside the tile
                bool valid = kk >= lo_t && kk <= hi_t;
                if constexpr (!CAUSAL) valid = valid && kk != self_t;
                float nlog2 = 0.f;
                if constexpr (NW > 0) {
                    const u32x4 k0 = *reinterpret_cast<const u32x4*>(&sig[kbase + e][0]);
                    int nm = 0;
#pragma unroll
                    for (int w = 0; w < (NW < 4 ? NW : 4); ++w)
                        nm += __popc(((qsig[w] ^ k0[w]) + kSigAdd) & kSigGuard);
                    if constexpr (NW > 4) {
                        const u32x4 k1 = *reinterpret_cast<const u32x4*>(&sig[kbase + e][4]);
#pragma unroll
                        for (int w = 4; w < NW; ++w)
                            nm += __popc(((qsig[w] ^ k1[w - 4]) + kSigAdd) & kSigGuard);
                    }
                    nlog2 = __log2f((float)(n_r - nm));
                }
                const float cfk = e < 4 ? c0[e] : c1[e - 4];
                const float x = fmaf(acc[kt][j], cfk, -nlog2);
                acc[kt][j] = valid ? x : -__builtin_inff();
                mrow = fmaxf(mrow, acc[kt][j]);
            }
        }
    }
    mrow = fmaxf(mrow, __shfl_xor(mrow, 32));
    const bool alone = !(mrow > -__builtin_inff());  // only itself left as a target

    // Rows left with only themselves still take part in the matrix-core
    // products below (every lane supplies operands); their probabilities are 0.
    const float msub = alone ? 0.f : mrow;

    // pass 2: probabilities, row sum, bf16 B operands for P V
    float lsum = 0.f;
    u32x4 pk[4][2];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        if (!act[kt]) continue;
#pragma unroll
        for (int ku = 0; ku < 2; ++ku)
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
                const int j = 8 * ku + 2 * e2;
                const float p0 = __builtin_amdgcn_exp2f(acc[kt][j] - msub);
                const float p1 = __builtin_amdgcn_exp2f(acc[kt][j + 1] - msub);
                lsum += p0 + p1;
                pk[kt][ku][e2] = pack_bf16x2(p0, p1);
            }
    }
    lsum += __shfl_xor(lsum, 32);

    f32x16 oacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        if (!act[kt]) continue;
#pragma unroll
        for (int ku = 0; ku < 2; ++ku) {
            const bf16x8 pb = as_bf16x8(pk[kt][ku]);
            const int vr = kb + kt * 32 + 16 * ku + 8 * h;
#pragma unroll
            for (int dt = 0; dt < 2; ++dt) {
                const int dcol = 32 * dt + n;
                u32x4 va;
#pragma unroll
                for (int e2 = 0; e2 < 4; ++e2)
                    va[e2] = (uint32_t)Vs[vr + 2 * e2][dcol] | ((uint32_t)Vs[vr + 2 * e2 + 1][dcol] << 16);
                oacc[dt] = mfma32x32x16(as_bf16x8(va), pb, oacc[dt]);
            }
        }
    }

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
                o[e] = alone ? bf16_bits_to_f32(Vs[rq][d0 + e]) : oacc[dt][4 * i + e] * inv;
            *reinterpret_cast<f32x4*>(orow + d0) = o;
        }
    // z = scale*|q_i| - self_mask when the token is its own only target
    if (h == 0)
        lse_rounds[seg * L + s_q] = alone ? scale * nrm[rq] - self_mask : (mrow + __log2f(lsum)) * kLn2;
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
                       float* lse, int L, int n_r, int n_b, float scale, float self_mask,
                       hipStream_t stream) {
    if (causal)
        attn_fwd_bf16_kernel<NW, true><<<grid, 256, 0, stream>>>(q, v, buckets, perm, bs, o, lse, L,
                                                                 n_r, n_b, scale, self_mask);
    else
        attn_fwd_bf16_kernel<NW, false><<<grid, 256, 0, stream>>>(q, v, buckets, perm, bs, o, lse, L,
                                                                  n_r, n_b, scale, self_mask);
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
    const dim3 grid((unsigned)((L / kChunk + 1) / 2), segs);
    const uint16_t* qb = static_cast<const uint16_t*>(q);
    const uint16_t* vb = static_cast<const uint16_t*>(v);
    const int nw = n_rounds == 1 ? 0 : (n_rounds + 1) / 2;
#define LSH_FWD_CASE(W)                                                                         \
    case W:                                                                                     \
        return launch_bf16<W>(grid, causal, qb, vb, buckets, perm, bucket_start, o_rounds,      \
                              lse_rounds, L, n_rounds, n_buckets, scale, self_mask, stream);
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

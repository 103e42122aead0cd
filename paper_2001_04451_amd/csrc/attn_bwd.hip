// Backward of chunked LSH attention (gradients with respect to q and v,
// buckets held fixed).  The paper gives no LSH backward; it recomputes
// attention in the backward pass of its memory-efficient attention (Sec. 2),
// and this follows that: the logits of every round are recomputed from q,
// perm and the forward's total log-partition z_i, with
//   P = exp(a - z_i),  dA = P (dO_i . v_j - D_i),  D_i = dO_i . o_i,
//   dv_j += P dO_i,  dq_i += scale dA k_j,  dk_j += scale dA q_i,
// and dk flows back through k_j = q_j/|q_j| in the final reduction.
//
// Kernels (gfx950):
//  * bwd_prep:   D_i per position.
//  * bwd_fused:  per chunk c of a round, one staged window (chunks c-1, c,
//                c+1).  Two waves take the key role for chunk c's keys
//                (lanes on keys): S = Q K^T and dP = dO V^T on the matrix
//                cores against the queries of chunks c and c+1 (the only ones
//                whose window holds chunk c), then dV^T += dO^T P and
//                dK^T += Q^T dA.  Two waves take the query role for chunk c's
//                queries (lanes on queries, as in the forward): S^T = K Q^T,
//                dP^T = V dO^T over chunks c-1 and c, then dQ^T += K^T dA^T.
//                The key role hands dK to the query role through LDS, which
//                adds it through the normalisation Jacobian and writes one
//                per-round dq partial; the key role writes the dv partial.
//  * bwd_reduce: per position, sum the rounds through `undo`, write dq, dv.
// Every (query, key) pair of a round is owned by exactly one lane of each
// role, so no atomics are used and results are deterministic.
#include "attn_common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr int kWin = 192;  // staged rows: three chunks
constexpr int kMaskedIndex = 32;  // table index of a masked-out pair

template <int NW>
struct SigStride {
    static constexpr int value = NW <= 1 ? 1 : (NW <= 2 ? 2 : (NW <= 4 ? 4 : 8));
};

// Row metadata of the staged window (one entry per staged row).
template <int NW>
struct RowMeta {
    float cf[kWin];  // scale*log2(e)/|q_row|
    float z2[kWin];  // the row's total log-partition, log2 units
    float D[kWin];   // dO_row . o_row
    int lo[kWin];    // slot interval of the row's valid keys (as a query)
    int hi[kWin];
    uint32_t sig[kWin][SigStride<NW>::value];
    float tab[kMaskedIndex + 1];  // -log2 N by mismatch count; -inf = masked
};

template <int NW>
__device__ __forceinline__ void load_sig(const RowMeta<NW>& M, int row, uint32_t (&out)[NW > 0 ? NW : 1]) {
    if constexpr (NW == 1) {
        out[0] = M.sig[row][0];
    } else if constexpr (NW == 2) {
        const uint2 v = *reinterpret_cast<const uint2*>(&M.sig[row][0]);
        out[0] = v.x;
        out[1] = v.y;
    } else if constexpr (NW > 2) {
#pragma unroll
        for (int w4 = 0; w4 < (NW + 3) / 4; ++w4) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(&M.sig[row][4 * w4]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (4 * w4 + e < NW) out[4 * w4 + e] = v[e];
        }
    }
}

// Number of rounds in which two tokens' bucket ids differ (0 when there is
// one round, which needs no signatures).
template <int NW>
__device__ __forceinline__ int n_mismatch(const uint32_t (&a)[NW > 0 ? NW : 1],
                                          const uint32_t (&b)[NW > 0 ? NW : 1]) {
    int nm = 0;
    if constexpr (NW > 0) {
#pragma unroll
        for (int w = 0; w < NW; ++w) nm += sig_mismatches(a[w], b[w]);
    }
    return nm;
}

// Stage rows [slot0, slot0 + 192) of one segment, gathered through perm:
// q rows into Qs (all rows), v rows into Vs for rows [v_lo, v_hi), dO rows
// into Ds for rows [d_lo, d_hi) (stored at row - d_lo), and per-row metadata.
template <int NW, bool CAUSAL>
__device__ __forceinline__ void stage_window(
    char* Qs, char* Vs, int v_lo, int v_hi, char* Ds, int d_lo, int d_hi, RowMeta<NW>& M,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse_total,
    const float* __restrict__ Dbuf, const int32_t* __restrict__ buckets,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ bstart, int64_t seg,
    int64_t bh, int r, int slot0, int L, int n_r, int n_b, float scale_log2e) {
    // Three phases, each issuing all of its loads before any result is used:
    // the staged slots' positions, then (through them) the rows, bucket ids,
    // log-partitions and D, then (through the ids) the bucket bounds.  Every
    // address is clamped to a valid one, so no load sits under a per-lane
    // condition (which would make it a branch with its own wait); slots
    // outside the sequence get zero rows and an empty interval afterwards.
    constexpr int kIt = kWin * 8 / 256;
    const int tid = threadIdx.x, part = tid & 7;
    const int32_t* bs = bstart + seg * (n_b + 1);
    const int32_t* pseg = perm + seg * L;
    if (tid <= kMaskedIndex) M.tab[tid] = tid < n_r ? -__log2f((float)(n_r - tid)) : -__builtin_inff();
    const u32x4 zero = {0, 0, 0, 0};

    int pos[kIt];
#pragma unroll
    for (int i = 0; i < kIt; ++i) {
        const int slot = slot0 + ((tid + 256 * i) >> 3);
        pos[i] = pseg[min(max(slot, 0), L - 1)];
    }

    u32x4 qq[kIt], vv[kIt], dd[kIt];
    int beta[kIt];
    uint32_t lo_id[kIt], hi_id[kIt];
    float zl[kIt], Dl[kIt];
#pragma unroll
    for (int i = 0; i < kIt; ++i) {
        const int rho = (tid + 256 * i) >> 3;  // the same for the whole wave's 8 rows' range test
        const int64_t grow = bh * L + min(max(pos[i], 0), L - 1);
        const int64_t off = grow * kHeadDim + part * 8;
        qq[i] = *reinterpret_cast<const u32x4*>(q + off);
        vv[i] = zero;
        if (rho >= v_lo && rho < v_hi) vv[i] = *reinterpret_cast<const u32x4*>(v + off);
        dd[i] = zero;
        if (rho >= d_lo && rho < d_hi) dd[i] = *reinterpret_cast<const u32x4*>(dout + off);
        const int32_t* brow = buckets + grow * n_r;
        beta[i] = brow[r];
        lo_id[i] = (uint32_t)brow[min(2 * part, n_r - 1)];
        hi_id[i] = (uint32_t)brow[min(2 * part + 1, n_r - 1)];
        zl[i] = lse_total[grow];
        Dl[i] = Dbuf[grow];
    }

    int b0[kIt], b1[kIt];
#pragma unroll
    for (int i = 0; i < kIt; ++i) {
        const int bb = min(max(beta[i], 0), n_b - 1);
        b0[i] = bs[bb];
        b1[i] = bs[bb + 1];
    }

#pragma unroll
    for (int i = 0; i < kIt; ++i) {
        const int rho = (tid + 256 * i) >> 3;
        const int slot = slot0 + rho;
        const bool ok = slot >= 0 && slot < L;
        const u32x4 qv = ok ? qq[i] : zero;
        lds_store_piece(Qs, rho, part, qv);
        if (rho >= v_lo && rho < v_hi) lds_store_piece(Vs, rho - v_lo, part, ok ? vv[i] : zero);
        if (rho >= d_lo && rho < d_hi) lds_store_piece(Ds, rho - d_lo, part, ok ? dd[i] : zero);
        float ss = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float a = __uint_as_float(qv[e] << 16), b = __uint_as_float(qv[e] & 0xFFFF0000u);
            ss = fmaf(a, a, fmaf(b, b, ss));
        }
        ss += __shfl_xor(ss, 1);
        ss += __shfl_xor(ss, 2);
        ss += __shfl_xor(ss, 4);
        if (part == 0) {
            const float nn = sqrtf(ss);
            M.cf[rho] = nn > 0.f ? scale_log2e / nn : 0.f;
            M.z2[rho] = ok ? zl[i] * kLog2e : 0.f;
            M.D[rho] = ok ? Dl[i] : 0.f;
            const int c = (slot >= 0 ? slot : 0) / kChunk;
            const int wlo = max(0, (c - 1) * kChunk);
            M.lo[rho] = ok ? max(b0[i], wlo) : 1;
            M.hi[rho] = ok ? (CAUSAL ? slot - 1 : min(b1[i], (c + 1) * kChunk) - 1) : 0;
        }
        if constexpr (NW > 0) {
            if (part < SigStride<NW>::value) {
                uint32_t w = 0;
                if (ok && part < NW) {
                    w = lo_id[i];
                    if (2 * part + 1 < n_r) w |= hi_id[i] << 11;
                }
                M.sig[rho][part] = w;
            }
        }
    }
}

// ---- fused: per chunk c, the key role (dK, dV of chunk c's keys, lanes on
// keys) and the query role (dQ of chunk c's queries, lanes on queries) over
// one staged window, chunks c-1, c and c+1 ----
// Waves 0 and 1 take the key role: S = Q K^T and dP = dO V^T against the
// queries of chunks c and c+1 (the only ones whose window holds chunk c),
// then dV^T += dO^T P and dK^T += Q^T dA.  Waves 2 and 3 take the query role:
// S^T = K Q^T, dP^T = V dO^T over chunks c-1 and c, then dQ^T += K^T dA^T.
// Both roles cover the same 64 tokens, so the key role hands dK_i to the
// query role through LDS, which adds it through the normalisation Jacobian
// (dq_i += (dk_i - (dk_i.k_i) k_i)/|q_i|, linear, so per round is exact) and
// writes one per-round partial for dq and one for dv.
template <int NW, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void bwd_fused_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse_total,
    const float* __restrict__ Dbuf, const int32_t* __restrict__ buckets,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ bstart,
    float* __restrict__ dq_r, float* __restrict__ dv_r, int L, int n_r, int n_b, float scale) {
    __shared__ __attribute__((aligned(16))) char Qs[kWin * 128];
    __shared__ __attribute__((aligned(16))) char Vs[128 * 128];    // chunks c-1, c
    __shared__ __attribute__((aligned(16))) char Ds[128 * 128];    // chunks c, c+1; then dK of chunk c
    __shared__ __attribute__((aligned(16))) RowMeta<NW> M;

    const int64_t seg = blockIdx.y;
    const int64_t bh = seg / n_r;
    const int r = (int)(seg % n_r);
    const int c = blockIdx.x;
    const int slot0 = (c - 1) * kChunk;  // row 0 = first slot of chunk c - 1
    stage_window<NW, CAUSAL>(Qs, Vs, 0, 2 * kChunk, Ds, kChunk, kWin, M, q, v, dout, lse_total,
                             Dbuf, buckets, perm, bstart, seg, bh, r, slot0, L, n_r, n_b,
                             scale * kLog2e);
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, h = lane >> 5, n = lane & 31;
    f32x16 accA[2] = {f32x16{}, f32x16{}};  // key role: dK; query role: dQ
    f32x16 accB[2] = {f32x16{}, f32x16{}};  // key role: dV
    if (wave < 2) {
        const int kh = wave & 1;
        const int kr = kChunk + kh * 32 + n;  // this lane's key row (chunk c)
        const int t_key = slot0 + kr;
        const float cf_k = M.cf[kr];
        uint32_t sig_k[NW > 0 ? NW : 1];
        load_sig<NW>(M, kr, sig_k);
        bf16x8 bk[4], bv[4];
    #pragma unroll
        for (int s = 0; s < 4; ++s) {
            bk[s] = row_operand(Qs, kr, h, s);
            bv[s] = row_operand(Vs, kr, h, s);
        }
        const int key_lo = slot0 + kChunk + kh * 32;  // slot range of the wave's keys
        const int key_hi = key_lo + 31;

        const int qrow0 = kChunk;  // queries: chunks c and c+1
    #pragma unroll 1
        for (int qt = 0; qt < 4; ++qt) {
            const int qr0 = qrow0 + qt * 32;
            // skip query tiles none of whose intervals reaches the wave's keys
            const int lo_n = M.lo[qr0 + n], hi_n = M.hi[qr0 + n];
            if (__ballot(lo_n <= hi_n && lo_n <= key_hi && hi_n >= key_lo) == 0) continue;

            f32x16 sacc = {}, dpacc = {};
            const int arow = qr0 + kappa(n);
    #pragma unroll
            for (int s = 0; s < 4; ++s) {
                sacc = mfma32x32x16(row_operand(Qs, arow, h, s), bk[s], sacc);
                dpacc = mfma32x32x16(row_operand(Ds, arow - kChunk, h, s), bv[s], dpacc);
            }
            u32x4 pk[2], pl[2], dak[2];  // P as bf16 hi + lo planes (dV), dA as bf16 (dK)
    #pragma unroll
            for (int run = 0; run < 2; ++run) {
                const int qb = qr0 + 16 * run + 8 * h;  // first query row of the lane's run
                // the run's eight queries: interval, log-partition, D
                int lo8[8], hi8[8];
                float z8[8], D8[8];
    #pragma unroll
                for (int e = 0; e < 8; ++e) {
                    lo8[e] = M.lo[qb + e];
                    hi8[e] = M.hi[qb + e];
                    z8[e] = M.z2[qb + e];
                    D8[e] = M.D[qb + e];
                }
    #pragma unroll
                for (int e2 = 0; e2 < 4; ++e2) {
                    float pv[2], dav[2];
    #pragma unroll
                    for (int u = 0; u < 2; ++u) {
                        const int e = 2 * e2 + u;
                        const int qi = qb + e;
                        const int j = 8 * run + e;
                        bool valid = t_key >= lo8[e] && t_key <= hi8[e];
                        if constexpr (!CAUSAL) valid = valid && t_key != slot0 + qi;
                        uint32_t sig_q[NW > 0 ? NW : 1];
                        load_sig<NW>(M, qi, sig_q);
                        // -log2 N_ij, or -inf for a pair outside the query's interval
                        const float mterm = M.tab[valid ? n_mismatch<NW>(sig_q, sig_k) : kMaskedIndex];
                        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[j], cf_k, mterm) - z8[e]);
                        pv[u] = p;
                        dav[u] = p * (dpacc[j] - D8[e]);
                    }
                    const uint32_t hi = pack_bf16x2(pv[0], pv[1]);
                    pk[run][e2] = hi;
                    pl[run][e2] = pack_bf16x2(pv[0] - __uint_as_float(hi << 16),
                                              pv[1] - __uint_as_float(hi & 0xFFFF0000u));
                    dak[run][e2] = pack_bf16x2(dav[0], dav[1]);
                }
            }
            // dV^T += dO^T (P_hi + P_lo),  dK^T += Q^T dA  (k = queries of the tile).
            // dO is exact in bf16 and P_hi + P_lo carries P to ~2^-16, so dV keeps
            // fp32-level accuracy; dA (then scaled and summed) stays one plane.
    #pragma unroll
            for (int ku = 0; ku < 2; ++ku) {
                const int r0 = qr0 + 16 * ku + 8 * h;
    #pragma unroll
                for (int dt = 0; dt < 2; ++dt) {
                    const bf16x8 dOt = col_operand(Ds, r0 - kChunk, 32 * dt + n);
                    accB[dt] = mfma32x32x16(dOt, as_bf16x8(pk[ku]), accB[dt]);
                    accB[dt] = mfma32x32x16(dOt, as_bf16x8(pl[ku]), accB[dt]);
                    accA[dt] = mfma32x32x16(col_operand(Qs, r0, 32 * dt + n), as_bf16x8(dak[ku]), accA[dt]);
                }
            }
        }
    } else {
        const int qh = wave & 1;
        const int kb = 0;                          // first key row of the window
        const int rq = kb + kChunk + qh * 32 + n;  // this lane's query row
        const int s_q = slot0 + rq;
        const int lo = M.lo[rq], hi = M.hi[rq];
        const float z2 = M.z2[rq], Dq = M.D[rq];
        uint32_t sig_q[NW > 0 ? NW : 1];
        load_sig<NW>(M, rq, sig_q);
        bf16x8 bq[4], bdo[4];
    #pragma unroll
        for (int s = 0; s < 4; ++s) {
            bq[s] = row_operand(Qs, rq, h, s);
            bdo[s] = row_operand(Ds, rq - kChunk, h, s);
        }

    #pragma unroll 1
        for (int kt = 0; kt < 4; ++kt) {
            const int tb = slot0 + kb + kt * 32;
            if (__ballot(lo <= hi && lo <= tb + 31 && hi >= tb) == 0) continue;
            const int kr0 = kb + kt * 32;
            f32x16 sacc = {}, dpacc = {};
            const int arow = kr0 + kappa(n);
    #pragma unroll
            for (int s = 0; s < 4; ++s) {
                sacc = mfma32x32x16(row_operand(Qs, arow, h, s), bq[s], sacc);
                dpacc = mfma32x32x16(row_operand(Vs, arow, h, s), bdo[s], dpacc);
            }
            u32x4 dak[2];
    #pragma unroll
            for (int run = 0; run < 2; ++run) {
                const int krb = kr0 + 16 * run + 8 * h;
                float cf8[8];  // the run's eight key scales
    #pragma unroll
                for (int e = 0; e < 8; ++e) cf8[e] = M.cf[krb + e];
    #pragma unroll
                for (int e2 = 0; e2 < 4; ++e2) {
                    float dav[2];
    #pragma unroll
                    for (int u = 0; u < 2; ++u) {
                        const int e = 2 * e2 + u;
                        const int kj = krb + e;
                        const int j = 8 * run + e;
                        const int t = slot0 + kj;
                        bool valid = t >= lo && t <= hi;
                        if constexpr (!CAUSAL) valid = valid && t != s_q;
                        uint32_t sig_k[NW > 0 ? NW : 1];
                        load_sig<NW>(M, kj, sig_k);
                        const float cfk = cf8[e];
                        // -log2 N_ij, or -inf for a key outside the query's interval
                        const float mterm = M.tab[valid ? n_mismatch<NW>(sig_q, sig_k) : kMaskedIndex];
                        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[j], cfk, mterm) - z2);
                        // scale/|q_j| = cf_j / log2(e); the 1/log2(e) is applied at the end
                        dav[u] = p * (dpacc[j] - Dq) * cfk;
                    }
                    dak[run][e2] = pack_bf16x2(dav[0], dav[1]);
                }
            }
    #pragma unroll
            for (int ku = 0; ku < 2; ++ku) {
                const int r0 = kr0 + 16 * ku + 8 * h;
    #pragma unroll
                for (int dt = 0; dt < 2; ++dt)
                    accA[dt] = mfma32x32x16(col_operand(Qs, r0, 32 * dt + n), as_bf16x8(dak[ku]), accA[dt]);
            }
        }
    }
    __syncthreads();  // every wave is done with Ds: it now carries dK
    float* X = reinterpret_cast<float*>(Ds);  // [64 tokens of chunk c][64] fp32
    const int xr = (wave & 1) * 32 + n;      // this lane's token in chunk c
    const int tok = slot0 + kChunk + xr;     // its slot
    if (wave < 2) {
        // lane holds key xr, d = 32dt + 8i + 4h + e
#pragma unroll
        for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int d0 = 32 * dt + 8 * i + 4 * h;
                f32x4 b;
#pragma unroll
                for (int e = 0; e < 4; ++e) b[e] = scale * accA[dt][4 * i + e];
                *reinterpret_cast<f32x4*>(X + xr * kHeadDim + d0) = b;
            }
        if (tok < L) {  // a slot past L (a partial last chunk) has no row
            float* dvrow = dv_r + (seg * L + tok) * kHeadDim;
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    f32x4 a;
#pragma unroll
                    for (int e = 0; e < 4; ++e) a[e] = accB[dt][4 * i + e];
                    *reinterpret_cast<f32x4*>(dvrow + 32 * dt + 8 * i + 4 * h) = a;
                }
        }
    }
    __syncthreads();
    if (wave >= 2) {
        // lane holds query xr, d = 32dt + 8i + 4h + e: its q values (bf16, the
        // row's pieces in Qs) and its dK from the key role
        const int rq = kChunk + xr;
        f32x4 dk[2][4], qv[2][4];
        float ss = 0.f, kd = 0.f;
#pragma unroll
        for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                dk[dt][i] = *reinterpret_cast<const f32x4*>(X + xr * kHeadDim + 32 * dt + 8 * i + 4 * h);
                const u32x4 pc = lds_piece(Qs, rq, 4 * dt + i);
                const uint32_t w0 = pc[2 * h], w1 = pc[2 * h + 1];
                qv[dt][i] = f32x4{__uint_as_float(w0 << 16), __uint_as_float(w0 & 0xFFFF0000u),
                                  __uint_as_float(w1 << 16), __uint_as_float(w1 & 0xFFFF0000u)};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    ss = fmaf(qv[dt][i][e], qv[dt][i][e], ss);
                    kd = fmaf(dk[dt][i][e], qv[dt][i][e], kd);
                }
            }
        ss += __shfl_xor(ss, 32);
        kd += __shfl_xor(kd, 32);
        const float nn = sqrtf(ss);
        const float inv = nn > 0.f ? 1.f / nn : 0.f;  // a zero query has k = 0 and no key gradient
        const float proj = kd * inv;                  // dk . k
        if (tok < L) {
            float* dqrow = dq_r + (seg * L + tok) * kHeadDim;
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    f32x4 a;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        a[e] = kLn2 * accA[dt][4 * i + e] + (dk[dt][i][e] - proj * qv[dt][i][e] * inv) * inv;
                    *reinterpret_cast<f32x4*>(dqrow + 32 * dt + 8 * i + 4 * h) = a;
                }
        }
    }
}

// D_i = dO_i . o_i, 16 lanes per row.
__global__ __launch_bounds__(256) void bwd_prep_kernel(const uint16_t* __restrict__ out,
                                                       const uint16_t* __restrict__ dout,
                                                       int64_t rows, float* __restrict__ Dbuf) {
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
    const int part = threadIdx.x & 15;
    if (row >= rows) return;  // whole 16-lane groups leave together
    const uint2 o = *reinterpret_cast<const uint2*>(out + row * kHeadDim + part * 4);
    const uint2 g = *reinterpret_cast<const uint2*>(dout + row * kHeadDim + part * 4);
    float s = bf16_bits_to_f32(o.x & 0xFFFF) * bf16_bits_to_f32(g.x & 0xFFFF);
    s = fmaf(bf16_bits_to_f32(o.x >> 16), bf16_bits_to_f32(g.x >> 16), s);
    s = fmaf(bf16_bits_to_f32(o.y & 0xFFFF), bf16_bits_to_f32(g.y & 0xFFFF), s);
    s = fmaf(bf16_bits_to_f32(o.y >> 16), bf16_bits_to_f32(g.y >> 16), s);
    for (int off = 8; off >= 1; off >>= 1) s += __shfl_xor(s, off);
    if (part == 0) Dbuf[row] = s;
}

constexpr int kMaxRounds = 16;

// Sum the rounds per position and add the key role:
//   dq_j = sum_r dq_r + (dk_j - (dk_j . k_j) k_j) / |q_j|,  dv_j = sum_r dv_r,
// plus dO_j for a token whose only target in every round was itself (its
// weights are then 1/n_rounds on each round's self entry).
__global__ __launch_bounds__(256) void bwd_reduce_kernel(
    const uint16_t* __restrict__ dout, const float* __restrict__ lse_total,
    const int32_t* __restrict__ undo, const float* __restrict__ dq_r,
    const float* __restrict__ dv_r, int64_t rows, int L, int n_r, float self_mask,
    float* __restrict__ dq, float* __restrict__ dv) {
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
    const int part = threadIdx.x & 15;
    if (row >= rows) return;  // whole 16-lane groups leave together
    const int64_t bh = row / L, i = row % L;
    int64_t base[kMaxRounds];
#pragma unroll
    for (int r = 0; r < kMaxRounds; ++r)
        if (r < n_r) base[r] = ((bh * n_r + r) * L + min(max(undo[(bh * n_r + r) * L + i], 0), L - 1)) * kHeadDim + part * 4;
    f32x4 aq = {0, 0, 0, 0}, av = {0, 0, 0, 0};
#pragma unroll
    for (int r = 0; r < kMaxRounds; ++r)
        if (r < n_r) {
            const f32x4 x = *reinterpret_cast<const f32x4*>(dq_r + base[r]);
            const f32x4 z = *reinterpret_cast<const f32x4*>(dv_r + base[r]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                aq[e] += x[e];
                av[e] += z[e];
            }
        }
    if (lse_total[row] < -0.5f * self_mask) {
        const uint2 g = *reinterpret_cast<const uint2*>(dout + row * kHeadDim + part * 4);
        av[0] += bf16_bits_to_f32(g.x & 0xFFFF);
        av[1] += bf16_bits_to_f32(g.x >> 16);
        av[2] += bf16_bits_to_f32(g.y & 0xFFFF);
        av[3] += bf16_bits_to_f32(g.y >> 16);
    }
    *reinterpret_cast<f32x4*>(dq + row * kHeadDim + part * 4) = aq;
    *reinterpret_cast<f32x4*>(dv + row * kHeadDim + part * 4) = av;
}

struct BwdWs {
    float* dq_r;  // per round: dq through the query role plus the key role's dk through k = q/|q|
    float* dv_r;
    float* D;
    size_t bytes;
};

BwdWs carve(void* base, int64_t BH, int L, int n_rounds) {
    const size_t rr = (size_t)BH * n_rounds * L;
    char* p = static_cast<char*>(base);
    BwdWs w{};
    size_t off = 0;
    w.dq_r = reinterpret_cast<float*>(p + off);
    off += align256(rr * kHeadDim * 4);
    w.dv_r = reinterpret_cast<float*>(p + off);
    off += align256(rr * kHeadDim * 4);
    w.D = reinterpret_cast<float*>(p + off);
    off += align256((size_t)BH * L * 4);
    w.bytes = off;
    return w;
}

template <int NW, bool CAUSAL>
void launch_chunks(dim3 grid, hipStream_t stream, const uint16_t* q, const uint16_t* v,
                   const uint16_t* dout, const float* lse, const float* D, const int32_t* buckets,
                   const int32_t* perm, const int32_t* bs, float* dq_r, float* dv_r, int L, int n_r,
                   int n_b, float scale) {
    bwd_fused_kernel<NW, CAUSAL><<<grid, 256, 0, stream>>>(q, v, dout, lse, D, buckets, perm, bs,
                                                           dq_r, dv_r, L, n_r, n_b, scale);
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
    const unsigned row_grid = (unsigned)((rows * 16 + 255) / 256);
    bwd_prep_kernel<<<row_grid, 256, 0, stream>>>(out, dout, rows, w.D);
    // one workgroup per chunk; a partial last chunk (L not a multiple of the
    // chunk) counts as a chunk
    const dim3 grid((unsigned)((L + kChunk - 1) / kChunk), (unsigned)(BH * n_rounds));
    const int nw = n_rounds == 1 ? 0 : (n_rounds + 1) / 2;
#define LSH_BWD_CASE(W)                                                                          \
    case W:                                                                                      \
        if (causal)                                                                              \
            launch_chunks<W, true>(grid, stream, q, v, dout, lse_total, w.D, buckets, perm,      \
                                   bucket_start, w.dq_r, w.dv_r, L, n_rounds, n_buckets,        \
                                   scale);                                                       \
        else                                                                                     \
            launch_chunks<W, false>(grid, stream, q, v, dout, lse_total, w.D, buckets, perm,     \
                                    bucket_start, w.dq_r, w.dv_r, L, n_rounds,                   \
                                    n_buckets, scale);                                           \
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
    bwd_reduce_kernel<<<row_grid, 256, 0, stream>>>(dout, lse_total, undo, w.dq_r, w.dv_r, rows, L,
                                                    n_rounds, self_mask, dq, dv);
    return hipGetLastError();
}

}  // namespace lsh

// Full shared-QK attention, forward: the memory-efficient baseline of Sec. 2
// (every query's softmax over all keys, without materialising QK^T), which
// the LSH forward approximates and which the paper's speed-versus-length
// comparison (Sec. 5) sets it against.  Keys are k_j = q_j/|q_j|; the logit
// of query i and key j is scale*q_i.k_j, the self key j == i carries the
// App. A mask (its weight exp(-1e5) vanishes in fp32 whenever the query has
// another key; without one the output is v_i and the log-partition is
// scale*|q_i| - self_mask), and under causal masking no later key counts.
//
// gfx950 design.  A workgroup of four waves owns 128 consecutive queries of
// one (batch, head); each wave holds 32 of them (two 16-query tiles) as
// matrix-core B operands in registers for the whole kernel.  The workgroup
// walks the keys in blocks of 64: the next block's k and v rows and key
// scales are copied from global memory straight into the free half of a
// double-buffered LDS area (global_load_lds) while the current block is
// used, with one barrier per block.  Per block and query tile the scores
// come as S^T = K Q^T (four 16-key tiles, mfma_f32_16x16x32_bf16: lane l
// holds keys 4(l/16)..+3 of query l%16), the softmax weights are packed to
// bf16 in place, and O^T += V^T P^T runs on mfma_f32_16x16x16_bf16 with V^T
// read through the LDS transpose read.  As in the chunked kernel, no running
// maximum is needed while the wave's logit bound B_i = scale*log2(e)*|q_i|
// (Cauchy-Schwarz: every logit lies in [-B_i, B_i]) is at most 60, since
// exp2 then neither overflows nor underflows; waves with a larger bound keep
// the online maximum.  Three workgroups share a CU (a few registers spill;
// measured faster than two without spills, most of all for short
// sequences, where a workgroup walks few blocks).  Masks are applied only in
// blocks that hold a query's own position or the sequence end; under causal
// masking a wave stops after the block holding its last query, and
// workgroups of later queries (more keys) are dispatched first.
#include "attn_common.h"
#include "launch.h"

namespace lsh {
namespace {

constexpr int kDenseWaves = 4;
constexpr int kDenseQueries = 32 * kDenseWaves;  // per workgroup
constexpr int kKeyBlock = 64;
constexpr float kDenseFastBound = 60.f;

struct DenseShared {
    char Ks[2][kKeyBlock * 128];  // k rows (the stored q), swizzled 16-byte pieces
    char Vs[2][kKeyBlock * 128];  // v rows, same layout
    float cf[2][kKeyBlock];       // scale*log2(e)/|q_j|, 0 for a zero row
};

template <bool B>
struct Tag {
    static constexpr bool value = B;
};

// Key scale of every row: scale*log2(e)/|q_j| (0 for a zero row, whose key is
// the zero vector).  Eight lanes per row, 16 bytes each.
__global__ __launch_bounds__(256) void dense_prep_kernel(const uint16_t* __restrict__ q,
                                                         float* __restrict__ cf, int64_t rows,
                                                         float scale_log2e) {
    const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 3;
    const int part = threadIdx.x & 7;
    if (row >= rows) return;  // whole 8-lane groups leave
    const u32x4 x = *reinterpret_cast<const u32x4*>(q + row * kHeadDim + part * 8);
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float a = __uint_as_float(x[e] << 16), b = __uint_as_float(x[e] & 0xFFFF0000u);
        ss = fmaf(a, a, fmaf(b, b, ss));
    }
    ss += __shfl_xor(ss, 1);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 4);
    if (part == 0) cf[row] = ss > 0.f ? scale_log2e / sqrtf(ss) : 0.f;
}

template <bool CAUSAL>
__global__ __launch_bounds__(256, 3) void dense_attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v, const float* __restrict__ cf,
    uint16_t* __restrict__ out, float* __restrict__ lse, int L, float scale_log2e, float self_mask) {
    __shared__ __attribute__((aligned(16))) DenseShared S;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = lane & 15, g = lane >> 4;
    const int64_t bh = blockIdx.y;
    const int qb = CAUSAL ? (int)(gridDim.x - 1 - blockIdx.x) : (int)blockIdx.x;
    const int q0 = qb * kDenseQueries;
    const int qw0 = q0 + 32 * wave;  // this wave's first query
    const uint16_t* qh = q + bh * L * kHeadDim;
    const uint16_t* vh = v + bh * L * kHeadDim;
    const float* cfh = cf + bh * L;

    const int n_blocks = (L + kKeyBlock - 1) / kKeyBlock;
    // blocks the workgroup walks, and the last one this wave needs
    const int wg_end = CAUSAL ? (min(q0 + kDenseQueries, L) - 1) / kKeyBlock + 1 : n_blocks;
    const bool active = qw0 < L;
    const int wave_end = !active ? 0 : (CAUSAL ? (min(qw0 + 32, L) - 1) / kKeyBlock + 1 : n_blocks);

    // Query operands: lane holds query qw0 + 16qt + n, dims 32ks + 8g .. +7.
    bf16x8 qop[2][2];
    float bound[2];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        const int row = min(qw0 + 16 * qt + n, L - 1);
        float ss = 0.f;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const u32x4 x = *reinterpret_cast<const u32x4*>(qh + (int64_t)row * kHeadDim + 32 * ks + 8 * g);
            qop[qt][ks] = as_bf16x8(x);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float a = __uint_as_float(x[e] << 16), b = __uint_as_float(x[e] & 0xFFFF0000u);
                ss = fmaf(a, a, fmaf(b, b, ss));
            }
        }
        ss += __shfl_xor(ss, 16);
        ss += __shfl_xor(ss, 32);
        bound[qt] = scale_log2e * sqrtf(ss);
    }
    const bool fast = __ballot(!(bound[0] <= kDenseFastBound && bound[1] <= kDenseFastBound)) == 0;

    // Stage key block kb into buffer b: wave w copies rows 16w .. 16w+15 of k
    // and of v (each lane the piece that belongs at its LDS slot), wave 0 the
    // 64 key scales.  Rows past L repeat row L-1 and are masked out.
    auto stage = [&](int kb, int b) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int row = 16 * wave + 8 * k + (lane >> 3);
            const int key = min(kb * kKeyBlock + row, L - 1);
            const int64_t off = (int64_t)key * kHeadDim + swz(row, lane & 7) * 8;
            copy16_to_lds(qh + off, S.Ks[b] + (16 * wave + 8 * k) * 128);
            copy16_to_lds(vh + off, S.Vs[b] + (16 * wave + 8 * k) * 128);
        }
        if (wave == 0) copy4_to_lds(cfh + min(kb * kKeyBlock + lane, L - 1), &S.cf[b][0]);
    };

    float m[2] = {-__builtin_inff(), -__builtin_inff()};  // running maxima (slow path)
    float lsum[2] = {0.f, 0.f};
    f32x4 oacc[2][4] = {};

    // One key block for both query tiles.  EDGE: the block holds one of the
    // wave's own positions or the sequence end, so keys are tested one by one.
    auto attend = [&](const char* Ks, const char* Vs, const float* cfb, int kb, auto fast_tag,
                      auto edge_tag) {
        constexpr bool FAST = decltype(fast_tag)::value;
        constexpr bool EDGE = decltype(edge_tag)::value;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
            const bf16x8 k0 = as_bf16x8(lds_piece(Ks, 16 * kt + n, g));
            const bf16x8 k1 = as_bf16x8(lds_piece(Ks, 16 * kt + n, 4 + g));
            const f32x4 cfk = *reinterpret_cast<const f32x4*>(cfb + 16 * kt + 4 * g);
            const int key0 = kb * kKeyBlock + 16 * kt + 4 * g;  // this lane's first key
            bf16x4 pk[2];
#pragma unroll
            for (int qt = 0; qt < 2; ++qt) {
                f32x4 acc = mfma16x16x32(k0, qop[qt][0], f32x4{});
                acc = mfma16x16x32(k1, qop[qt][1], acc);
                const int query = qw0 + 16 * qt + n;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc[j] *= cfk[j];
                    if constexpr (EDGE) {
                        const int key = key0 + j;
                        const bool ok = key < L && (CAUSAL ? key < query : key != query);
                        acc[j] = ok ? acc[j] : -__builtin_inff();
                    }
                }
                float off = 0.f;
                if constexpr (!FAST) {  // online maximum over the four lane groups of a query
                    float mt = fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3]));
                    mt = fmaxf(mt, __shfl_xor(mt, 16));
                    mt = fmaxf(mt, __shfl_xor(mt, 32));
                    const float m_new = fmaxf(m[qt], mt);
                    off = m_new > -__builtin_inff() ? m_new : 0.f;
                    const float corr = __builtin_amdgcn_exp2f(m[qt] - off);
                    lsum[qt] *= corr;
#pragma unroll
                    for (int dt = 0; dt < 4; ++dt) oacc[qt][dt] *= corr;
                    m[qt] = m_new;
                }
                uint32_t pw[2];
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) {
                    const float pa = __builtin_amdgcn_exp2f(acc[2 * h2] - off);
                    const float pb = __builtin_amdgcn_exp2f(acc[2 * h2 + 1] - off);
                    pw[h2] = pack_bf16x2(pa, pb);
                    // the row sum takes the bf16 weights that enter P V
                    lsum[qt] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw[h2]), kOnes,
                                                               lsum[qt], false);
                }
                pk[qt] = __builtin_bit_cast(bf16x4, make_uint2(pw[0], pw[1]));
            }
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) {
                const bf16x4 vt = vt_read(Vs + vt_offset(16 * kt, 16 * dt, lane));
#pragma unroll
                for (int qt = 0; qt < 2; ++qt) oacc[qt][dt] = mfma16x16x16(vt, pk[qt], oacc[qt][dt]);
            }
        }
    };

    stage(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int kb = 0; kb < wg_end; ++kb) {
        const int b = kb & 1;
        if (kb + 1 < wg_end) stage(kb + 1, b ^ 1);
        if (kb < wave_end) {
            const int k_lo = kb * kKeyBlock;
            const bool edge = k_lo + kKeyBlock > L || (k_lo + kKeyBlock > qw0 && k_lo < qw0 + 32);
            if (fast) {
                if (edge)
                    attend(S.Ks[b], S.Vs[b], S.cf[b], kb, Tag<true>{}, Tag<true>{});
                else
                    attend(S.Ks[b], S.Vs[b], S.cf[b], kb, Tag<true>{}, Tag<false>{});
            } else {
                if (edge)
                    attend(S.Ks[b], S.Vs[b], S.cf[b], kb, Tag<false>{}, Tag<true>{});
                else
                    attend(S.Ks[b], S.Vs[b], S.cf[b], kb, Tag<false>{}, Tag<false>{});
            }
        }
        __builtin_amdgcn_s_waitcnt(0);  // this wave's copies of block kb+1 have landed
        __syncthreads();                // ... and every wave is done with block kb
    }
    if (!active) return;

    // Lane holds O^T[d = 16dt + 4g + e][query qw0 + 16qt + n].
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        const int query = qw0 + 16 * qt + n;
        float l = lsum[qt];
        l += __shfl_xor(l, 16);
        l += __shfl_xor(l, 32);
        if (query >= L) continue;
        uint16_t* orow = out + (bh * L + query) * kHeadDim;
        if (l > 0.f) {
            const float inv = __builtin_amdgcn_rcpf(l);
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) {
                const uint2 w = make_uint2(pack_bf16x2(oacc[qt][dt][0] * inv, oacc[qt][dt][1] * inv),
                                           pack_bf16x2(oacc[qt][dt][2] * inv, oacc[qt][dt][3] * inv));
                *reinterpret_cast<uint2*>(orow + 16 * dt + 4 * g) = w;
            }
            if (lse && g == 0) lse[bh * L + query] = ((fast ? 0.f : m[qt]) + __log2f(l)) * kLn2;
        } else {
            // the query's only key is itself: output v_i
            const uint16_t* vrow = vh + (int64_t)query * kHeadDim;
#pragma unroll
            for (int dt = 0; dt < 4; ++dt)
                *reinterpret_cast<uint2*>(orow + 16 * dt + 4 * g) =
                    *reinterpret_cast<const uint2*>(vrow + 16 * dt + 4 * g);
            if (lse && g == 0) lse[bh * L + query] = bound[qt] * kLn2 - self_mask;
        }
    }
}

}  // namespace

size_t dense_workspace_bytes(int64_t BH, int L) { return align256((size_t)BH * L * sizeof(float)); }

hipError_t launch_dense_fwd(int64_t BH, int L, bool causal, float scale, float self_mask,
                            const void* q_, const void* v_, void* out_, float* lse, void* workspace,
                            hipStream_t stream) {
    if (BH == 0 || L == 0) return hipSuccess;
    const uint16_t* q = static_cast<const uint16_t*>(q_);
    const uint16_t* v = static_cast<const uint16_t*>(v_);
    uint16_t* out = static_cast<uint16_t*>(out_);
    float* cf = static_cast<float*>(workspace);
    const int64_t rows = BH * L;
    const float scale_log2e = scale * kLog2e;
    dense_prep_kernel<<<(unsigned)((rows * 8 + 255) / 256), 256, 0, stream>>>(q, cf, rows, scale_log2e);
    const dim3 grid((unsigned)((L + kDenseQueries - 1) / kDenseQueries), (unsigned)BH);
    if (causal)
        dense_attn_fwd_kernel<true><<<grid, 256, 0, stream>>>(q, v, cf, out, lse, L, scale_log2e, self_mask);
    else
        dense_attn_fwd_kernel<false><<<grid, 256, 0, stream>>>(q, v, cf, out, lse, L, scale_log2e, self_mask);
    return hipGetLastError();
}

}  // namespace lsh

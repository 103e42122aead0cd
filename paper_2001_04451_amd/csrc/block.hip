// The reversible block around LSH attention (Reformer Sec. 3, "RevNets",
// "Reversible Transformer" and "Chunking"): the layer normalisations inside
// the residual branches and the block's dense products.  The attention
// itself is the library's LSH forward; the block's entry points (block_api.cpp)
// chain these kernels with it.
//
// LayerNorm: one wave per row, the row held in registers, mean and variance
// in fp32 by wave reductions, bf16 output (the products' operand precision).
//
// Products: C = A W^T with A the activations (rows of K bf16 values, or the
// attention's output in its [B, H, L, 64] layout) and W a weight matrix
// [N][K] in bf16, fp32 accumulation on the matrix cores
// (mfma_f32_16x16x32_bf16).  A workgroup of four waves computes a 128 x 128
// tile of C; each wave a 64 x 64 quarter as 4 x 4 products of 16 x 16 with W
// as the first operand, so a lane ends up with four consecutive output
// columns of one row.  A and W tiles of 128 rows x 64 k stream through LDS by
// buffer loads straight into LDS, double-buffered, one barrier per k-tile;
// piece p (16 B) of tile row r sits at slot p ^ (r & 7), so the 16 rows an
// operand load reads hit distinct banks.  Rows past M read as zero (the
// buffer's bound) and are not stored.  Workgroups are numbered so that the N
// tiles of one row tile run on one XCD, which then reads those rows of A from
// memory once.  The epilogue adds the bias and either
//  * adds the product, times a sign, to an fp32 residual (the branch outputs:
//    y = x + F or x = y - F),
//  * applies ReLU and stores bf16 (the feed-forward's hidden layer), or
//  * stores bf16 q or v in the attention's [B, H, L, 64] layout.
#include "attn_common.h"
#include "launch.h"

namespace lsh {
namespace {

// ---------------------------------------------------------------------------
// LayerNorm

constexpr int kLnMaxPairs = 32;  // rows of up to 64 x 2 x 32 = 4096 values

__device__ __forceinline__ float wave_sum(float x) {
    // butterfly: every lane ends with the same (commutative) sums
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

__global__ __launch_bounds__(256) void layer_norm_kernel(const float* __restrict__ x, const float* __restrict__ g,
                                                         const float* __restrict__ b, uint32_t* __restrict__ out,
                                                         int64_t rows, int D, float eps) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;  // uniform per wave
    const int P = D / 128;    // value pairs per lane
    const float2* xr = reinterpret_cast<const float2*>(x + row * D);
    float2 v[kLnMaxPairs];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kLnMaxPairs; ++i)
        if (i < P) {
            v[i] = xr[lane + 64 * i];
            s += v[i].x + v[i].y;
        }
    const float mu = wave_sum(s) / (float)D;
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < kLnMaxPairs; ++i)
        if (i < P) {
            const float dx = v[i].x - mu, dy = v[i].y - mu;
            ss += dx * dx + dy * dy;
        }
    const float rstd = 1.0f / sqrtf(wave_sum(ss) / (float)D + eps);
    const float2* g2 = reinterpret_cast<const float2*>(g);
    const float2* b2 = reinterpret_cast<const float2*>(b);
    uint32_t* orow = out + row * (D / 2);
#pragma unroll
    for (int i = 0; i < kLnMaxPairs; ++i)
        if (i < P) {
            const int c = lane + 64 * i;
            const float2 gg = g2[c], bb = b2[c];
            orow[c] = pack_bf16x2((v[i].x - mu) * rstd * gg.x + bb.x, (v[i].y - mu) * rstd * gg.y + bb.y);
        }
}

// ---------------------------------------------------------------------------
// Products

constexpr int kTile = 128;                 // rows of A and of W per workgroup
constexpr int kBK = 64;                    // k per LDS tile
constexpr uint32_t kTileBytes = kTile * kBK * 2;
constexpr int kGemmThreads = 256;

// Raw buffer (word 3: raw, untyped 32-bit data); loads past num_records read 0.
constexpr int kRawBufferWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_buffer(const void* p, uint64_t bytes) {
    const uint32_t n = bytes >= 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)n, kRawBufferWord3);
}

enum : int { kInRows = 0, kInHeads = 1 };                    // A layout
enum : int { kOutResid = 0, kOutReluBf16 = 1, kOutHeads = 2 };  // epilogue

struct GemmArgs {
    const uint16_t* a;      // [M][K] rows, or [B][H][L][64] (kInHeads: K = 64 H, M = B L)
    const uint16_t* w;      // [N][K]
    int64_t M;
    int N, K;
    int L, H;               // kInHeads / kOutHeads: sequence length and heads
    const float* bias;      // [N] or null
    const float* resid;     // kOutResid: [M][N] fp32 or null (then 0)
    float sign;             // kOutResid: out = resid + sign (A W^T + bias)
    float* out_f32;         // kOutResid: [M][N]
    uint16_t* out_bf16;     // kOutReluBf16: [M][N]; kOutHeads: [B][H][L][64]
};

template <int IN, int OUT>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_bf16_kernel(GemmArgs g) {
    __shared__ __attribute__((aligned(16))) char sa[2][kTileBytes];
    __shared__ __attribute__((aligned(16))) char sw[2][kTileBytes];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // tile of this workgroup: N tiles of one row tile on one XCD when the
    // tile count allows (workgroup b runs on XCD b % 8)
    const int nN = g.N / kTile;
    const int64_t nM = (g.M + kTile - 1) / kTile;
    const int64_t T = nN * nM;
    int64_t t = blockIdx.x;
    if (T % 8 == 0) t = (t % 8) * (T / 8) + t / 8;
    const int64_t m0 = (t / nN) * kTile;
    const int n0 = (int)(t % nN) * kTile;
    const int KT = g.K / kBK;

    // Loads: wave w moves LDS rows 32w .. 32w+31 of both tiles, 8 rows per
    // instruction; lane l fills row 8j + l/8, slot l%8 with piece
    // (l%8) ^ (l/8) of that row (the row's low three bits are l/8).
    const int lr = lane >> 3;
    const uint32_t lp = (uint32_t)((lane & 7) ^ lr);
    const __amdgpu_buffer_rsrc_t ra = raw_buffer(g.a, (uint64_t)g.M * g.K * 2);
    const __amdgpu_buffer_rsrc_t rw = raw_buffer(g.w, (uint64_t)g.N * g.K * 2);
    uint32_t a_off[4], w_off[4];  // byte offsets of the lane's piece at k-tile 0
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = 32 * wave + 8 * j + lr;
        const int64_t m = m0 + r;
        if constexpr (IN == kInRows) {
            a_off[j] = m < g.M ? (uint32_t)((m * g.K + 8 * lp) * 2) : 0xFFFFFFF0u;
        } else {
            const int64_t bb = m / g.L, l = m % g.L;
            a_off[j] = m < g.M ? (uint32_t)(((bb * g.H * g.L + l) * 64 + 8 * lp) * 2) : 0xFFFFFFF0u;
        }
        w_off[j] = (uint32_t)(((int64_t)(n0 + r) * g.K + 8 * lp) * 2);
    }
    // advance per k-tile: 64 values along a row, or one head
    const uint32_t a_step = IN == kInRows ? kBK * 2 : (uint32_t)g.L * 64 * 2;
    auto load_tiles = [&](int kt, int buf) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int chunk = 4 * wave + j;  // 1 KB chunk: rows 8 chunk .. 8 chunk + 7
            const uint32_t ao = a_off[j] == 0xFFFFFFF0u ? 0xFFFFFFF0u : a_off[j] + (uint32_t)kt * a_step;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (__attribute__((address_space(3))) void*)(sa[buf] + 1024 * chunk),
                                                     16, ao, 0, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (__attribute__((address_space(3))) void*)(sw[buf] + 1024 * chunk),
                                                     16, w_off[j] + (uint32_t)kt * (kBK * 2), 0, 0, 0);
        }
    };

    // Operand reads: wave (wm, wn) covers A rows 64 wm .. +63 and W rows
    // 64 wn .. +63; lane l reads row 16 i + l%16 of its quarter, piece
    // 4 ks + l/16 (k-step ks of 32), at slot piece ^ (l & 7).
    const int wm = wave & 1, wn = wave >> 1;
    const uint32_t row_l = (uint32_t)(lane & 15);
    uint32_t op_off[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) op_off[ks] = row_l * 128 + ((((uint32_t)(4 * ks + (lane >> 4))) ^ (lane & 7)) << 4);

    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    load_tiles(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < KT) load_tiles(kt + 1, buf ^ 1);
        const char* A = sa[buf] + wm * 64 * 128;
        const char* Wt = sw[buf] + wn * 64 * 128;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            bf16x8 wf[4], af[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                wf[i] = as_bf16x8(*reinterpret_cast<const u32x4*>(Wt + op_off[ks] + i * 16 * 128));
                af[i] = as_bf16x8(*reinterpret_cast<const u32x4*>(A + op_off[ks] + i * 16 * 128));
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(wf[i], af[j], acc[i][j]);
        }
        __builtin_amdgcn_s_waitcnt(0);  // this wave's copies of the next tiles have landed
        __syncthreads();                // ... and every wave is done with this buffer
    }

    // Epilogue: acc[i][j] holds C[m][n .. n+3] with m = m0 + 64 wm + 16 j +
    // l%16 and n = n0 + 64 wn + 16 i + 4 (l/16).
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t m = m0 + 64 * wm + 16 * j + (lane & 15);
        if (m >= g.M) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int n = n0 + 64 * wn + 16 * i + 4 * (lane >> 4);
            f32x4 c = acc[i][j];
            if (g.bias) {
                const f32x4 bv = *reinterpret_cast<const f32x4*>(g.bias + n);
                c += bv;
            }
            if constexpr (OUT == kOutResid) {
                f32x4 r = g.resid ? *reinterpret_cast<const f32x4*>(g.resid + m * g.N + n) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int e = 0; e < 4; ++e) r[e] = fmaf(g.sign, c[e], r[e]);
                *reinterpret_cast<f32x4*>(g.out_f32 + m * g.N + n) = r;
            } else if constexpr (OUT == kOutReluBf16) {
                const uint2 p = make_uint2(pack_bf16x2(fmaxf(c[0], 0.f), fmaxf(c[1], 0.f)),
                                           pack_bf16x2(fmaxf(c[2], 0.f), fmaxf(c[3], 0.f)));
                *reinterpret_cast<uint2*>(g.out_bf16 + m * g.N + n) = p;
            } else {
                const int64_t bb = m / g.L, l = m % g.L;
                const int h = n >> 6, e = n & 63;
                const uint2 p = make_uint2(pack_bf16x2(c[0], c[1]), pack_bf16x2(c[2], c[3]));
                *reinterpret_cast<uint2*>(g.out_bf16 + ((bb * g.H + h) * g.L + l) * 64 + e) = p;
            }
        }
    }
}

template <int IN, int OUT>
hipError_t launch_gemm(const GemmArgs& g, hipStream_t stream) {
    const int64_t tiles = (int64_t)(g.N / kTile) * ((g.M + kTile - 1) / kTile);
    if (tiles == 0) return hipSuccess;
    gemm_bf16_kernel<IN, OUT><<<(unsigned)tiles, kGemmThreads, 0, stream>>>(g);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_layer_norm(const float* x, const float* g, const float* b, uint16_t* out, int64_t rows, int D,
                             float eps, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    layer_norm_kernel<<<(unsigned)((rows + 3) / 4), 256, 0, stream>>>(x, g, b, reinterpret_cast<uint32_t*>(out),
                                                                      rows, D, eps);
    return hipGetLastError();
}

hipError_t launch_linear(const uint16_t* a, bool a_heads, int L, int H, const uint16_t* w, int64_t M, int N, int K,
                         const float* bias, int out_kind, const float* resid, float sign, float* out_f32,
                         uint16_t* out_bf16, hipStream_t stream) {
    GemmArgs g{a, w, M, N, K, L, H, bias, resid, sign, out_f32, out_bf16};
    if (a_heads) {
        if (out_kind != kLinearResid) return hipErrorInvalidValue;
        return launch_gemm<kInHeads, kOutResid>(g, stream);
    }
    switch (out_kind) {
        case kLinearResid: return launch_gemm<kInRows, kOutResid>(g, stream);
        case kLinearReluBf16: return launch_gemm<kInRows, kOutReluBf16>(g, stream);
        case kLinearHeads: return launch_gemm<kInRows, kOutHeads>(g, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lsh

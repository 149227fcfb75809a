// Stage-sum linear layer on an RRQ package (the prefill / decode product of
// Eq. 20): Y[m][o] = sum over the first K stages t and inputs i of
// X[m][i] (Q_t[o][i] - z_t) s_t, with X bfloat16 [M][cols] and Y binary32
// [M][rows], on gfx950 matrix cores.
//
// Per group g of G inputs and stage t the sum over the group factors as
//   s_t (sum_i x_i Q_i - z_t sum_i x_i),
// and both inner sums run on v_mfma_f32_16x16x32_bf16 with fp32 accumulation:
//   * A operand: 16 tokens x 32 inputs of X (bfloat16, exact);
//   * B operand: 32 inputs x 16 output rows of codes, each code Q encoded as
//     the bfloat16 1 + Q/4 (bits 0x3F80 | Q << 5: the code lands in the top
//     two mantissa bits with one shift, one AND and one OR per pair of
//     codes), so the MFMA yields P = sum x (1 + Q/4) and
//     sum x Q = 4 P - 4 Sx exactly in real arithmetic;
//   * Sx = sum x over the group comes from the same MFMA with a B operand of
//     bfloat16 ones.
// The group's contribution s (4 P - (4 + z) Sx) is added to the lane's fp32
// accumulators with two fused multiply-adds. Every product of the MFMAs is
// exact; fp32 rounding enters only in the accumulations (error bound in the
// tests).
//
// Work split: a workgroup of 8 waves owns 16 output rows; the groups of a
// row are split into 8 contiguous ranges, one per wave; the 8 partial
// results are summed through LDS in wave order (deterministic). Tokens are
// processed 16 at a time. Lane l of a wave: A row / B column l % 16, input
// slice j = l / 16 of each 32-input block. With nb = G / 32 blocks per group,
// block b takes code word b + (j / 2) nb of the row's group (so a lane loads
// its nb words with one load per stage) and, of that word, the element pairs
// (p, p + 8) for p = 4 (j % 2) .. 4 (j % 2) + 3; the A operand holds the
// activations of the same inputs in the same order.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rrq_launch.h"

namespace rrq_detail {
namespace {

using rsrc_t = __amdgpu_buffer_rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr uint32_t kOnePair = 0x3F803F80u;    // two bfloat16 1.0
constexpr uint32_t kCodeMask = 0x00600060u;   // top two mantissa bits of both halves

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

__device__ __forceinline__ f32x4 mfma(const u32x4 &a, const u32x4 &b, const f32x4 &c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// B operand of one block: codes q = 0..3 of the (pre-shifted) word w sit at
// bits 2q and 16 + 2q; register q gets codes q and q + 8 as 1 + code / 4.
__device__ __forceinline__ u32x4 code_operand(uint32_t w)
{
    u32x4 b;
    b[0] = ((w << 5) & kCodeMask) | kOnePair;
    b[1] = ((w << 3) & kCodeMask) | kOnePair;
    b[2] = ((w << 1) & kCodeMask) | kOnePair;
    b[3] = ((w >> 1) & kCodeMask) | kOnePair;
    return b;
}

// A operand of one block from two runs of 4 activations (inputs p0 .. p0 + 3
// and p0 + 8 .. p0 + 11 of a 16-input word): register q = (x[p0 + q],
// x[p0 + 8 + q]).
__device__ __forceinline__ u32x4 act_operand(const u32x2 &run1, const u32x2 &run2)
{
    u32x4 a;
    a[0] = __builtin_amdgcn_perm(run2[0], run1[0], 0x05040100u);
    a[1] = __builtin_amdgcn_perm(run2[0], run1[0], 0x07060302u);
    a[2] = __builtin_amdgcn_perm(run2[1], run1[1], 0x05040100u);
    a[3] = __builtin_amdgcn_perm(run2[1], run1[1], 0x07060302u);
    return a;
}

template <int NB>
__device__ __forceinline__ void load_words(rsrc_t r, uint32_t off, uint32_t (&w)[NB])
{
    if constexpr (NB == 4) {
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
        w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
    } else if constexpr (NB == 2) {
        const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
        w[0] = v[0]; w[1] = v[1];
    } else {
        w[0] = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
    }
}

template <int G, int K>
__global__ __launch_bounds__(kLinearThreads) void linear_kernel(
    const uint32_t *__restrict__ codes, const float *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int64_t n_tokens,
    float *__restrict__ Y)
{
    constexpr int NB = G / 32;          // 32-input blocks per group
    constexpr int WPG = G / 16;         // code words per group and row
    constexpr int NW = kLinearThreads / 64;
    __shared__ f32x4 red[NW][64];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r = lane & 15;            // B column (output row) and A row (token)
    const int j = lane >> 4;            // input slice within a 32-input block
    const int half = j & 1;             // element pairs 4 half .. 4 half + 3
    const int wsel = j >> 1;            // which of the block's two words

    const int64_t o0 = (int64_t)blockIdx.x * 16;
    const uint32_t rows_here = (uint32_t)(rows - o0 < 16 ? rows - o0 : 16);
    const int64_t gpr = cols / G;       // groups per row
    const int64_t wpr = cols / 16;      // code words per row
    // This wave's contiguous range of groups.
    const int64_t per_wave = (gpr + NW - 1) / NW;
    const int64_t g_begin = per_wave * wave < gpr ? per_wave * wave : gpr;
    const int64_t g_end = g_begin + per_wave < gpr ? g_begin + per_wave : gpr;

    // Package resources of this row tile, one per stage (rows past the end
    // read zero codes and zero scales).
    rsrc_t rc[K], rs[K], rz[K];
#pragma unroll
    for (int t = 0; t < K; ++t) {
        rc[t] = make_rsrc(codes + t * plane_words + o0 * wpr, rows_here * (uint32_t)wpr * 4);
        rs[t] = make_rsrc(scales + t * plane_groups + o0 * gpr, rows_here * (uint32_t)gpr * 4);
        rz[t] = make_rsrc(zeros + t * plane_groups + o0 * gpr, rows_here * (uint32_t)gpr * 4);
    }
    const uint32_t row_word_off = (uint32_t)(r * wpr) * 4;
    const uint32_t row_group_off = (uint32_t)(r * gpr) * 4;
    const u32x4 ones = {kOnePair, kOnePair, kOnePair, kOnePair};

    for (int64_t m0 = 0; m0 < n_tokens; m0 += 16) {
        const uint32_t m_here = (uint32_t)(n_tokens - m0 < 16 ? n_tokens - m0 : 16);
        const rsrc_t rx = make_rsrc(X + m0 * cols, m_here * (uint32_t)cols * 2);
        const uint32_t tok_off = (uint32_t)(r * cols) * 2;

        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int64_t g = g_begin; g < g_end; ++g) {
            // Activations of this lane's inputs of group g, all blocks.
            u32x4 a[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const uint32_t in0 = (uint32_t)(g * G) + 16 * (b + wsel * NB) + 4 * half;
                const u32x2 run1 = __builtin_amdgcn_raw_buffer_load_b64(rx, tok_off + in0 * 2, 0, 0);
                const u32x2 run2 = __builtin_amdgcn_raw_buffer_load_b64(rx, tok_off + (in0 + 8) * 2, 0, 0);
                a[b] = act_operand(run1, run2);
            }
            // Package data of group g for every stage.
            uint32_t w[K][NB];
            float s[K], z[K];
#pragma unroll
            for (int t = 0; t < K; ++t) {
                load_words<NB>(rc[t], row_word_off + (uint32_t)(g * WPG + wsel * NB) * 4, w[t]);
                s[t] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs[t], row_group_off + (uint32_t)g * 4, 0, 0));
                z[t] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rz[t], row_group_off + (uint32_t)g * 4, 0, 0));
            }

            f32x4 sx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int b = 0; b < NB; ++b) sx = mfma(a[b], ones, sx);
#pragma unroll
            for (int t = 0; t < K; ++t) {
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int b = 0; b < NB; ++b) p = mfma(a[b], code_operand(w[t][b] >> (8 * half)), p);
                // s (sum x Q - z Sx) = 4 s P - s (4 + z) Sx
                const float s4 = 4.0f * s[t];
                const float scz = s[t] * (4.0f + z[t]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    acc[i] = __builtin_fmaf(s4, p[i], acc[i]);
                    acc[i] = __builtin_fmaf(-scz, sx[i], acc[i]);
                }
            }
        }

        // Sum the waves' partial results in wave order and store: lane l
        // holds tokens m0 + 4 j + i of output row o0 + r.
        red[wave][lane] = acc;
        __syncthreads();
        if (wave == 0) {
            f32x4 y = red[0][lane];
#pragma unroll
            for (int v = 1; v < NW; ++v) {
                const f32x4 q = red[v][lane];
                y[0] += q[0]; y[1] += q[1]; y[2] += q[2]; y[3] += q[3];
            }
            if ((uint32_t)r < rows_here) {
                const rsrc_t ry = make_rsrc(Y + m0 * rows, m_here * (uint32_t)rows * 4);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    __builtin_amdgcn_raw_buffer_store_b32(
                        __float_as_uint(y[i]), ry, (uint32_t)((4 * j + i) * rows + o0 + r) * 4, 0, 0);
            }
        }
        __syncthreads();   // red is reused by the next token tile
    }
}

template <typename... Args>
hipError_t launch(void (*kernel)(Args...), int grid, int block, hipStream_t stream,
                  Args... args)
{
    void *argv[] = {static_cast<void *>(&args)...};
    return hipLaunchKernel(reinterpret_cast<const void *>(kernel), dim3(grid), dim3(block),
                           argv, 0, stream);
}

template <int G>
hipError_t launch_linear_g(const uint32_t *codes, const float *scales, const float *zeros,
                           int64_t rows, int64_t cols, int S, int k, const uint16_t *X,
                           int64_t n_tokens, float *Y, hipStream_t stream)
{
    const int64_t plane_words = rows * cols / 16;
    const int64_t plane_groups = rows * cols / G;
    const int grid = (int)((rows + 15) / 16);
    (void)S;
    switch (k) {
    case 1: return launch(linear_kernel<G, 1>, grid, kLinearThreads, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y);
    case 2: return launch(linear_kernel<G, 2>, grid, kLinearThreads, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y);
    case 3: return launch(linear_kernel<G, 3>, grid, kLinearThreads, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y);
    case 4: return launch(linear_kernel<G, 4>, grid, kLinearThreads, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_linear(const uint32_t *codes, const float *scales, const float *zeros,
                         int64_t rows, int64_t cols, int G, int S, int k, const uint16_t *X,
                         int64_t n_tokens, float *Y, hipStream_t stream)
{
    switch (G) {
    case 32: return launch_linear_g<32>(codes, scales, zeros, rows, cols, S, k, X, n_tokens, Y, stream);
    case 64: return launch_linear_g<64>(codes, scales, zeros, rows, cols, S, k, X, n_tokens, Y, stream);
    case 128: return launch_linear_g<128>(codes, scales, zeros, rows, cols, S, k, X, n_tokens, Y, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace rrq_detail

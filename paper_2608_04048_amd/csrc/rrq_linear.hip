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
// row are split into 8 contiguous ranges, one per wave, each wave keeping
// the loads of two groups in flight; the partial results are summed through
// LDS in wave order (deterministic). Tokens are processed 16 at a time. The
// loads are shaped for the vector-memory address path, which bounds this
// kernel before HBM does: no lane loads a code word another lane of its row
// loads (G = 128, 64), activations come in 16-byte loads and only for live
// tokens, scales and zero-points for two groups per load.

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

// Lane layout of one group (G inputs of 16 output rows, nb = G / 32 MFMA
// blocks of 32 inputs). Lane l: row / token r = l % 16, slice j = l / 16.
//   G = 128: lane j owns code words 2j, 2j + 1 of the row's group (one 8-byte
//            load per stage) and the activations of their 32 inputs; block b
//            takes word 2j + b / 2, element pairs of half b % 2.
//   G = 64:  lane j owns word j; block b takes its half b.
//   G = 32:  lanes j = 2w, 2w + 1 share word w; block 0 takes half j % 2.
// Half h of a word holds the element pairs (p, p + 8), p = 4h .. 4h + 3.
template <int G>
struct LaneMap {
    static constexpr int NB = G / 32;
    static constexpr int WL = G == 128 ? 2 : 1;        // words loaded per lane
    static constexpr int XD = G == 32 ? 4 : 8 * WL;    // activation dwords per lane
};

template <int G, int K>
struct GroupLoads {
    uint32_t w[K][LaneMap<G>::WL];        // code words, per stage
    uint32_t x[LaneMap<G>::XD];           // activations (bfloat16 pairs)
};

// A group at or past g_end (the next wave's, or past the row) is not fetched:
// its offsets are moved 2^31 bytes up, past every resource's size (all are
// below 2^28 bytes), so the loads return zeros without touching memory.
// Token lanes past the tile's last token skip their activation loads.
template <int G, int K>
__device__ __forceinline__ void load_group(GroupLoads<G, K> &d, int64_t g, int64_t g_end,
                                           rsrc_t rx, uint32_t tok_off, bool tok_live,
                                           const rsrc_t (&rc)[K], uint32_t row_word_off,
                                           int j)
{
    constexpr int WPG = G / 16;
    const uint32_t skip = g < g_end ? 0u : 0x80000000u;
    // first word of this lane within the group, and its first input
    const int w0 = G == 128 ? 2 * j : G == 64 ? j : (j >> 1);
    const uint32_t word_off = skip + row_word_off + (uint32_t)(g * WPG + w0) * 4;
#pragma unroll
    for (int t = 0; t < K; ++t) {
        if constexpr (G == 128) {
            const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rc[t], word_off, 0, 0);
            d.w[t][0] = v[0];
            d.w[t][1] = v[1];
        } else {
            d.w[t][0] = __builtin_amdgcn_raw_buffer_load_b32(rc[t], word_off, 0, 0);
        }
    }
    const uint32_t in0 = (uint32_t)(g * G) + 16 * w0;
    const uint32_t xoff = skip + tok_off + in0 * 2;
#pragma unroll
    for (int i = 0; i < LaneMap<G>::XD; ++i) d.x[i] = 0u;
    if (tok_live) {
        if constexpr (G == 32) {
            // only this lane's half: inputs 4h .. 4h + 3 and 8 + 4h .. 8 + 4h + 3
            const uint32_t h = (uint32_t)(j & 1);
            const u32x2 a = __builtin_amdgcn_raw_buffer_load_b64(rx, xoff + 8 * h, 0, 0);
            const u32x2 b = __builtin_amdgcn_raw_buffer_load_b64(rx, xoff + 16 + 8 * h, 0, 0);
            d.x[0] = a[0]; d.x[1] = a[1]; d.x[2] = b[0]; d.x[3] = b[1];
        } else {
#pragma unroll
            for (int q = 0; q < LaneMap<G>::XD / 4; ++q) {
                const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rx, xoff + 16 * q, 0, 0);
                d.x[4 * q] = v[0]; d.x[4 * q + 1] = v[1]; d.x[4 * q + 2] = v[2]; d.x[4 * q + 3] = v[3];
            }
        }
    }
}

// Package stage format (values of the C ABI's enums).
constexpr int kZpSymmetric = 2;
constexpr int kScaleF32 = 0, kScaleF16 = 1;

// Scales and zero-points of groups g, g + 1, as binary32 (one load each per
// stage): 16-bit scales are widened, symmetric stages have z = 2. gi is the
// group's index within the row tile's plane segment.
template <int K>
__device__ __forceinline__ void load_sz(u32x2 (&s)[K], u32x2 (&z)[K], int64_t g, int64_t g_end,
                                        const rsrc_t (&rs)[K], const rsrc_t (&rz)[K],
                                        uint32_t row_group, int scale_type, bool sym)
{
    const uint32_t skip = g < g_end ? 0u : 0x80000000u;
    const uint32_t gi = row_group + (uint32_t)g;     // group index within the row tile
#pragma unroll
    for (int t = 0; t < K; ++t) {
        if (scale_type == kScaleF32) {
            s[t] = __builtin_amdgcn_raw_buffer_load_b64(rs[t], skip + gi * 4, 0, 0);
        } else {
            // two 16-bit scales (2-byte aligned: a row may start at an odd group)
            const uint16_t b0 = __builtin_amdgcn_raw_buffer_load_b16(rs[t], skip + gi * 2, 0, 0);
            const uint16_t b1 = __builtin_amdgcn_raw_buffer_load_b16(rs[t], skip + gi * 2 + 2, 0, 0);
            if (scale_type == kScaleF16) {
                s[t][0] = __float_as_uint((float)__builtin_bit_cast(_Float16, b0));
                s[t][1] = __float_as_uint((float)__builtin_bit_cast(_Float16, b1));
            } else {
                s[t][0] = (uint32_t)b0 << 16;
                s[t][1] = (uint32_t)b1 << 16;
            }
        }
        if (sym) {
            z[t][0] = z[t][1] = __float_as_uint(2.0f);
        } else {
            z[t] = __builtin_amdgcn_raw_buffer_load_b64(rz[t], skip + gi * 4, 0, 0);
        }
    }
}

// One group's contribution to the lane's 4 outputs: Sx, then per stage P and
// acc += 4 s P - s (4 + z) Sx.
template <int G, int K>
__device__ __forceinline__ void compute_group(const GroupLoads<G, K> &d, const float (&s)[K],
                                              const float (&z)[K], int j, f32x4 &acc)
{
    constexpr int NB = G / 32;
    const u32x4 ones = {kOnePair, kOnePair, kOnePair, kOnePair};
    u32x4 a[NB];
    if constexpr (G == 32) {
        a[0] = act_operand((u32x2){d.x[0], d.x[1]}, (u32x2){d.x[2], d.x[3]});
    } else {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            // word b / 2 of the lane (G = 128) or its only word (G = 64), half b % 2
            const int base = (G == 128 ? 8 * (b >> 1) : 0) + 2 * (b & 1);
            a[b] = act_operand((u32x2){d.x[base], d.x[base + 1]},
                               (u32x2){d.x[base + 4], d.x[base + 5]});
        }
    }
    f32x4 sx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < NB; ++b) sx = mfma(a[b], ones, sx);
#pragma unroll
    for (int t = 0; t < K; ++t) {
        f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            uint32_t word;
            int h;
            if constexpr (G == 128) { word = d.w[t][b >> 1]; h = b & 1; }
            else if constexpr (G == 64) { word = d.w[t][0]; h = b; }
            else { word = d.w[t][0]; h = j & 1; }
            p = mfma(a[b], code_operand(h ? word >> 8 : word), p);
        }
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

template <int G, int K>
__global__ __launch_bounds__(kLinearThreads) void linear_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int64_t n_tokens,
    float *__restrict__ Y, int zero_point, int scale_type)
{
    constexpr int NW = kLinearThreads / 64;
    const bool sym = zero_point == kZpSymmetric;
    const uint32_t sbytes = scale_type == kScaleF32 ? 4 : 2;
    __shared__ f32x4 red[NW][64];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r = lane & 15;            // B column (output row) and A row (token)
    const int j = lane >> 4;            // input slice

    const int64_t o0 = (int64_t)blockIdx.x * 16;
    const uint32_t rows_here = (uint32_t)(rows - o0 < 16 ? rows - o0 : 16);
    const int64_t gpr = cols / G;       // groups per row
    const int64_t wpr = cols / 16;      // code words per row
    // This wave's contiguous range of groups (an even count, so that scales
    // and zero-points come in pairs of groups).
    const int64_t per_wave = ((gpr + NW - 1) / NW + 1) & ~int64_t(1);
    const int64_t g_begin = per_wave * wave < gpr ? per_wave * wave : gpr;
    const int64_t g_end = g_begin + per_wave < gpr ? g_begin + per_wave : gpr;

    // Package resources of this row tile, one per stage (rows past the end
    // read zero codes and zero scales).
    rsrc_t rc[K], rs[K], rz[K];
#pragma unroll
    for (int t = 0; t < K; ++t) {
        rc[t] = make_rsrc(codes + t * plane_words + o0 * wpr, rows_here * (uint32_t)wpr * 4);
        rs[t] = make_rsrc(scales + (t * plane_groups + o0 * gpr) * sbytes,
                          rows_here * (uint32_t)gpr * sbytes);
        rz[t] = make_rsrc(zeros + t * plane_groups + o0 * gpr, rows_here * (uint32_t)gpr * 4);
    }
    const uint32_t row_word_off = (uint32_t)(r * wpr) * 4;
    const uint32_t row_group = (uint32_t)(r * gpr);

    for (int64_t m0 = 0; m0 < n_tokens; m0 += 16) {
        const uint32_t m_here = (uint32_t)(n_tokens - m0 < 16 ? n_tokens - m0 : 16);
        const rsrc_t rx = make_rsrc(X + m0 * cols, m_here * (uint32_t)cols * 2);
        const uint32_t tok_off = (uint32_t)(r * cols) * 2;
        const bool tok_live = (uint32_t)r < m_here;

        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        // Groups in pairs; the loads of the next group are issued before the
        // current one is computed.
        GroupLoads<G, K> cur, nxt;
        u32x2 s2[K], z2[K];
        load_group<G, K>(cur, g_begin, g_end, rx, tok_off, tok_live, rc, row_word_off, j);
        load_sz<K>(s2, z2, g_begin, g_end, rs, rz, row_group, scale_type, sym);
        for (int64_t g = g_begin; g < g_end; g += 2) {
            float s[K], z[K];
            load_group<G, K>(nxt, g + 1, g_end, rx, tok_off, tok_live, rc, row_word_off, j);
#pragma unroll
            for (int t = 0; t < K; ++t) { s[t] = __uint_as_float(s2[t][0]); z[t] = __uint_as_float(z2[t][0]); }
            compute_group<G, K>(cur, s, z, j, acc);
            if (g + 1 >= g_end) break;
#pragma unroll
            for (int t = 0; t < K; ++t) { s[t] = __uint_as_float(s2[t][1]); z[t] = __uint_as_float(z2[t][1]); }
            load_group<G, K>(cur, g + 2, g_end, rx, tok_off, tok_live, rc, row_word_off, j);
            load_sz<K>(s2, z2, g + 2, g_end, rs, rz, row_group, scale_type, sym);
            compute_group<G, K>(nxt, s, z, j, acc);
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
hipError_t launch_linear_g(const uint32_t *codes, const char *scales, const float *zeros,
                           int64_t rows, int64_t cols, int S, int k, int zp, int sdt,
                           const uint16_t *X, int64_t n_tokens, float *Y, hipStream_t stream)
{
    const int64_t plane_words = rows * cols / 16;
    const int64_t plane_groups = rows * cols / G;
    const int grid = (int)((rows + 15) / 16);
    (void)S;
    switch (k) {
    case 1: return launch(linear_kernel<G, 1>, grid, kLinearThreads, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y, zp, sdt);
    case 2: return launch(linear_kernel<G, 2>, grid, kLinearThreads, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y, zp, sdt);
    case 3: return launch(linear_kernel<G, 3>, grid, kLinearThreads, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y, zp, sdt);
    case 4: return launch(linear_kernel<G, 4>, grid, kLinearThreads, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y, zp, sdt);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_linear(const uint32_t *codes, const void *scales, const float *zeros,
                         int64_t rows, int64_t cols, int G, int S, int k, int zero_point,
                         int scale_type, const uint16_t *X, int64_t n_tokens, float *Y,
                         hipStream_t stream)
{
    const char *sc = static_cast<const char *>(scales);
    switch (G) {
    case 32: return launch_linear_g<32>(codes, sc, zeros, rows, cols, S, k, zero_point, scale_type, X, n_tokens, Y, stream);
    case 64: return launch_linear_g<64>(codes, sc, zeros, rows, cols, S, k, zero_point, scale_type, X, n_tokens, Y, stream);
    case 128: return launch_linear_g<128>(codes, sc, zeros, rows, cols, S, k, zero_point, scale_type, X, n_tokens, Y, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace rrq_detail

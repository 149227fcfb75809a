// Prefill form of the stage-sum linear layer (Eq. 20) for many tokens and
// groups of 128: Y[m][o] = sum over stages t < K and groups g of
// s_t,o,g (sum_i x_m,i Q_t,o,i - z_t,o,g sum_i x_m,i), the product the general
// kernel of rrq_linear.hip computes 16 tokens at a time, organised here as a
// matrix-core product that reuses every operand it builds.
//
// Per group and stage the inner sums run on v_mfma_f32_16x16x32_bf16 with the
// general kernel's operand layouts: A = 16 tokens x 32 inputs of X, B = 32
// inputs x 16 output rows of codes, each code the bfloat16 4 + Q, so that
// P = sum x (4 + Q) and Sx = sum x (the same MFMA with a ones operand) give
// sum x Q = P - 4 Sx. Each output accumulates, per group, sum over stages of
// s P then - (sum over stages of s (4 + z)) Sx.
//
// Work: a workgroup of 4 waves owns a tile of 64 tokens x 64 output rows;
// wave w owns rows 16 w .. 16 w + 15 of it for all 64 tokens, so a B operand
// (one stage of one group of its 16 rows) feeds 4 MFMAs, and the A operands
// of a group (its 64 tokens) are built once and serve every stage. The
// waves walk the groups of a row together: a group's activations (64 tokens
// x 256 bytes) are staged once in LDS for all 4 waves, each wave stages its
// own rows' codes, scales and zero-points, all by LDS-DMA loads into a ring
// of 3 buffers (2 groups in flight while one is computed), with one barrier
// per group.
//
// Accumulation order: each output is accumulated over 4 contiguous quarters
// of the groups (quarter length: the groups per wave of the general kernel's
// 16-token tile, 4 waves, 2-group chunks), starting from 0 each, and the
// quarters are summed in order, ((Q0 + Q1) + Q2) + Q3: the same operations in
// the same order as the general kernel, so the results are identical to its
// and the error bound in rrq.h holds unchanged.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rrq_code_operands.h"
#include "rrq_dma.h"
#include "rrq_launch.h"

namespace rrq_detail {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kWaves = 4;                      // waves per workgroup, 16 rows each
constexpr int kTokens = 64;                    // tokens per workgroup tile
constexpr int kRows = 16 * kWaves;             // output rows per workgroup tile
constexpr int kBuffers = 3;                    // group ring depth
constexpr uint32_t kOnePair = 0x3F803F80u;     // two bfloat16 1.0
constexpr uint32_t kFourPair = 0x40804080u;    // two bfloat16 4.0: code operands 4 + Q
constexpr uint32_t kCodeMask = 0x00600060u;    // top two mantissa bits of both halves
constexpr int kZpSymmetric = 2;
constexpr int kScaleF32 = 0, kScaleF16 = 1;

__device__ __forceinline__ f32x4 mfma(const u32x4 &a, const u32x4 &b, const f32x4 &c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// One ring buffer (one group): the activations of the tile's 64 tokens (16
// slots of 16 bytes per token, slot p of token m holding piece p ^ (m % 16)
// of its 256 bytes, so that the 16 tokens an MFMA reads hit different LDS
// banks), then per wave its 16 rows' codes (stage t at 1024 (t / 2) +
// 512 (t % 2), row-major 16 x 32 bytes), scales and zero-points (32-bit
// words, stage t of row r at 4 (16 t + r)).
template <int K>
struct GroupBuf {
    static constexpr int X_BYTES = kTokens * 256;
    static constexpr int X_DMA = X_BYTES / 1024 / kWaves;   // 1 KiB loads per wave
    static constexpr int CODE_DMA = (K + 1) / 2;            // two stages per load
    static constexpr int SCALES = CODE_DMA * 1024;          // within a wave's part
    static constexpr int ZEROS = SCALES + 256;
    static constexpr int WAVE_BYTES = ZEROS + 256;
    static constexpr int BYTES = X_BYTES + kWaves * WAVE_BYTES;
    static constexpr int DMA = X_DMA + CODE_DMA + 2;        // loads per wave per group
};

// A operands of one 16-token tile for the lane (token n of the tile, k-slice
// j) from its inputs 32 j .. 32 j + 31 of the group, four runs of 8: block b
// = 16-input run 2 j + b / 2, half b % 2, register v = (x[v'], x[v' + 8]).
__device__ __forceinline__ void act_operands(const u32x4 (&run)[4], u32x4 (&a)[4])
{
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        const u32x4 &lo = run[2 * (b >> 1)], &hi = run[2 * (b >> 1) + 1];
        const int h = 2 * (b & 1);
        a[b][0] = __builtin_amdgcn_perm(hi[h], lo[h], 0x05040100u);
        a[b][1] = __builtin_amdgcn_perm(hi[h], lo[h], 0x07060302u);
        a[b][2] = __builtin_amdgcn_perm(hi[h + 1], lo[h + 1], 0x05040100u);
        a[b][3] = __builtin_amdgcn_perm(hi[h + 1], lo[h + 1], 0x07060302u);
    }
}

template <int K, bool DEF, bool MFMA_PRIO>
__global__ __launch_bounds__(64 * kWaves) void prefill_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int64_t n_tokens,
    float *__restrict__ Y, int zero_point, int scale_type, int row_tiles)
{
    using B = GroupBuf<K>;
    __shared__ __attribute__((aligned(16))) char buf[kBuffers][B::BYTES];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;            // A row (token of a 16-token tile) and B column (row)
    const int j = lane >> 4;            // k-slice
    const bool sym = zero_point == kZpSymmetric;
    uint32_t mask, one;
    asm volatile("s_mov_b32 %0, %1" : "=s"(mask) : "n"(kCodeMask));
    asm volatile("v_mov_b32 %0, %1" : "=v"(one) : "n"(kOnePair));
    uint32_t four;
    asm volatile("v_mov_b32 %0, %1" : "=v"(four) : "n"(kFourPair));

    // Tiles: consecutive workgroups share the token tile (its activations
    // stay in L2 while the row tiles stream their codes).
    const int64_t m0 = (int64_t)(blockIdx.x / row_tiles) * kTokens;
    const int64_t o0 = (int64_t)(blockIdx.x % row_tiles) * kRows + 16 * wave;
    const uint32_t tokens_here = (uint32_t)(n_tokens - m0 < kTokens ? n_tokens - m0 : kTokens);
    const int64_t rem = rows - o0;
    const uint32_t rows_here = rem <= 0 ? 0u : (uint32_t)(rem < 16 ? rem : 16);
    const uint32_t gpr = (uint32_t)(cols / 128);        // groups per row
    const uint32_t row_bytes = (uint32_t)(cols / 4);
    const uint32_t x_row = (uint32_t)cols * 2;
    const uint32_t sbytes = scale_type == kScaleF32 ? 4 : 2;
    const uint32_t code_plane = (uint32_t)plane_words * 4;
    const uint32_t scale_plane = (uint32_t)plane_groups * sbytes;
    const uint32_t zero_plane = (uint32_t)plane_groups * 4;
    const int64_t o_first = rows_here ? o0 : 0;         // rows past the end read nothing
    const u32x4 dx = make_desc(X + m0 * cols, tokens_here * x_row);
    const u32x4 dc = make_desc(codes + o_first * (cols / 16),
                               rows_here ? (K - 1) * code_plane + rows_here * row_bytes : 0u);
    const u32x4 ds = make_desc(scales + o_first * gpr * sbytes,
                               rows_here ? (K - 1) * scale_plane + rows_here * gpr * sbytes : 0u);
    const u32x4 dz = make_desc(sym ? nullptr : zeros + o_first * gpr,
                               sym || !rows_here ? 0u : (K - 1) * zero_plane + rows_here * gpr * 4);

    // DMA lane offsets. Activations: this wave's X_DMA loads fill slots
    // 64 (X_DMA wave + i) + lane, slot s -> token s / 16, piece
    // (s % 16) ^ (token % 16); tokens past the tile read nothing.
    uint32_t dma_x[B::X_DMA];
#pragma unroll
    for (int i = 0; i < B::X_DMA; ++i) {
        const uint32_t s = (uint32_t)((B::X_DMA * wave + i) * 64 + lane);
        const uint32_t tok = s >> 4, pc = (s & 15) ^ (tok & 15);
        dma_x[i] = (tok < tokens_here ? 0u : kSkip) + tok * x_row + 16 * pc;
    }
    // Codes: lane l fills bytes 16 l of a 1 KiB load: stage 2 i + l / 32,
    // row (l % 32) / 2, bytes 16 (l % 2) .. + 15 of the row's 32 bytes of the
    // group (a stage past K - 1 reads past the descriptor).
    const uint32_t dma_code = (uint32_t)((lane & 31) >> 1) * row_bytes + 16 * (uint32_t)(lane & 1) +
                              (uint32_t)(lane >> 5) * code_plane;
    // Scales and zero-points: lane l -> stage l / 16, row l % 16; stages past
    // K - 1 read nothing.
    const uint32_t pst = (uint32_t)lane >> 4;
    const uint32_t dma_scale = pst < (uint32_t)K ? (uint32_t)n * gpr * sbytes + pst * scale_plane : kSkip;
    const uint32_t dma_zero = pst < (uint32_t)K ? (uint32_t)n * gpr * 4 + pst * zero_plane : kSkip;

    const uint32_t lds0 = lds_address(&buf[0][0]);
    auto issue = [&](uint32_t g, int b) {
        const uint32_t lds = lds0 + (uint32_t)b * B::BYTES;
#pragma unroll
        for (int i = 0; i < B::X_DMA; ++i)
            dma_x4(dx, g * 256, lds + (uint32_t)(B::X_DMA * wave + i) * 1024, dma_x[i]);
        const uint32_t lw = lds + B::X_BYTES + (uint32_t)wave * B::WAVE_BYTES;
#pragma unroll
        for (int i = 0; i < B::CODE_DMA; ++i)
            dma_x4(dc, g * 32 + 2u * i * code_plane, lw + 1024u * i, dma_code);
        if (DEF || scale_type == kScaleF32)
            dma_dword(ds, g * 4, lw + B::SCALES, dma_scale);
        else
            dma_ushort(ds, g * 2, lw + B::SCALES, dma_scale);
        dma_dword(dz, g * 4, lw + B::ZEROS, dma_zero);
    };

    // Quarter length as in the general kernel (4 waves, 2-group chunks).
    const uint32_t per_q = (((gpr + 3) / 4 + 1) / 2) * 2;
    const u32x4 ones = {one, one, one, one};
    // MFMA_PRIO (2 to 4 stages, long token runs): the stage products of a
    // group (its MFMA stretch) are issued at a raised wave priority, so that
    // the matrix core keeps being fed while the other wave of the SIMD builds
    // operands (measured 4-9% faster from 1024 tokens; not for short runs).

    f32x4 run[4], cur[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) cur[tt] = (f32x4){0.f, 0.f, 0.f, 0.f};
    int quarter = 0;

    issue(0, 0);
    if (gpr > 1) issue(1, 1);
    for (uint32_t g = 0; g < gpr; ++g) {
        // this wave's loads of group g have landed (group g + 1's may not),
        // and after the barrier every wave's have: the buffer of group
        // g - 1 is free again
        if (g + 1 < gpr) wait_vm<B::DMA>(); else wait_vm<0>();
        __syncthreads();
        if (g + 2 < gpr) issue(g + 2, (int)((g + 2) % kBuffers));
        const char *lb = &buf[g % kBuffers][0];
        const char *lw = lb + B::X_BYTES + wave * B::WAVE_BYTES;

        // per-stage s and c = sum over stages of s (4 + z) for the lane's row
        float s4[K], c = 0.0f;
#pragma unroll
        for (int t = 0; t < K; ++t) {
            const uint32_t sw = *reinterpret_cast<const uint32_t *>(lw + B::SCALES + 4 * (16 * t + n));
            const uint32_t zw = *reinterpret_cast<const uint32_t *>(lw + B::ZEROS + 4 * (16 * t + n));
            float s, z;
            if constexpr (DEF) {
                s = __uint_as_float(sw);
                z = __uint_as_float(zw);
            } else {
                s = scale_type == kScaleF32 ? __uint_as_float(sw)
                    : scale_type == kScaleF16
                        ? (float)__builtin_bit_cast(_Float16, (uint16_t)(sw & 0xFFFFu))
                        : __uint_as_float(sw << 16);
                z = sym ? 2.0f : __uint_as_float(zw);
            }
            s4[t] = s;
            c = __builtin_fmaf(s, 4.0f + z, c);
        }
        // A operands and group sums of the 4 token tiles
        u32x4 a[4][4];
        f32x4 sx[4];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) {
            const char *xt = lb + (16 * tt + n) * 256;
            u32x4 runs[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                runs[i] = *reinterpret_cast<const u32x4 *>(xt + 16 * ((4 * j + i) ^ n));
            act_operands(runs, a[tt]);
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int b = 0; b < 4; ++b) acc = mfma(a[tt][b], ones, acc);
            sx[tt] = acc;
        }
        if constexpr (MFMA_PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int t = 0; t < K; ++t) {
            const u32x2 w = *reinterpret_cast<const u32x2 *>(
                lw + 1024 * (t >> 1) + 512 * (t & 1) + n * 32 + 8 * j);
            u32x4 bop[2][2];
            code_operands_pair(w[0], w[1], mask, four, bop);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int b = 0; b < 4; ++b) p = mfma(a[tt][b], bop[b >> 1][b & 1], p);
#pragma unroll
                for (int i = 0; i < 4; ++i) cur[tt][i] = __builtin_fmaf(s4[t], p[i], cur[tt][i]);
            }
        }
        if constexpr (MFMA_PRIO) __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int i = 0; i < 4; ++i) cur[tt][i] = __builtin_fmaf(-c, sx[tt][i], cur[tt][i]);
        // end of a quarter: fold it into the running sum
        if ((g + 1) % per_q == 0 || g + 1 == gpr) {
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                if (quarter == 0) {
                    run[tt] = cur[tt];
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) run[tt][i] = run[tt][i] + cur[tt][i];
                }
                cur[tt] = (f32x4){0.f, 0.f, 0.f, 0.f};
            }
            ++quarter;
        }
    }
    // quarters with no groups add zeros, as the general kernel's idle waves do
    for (; quarter < 4; ++quarter)
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int i = 0; i < 4; ++i) run[tt][i] = run[tt][i] + 0.0f;

    // lane: tokens m0 + 16 tt + 4 j + i of output row o0 + n
    if ((uint32_t)n < rows_here) {
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t tk = (uint32_t)(16 * tt + 4 * j + i);
                if (tk < tokens_here) Y[(m0 + tk) * rows + o0 + n] = run[tt][i];
            }
    }
}

template <typename... Args>
hipError_t launch(void (*kernel)(Args...), int grid, int block, hipStream_t stream, Args... args)
{
    void *argv[] = {static_cast<void *>(&args)...};
    return hipLaunchKernel(reinterpret_cast<const void *>(kernel), dim3(grid), dim3(block),
                           argv, 0, stream);
}

// From this many tokens the 2-4 stage kernels issue their MFMA stretches at
// a raised wave priority (A/B: faster from 1024 tokens, slower at 256).
constexpr int64_t kPrefillPrioTokens = 1024;

template <bool DEF>
hipError_t launch_d(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int64_t n_tokens,
                    float *Y, hipStream_t stream)
{
    const int row_tiles = (int)((rows + kRows - 1) / kRows);
    const int64_t tiles = (int64_t)row_tiles * ((n_tokens + kTokens - 1) / kTokens);
    const int grid = (int)tiles;
    const int64_t pw = rows * cols / 16, pg = rows * cols / 128;
    const bool prio = n_tokens >= kPrefillPrioTokens;
    switch (k) {
    case 1: return launch(prefill_kernel<1, DEF, false>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles);
    case 2: return prio ? launch(prefill_kernel<2, DEF, true>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles)
                        : launch(prefill_kernel<2, DEF, false>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles);
    case 3: return prio ? launch(prefill_kernel<3, DEF, true>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles)
                        : launch(prefill_kernel<3, DEF, false>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles);
    case 4: return prio ? launch(prefill_kernel<4, DEF, true>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles)
                        : launch(prefill_kernel<4, DEF, false>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool linear_prefill_fits(int64_t rows, int64_t cols, int G, int64_t n_tokens)
{
    // 64-token tiles: the activation descriptor spans 64 rows of X (under
    // 2^31 bytes), and the grid (row tiles x token tiles) fits an int.
    const int64_t tiles = ((rows + kRows - 1) / kRows) * ((n_tokens + kTokens - 1) / kTokens);
    return G == 128 && n_tokens >= kPrefillMinTokens && cols <= 65536 && tiles < (1ll << 31);
}

hipError_t launch_linear_prefill(const uint32_t *codes, const void *scales, const float *zeros,
                                 int64_t rows, int64_t cols, int k, int zero_point,
                                 int scale_type, const uint16_t *X, int64_t n_tokens, float *Y,
                                 hipStream_t stream)
{
    const char *sc = static_cast<const char *>(scales);
    const bool def = scale_type == kScaleF32 && zero_point != kZpSymmetric;
    return def ? launch_d<true>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X,
                                n_tokens, Y, stream)
               : launch_d<false>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X,
                                 n_tokens, Y, stream);
}

}  // namespace rrq_detail

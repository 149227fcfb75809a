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
// Work: a workgroup of WV waves owns a tile of 16 T tokens x 16 NR WV
// output rows (8 waves and 128 x 128 when that still fills the GPU, else 4
// waves and 64 x 64; at one stage 8 waves of 32 rows, 256 x 128); wave w
// owns rows 16 NR w .. 16 NR (w + 1) - 1 of it for all 16 T tokens, so a B
// operand (one stage of one group of 16 rows) feeds T MFMAs and an A
// operand (16 tokens of a group) NR K of them, one per row tile and stage.
// The waves walk the groups of a row together. A group's
// activations (16 T tokens x 256 bytes) are staged once in LDS for all the
// waves, each wave staging its share of T / WV 16-token tiles, and its own
// rows' codes, scales and zero-points, all by LDS-DMA loads into a ring of
// 3 buffers (2 groups in flight while one is computed), with one barrier
// per group. Once its loads of a group have landed, a wave prepares its
// share of the activations for every wave: it rewrites its tiles in place
// as A operands (the order the code operands need) and stores their sums Sx
// in LDS, so that each operand is built and each sum is taken once per
// workgroup instead of once per wave. A wave prepares group g + 1 when it
// is done computing group g, and the barrier that opens group g + 1
// publishes it.
//
// Accumulation order: each output is accumulated over 4 contiguous quarters
// of the groups (quarter length: the groups per wave of the general kernel's
// 16-token tile, 4 waves, 2-group chunks), starting from 0 each, and the
// quarters are summed in order, ((Q0 + Q1) + Q2) + Q3 (taken as
// (((+0 + Q0) + Q1) + Q2) + Q3, the same value: a quarter sum is never -0):
// the same operations in the same order as the general kernel, so the
// results are identical to its and the error bound in rrq.h holds
// unchanged.

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

// One ring buffer (one group) of a tile of 16 T tokens and WV waves of
// 16 NR rows each: the activations (16 slots of 16 bytes per token, slot p
// of token m holding piece p ^ (m % 16) of its 256 bytes, so that the 16
// tokens an MFMA reads hit different LDS banks; once prepared, the same
// slots hold the token's A operands), the tokens' sums Sx (one float each),
// then per wave its rows' codes, scales and zero-points. With 16 rows per
// wave (NR = 1) the codes of stage t sit at 1024 (t / 2) + 512 (t % 2),
// row-major 16 x 32 bytes, and the scale (zero-point) of stage t, row r at
// 4 (16 t + r); with 32 rows (NR = 2, at most 2 stages) the codes of stage
// t sit at 1024 t, row-major 32 x 32 bytes, and the scale of stage t, row r
// at 4 (32 t + r).
template <int K, int WV, int T, int NR>
struct GroupBuf {
    static_assert(T % WV == 0, "every wave prepares the same number of token tiles");
    static_assert(NR == 1 || (NR == 2 && K <= 2), "32-row waves take at most 2 stages");
    static constexpr int PT = T / WV;                       // token tiles a wave prepares
    static constexpr int X_BYTES = 16 * T * 256;
    static constexpr int SX = X_BYTES;
    static constexpr int WAVES = SX + 16 * T * 4;
    static constexpr int X_DMA = 4 * PT;                    // 1 KiB loads per wave
    static constexpr int CODE_DMA = NR == 1 ? (K + 1) / 2 : K;
    static constexpr int SCALES = CODE_DMA * 1024;          // within a wave's part
    static constexpr int ZEROS = SCALES + 256;
    static constexpr int WAVE_BYTES = ZEROS + 256;
    static constexpr int BYTES = WAVES + WV * WAVE_BYTES;
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

template <int K, bool DEF, int WV, int T, int NR, bool MFMA_PRIO>
__global__ __launch_bounds__(64 * WV) void prefill_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int64_t n_tokens,
    float *__restrict__ Y, int zero_point, int scale_type, int row_tiles)
{
    using B = GroupBuf<K, WV, T, NR>;
    constexpr int RW = 16 * NR;                          // rows per wave
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
    const int64_t m0 = (int64_t)(blockIdx.x / row_tiles) * (16 * T);
    const int64_t o0 = (int64_t)(blockIdx.x % row_tiles) * (RW * WV) + RW * wave;
    const uint32_t tokens_here = (uint32_t)(n_tokens - m0 < 16 * T ? n_tokens - m0 : 16 * T);
    const int64_t rem = rows - o0;
    const uint32_t rows_here = rem <= 0 ? 0u : (uint32_t)(rem < RW ? rem : RW);
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
    // 64 (X_DMA wave + i) + lane (the tokens of its token tiles
    // PT wave .. PT wave + PT - 1), slot s -> token s / 16, piece
    // (s % 16) ^ (token % 16); tokens past the tile read nothing.
    uint32_t dma_x[B::X_DMA];
#pragma unroll
    for (int i = 0; i < B::X_DMA; ++i) {
        const uint32_t s = (uint32_t)((B::X_DMA * wave + i) * 64 + lane);
        const uint32_t tok = s >> 4, pc = (s & 15) ^ (tok & 15);
        dma_x[i] = (tok < tokens_here ? 0u : kSkip) + tok * x_row + 16 * pc;
    }
    // Codes: lane l fills bytes 16 l of a 1 KiB load i, bytes 16 (l % 2) ..
    // + 15 of a row's 32 bytes of the group: with NR = 1 stage 2 i + l / 32,
    // row (l % 32) / 2; with NR = 2 stage i, row (l / 2) (a stage past K - 1
    // reads past the descriptor).
    const uint32_t dma_code = NR == 1
        ? (uint32_t)((lane & 31) >> 1) * row_bytes + 16 * (uint32_t)(lane & 1) +
              (uint32_t)(lane >> 5) * code_plane
        : (uint32_t)(lane >> 1) * row_bytes + 16 * (uint32_t)(lane & 1);
    const uint32_t code_step = NR == 1 ? 2u * code_plane : code_plane;
    // Scales and zero-points: lane l -> stage l / RW, row l % RW; stages past
    // K - 1 read nothing.
    const uint32_t pst = (uint32_t)lane / RW, prow = (uint32_t)lane % RW;
    const uint32_t dma_scale = pst < (uint32_t)K ? prow * gpr * sbytes + pst * scale_plane : kSkip;
    const uint32_t dma_zero = pst < (uint32_t)K ? prow * gpr * 4 + pst * zero_plane : kSkip;

    const uint32_t lds0 = lds_address(&buf[0][0]);
    auto issue = [&](uint32_t g, int b) {
        const uint32_t lds = lds0 + (uint32_t)b * B::BYTES;
#pragma unroll
        for (int i = 0; i < B::X_DMA; ++i)
            dma_x4(dx, g * 256, lds + (uint32_t)(B::X_DMA * wave + i) * 1024, dma_x[i]);
        const uint32_t lw = lds + B::WAVES + (uint32_t)wave * B::WAVE_BYTES;
#pragma unroll
        for (int i = 0; i < B::CODE_DMA; ++i)
            dma_x4(dc, g * 32 + i * code_step, lw + 1024u * i, dma_code);
        if (DEF || scale_type == kScaleF32)
            dma_dword(ds, g * 4, lw + B::SCALES, dma_scale);
        else
            dma_ushort(ds, g * 2, lw + B::SCALES, dma_scale);
        dma_dword(dz, g * 4, lw + B::ZEROS, dma_zero);
    };

    const u32x4 ones = {one, one, one, one};

    // This wave's token tiles of buffer b, once its loads have landed: each
    // lane reads its 64 bytes (token n, inputs 32 j .. 32 j + 31), rewrites
    // them in place as its four A operands (slot (4 j + i) ^ n then holds
    // block i) and the tile's sums (the MFMA with a ones operand, lane (n,
    // j) holding tokens 4 j .. 4 j + 3) go to the group's Sx, from n = 0.
    auto prepare = [&](int b) {
        char *lb = &buf[b][0];
#pragma unroll
        for (int q = 0; q < B::PT; ++q) {
            const int tt = B::PT * wave + q;
            char *xt = lb + (16 * tt + n) * 256;
            u32x4 runs[4], a[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                runs[i] = *reinterpret_cast<const u32x4 *>(xt + 16 * ((4 * j + i) ^ n));
            act_operands(runs, a);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                *reinterpret_cast<u32x4 *>(xt + 16 * ((4 * j + i) ^ n)) = a[i];
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int i = 0; i < 4; ++i) acc = mfma(a[i], ones, acc);
            if (n == 0) *reinterpret_cast<f32x4 *>(lb + B::SX + 4 * (16 * tt + 4 * j)) = acc;
        }
    };

    // A operands and sums of a token tile, from LDS.
    auto read_tile = [&](const char *lb, int tt, u32x4 (&a)[4], f32x4 &sx) {
        const char *xt = lb + (16 * tt + n) * 256;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            a[i] = *reinterpret_cast<const u32x4 *>(xt + 16 * ((4 * j + i) ^ n));
        sx = *reinterpret_cast<const f32x4 *>(lb + B::SX + 4 * (16 * tt + 4 * j));
    };

    // Per stage and row tile r the scale s and c = sum over stages of
    // s (4 + z) for the lane's row 16 r + n, and the code operands, from this
    // wave's part of a buffer (its own loads: no barrier needed).
    float s4[K][NR], c[NR];
    u32x4 bop[K][NR][2][2];
    auto params = [&](int b) {
        const char *lw = &buf[b][0] + B::WAVES + wave * B::WAVE_BYTES;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            c[r] = 0.0f;
#pragma unroll
            for (int t = 0; t < K; ++t) {
                const int e = 4 * (RW * t + 16 * r + n);
                const uint32_t sw = *reinterpret_cast<const uint32_t *>(lw + B::SCALES + e);
                const uint32_t zw = *reinterpret_cast<const uint32_t *>(lw + B::ZEROS + e);
                float sc, z;
                if constexpr (DEF) {
                    sc = __uint_as_float(sw);
                    z = __uint_as_float(zw);
                } else {
                    sc = scale_type == kScaleF32 ? __uint_as_float(sw)
                         : scale_type == kScaleF16
                             ? (float)__builtin_bit_cast(_Float16, (uint16_t)(sw & 0xFFFFu))
                             : __uint_as_float(sw << 16);
                    z = sym ? 2.0f : __uint_as_float(zw);
                }
                s4[t][r] = sc;
                c[r] = __builtin_fmaf(sc, 4.0f + z, c[r]);
            }
#pragma unroll
            for (int t = 0; t < K; ++t) {
                const int off = NR == 1 ? 1024 * (t >> 1) + 512 * (t & 1) : 1024 * t + 512 * r;
                const u32x2 w = *reinterpret_cast<const u32x2 *>(lw + off + n * 32 + 8 * j);
                code_operands_pair(w[0], w[1], mask, four, bop[t][r]);
            }
        }
    };

    f32x4 run[T][NR], cur[T][NR];
#pragma unroll
    for (int q = 0; q < T; ++q)
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            cur[q][r] = (f32x4){0.f, 0.f, 0.f, 0.f};
            run[q][r] = cur[q][r];
        }
    // One group's stage products for token tile q: per row tile and stage
    // s P, then - c Sx.
    auto tile = [&](int q, const u32x4 (&a)[4], const f32x4 &sx) {
#pragma unroll
        for (int r = 0; r < NR; ++r) {
#pragma unroll
            for (int t = 0; t < K; ++t) {
                f32x4 pr = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int b = 0; b < 4; ++b) pr = mfma(a[b], bop[t][r][b >> 1][b & 1], pr);
#pragma unroll
                for (int i = 0; i < 4; ++i) cur[q][r][i] = __builtin_fmaf(s4[t][r], pr[i], cur[q][r][i]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) cur[q][r][i] = __builtin_fmaf(-c[r], sx[i], cur[q][r][i]);
        }
    };

    // Quarter length as in the general kernel (4 waves, 2-group chunks).
    const uint32_t per_q = (((gpr + 3) / 4 + 1) / 2) * 2;
    // MFMA_PRIO (2 to 4 stages, long token runs): a group's stage products
    // (its MFMA stretch) are issued at a raised wave priority, so that the
    // matrix core keeps being fed while the other waves of the SIMD build
    // operands.
    int quarter = 0;

    issue(0, 0);
    if (gpr > 1) {
        issue(1, 1);
        wait_vm<B::DMA>();
    } else {
        wait_vm<0>();
    }
    prepare(0);
    for (uint32_t g = 0; g < gpr; ++g) {
        // every wave has prepared group g, and every wave is done with the
        // buffer of group g - 1: it is free again
        __syncthreads();
        if (g + 2 < gpr) issue(g + 2, (int)((g + 2) % kBuffers));
        const char *lb = &buf[g % kBuffers][0];
        params((int)(g % kBuffers));
        u32x4 a_next[4];
        f32x4 sx_next;
        read_tile(lb, 0, a_next, sx_next);
        if constexpr (MFMA_PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int q = 0; q < T; ++q) {
            u32x4 a[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = a_next[i];
            const f32x4 sx = sx_next;
            if (q + 1 < T) read_tile(lb, q + 1, a_next, sx_next);
            tile(q, a, sx);
        }
        if constexpr (MFMA_PRIO) __builtin_amdgcn_s_setprio(0);
        // end of a quarter: fold it into the running sum (which starts at
        // +0: a quarter sum is never -0, as it starts at +0 and rounds to
        // nearest, so +0 + Q0 is Q0 bit for bit)
        if ((g + 1) % per_q == 0 || g + 1 == gpr) {
#pragma unroll
            for (int q = 0; q < T; ++q)
#pragma unroll
                for (int r = 0; r < NR; ++r) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) run[q][r][i] = run[q][r][i] + cur[q][r][i];
                    cur[q][r] = (f32x4){0.f, 0.f, 0.f, 0.f};
                }
            ++quarter;
        }
        // this wave's loads of group g + 1 have landed (group g + 2's may
        // not): prepare its share of them
        if (g + 1 < gpr) {
            if (g + 2 < gpr) wait_vm<B::DMA>(); else wait_vm<0>();
            prepare((int)((g + 1) % kBuffers));
        }
    }
    // quarters with no groups add zeros, as the general kernel's idle waves do
    for (; quarter < 4; ++quarter)
#pragma unroll
        for (int q = 0; q < T; ++q)
#pragma unroll
            for (int r = 0; r < NR; ++r)
#pragma unroll
                for (int i = 0; i < 4; ++i) run[q][r][i] = run[q][r][i] + 0.0f;

    // lane: tokens m0 + 16 q + 4 j + i of output row o0 + 16 r + n
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        if ((uint32_t)(16 * r + n) < rows_here) {
#pragma unroll
            for (int q = 0; q < T; ++q)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t tk = (uint32_t)(16 * q + 4 * j + i);
                    if (tk < tokens_here) Y[(m0 + tk) * rows + o0 + 16 * r + n] = run[q][r][i];
                }
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
// a raised wave priority.
constexpr int64_t kPrefillPrioTokens = 1024;

template <int K, bool DEF, int WV, int T, int NR>
hipError_t launch_t(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int zp, int sdt, const uint16_t *X, int64_t n_tokens, float *Y,
                    hipStream_t stream)
{
    const int row_tiles = (int)((rows + 16 * NR * WV - 1) / (16 * NR * WV));
    const int grid = (int)((int64_t)row_tiles * ((n_tokens + 16 * T - 1) / (16 * T)));
    const int64_t pw = rows * cols / 16, pg = rows * cols / 128;
    const bool prio = K > 1 && n_tokens >= kPrefillPrioTokens;
    return prio ? launch(prefill_kernel<K, DEF, WV, T, NR, true>, grid, 64 * WV, stream, codes,
                         scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles)
                : launch(prefill_kernel<K, DEF, WV, T, NR, false>, grid, 64 * WV, stream, codes,
                         scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt, row_tiles);
}

template <bool DEF, int WV, int T>
hipError_t launch_k(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int64_t n_tokens,
                    float *Y, hipStream_t stream)
{
    switch (k) {
    case 1: return launch_t<1, DEF, WV, T, 1>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, stream);
    case 2: return launch_t<2, DEF, WV, T, 1>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, stream);
    case 3: return launch_t<3, DEF, WV, T, 1>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, stream);
    case 4: return launch_t<4, DEF, WV, T, 1>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, stream);
    default: return hipErrorInvalidValue;
    }
}

// Tile shape: the large tile (8 waves, 128 rows x 128 tokens: every code
// operand serves 8 token tiles) when it gives at least 3/4 of the compute
// units a workgroup, else the small one (4 waves, 64 rows x 64 tokens).
// Measured on 4096 x 4096, 12288 x 4096 and 4096 x 12288 from 256 to 2048
// tokens, the large tile is the faster one exactly there.
bool large_tiles(int64_t rows, int64_t n_tokens, int cus)
{
    return 4 * ((rows + 127) / 128) * ((n_tokens + 127) / 128) >= 3 * (int64_t)cus;
}

// One stage: waves of 32 rows (8 waves, 256 rows x 128 tokens), so that each
// A operand read from LDS serves two row tiles, when that still gives every
// compute unit a workgroup (30% faster than 16-row waves on the three
// shapes at 2048 tokens; slower where it leaves compute units idle). With
// more stages the 32-row waves' code operands do not fit the registers of
// 128 tokens, and 64 tokens were slower than 16-row waves.
bool wide_tiles(int k, int64_t rows, int64_t n_tokens, int cus)
{
    return k == 1 && ((rows + 255) / 256) * ((n_tokens + 127) / 128) >= cus;
}

template <bool DEF>
hipError_t launch_d(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int64_t n_tokens,
                    float *Y, int cus, hipStream_t stream)
{
    if (wide_tiles(k, rows, n_tokens, cus))
        return launch_t<1, DEF, 8, 8, 2>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y,
                                         stream);
    return large_tiles(rows, n_tokens, cus)
        ? launch_k<DEF, 8, 8>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, stream)
        : launch_k<DEF, 4, 4>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, stream);
}

}  // namespace

bool linear_prefill_fits(int64_t rows, int64_t cols, int G, int64_t n_tokens)
{
    // The activation descriptor spans at most 128 rows of X (under 2^31
    // bytes), and the grid (row tiles x token tiles, at most 64 x 64 each)
    // fits an int.
    const int64_t tiles = ((rows + 63) / 64) * ((n_tokens + 63) / 64);
    return G == 128 && n_tokens >= kPrefillMinTokens && cols <= 65536 && tiles < (1ll << 31);
}

hipError_t launch_linear_prefill(const uint32_t *codes, const void *scales, const float *zeros,
                                 int64_t rows, int64_t cols, int k, int zero_point,
                                 int scale_type, const uint16_t *X, int64_t n_tokens, float *Y,
                                 int cus, hipStream_t stream)
{
    const char *sc = static_cast<const char *>(scales);
    const bool def = scale_type == kScaleF32 && zero_point != kZpSymmetric;
    return def ? launch_d<true>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X,
                                n_tokens, Y, cus, stream)
               : launch_d<false>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X,
                                 n_tokens, Y, cus, stream);
}

}  // namespace rrq_detail

// Internal launch interface between the C ABI layer (rrq_api.cpp) and the
// HIP kernels (rrq_kernels.hip). Arguments are already validated.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace rrq_detail {

// Package construction of n_groups groups of G bfloat16 weights, S stages,
// in stage format (zero_point, scale_type) of rrq.h (scales are binary32 or
// 16-bit patterns; zeros are not written for symmetric stages).
// from_base: stage 0 of the package is an input (a base checkpoint) and only
// stages 1 .. S-1 are written.
// pmr (NULL for none; ignored with from_base): per-group peak-to-mean
// ratios of W as a side output.
// lanes: lanes per group (construct_lanes), grid: workgroups of one wave.
hipError_t launch_construct(const uint16_t *W, int64_t n_groups, int G, int S,
                            uint32_t *codes, void *scales, float *zeros, float *pmr,
                            bool from_base, int zero_point, int scale_type, int lanes, int grid,
                            hipStream_t stream);

// Several tensors (each its own package, integer zero-points, binary32
// scales) in one launch: tensor i has n_groups[i] groups at W[i] and its
// package at codes[i], scales[i], zeros[i]; its tiles (of 64 lane shares at
// the launch's lanes per group) are the launch's tiles tile_first[i] ..
// tile_first[i + 1] - 1. At most kConstructManyPerLaunch tensors per launch
// (the table travels in the kernel arguments, 3 KiB).
constexpr int kConstructManyPerLaunch = 64;
struct ConstructMany {
    int64_t tile_first[kConstructManyPerLaunch + 1];
    const void *W[kConstructManyPerLaunch];
    void *codes[kConstructManyPerLaunch];
    void *scales[kConstructManyPerLaunch];
    void *zeros[kConstructManyPerLaunch];
    int64_t n_groups[kConstructManyPerLaunch];
    int32_t n;
};
hipError_t launch_construct_many(const ConstructMany &a, int G, int S, int lanes, int grid,
                                 hipStream_t stream);

// Per-group peak-to-mean ratios of W only.
hipError_t launch_group_pmr(const uint16_t *W, int64_t n_groups, int G, float *pmr, int grid,
                            hipStream_t stream);

// Prefix-k reconstruction of a package with n_groups groups of G, S stages.
hipError_t launch_reconstruct(const uint32_t *codes, const void *scales,
                              const float *zeros, int64_t n_groups, int G, int S,
                              int k, void *out, bool out_bf16, int zero_point,
                              int scale_type, int grid, hipStream_t stream);

// Stage-sum linear layer Y = X W~_(k)^T on a package of rows x cols weights.
hipError_t launch_linear(const uint32_t *codes, const void *scales, const float *zeros,
                         int64_t rows, int64_t cols, int G, int S, int k, int zero_point,
                         int scale_type, const uint16_t *X, int64_t n_tokens, float *Y,
                         hipStream_t stream);

// The decode form of the linear layer (up to 4 tokens, groups of 128, cols
// a multiple of 4096 up to kDecodeMaxCols, or 5 to 16 tokens on rows of 4096
// inputs; and the stage, row and token counts where it is the faster one:
// linear_decode_fits);
// launch_linear covers every other case.
constexpr int kDecodeMaxCols = 16384;
// The batch form (groups of 128, kBatchMinTokens to 16 tokens, at most 4096
// cols: the A operands of a wave's groups stay in its registers; and the
// row, column, stage and token counts where it is the faster one:
// linear_batch_fits).
constexpr int kBatchMinTokens = 5;
bool linear_batch_fits(int64_t rows, int64_t cols, int G, int k, int64_t n_tokens);
hipError_t launch_linear_batch(const uint32_t *codes, const void *scales, const float *zeros,
                               int64_t rows, int64_t cols, int k, int zero_point, int scale_type,
                               const uint16_t *X, int64_t n_tokens, float *Y, int cus,
                               hipStream_t stream);
// The prefill form (groups of 128, at least kPrefillMinTokens tokens;
// 128-token x 128-row tiles when they still give every compute unit one,
// else 64 x 64). Measured against the general kernel on the Qwen3-8B shapes:
// from 128 tokens it is faster on all of them (2-3x from 256); below that a
// matrix of a few thousand rows gives too few tiles to fill the GPU.
constexpr int kPrefillMinTokens = 128;
bool linear_prefill_fits(int64_t rows, int64_t cols, int G, int64_t n_tokens);
hipError_t launch_linear_prefill(const uint32_t *codes, const void *scales, const float *zeros,
                                 int64_t rows, int64_t cols, int k, int zero_point,
                                 int scale_type, const uint16_t *X, int64_t n_tokens, float *Y,
                                 int cus, hipStream_t stream);
bool linear_decode_fits(int64_t rows, int64_t cols, int G, int k, int64_t n_tokens);
hipError_t launch_linear_decode(const uint32_t *codes, const void *scales, const float *zeros,
                                int64_t rows, int64_t cols, int k, int zero_point, int scale_type,
                                const uint16_t *X, int64_t n_tokens, float *Y, int cus,
                                hipStream_t stream);

// rows and cols of the linear kernel stay below this bound, so its 32-bit
// buffer sizes and offsets (at most 16 * rows * 4 bytes) cannot wrap.
constexpr int64_t kLinearMaxDim = int64_t(1) << 26;

// Stages a package holds at most (RRQ_MAX_STAGES of rrq.h).
constexpr int kMaxStages = 4;

// Workgroups (one wave each) the construct kernel keeps resident per compute
// unit with one lane per group: two per SIMD.
constexpr int kConstructBlocksPerCU = 8;
// Lanes per group of the construct kernel. A wave takes tiles of 64 lane
// shares; one share (a whole group at L = 1) is a long serial stretch of work
// per wave (4 stages x G elements), and a call ends with its waves' last
// tiles. A call with few tiles per resident wave therefore ends on that
// latency, so such calls split each group over L = G / 32 lanes (32 elements
// each): the serial work per wave drops L-fold and four waves per SIMD fit
// instead of two. Measured on Qwen3-8B shapes at G = 128 (per call, MALL
// flushed): 1024 x 4096 12.4 -> 7.9 us, 4096 x 4096 21.9 -> 20.0 us,
// 12288 x 4096 53.8 -> 49.4 us (3 tiles per slot), 47104 x 4096 equal at
// 11.5 tiles per slot; L = 2 at G = 128 was never the fastest. The
// peak-to-mean side output needs one lane per group. tiles1 = tiles at L = 1.
constexpr int64_t kConstructSplitMaxTilesPerSlot = 8;
inline int construct_lanes(int64_t n_groups, int G, bool pmr, int cus)
{
    if (pmr || G == 32) return 1;
    const int64_t tiles1 = (n_groups + 63) / 64;
    const int64_t slots = (int64_t)cus * kConstructBlocksPerCU;
    return tiles1 <= kConstructSplitMaxTilesPerSlot * slots ? G / 32 : 1;
}
// Resident one-wave workgroups per compute unit at L lanes per group: the
// waves per SIMD the registers allow (two at 128 elements per lane, four at
// 32), capped by LDS at 32 elements per lane (a wave's transpose buffer and
// dequantization table take 11 KiB of 160).
constexpr int construct_blocks_per_cu(int G, int lanes)
{
    return lanes == 1 ? kConstructBlocksPerCU : (G / lanes >= 64 ? 12 : 14);
}
// Reconstruct: threads per workgroup (4 waves), 16-byte output chunks per
// lane per tile (8 bfloat16 or 4 binary32 elements each) and resident
// workgroups per CU, as measured on the 36-layer stack (6.9e9 weights): 8
// chunks per lane keep more loads in flight for 1 or 2 stages, 4 are faster
// from 3 stages on (the loads of K stages x 8 chunks crowd the registers);
// 2 workgroups per CU write faster than 8 (fewer concurrent write streams),
// except for binary32 output from 3 stages on.
constexpr int kReconstructThreads = 256;
constexpr int reconstruct_chunks(int k, bool bf16) { return (void)bf16, k <= 2 ? 8 : 4; }
constexpr int reconstruct_blocks_per_cu(int k, bool bf16) { return bf16 || k <= 2 ? 2 : 8; }

}  // namespace rrq_detail

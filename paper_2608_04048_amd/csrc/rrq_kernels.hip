// HIP kernels for RRQ package construction and prefix reconstruction on
// gfx950 (MI355X).
//
// Construction follows Algorithm 1 (no base checkpoint) with the per-group
// affine RTN stage of Eq. 1-3 applied S times, each stage to the residual the
// earlier stages left (Eq. 4-7). Reconstruction is the prefix sum of Eq. 8 /
// Eq. 18-19. The arithmetic is the fixed binary32 reading stated in rrq.h;
// the kernels reproduce it bit for bit (build with -ffp-contract=off, no fast
// math, denormals kept).
//
// Construct kernel layout:
//   * one wave (64 lanes) per workgroup; the wave takes tiles of 64
//     consecutive groups in a grid-stride loop, and each lane owns one whole
//     group, held in registers (G binary32 residuals) through every stage, so
//     the bfloat16 input is read from HBM once and residuals never leave the
//     register file;
//   * the tile is loaded with fully coalesced 16-byte-per-lane loads and
//     transposed through LDS (an XOR swizzle on the 16-byte chunk index keeps
//     both the row writes and the per-lane group reads free of bank
//     conflicts), so every lane receives the G contiguous elements of its
//     group;
//   * the group's range, scale, reciprocal and zero-point are computed once
//     per lane per stage, i.e. once per group;
//   * per element and stage: t = r * inv; u = t + (1.5 * 2^23 + z), which is
//     the single nearest-even rounding of the exact t + z (u lies in
//     [2^23, 2^24), where binary32 spacing is 1) and leaves the code in the
//     two low mantissa bits of u; codes are packed by shift-adding u's bits
//     (the constant upper bits of the 16 shifted words sum to a known
//     constant, subtracted once per word); Q - z = u - (1.5 * 2^23 + z) exactly;
//     rhat = (Q - z) * s; r = r - rhat.
//   * Lower clamp: no element can round below code 0, because z is computed
//     from the same fl(-lo * inv) that bounds every fl(r * inv) from below.
//     Upper clamp: only the group maximum can reach code 4, so each lane tests
//     its maximum first and the wave runs the clamped element loop only when
//     one of its groups needs it.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rrq_launch.h"

namespace rrq_detail {
namespace {

constexpr float kMagic = 12582912.0f;          // 1.5 * 2^23
constexpr uint32_t kMagicBits = 0x4B400000u;   // its binary32 bit pattern
constexpr float kTopCode = kMagic + 3.0f;      // u of code 3

// Sum over the 16 code slots of the constant upper bits of u, shifted to each
// slot; subtracting it from the shift-added u words leaves the packed codes.
constexpr uint32_t pack_bias()
{
    uint32_t b = 0;
    for (int e = 0; e < 16; ++e) b += kMagicBits << (2 * e);
    return b;
}
constexpr uint32_t kPackBias = pack_bias();

// Raw buffer resources (gfx9 family descriptor). Accesses beyond num_records
// bytes read as zero and stores there are dropped, which handles the ragged
// last tile without branches. A resource is rebuilt per tile, so 32-bit
// num_records and offsets suffice for inputs of any size.
using rsrc_t = __amdgpu_buffer_rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

// acc + (bits << sh) as one v_lshl_add_u32 (the compiler would otherwise
// re-associate the packing sums into shift + add3 pairs). sh is a constant
// after unrolling, so the switch folds to one instruction.
#define RRQ_LSHL_ADD_CASE(SH)                                                      \
    case SH:                                                                     \
        asm("v_lshl_add_u32 %0, %1, " #SH ", %2" : "=v"(out) : "v"(bits), "v"(acc)); \
        break;
__device__ __forceinline__ uint32_t lshl_add(uint32_t bits, int sh, uint32_t acc)
{
    uint32_t out;
    switch (sh) {
        RRQ_LSHL_ADD_CASE(2) RRQ_LSHL_ADD_CASE(4) RRQ_LSHL_ADD_CASE(6) RRQ_LSHL_ADD_CASE(8)
        RRQ_LSHL_ADD_CASE(10) RRQ_LSHL_ADD_CASE(12) RRQ_LSHL_ADD_CASE(14) RRQ_LSHL_ADD_CASE(16)
        RRQ_LSHL_ADD_CASE(18) RRQ_LSHL_ADD_CASE(20) RRQ_LSHL_ADD_CASE(22) RRQ_LSHL_ADD_CASE(24)
        RRQ_LSHL_ADD_CASE(26) RRQ_LSHL_ADD_CASE(28) RRQ_LSHL_ADD_CASE(30)
    default: out = acc + (bits << sh); break;
    }
    return out;
}
#undef RRQ_LSHL_ADD_CASE

// Element loop of one stage for one lane's group: the stage's codes into
// words[]; with UPDATE also the residual r <- r - (Q - z) s and the range of
// the new residual (lo, hi, zero included) for the next stage.
template <int G, bool CLAMP, bool UPDATE>
__device__ __forceinline__ void stage_elements(float (&r)[G], float inv, float m, float s,
                                               uint32_t (&words)[G / 16], float &lo, float &hi)
{
    float l0 = 0.f, l1 = 0.f, h0 = 0.f, h1 = 0.f;
#pragma unroll
    for (int w = 0; w < G / 16; ++w) {
        uint32_t acc = 0;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int j = w * 16 + e;
            const float t = r[j] * inv;
            float u = t + m;
            if (CLAMP) u = fminf(u, kTopCode);
            if (e == 0) acc = __float_as_uint(u);
            else acc = lshl_add(__float_as_uint(u), 2 * e, acc);
            if (UPDATE) {
                const float qz = u - m;      // Q - z, exact
                const float rh = qz * s;     // fl((Q - z) s)
                r[j] = r[j] - rh;
            }
        }
        words[w] = acc - kPackBias;
        if (UPDATE) {
            // min3 / max3 over pairs of the new residuals, two chains each
#pragma unroll
            for (int e = 0; e < 16; e += 4) {
                const int j = w * 16 + e;
                l0 = fminf(fminf(l0, r[j]), r[j + 1]);
                h0 = fmaxf(fmaxf(h0, r[j]), r[j + 1]);
                l1 = fminf(fminf(l1, r[j + 2]), r[j + 3]);
                h1 = fmaxf(fmaxf(h1, r[j + 2]), r[j + 3]);
            }
        }
        // Keep the scheduler from hoisting the next word's products above
        // this word's updates: that would hold a second G-wide array of
        // temporaries live and spill the residuals out of the register file.
        __builtin_amdgcn_sched_barrier(0);
    }
    lo = fminf(l0, l1);
    hi = fmaxf(h0, h1);
}

template <int G>
__device__ __forceinline__ void group_range(const float (&r)[G], float &lo, float &hi)
{
    float l0 = 0.f, l1 = 0.f, h0 = 0.f, h1 = 0.f;
#pragma unroll
    for (int j = 0; j < G; j += 4) {
        l0 = fminf(fminf(l0, r[j]), r[j + 1]);
        h0 = fmaxf(fmaxf(h0, r[j]), r[j + 1]);
        l1 = fminf(fminf(l1, r[j + 2]), r[j + 3]);
        h1 = fmaxf(fmaxf(h1, r[j + 2]), r[j + 3]);
    }
    lo = fminf(l0, l1);
    hi = fmaxf(h0, h1);
}

// Stores one lane's code words of one stage at byte offset off of the
// stage's per-tile resource.
template <int G>
__device__ __forceinline__ void store_words(rsrc_t dst, uint32_t off, const uint32_t (&w)[G / 16])
{
    if constexpr (G / 16 >= 4) {
#pragma unroll
        for (int i = 0; i < G / 16; i += 4) {
            const u32x4 v = {w[i], w[i + 1], w[i + 2], w[i + 3]};
            __builtin_amdgcn_raw_buffer_store_b128(v, dst, off + 4 * i, 0, 0);
        }
    } else {
        const u32x2 v = {w[0], w[1]};
        __builtin_amdgcn_raw_buffer_store_b64(v, dst, off, 0, 0);
    }
}

// Loads this lane's share of one tile (64 groups): chunk q = 64 i + lane of
// the tile's 16-byte chunks, so each load instruction covers 1 KiB
// contiguously. Chunks past the end of the input read as zero.
template <int CH>
__device__ __forceinline__ void load_tile(const uint4 *__restrict__ W, int64_t n_groups,
                                          int64_t tile, int lane, uint4 (&v)[CH])
{
    const int64_t g0 = tile * 64;
    const int64_t left = n_groups - g0;
    const uint32_t bytes = (uint32_t)(left < 64 ? left : 64) * CH * 16;
    const rsrc_t src = make_rsrc(W + g0 * CH, bytes);
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(src, (i * 64 + lane) * 16, 0, 0);
        v[i] = make_uint4(x.x, x.y, x.z, x.w);
    }
}

template <int G>
__global__ __launch_bounds__(64) void construct_kernel(const uint4 *__restrict__ W,
                                                       int64_t n_groups, int n_stages,
                                                       uint32_t *__restrict__ codes,
                                                       float *__restrict__ scales,
                                                       float *__restrict__ zeros)
{
    constexpr int CH = G / 8;            // 16-byte chunks (8 bfloat16) per group
    constexpr int WPG = G / 16;          // code words per group and stage
    constexpr int ROW = CH + 1;          // LDS row of one group, padded by 16 bytes
    constexpr int GROUPS_PER_LOAD = 64 / CH;
    // Padding each group's row by one chunk spreads both access patterns over
    // all banks: a row write (lanes -> consecutive chunks of a group) and a
    // column read (lanes -> the same chunk of consecutive groups).
    __shared__ uint4 tile_lds[64 * ROW];

    const int lane = threadIdx.x;
    const int64_t n_tiles = (n_groups + 63) / 64;
    const int64_t words_per_stage = n_groups * WPG;
    uint4 *const wr_base = tile_lds + (lane / CH) * ROW + (lane % CH);
    const uint4 *const rd_base = tile_lds + lane * ROW;

    int64_t tile = blockIdx.x;
    uint4 v[CH];
    if (tile < n_tiles) load_tile<CH>(W, n_groups, tile, lane, v);

    for (; tile < n_tiles; tile += gridDim.x) {
        __syncthreads();   // the previous tile's LDS reads are complete
#pragma unroll
        for (int i = 0; i < CH; ++i) wr_base[i * GROUPS_PER_LOAD * ROW] = v[i];
        __syncthreads();

        // Each lane gathers its own group and widens bfloat16 to binary32.
        float r[G];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const uint4 w = rd_base[c];
            const uint32_t p[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                r[8 * c + 2 * h] = __uint_as_float(p[h] << 16);
                r[8 * c + 2 * h + 1] = __uint_as_float(p[h] & 0xFFFF0000u);
            }
        }

        // Prefetch the next tile while this one is quantized.
        const int64_t next = tile + gridDim.x;
        if (next < n_tiles) load_tile<CH>(W, n_groups, next, lane, v);

        const int64_t g0 = tile * 64;
        const uint32_t groups_here = (uint32_t)(n_groups - g0 < 64 ? n_groups - g0 : 64);
        float lo, hi;
        group_range<G>(r, lo, hi);
        for (int k = 0; k < n_stages; ++k) {
            const float d = hi - lo;
            const float s = d / 3.0f;
            const bool degenerate = !(s >= 0x1p-126f);
            const float inv = degenerate ? 0.0f : 1.0f / s;
            const float sq = degenerate ? 0.0f : s;
            // lo <= 0, so |lo| is exactly 0 - lo, +0 included. Written as fabs:
            // the code generator folds 0 - lo into a negate modifier, which
            // turns lo = +0 into -0 and would store z = -0.
            const float z = rintf(fabsf(lo) * inv);
            const float m = kMagic + z;
            const float u_hi = hi * inv + m;
            const bool clamp = __any(u_hi > kTopCode);

            uint32_t words[WPG];
            (void)clamp;
            stage_elements<G, true, true>(r, inv, m, sq, words, lo, hi);
            // Lanes past the last group fall outside the resources and
            // their stores are dropped.
            store_words<G>(make_rsrc(codes + k * words_per_stage + g0 * WPG, groups_here * WPG * 4),
                           lane * WPG * 4, words);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(sq),
                                                  make_rsrc(scales + k * n_groups + g0, groups_here * 4),
                                                  lane * 4, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(z),
                                                  make_rsrc(zeros + k * n_groups + g0, groups_here * 4),
                                                  lane * 4, 0, 0);
        }
    }
}

// Reconstruction: each thread owns 16 consecutive elements (one code word per
// stage) and sums (Q - z) s over the first k stages, left to right.
template <bool OUT_BF16>
__global__ __launch_bounds__(kReconstructThreads) void reconstruct_kernel(
    const uint32_t *__restrict__ codes, const float *__restrict__ scales,
    const float *__restrict__ zeros, int64_t n_words, int64_t n_groups, int wpg_shift,
    int k, void *__restrict__ out)
{
    const int64_t stride = (int64_t)gridDim.x * kReconstructThreads;
    for (int64_t w = (int64_t)blockIdx.x * kReconstructThreads + threadIdx.x; w < n_words;
         w += stride) {
        const int64_t g = w >> wpg_shift;
        float acc[16];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            if (t >= k) break;
            const uint32_t word = codes[t * n_words + w];
            const float s = scales[t * n_groups + g];
            const float z = zeros[t * n_groups + g];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float q = (float)((word >> (2 * e)) & 3u);
                const float rh = (q - z) * s;
                acc[e] = t == 0 ? rh : acc[e] + rh;
            }
        }
        if (OUT_BF16) {
            uint32_t packed[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                // nearest-even binary32 -> bfloat16 of a finite value
                uint32_t lo = __float_as_uint(acc[2 * i]);
                uint32_t hi = __float_as_uint(acc[2 * i + 1]);
                lo = (lo + 0x7FFFu + ((lo >> 16) & 1u)) >> 16;
                hi = (hi + 0x7FFFu + ((hi >> 16) & 1u)) >> 16;
                packed[i] = lo | (hi << 16);
            }
            uint4 *dst = reinterpret_cast<uint4 *>(static_cast<uint16_t *>(out) + w * 16);
            dst[0] = make_uint4(packed[0], packed[1], packed[2], packed[3]);
            dst[1] = make_uint4(packed[4], packed[5], packed[6], packed[7]);
        } else {
            float4 *dst = reinterpret_cast<float4 *>(static_cast<float *>(out) + w * 16);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                dst[i] = make_float4(acc[4 * i], acc[4 * i + 1], acc[4 * i + 2], acc[4 * i + 3]);
        }
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

}  // namespace

hipError_t launch_construct(const uint16_t *W, int64_t n_groups, int G, int S,
                            uint32_t *codes, float *scales, float *zeros, int grid,
                            hipStream_t stream)
{
    const uint4 *w4 = reinterpret_cast<const uint4 *>(W);
    switch (G) {
    case 32: return launch(construct_kernel<32>, grid, 64, stream, w4, n_groups, S, codes, scales, zeros);
    case 64: return launch(construct_kernel<64>, grid, 64, stream, w4, n_groups, S, codes, scales, zeros);
    case 128: return launch(construct_kernel<128>, grid, 64, stream, w4, n_groups, S, codes, scales, zeros);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_reconstruct(const uint32_t *codes, const float *scales, const float *zeros,
                              int64_t n_groups, int G, int S, int k, void *out, bool out_bf16,
                              int grid, hipStream_t stream)
{
    (void)S;
    const int64_t n_words = n_groups * (G / 16);
    const int wpg_shift = G == 32 ? 1 : G == 64 ? 2 : 3;
    if (out_bf16)
        return launch(reconstruct_kernel<true>, grid, kReconstructThreads, stream, codes, scales,
                      zeros, n_words, n_groups, wpg_shift, k, out);
    return launch(reconstruct_kernel<false>, grid, kReconstructThreads, stream, codes, scales,
                  zeros, n_words, n_groups, wpg_shift, k, out);
}

}  // namespace rrq_detail

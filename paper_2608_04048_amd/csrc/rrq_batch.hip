// Batch form of the stage-sum linear layer (Eq. 20) for 5 to 16 tokens and
// groups of 128: Y[m][o] = sum over stages t < K and groups g of
// s_t,o,g (sum_i x_m,i Q_t,o,i - z_t,o,g sum_i x_m,i), the product the general
// kernel of rrq_linear.hip computes 16 tokens at a time, organised here, like
// the decode form, for streaming the package when the activations fit in
// registers.
//
// Matrix cores (v_mfma_f32_16x16x32_bf16, lane l: row / column n = l % 16,
// k-slice j = l / 16), the general kernel's operand layouts: A = 16 tokens x
// 32 inputs of X, B = 32 inputs x 16 output rows of codes (each the bfloat16
// 1 + Q/4), so P = sum x (1 + Q/4) and Sx = sum x (the same MFMA with a ones
// operand) give sum x Q = 4 P - 4 Sx; every output of an MFMA is used.
//
// Work: the 8 waves of a workgroup split the groups of a row into contiguous
// ranges of at most 8 (the general kernel's split for 8 waves), so a wave's A
// operands and group sums (16 tokens x its groups) are loaded and formed once
// and stay in registers. A workgroup takes 16-row tiles in turn; an item is
// one group of a 16-row tile, all K stages: its codes, scales and
// zero-points go from HBM into a ring of D LDS slots per wave by LDS-DMA
// loads, a fixed count per item, and the wave waits for exactly the item it
// reads. At the end of a tile the 8 waves' partial sums meet in LDS and are
// summed in wave order: per output, the wave's groups in order (k FMAs and
// the Sx term each) and then the 8 partials, the accumulation structure of
// the general kernel's 8-wave tiles, so its error bound holds unchanged.

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

constexpr int kWaves = 8;                      // waves per workgroup
constexpr int kMaxGroupsPerWave = 8;           // A operands held in registers
constexpr uint32_t kOnePair = 0x3F803F80u;     // two bfloat16 1.0
constexpr uint32_t kCodeMask = 0x00600060u;    // top two mantissa bits of both halves
constexpr int kZpSymmetric = 2;
constexpr int kScaleF32 = 0, kScaleF16 = 1;

__device__ __forceinline__ f32x4 mfma(const u32x4 &a, const u32x4 &b, const f32x4 &c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// One item's LDS slot (one group of a 16-row tile, all K stages): codes of
// stage t at 1024 (t / 2) + 512 (t % 2), row-major 16 x 32 bytes; scales and
// zero-points as 32-bit words, stage t of row r at 4 (16 t + r).
template <int K>
struct ItemSlot {
    static constexpr int CODE_DMA = (K + 1) / 2;   // 1 KiB loads, two stages each
    static constexpr int SCALES = CODE_DMA * 1024;
    static constexpr int ZEROS = SCALES + 256;
    static constexpr int BYTES = ZEROS + 256;
    static constexpr int DMA = CODE_DMA + 2;       // vector-memory loads per item
};

// Groups per wave GPW: the A operands of a wave's groups stay in its
// registers (16 tokens x GPW groups, 16 GPW VGPRs). GPW = 4 serves rows of up
// to 4096 inputs in at most 128 VGPRs, GPW = 8 up to 8192. One workgroup per
// CU: with GPW = 4 two fit (four waves per SIMD), but measured on
// 24576 x 4096 and 12288 x 4096 at 16 tokens that was 12-18% slower than
// one (the rings are then shallower, 64 KiB per workgroup); the smaller
// register set alone was 2-7% faster than GPW = 8 at one workgroup.
constexpr int wgs_per_cu(int gpw) { return (void)gpw, 1; }

// Ring depth: the 6-bit vmcnt counter and 96 KiB of LDS for the 8 rings.
template <int K, int GPW>
constexpr int depth_for()
{
    constexpr int by_count = 63 / ItemSlot<K>::DMA;
    constexpr int by_lds = 96 * 1024 / (kWaves * ItemSlot<K>::BYTES);
    constexpr int d = by_count < by_lds ? by_count : by_lds;
    return d < 16 ? d : 16;
}

// A operands of one group for the lane (token n, k-slice j) from its inputs
// 32 j .. 32 j + 31, four runs of 8: block b = 16-input run 2 j + b / 2, half
// b % 2, register v = (x[v'], x[v' + 8]).
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

// Activation run loaded behind the compiler's back (see the wait below): a
// compiler-visible load would be followed by a wait that also drains the
// ring's DMA loads, which the compiler does not count.
__device__ __forceinline__ u32x4 load_run(const u32x4 &desc, uint32_t voff)
{
    u32x4 v;
    asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen" : "=v"(v) : "v"(voff), "s"(desc));
    return v;
}

template <int K, bool DEF, int GPW>
__global__ __launch_bounds__(64 * kWaves, 2 * wgs_per_cu(GPW)) void batch_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int n_tokens, float *__restrict__ Y,
    int zero_point, int scale_type)
{
    using L = ItemSlot<K>;
    constexpr int D = depth_for<K, GPW>();
    __shared__ __attribute__((aligned(16))) char ring[kWaves][D][L::BYTES];
    __shared__ f32x4 red[2][kWaves][64];
    // group sums of the wave's groups: Sx depends on the token only, so a
    // wave keeps its 16 tokens x GPW groups here rather than in registers
    // (lane k-slice j reads tokens 4 j .. 4 j + 3 as one 16-byte broadcast)
    __shared__ f32x4 sx_lds[kWaves][GPW][4];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;
    const int j = lane >> 4;
    const bool sym = zero_point == kZpSymmetric;
    const int gpr = (int)(cols / 128);                  // groups per row
    uint32_t mask, one;
    asm volatile("s_mov_b32 %0, %1" : "=s"(mask) : "n"(kCodeMask));
    asm volatile("v_mov_b32 %0, %1" : "=v"(one) : "n"(kOnePair));

    // This wave's groups: the general kernel's split for 8 waves (ranges of a
    // whole number of 2-group chunks).
    const int per_wave = ((gpr + kWaves - 1) / kWaves + 1) / 2 * 2;
    const int g_begin = per_wave * wave < gpr ? per_wave * wave : gpr;
    const int g_end = g_begin + per_wave < gpr ? g_begin + per_wave : gpr;
    const int gw = g_end - g_begin;                     // 0 .. GPW

    const uint32_t row_bytes = (uint32_t)(cols / 4);
    const uint32_t plane_bytes = (uint32_t)plane_words * 4;
    const uint32_t sbytes = scale_type == kScaleF32 ? 4 : 2;
    const uint32_t scale_plane = (uint32_t)plane_groups * sbytes;
    const uint32_t zero_plane = (uint32_t)plane_groups * 4;
    const u32x4 dc = make_desc(codes, (uint32_t)K * plane_bytes);
    const u32x4 ds = make_desc(scales, (uint32_t)K * scale_plane);
    const u32x4 dz = make_desc(sym ? nullptr : zeros, sym ? 0u : (uint32_t)K * zero_plane);

    // DMA lane offsets within an item. Codes: lane l fills bytes 16 l of a
    // 1 KiB load: stage 2 i + l / 32, row (l % 32) / 2, bytes 16 (l % 2) .. + 15
    // of the row's 32 bytes of the group (a stage past K - 1 reads past the
    // descriptor, or other data that is never read).
    const uint32_t dma_code = (uint32_t)((lane & 31) >> 1) * row_bytes + 16 * (uint32_t)(lane & 1) +
                              (uint32_t)(lane >> 5) * plane_bytes;
    // Scales and zero-points: lane l -> stage l / 16, row l % 16; stages past
    // K - 1 read nothing.
    const uint32_t pst = (uint32_t)lane >> 4;
    const uint32_t prow = (uint32_t)(lane & 15) * (uint32_t)gpr;
    const uint32_t dma_scale = pst < (uint32_t)K ? (prow * sbytes + pst * scale_plane) : kSkip;
    const uint32_t dma_zero = pst < (uint32_t)K ? (prow * 4 + pst * zero_plane) : kSkip;

    const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
        Y, (short)0, (int)((uint32_t)n_tokens * (uint32_t)rows * 4u), (int)kRsrcWord3);
    const uint32_t lds_ring = lds_address(&ring[wave][0][0]);
    const char *my_ring = &ring[wave][0][0];

    // Row tiles of this workgroup: blockIdx, blockIdx + grid, ...
    const int tiles = (int)((rows + 15) / 16);
    const int my_tiles = (int)blockIdx.x < tiles ? (tiles - 1 - (int)blockIdx.x) / (int)gridDim.x + 1 : 0;
    const int total = my_tiles * gw;                    // items of this wave

    // DMA of the items in order (tile-major, then this wave's groups), one
    // call per item, position kept in running counters; items past the end
    // and rows past the last read through descriptors of size 0 or past
    // their end (zeros).
    int is_g = 0, is_slot = 0, issued = 0;
    int is_tile = (int)blockIdx.x;
    auto issue_next = [&]() {
        const bool live = issued < total;
        const uint32_t row0 = live ? (uint32_t)is_tile * 16 : 0u;
        const uint32_t g = (uint32_t)(g_begin + is_g);
        const uint32_t code_base = row0 * row_bytes + g * 32;
        const uint32_t grp = row0 * (uint32_t)gpr + g;
        const uint32_t lds = lds_ring + (uint32_t)is_slot * L::BYTES;
        u32x4 c_src = dc, s_src = ds, z_src = dz;
        if (!live) c_src[2] = s_src[2] = z_src[2] = 0u;
        // the reads of the item that used this slot have completed
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int i = 0; i < L::CODE_DMA; ++i)
            dma_x4(c_src, code_base + 2u * i * plane_bytes, lds + 1024u * i, dma_code);
        if (DEF || scale_type == kScaleF32)
            dma_dword(s_src, grp * 4, lds + L::SCALES, dma_scale);
        else
            dma_ushort(s_src, grp * 2, lds + L::SCALES, dma_scale);
        dma_dword(z_src, grp * 4, lds + L::ZEROS, dma_zero);
        ++issued;
        if (++is_slot == D) is_slot = 0;
        if (++is_g == gw) {
            is_g = 0;
            is_tile += (int)gridDim.x;
        }
    };

    // The ring's first items, then the activations of this wave's groups
    // (lane as A row: token n, tokens past n_tokens reading zeros), waited
    // for explicitly with the runs tied to the wait. The prologue runs at a
    // raised wave priority (measured 1-5% faster at 2 to 4 stages, same
    // outputs): it is a serial stretch that every later item waits for.
    __builtin_amdgcn_s_setprio(2);
#pragma unroll
    for (int d = 0; d < D; ++d) issue_next();
    u32x4 a[GPW][4];
    {
        const u32x4 xs = make_desc(X, (uint32_t)n_tokens * (uint32_t)cols * 2);
        const uint32_t xrow = (n < n_tokens ? 0u : kSkip) + (uint32_t)n * (uint32_t)cols * 2;
        u32x4 run[GPW][4];
#pragma unroll
        for (int g = 0; g < GPW; ++g) {
            // groups past this wave's range load nothing (an offset past the
            // buffer) and are never used
            const uint32_t off = (g < gw ? xrow : kSkip) + (uint32_t)(g_begin + g) * 256 + 64 * (uint32_t)j;
#pragma unroll
            for (int i = 0; i < 4; ++i) run[g][i] = load_run(xs, off + 16 * i);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
        for (int g = 0; g < GPW; ++g)
            asm volatile("" : "+v"(run[g][0]), "+v"(run[g][1]), "+v"(run[g][2]), "+v"(run[g][3]));
        const u32x4 ones = {one, one, one, one};
#pragma unroll
        for (int g = 0; g < GPW; ++g) {
            act_operands(run[g], a[g]);
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int b = 0; b < 4; ++b) acc = mfma(a[g][b], ones, acc);
            // C rows 4 j + i = tokens, the same in every column n
            if (n == 0) sx_lds[wave][g][j] = acc;
        }
    }

    __builtin_amdgcn_s_setprio(0);
    int slot_i = 0, n_red = 0;
    for (int ti = 0; ti < my_tiles; ++ti) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int g = 0; g < GPW; ++g) {
            if (g >= gw) break;
            // this item's loads have landed; the next D - 1 items' may not
            wait_vm<(D - 1) * L::DMA>();
            const char *slot = my_ring + slot_i * L::BYTES;
            float c = 0.0f;
#pragma unroll
            for (int st = 0; st < K; ++st) {
                const u32x2 w = *reinterpret_cast<const u32x2 *>(
                    slot + 1024 * (st >> 1) + 512 * (st & 1) + n * 32 + j * 8);
                u32x4 b[2][2];
                code_operands_pair(w[0], w[1], mask, one, b);
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < 4; ++q) p = mfma(a[g][q], b[q >> 1][q & 1], p);
                const uint32_t sw = *reinterpret_cast<const uint32_t *>(slot + L::SCALES + 4 * (16 * st + n));
                const uint32_t zw = *reinterpret_cast<const uint32_t *>(slot + L::ZEROS + 4 * (16 * st + n));
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
                const float s4 = 4.0f * s;
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(s4, p[i], acc[i]);
                c = __builtin_fmaf(s, 4.0f + z, c);
            }
            const f32x4 sxg = sx_lds[wave][g][j];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(-c, sxg[i], acc[i]);
            // the slot is free: refill it with the item D ahead
            issue_next();
            if (++slot_i == D) slot_i = 0;
        }
        // end of the tile: the waves' partial sums in wave order. The buffer
        // written here is next written two tiles later, after a barrier that
        // the summing wave reaches only once it has read it.
        red[n_red & 1][wave][lane] = acc;
        __syncthreads();
        if (wave == 0) {
            f32x4 y = red[n_red & 1][0][lane];
#pragma unroll
            for (int v = 1; v < kWaves; ++v) {
                const f32x4 q = red[n_red & 1][v][lane];
                y[0] += q[0]; y[1] += q[1]; y[2] += q[2]; y[3] += q[3];
            }
            // lane: tokens 4 j + i of output row 16 tile + n; 32-bit byte
            // offsets into Y (n_tokens rows < 2^26 x 16 x 4 bytes < 2^32)
            const uint32_t o = (uint32_t)((int)blockIdx.x + ti * (int)gridDim.x) * 16 + (uint32_t)n;
            if (o < (uint32_t)rows) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * j + i < n_tokens)
                        __builtin_amdgcn_raw_buffer_store_b32(
                            __float_as_uint(y[i]), yr, ((uint32_t)(4 * j + i) * (uint32_t)rows + o) * 4,
                            0, 0);
            }
        }
        ++n_red;
    }
    // no DMA load may still write this workgroup's LDS once it ends
    wait_vm<0>();
}

template <typename... Args>
hipError_t launch(void (*kernel)(Args...), int grid, int block, hipStream_t stream, Args... args)
{
    void *argv[] = {static_cast<void *>(&args)...};
    return hipLaunchKernel(reinterpret_cast<const void *>(kernel), dim3(grid), dim3(block),
                           argv, 0, stream);
}

template <bool DEF, int GPW>
hipError_t launch_d(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int n_tokens,
                    float *Y, int grid, hipStream_t stream)
{
    const int64_t pw = rows * cols / 16, pg = rows * cols / 128;
    switch (k) {
    case 1: return launch(batch_kernel<1, DEF, GPW>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt);
    case 2: return launch(batch_kernel<2, DEF, GPW>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt);
    case 3: return launch(batch_kernel<3, DEF, GPW>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt);
    case 4: return launch(batch_kernel<4, DEF, GPW>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt);
    default: return hipErrorInvalidValue;
    }
}

// Groups per wave of a row of cols inputs (the general kernel's 8-wave split).
int64_t groups_per_wave(int64_t cols)
{
    const int64_t gpr = cols / 128;
    return ((gpr + kWaves - 1) / kWaves + 1) / 2 * 2;
}

}  // namespace

bool linear_batch_fits(int64_t rows, int64_t cols, int G, int k, int64_t n_tokens)
{
    // The A operands of a wave's groups (16 tokens x at most 8 groups) fit its
    // registers for cols up to 8 x 8 x 128. The form pays a fixed prologue per
    // workgroup (every wave loads its activations before its first product), so
    // it only gains where each workgroup streams several row tiles: measured
    // ahead of the general kernel from 12288 rows at 4096 columns or fewer (2 to
    // 4 stages), and from 24576 rows for one stage; behind it below.
    const int64_t per_wave = groups_per_wave(cols);
    if (G != 128 || n_tokens < kBatchMinTokens || n_tokens > 16 || per_wave > kMaxGroupsPerWave)
        return false;
    return cols <= 4096 && (k >= 2 ? rows >= 12288 : rows >= 24576);
}

hipError_t launch_linear_batch(const uint32_t *codes, const void *scales, const float *zeros,
                               int64_t rows, int64_t cols, int k, int zero_point, int scale_type,
                               const uint16_t *X, int64_t n_tokens, float *Y, int cus,
                               hipStream_t stream)
{
    const char *sc = static_cast<const char *>(scales);
    const int64_t tiles = (rows + 15) / 16;
    const bool small = groups_per_wave(cols) <= 4;
    const int64_t slots = (int64_t)cus * (small ? wgs_per_cu(4) : wgs_per_cu(8));
    const int grid = (int)(tiles < slots ? tiles : slots);
    const bool def = scale_type == kScaleF32 && zero_point != kZpSymmetric;
    const int nt = (int)n_tokens;
    if (small)
        return def ? launch_d<true, 4>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X,
                                       nt, Y, grid, stream)
                   : launch_d<false, 4>(codes, sc, zeros, rows, cols, k, zero_point, scale_type,
                                        X, nt, Y, grid, stream);
    return def ? launch_d<true, 8>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, nt,
                                   Y, grid, stream)
               : launch_d<false, 8>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X,
                                    nt, Y, grid, stream);
}

}  // namespace rrq_detail

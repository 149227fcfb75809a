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
// 4 + Q), so P = sum x (4 + Q) and Sx = sum x (the same MFMA with a ones
// operand) give sum x Q = P - 4 Sx; every output of an MFMA is used.
//
// Work: wave w of a workgroup's 8 owns the set of groups 4 w .. 4 w + 3 of
// every row (rows of up to 4096 inputs), so its A operands (16 tokens x 4
// groups) are loaded and formed once and stay in registers. A workgroup
// takes 16-row tiles in turn; each wave walks its (tile, stage) items as one
// sequence, accumulating per output (lane: tokens 4 j .. 4 j + 3 of row n)
// the stages' and groups' s P, and per group the stages' s (4 + z). At the
// end of a tile the wave subtracts each group's c Sx and the 8 waves' sums
// meet in LDS, summed in wave order: one barrier per tile.
//
// Memory path (the decode form's): an item's codes (16 rows x the set's 128
// contiguous bytes, one stage), scales and zero-points (16 rows x 4 groups)
// go from HBM straight into a ring of D LDS slots per wave by LDS-DMA loads,
// a fixed count per item; the wave keeps the next D - 1 items in flight and
// waits for exactly the item it is about to read. Code pieces sit in the
// slot XOR-swizzled by row so that an MFMA's 16 rows read distinct banks.
// One accumulator per output takes every group and stage (one per group was
// slower: the compiler then holds more MFMA results), so after the
// matrix-core sum each product term passes through at most 4 k + 11
// roundings (4 k in the wave's sum over stages and groups, 4 with the groups'
// c Sx terms, 7 across the waves), within the 2 n + 24 (n >= 2 k) of the
// error bound of include/rrq.h.
//
// The form's first version streamed each unit (one stage of a tile, every
// group) through a ring shared by the 8 waves, with a barrier per two units;
// per-wave rings with one barrier per tile are 4-15% faster on the Qwen3-8B
// shapes at 2 to 4 stages (24576 x 4096, 16 tokens, 4 / 2 stages: 39.5 /
// 27.7 -> 37.8 / 26.5 us; 6144 x 4096: 18.6 / 14.5 -> 17.3 / 12.4 us).

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
constexpr int kGroupsPerWave = 4;             // A operands held in registers (cols <= 4096)
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

// One item's LDS slot (a 16-row tile, the wave's set of 4 groups, one
// stage): the codes, row r's 16-byte piece p at 128 r + 16 (p ^ (r & 7)) (an
// MFMA's 16 rows then fall on distinct banks but for rows 8 apart); then the
// scales and the zero-points as 32-bit words, row r group g at 4 (4 r + g)
// of their block (a 16-bit scale in the low half).
struct ItemSlot {
    static constexpr int SCALES = 2048;
    static constexpr int ZEROS = SCALES + 256;
    static constexpr int BYTES = ZEROS + 256;
    static constexpr int DMA = 4;               // two 1 KiB code loads, scales, zero-points
};

// One workgroup per CU (up to 256 VGPRs a lane: the A operands of 4 groups
// take 64; two per CU, at 128, spilled from 2 stages and were up to 40%
// slower) and the ring depth its 160 KiB of LDS allows beside the reduction
// buffers and group sums, within the 6-bit vmcnt with the activations' loads.
constexpr int kRedBytes = 2 * kWaves * 64 * 16;
constexpr int kSxBytes = kWaves * kGroupsPerWave * 64;
constexpr int depth_for()
{
    constexpr int by_lds = (160 * 1024 - kRedBytes - kSxBytes) / (kWaves * ItemSlot::BYTES);
    constexpr int by_count = (63 - 4 * kGroupsPerWave) / ItemSlot::DMA;
    return by_lds < by_count ? by_lds : by_count;
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

template <int K, int D, bool DEF>
__global__ __launch_bounds__(64 * kWaves, 2) void batch_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int n_tokens, float *__restrict__ Y,
    int zero_point, int scale_type)
{
    using L = ItemSlot;
    constexpr int GPW = kGroupsPerWave;
    __shared__ __attribute__((aligned(16))) char ring[kWaves][D][L::BYTES];
    __shared__ f32x4 red[2][kWaves][64];
    // group sums of the wave's groups: Sx depends on the token only (lane
    // k-slice j reads tokens 4 j .. 4 j + 3 as one 16-byte broadcast)
    __shared__ f32x4 sx_lds[kWaves][GPW][4];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;
    const int j = lane >> 4;
    const bool sym = zero_point == kZpSymmetric;
    const int gpr = (int)(cols / 128);                  // groups per row
    const int g_begin = GPW * wave;                     // this wave's set
    const int gw = gpr - g_begin < GPW ? (gpr - g_begin > 0 ? gpr - g_begin : 0) : GPW;
    uint32_t mask, one;
    asm volatile("s_mov_b32 %0, %1" : "=s"(mask) : "n"(kCodeMask));
    asm volatile("v_mov_b32 %0, %1" : "=v"(one) : "n"(kOnePair));
    uint32_t four;
    asm volatile("v_mov_b32 %0, %1" : "=v"(four) : "n"(kFourPair));

    const uint32_t row_bytes = (uint32_t)(cols / 4);
    const uint32_t plane_bytes = (uint32_t)plane_words * 4;
    const uint32_t sbytes = scale_type == kScaleF32 ? 4 : 2;
    const u32x4 dc = make_desc(codes, (uint32_t)K * plane_bytes);
    const u32x4 ds = make_desc(scales, (uint32_t)K * (uint32_t)plane_groups * sbytes);
    const u32x4 dz = make_desc(sym ? nullptr : zeros, sym ? 0u : (uint32_t)K * (uint32_t)plane_groups * 4);

    // DMA lane offsets within an item (from the tile's first row of the
    // stage plane, the set's first byte). Codes: load i, lane l -> slot
    // bytes 1024 i + 16 l = row r = 8 i + l / 8, slot piece l % 8, holding
    // the row's piece (l % 8) ^ (r & 7) (8 runs of 128 bytes per load);
    // pieces of groups past the row read nothing. Scales and zero-points:
    // lane l -> row l / 4, group l % 4.
    uint32_t dma_code[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int r = 8 * i + (lane >> 3);
        const int p = (lane & 7) ^ (r & 7);
        dma_code[i] = p < 2 * gw ? (uint32_t)r * row_bytes + 16u * (uint32_t)p : kSkip;
    }
    const int pg = lane & 3;
    const uint32_t pel = (uint32_t)(lane >> 2) * (uint32_t)gpr + (uint32_t)pg;
    const uint32_t dma_scale = pg < gw ? pel * sbytes : kSkip;
    const uint32_t dma_zero = pg < gw ? pel * 4 : kSkip;
    // This lane's reads (B column: row n, k-slice j): group g's 8 code bytes
    // at code_rd[g], its scale and zero-point at par_rd + 4 g.
    uint32_t code_rd[GPW];
#pragma unroll
    for (int g = 0; g < GPW; ++g)
        code_rd[g] = 128u * (uint32_t)n + 16u * (uint32_t)((2 * g + (j >> 1)) ^ (n & 7)) +
                     8u * (uint32_t)(j & 1);
    const uint32_t par_rd = 16u * (uint32_t)n;

    const uint32_t lds_ring = lds_address(&ring[wave][0][0]);
    const char *my_ring = &ring[wave][0][0];

    // Row tiles of this workgroup: blockIdx, blockIdx + grid, ...; items in
    // order: tile t, stage st = item t K + st.
    const int tiles = (int)((rows + 15) / 16);
    const int my_tiles = (int)blockIdx.x < tiles ? (tiles - 1 - (int)blockIdx.x) / (int)gridDim.x + 1 : 0;
    const int total = my_tiles * K;

    // DMA of the items in order, one call per item, position in running
    // counters; items past the end read through descriptors of size 0.
    int issued = 0, is_st = 0, is_slot = 0;
    int is_tile = (int)blockIdx.x;
    auto issue_next = [&]() {
        const bool live = issued < total;
        const uint32_t row0 = live ? (uint32_t)is_tile * 16 : 0u;
        const uint32_t code_off = (uint32_t)is_st * plane_bytes + row0 * row_bytes + (uint32_t)g_begin * 32;
        const uint32_t par_el = (uint32_t)is_st * (uint32_t)plane_groups + row0 * (uint32_t)gpr + (uint32_t)g_begin;
        const uint32_t lds = lds_ring + (uint32_t)is_slot * L::BYTES;
        u32x4 c_src = dc, s_src = ds, z_src = dz;
        if (!live) c_src[2] = s_src[2] = z_src[2] = 0u;
        // the reads of the item that used this slot have completed
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        dma_x4(c_src, code_off, lds, dma_code[0]);
        dma_x4(c_src, code_off, lds + 1024u, dma_code[1]);
        if (DEF || scale_type == kScaleF32)
            dma_dword(s_src, par_el * 4, lds + L::SCALES, dma_scale);
        else
            dma_ushort(s_src, par_el * 2, lds + L::SCALES, dma_scale);
        dma_dword(z_src, par_el * 4, lds + L::ZEROS, dma_zero);
        ++issued;
        if (++is_slot == D) is_slot = 0;
        if (++is_st == K) {
            is_st = 0;
            is_tile += (int)gridDim.x;
        }
    };

    // The activations of this wave's groups first (lane as A row: token n,
    // tokens past n_tokens and groups past the row reading zeros), then the
    // ring's first items; the activations are waited for explicitly, with
    // the runs tied to the wait, leaving the ring's loads in flight.
    u32x4 a[GPW][4];
    {
        const u32x4 xs = make_desc(X, (uint32_t)n_tokens * (uint32_t)cols * 2);
        const uint32_t xrow = (n < n_tokens ? 0u : kSkip) + (uint32_t)n * (uint32_t)cols * 2;
        u32x4 run[GPW][4];
#pragma unroll
        for (int g = 0; g < GPW; ++g) {
            const uint32_t off = (g < gw ? xrow : kSkip) + (uint32_t)(g_begin + g) * 256 + 64 * (uint32_t)j;
#pragma unroll
            for (int i = 0; i < 4; ++i) run[g][i] = load_run(xs, off + 16 * i);
        }
#pragma unroll
        for (int d = 0; d < D; ++d) issue_next();
        wait_vm<D * L::DMA>();
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

    const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
        Y, (short)0, (int)((uint32_t)n_tokens * (uint32_t)rows * 4u), (int)kRsrcWord3);
    int slot_i = 0, n_red = 0;
    for (int ti = 0; ti < my_tiles; ++ti) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        float cz[GPW];
#pragma unroll
        for (int g = 0; g < GPW; ++g) cz[g] = 0.0f;
#pragma unroll
        for (int st = 0; st < K; ++st) {
            // this item's loads have landed; the next D - 1 items' may not
            wait_vm<(D - 1) * L::DMA>();
            const char *slot = my_ring + slot_i * L::BYTES;
            // every group of the set, also past the row (zero activations,
            // zero codes): independent chains to interleave
#pragma unroll
            for (int g = 0; g < GPW; ++g) {
                const u32x2 w = *reinterpret_cast<const u32x2 *>(slot + code_rd[g]);
                u32x4 b[2][2];
                code_operands_pair(w[0], w[1], mask, four, b);
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < 4; ++q) p = mfma(a[g][q], b[q >> 1][q & 1], p);
                const uint32_t sw = *reinterpret_cast<const uint32_t *>(slot + L::SCALES + par_rd + 4 * g);
                const uint32_t zw = *reinterpret_cast<const uint32_t *>(slot + L::ZEROS + par_rd + 4 * g);
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
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(s, p[i], acc[i]);
                cz[g] = __builtin_fmaf(s, 4.0f + z, cz[g]);
            }
            // the slot is free: refill it with the item D ahead
            issue_next();
            if (++slot_i == D) slot_i = 0;
        }

        // end of the tile: less each group's c Sx in group order, then the
        // waves' sums in wave order. The buffer written here is next written
        // two tiles later, after a barrier that the summing wave reaches only
        // once it has read it.
#pragma unroll
        for (int g = 0; g < GPW; ++g) {
            const f32x4 sxg = sx_lds[wave][g][j];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(-cz[g], sxg[i], acc[i]);
        }
        red[n_red & 1][wave][lane] = acc;
        __syncthreads();
        if (wave == 0) {
            f32x4 yo = red[n_red & 1][0][lane];
#pragma unroll
            for (int v = 1; v < kWaves; ++v) {
                const f32x4 q = red[n_red & 1][v][lane];
                yo[0] += q[0]; yo[1] += q[1]; yo[2] += q[2]; yo[3] += q[3];
            }
            // lane: tokens 4 j + i of output row 16 tile + n; 32-bit byte
            // offsets into Y (n_tokens rows < 2^26 x 16 x 4 bytes < 2^32)
            const uint32_t o = (uint32_t)((int)blockIdx.x + ti * (int)gridDim.x) * 16 + (uint32_t)n;
            if (o < (uint32_t)rows) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * j + i < n_tokens)
                        __builtin_amdgcn_raw_buffer_store_b32(
                            __float_as_uint(yo[i]), yr,
                            ((uint32_t)(4 * j + i) * (uint32_t)rows + o) * 4, 0, 0);
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

template <bool DEF>
hipError_t launch_d(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int n_tokens,
                    float *Y, int grid, hipStream_t stream)
{
    constexpr int D = depth_for();
    const int64_t pw = rows * cols / 16, pg = rows * cols / 128;
    switch (k) {
    case 1: return launch(batch_kernel<1, D, DEF>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt);
    case 2: return launch(batch_kernel<2, D, DEF>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt);
    case 3: return launch(batch_kernel<3, D, DEF>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt);
    case 4: return launch(batch_kernel<4, D, DEF>, grid, 64 * kWaves, stream, codes, scales, zeros, rows, cols, pw, pg, X, n_tokens, Y, zp, sdt);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool linear_batch_fits(int64_t rows, int64_t cols, int G, int k, int64_t n_tokens)
{
    // Measured against the general kernel (5, 8 and 16 tokens, packages read
    // from HBM, rows counted in 4096-input equivalents e): ahead from e =
    // 3072 at 4 stages (16 tokens 3072 x 4096: 12.2 against 12.5 us; 4096 x
    // 4096: 12.5 against 13.4), and with up to 8 tokens from 3072 at 3
    // stages, 4096 at 2 and 6144 at 1; with 16 tokens from 6144 at 2 and 3
    // stages and 12288 at 1 (below, a workgroup's fixed start outweighs its
    // few tiles). Rows of fewer than 2048 inputs leave most waves without
    // groups (16384 x 1024: behind at 1, 3 and 4 stages).
    if (G != 128 || n_tokens < kBatchMinTokens || n_tokens > 16 || cols > 4096 || cols < 2048)
        return false;
    const int64_t e = rows * cols / 4096;
    const bool few = n_tokens <= 8;
    switch (k) {
    case 1: return e >= (few ? 6144 : 12288);
    case 2: return e >= (few ? 4096 : 6144);
    case 3: return e >= (few ? 3072 : 6144);
    default: return e >= 3072;
    }
}

hipError_t launch_linear_batch(const uint32_t *codes, const void *scales, const float *zeros,
                               int64_t rows, int64_t cols, int k, int zero_point, int scale_type,
                               const uint16_t *X, int64_t n_tokens, float *Y, int cus,
                               hipStream_t stream)
{
    if (cols > 4096 || n_tokens > 16) return hipErrorInvalidValue;
    const char *sc = static_cast<const char *>(scales);
    const int64_t tiles = (rows + 15) / 16;
    const int grid = (int)(tiles < cus ? tiles : (int64_t)cus);
    const bool def = scale_type == kScaleF32 && zero_point != kZpSymmetric;
    const int nt = (int)n_tokens;
    return def ? launch_d<true>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, nt, Y,
                                grid, stream)
               : launch_d<false>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, nt,
                                 Y, grid, stream);
}

}  // namespace rrq_detail

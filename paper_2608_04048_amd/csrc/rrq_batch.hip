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
// Work: the 8 waves of a workgroup split the groups of a row into contiguous
// ranges of at most 4 (the general kernel's split for 8 waves), so a wave's A
// operands and group sums (16 tokens x its groups) are loaded and formed once
// and stay in registers. A workgroup takes 16-row tiles in turn and streams
// each tile stage by stage: a unit (one stage of the tile's 16 rows, every
// group) goes from HBM into a ring of LDS slots shared by the 8 waves by
// LDS-DMA loads, each wave issuing a fixed share of whole-row code runs and
// 64-element runs of scales and zero-points (a 16-row slice of one group
// would be 16 runs of 32 bytes, and its parameters 64 single words, which
// the memory system serves far below its streaming rate). A wave waits for
// its own shares of the next two units, one barrier then makes every share
// visible, and the wave works on its groups of the units: per group, an
// accumulator of the stages' s P and a sum of the stages' s (4 + z). At
// the end of a tile, per output, the wave adds its groups in order (each
// its stage sum less c Sx) and the 8 waves' partial sums meet in LDS and are
// summed in wave order. After the matrix-core sum each product term passes
// through at most k + 11 roundings (k in its group's stage sum, one with the
// c Sx term, 3 across the wave's groups, 7 across the waves), within the
// 2 n + 24 (n >= 2 k) of the error bound of include/rrq.h.

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

// A unit: one stage of a 16-row tile, every group of the rows, as the
// workgroup's 8 waves share it in LDS: the 16 rows' codes (row r at r RB
// bytes, RB = cols / 4, its 16-byte pieces XOR-swizzled within aligned runs
// of 16 so that an MFMA's 16 rows read distinct banks), then the scales and
// the zero-points of the 16 rows (one 32-bit word per element, group-major:
// row r group g at 16 g + r, so that an MFMA's 16 rows read consecutive
// words; a 16-bit scale in the low half). The waves fetch a unit together,
// each a fixed share of 1 KiB code loads (whole rows) and 64-element
// parameter loads (4 groups of the 16 rows); loads past the unit's end read
// nothing, so every wave issues the same loads per unit.
template <int GPW>
struct Unit {
    static constexpr int CODE = 16 * GPW * kWaves * 32;      // 16 rows of at most GPW x 8 groups
    static constexpr int PAR = 16 * GPW * kWaves * 4;        // 16 rows x groups, one word each
    static constexpr int BYTES = CODE + 2 * PAR;
    static constexpr int CI = CODE / 1024 / kWaves;          // code loads per wave
    static constexpr int PI = PAR / 256 / kWaves;            // loads per wave per parameter buffer
    static constexpr int DMA = CI + 2 * PI;                  // loads per wave per unit
};

// Groups per wave GPW: the A operands of a wave's groups stay in its
// registers (16 tokens x GPW groups, 16 GPW VGPRs); GPW = 4 serves rows of up
// to 4096 inputs. One workgroup per CU.
constexpr int kRedBytes = 2 * kWaves * 64 * 16;

// Units resident: as many as the CU's 160 KiB of LDS holds beside the
// reduction buffers and the group sums. The waves keep all but the two being
// worked on in flight: a unit's slot is refilled only once every wave has
// passed the next barrier, i.e. is done with it.
template <int GPW>
constexpr int unit_slots()
{
    return (160 * 1024 - kRedBytes - kWaves * GPW * 64) / Unit<GPW>::BYTES;
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
__global__ __launch_bounds__(64 * kWaves, 2) void batch_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int n_tokens, float *__restrict__ Y,
    int zero_point, int scale_type)
{
    using U = Unit<GPW>;
    constexpr int NS = unit_slots<GPW>();
    // Two units per barrier (half the barriers, twice the independent chains
    // between them); a loop step covers TPB whole tiles, two where a tile has
    // an odd number of stages, so that every unit's tile is known at compile
    // time.
    constexpr int UPB = 2;
    constexpr int TPB = K % 2 == 0 ? 1 : 2;
    constexpr int PAIRS = TPB * K / UPB;
    // Units in flight: the refills after a barrier overwrite the slots of
    // the UPB units before it, which every wave is done with by then.
    constexpr int D = NS - UPB;
    static_assert(D >= 2 * UPB && D * U::DMA + 4 * GPW <= 63, "unit ring");
    __shared__ __attribute__((aligned(16))) char ring[NS][U::BYTES];
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
    const int cpr = (int)(cols / 64);                   // 16-byte code pieces per row
    uint32_t mask, one;
    asm volatile("s_mov_b32 %0, %1" : "=s"(mask) : "n"(kCodeMask));
    asm volatile("v_mov_b32 %0, %1" : "=v"(one) : "n"(kOnePair));
    uint32_t four;
    asm volatile("v_mov_b32 %0, %1" : "=v"(four) : "n"(kFourPair));

    // This wave's groups: the general kernel's split for 8 waves (ranges of a
    // whole number of 2-group chunks).
    const int per_wave = ((gpr + kWaves - 1) / kWaves + 1) / 2 * 2;
    const int g_begin = per_wave * wave < gpr ? per_wave * wave : gpr;
    const int g_end = g_begin + per_wave < gpr ? g_begin + per_wave : gpr;
    const int gw = g_end - g_begin;                     // 0 .. GPW

    const uint32_t row_bytes = (uint32_t)(cols / 4);
    const uint32_t plane_bytes = (uint32_t)plane_words * 4;
    const uint32_t sbytes = scale_type == kScaleF32 ? 4 : 2;
    const u32x4 dc = make_desc(codes, (uint32_t)K * plane_bytes);
    const u32x4 ds = make_desc(scales, (uint32_t)K * (uint32_t)plane_groups * sbytes);
    const u32x4 dz = make_desc(sym ? nullptr : zeros, sym ? 0u : (uint32_t)K * (uint32_t)plane_groups * 4);
    u32x4 dc0 = dc, ds0 = ds, dz0 = dz;                 // size 0: no access
    dc0[2] = ds0[2] = dz0[2] = 0u;

    // Code pieces within a row are swizzled by XOR with the row's low bits,
    // over the largest run of 16 or fewer pieces that divides the row.
    const int swz = (cpr & -cpr) < 16 ? (cpr & -cpr) - 1 : 15;
    // This lane's loads of a unit (offsets from the unit's first row of the
    // plane): code piece q = 64 (wave CI + i) + lane is row q / cpr, LDS piece
    // q % cpr holding the row's piece (q % cpr) ^ (row & swz); parameter word
    // e = 64 (wave PI + i) + lane holds row e % 16, group e / 16.
    uint32_t v_code[U::CI], v_scale[U::PI], v_zero[U::PI];
#pragma unroll
    for (int i = 0; i < U::CI; ++i) {
        const int q = 64 * (wave * U::CI + i) + lane;
        const int r = q / cpr, c = q - r * cpr;
        v_code[i] = q < 16 * cpr ? (uint32_t)r * row_bytes + (uint32_t)(c ^ (r & swz)) * 16 : kSkip;
    }
#pragma unroll
    for (int i = 0; i < U::PI; ++i) {
        const int e = 64 * (wave * U::PI + i) + lane;
        const uint32_t el = (uint32_t)((e & 15) * gpr + (e >> 4));
        v_scale[i] = e < 16 * gpr ? el * sbytes : kSkip;
        v_zero[i] = e < 16 * gpr ? el * 4 : kSkip;
    }
    // This lane's reads (B column: row n, k-slice j): the 8 code bytes of
    // group g_begin + g at code_rd[g] within a unit, its parameters at
    // par_rd + 64 g.
    uint32_t code_rd[GPW];
#pragma unroll
    for (int g = 0; g < GPW; ++g) {
        const int c = 2 * (g_begin + g) + (j >> 1);
        code_rd[g] = (uint32_t)n * row_bytes + (uint32_t)(c ^ (n & swz)) * 16 + (uint32_t)(j & 1) * 8;
    }
    const uint32_t par_rd = U::CODE + 4 * (uint32_t)(16 * g_begin + n);

    const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
        Y, (short)0, (int)((uint32_t)n_tokens * (uint32_t)rows * 4u), (int)kRsrcWord3);
    const uint32_t lds_ring = lds_address(&ring[0][0]);

    // Row tiles of this workgroup: blockIdx, blockIdx + grid, ...; units in
    // order: tile t, stage st = unit t K + st.
    const int tiles = (int)((rows + 15) / 16);
    const int my_tiles = (int)blockIdx.x < tiles ? (tiles - 1 - (int)blockIdx.x) / (int)gridDim.x + 1 : 0;
    const int n_units = my_tiles * K;

    // DMA of this wave's share of the units in order, one call per unit,
    // position in running counters; units past the end read through
    // descriptors of size 0 (zeros).
    int is_u = 0, is_st = 0, is_slot = 0;
    int is_tile = (int)blockIdx.x;
    auto issue_next = [&]() {
        const bool live = is_u < n_units;
        const uint32_t row0 = live ? (uint32_t)is_tile * 16 : 0u;
        const uint32_t lds = lds_ring + (uint32_t)is_slot * U::BYTES;
        const uint32_t code_off = (uint32_t)is_st * plane_bytes + row0 * row_bytes;
        const uint32_t par_el = (uint32_t)is_st * (uint32_t)plane_groups + row0 * (uint32_t)gpr;
        const u32x4 c_src = live ? dc : dc0, s_src = live ? ds : ds0, z_src = live ? dz : dz0;
#pragma unroll
        for (int i = 0; i < U::CI; ++i)
            dma_x4(c_src, code_off, lds + 1024u * (uint32_t)(wave * U::CI + i), v_code[i]);
#pragma unroll
        for (int i = 0; i < U::PI; ++i) {
            const uint32_t at = 256u * (uint32_t)(wave * U::PI + i);
            if (DEF || scale_type == kScaleF32)
                dma_dword(s_src, par_el * 4, lds + U::CODE + at, v_scale[i]);
            else
                dma_ushort(s_src, par_el * 2, lds + U::CODE + at, v_scale[i]);
            dma_dword(z_src, par_el * 4, lds + U::CODE + U::PAR + at, v_zero[i]);
        }
        ++is_u;
        if (++is_slot == NS) is_slot = 0;
        if (++is_st == K) {
            is_st = 0;
            is_tile += (int)gridDim.x;
        }
    };

    // The ring's first units, then the activations of this wave's groups
    // (lane as A row: token n, tokens past n_tokens reading zeros), waited
    // for explicitly with the runs tied to the wait. The prologue runs at a
    // raised wave priority: it is a serial stretch that every later unit
    // waits for.
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

    // Per tile of the step and group of the wave: acc[t][g] = sum over
    // stages of s P and cz[t][g] = sum over stages of s (4 + z), stage by
    // stage as the units come.
    int slot_i = 0, n_red = 0;
    f32x4 acc[TPB][GPW];
    float cz[TPB][GPW];
#pragma unroll
    for (int t = 0; t < TPB; ++t)
#pragma unroll
        for (int g = 0; g < GPW; ++g) {
            acc[t][g] = f32x4{0.f, 0.f, 0.f, 0.f};
            cz[t][g] = 0.0f;
        }
    // (a last step past this workgroup's tiles reads units through
    // descriptors of size 0, whose sums are never stored)
    for (int tb = 0; tb < my_tiles; tb += TPB) {
#pragma unroll
        for (int pr = 0; pr < PAIRS; ++pr) {
            // this wave's loads of the next UPB units have landed; then every
            // wave's have, and every wave is done with the UPB units before
            // (whose slots the refills below overwrite)
            wait_vm<(D - UPB) * U::DMA>();
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __syncthreads();
#pragma unroll
            for (int h = 0; h < UPB; ++h) {
                const int t = (UPB * pr + h) / K;      // tile of the step
                const char *unit = &ring[slot_i][0];
                // every group slot, also past this wave's range (its
                // activations are zero, the codes there other bytes of the
                // unit): independent chains to interleave; only groups in
                // range enter the tile's sum
#pragma unroll
                for (int g = 0; g < GPW; ++g) {
                    const u32x2 w = *reinterpret_cast<const u32x2 *>(unit + code_rd[g]);
                    u32x4 b[2][2];
                    code_operands_pair(w[0], w[1], mask, four, b);
                    f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int q = 0; q < 4; ++q) p = mfma(a[g][q], b[q >> 1][q & 1], p);
                    const uint32_t sw = *reinterpret_cast<const uint32_t *>(unit + par_rd + 64 * g);
                    const uint32_t zw = *reinterpret_cast<const uint32_t *>(unit + U::PAR + par_rd + 64 * g);
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
                    for (int i = 0; i < 4; ++i) acc[t][g][i] = __builtin_fmaf(s, p[i], acc[t][g][i]);
                    cz[t][g] = __builtin_fmaf(s, 4.0f + z, cz[t][g]);
                }
                if (++slot_i == NS) slot_i = 0;
            }
            // the slots of the units before are free: refill them, UPB units on
#pragma unroll
            for (int h = 0; h < UPB; ++h) issue_next();
        }

        // end of the step's tiles: per output, the wave's groups in order
        // (each its stages' sum less c Sx), then the waves' partial sums in
        // wave order. The buffer written here is next written two tiles
        // later, after a barrier that the summing wave reaches only once it
        // has read it.
#pragma unroll
        for (int t = 0; t < TPB; ++t) {
            f32x4 y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int g = 0; g < GPW; ++g) {
                if (g >= gw) break;
                const f32x4 sxg = sx_lds[wave][g][j];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float v = __builtin_fmaf(-cz[t][g], sxg[i], acc[t][g][i]);
                    y[i] = g == 0 ? v : y[i] + v;
                }
            }
#pragma unroll
            for (int g = 0; g < GPW; ++g) {
                acc[t][g] = f32x4{0.f, 0.f, 0.f, 0.f};
                cz[t][g] = 0.0f;
            }
            red[n_red & 1][wave][lane] = y;
            __syncthreads();
            const int ti = tb + t;
            if (wave == 0 && ti < my_tiles) {
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
    // The A operands of a wave's groups (16 tokens x at most 4 groups) fit its
    // registers for cols up to 8 x 4 x 128. The form pays a fixed prologue per
    // workgroup (every wave loads its activations before its first product), so
    // it only gains where each workgroup streams several row tiles: measured
    // ahead of the general kernel (16 tokens, 4096 columns) from 6144 rows at 2
    // to 4 stages and from 24576 rows at one stage; behind it at 4096 rows, and
    // at one stage up to 12288.
    if (G != 128 || n_tokens < kBatchMinTokens || n_tokens > 16 ||
        groups_per_wave(cols) > kGroupsPerWave)
        return false;
    return k >= 2 ? rows >= 6144 : rows >= 24576;
}

hipError_t launch_linear_batch(const uint32_t *codes, const void *scales, const float *zeros,
                               int64_t rows, int64_t cols, int k, int zero_point, int scale_type,
                               const uint16_t *X, int64_t n_tokens, float *Y, int cus,
                               hipStream_t stream)
{
    if (groups_per_wave(cols) > kGroupsPerWave || n_tokens > 16)
        return hipErrorInvalidValue;
    const char *sc = static_cast<const char *>(scales);
    const int64_t tiles = (rows + 15) / 16;
    const int grid = (int)(tiles < cus ? tiles : (int64_t)cus);
    const bool def = scale_type == kScaleF32 && zero_point != kZpSymmetric;
    const int nt = (int)n_tokens;
    return def ? launch_d<true, kGroupsPerWave>(codes, sc, zeros, rows, cols, k, zero_point,
                                                scale_type, X, nt, Y, grid, stream)
               : launch_d<false, kGroupsPerWave>(codes, sc, zeros, rows, cols, k, zero_point,
                                                 scale_type, X, nt, Y, grid, stream);
}

}  // namespace rrq_detail

// Stage-sum linear layer on an RRQ package (the prefill / decode product of
// Eq. 20): Y[m][o] = sum over the first K stages t and inputs i of
// X[m][i] (Q_t[o][i] - z_t) s_t, with X bfloat16 [M][cols] and Y binary32
// [M][rows], on gfx950 matrix cores.
//
// Per group g of G inputs and stage t the sum over the group factors as
//   s_t (sum_i x_i Q_i - z_t sum_i x_i),
// and both inner sums run on v_mfma_f32_16x16x32_bf16 with fp32 accumulation:
//   * A operand: 16 token rows x 32 inputs of X (bfloat16, exact);
//   * B operand: 32 inputs x 16 output rows of codes, each code Q encoded as
//     the bfloat16 4 + Q (bits 0x4080 | Q << 5: the code lands in the top
//     two mantissa bits of 4 with one shift and one AND-OR per pair of
//     codes), so the MFMA yields P_t = sum x (4 + Q) and sum x Q = P_t - 4 Sx
//     exactly in real arithmetic;
//   * Sx = sum x over the group comes from the same MFMA with a B operand of
//     bfloat16 ones.
// The group's contribution sum_t s_t (P_t - (4 + z_t) Sx) is added to the
// lane's fp32 accumulators as sum_t s_t P_t (one fused multiply-add per
// output and stage) minus c Sx with c = sum_t s_t (4 + z_t) (one per output
// and group). Every product of the MFMAs is exact; fp32 rounding enters only
// in the accumulations (error bound in the tests).
//
// Work split: a workgroup of NW waves owns 16 output rows; the groups of a
// row are split into NW contiguous ranges, one per wave, and each wave walks
// its range in chunks of 2 groups. The partial results are summed through
// LDS in wave order (deterministic). Up to 4 tokens are served by one pass
// over the package with 8 waves per workgroup; more tokens go 16 at a time
// with 4 waves (a chunk's activations take 4 times the LDS).
//
// Memory path: everything a chunk needs (codes of 16 rows per stage, scales
// and zero-points, activations of the tile's tokens) goes from memory
// straight into LDS with LDS-DMA buffer loads and is read back in the MFMA
// operand layout. Every wave double-buffers its chunks, so the next chunk is
// in flight while the current one is computed. The DMA instructions are
// issued from inline assembly, a fixed number per chunk, and the wave waits
// for exactly the chunk it is about to read (s_waitcnt vmcnt(n) with n = one
// chunk's instructions); no other vector-memory loads are issued in the
// loop. LDS slots are XOR-swizzled so that the reads of 16 rows (or of the
// tile's tokens) fall in distinct banks.

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

constexpr uint32_t kOnePair = 0x3F803F80u;    // two bfloat16 1.0
constexpr uint32_t kFourPair = 0x40804080u;    // two bfloat16 4.0: code operands 4 + Q
constexpr uint32_t kCodeMask = 0x00600060u;   // top two mantissa bits of both halves

// Package stage format (values of the C ABI's enums).
constexpr int kZpSymmetric = 2;
constexpr int kScaleF32 = 0, kScaleF16 = 1;

// Waves per workgroup for a token tile of TT.
constexpr int tile_waves(int TT) { return TT == 4 ? 8 : 4; }

// LDS image of one chunk of 2 groups (per wave and buffer), in 16-byte
// slots:
//   codes   K stages x 16 rows x RB = G / 2 bytes (a stage takes at least
//           the 1 KiB one DMA instruction writes),
//   scales  K stages x 16 rows x 2 groups, one dword each (a stage takes
//           the 256 bytes one dword DMA writes),
//   zeros   the same,
//   X       TT tokens x 2 G inputs x 2 bytes (whole KiB: the DMA lanes past
//           the last token read zeros into the padding).
template <int G, int K, int TT>
struct Chunk {
    static constexpr int NW = tile_waves(TT);
    static constexpr int CG = 2;                                  // groups per chunk
    static constexpr int RB = CG * G / 4;                         // code bytes per row
    static constexpr int SLOTS = RB / 16;                         // code slots per row
    static constexpr int CODE_BYTES = 16 * RB > 1024 ? 16 * RB : 1024;
    static constexpr int CODE_DMA = CODE_BYTES / 1024;            // per stage
    static constexpr int PARAM_BYTES = 256;
    static constexpr int SCALES = K * CODE_BYTES;
    static constexpr int ZEROS = SCALES + K * PARAM_BYTES;
    static constexpr int XOFF = ZEROS + K * PARAM_BYTES;
    static constexpr int X_ROW = CG * G * 2;                      // one token
    static constexpr int X_SLOTS = X_ROW / 16;
    static constexpr int X_DMA = (TT * X_ROW + 1023) / 1024;
    static constexpr int BYTES = XOFF + X_DMA * 1024;
    // DMA instructions per chunk: what one wait leaves in flight
    static constexpr int DMA = K * (CODE_DMA + 2) + X_DMA;
    static_assert(DMA <= 31, "two chunks in flight must fit the vmcnt counter");
    static_assert(16 * CG * 4 <= PARAM_BYTES, "chunk shape");

    // Slot k of code row r holds the row's piece k ^ code_swizzle(r): rows
    // that share LDS banks (256 / RB rows apart) get different slots.
    static __device__ __forceinline__ int code_swizzle(int r)
    {
        return SLOTS > 1 ? (r * RB / 256) & (SLOTS - 1) : 0;
    }
    // Slot p of token row tk holds piece p ^ x_swizzle(tk): token rows that
    // share banks get different slots where the row has enough of them.
    static __device__ __forceinline__ int x_swizzle(int tk)
    {
        return (TT == 4 ? 4 * tk : tk) & (X_SLOTS - 1);
    }
};

__device__ __forceinline__ f32x4 mfma(const u32x4 &a, const u32x4 &b, const f32x4 &c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// B operand of one block: codes q = 0..3 of the (pre-shifted) word w sit at
// bits 2q and 16 + 2q; register q gets codes q and q + 8 as 4 + code.
// mask and four hold kCodeMask and kFourPair in registers, so that each
// register costs a shift and one AND-OR.
__device__ __forceinline__ u32x4 code_operand(uint32_t w, uint32_t mask, uint32_t four)
{
    u32x4 b;
    b[0] = ((w << 5) & mask) | four;
    b[1] = ((w << 3) & mask) | four;
    b[2] = ((w << 1) & mask) | four;
    b[3] = ((w >> 1) & mask) | four;
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

// Buffers of one row tile and token tile: one descriptor per package
// array, from the row tile in stage 0 to its end in stage K - 1, and the
// byte stride between stage planes (the loads' scalar offset). Rows past
// the last row read the next plane's data (never used) or, in the last
// plane, zeros.
struct Sources {
    u32x4 codes, scales, zeros;
    uint32_t code_plane, scale_plane, zero_plane;
    u32x4 x;
    uint32_t row_bytes;   // code bytes per row: cols / 4
    uint32_t gpr;         // groups per row
    uint32_t x_row;       // activation bytes per token: cols * 2
    uint32_t m_here;      // live tokens of the tile
    int scale_type;
};

// Issue the DMA of the chunk whose first group is g0 into the LDS buffer
// at byte address lds: Chunk<G, K, TT>::DMA instructions, whatever the
// format (symmetric stages read zeros through a zero-sized descriptor,
// tokens past the tile read zeros without touching memory). Code rows past
// the tile and inputs past the row read zeros or other rows' data: those
// groups are never computed.
template <int G, int K, int TT>
__device__ __forceinline__ void load_chunk(uint32_t lds, const Sources &src, uint32_t g0,
                                           int lane)
{
    using C = Chunk<G, K, TT>;
    // the reads of the previous chunk in this buffer have completed
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    const uint32_t cbase = g0 * (G / 4);
#pragma unroll
    for (int t = 0; t < K; ++t) {
#pragma unroll
        for (int i = 0; i < C::CODE_DMA; ++i) {
            const int sl = i * 64 + lane;
            const int rho = sl / C::SLOTS;
            const int k = sl % C::SLOTS;
            // lanes past row 15 fill the stage's padding (with row 0's data)
            const uint32_t off = rho < 16 ? (uint32_t)rho * src.row_bytes + cbase +
                                                16u * (uint32_t)(k ^ C::code_swizzle(rho))
                                          : 0u;
            dma_x4(src.codes, t * src.code_plane, lds + t * C::CODE_BYTES + i * 1024, off);
        }
    }
    // scales and zero-points: lane l -> row l / CG, group g0 + l % CG (lanes
    // past row 15 fill the padding with group 0)
    const int prow = lane / C::CG;
    const uint32_t gi = prow < 16 ? (uint32_t)prow * src.gpr + g0 + (uint32_t)(lane % C::CG) : 0u;
#pragma unroll
    for (int t = 0; t < K; ++t) {
        if (src.scale_type == kScaleF32)
            dma_dword(src.scales, t * src.scale_plane, lds + C::SCALES + t * C::PARAM_BYTES, gi * 4);
        else
            dma_ushort(src.scales, t * src.scale_plane, lds + C::SCALES + t * C::PARAM_BYTES, gi * 2);
        dma_dword(src.zeros, t * src.zero_plane, lds + C::ZEROS + t * C::PARAM_BYTES, gi * 4);
    }
    const uint32_t xbase = g0 * (G * 2);
#pragma unroll
    for (int i = 0; i < C::X_DMA; ++i) {
        const int sl = i * 64 + lane;
        const int tk = sl / C::X_SLOTS;
        const int pc = sl % C::X_SLOTS;
        const uint32_t off = ((uint32_t)tk < src.m_here ? 0u : kSkip) + (uint32_t)tk * src.x_row +
                             xbase + 16u * (uint32_t)(pc ^ C::x_swizzle(tk));
        dma_x4(src.x, 0u, lds + C::XOFF + i * 1024, off);
    }
}

// Lane layout (lane l: A row / B column r = l % 16, k-slice j = l / 16).
// A group's 128 / 64 / 32 inputs form 4 / 2 / 1 MFMA blocks:
//   G = 128: lane j takes code words 2j, 2j + 1 of the group; block b takes
//            word 2j + b / 2, half b % 2.
//   G = 64:  lane j takes word j; block b takes its half b.
//   G = 32:  lanes j = 2w, 2w + 1 share word w; block 0 takes half j % 2.
// Half h of a word holds the element pairs (p, p + 8), p = 4h .. 4h + 3.
//
// Adds the first n_groups groups (1..CG, wave-uniform) of the chunk in the
// LDS buffer lds to acc; the lane's A row is token tk of the tile. DEF: the
// default stage format (binary32 scales, stored zero-points), with no format
// branches; otherwise scale_type and sym are read at run time.
template <int G, int K, int TT, bool DEF>
__device__ __forceinline__ void compute_chunk(const char *lds, int n_groups, int r, int j, int tk,
                                              int scale_type, bool sym, uint32_t mask,
                                              uint32_t one, uint32_t four, f32x4 &acc)
{
    using C = Chunk<G, K, TT>;
    constexpr int CG = C::CG;
    constexpr int NB = G / 32;
    const u32x4 ones = {one, one, one, one};
    // s_t and c = sum_t s_t (4 + z_t) per group of the lane's row
    float s4[K][CG], c[CG];
#pragma unroll
    for (int q = 0; q < CG; ++q) c[q] = 0.0f;
#pragma unroll
    for (int t = 0; t < K; ++t) {
        const u32x2 sv = *reinterpret_cast<const u32x2 *>(lds + C::SCALES + t * C::PARAM_BYTES + 8 * r);
        const u32x2 zv = *reinterpret_cast<const u32x2 *>(lds + C::ZEROS + t * C::PARAM_BYTES + 8 * r);
#pragma unroll
        for (int q = 0; q < CG; ++q) {
            float s, z;
            if constexpr (DEF) {
                s = __uint_as_float(sv[q]);
                z = __uint_as_float(zv[q]);
            } else {
                s = scale_type == kScaleF32 ? __uint_as_float(sv[q])
                    : scale_type == kScaleF16
                        ? (float)__builtin_bit_cast(_Float16, (uint16_t)(sv[q] & 0xFFFFu))
                        : __uint_as_float(sv[q] << 16);
                z = sym ? 2.0f : __uint_as_float(zv[q]);
            }
            s4[t][q] = s;
            c[q] = __builtin_fmaf(s, 4.0f + z, c[q]);
        }
    }
    const char *xl = lds + C::XOFF + tk * C::X_ROW;
    const int xs = C::x_swizzle(tk);
    const int cs = C::code_swizzle(r);
#pragma unroll
    for (int q = 0; q < CG; ++q) {
        if (q >= n_groups) break;
        // activations of the lane's token and k-slice
        u32x4 a[NB];
        if constexpr (G == 128) {
            uint32_t x[16];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const u32x4 d = *reinterpret_cast<const u32x4 *>(xl + 16 * ((q * 16 + 4 * j + v) ^ xs));
                x[4 * v] = d[0]; x[4 * v + 1] = d[1]; x[4 * v + 2] = d[2]; x[4 * v + 3] = d[3];
            }
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const int base = 8 * (b >> 1) + 2 * (b & 1);
                a[b] = act_operand((u32x2){x[base], x[base + 1]}, (u32x2){x[base + 4], x[base + 5]});
            }
        } else if constexpr (G == 64) {
            uint32_t x[8];
#pragma unroll
            for (int v = 0; v < 2; ++v) {
                const u32x4 d = *reinterpret_cast<const u32x4 *>(xl + 16 * ((q * 8 + 2 * j + v) ^ xs));
                x[4 * v] = d[0]; x[4 * v + 1] = d[1]; x[4 * v + 2] = d[2]; x[4 * v + 3] = d[3];
            }
#pragma unroll
            for (int b = 0; b < NB; ++b)
                a[b] = act_operand((u32x2){x[2 * b], x[2 * b + 1]}, (u32x2){x[2 * b + 4], x[2 * b + 5]});
        } else {
            // inputs 16 w + 4h .. + 3 and 16 w + 8 + 4h .. + 3 of the group,
            // w = j / 2, h = j % 2: 8 bytes at 8h in pieces 2w and 2w + 1
            const int piece = q * 4 + 2 * (j >> 1);
            const int h8 = 8 * (j & 1);
            const u32x2 lo = *reinterpret_cast<const u32x2 *>(xl + 16 * (piece ^ xs) + h8);
            const u32x2 hi = *reinterpret_cast<const u32x2 *>(xl + 16 * ((piece + 1) ^ xs) + h8);
            a[0] = act_operand(lo, hi);
        }
        f32x4 sx = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int b = 0; b < NB; ++b) sx = mfma(a[b], ones, sx);
#pragma unroll
        for (int t = 0; t < K; ++t) {
            const char *row = lds + t * C::CODE_BYTES + r * C::RB;
            f32x4 pq = {0.f, 0.f, 0.f, 0.f};
            if constexpr (G == 128) {
                const u32x2 w = *reinterpret_cast<const u32x2 *>(
                    row + 16 * ((2 * q + (j >> 1)) ^ cs) + 8 * (j & 1));
                u32x4 bop[2][2];
                code_operands_pair(w[0], w[1], mask, four, bop);
#pragma unroll
                for (int b = 0; b < NB; ++b) pq = mfma(a[b], bop[b >> 1][b & 1], pq);
            } else if constexpr (G == 64) {
                const uint32_t word = *reinterpret_cast<const uint32_t *>(row + 16 * (q ^ cs) + 4 * j);
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    pq = mfma(a[b], code_operand(b ? word >> 8 : word, mask, four), pq);
            } else {
                const uint32_t word = *reinterpret_cast<const uint32_t *>(
                    row + 16 * ((q >> 1) ^ cs) + 8 * (q & 1) + 4 * (j >> 1));
                pq = mfma(a[0], code_operand((j & 1) ? word >> 8 : word, mask, four), pq);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(s4[t][q], pq[i], acc[i]);
        }
        // - c Sx, c = sum_t s_t (4 + z_t)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(-c[q], sx[i], acc[i]);
    }
}

template <int G, int K, int TT, bool DEF>
__global__ __launch_bounds__(64 * tile_waves(TT)) void linear_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int64_t n_tokens,
    float *__restrict__ Y, int zero_point, int scale_type)
{
    using C = Chunk<G, K, TT>;
    constexpr int CG = C::CG;
    constexpr int NW = C::NW;
    // two chunk buffers per wave
    __shared__ __attribute__((aligned(16))) char buf[2][NW][C::BYTES];
    __shared__ f32x4 red[NW][64];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r = lane & 15;            // B column (output row) and A row (token)
    const int j = lane >> 4;            // k-slice
    const int tk = r < TT ? r : TT - 1; // A rows past the tile repeat its last token
    const bool sym = zero_point == kZpSymmetric;
    // the code operand's constants in registers (opaque to constant folding,
    // so that the AND and OR fuse)
    uint32_t mask, one;
    asm volatile("s_mov_b32 %0, %1" : "=s"(mask) : "n"(kCodeMask));
    asm volatile("v_mov_b32 %0, %1" : "=v"(one) : "n"(kOnePair));
    uint32_t four;
    asm volatile("v_mov_b32 %0, %1" : "=v"(four) : "n"(kFourPair));

    const int64_t o0 = (int64_t)blockIdx.x * 16;
    const uint32_t rows_here = (uint32_t)(rows - o0 < 16 ? rows - o0 : 16);
    const int64_t gpr = cols / G;       // groups per row
    const int64_t wpr = cols / 16;      // code words per row
    // This wave's contiguous range of groups, a whole number of chunks.
    const int64_t per_wave = ((gpr + NW - 1) / NW + CG - 1) / CG * CG;
    const int64_t g_begin = per_wave * wave < gpr ? per_wave * wave : gpr;
    const int64_t g_end = g_begin + per_wave < gpr ? g_begin + per_wave : gpr;
    const int n_chunks = (int)((g_end - g_begin + CG - 1) / CG);

    // Package buffers of this row tile (rows past the end read zero).
    Sources src;
    const uint32_t sbytes = scale_type == kScaleF32 ? 4 : 2;
    src.code_plane = (uint32_t)plane_words * 4;
    src.scale_plane = (uint32_t)plane_groups * sbytes;
    src.zero_plane = (uint32_t)plane_groups * 4;
    src.codes = make_desc(codes + o0 * wpr,
                          (K - 1) * src.code_plane + rows_here * (uint32_t)wpr * 4);
    src.scales = make_desc(scales + o0 * gpr * sbytes,
                           (K - 1) * src.scale_plane + rows_here * (uint32_t)gpr * sbytes);
    src.zeros = make_desc(sym ? nullptr : zeros + o0 * gpr,
                          sym ? 0u : (K - 1) * src.zero_plane + rows_here * (uint32_t)gpr * 4);
    src.row_bytes = (uint32_t)wpr * 4;
    src.gpr = (uint32_t)gpr;
    src.x_row = (uint32_t)cols * 2;
    src.scale_type = scale_type;
    const uint32_t lds_a = (uint32_t)reinterpret_cast<uintptr_t>(
        (__attribute__((address_space(3))) char *)&buf[0][wave][0]);
    const uint32_t lds_b = (uint32_t)reinterpret_cast<uintptr_t>(
        (__attribute__((address_space(3))) char *)&buf[1][wave][0]);
    const char *la = &buf[0][wave][0];
    const char *lb = &buf[1][wave][0];

    for (int64_t m0 = 0; m0 < n_tokens; m0 += TT) {
        src.m_here = (uint32_t)(n_tokens - m0 < TT ? n_tokens - m0 : TT);
        src.x = make_desc(X + m0 * cols, src.m_here * src.x_row);

        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        const uint32_t g0 = (uint32_t)g_begin;
        if (n_chunks > 0) load_chunk<G, K, TT>(lds_a, src, g0, lane);
        if (n_chunks > 1) load_chunk<G, K, TT>(lds_b, src, g0 + CG, lane);
        for (int c = 0; c < n_chunks; c += 2) {
            const uint32_t ga = g0 + (uint32_t)c * CG;
            const int na = (int)(g_end - ga < CG ? g_end - ga : CG);
            // chunk c is in buffer a; chunk c + 1, if any, may stay in flight
            if (c + 1 < n_chunks) wait_vm<C::DMA>(); else wait_vm<0>();
            compute_chunk<G, K, TT, DEF>(la, na, r, j, tk, scale_type, sym, mask, one, four, acc);
            if (c + 2 < n_chunks) load_chunk<G, K, TT>(lds_a, src, ga + 2 * CG, lane);
            if (c + 1 >= n_chunks) break;
            const uint32_t gb = ga + CG;
            const int nb = (int)(g_end - gb < CG ? g_end - gb : CG);
            if (c + 2 < n_chunks) wait_vm<C::DMA>(); else wait_vm<0>();
            compute_chunk<G, K, TT, DEF>(lb, nb, r, j, tk, scale_type, sym, mask, one, four, acc);
            if (c + 3 < n_chunks) load_chunk<G, K, TT>(lds_b, src, gb + 2 * CG, lane);
        }

        // Sum the waves' partial results in wave order and store: lane l
        // holds tokens m0 + 4 j + i of output row o0 + r.
        red[wave][lane] = acc;
        __syncthreads();
        if (wave == 0 && 4 * j < TT) {
            f32x4 y = red[0][lane];
#pragma unroll
            for (int v = 1; v < NW; ++v) {
                const f32x4 q = red[v][lane];
                y[0] += q[0]; y[1] += q[1]; y[2] += q[2]; y[3] += q[3];
            }
            if ((uint32_t)r < rows_here) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if ((uint32_t)(4 * j + i) < src.m_here) Y[(m0 + 4 * j + i) * rows + o0 + r] = y[i];
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

template <int G, int TT, bool DEF>
hipError_t launch_linear_gtd(const uint32_t *codes, const char *scales, const float *zeros,
                             int64_t rows, int64_t cols, int k, int zp, int sdt, const uint16_t *X,
                             int64_t n_tokens, float *Y, hipStream_t stream)
{
    const int64_t plane_words = rows * cols / 16;
    const int64_t plane_groups = rows * cols / G;
    const int grid = (int)((rows + 15) / 16);
    const int block = 64 * tile_waves(TT);
    switch (k) {
    case 1: return launch(linear_kernel<G, 1, TT, DEF>, grid, block, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y, zp, sdt);
    case 2: return launch(linear_kernel<G, 2, TT, DEF>, grid, block, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y, zp, sdt);
    case 3: return launch(linear_kernel<G, 3, TT, DEF>, grid, block, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y, zp, sdt);
    case 4: return launch(linear_kernel<G, 4, TT, DEF>, grid, block, stream, codes, scales, zeros, rows, cols, plane_words, plane_groups, X, n_tokens, Y, zp, sdt);
    default: return hipErrorInvalidValue;
    }
}

// Up to 4 tokens: one pass with 4-token tiles; more: 16-token tiles. The
// default format (binary32 scales, stored zero-points) has its own kernels.
template <int G>
hipError_t launch_linear_g(const uint32_t *codes, const char *scales, const float *zeros,
                           int64_t rows, int64_t cols, int k, int zp, int sdt, const uint16_t *X,
                           int64_t n_tokens, float *Y, hipStream_t stream)
{
    const bool def = sdt == kScaleF32 && zp != kZpSymmetric;
    if (n_tokens <= 4)
        return def ? launch_linear_gtd<G, 4, true>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, stream)
                   : launch_linear_gtd<G, 4, false>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, stream);
    return def ? launch_linear_gtd<G, 16, true>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, stream)
               : launch_linear_gtd<G, 16, false>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, stream);
}

}  // namespace

hipError_t launch_linear(const uint32_t *codes, const void *scales, const float *zeros,
                         int64_t rows, int64_t cols, int G, int S, int k, int zero_point,
                         int scale_type, const uint16_t *X, int64_t n_tokens, float *Y,
                         hipStream_t stream)
{
    const char *sc = static_cast<const char *>(scales);
    (void)S;
    switch (G) {
    case 32: return launch_linear_g<32>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, n_tokens, Y, stream);
    case 64: return launch_linear_g<64>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, n_tokens, Y, stream);
    case 128: return launch_linear_g<128>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, n_tokens, Y, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace rrq_detail

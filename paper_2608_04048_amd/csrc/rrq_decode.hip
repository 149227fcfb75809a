// Decode form of the stage-sum linear layer (Eq. 20) for up to 4 tokens (5
// to 16 on rows of 4096 inputs) and groups of 128: Y[m][o] = sum over stages
// t < K and groups g of
// s_t,o,g (sum_i x_m,i Q_t,o,i - z_t,o,g sum_i x_m,i), the product
// rrq_linear.hip computes for any shape, organised here for streaming the
// package from HBM at full width when the activations are few.
//
// Matrix-core mapping (v_mfma_f32_16x16x32_bf16, lane l: row / column
// n = l % 16, k-slice j = l / 16):
//   * B columns are 4 output rows x 4 consecutive groups (n = 4 r + g'); lane
//     j owns inputs 32 j .. 32 j + 31 of its group, i.e. 8 contiguous bytes
//     of codes per stage. Codes become the bfloat16 4 + Q (one shift and
//     one AND-OR per pair of codes, codes q and q + 8 of a word per register);
//   * A rows are 4 tokens x the same 4 groups (m = 4 t + g), so C[m][n] is a
//     group's dot product only on the diagonal g = g': lane l keeps all four
//     of its C rows (tokens j, groups 0..3) and uses row g' = n % 4 at the end;
//   * a wave works on a fixed range of columns (its sets of 4 groups), so its
//     A operands (the activations, in pairs (x[v], x[v + 8]) of every 16
//     inputs) and the group sums Sx (from the same MFMA with a ones operand)
//     are loaded and formed once and stay in registers.
// With 5 to 8 (9 to 16) tokens, TQ = 2 (4) quads of 4 tokens, each quad has
// its own A operands and group sums, and a stage's B operands serve every
// quad's MFMAs: the operand building, most of the instruction count, is
// shared.
// Each lane accumulates sum over stages of s P - (sum over stages of
// s (4 + z)) Sx for its token, row and group (P = sum x (4 + Q) = 4 Sx +
// sum x Q); the four
// groups of a set are summed across lanes and the waves' column ranges
// through LDS, in a fixed order. Every matrix-core product is exact; fp32
// rounding is in the accumulations only.
//
// Work: the waves of a workgroup (8; 12 and 16 on rows of 12288 and 16384
// inputs) split every 4-row tile's columns, so at any moment a workgroup
// reads whole rows and neighbouring workgroups read neighbouring rows; a
// workgroup takes batches of consecutive tiles in turn.
// Each wave walks its (tile, set) items as one sequence.
//
// Memory path: an item's codes (4 rows x 128 contiguous bytes per stage),
// scales and zero-points go from HBM straight into a ring of D LDS slots per
// wave by LDS-DMA loads: one 1 KiB load per two stages of codes, one load
// for the scales and one for the zero-points of all stages, a fixed count
// per item. The wave keeps the next D - 1 items in flight and waits for
// exactly the item it is about to read (s_waitcnt vmcnt with the later
// items' load count); with no register destinations there is nothing for
// the compiler to drain at the loop's back edge. Each lane then reads its 8
// code bytes per stage and its scales and zero-points from the slot: the 64
// lanes' code reads cover the stage's 512 bytes once, so they are free of
// bank conflicts.

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

// One item's LDS slot (a 4-row tile and a set of 4 groups, all K stages):
// codes of stage t at 1024 (t / 2) + 512 (t % 2), row-major 4 x 128 bytes;
// scales and zero-points as 32-bit words, stage t of pair n = 4 row + group
// at 4 (16 t + n) of their block.
template <int K>
struct ItemSlot {
    static constexpr int CODE_DMA = (K + 1) / 2;   // 1 KiB loads, two stages each
    static constexpr int SCALES = CODE_DMA * 1024;
    static constexpr int ZEROS = SCALES + 256;
    static constexpr int BYTES = ZEROS + 256;
    static constexpr int DMA = CODE_DMA + 2;       // vector-memory loads per item
};

// Partial row sums of a batch of up to kBatch tiles, double-buffered.
constexpr int kBatch = 8;
constexpr int red_bytes(int wv, int tq) { return 2 * wv * kBatch * 16 * tq * 4; }

// Waves per workgroup (WV) and sets of 4 groups per wave (SPW) by the sets
// in a row (cols / 512; up to 4 tokens): 8 x 1 and 8 x 2 for rows of 4096
// and 8192 inputs, 12 x 2 and 16 x 2 for 12288 and 16384. A set's A operands
// take 16 VGPRs for the whole call, so at 3 sets per wave the 8-wave
// workgroup fitted only once per CU (two waves per SIMD; twice it spilled at 4
// stages); 12 or 16 waves of 2 sets keep 3 or 4 waves per SIMD busy
// (measured 4096 x 12288 at 4 / 2 stages: 21.9 / 14.8 -> 19.3 / 13.9 us,
// 4096 x 16384: 27.4 / 18.9 -> 25.7 / 16.6 us).
constexpr int waves_for(int sets) { return sets <= 16 ? 8 : sets / 2; }
constexpr int sets_per_wave(int sets) { return sets / waves_for(sets); }

// Workgroups per CU: three with 8 waves of one set of 4 groups (at most 85
// VGPRs: 24 waves per CU give the slow-issue integer work of the code
// operands more waves to pair with; measured 2-6% faster than two on the
// Qwen3-8B shapes at 2 to 4 stages, rings 2-3 items deep instead of 3-5),
// two with 8 waves of 2 sets (at most 128 VGPRs), one with 12 or 16 waves.
// The rings share the CU's 160 KiB of LDS with the reduction buffers
// accordingly. With 5 to 8 tokens (two quads of tokens, 8 waves of one set)
// the A operands take 32 VGPRs: two workgroups per CU, with the larger
// reduction buffers; with 9 to 16 (four quads) 64: one.
constexpr int wgs_per_cu(int wv, int spw, int tq)
{
    return wv > 8 || tq > 2 ? 1 : tq > 1 ? 2 : spw == 1 ? 3 : 2;
}
constexpr int ring_bytes(int wv, int spw, int tq)
{
    return wgs_per_cu(wv, spw, tq) == 3   ? 44 * 1024
           : wgs_per_cu(wv, spw, tq) == 2 ? 64 * 1024 - 8 * 1024 * (tq - 1)
                                          : 160 * 1024 - red_bytes(wv, tq);
}

// Ring depth: as deep as the 6-bit vmcnt counter (all in-flight items'
// loads) and the LDS for the waves' rings allow, at most 16.
template <int K, int WV, int SPW, int TQ>
constexpr int depth_for()
{
    constexpr int by_count = 63 / ItemSlot<K>::DMA;
    constexpr int by_lds = ring_bytes(WV, SPW, TQ) / (WV * ItemSlot<K>::BYTES);
    constexpr int d = by_count < by_lds ? by_count : by_lds;
    return d < 16 ? d : 16;
}

// A operands of one set of 4 groups for the lane (token t, group g, k-slice
// j) from its 32 inputs 32 j .. 32 j + 31 of group g, as four runs of 8
// (x[32 j .. +7], [+8 .. +15], [+16 .. +23], [+24 .. +31]): block b = 16-input
// run 2 j + b / 2, half b % 2, register v = (x[v'], x[v' + 8]) of the run's
// half.
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

// Activation run loaded behind the compiler's back: the loads are issued
// before the ring's first DMA loads and waited for explicitly, so that the
// wait does not also drain the ring (a compiler-visible load would be
// followed by a full drain, as the compiler does not count the DMA loads).
// The value is only read after wait_runs.
__device__ __forceinline__ u32x4 load_run(const u32x4 &desc, uint32_t voff)
{
    u32x4 v;
    asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen" : "=v"(v) : "v"(voff), "s"(desc));
    return v;
}

// Wait until at most N vector-memory loads are in flight, with the runs as
// operands, so that no use of them can move above the wait.
template <int N, int SPW>
__device__ __forceinline__ void wait_runs(u32x4 (&run)[SPW][4])
{
    if constexpr (SPW == 1) {
        asm volatile("s_waitcnt vmcnt(%4)"
                     : "+v"(run[0][0]), "+v"(run[0][1]), "+v"(run[0][2]), "+v"(run[0][3])
                     : "n"(N) : "memory");
    } else {
        asm volatile("s_waitcnt vmcnt(%4)"
                     : "+v"(run[0][0]), "+v"(run[0][1]), "+v"(run[0][2]), "+v"(run[0][3])
                     : "n"(N) : "memory");
#pragma unroll
        for (int s = 1; s < SPW; ++s)
            asm volatile(""
                         : "+v"(run[s][0]), "+v"(run[s][1]), "+v"(run[s][2]), "+v"(run[s][3])
                         :: "memory");
    }
}

// Workgroup: WV waves share each 4-row tile, wave w taking sets
// w SPW .. w SPW + SPW - 1 of its WV SPW sets of 4 groups (so the waves of a
// workgroup read whole rows together); a batch of up to 8 consecutive tiles
// is reduced across the waves through LDS. Batches go to workgroups in turn.
template <int K, int D, int WV, int SPW, int TQ, bool DEF>
__global__ __launch_bounds__(64 * WV, WV * wgs_per_cu(WV, SPW, TQ) / 4) void decode_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int n_tokens, float *__restrict__ Y,
    int zero_point, int scale_type, int batch)
{
    using L = ItemSlot<K>;
    // the waves' item rings
    __shared__ __attribute__((aligned(16))) char ring[WV][D][L::BYTES];
    // partial row sums: [buffer][wave][tile of the batch][token][row]
    __shared__ float red[2][WV][kBatch][16 * TQ];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;
    const int j = lane >> 4;
    const bool sym = zero_point == kZpSymmetric;
    const uint32_t gpr = (uint32_t)(cols / 128);        // groups per row

    uint32_t mask, one;
    asm volatile("s_mov_b32 %0, %1" : "=s"(mask) : "n"(kCodeMask));
    asm volatile("v_mov_b32 %0, %1" : "=v"(one) : "n"(kOnePair));
    uint32_t four;
    asm volatile("v_mov_b32 %0, %1" : "=v"(four) : "n"(kFourPair));

    // This lane as B column: row r of the tile, group gb of the set.
    const uint32_t r = n >> 2, gb = n & 3;
    const uint32_t row_bytes = (uint32_t)(cols / 4);
    const uint32_t plane_bytes = (uint32_t)plane_words * 4;
    const uint32_t sbytes = scale_type == kScaleF32 ? 4 : 2;
    const u32x4 dc = make_desc(codes, (uint32_t)K * plane_bytes);
    const u32x4 ds = make_desc(scales, (uint32_t)K * (uint32_t)plane_groups * sbytes);
    const u32x4 dz = make_desc(sym ? nullptr : zeros,
                               sym ? 0u : (uint32_t)K * (uint32_t)plane_groups * 4);
    const uint32_t set0 = (uint32_t)wave * SPW;

    // DMA lane offsets within an item. Codes: lane l fills bytes 16 l of a
    // 1 KiB load, i.e. stage 2 i + l / 32, row (l % 32) / 8, bytes
    // 16 (l % 8) .. + 15 of the set's 128-byte run of the row (a stage past
    // K - 1 reads past the descriptor, or other data that is never read).
    const uint32_t dma_code = (uint32_t)((lane & 31) >> 3) * row_bytes +
                              (uint32_t)(lane & 7) * 16 + (uint32_t)(lane >> 5) * plane_bytes;
    // Scales and zero-points: lane l -> stage l / 16, row (l % 16) / 4, group
    // l % 4 of the set; lanes of stages past K - 1 read nothing.
    const uint32_t pst = (uint32_t)lane >> 4;
    const uint32_t pgrp = ((uint32_t)(lane & 15) >> 2) * gpr + (uint32_t)(lane & 3) +
                          pst * (uint32_t)plane_groups;
    const uint32_t dma_scale = pst < (uint32_t)K ? pgrp * sbytes : kSkip;
    const uint32_t dma_zero = pst < (uint32_t)K ? pgrp * 4 : kSkip;

    const uint32_t lds_ring = lds_address(&ring[wave][0][0]);
    const char *my_ring = &ring[wave][0][0];

    const int64_t n_tiles = (rows + 3) / 4;
    const int64_t n_batches = (n_tiles + batch - 1) / batch;
    const int my_batches = blockIdx.x < n_batches
                               ? (int)((n_batches - 1 - blockIdx.x) / gridDim.x + 1) : 0;
    const int my_tiles = my_batches * batch;
    const int total = my_tiles * SPW;                  // items

    // DMA of the items in order, one call per item: item it is tile it / SPW
    // of this workgroup's sequence (batch b, tile t of it: tile
    // (blockIdx + b grid) batch + t), set it % SPW of this wave's, into slot
    // it % D. The position is kept as running counters, so an item costs a
    // few scalar additions rather than divisions. Items past the end, and
    // tiles past the last row, read through descriptors of size 0 (no
    // memory access, zeros in the slot): every item issues the same loads.
    // (tile indices fit 32 bits: rows < 2^26)
    int is_set = 0, is_tt = 0, is_slot = 0, issued = 0;
    int is_tile = (int)blockIdx.x * batch;
    const int batch_jump = ((int)gridDim.x - 1) * batch + 1;
    const int tiles = (int)n_tiles;
    auto issue_next = [&]() {
        const bool live = issued < total && is_tile < tiles;
        const uint32_t set = set0 + (uint32_t)is_set;
        const uint32_t row4 = live ? (uint32_t)is_tile * 4 : 0u;
        const uint32_t code_base = row4 * row_bytes + set * 128;
        const uint32_t grp_base = row4 * gpr + set * 4;
        const uint32_t lds = lds_ring + (uint32_t)is_slot * L::BYTES;
        u32x4 c_src = dc, s_src = ds, z_src = dz;
        if (!live) c_src[2] = s_src[2] = z_src[2] = 0u;
        // the reads of the item that used this slot have completed
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int i = 0; i < L::CODE_DMA; ++i)
            dma_x4(c_src, code_base + 2u * i * plane_bytes, lds + 1024u * i, dma_code);
        if (DEF || scale_type == kScaleF32)
            dma_dword(s_src, grp_base * 4, lds + L::SCALES, dma_scale);
        else
            dma_ushort(s_src, grp_base * 2, lds + L::SCALES, dma_scale);
        dma_dword(z_src, grp_base * 4, lds + L::ZEROS, dma_zero);
        ++issued;
        if (++is_slot == D) is_slot = 0;
        if (++is_set == SPW) {
            is_set = 0;
            if (++is_tt == batch) {
                is_tt = 0;
                is_tile += batch_jump;
            } else {
                ++is_tile;
            }
        }
    };

    // Activations first (the lane as A row of quad q: token 4 q + n / 4,
    // tokens past n_tokens repeating the last one, group ga of each of its
    // sets; operand set u = TQ set + q), then the ring.
    const uint32_t ga = n & 3;
    u32x4 run[SPW * TQ][4];
    {
        const u32x4 xs = make_desc(X, (uint32_t)n_tokens * (uint32_t)cols * 2);
#pragma unroll
        for (int s = 0; s < SPW; ++s)
#pragma unroll
            for (int q = 0; q < TQ; ++q) {
                const int t = 4 * q + (n >> 2);
                const uint32_t ta = (uint32_t)(t < n_tokens ? t : n_tokens - 1);
                const uint32_t gi = ((uint32_t)wave * SPW + s) * 4 + ga;
                const uint32_t off = ta * (uint32_t)cols * 2 + gi * 256 + 64 * (uint32_t)j;
#pragma unroll
                for (int i = 0; i < 4; ++i) run[TQ * s + q][i] = load_run(xs, off + 16 * i);
            }
    }
#pragma unroll
    for (int d = 0; d < D; ++d) issue_next();
    wait_runs<D * L::DMA>(run);

    u32x4 a[SPW * TQ][4];
    float sxd[SPW * TQ];
    {
        const u32x4 ones = {one, one, one, one};
#pragma unroll
        for (int s = 0; s < SPW * TQ; ++s) {
            act_operands(run[s], a[s]);
            // Sx: C rows 4 j + i = token j, group i of the set
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int b = 0; b < 4; ++b) acc = mfma(a[s][b], ones, acc);
            // the lane's diagonal entry (token j, group gb) is the one used
            sxd[s] = gb == 0 ? acc[0] : gb == 1 ? acc[1] : gb == 2 ? acc[2] : acc[3];
        }
    }

    int n_red = 0, slot_i = 0, tt = 0, bi = 0;
    for (int ti = 0; ti < my_tiles; ++ti) {
        f32x4 acc[TQ];
#pragma unroll
        for (int q = 0; q < TQ; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        float c[SPW];
#pragma unroll
        for (int set = 0; set < SPW; ++set) {
            // this item's loads have landed; the next D - 1 items' may not
            wait_vm<(D - 1) * L::DMA>();
            const char *slot = my_ring + slot_i * L::BYTES;
            c[set] = 0.0f;
#pragma unroll
            for (int st = 0; st < K; ++st) {
                const u32x2 w = *reinterpret_cast<const u32x2 *>(
                    slot + 1024 * (st >> 1) + 512 * (st & 1) + r * 128 + gb * 32 + j * 8);
                u32x4 b[2][2];
                code_operands_pair(w[0], w[1], mask, four, b);
                // the stage's B operands serve every quad of tokens
                f32x4 p[TQ];
#pragma unroll
                for (int q = 0; q < TQ; ++q) {
                    p[q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int v = 0; v < 4; ++v) p[q] = mfma(a[TQ * set + q][v], b[v >> 1][v & 1], p[q]);
                }
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
#pragma unroll
                for (int q = 0; q < TQ; ++q)
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[q][i] = __builtin_fmaf(s, p[q][i], acc[q][i]);
                c[set] = __builtin_fmaf(s, 4.0f + z, c[set]);
            }
            // the slot is free: refill it with the item D ahead
            issue_next();
            if (++slot_i == D) slot_i = 0;
        }
        // end of this wave's share of the tile: its diagonal entry (token j,
        // row r, group gb) less the sets' c Sx terms, summed over the 4
        // groups of the lanes n = 4 r .. 4 r + 3, kept for the batch reduction
#pragma unroll
        for (int q = 0; q < TQ; ++q) {
            float y = gb == 0 ? acc[q][0] : gb == 1 ? acc[q][1] : gb == 2 ? acc[q][2] : acc[q][3];
#pragma unroll
            for (int set = 0; set < SPW; ++set) y = __builtin_fmaf(-c[set], sxd[TQ * set + q], y);
            // (quad permutations [1 0 3 2] and [2 3 0 1]: lanes n ^ 1, n ^ 2)
            y += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, y), 0xB1, 0xF, 0xF, false));
            y += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, y), 0x4E, 0xF, 0xF, false));
            if (gb == 0) red[n_red & 1][wave][tt][16 * q + 4 * j + r] = y;
        }
        if (tt == batch - 1) {
            // end of the batch: sum the waves' partial sums in wave order
            // and store. The buffer written here is next written two batches
            // later, after a barrier that the summing threads reach only once
            // they have read it.
            __syncthreads();
            const int tid = threadIdx.x;
            if (tid < batch * 16 * TQ) {
                const int tb = tid / (16 * TQ), e = tid % (16 * TQ);   // e = 4 token + row
                float out = red[n_red & 1][0][tb][e];
#pragma unroll
                for (int w = 1; w < WV; ++w) out += red[n_red & 1][w][tb][e];
                const int64_t tile = ((int64_t)blockIdx.x + (int64_t)bi * gridDim.x) * batch + tb;
                const int64_t o = tile * 4 + (e & 3);
                const int tok = e >> 2;
                if (tok < n_tokens && o < rows) Y[(int64_t)tok * rows + o] = out;
            }
            ++n_red;
            tt = 0;
            ++bi;
        } else {
            ++tt;
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

template <int K, int WV, int SPW, int TQ, bool DEF>
hipError_t launch_k(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int zp, int sdt, const uint16_t *X, int n_tokens, float *Y,
                    int grid, int batch, hipStream_t stream)
{
    static_assert(wgs_per_cu(WV, SPW, TQ) * (ring_bytes(WV, SPW, TQ) + red_bytes(WV, TQ)) <=
                      160 * 1024, "the workgroups of a CU share its 160 KiB of LDS");
    constexpr int D = depth_for<K, WV, SPW, TQ>();
    return launch(decode_kernel<K, D, WV, SPW, TQ, DEF>, grid, 64 * WV, stream, codes, scales,
                  zeros, rows, cols, rows * cols / 16, rows * cols / 128, X, n_tokens, Y, zp, sdt,
                  batch);
}

template <int WV, int SPW, int TQ, bool DEF>
hipError_t launch_s(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int n_tokens,
                    float *Y, int grid, int batch, hipStream_t stream)
{
    switch (k) {
    case 1: return launch_k<1, WV, SPW, TQ, DEF>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 2: return launch_k<2, WV, SPW, TQ, DEF>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 3: return launch_k<3, WV, SPW, TQ, DEF>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 4: return launch_k<4, WV, SPW, TQ, DEF>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    default: return hipErrorInvalidValue;
    }
}

template <bool DEF>
hipError_t launch_d(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int n_tokens,
                    float *Y, int grid, int batch, hipStream_t stream)
{
    if (n_tokens > 8) {   // four quads of tokens, one set of 4 groups per wave
        if (cols != 4096 || n_tokens > 16) return hipErrorInvalidValue;
        return launch_s<8, 1, 4, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    }
    if (n_tokens > 4) {   // two quads of tokens, one set of 4 groups per wave
        if (cols != 4096 || n_tokens > 8) return hipErrorInvalidValue;
        return launch_s<8, 1, 2, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    }
    switch (cols / 4096) {   // sets of 4 groups per row / 8
    case 1: return launch_s<waves_for(8), sets_per_wave(8), 1, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 2: return launch_s<waves_for(16), sets_per_wave(16), 1, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 3: return launch_s<waves_for(24), sets_per_wave(24), 1, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 4: return launch_s<waves_for(32), sets_per_wave(32), 1, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool linear_decode_fits(int64_t rows, int64_t cols, int G, int k, int64_t n_tokens)
{
    if (G != 128 || n_tokens < 1 || n_tokens > 16 || cols % 4096 != 0 ||
        cols > kDecodeMaxCols)
        return false;
    // 5 to 8 tokens (two quads, rows of 4096 inputs): measured against the
    // batch form and the general kernel at 5 and 8 tokens, ahead up to 1024
    // rows at every stage count (5.9 against 9.8 us at 4 stages, 8 tokens),
    // and from 3 stages up to 2048 rows (8 tokens, 4 stages: 9.2 against 10.3
    // us) and from 4097 to 6144 rows, where the batch form's 16-row tiles
    // leave a round of workgroups half full (6144 x 4096, 5 tokens, 4 stages:
    // 14.0 against 15.2 us); behind or even elsewhere.
    // 9 to 16 tokens (four quads, rows of 4096 inputs, one workgroup per CU):
    // ahead of the general kernel, whose 16-row tiles leave most CUs idle on
    // so few rows, from 3 stages up to 1024 rows (1024 x 4096, 16 tokens, 4 /
    // 3 stages: 9.0 / 8.7 against 10.8 / 9.3 us; 256 rows, 4 stages: 8.2
    // against 9.5); behind at 1 and 2 stages (8.1 against 7.3 us at 2) and
    // even from 2048 rows.
    if (n_tokens > 8) return cols == 4096 && rows <= 1024 && k >= 3;
    if (n_tokens > 4) {
        if (cols != 4096) return false;
        return rows <= 1024 || (k >= 3 && (rows <= 2048 || (rows > 4096 && rows <= 6144)));
    }
    // Measured crossover against the general kernel (one token, packages
    // read from HBM): from 2 stages this form is as fast or faster on every
    // shape; with 1 stage an item is small and its per-item work costs more
    // than the general kernel's less efficient loads, except on small
    // matrices (latency-bound: this form fills the GPU with 4-row tiles) and
    // on tall ones with up to 2 sets of 4 groups per wave (two or three
    // workgroups per CU).
    if (k >= 2) return true;
    return rows <= 1024 || (rows >= 12288 && cols <= 8192);
}

hipError_t launch_linear_decode(const uint32_t *codes, const void *scales, const float *zeros,
                                int64_t rows, int64_t cols, int k, int zero_point, int scale_type,
                                const uint16_t *X, int64_t n_tokens, float *Y, int cus,
                                hipStream_t stream)
{
    if (n_tokens < 1 || n_tokens > 16 || (n_tokens > 4 && cols != 4096)) return hipErrorInvalidValue;
    const char *sc = static_cast<const char *>(scales);
    // Batches of up to 8 tiles, sized so that every resident workgroup
    // gets the same number of batches: R rounds of one batch per workgroup.
    const int sets = (int)(cols / 512), tq = n_tokens > 8 ? 4 : n_tokens > 4 ? 2 : 1;
    const int64_t slots = (int64_t)cus * (tq > 1 ? wgs_per_cu(8, 1, tq)
                                                 : wgs_per_cu(waves_for(sets), sets_per_wave(sets), 1));
    const int64_t tiles = (rows + 3) / 4;
    const int64_t rounds = (tiles + slots * kBatch - 1) / (slots * kBatch);
    const int64_t batch = (tiles + slots * rounds - 1) / (slots * rounds);
    const int64_t batches = (tiles + batch - 1) / batch;
    const int grid = (int)(batches < slots ? batches : slots);
    const int nt = (int)n_tokens;
    const bool def = scale_type == kScaleF32 && zero_point != kZpSymmetric;
    return def ? launch_d<true>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, nt, Y,
                                grid, (int)batch, stream)
               : launch_d<false>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, nt, Y,
                                 grid, (int)batch, stream);
}

}  // namespace rrq_detail

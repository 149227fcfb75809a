// Decode form of the stage-sum linear layer (Eq. 20) for up to 4 tokens and
// groups of 128: Y[m][o] = sum over stages t < K and groups g of
// s_t,o,g (sum_i x_m,i Q_t,o,i - z_t,o,g sum_i x_m,i), the product
// rrq_linear.hip computes for any shape, organised here for streaming the
// package from HBM at full width when the activations are few.
//
// Matrix-core mapping (v_mfma_f32_16x16x32_bf16, lane l: row / column
// n = l % 16, k-slice j = l / 16):
//   * B columns are 4 output rows x 4 consecutive groups (n = 4 r + g'); lane
//     j owns inputs 32 j .. 32 j + 31 of its group, i.e. 8 contiguous bytes
//     of codes per stage. One load instruction of a wave reads 4 rows x 128
//     contiguous bytes with consecutive lanes on consecutive 8-byte pieces,
//     and a cross-lane permutation (ds_bpermute) hands each piece to its
//     MFMA lane. Codes become the bfloat16 1 + Q/4 (one shift and one AND-OR
//     per pair of codes, codes q and q + 8 of a word per register);
//   * A rows are 4 tokens x the same 4 groups (m = 4 t + g), so C[m][n] is a
//     group's dot product only on the diagonal g = g': lane l keeps all four
//     of its C rows (tokens j, groups 0..3) and uses row g' = n % 4 at the end;
//   * a wave works on a fixed range of columns (its sets of 4 groups), so its
//     A operands (the activations, in pairs (x[v], x[v + 8]) of every 16
//     inputs) and the group sums Sx (from the same MFMA with a ones operand)
//     are loaded and formed once and stay in registers.
// Each lane accumulates sum over stages of (4 s) P - (sum over stages of
// s (4 + z)) Sx for its token, row and group (P = sum x (1 + Q/4)); the four
// groups of a set are summed across lanes and the waves' column ranges
// through LDS, in a fixed order. Every matrix-core product is exact; fp32
// rounding is in the accumulations only.
//
// Work: the 8 waves of a workgroup split every 4-row tile's columns, so at
// any moment a workgroup reads whole rows and neighbouring workgroups read
// neighbouring rows; a workgroup takes batches of consecutive tiles in turn.
// Each wave walks its (tile, set) items as one sequence and keeps the loads
// of the next D - 1 items in flight in registers (codes, scales and
// zero-points of the K stages).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rrq_launch.h"

namespace rrq_detail {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
using rsrc_t = __amdgpu_buffer_rsrc_t;

constexpr int kWaves = 8;                      // waves per workgroup
constexpr uint32_t kOnePair = 0x3F803F80u;     // two bfloat16 1.0
constexpr uint32_t kCodeMask = 0x00600060u;    // top two mantissa bits of both halves
constexpr int kZpSymmetric = 2;
constexpr int kScaleF32 = 0, kScaleF16 = 1;

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ f32x4 mfma(const u32x4 &a, const u32x4 &b, const f32x4 &c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// B operands of the two blocks of one code word: register q (of 8) holds
// codes q and q + 8 as 1 + code / 4; block 0 takes registers 0..3, block 1
// registers 4..7.
__device__ __forceinline__ void word_operands(uint32_t w, uint32_t mask, uint32_t one,
                                              u32x4 &b0, u32x4 &b1)
{
    b0[0] = ((w << 5) & mask) | one;
    b0[1] = ((w << 3) & mask) | one;
    b0[2] = ((w << 1) & mask) | one;
    b0[3] = ((w >> 1) & mask) | one;
    b1[0] = ((w >> 3) & mask) | one;
    b1[1] = ((w >> 5) & mask) | one;
    b1[2] = ((w >> 7) & mask) | one;
    b1[3] = ((w >> 9) & mask) | one;
}

// The loads of one item (a 4-row tile and a set of 4 groups) for all K
// stages: this lane's 8 code bytes, scale and zero-point per stage.
template <int K>
struct Item {
    u32x2 c[K];
    uint32_t s[K], z[K];
};

// A operands of one set of 4 groups for the lane (token t, group g, k-slice
// j): its 32 inputs 32 j .. 32 j + 31 of group g, block b = 16-input run
// 2 j + b / 2, half b % 2, register v = (x[v'], x[v' + 8]) of the run's half.
__device__ __forceinline__ void act_operands(const rsrc_t &xs, uint32_t off, u32x4 (&a)[4])
{
    u32x4 run[4];   // x[32 j .. +7], [+8 .. +15], [+16 .. +23], [+24 .. +31]
#pragma unroll
    for (int i = 0; i < 4; ++i) run[i] = __builtin_amdgcn_raw_buffer_load_b128(xs, off + 16 * i, 0, 0);
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

// Workgroup: 8 waves share each 4-row tile, wave w taking sets
// w SPW .. w SPW + SPW - 1 of its 8 SPW sets of 4 groups (so the waves of a
// workgroup read whole rows together); a batch of up to 8 consecutive tiles
// is reduced across the waves through LDS. Batches go to workgroups in turn.
constexpr int kBatch = 8;

template <int K, int D, int SPW, bool DEF>
__global__ __launch_bounds__(64 * kWaves) void decode_kernel(
    const uint32_t *__restrict__ codes, const char *__restrict__ scales,
    const float *__restrict__ zeros, int64_t rows, int64_t cols, int64_t plane_words,
    int64_t plane_groups, const uint16_t *__restrict__ X, int n_tokens, float *__restrict__ Y,
    int zero_point, int scale_type, int batch)
{
    // partial row sums: [buffer][wave][tile of the batch][token][row]
    __shared__ float red[2][kWaves][kBatch][16];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 15;
    const int j = lane >> 4;
    const bool sym = zero_point == kZpSymmetric;
    const uint32_t gpr = (uint32_t)(cols / 128);        // groups per row

    uint32_t mask, one;
    asm volatile("s_mov_b32 %0, %1" : "=s"(mask) : "n"(kCodeMask));
    asm volatile("v_mov_b32 %0, %1" : "=v"(one) : "n"(kOnePair));

    // This lane as B column: row r of the tile, group gb of the set.
    const uint32_t r = n >> 2, gb = n & 3;
    const uint32_t row_bytes = (uint32_t)(cols / 4);
    const uint32_t plane_bytes = (uint32_t)plane_words * 4;
    const uint32_t sbytes = scale_type == kScaleF32 ? 4 : 2;
    const rsrc_t rc = make_rsrc(codes, (uint32_t)K * plane_bytes);
    const rsrc_t rs = make_rsrc(scales, (uint32_t)K * (uint32_t)plane_groups * sbytes);
    const rsrc_t rz = make_rsrc(sym ? nullptr : zeros, sym ? 0u : (uint32_t)K * (uint32_t)plane_groups * 4);
    const rsrc_t rnone = make_rsrc(codes, 0u);
    const uint32_t set0 = (uint32_t)wave * SPW;
    // Codes are loaded coalesced: lane l takes bytes 8 (l % 16) of row l / 16
    // of the set's 4 rows x 128 bytes, and a cross-lane permutation moves
    // each 8-byte piece to the lane that uses it (row r, group gb, slice j),
    // i.e. from lane 16 r + 4 gb + j.
    const uint32_t lane_code = (uint32_t)j * row_bytes + set0 * 128 + 8 * (uint32_t)n;
    const int perm_src = 4 * (int)(16 * r + 4 * gb + (uint32_t)j);   // ds_bpermute byte address
    const uint32_t lane_grp = r * gpr + set0 * 4 + gb;

    const int64_t n_tiles = (rows + 3) / 4;
    const int64_t n_batches = (n_tiles + batch - 1) / batch;
    const int my_batches = blockIdx.x < n_batches
                               ? (int)((n_batches - 1 - blockIdx.x) / gridDim.x + 1) : 0;
    const int per_batch = batch * SPW;                 // items per batch
    const int total = my_batches * per_batch;

    // Loads of item it: batch it / per_batch, tile (it % per_batch) / SPW of
    // it, set it % SPW of this wave's. Items past the end, and tiles past the
    // last row, load from an empty resource (no memory access).
    auto issue = [&](int it, Item<K> &dst) {
        const int bi = it / per_batch, rest = it % per_batch;
        const int64_t tile = ((int64_t)blockIdx.x + (int64_t)bi * gridDim.x) * batch + rest / SPW;
        const uint32_t set = (uint32_t)(rest % SPW);
        const bool live = it < total && tile < n_tiles;
        const uint32_t code_off = live ? (uint32_t)(tile * 4) * row_bytes + set * 128 + lane_code : 0u;
        const uint32_t grp = live ? (uint32_t)(tile * 4) * gpr + set * 4 + lane_grp : 0u;
        const rsrc_t c_src = live ? rc : rnone, s_src = live ? rs : rnone, z_src = live ? rz : rnone;
#pragma unroll
        for (int st = 0; st < K; ++st) {
            dst.c[st] = __builtin_amdgcn_raw_buffer_load_b64(c_src, code_off, st * plane_bytes, 0);
            if (DEF || scale_type == kScaleF32)
                dst.s[st] = __builtin_amdgcn_raw_buffer_load_b32(
                    s_src, grp * 4, st * (uint32_t)plane_groups * 4, 0);
            else
                dst.s[st] = __builtin_amdgcn_raw_buffer_load_b16(
                    s_src, grp * 2, st * (uint32_t)plane_groups * 2, 0);
            dst.z[st] = __builtin_amdgcn_raw_buffer_load_b32(
                z_src, grp * 4, st * (uint32_t)plane_groups * 4, 0);
        }
    };

    Item<K> ring[D];
#pragma unroll
    for (int d = 0; d < D; ++d) issue(d, ring[d]);

    // A operands and group sums of this wave's sets (fixed for the whole
    // kernel, loaded once the first items' loads are in flight): lane as A
    // row = token ta (tokens past n_tokens repeat the last one), group ga of
    // the set.
    const uint32_t ta = (uint32_t)((n >> 2) < n_tokens ? (n >> 2) : n_tokens - 1);
    const uint32_t ga = n & 3;
    u32x4 a[SPW][4];
    f32x4 sx[SPW];
    {
        const rsrc_t xs = make_rsrc(X, (uint32_t)n_tokens * (uint32_t)cols * 2);
        const u32x4 ones = {one, one, one, one};
#pragma unroll
        for (int s = 0; s < SPW; ++s) {
            const uint32_t gi = ((uint32_t)wave * SPW + s) * 4 + ga;
            act_operands(xs, ta * (uint32_t)cols * 2 + gi * 256 + 64 * (uint32_t)j, a[s]);
            // Sx: C rows 4 j + i = token j, group i of the set
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int b = 0; b < 4; ++b) acc = mfma(a[s][b], ones, acc);
            sx[s] = acc;
        }
    }


    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    int n_red = 0;
    for (int base = 0; base < total; base += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            const int it = base + d;
            if (it >= total) break;
            const int rest = it % per_batch;
            const int set = rest % SPW;
            const Item<K> &cur = ring[d];
            float c = 0.0f;
#pragma unroll
            for (int st = 0; st < K; ++st) {
                const uint32_t w0 = (uint32_t)__builtin_amdgcn_ds_bpermute(perm_src, (int)cur.c[st][0]);
                const uint32_t w1 = (uint32_t)__builtin_amdgcn_ds_bpermute(perm_src, (int)cur.c[st][1]);
                u32x4 b[4];
                word_operands(w0, mask, one, b[0], b[1]);
                word_operands(w1, mask, one, b[2], b[3]);
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    // the set index is wave-uniform and SPW is small: select
                    // the A operand without indexing registers dynamically
                    u32x4 aq = a[0][q];
#pragma unroll
                    for (int s2 = 1; s2 < SPW; ++s2)
                        if (set == s2) aq = a[s2][q];
                    p = mfma(aq, b[q], p);
                }
                float s, z;
                if constexpr (DEF) {
                    s = __uint_as_float(cur.s[st]);
                    z = __uint_as_float(cur.z[st]);
                } else {
                    s = scale_type == kScaleF32 ? __uint_as_float(cur.s[st])
                        : scale_type == kScaleF16
                            ? (float)__builtin_bit_cast(_Float16, (uint16_t)(cur.s[st] & 0xFFFFu))
                            : __uint_as_float(cur.s[st] << 16);
                    z = sym ? 2.0f : __uint_as_float(cur.z[st]);
                }
                const float s4 = 4.0f * s;
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(s4, p[i], acc[i]);
                c = __builtin_fmaf(s, 4.0f + z, c);
            }
            f32x4 sxs = sx[0];
#pragma unroll
            for (int s2 = 1; s2 < SPW; ++s2)
                if (set == s2) sxs = sx[s2];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(-c, sxs[i], acc[i]);
            // reuse the slot for the item D ahead
            issue(it + D, ring[d]);

            if (set == SPW - 1) {
                // end of this wave's share of a tile: its diagonal entry
                // (token j, row r, group gb) summed over the 4 groups of the
                // lanes n = 4 r .. 4 r + 3, kept for the batch reduction
                float y = gb == 0 ? acc[0] : gb == 1 ? acc[1] : gb == 2 ? acc[2] : acc[3];
                y += __shfl_xor(y, 1, 64);
                y += __shfl_xor(y, 2, 64);
                const int ti = rest / SPW;
                if (gb == 0) red[n_red & 1][wave][ti][4 * j + r] = y;
                acc = (f32x4){0.f, 0.f, 0.f, 0.f};
                if (rest == per_batch - 1) {
                    // end of the batch: sum the waves' partial sums in wave
                    // order and store. The buffer written here is next
                    // written two batches later, after a barrier that the
                    // summing threads reach only once they have read it.
                    __syncthreads();
                    const int tid = threadIdx.x;
                    if (tid < batch * 16) {
                        const int tt = tid / 16, e = tid % 16;   // e = 4 token + row
                        float out = red[n_red & 1][0][tt][e];
#pragma unroll
                        for (int w = 1; w < kWaves; ++w) out += red[n_red & 1][w][tt][e];
                        const int bi = it / per_batch;
                        const int64_t tile = ((int64_t)blockIdx.x + (int64_t)bi * gridDim.x) * batch + tt;
                        const int64_t o = tile * 4 + (e & 3);
                        const int tok = e >> 2;
                        if (tok < n_tokens && o < rows) Y[(int64_t)tok * rows + o] = out;
                    }
                    ++n_red;
                }
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

// Items in flight per wave: as many as keep all their loads (3 K per item)
// within the 6-bit vmcnt counter, at most 8.
constexpr int depth_for(int K) { return 63 / (3 * K) < 8 ? 63 / (3 * K) : 8; }

template <int K, int SPW, bool DEF>
hipError_t launch_k(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int zp, int sdt, const uint16_t *X, int n_tokens, float *Y,
                    int grid, int batch, hipStream_t stream)
{
    constexpr int D = depth_for(K);
    return launch(decode_kernel<K, D, SPW, DEF>, grid, 64 * kWaves, stream, codes, scales, zeros,
                  rows, cols, rows * cols / 16, rows * cols / 128, X, n_tokens, Y, zp, sdt, batch);
}

template <int SPW, bool DEF>
hipError_t launch_s(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int n_tokens,
                    float *Y, int grid, int batch, hipStream_t stream)
{
    switch (k) {
    case 1: return launch_k<1, SPW, DEF>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 2: return launch_k<2, SPW, DEF>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 3: return launch_k<3, SPW, DEF>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 4: return launch_k<4, SPW, DEF>(codes, scales, zeros, rows, cols, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    default: return hipErrorInvalidValue;
    }
}

template <bool DEF>
hipError_t launch_d(const uint32_t *codes, const char *scales, const float *zeros, int64_t rows,
                    int64_t cols, int k, int zp, int sdt, const uint16_t *X, int n_tokens,
                    float *Y, int grid, int batch, hipStream_t stream)
{
    switch (cols / 4096) {   // sets of 4 groups per wave
    case 1: return launch_s<1, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 2: return launch_s<2, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 3: return launch_s<3, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    case 4: return launch_s<4, DEF>(codes, scales, zeros, rows, cols, k, zp, sdt, X, n_tokens, Y, grid, batch, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool linear_decode_fits(int64_t rows, int64_t cols, int G, int k, int64_t n_tokens)
{
    // Measured crossover: with one stage the items are too small to amortise
    // their loads of scales and zero-points, and below about 6144 rows a
    // wave gets too few items to amortise the kernel's start (activations,
    // group sums, first loads); the general kernel is faster there.
    return G == 128 && k >= 2 && rows >= 6144 && n_tokens >= 1 && n_tokens <= 4 &&
           cols % 4096 == 0 && cols / 4096 <= kDecodeMaxSetsPerWave;
}

hipError_t launch_linear_decode(const uint32_t *codes, const void *scales, const float *zeros,
                                int64_t rows, int64_t cols, int k, int zero_point, int scale_type,
                                const uint16_t *X, int64_t n_tokens, float *Y, int cus,
                                hipStream_t stream)
{
    const char *sc = static_cast<const char *>(scales);
    // Batches of up to 8 tiles, sized so that every workgroup (one per CU)
    // gets the same number of batches: R rounds of cus batches.
    const int64_t tiles = (rows + 3) / 4;
    const int64_t rounds = (tiles + (int64_t)cus * kBatch - 1) / ((int64_t)cus * kBatch);
    const int64_t batch = (tiles + (int64_t)cus * rounds - 1) / ((int64_t)cus * rounds);
    const int64_t batches = (tiles + batch - 1) / batch;
    const int grid = (int)(batches < cus ? batches : cus);
    const int nt = (int)n_tokens;
    const bool def = scale_type == kScaleF32 && zero_point != kZpSymmetric;
    return def ? launch_d<true>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, nt, Y,
                                grid, (int)batch, stream)
               : launch_d<false>(codes, sc, zeros, rows, cols, k, zero_point, scale_type, X, nt, Y,
                                 grid, (int)batch, stream);
}

}  // namespace rrq_detail

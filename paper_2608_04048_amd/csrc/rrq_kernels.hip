// HIP kernels for RRQ package construction and prefix reconstruction on
// gfx950 (MI355X).
//
// Construction follows Algorithm 1 with the per-group affine RTN stage of
// Eq. 1-3 applied S times, each stage to the residual the earlier stages left
// (Eq. 4-7); either the base stage is quantized too, or (Algorithm 1's first
// branch) a given base stage is dequantized and only the residual stages are
// built. Reconstruction is the prefix sum of Eq. 8 /
// Eq. 18-19. The arithmetic is the fixed binary32 reading stated in rrq.h;
// the kernels reproduce it bit for bit (build with -ffp-contract=off, no fast
// math, denormals kept).
//
// Construct kernel:
//   * one wave (64 lanes) per workgroup, two waves per SIMD; the wave takes
//     tiles of 64 consecutive groups in a grid-stride loop, and each lane owns
//     one whole group, held in registers (G binary32 residuals) through every
//     stage, so the bfloat16 input is read from HBM once and residuals never
//     leave the register file. The next tile is prefetched into registers
//     while the current one is quantized;
//   * the tile is loaded with fully coalesced 16-byte-per-lane buffer loads
//     and transposed through LDS half a group at a time (rows padded by 16
//     bytes, so row writes and per-lane column reads are free of bank
//     conflicts); every lane then holds the G contiguous elements of its group;
//   * per group and stage (once per lane): range lo = min(0, min r),
//     hi = max(0, max r) (two-chain min3/max3, fused into the previous stage's
//     residual update), s = fl((hi - lo) / 3), inv = fl(1 / s),
//     z = RNE(|lo| inv) (the exact product), and a per-lane LDS table of
//     dequantized pairs;
//   * per element and stage: u = fma(r, inv, 1.5 * 2^23 + z) is the single
//     nearest-even rounding of the exact r inv + z (u lies in [2^23, 2^24),
//     where binary32 spacing is 1); one clamped FMA turns u into a tiny
//     binary32 whose bit pattern is 3 - min(Q, 3); exact FMAs on such values
//     pack the codes and form the LDS address of each element pair's
//     dequantized values fl((Q - z) s); r = fl(r - rhat). Lanes past the input
//     compute on zeros and their stores fall outside the buffer resources.
//   * Clamp: no element can round below code 0 (z = RNE(|lo| inv) of the same
//     exact product that bounds every r inv from below, so r inv + z >= -1/2,
//     and -1/2 rounds to -0, code 0); the upper clamp
//     is needed in most tiles (a residual range symmetric about zero gives
//     z = RNE(1.5) = 2 and puts its top element on code 4) and costs nothing
//     here: it is the clamp modifier of the FMA above.
// gfx950 issues fused multiply-add, add, multiply and bitwise logic at twice
// the rate of shifts, min/max, three-operand integer and conversion
// instructions (two waves dual-issue the former); the element loop is written
// with the former wherever the arithmetic allows.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rrq_launch.h"

namespace rrq_detail {
namespace {

constexpr float kMagic = 12582912.0f;          // 1.5 * 2^23

// Stage formats (values of the C ABI's zero-point and scale-type enums).
constexpr int kZpInteger = 0;    // z = RNE(|lo| inv), exact product, stored
constexpr int kZpReal = 1;       // z = fl(|lo| inv), stored
constexpr int kZpSymmetric = 2;  // range [-amax, amax], z = 2, not stored
constexpr int kScaleF32 = 0, kScaleF16 = 1, kScaleBF16 = 2;

// Codes as bit patterns of tiny binary32 values. For u = 1.5 * 2^23 + Q
// (Q = RNE(t + z) in 0..4), fma(u, -2^-149, (1.5 * 2^23 + 3) 2^-149) is
// exactly (3 - Q) 2^-149, and the instruction's clamp-to-[0, 1] modifier turns
// Q = 4 into 0: the result's bit pattern is the integer k = 3 - min(Q, 3).
// Every value below stays under 2^24 * 2^-149, where binary32 bit patterns
// equal the integer multiple of 2^-149 and fused multiply-adds of such values
// by powers of two are exact; so packing codes and forming LDS addresses are
// single exact FMAs (full-rate on gfx950, unlike shifts, min/max or
// three-operand integer instructions, which issue at half that rate).
constexpr float kNegTiny = -0x1p-149f;              // -2^-149
constexpr float kTopTiny = 0x1.800006p-126f;        // (1.5 * 2^23 + 3) * 2^-149

// Raw buffer resources (gfx9 family descriptor). Accesses beyond num_records
// bytes read as zero and stores there are dropped, which handles the ragged
// last tile without branches. A resource is rebuilt per tile, so 32-bit
// num_records and offsets suffice for inputs of any size.
using rsrc_t = __amdgpu_buffer_rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

// Per-lane dequantization tables in LDS, one per wave. Entry idx = k[e] +
// 4 k[e + 1] (k = 3 - code) of lane l holds the pair of dequantized values
// {fl((Q[e] - z) s), fl((Q[e + 1] - z) s)} of the lane's group for the current
// stage, the first at byte offset idx * 512 + l * 4 and the second 256 bytes
// further: one two-address LDS read fetches a pair, a wave's 64 lookups of one
// pair of elements touch every bank once per value, and the lane's whole
// table is written from a single address register.
struct DequantTable {
    float *base;      // this wave's 16 x 2 x 64 floats
    float lane_off;   // binary32 whose bit pattern is l * 4
};

// The pair of dequantized values at byte offset off of the table.
__device__ __forceinline__ f32x2 table_pair(const char *tbase, uint32_t off)
{
    const float *p = reinterpret_cast<const float *>(tbase + off);
    return (f32x2){p[0], p[64]};
}

// Code of one element as the tiny binary32 (3 - min(Q, 3)) 2^-149, where
// Q = RNE(r inv + z) of the exact value: u = fma(r, inv, 1.5 * 2^23 + z) rounds
// the exact r inv + z once to the nearest integer, ties to even (u lies in
// [2^23, 2^24), where binary32 spacing is 1).
__device__ __forceinline__ float tiny_code(float r, float inv, float m)
{
    const float u = __builtin_fmaf(r, inv, m);
    return __builtin_amdgcn_fmed3f(__builtin_fmaf(u, kNegTiny, kTopTiny), 0.0f, 1.0f);
}

// With a real-valued zero-point, Q = RNE(fl(t + z)): the sum is rounded to
// binary32 first, then to the nearest integer by the magic addend.
__device__ __forceinline__ float tiny_code_real(float r, float inv, float z)
{
    const float v = r * inv + z;   // fl(fl(r inv) + z)
    const float u = v + kMagic;
    return __builtin_amdgcn_fmed3f(__builtin_fmaf(u, kNegTiny, kTopTiny), 0.0f, 1.0f);
}

// Issue priority of the wave. Two waves share a SIMD; each tile and stage
// has serial stretches (the LDS transpose, the last residual updates and the
// range reduction, scale and reciprocal, the table writes and the first
// lookups) between long runs of independent element work. The serial stretches run at a raised priority,
// so that the SIMD's arbiter favours them and the other wave's element work
// fills their latency (measured 4% faster, identical outputs).
__device__ __forceinline__ void serial_priority(bool on)
{
    if (on) __builtin_amdgcn_s_setprio(2);
    else __builtin_amdgcn_s_setprio(0);
}

// Element loop of one stage for one lane's group: the stage's codes into
// words[]; with UPDATE also the residual r <- r - (Q - z) s and the range of
// the new residual (lo, hi, zero included) for the next stage. ZP selects the
// zero-point kind (integer and symmetric stages round t + z in one step).
template <int G, bool UPDATE, int ZP>
__device__ __forceinline__ void stage_elements(float (&r)[G], float inv, float m, float z,
                                               const DequantTable &tab,
                                               uint32_t (&words)[G / 16], float &lo, float &hi)
{
    float l0 = 0.f, l1 = 0.f, h0 = 0.f, h1 = 0.f;
    const char *tbase = reinterpret_cast<const char *>(tab.base);
    f32x2 rh[2][8];   // table lookups of two consecutive words in flight

    // Codes of word w and (UPDATE) the lookups of its dequantized values.
    auto quantize_word = [&](int w, f32x2 (&rhw)[8]) {
        float x[8];   // pair p: k[2p] + 4 k[2p + 1], as a tiny binary32
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            const int j = w * 16 + 2 * p;
            if constexpr (ZP == kZpReal)
                x[p] = __builtin_fmaf(tiny_code_real(r[j + 1], inv, z), 4.0f,
                                      tiny_code_real(r[j], inv, z));
            else
                x[p] = __builtin_fmaf(tiny_code(r[j + 1], inv, m), 4.0f, tiny_code(r[j], inv, m));
            if (UPDATE) {
                const uint32_t off = __float_as_uint(__builtin_fmaf(x[p], 512.0f, tab.lane_off));
                rhw[p] = table_pair(tbase, off);
            }
        }
        float q[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) q[i] = __builtin_fmaf(x[2 * i + 1], 16.0f, x[2 * i]);
        const uint32_t lo16 = __float_as_uint(__builtin_fmaf(q[1], 256.0f, q[0]));
        const uint32_t hi16 = __float_as_uint(__builtin_fmaf(q[3], 256.0f, q[2]));
        // fields hold 3 - Q = Q ^ 3: complement to get the codes
        words[w] = ~(lo16 | (hi16 << 16));
    };
    // Residual update of word w and its contribution to the next range.
    auto update_word = [&](int w, const f32x2 (&rhw)[8]) {
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            r[w * 16 + 2 * p] = r[w * 16 + 2 * p] - rhw[p].x;
            r[w * 16 + 2 * p + 1] = r[w * 16 + 2 * p + 1] - rhw[p].y;
        }
#pragma unroll
        for (int e = 0; e < 16; e += 4) {
            const int j = w * 16 + e;
            l0 = fminf(fminf(l0, r[j]), r[j + 1]);
            h0 = fmaxf(fmaxf(h0, r[j]), r[j + 1]);
            l1 = fminf(fminf(l1, r[j + 2]), r[j + 3]);
            h1 = fmaxf(fmaxf(h1, r[j + 2]), r[j + 3]);
        }
    };

    // Software pipeline: word w + 1's lookups are issued before word w's
    // results are consumed, so LDS latency overlaps VALU work. The
    // scheduling barriers keep the compiler from hoisting further ahead,
    // which would hold extra G-wide temporaries and spill the residuals.
    quantize_word(0, rh[0]);
    serial_priority(false);   // raised by the caller for the stage's set-up
#pragma unroll
    for (int w = 0; w < G / 16; ++w) {
        if (w + 1 < G / 16) quantize_word(w + 1, rh[(w + 1) & 1]);
        // the last word's residuals give the range the next stage waits for
        if (w + 1 == G / 16) serial_priority(true);
        if (UPDATE) update_word(w, rh[w & 1]);
        __builtin_amdgcn_sched_barrier(0);
    }
    lo = fminf(l0, l1);
    hi = fmaxf(h0, h1);
}

// Base stage of a loaded checkpoint (Algorithm 1, first branch), for half
// HALF of the lane's group (G / 2 elements): each element becomes
// r - fl(fl(Q_0 - z_0) s_0), looked up in the lane's pair table (filled for
// s_0, z_0), and the result's range is folded into (l0, l1, h0, h1). The
// table index of an element pair is k0 + 4 k1 with k = 3 - Q, which is the
// pair's nibble of the complemented code word.
template <int G, int HALF>
__device__ __forceinline__ void subtract_base_half(float (&r)[G], const uint32_t (&bw)[G / 16],
                                                   const DequantTable &tab, float &l0, float &l1,
                                                   float &h0, float &h1)
{
    const char *tbase = reinterpret_cast<const char *>(tab.base);
    const uint32_t lane_off = __float_as_uint(tab.lane_off);   // lane * 4 < 256
    f32x2 rh[2][4];   // lookups of two consecutive 8-element pieces in flight
    constexpr int H0 = HALF * (G / 16), H1 = H0 + G / 16;    // 8-element pieces

    auto lookup = [&](int h, f32x2 (&rhh)[4]) {
        const uint32_t kw = ~bw[h >> 1];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int p = (h & 1) * 4 + i;
            // nibble p of kw, times 512
            const uint32_t nib = (4 * p <= 9) ? (kw << (9 - 4 * p)) & 0x1E00u
                                              : (kw >> (4 * p - 9)) & 0x1E00u;
            rhh[i] = table_pair(tbase, nib | lane_off);
        }
    };
    auto apply = [&](int h, const f32x2 (&rhh)[4]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            r[h * 8 + 2 * i] = r[h * 8 + 2 * i] - rhh[i].x;
            r[h * 8 + 2 * i + 1] = r[h * 8 + 2 * i + 1] - rhh[i].y;
        }
#pragma unroll
        for (int e = 0; e < 8; e += 4) {
            const int j = h * 8 + e;
            l0 = fminf(fminf(l0, r[j]), r[j + 1]);
            h0 = fmaxf(fmaxf(h0, r[j]), r[j + 1]);
            l1 = fminf(fminf(l1, r[j + 2]), r[j + 3]);
            h1 = fmaxf(fmaxf(h1, r[j + 2]), r[j + 3]);
        }
    };

    lookup(H0, rh[0]);
#pragma unroll
    for (int h = H0; h < H1; ++h) {
        if (h + 1 < H1) lookup(h + 1, rh[(h + 1) & 1]);
        apply(h, rh[h & 1]);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Sum of |x| over the lane's group in the order that defines the peak-to-mean
// ratio: four partial sums over j = 0, 1, 2, 3 (mod 4), each in increasing j,
// combined as (p0 + p1) + (p2 + p3).
template <int G>
__device__ __forceinline__ float group_abs_sum(const float (&r)[G])
{
    float p0 = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f;
#pragma unroll
    for (int j = 0; j < G; j += 4) {
        p0 = p0 + fabsf(r[j]);
        p1 = p1 + fabsf(r[j + 1]);
        p2 = p2 + fabsf(r[j + 2]);
        p3 = p3 + fabsf(r[j + 3]);
    }
    return (p0 + p1) + (p2 + p3);
}

// Peak-to-mean ratio K / fl(S / G) of a group (0 for a group of zeros) from
// its zero-included range (K = max(|lo|, hi)) and its |x| sum S; stored at
// the lane's group.
template <int G>
__device__ __forceinline__ void store_pmr(float *pmr, int64_t g0, uint32_t groups_here, int lane,
                                          float lo, float hi, float S)
{
    const float K = fmaxf(fabsf(lo), hi);
    const float mae = S * (1.0f / (float)G);             // exact: G is a power of two
    const float v = S > 0.0f ? K / mae : 0.0f;
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), make_rsrc(pmr + g0, groups_here * 4),
                                          lane * 4, 0, 0);
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

// Range of a group split over L consecutive lanes (L = 1, 2 or 4): each lane
// holds a contiguous share of the group and its own partial lo, hi; DPP quad
// permutes exchange them (min and max are exact, so the order of combination
// does not matter).
template <int CTRL>
__device__ __forceinline__ float dpp_quad(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

template <int L>
__device__ __forceinline__ void combine_range(float &lo, float &hi)
{
    static_assert(L == 1 || L == 2 || L == 4, "lanes per group");
    if constexpr (L >= 2) {   // partner lane ^ 1: quad_perm [1, 0, 3, 2]
        lo = fminf(lo, dpp_quad<0xB1>(lo));
        hi = fmaxf(hi, dpp_quad<0xB1>(hi));
    }
    if constexpr (L >= 4) {   // partner lane ^ 2: quad_perm [2, 3, 0, 1]
        lo = fminf(lo, dpp_quad<0x4E>(lo));
        hi = fmaxf(hi, dpp_quad<0x4E>(hi));
    }
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
// contiguously. Chunks past the end of the input read as zero, and a tile
// past the end reads all zeros (a zero-sized resource): the prefetch of a
// next tile needs no branch, which keeps the compiler from moving the
// current tile's arithmetic across one.
template <int CH>
__device__ __forceinline__ void load_tile(const uint4 *__restrict__ W, int64_t n_groups,
                                          int64_t tile, int lane, uint4 (&v)[CH])
{
    const int64_t g0 = tile * 64;
    const int64_t left = n_groups - g0;
    const uint32_t bytes = left <= 0 ? 0u : (uint32_t)(left < 64 ? left : 64) * CH * 16;
    const rsrc_t src = make_rsrc(W + (left <= 0 ? 0 : g0 * CH), bytes);
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(src, (i * 64 + lane) * 16, 0, 0);
        v[i] = make_uint4(x.x, x.y, x.z, x.w);
    }
}

// Reads half h of this lane's group (G / 2 elements) from the transposed LDS
// buffer and widens bfloat16 to binary32.
template <int G>
__device__ __forceinline__ void gather_half(const uint4 *rd_base, int h, float (&r)[G])
{
#pragma unroll
    for (int c = 0; c < G / 16; ++c) {
        const uint4 w = rd_base[c];
        const uint32_t p[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            r[h * (G / 2) + 8 * c + 2 * q] = __uint_as_float(p[q] << 16);
            r[h * (G / 2) + 8 * c + 2 * q + 1] = __uint_as_float(p[q] & 0xFFFF0000u);
        }
    }
}

// Output resources of one tile: codes, scales and zeros of stage 0; stage k
// is reached by advancing the base pointers k planes.
struct TileOut {
    uint32_t *codes;
    char *scales;        // binary32, or 16-bit patterns (the kernel's SC)
    float *zeros;
    int64_t words_per_stage, n_groups;
    uint32_t shares_here;   // lane shares of groups in the tile (codes)
    uint32_t groups_here;   // groups in the tile (scales, zeros)
};

// Scale storage SC (kScaleF32, kScaleF16, kScaleBF16): the binary32 value of
// the stored scale, nearest-even, and its stored bit pattern.
template <int SC>
__device__ __forceinline__ float round_scale(float s)
{
    if constexpr (SC == kScaleF16) {
        return (float)(_Float16)s;
    } else if constexpr (SC == kScaleBF16) {
        uint32_t u = __float_as_uint(s);
        u = (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;   // finite, non-negative s
        return __uint_as_float(u);
    } else {
        return s;
    }
}

// Stores one stage of a tile. With active false the same store instructions
// go to zero-sized resources and are dropped: every tile then issues the same
// sequence of vector-memory operations whatever the stage count, which lets
// the wait for the prefetched tile at the top of the tile loop count past
// the previous tile's stores instead of draining them (loads and stores share
// one in-order counter on this architecture).
template <int E, int L, int ZP, int SC>
__device__ __forceinline__ void store_stage(const TileOut &o, int k, int lane,
                                            const uint32_t (&words)[E / 16], float s, float z,
                                            bool active = true)
{
    // Lanes past the last group fall outside the resources; their stores
    // are dropped. The L lanes of a group store the same scale and zero-point
    // to the same address.
    // (read back as wave-uniform values: the resources must stay scalar)
    const uint32_t shares = __builtin_amdgcn_readfirstlane(active ? o.shares_here : 0u);
    const uint32_t groups = __builtin_amdgcn_readfirstlane(active ? o.groups_here : 0u);
    const uint32_t gl = (uint32_t)lane / L;
    store_words<E>(make_rsrc(o.codes + k * o.words_per_stage, shares * (E / 16) * 4),
                   lane * (E / 16) * 4, words);
    if constexpr (SC == kScaleF32) {
        __builtin_amdgcn_raw_buffer_store_b32(
            __float_as_uint(s), make_rsrc(o.scales + k * o.n_groups * 4, groups * 4),
            gl * 4, 0, 0);
    } else {
        // s already holds a value of the 16-bit type: the conversion is exact
        const uint16_t b = SC == kScaleF16 ? __builtin_bit_cast(uint16_t, (_Float16)s)
                                           : (uint16_t)(__float_as_uint(s) >> 16);
        __builtin_amdgcn_raw_buffer_store_b16(
            b, make_rsrc(o.scales + k * o.n_groups * 2, groups * 2), gl * 2, 0, 0);
    }
    if constexpr (ZP != kZpSymmetric)
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(z),
                                              make_rsrc(o.zeros + k * o.n_groups, groups * 4),
                                              gl * 4, 0, 0);
}

// fl(d / 3) for every finite d >= 0 in five fewer dependent steps than the
// IEEE division sequence: q = fl(d fl(1/3)) is within an ulp of d / 3, the
// first FMA gives the remainder d - 3q exactly, and the second rounds the
// corrected quotient q + (d - 3q) fl(1/3) once. It equals IEEE d / 3 on every
// non-negative finite binary32 (an exhaustive check of the same arithmetic
// runs with the CPU tests).
__device__ __forceinline__ float div3(float d)
{
    constexpr float kThird = 0x1.555556p-2f;   // fl(1/3)
    const float q = d * kThird;
    const float rem = __builtin_fmaf(-3.0f, q, d);
    return __builtin_fmaf(rem, kThird, q);
}

// Scale, reciprocal, zero-point and magic addend of one stage from the
// group's range (lo <= 0 <= hi), in stage format (ZP, SC): the scale
// is rounded to its storage type first and the rounded value is used.
template <int ZP, int SC>
__device__ __forceinline__ void stage_params(float lo, float hi, float &inv, float &sq, float &z,
                                             float &m)
{
    // lo <= 0, so |lo| is exactly 0 - lo, +0 included. Written as fabs: the
    // code generator folds 0 - lo into a negate modifier, which turns lo = +0
    // into -0 and would store z = -0.
    float d;
    if constexpr (ZP == kZpSymmetric) {
        const float amax = fmaxf(fabsf(lo), hi);
        d = amax + amax;                     // range [-amax, amax]
    } else {
        d = hi - lo;
    }
    const float s = round_scale<SC>(div3(d));
    const bool degenerate = !(s >= 0x1p-126f);
    inv = degenerate ? 0.0f : 1.0f / s;
    sq = degenerate ? 0.0f : s;
    // integer zero-point: RNE of the exact |lo| inv, by the same magic addend
    if constexpr (ZP == kZpInteger) z = __builtin_fmaf(fabsf(lo), inv, kMagic) - kMagic;
    else if constexpr (ZP == kZpReal) z = fabsf(lo) * inv;
    else z = 2.0f;
    m = kMagic + z;
}

// Two 32-bit LDS writes at addr + O0 * 256 and addr + O1 * 256 bytes, from two
// independent registers (a 64-bit write would need them in adjacent
// registers, i.e. copies).
template <int O0, int O1>
__device__ __forceinline__ void lds_write2st64(uint32_t addr, float a, float b)
{
    asm volatile("ds_write2st64_b32 %0, %1, %2 offset0:%3 offset1:%4"
                 :: "v"(addr), "v"(a), "v"(b), "i"(O0), "i"(O1) : "memory");
}

template <int I = 0>
__device__ __forceinline__ void write_table_entries(uint32_t addr, const float (&t)[4])
{
    if constexpr (I < 16) {
        // entry I: its two values at I * 512 and I * 512 + 256 bytes
        lds_write2st64<2 * I, 2 * I + 1>(addr, t[I & 3], t[I >> 2]);
        write_table_entries<I + 1>(addr, t);
    }
}

// Fills this lane's dequantization table for the stage: entry k0 + 4 k1 is
// {fl((3 - k0 - z) s), fl((3 - k1 - z) s)}.
__device__ __forceinline__ void fill_table(const DequantTable &tab, int lane, float sq, float z)
{
    float t[4];   // t[k] = fl((Q - z) s) for Q = 3 - k
#pragma unroll
    for (int k = 0; k < 4; ++k) t[k] = ((float)(3 - k) - z) * sq;
    typedef __attribute__((address_space(3))) float lds_float;
    write_table_entries((uint32_t)(uintptr_t)(lds_float *)(tab.base + lane), t);
}

// Loads one lane's base stage (plane 0 of the package) for tile `tile`: its
// share's code words (E elements, L lanes per group), the group's scale and
// zero-point. Lanes past the input, and a tile past the end, read zeros.
template <int E, int L, int ZP, int SC>
__device__ __forceinline__ void load_base(const uint32_t *codes, const char *scales,
                                          const float *zeros, int64_t n_groups, int64_t tile,
                                          int lane, uint32_t (&bw)[E / 16], float &s0, float &z0)
{
    const int64_t left = n_groups * L - tile * 64;
    const int64_t first = left <= 0 ? 0 : tile * 64;          // first share of the tile
    const uint32_t shares_here = left <= 0 ? 0u : (uint32_t)(left < 64 ? left : 64);
    const int64_t g0 = first / L;
    const uint32_t groups_here = shares_here / L;
    const uint32_t gl = (uint32_t)lane / L;
    const rsrc_t rc = make_rsrc(codes + first * (E / 16), shares_here * (E / 16) * 4);
    if constexpr (E / 16 >= 4) {
#pragma unroll
        for (int i = 0; i < E / 16; i += 4) {
            const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(rc, lane * (E / 16) * 4 + 4 * i, 0, 0);
            bw[i] = x.x; bw[i + 1] = x.y; bw[i + 2] = x.z; bw[i + 3] = x.w;
        }
    } else {
        const u32x2 x = __builtin_amdgcn_raw_buffer_load_b64(rc, lane * (E / 16) * 4, 0, 0);
        bw[0] = x.x; bw[1] = x.y;
    }
    if constexpr (SC == kScaleF32) {
        s0 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
            make_rsrc(scales + g0 * 4, groups_here * 4), gl * 4, 0, 0));
    } else {
        const uint16_t b = __builtin_amdgcn_raw_buffer_load_b16(
            make_rsrc(scales + g0 * 2, groups_here * 2), gl * 2, 0, 0);
        s0 = SC == kScaleF16 ? (float)__builtin_bit_cast(_Float16, b)
                             : __uint_as_float((uint32_t)b << 16);
    }
    if constexpr (ZP == kZpSymmetric)
        z0 = 2.0f;
    else
        z0 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
            make_rsrc(zeros + g0, groups_here * 4), gl * 4, 0, 0));
}

// One group per lane (L = 1), or a group split over L = 2 or 4 consecutive
// lanes, each holding a contiguous share of E = G / L elements (for calls too
// small to give every wave many tiles: the serial work per wave and tile
// drops L-fold). A tile is 64 shares; every per-element step is the same, the
// group's range is combined across its lanes, and each lane then forms the
// same scale, reciprocal and zero-point.
// Waves per SIMD: a lane holding E = 128 elements keeps 128 residuals plus
// the prefetched next tile, so 256 VGPRs is the budget (two waves); E = 64
// needs 156 (three waves: the lookups in flight stay the same), E = 32 about
// 80 (four waves).
// FROM_BASE: plane 0 of codes / scales / zeros holds a base checkpoint on
// entry (read only); the kernel forms R_0 = W - dequant(base) and writes the
// residual stages 1 .. n_stages - 1 (n_stages >= 2).
// ZP: zero-point kind; SC: scale storage type. pmr (may be NULL; L = 1
// only): per-group peak-to-mean ratios of W as a side output. STATS_ONLY:
// only pmr.
constexpr int construct_waves_per_simd(int E) { return E >= 128 ? 2 : E >= 64 ? 3 : 4; }

// The tensors a construct launch covers. Tiles are numbered over the whole
// launch; a workgroup takes tiles first, first + stride, ... (the grid-stride
// loop), and each tile lies in one tensor: `locate` advances a tensor index
// (wave-uniform, only ever forward) to the tensor of tile t, `local` gives the
// tile's number within it.
struct OneTensor {
    const uint4 *W;
    uint32_t *codes;
    char *scales;
    float *zeros;
    int64_t groups;
    __device__ int64_t total_tiles(int L) const { return (groups * L + 63) / 64; }
    __device__ void locate(int64_t, int &) const {}
    __device__ int64_t local(int64_t t, int) const { return t; }
    __device__ const uint4 *w(int) const { return W; }
    __device__ uint32_t *c(int) const { return codes; }
    __device__ char *sc(int) const { return scales; }
    __device__ float *z(int) const { return zeros; }
    __device__ int64_t n_groups(int) const { return groups; }
};

// Several tensors, each its own package, their tiles back to back
// (ConstructMany of rrq_launch.h, in the kernel arguments): the resident
// waves walk the tiles in order, as over one flat stack, so that at any time
// they read and write one or two tensors' neighbouring tiles.
struct ManyTensors {
    const ConstructMany &a;
    __device__ int64_t total_tiles(int) const { return a.tile_first[a.n]; }
    __device__ void locate(int64_t t, int &i) const
    {
        while (i + 1 < a.n && t >= a.tile_first[i + 1]) ++i;
        i = __builtin_amdgcn_readfirstlane(i);
    }
    __device__ int64_t local(int64_t t, int i) const { return t - a.tile_first[i]; }
    __device__ const uint4 *w(int i) const { return static_cast<const uint4 *>(a.W[i]); }
    __device__ uint32_t *c(int i) const { return static_cast<uint32_t *>(a.codes[i]); }
    __device__ char *sc(int i) const { return static_cast<char *>(a.scales[i]); }
    __device__ float *z(int i) const { return static_cast<float *>(a.zeros[i]); }
    __device__ int64_t n_groups(int i) const { return a.n_groups[i]; }
};

template <int G, bool FROM_BASE, int ZP, int SC, bool STATS_ONLY, int L, class SRC>
__device__ __forceinline__ void construct_tiles(const SRC &src, int n_stages,
                                                float *__restrict__ pmr, int64_t first,
                                                int64_t stride)
{
    static_assert(L == 1 || !STATS_ONLY, "the peak-to-mean ratio needs one lane per group");
    if (FROM_BASE && n_stages < 2) return;
    constexpr int E = G / L;             // elements per lane
    static_assert(E >= 32, "a lane holds at least 32 elements");
    constexpr int CH = E / 8;            // 16-byte chunks (8 bfloat16) per lane share
    constexpr int HC = CH / 2;           // chunks per half share
    constexpr int WPG = E / 16;          // code words per lane share and stage
    constexpr int ROW = HC + 1;          // LDS row of one half share, padded by 16 bytes
    constexpr int SHARES_PER_LOAD = 64 / CH;
    // The tile is transposed through LDS half a share at a time. Padding each
    // row by one chunk spreads both access patterns over all banks: a row
    // write (lanes -> consecutive chunks of a share) and a column read
    // (lanes -> the same chunk of consecutive shares).
    __shared__ uint4 tile_lds[64 * ROW];
    __shared__ f32x2 table_lds[16 * 64];

    const int lane = threadIdx.x;
    const int64_t n_tiles = src.total_tiles(L);
    // A lane's loaded chunks all have the same index within their share
    // (lane % CH), so each lane writes in exactly one of the two passes.
    const int my_half = (lane % CH) / HC;
    uint4 *const wr_base = tile_lds + (lane / CH) * ROW + (lane % HC);
    const uint4 *const rd_base = tile_lds + lane * ROW;
    const DequantTable tab = {reinterpret_cast<float *>(table_lds),
                              __uint_as_float((uint32_t)lane * 4)};

    int64_t tile = first;
    int ti = 0;                  // tensor of the current tile
    src.locate(tile, ti);
    uint4 v[CH];
    uint32_t bw[WPG];            // base stage of the tile in v (with a base)
    float bs = 0.f, bz = 0.f;
    if (tile < n_tiles) {
        load_tile<CH>(src.w(ti), src.n_groups(ti) * L, src.local(tile, ti), lane, v);
        if constexpr (FROM_BASE)
            load_base<E, L, ZP, SC>(src.c(ti), src.sc(ti), src.z(ti), src.n_groups(ti),
                                    src.local(tile, ti), lane, bw, bs, bz);
    }
    // The stores of one tile, dropped (see store_stage): the loop is entered
    // with the same operations outstanding as after each tile.
    {
        // (distinct planes, so that no store looks overwritten by the next)
        const TileOut none = {src.c(ti), src.sc(ti), src.z(ti), 1, 1, 0u, 0u};
        const uint32_t zw[WPG] = {};
        if constexpr (L == 1) store_pmr<G>(pmr, 0, 0u, lane, 0.f, 0.f, 0.f);
        if constexpr (!STATS_ONLY) {
#pragma unroll
            for (int k = 0; k < kMaxStages; ++k)
                store_stage<E, L, ZP, SC>(none, k, lane, zw, 0.f, 0.f, false);
        }
    }

    for (; tile < n_tiles; tile += stride) {
        const int64_t n_groups = src.n_groups(ti);
        const int64_t n_shares = n_groups * L;
        const int64_t s0 = src.local(tile, ti) * 64;   // first share of the tile
        const uint32_t shares_here = (uint32_t)(n_shares - s0 < 64 ? n_shares - s0 : 64);
        const int64_t g0 = s0 / L;                     // first group of the tile
        const uint32_t groups_here = shares_here / L;

        float r[E];
        float bl0 = 0.f, bl1 = 0.f, bh0 = 0.f, bh1 = 0.f;   // range of R_0 (with a base)
        serial_priority(true);
        if constexpr (FROM_BASE) fill_table(tab, lane, bs, bz);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            __syncthreads();   // earlier reads of the buffer are complete
            if (my_half == h) {
#pragma unroll
                for (int i = 0; i < CH; ++i) wr_base[i * SHARES_PER_LOAD * ROW] = v[i];
            }
            __syncthreads();
            gather_half<E>(rd_base, h, r);
            // With a base checkpoint, R_0 = W - dequant(base), half by half.
            if constexpr (FROM_BASE) {
                if (h == 0) subtract_base_half<E, 0>(r, bw, tab, bl0, bl1, bh0, bh1);
                else subtract_base_half<E, 1>(r, bw, tab, bl0, bl1, bh0, bh1);
            }
        }

        serial_priority(false);
        // |x| sum for the peak-to-mean side output (the weights, before any stage)
        const bool stats = L == 1 && !FROM_BASE && pmr != nullptr;
        float abs_sum = 0.f;
        if (stats) abs_sum = group_abs_sum<E>(r);

        // Prefetch the next tile while this one is quantized.
        int tn = ti;             // tensor of the next tile
        src.locate(tile + stride, tn);
        load_tile<CH>(src.w(tn), src.n_groups(tn) * L, src.local(tile + stride, tn), lane, v);

        constexpr int64_t scale_bytes = SC == kScaleF32 ? 4 : 2;
        const TileOut out = {src.c(ti) + s0 * WPG, src.sc(ti) + g0 * scale_bytes, src.z(ti) + g0,
                             n_shares * WPG, n_groups, shares_here, groups_here};

        float lo, hi, inv = 0.f, sq = 0.f, z = 0.f, m = 0.f;
        uint32_t words[WPG] = {};
        if constexpr (FROM_BASE) {
            lo = fminf(bl0, bl1);
            hi = fmaxf(bh0, bh1);
            combine_range<L>(lo, hi);
        } else {
            serial_priority(true);
            group_range<E>(r, lo, hi);
            combine_range<L>(lo, hi);
            serial_priority(false);
        }
        if constexpr (L == 1) store_pmr<G>(pmr, g0, stats ? groups_here : 0u, lane, lo, hi, abs_sum);
        if constexpr (STATS_ONLY) continue;
        // Stage slots 0 .. kMaxStages - 2 hold the stages that update the
        // residual; a slot outside 1 + FROM_BASE .. n_stages - 1 computes
        // nothing and drops its stores.
#pragma unroll
        for (int k = 0; k + 1 < kMaxStages; ++k) {
            const bool active = k >= (FROM_BASE ? 1 : 0) && k + 1 < n_stages;
            if (active) {
                serial_priority(true);
                stage_params<ZP, SC>(lo, hi, inv, sq, z, m);
                fill_table(tab, lane, sq, z);
                stage_elements<E, true, ZP>(r, inv, m, z, tab, words, lo, hi);
                combine_range<L>(lo, hi);
            }
            store_stage<E, L, ZP, SC>(out, k, lane, words, sq, z, active);
        }
        // The next tile's base stage, loaded where the last stage leaves
        // registers free; only this stage's stores are issued after it.
        if constexpr (FROM_BASE)
            load_base<E, L, ZP, SC>(src.c(tn), src.sc(tn), src.z(tn), src.n_groups(tn),
                                    src.local(tile + stride, tn), lane, bw, bs, bz);
        serial_priority(true);
        stage_params<ZP, SC>(lo, hi, inv, sq, z, m);
        stage_elements<E, false, ZP>(r, inv, m, z, tab, words, lo, hi);
        store_stage<E, L, ZP, SC>(out, n_stages - 1, lane, words, sq, z);
        ti = tn;
    }
}

template <int G, bool FROM_BASE, int ZP, int SC, bool STATS_ONLY = false, int L = 1>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(
    construct_waves_per_simd(G / L), construct_waves_per_simd(G / L)))) void construct_kernel(
    const uint4 *__restrict__ W, int64_t n_groups, int n_stages, uint32_t *__restrict__ codes,
    char *__restrict__ scales, float *__restrict__ zeros, float *__restrict__ pmr)
{
    const OneTensor src = {W, codes, scales, zeros, n_groups};
    construct_tiles<G, FROM_BASE, ZP, SC, STATS_ONLY, L>(src, n_stages, pmr, blockIdx.x,
                                                         gridDim.x);
}

// Several tensors in one launch, each into its own package (integer
// zero-points, binary32 scales).
template <int G, int L>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(
    construct_waves_per_simd(G / L), construct_waves_per_simd(G / L)))) void construct_many_kernel(
    const ConstructMany a, int n_stages)
{
    const ManyTensors src = {a};
    construct_tiles<G, false, kZpInteger, kScaleF32, false, L>(src, n_stages, nullptr,
                                                               blockIdx.x, gridDim.x);
}

// Reconstruction. Lane work unit: a chunk of E consecutive elements whose
// output is 16 bytes (E = 8 for bfloat16, 4 for binary32), so that each store
// instruction of a wave writes 1 KiB contiguously. A wave handles tiles of
// 64 * U chunks; lane l owns chunks l, l + 64, ... of the tile, issues all of
// its loads (codes, scales, zeros of the K stages) before any arithmetic, and
// sums the stages of each element left to right: acc = rhat_0,
// acc = fl(acc + rhat_t).
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// x & 0x03030303, opaque to the compiler so that the byte conversions below
// stay single v_cvt_f32_ubyte instructions.
__device__ __forceinline__ uint32_t code_bytes(uint32_t x)
{
    uint32_t out;
    asm("v_and_b32 %0, 0x3030303, %1" : "=v"(out) : "v"(x));
    return out;
}

// SC16: 16-bit scales (binary16 when f16 is set, else bfloat16); SYM:
// symmetric stages (z = 2, no zeros stored).
// Cache-policy operand of the buffer intrinsics: nontemporal (gfx950 nt bit).
constexpr int kNontemporal = 2;

template <int K, bool OUT_BF16, int U, bool SC16, bool SYM>
__global__ __launch_bounds__(256) void reconstruct_kernel(const uint32_t *__restrict__ codes,
                                                          const char *__restrict__ scales,
                                                          const float *__restrict__ zeros,
                                                          int64_t n_elems, int64_t n_groups,
                                                          int g_shift, void *__restrict__ out,
                                                          int f16)
{
    constexpr int SB = SC16 ? 2 : 4;             // bytes per stored scale
    constexpr int E = OUT_BF16 ? 8 : 4;          // elements per chunk (16 output bytes)
    constexpr int CPW = 16 / E;                  // chunks per code word
    constexpr int TILE = 64 * U;                 // chunks per tile
    const int lane = threadIdx.x & 63;
    const int64_t n_chunks = n_elems / E;
    const int64_t n_words = n_elems / 16;
    const int64_t n_tiles = (n_chunks + TILE - 1) / TILE;
    const int64_t n_waves = (int64_t)gridDim.x * 4;
    // The wave index is uniform across the wave; saying so keeps the buffer
    // resources below in scalar registers.
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    for (int64_t tile = (int64_t)blockIdx.x * 4 + wave; tile < n_tiles; tile += n_waves) {
        const int64_t c0 = tile * TILE;                       // first chunk
        const uint32_t chunks_here = (uint32_t)(n_chunks - c0 < TILE ? n_chunks - c0 : TILE);
        const int64_t wfirst = c0 / CPW;
        const uint32_t words_here = (chunks_here + CPW - 1) / CPW;
        const int64_t gfirst = (c0 * E) >> g_shift;
        const uint32_t groups_here =
            (uint32_t)((((c0 + chunks_here) * E - 1) >> g_shift) - gfirst + 1);

        uint32_t cw[K][U];
        float sc[K][U], ze[K][U];
#pragma unroll
        for (int t = 0; t < K; ++t) {
            const rsrc_t rc = make_rsrc(codes + t * n_words + wfirst, words_here * 4);
            const rsrc_t rs = make_rsrc(scales + (t * n_groups + gfirst) * SB, groups_here * SB);
            const rsrc_t rz = make_rsrc(zeros + t * n_groups + gfirst, groups_here * 4);
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const uint32_t cl = j * 64 + lane;   // chunk within the tile
                const uint32_t gl = (uint32_t)((((c0 + cl) * E) >> g_shift) - gfirst);
                cw[t][j] = __builtin_amdgcn_raw_buffer_load_b32(rc, (cl / CPW) * 4, 0, 0);
                if constexpr (SC16) {
                    const uint16_t b = __builtin_amdgcn_raw_buffer_load_b16(rs, gl * 2, 0, 0);
                    sc[t][j] = f16 ? (float)__builtin_bit_cast(_Float16, b)
                                   : __uint_as_float((uint32_t)b << 16);
                } else {
                    sc[t][j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, gl * 4, 0, 0));
                }
                if constexpr (SYM)
                    ze[t][j] = 2.0f;
                else
                    ze[t][j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rz, gl * 4, 0, 0));
            }
        }

        const rsrc_t ro = make_rsrc(static_cast<char *>(out) + c0 * 16, chunks_here * 16);
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const uint32_t cl = j * 64 + lane;
            const int shift = (int)((c0 + cl) % CPW) * 2 * E;   // this chunk's codes in the word
            float acc[E];
#pragma unroll
            for (int t = 0; t < K; ++t) {
                const uint32_t bits = cw[t][j] >> shift;
                // byte b of cb[p] holds the code of element 4 b + p
                uint32_t cb[4];
#pragma unroll
                for (int p = 0; p < 4; ++p) cb[p] = code_bytes(bits >> (2 * p));
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const float q = (float)((cb[e & 3] >> (8 * (e >> 2))) & 0xFFu);
                    const float rh = (q - ze[t][j]) * sc[t][j];
                    acc[e] = t == 0 ? rh : acc[e] + rh;
                }
            }
            u32x4 v;
            if constexpr (OUT_BF16) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const f32x2 f = {acc[2 * i], acc[2 * i + 1]};
                    v[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
                }
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(acc[i]);
            }
            // nontemporal: the output is written once and not read back here
            // (1-2% faster than default stores in an A/B on the stack's size)
            __builtin_amdgcn_raw_buffer_store_b128(v, ro, cl * 16, 0, kNontemporal);
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

template <bool FROM_BASE, int ZP, int SC>
hipError_t launch_construct_s(const uint4 *w4, int64_t n_groups, int G, int S, uint32_t *codes,
                              char *scales, float *zeros, float *pmr, int lanes, int grid,
                              hipStream_t stream)
{
#define RRQ_CONSTRUCT_CASE(GS, LS)                                                                 \
    if (G == GS && lanes == LS)                                                                    \
        return launch(construct_kernel<GS, FROM_BASE, ZP, SC, false, LS>, grid, 64, stream, w4,   \
                      n_groups, S, codes, scales, zeros, pmr);
    RRQ_CONSTRUCT_CASE(32, 1) RRQ_CONSTRUCT_CASE(64, 1) RRQ_CONSTRUCT_CASE(128, 1)
    RRQ_CONSTRUCT_CASE(64, 2) RRQ_CONSTRUCT_CASE(128, 4)
#undef RRQ_CONSTRUCT_CASE
    return hipErrorInvalidValue;
}

template <bool FROM_BASE, int ZP>
hipError_t launch_construct_g(const uint4 *w4, int64_t n_groups, int G, int S, uint32_t *codes,
                              char *scales, float *zeros, float *pmr, int scale_type, int lanes,
                              int grid, hipStream_t stream)
{
    switch (scale_type) {
    case kScaleF32: return launch_construct_s<FROM_BASE, ZP, kScaleF32>(w4, n_groups, G, S, codes, scales, zeros, pmr, lanes, grid, stream);
    case kScaleF16: return launch_construct_s<FROM_BASE, ZP, kScaleF16>(w4, n_groups, G, S, codes, scales, zeros, pmr, lanes, grid, stream);
    case kScaleBF16: return launch_construct_s<FROM_BASE, ZP, kScaleBF16>(w4, n_groups, G, S, codes, scales, zeros, pmr, lanes, grid, stream);
    default: return hipErrorInvalidValue;
    }
}

template <bool FROM_BASE>
hipError_t launch_construct_b(const uint4 *w4, int64_t n_groups, int G, int S, uint32_t *codes,
                              char *scales, float *zeros, float *pmr, int zero_point,
                              int scale_type, int lanes, int grid, hipStream_t stream)
{
    switch (zero_point) {
    case kZpInteger: return launch_construct_g<FROM_BASE, kZpInteger>(w4, n_groups, G, S, codes, scales, zeros, pmr, scale_type, lanes, grid, stream);
    case kZpReal: return launch_construct_g<FROM_BASE, kZpReal>(w4, n_groups, G, S, codes, scales, zeros, pmr, scale_type, lanes, grid, stream);
    case kZpSymmetric: return launch_construct_g<FROM_BASE, kZpSymmetric>(w4, n_groups, G, S, codes, scales, zeros, pmr, scale_type, lanes, grid, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_construct(const uint16_t *W, int64_t n_groups, int G, int S,
                            uint32_t *codes, void *scales, float *zeros, float *pmr,
                            bool from_base, int zero_point, int scale_type, int lanes, int grid,
                            hipStream_t stream)
{
    if (lanes != 1 && pmr != nullptr) return hipErrorInvalidValue;
    const uint4 *w4 = reinterpret_cast<const uint4 *>(W);
    char *sc = static_cast<char *>(scales);
    return from_base ? launch_construct_b<true>(w4, n_groups, G, S, codes, sc, zeros, nullptr,
                                                zero_point, scale_type, lanes, grid, stream)
                     : launch_construct_b<false>(w4, n_groups, G, S, codes, sc, zeros, pmr,
                                                 zero_point, scale_type, lanes, grid, stream);
}

hipError_t launch_construct_many(const ConstructMany &a, int G, int S, int lanes, int grid,
                                 hipStream_t stream)
{
#define RRQ_MANY_CASE(GS, LS)                                                                      \
    if (G == GS && lanes == LS)                                                                    \
        return launch(construct_many_kernel<GS, LS>, grid, 64, stream, a, S);
    RRQ_MANY_CASE(32, 1) RRQ_MANY_CASE(64, 1) RRQ_MANY_CASE(128, 1)
    RRQ_MANY_CASE(64, 2) RRQ_MANY_CASE(128, 4)
#undef RRQ_MANY_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_group_pmr(const uint16_t *W, int64_t n_groups, int G, float *pmr, int grid,
                            hipStream_t stream)
{
    const uint4 *w4 = reinterpret_cast<const uint4 *>(W);
    uint32_t *nc = nullptr;
    char *ns = nullptr;
    float *nz = nullptr;
    switch (G) {
    case 32: return launch(construct_kernel<32, false, kZpInteger, kScaleF32, true>, grid, 64, stream, w4, n_groups, 1, nc, ns, nz, pmr);
    case 64: return launch(construct_kernel<64, false, kZpInteger, kScaleF32, true>, grid, 64, stream, w4, n_groups, 1, nc, ns, nz, pmr);
    case 128: return launch(construct_kernel<128, false, kZpInteger, kScaleF32, true>, grid, 64, stream, w4, n_groups, 1, nc, ns, nz, pmr);
    default: return hipErrorInvalidValue;
    }
}

template <int K, bool BF16, bool SC16, bool SYM>
hipError_t launch_reconstruct_k(const uint32_t *codes, const char *scales, const float *zeros,
                                int64_t n_elems, int64_t n_groups, int g_shift, void *out,
                                int f16, int grid, hipStream_t stream)
{
    return launch(reconstruct_kernel<K, BF16, reconstruct_chunks(K, BF16), SC16, SYM>,
                  grid, kReconstructThreads, stream, codes, scales, zeros, n_elems, n_groups,
                  g_shift, out, f16);
}

template <bool SC16, bool SYM>
hipError_t launch_reconstruct_f(const uint32_t *codes, const char *scales, const float *zeros,
                                int64_t n_elems, int64_t n_groups, int g_shift, int k, void *out,
                                bool out_bf16, int f16, int grid, hipStream_t stream)
{
#define RRQ_RECON_CASE(K)                                                                          \
    case K:                                                                                        \
        return out_bf16 ? launch_reconstruct_k<K, true, SC16, SYM>(codes, scales, zeros, n_elems,  \
                                                                   n_groups, g_shift, out, f16,    \
                                                                   grid, stream)                   \
                        : launch_reconstruct_k<K, false, SC16, SYM>(codes, scales, zeros, n_elems, \
                                                                    n_groups, g_shift, out, f16,   \
                                                                    grid, stream);
    switch (k) {
        RRQ_RECON_CASE(1) RRQ_RECON_CASE(2) RRQ_RECON_CASE(3) RRQ_RECON_CASE(4)
    default: return hipErrorInvalidValue;
    }
#undef RRQ_RECON_CASE
}

hipError_t launch_reconstruct(const uint32_t *codes, const void *scales, const float *zeros,
                              int64_t n_groups, int G, int S, int k, void *out, bool out_bf16,
                              int zero_point, int scale_type, int grid, hipStream_t stream)
{
    (void)S;
    const int64_t n_elems = n_groups * G;
    const int g_shift = G == 32 ? 5 : G == 64 ? 6 : 7;
    const char *sc = static_cast<const char *>(scales);
    const bool sc16 = scale_type != kScaleF32, sym = zero_point == kZpSymmetric;
    const int f16 = scale_type == kScaleF16;
    if (!sc16 && !sym)
        return launch_reconstruct_f<false, false>(codes, sc, zeros, n_elems, n_groups, g_shift, k, out, out_bf16, f16, grid, stream);
    if (!sc16 && sym)
        return launch_reconstruct_f<false, true>(codes, sc, zeros, n_elems, n_groups, g_shift, k, out, out_bf16, f16, grid, stream);
    if (sc16 && !sym)
        return launch_reconstruct_f<true, false>(codes, sc, zeros, n_elems, n_groups, g_shift, k, out, out_bf16, f16, grid, stream);
    return launch_reconstruct_f<true, true>(codes, sc, zeros, n_elems, n_groups, g_shift, k, out, out_bf16, f16, grid, stream);
}

}  // namespace rrq_detail

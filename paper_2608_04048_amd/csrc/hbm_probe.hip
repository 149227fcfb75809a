// Streaming probes. The mixed one has construction's read/write ratio
// (2 : 1.25): it reads every 16-byte chunk of src and writes 5 of every 8
// chunks to dst, each lane keeping four loads in flight before it stores. The
// read-only and write-only ones bound each direction on its own. The
// construct-pattern probe replays package construction's own memory traffic
// (its tiles, loads, LDS transpose, prefetch and the 16 stores per tile over
// 12 output planes) with no quantization arithmetic, and the
// reconstruct-pattern probe does the same for reconstruction (bfloat16 out).
// Two machine probes time the terms the linear-layer kernels are built from:
// the issue of v_mfma_f32_16x16x32_bf16 and of binary32 FMAs, alone and
// interleaved, and 16-byte LDS reads, each wave reporting the clock ticks
// (s_memtime) of its loop.

#include "hbm_probe.h"

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;
constexpr int kBlocksPerCU = 8;
// The construct kernel's launch: one-wave workgroups, 8 per compute unit.
constexpr int kConstructProbeBlocksPerCU = 8;

__global__ __launch_bounds__(kThreads) void stream_probe_kernel(const uint4 *__restrict__ src,
                                                                uint4 *__restrict__ dst,
                                                                int64_t n16)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads * kUnroll;
    for (int64_t base = (int64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; base < n16;
         base += stride) {
        uint4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t i = base + (int64_t)u * kThreads;
            if (i < n16) v[u] = src[i];
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t i = base + (int64_t)u * kThreads;
            // n16 is a multiple of 8, so (i >> 3) * 5 + (i & 7) < n16 / 8 * 5.
            if (i < n16 && (i & 7) < 5) dst[(i >> 3) * 5 + (i & 7)] = v[u];
        }
    }
}

// Read-only: eight nontemporal 16-byte loads in flight per lane; the XOR of
// everything read is folded per wave and XORed into *out.
constexpr int kReadUnroll = 8;

__global__ __launch_bounds__(kThreads) void read_probe_kernel(const uint4 *__restrict__ src,
                                                              int64_t n16, uint32_t *out)
{
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    uint32_t acc = 0;
    const int64_t stride = (int64_t)gridDim.x * kThreads * kReadUnroll;
    for (int64_t base = (int64_t)blockIdx.x * kThreads * kReadUnroll + threadIdx.x; base < n16;
         base += stride) {
        u32x4 v[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) {
            const int64_t i = base + (int64_t)u * kThreads;
            v[u] = i < n16 ? __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(src) + i)
                           : (u32x4){0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) acc ^= __shfl_xor(acc, d, 64);
    if ((threadIdx.x & 63) == 0) atomicXor(out, acc);
}

// Write-only: a workgroup fills 16 KiB tiles (four 16-byte stores per lane,
// each wave instruction covering 1 KiB), tiles taken in a grid-stride loop;
// one workgroup per CU (more concurrent write streams write more slowly here).
__global__ __launch_bounds__(kThreads) void write_probe_kernel(uint4 *__restrict__ dst,
                                                               int64_t n16, uint32_t value)
{
    const uint4 v = make_uint4(value, value, value, value);
    const int64_t stride = (int64_t)gridDim.x * kThreads * kUnroll;
    for (int64_t base = (int64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; base < n16;
         base += stride) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t i = base + (int64_t)u * kThreads;
            if (i < n16) dst[i] = v;
        }
    }
}

// Construct-pattern probe. One wave per workgroup takes tiles of 64 groups of
// G bfloat16 weights in a grid-stride loop, exactly as the construct kernel
// does: 16-byte loads with each wave instruction covering 1 KiB, the next tile
// prefetched into registers while the current one is handled, the tile
// transposed through LDS half a group at a time (rows padded by 16 bytes), and
// per stage the same store instructions into the same planes: the lane's
// G / 16 code words (16-byte stores, 2 KiB per wave instruction at G = 128),
// one 32-bit scale and one 32-bit zero-point (256 bytes per wave
// instruction). The values stored are XORs of the group's 32-bit words, so
// every load is live and the stores are checkable:
//   code word j of stage k  = (XOR of the group's words j, j + G/16, ...) ^ k
//   scale of stage k        = (group word 0) ^ k
//   zero of stage k         = (group word 1) ^ k
// Buffer resources drop stores past the last group and read zeros past the
// input, as in the construct kernel.
typedef uint32_t pu32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t pu32x2 __attribute__((ext_vector_type(2)));
using prsrc_t = __amdgpu_buffer_rsrc_t;

__device__ __forceinline__ prsrc_t probe_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

template <int CH>
__device__ __forceinline__ void probe_load_tile(const uint4 *__restrict__ W, int64_t n_groups,
                                                int64_t tile, int lane, pu32x4 (&v)[CH])
{
    const int64_t g0 = tile * 64;
    const int64_t left = n_groups - g0;
    const uint32_t bytes = left <= 0 ? 0u : (uint32_t)(left < 64 ? left : 64) * CH * 16;
    const prsrc_t src = probe_rsrc(W + (left <= 0 ? 0 : g0 * CH), bytes);
#pragma unroll
    for (int i = 0; i < CH; ++i)
        v[i] = __builtin_amdgcn_raw_buffer_load_b128(src, (i * 64 + lane) * 16, 0, 0);
}

template <int G>
__global__ __launch_bounds__(64) void construct_probe_kernel(const uint4 *__restrict__ W,
                                                             int64_t n_groups, int n_stages,
                                                             uint32_t *__restrict__ codes,
                                                             uint32_t *__restrict__ scales,
                                                             uint32_t *__restrict__ zeros)
{
    constexpr int CH = G / 8, HC = CH / 2, WPG = G / 16, ROW = HC + 1;
    constexpr int GROUPS_PER_LOAD = 64 / CH;
    __shared__ pu32x4 tile_lds[64 * ROW];

    const int lane = threadIdx.x;
    const int64_t n_tiles = (n_groups + 63) / 64;
    const int my_half = (lane % CH) / HC;
    pu32x4 *const wr_base = tile_lds + (lane / CH) * ROW + (lane % HC);
    const pu32x4 *const rd_base = tile_lds + lane * ROW;

    int64_t tile = blockIdx.x;
    pu32x4 v[CH];
    if (tile < n_tiles) probe_load_tile<CH>(W, n_groups, tile, lane, v);
    for (; tile < n_tiles; tile += gridDim.x) {
        const int64_t g0 = tile * 64;
        const uint32_t groups_here = (uint32_t)(n_groups - g0 < 64 ? n_groups - g0 : 64);
        uint32_t acc[WPG] = {};
        uint32_t w0 = 0, w1 = 0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            __syncthreads();
            if (my_half == h) {
#pragma unroll
                for (int i = 0; i < CH; ++i) wr_base[i * GROUPS_PER_LOAD * ROW] = v[i];
            }
            __syncthreads();
#pragma unroll
            for (int c = 0; c < HC; ++c) {
                const pu32x4 x = rd_base[c];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int wi = (h * HC + c) * 4 + q;   // word index within the group
                    acc[wi % WPG] ^= x[q];
                    if (wi == 0) w0 = x[q];
                    if (wi == 1) w1 = x[q];
                }
            }
        }
        probe_load_tile<CH>(W, n_groups, tile + gridDim.x, lane, v);
        const int64_t words_per_stage = n_groups * WPG;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t groups =
                __builtin_amdgcn_readfirstlane(k < n_stages ? groups_here : 0u);
            const prsrc_t rc = probe_rsrc(codes + k * words_per_stage + g0 * WPG,
                                          groups * WPG * 4);
            if constexpr (WPG >= 4) {
#pragma unroll
                for (int i = 0; i < WPG; i += 4) {
                    const pu32x4 o = {acc[i] ^ k, acc[i + 1] ^ k, acc[i + 2] ^ k, acc[i + 3] ^ k};
                    __builtin_amdgcn_raw_buffer_store_b128(o, rc, lane * WPG * 4 + 4 * i, 0, 0);
                }
            } else {
                const pu32x2 o = {acc[0] ^ k, acc[1] ^ k};
                __builtin_amdgcn_raw_buffer_store_b64(o, rc, lane * WPG * 4, 0, 0);
            }
            __builtin_amdgcn_raw_buffer_store_b32(
                w0 ^ k, probe_rsrc(scales + k * n_groups + g0, groups * 4), lane * 4, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b32(
                w1 ^ k, probe_rsrc(zeros + k * n_groups + g0, groups * 4), lane * 4, 0, 0);
        }
    }
}

// Reconstruct-pattern probe: the reconstruct kernel's memory traffic for
// bfloat16 output with no dequantization arithmetic. Workgroups of four
// waves; a wave takes tiles of 64 U chunks of 8 elements (16 output bytes)
// in a grid-stride loop, lane l owning chunks l, l + 64, ...; for each of the
// k stages it loads the chunk's code word, its group's scale and its
// group's zero-point (32-bit each), then stores the chunk with one 16-byte
// store (each wave instruction covers 1 KiB). The stored chunk c is
// {x, x + 1, x + 2, x + 3} with x the XOR over the k stages of those three
// loaded words.
template <int K, int U>
__global__ __launch_bounds__(256) void reconstruct_probe_kernel(const uint32_t *__restrict__ codes,
                                                                const uint32_t *__restrict__ scales,
                                                                const uint32_t *__restrict__ zeros,
                                                                int64_t n_elems, int64_t n_groups,
                                                                int g_shift,
                                                                uint32_t *__restrict__ out)
{
    constexpr int E = 8, CPW = 2, TILE = 64 * U;
    const int lane = threadIdx.x & 63;
    const int64_t n_chunks = n_elems / E, n_words = n_elems / 16;
    const int64_t n_tiles = (n_chunks + TILE - 1) / TILE;
    const int64_t n_waves = (int64_t)gridDim.x * 4;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    for (int64_t tile = (int64_t)blockIdx.x * 4 + wave; tile < n_tiles; tile += n_waves) {
        const int64_t c0 = tile * TILE;
        const uint32_t chunks_here = (uint32_t)(n_chunks - c0 < TILE ? n_chunks - c0 : TILE);
        const int64_t wfirst = c0 / CPW;
        const uint32_t words_here = (chunks_here + CPW - 1) / CPW;
        const int64_t gfirst = (c0 * E) >> g_shift;
        const uint32_t groups_here =
            (uint32_t)((((c0 + chunks_here) * E - 1) >> g_shift) - gfirst + 1);
        uint32_t acc[U] = {};
#pragma unroll
        for (int t = 0; t < K; ++t) {
            const prsrc_t rc = probe_rsrc(codes + t * n_words + wfirst, words_here * 4);
            const prsrc_t rs = probe_rsrc(scales + t * n_groups + gfirst, groups_here * 4);
            const prsrc_t rz = probe_rsrc(zeros + t * n_groups + gfirst, groups_here * 4);
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const uint32_t cl = j * 64 + lane;
                const uint32_t gl = (uint32_t)((((c0 + cl) * E) >> g_shift) - gfirst);
                acc[j] ^= __builtin_amdgcn_raw_buffer_load_b32(rc, (cl / CPW) * 4, 0, 0) ^
                          __builtin_amdgcn_raw_buffer_load_b32(rs, gl * 4, 0, 0) ^
                          __builtin_amdgcn_raw_buffer_load_b32(rz, gl * 4, 0, 0);
            }
        }
        const prsrc_t ro = probe_rsrc(out + c0 * 4, chunks_here * 16);
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const pu32x4 v = {acc[j], acc[j] + 1, acc[j] + 2, acc[j] + 3};
            __builtin_amdgcn_raw_buffer_store_b128(v, ro, (j * 64 + lane) * 16, 0, 0);
        }
    }
}

int grid_limit(int per_cu, int64_t work, int per_block, int *grid)
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return 7;
    int64_t blocks = (work + per_block - 1) / per_block;
    if (blocks > (int64_t)cus * per_cu) blocks = (int64_t)cus * per_cu;
    *grid = (int)blocks;
    return 0;
}

}  // namespace

namespace {

// ---- machine probes ----

typedef float f32x4p __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8p __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4p __attribute__((ext_vector_type(4)));

// Per iteration: NM MFMAs over 4 accumulator chains (distinct operands per
// chain and round, so that none is folded away) and NV FMAs over 8 chains.
template <int NM, int NV>
__global__ __launch_bounds__(256) void issue_probe_kernel(float *out, long long *ticks, int iters)
{
    const uint32_t t = threadIdx.x;
    const u32x4p a0 = {0x3F803F80u ^ t, 0x3F803F81u, 0x3F803F82u, 0x3F803F83u};
    const u32x4p b0 = {0x3F803F84u, 0x3F803F85u ^ t, 0x3F803F86u, 0x3F803F87u};
    u32x4p b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) b[i] = b0 ^ (u32x4p){0u, (uint32_t)i << 1, 0u, 0u};
    f32x4p acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = (f32x4p){0.f, 0.f, 0.f, 0.f};
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (float)(t + i);
    u32x4p a = a0;
    const long long c0 = __builtin_amdgcn_s_memtime();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int m = 0; m < NM; ++m)
            acc[m & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8p, a), __builtin_bit_cast(bf16x8p, b[m & 3]), acc[m & 3], 0, 0, 0);
#pragma unroll
        for (int k = 0; k < NV; ++k) v[k & 7] = __builtin_fmaf(v[k & 7], 1.0001f, 0.5f);
        a[2] += 1u;
    }
    const long long c1 = __builtin_amdgcn_s_memtime();
    float r = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) r += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
#pragma unroll
    for (int i = 0; i < 8; ++i) r += v[i];
    const size_t idx = (size_t)blockIdx.x * blockDim.x + t;
    out[idx] = r;
    if ((t & 63) == 0) ticks[idx >> 6] = c1 - c0;
}

// Each lane reads 16 bytes per instruction from a 96 KiB LDS array (one
// workgroup per compute unit), distinct 16-byte slots across the wave, 16
// reads per iteration.
constexpr int kLdsProbeWords = 24576;   // 96 KiB
__global__ __launch_bounds__(512) void lds_probe_kernel(uint32_t *out, long long *ticks, int iters)
{
    __shared__ __attribute__((aligned(16))) uint32_t buf[kLdsProbeWords];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    for (int i = t; i < kLdsProbeWords; i += blockDim.x) buf[i] = (uint32_t)i * 2654435761u;
    __syncthreads();
    u32x4p acc = {0u, 0u, 0u, 0u};
    const uint32_t base = (uint32_t)(wave * 1024 + lane * 16);
    const long long c0 = __builtin_amdgcn_s_memtime();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const uint32_t off = (base + (uint32_t)k * 8192u + (uint32_t)it * 16u) % (4u * kLdsProbeWords);
            acc ^= *reinterpret_cast<const u32x4p *>(reinterpret_cast<const char *>(buf) + (off & ~15u));
        }
    }
    const long long c1 = __builtin_amdgcn_s_memtime();
    const size_t idx = (size_t)blockIdx.x * blockDim.x + t;
    out[idx] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
    if (lane == 0) ticks[idx >> 6] = c1 - c0;
}

int cu_count()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    return cus;
}

}  // namespace

extern "C" int hbm_probe_issue(int mode, int waves_per_simd, int iters, float *out, size_t out_len,
                               long long *ticks, size_t ticks_len, hipStream_t stream)
{
    if (!out || !ticks) return 1;
    if (mode < 0 || mode > 2 || waves_per_simd < 1 || waves_per_simd > 4 || iters < 1) return 3;
    const int cus = cu_count();
    if (cus <= 0) return 7;
    const int grid = cus * waves_per_simd;              // 4 waves per workgroup, one per SIMD
    if (out_len < (size_t)grid * 256 || ticks_len < (size_t)grid * 4) return 3;
    if (mode == 0)
        hipLaunchKernelGGL((issue_probe_kernel<16, 0>), dim3(grid), dim3(256), 0, stream, out, ticks, iters);
    else if (mode == 1)
        hipLaunchKernelGGL((issue_probe_kernel<0, 64>), dim3(grid), dim3(256), 0, stream, out, ticks, iters);
    else
        hipLaunchKernelGGL((issue_probe_kernel<16, 64>), dim3(grid), dim3(256), 0, stream, out, ticks, iters);
    return hipGetLastError() == hipSuccess ? 0 : 7;
}

extern "C" int hbm_probe_lds(int waves_per_cu, int iters, uint32_t *out, size_t out_len,
                             long long *ticks, size_t ticks_len, hipStream_t stream)
{
    if (!out || !ticks) return 1;
    if ((waves_per_cu != 4 && waves_per_cu != 8) || iters < 1) return 3;
    const int cus = cu_count();
    if (cus <= 0) return 7;
    const int block = 64 * waves_per_cu;
    if (out_len < (size_t)cus * block || ticks_len < (size_t)cus * waves_per_cu) return 3;
    hipLaunchKernelGGL(lds_probe_kernel, dim3(cus), dim3(block), 0, stream, out, ticks, iters);
    return hipGetLastError() == hipSuccess ? 0 : 7;
}

extern "C" int hbm_probe_read(const void *src, size_t src_bytes, uint32_t *out,
                              hipStream_t stream)
{
    if (!src || !out) return 1;
    if (reinterpret_cast<uintptr_t>(src) % 16 != 0 || reinterpret_cast<uintptr_t>(out) % 4 != 0)
        return 2;
    if (src_bytes == 0 || src_bytes % 16 != 0 || src_bytes > (size_t)INT64_MAX) return 3;
    const int64_t n16 = (int64_t)(src_bytes / 16);
    int grid = 0;
    if (grid_limit(kBlocksPerCU, n16, kThreads * kReadUnroll, &grid)) return 7;
    hipLaunchKernelGGL(read_probe_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream,
                       static_cast<const uint4 *>(src), n16, out);
    return hipGetLastError() == hipSuccess ? 0 : 7;
}

extern "C" int hbm_probe_write(void *dst, size_t dst_bytes, uint32_t value, hipStream_t stream)
{
    if (!dst) return 1;
    if (reinterpret_cast<uintptr_t>(dst) % 16 != 0) return 2;
    if (dst_bytes == 0 || dst_bytes % 16 != 0 || dst_bytes > (size_t)INT64_MAX) return 3;
    const int64_t n16 = (int64_t)(dst_bytes / 16);
    int grid = 0;
    if (grid_limit(1, n16, kThreads * kUnroll, &grid)) return 7;
    hipLaunchKernelGGL(write_probe_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream,
                       static_cast<uint4 *>(dst), n16, value);
    return hipGetLastError() == hipSuccess ? 0 : 7;
}

extern "C" int hbm_probe_stream(const void *src, size_t src_bytes, void *dst, hipStream_t stream)
{
    if (!src || !dst) return 1;
    if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16 != 0) return 2;
    if (src_bytes == 0 || src_bytes % 128 != 0 || src_bytes > (size_t)INT64_MAX) return 3;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return 7;
    const int64_t n16 = (int64_t)(src_bytes / 16);
    const int64_t per_block = (int64_t)kThreads * kUnroll;
    int64_t blocks = (n16 + per_block - 1) / per_block;
    if (blocks > (int64_t)cus * kBlocksPerCU) blocks = (int64_t)cus * kBlocksPerCU;
    hipLaunchKernelGGL(stream_probe_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                       static_cast<const uint4 *>(src), static_cast<uint4 *>(dst), n16);
    return hipGetLastError() == hipSuccess ? 0 : 7;
}

extern "C" int hbm_probe_construct(const void *W, int64_t n_groups, int32_t group_size,
                                   int32_t n_stages, uint32_t *codes, uint32_t *scales,
                                   uint32_t *zeros, int32_t blocks_per_cu, hipStream_t stream)
{
    if (!W || !codes || !scales || !zeros) return 1;
    if ((reinterpret_cast<uintptr_t>(W) | reinterpret_cast<uintptr_t>(codes)) % 16 != 0 ||
        (reinterpret_cast<uintptr_t>(scales) | reinterpret_cast<uintptr_t>(zeros)) % 4 != 0)
        return 2;
    if (group_size != 32 && group_size != 64 && group_size != 128) return 3;
    if (n_groups < 1 || n_stages < 1 || n_stages > 4 || blocks_per_cu < 0 || blocks_per_cu > 32)
        return 3;
    // per-tile offsets of every plane stay in 64-bit pointers; sizes per
    // tile fit 32 bits
    if (n_groups > INT64_MAX / (4 * group_size)) return 3;
    int grid = 0;
    if (grid_limit(blocks_per_cu ? blocks_per_cu : kConstructProbeBlocksPerCU, n_groups, 64,
                   &grid))
        return 7;
    const uint4 *w4 = static_cast<const uint4 *>(W);
    switch (group_size) {
    case 32:
        hipLaunchKernelGGL(construct_probe_kernel<32>, dim3((unsigned)grid), dim3(64), 0, stream,
                           w4, n_groups, (int)n_stages, codes, scales, zeros);
        break;
    case 64:
        hipLaunchKernelGGL(construct_probe_kernel<64>, dim3((unsigned)grid), dim3(64), 0, stream,
                           w4, n_groups, (int)n_stages, codes, scales, zeros);
        break;
    default:
        hipLaunchKernelGGL(construct_probe_kernel<128>, dim3((unsigned)grid), dim3(64), 0, stream,
                           w4, n_groups, (int)n_stages, codes, scales, zeros);
        break;
    }
    return hipGetLastError() == hipSuccess ? 0 : 7;
}

extern "C" int hbm_probe_reconstruct(const uint32_t *codes, const uint32_t *scales,
                                     const uint32_t *zeros, int64_t n_groups, int32_t group_size,
                                     int32_t k_stages, uint32_t *out, int32_t blocks_per_cu,
                                     hipStream_t stream)
{
    if (!codes || !scales || !zeros || !out) return 1;
    if ((reinterpret_cast<uintptr_t>(codes) | reinterpret_cast<uintptr_t>(out)) % 16 != 0 ||
        (reinterpret_cast<uintptr_t>(scales) | reinterpret_cast<uintptr_t>(zeros)) % 4 != 0)
        return 2;
    if (group_size != 32 && group_size != 64 && group_size != 128) return 3;
    if (n_groups < 1 || k_stages < 1 || k_stages > 4 || blocks_per_cu < 0 || blocks_per_cu > 32)
        return 3;
    if (n_groups > INT64_MAX / (4 * group_size)) return 3;
    const int64_t n = n_groups * group_size;
    const int g_shift = group_size == 32 ? 5 : group_size == 64 ? 6 : 7;
    // the reconstruct kernel's launch for bfloat16 output: 8 chunks per lane
    // for 1 or 2 stages, 4 from 3 on; two workgroups of 256 per CU
    const int U = k_stages <= 2 ? 8 : 4;
    int grid = 0;
    if (grid_limit(blocks_per_cu ? blocks_per_cu : 2, n, kThreads * U * 8, &grid)) return 7;
#define RRQ_PROBE_RECON(KK, UU)                                                                   \
    case KK:                                                                                       \
        hipLaunchKernelGGL((reconstruct_probe_kernel<KK, UU>), dim3((unsigned)grid), dim3(kThreads), \
                           0, stream, codes, scales, zeros, n, n_groups, g_shift, out);           \
        break;
    switch (k_stages) {
        RRQ_PROBE_RECON(1, 8) RRQ_PROBE_RECON(2, 8) RRQ_PROBE_RECON(3, 4) RRQ_PROBE_RECON(4, 4)
    default: return 3;
    }
#undef RRQ_PROBE_RECON
    return hipGetLastError() == hipSuccess ? 0 : 7;
}

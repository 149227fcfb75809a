// Streaming probes. The mixed one has construction's read/write ratio
// (2 : 1.25): it reads every 16-byte chunk of src and writes 5 of every 8
// chunks to dst, each lane keeping four loads in flight before it stores. The
// read-only and write-only ones bound each direction on its own.

#include "hbm_probe.h"

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;
constexpr int kBlocksPerCU = 8;

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

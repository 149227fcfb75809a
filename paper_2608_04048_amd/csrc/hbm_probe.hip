// Streaming probe with construction's read/write ratio (2 : 1.25): reads
// every 16-byte chunk of src and writes 5 of every 8 chunks to dst. Each lane
// keeps four loads in flight before it stores.

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

}  // namespace

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

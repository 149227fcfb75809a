// C ABI of librrq.so (declared in include/rrq.h): argument validation, package
// sizes, launch geometry and HIP error mapping. Every entry point validates
// its arguments before enqueueing anything and never throws.

#include "rrq.h"

#include <atomic>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "rrq_launch.h"

namespace {

constexpr int kMaxDevices = 64;
std::atomic<int> g_cu_count[kMaxDevices];   // 0 = not yet queried

// Compute units of the current device (cached; read-only after first use).
int current_cu_count()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return -1;
    if (dev < kMaxDevices) {
        int c = g_cu_count[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return -1;
    if (dev < kMaxDevices) g_cu_count[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Shape / group / stage checks shared by every entry point. On success *n is
// rows * cols.
int check_common(int64_t rows, int64_t cols, int32_t G, int32_t S, int64_t *n)
{
    if (G != 32 && G != 64 && G != 128) return RRQ_ERR_GROUP;
    if (S < 1 || S > RRQ_MAX_STAGES) return RRQ_ERR_STAGES;
    if (rows < 1 || cols < 1 || cols % G != 0) return RRQ_ERR_SHAPE;
    int64_t prod = 0;
    // Byte counts (up to 4 bytes per element) must fit in int64.
    if (__builtin_mul_overflow(rows, cols, &prod) || prod > INT64_MAX / 4) return RRQ_ERR_SHAPE;
    *n = prod;
    return RRQ_OK;
}

// Stage-format checks: zero-point kind, scale type, and the alignment and
// presence of the scales and zeros buffers they imply (zeros may be NULL for
// symmetric stages, which store none).
int check_format(int32_t zero_point, int32_t scale_type, const void *scales, const void *zeros)
{
    if (zero_point != RRQ_ZP_INTEGER && zero_point != RRQ_ZP_REAL &&
        zero_point != RRQ_ZP_SYMMETRIC)
        return RRQ_ERR_FORMAT;
    if (scale_type != RRQ_SCALE_F32 && scale_type != RRQ_SCALE_F16 && scale_type != RRQ_SCALE_BF16)
        return RRQ_ERR_FORMAT;
    if (!scales || (zero_point != RRQ_ZP_SYMMETRIC && !zeros)) return RRQ_ERR_NULL;
    if (!aligned(scales, scale_type == RRQ_SCALE_F32 ? 4 : 2) || (zeros && !aligned(zeros, 4)))
        return RRQ_ERR_ALIGN;
    return RRQ_OK;
}

int grid_for(int64_t work_items, int per_block, int blocks_per_cu, int *grid)
{
    const int cus = current_cu_count();
    if (cus <= 0) return RRQ_ERR_HIP;
    const int64_t blocks = (work_items + per_block - 1) / per_block;
    const int64_t cap = (int64_t)cus * blocks_per_cu;
    *grid = (int)(blocks < cap ? blocks : cap);
    return RRQ_OK;
}

// Construction with or without a base stage, in any stage format.
int construct_common(const uint16_t *W, int64_t rows, int64_t cols, int32_t group_size,
                     int32_t n_stages, int32_t zero_point, int32_t scale_type, uint32_t *codes,
                     void *scales, float *zeros, bool from_base, hipStream_t stream,
                     float *pmr = nullptr)
{
    if (!W || !codes) return RRQ_ERR_NULL;
    int64_t n = 0;
    int st = check_common(rows, cols, group_size, n_stages, &n);
    if (st != RRQ_OK) return st;
    st = check_format(zero_point, scale_type, scales, zeros);
    if (st != RRQ_OK) return st;
    if (!aligned(W, 16) || !aligned(codes, 16) || (pmr && !aligned(pmr, 4))) return RRQ_ERR_ALIGN;
    if (from_base && n_stages == 1) return RRQ_OK;   // the package is the base alone
    const int64_t n_groups = n / group_size;
    const int cus = current_cu_count();
    if (cus <= 0) return RRQ_ERR_HIP;
    const int lanes = rrq_detail::construct_lanes(n_groups, group_size, pmr != nullptr, cus);
    int grid = 0;
    st = grid_for(n_groups * lanes, 64, rrq_detail::construct_blocks_per_cu(group_size, lanes), &grid);
    if (st != RRQ_OK) return st;
    hipError_t e = rrq_detail::launch_construct(W, n_groups, group_size, n_stages, codes, scales,
                                                zeros, pmr, from_base, zero_point, scale_type,
                                                lanes, grid, stream);
    return e == hipSuccess ? RRQ_OK : RRQ_ERR_HIP;
}

int reconstruct_common(const uint32_t *codes, const void *scales, const float *zeros,
                       int64_t rows, int64_t cols, int32_t group_size, int32_t n_stages,
                       int32_t zero_point, int32_t scale_type, int32_t k_stages, void *W_out,
                       int32_t out_dtype, hipStream_t stream)
{
    if (!codes || !W_out) return RRQ_ERR_NULL;
    int64_t n = 0;
    int st = check_common(rows, cols, group_size, n_stages, &n);
    if (st != RRQ_OK) return st;
    st = check_format(zero_point, scale_type, scales, zeros);
    if (st != RRQ_OK) return st;
    if (k_stages < 1 || k_stages > n_stages) return RRQ_ERR_STAGES;
    if (out_dtype != RRQ_F32 && out_dtype != RRQ_BF16) return RRQ_ERR_DTYPE;
    if (!aligned(codes, 16) || !aligned(W_out, 16)) return RRQ_ERR_ALIGN;
    const int64_t n_groups = n / group_size;
    int grid = 0;
    // one wave tile = 64 lanes x (4 or 8) chunks x (8 or 4) elements; 4 waves
    // per workgroup
    const bool bf16 = out_dtype == RRQ_BF16;
    const int per_lane = rrq_detail::reconstruct_chunks(k_stages, bf16) * (bf16 ? 8 : 4);
    st = grid_for(n, rrq_detail::kReconstructThreads * per_lane,
                  rrq_detail::reconstruct_blocks_per_cu(k_stages, bf16), &grid);
    if (st != RRQ_OK) return st;
    hipError_t e = rrq_detail::launch_reconstruct(codes, scales, zeros, n_groups, group_size,
                                                  n_stages, k_stages, W_out,
                                                  out_dtype == RRQ_BF16, zero_point, scale_type,
                                                  grid, stream);
    return e == hipSuccess ? RRQ_OK : RRQ_ERR_HIP;
}

int linear_common(const uint32_t *codes, const void *scales, const float *zeros, int64_t rows,
                  int64_t cols, int32_t group_size, int32_t n_stages, int32_t zero_point,
                  int32_t scale_type, int32_t k_stages, const uint16_t *X, int64_t n_tokens,
                  float *Y, hipStream_t stream)
{
    if (!codes || !X || !Y) return RRQ_ERR_NULL;
    int64_t n = 0;
    int st = check_common(rows, cols, group_size, n_stages, &n);
    if (st != RRQ_OK) return st;
    st = check_format(zero_point, scale_type, scales, zeros);
    if (st != RRQ_OK) return st;
    if (k_stages < 1 || k_stages > n_stages) return RRQ_ERR_STAGES;
    if (n_tokens < 1 || rows >= rrq_detail::kLinearMaxDim || cols >= rrq_detail::kLinearMaxDim)
        return RRQ_ERR_SHAPE;
    // the k stage planes the kernel reads span less than 4 GiB of codes
    if ((uint64_t)k_stages * (uint64_t)(n / 4) >= (uint64_t(1) << 32)) return RRQ_ERR_SHAPE;
    if (!aligned(codes, 16) || !aligned(X, 16) || !aligned(Y, 4)) return RRQ_ERR_ALIGN;
    const int cus = current_cu_count();
    if (cus <= 0) return RRQ_ERR_HIP;
    hipError_t e;
    if (rrq_detail::linear_decode_fits(rows, cols, group_size, k_stages, n_tokens))
        e = rrq_detail::launch_linear_decode(codes, scales, zeros, rows, cols, k_stages, zero_point,
                                             scale_type, X, n_tokens, Y, cus, stream);
    else if (rrq_detail::linear_batch_fits(rows, cols, group_size, k_stages, n_tokens))
        e = rrq_detail::launch_linear_batch(codes, scales, zeros, rows, cols, k_stages, zero_point,
                                            scale_type, X, n_tokens, Y, cus, stream);
    else if (rrq_detail::linear_prefill_fits(rows, cols, group_size, n_tokens))
        e = rrq_detail::launch_linear_prefill(codes, scales, zeros, rows, cols, k_stages,
                                              zero_point, scale_type, X, n_tokens, Y, cus,
                                              stream);
    else
        e = rrq_detail::launch_linear(codes, scales, zeros, rows, cols, group_size, n_stages,
                                      k_stages, zero_point, scale_type, X, n_tokens, Y, stream);
    return e == hipSuccess ? RRQ_OK : RRQ_ERR_HIP;
}

}  // namespace

extern "C" int rrq_construct(const uint16_t *W, int64_t rows, int64_t cols, int32_t group_size,
                             int32_t n_stages, uint32_t *codes, float *scales, float *zeros,
                             hipStream_t stream)
{
    return construct_common(W, rows, cols, group_size, n_stages, RRQ_ZP_INTEGER, RRQ_SCALE_F32,
                            codes, scales, zeros, false, stream);
}

extern "C" int rrq_construct_many(const rrq_tensor *tensors, int32_t n_tensors,
                                  int32_t group_size, int32_t n_stages, hipStream_t stream)
{
    if (n_tensors < 0) return RRQ_ERR_SHAPE;
    if (n_tensors == 0) return RRQ_OK;
    if (!tensors) return RRQ_ERR_NULL;
    int64_t total_groups = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        const rrq_tensor &t = tensors[i];
        if (!t.W || !t.codes || !t.scales || !t.zeros) return RRQ_ERR_NULL;
        int64_t n = 0;
        const int st = check_common(t.rows, t.cols, group_size, n_stages, &n);
        if (st != RRQ_OK) return st;
        if (!aligned(t.W, 16) || !aligned(t.codes, 16) || !aligned(t.scales, 4) ||
            !aligned(t.zeros, 4))
            return RRQ_ERR_ALIGN;
        if (__builtin_add_overflow(total_groups, n / group_size, &total_groups))
            return RRQ_ERR_SHAPE;
    }
    const int cus = current_cu_count();
    if (cus <= 0) return RRQ_ERR_HIP;
    constexpr int kPer = rrq_detail::kConstructManyPerLaunch;
    for (int32_t c0 = 0; c0 < n_tensors; c0 += kPer) {
        const int32_t cn = n_tensors - c0 < kPer ? n_tensors - c0 : kPer;
        int64_t groups = 0;
        for (int32_t i = 0; i < cn; ++i)
            groups += tensors[c0 + i].rows * tensors[c0 + i].cols / group_size;
        // lanes per group and grid as for one flat call of this size
        const int lanes = rrq_detail::construct_lanes(groups, group_size, false, cus);
        rrq_detail::ConstructMany a = {};
        a.n = cn;
        int64_t tiles_all = 0;
        for (int32_t i = 0; i < cn; ++i) {
            const rrq_tensor &t = tensors[c0 + i];
            a.tile_first[i] = tiles_all;
            a.W[i] = t.W;
            a.codes[i] = t.codes;
            a.scales[i] = t.scales;
            a.zeros[i] = t.zeros;
            a.n_groups[i] = t.rows * t.cols / group_size;
            tiles_all += (a.n_groups[i] * lanes + 63) / 64;
        }
        a.tile_first[cn] = tiles_all;
        const int64_t cap = (int64_t)cus * rrq_detail::construct_blocks_per_cu(group_size, lanes);
        const int64_t wg = tiles_all < cap ? tiles_all : cap;
        const hipError_t e = rrq_detail::launch_construct_many(a, group_size, n_stages, lanes,
                                                               (int)wg, stream);
        if (e != hipSuccess) return RRQ_ERR_HIP;
    }
    return RRQ_OK;
}

extern "C" int rrq_construct_format(const uint16_t *W, int64_t rows, int64_t cols,
                                    int32_t group_size, int32_t n_stages, int32_t zero_point,
                                    int32_t scale_type, uint32_t *codes, void *scales,
                                    float *zeros, hipStream_t stream)
{
    return construct_common(W, rows, cols, group_size, n_stages, zero_point, scale_type, codes,
                            scales, zeros, false, stream);
}

extern "C" int rrq_construct_stats(const uint16_t *W, int64_t rows, int64_t cols,
                                   int32_t group_size, int32_t n_stages, int32_t zero_point,
                                   int32_t scale_type, uint32_t *codes, void *scales,
                                   float *zeros, float *pmr, hipStream_t stream)
{
    if (!pmr) return RRQ_ERR_NULL;
    return construct_common(W, rows, cols, group_size, n_stages, zero_point, scale_type, codes,
                            scales, zeros, false, stream, pmr);
}

extern "C" int rrq_group_pmr(const uint16_t *W, int64_t rows, int64_t cols, int32_t group_size,
                             float *pmr, hipStream_t stream)
{
    if (!W || !pmr) return RRQ_ERR_NULL;
    int64_t n = 0;
    int st = check_common(rows, cols, group_size, 1, &n);
    if (st != RRQ_OK) return st;
    if (!aligned(W, 16) || !aligned(pmr, 4)) return RRQ_ERR_ALIGN;
    const int64_t n_groups = n / group_size;
    int grid = 0;
    st = grid_for(n_groups, 64, rrq_detail::kConstructBlocksPerCU, &grid);
    if (st != RRQ_OK) return st;
    hipError_t e = rrq_detail::launch_group_pmr(W, n_groups, group_size, pmr, grid, stream);
    return e == hipSuccess ? RRQ_OK : RRQ_ERR_HIP;
}

extern "C" int rrq_construct_from_base(const uint16_t *W, int64_t rows, int64_t cols,
                                       int32_t group_size, int32_t n_stages, uint32_t *codes,
                                       float *scales, float *zeros, hipStream_t stream)
{
    return construct_common(W, rows, cols, group_size, n_stages, RRQ_ZP_INTEGER, RRQ_SCALE_F32,
                            codes, scales, zeros, true, stream);
}

extern "C" int rrq_construct_from_base_format(const uint16_t *W, int64_t rows, int64_t cols,
                                              int32_t group_size, int32_t n_stages,
                                              int32_t zero_point, int32_t scale_type,
                                              uint32_t *codes, void *scales, float *zeros,
                                              hipStream_t stream)
{
    return construct_common(W, rows, cols, group_size, n_stages, zero_point, scale_type, codes,
                            scales, zeros, true, stream);
}

extern "C" int rrq_reconstruct(const uint32_t *codes, const float *scales, const float *zeros,
                               int64_t rows, int64_t cols, int32_t group_size, int32_t n_stages,
                               int32_t k_stages, void *W_out, int32_t out_dtype,
                               hipStream_t stream)
{
    return reconstruct_common(codes, scales, zeros, rows, cols, group_size, n_stages,
                              RRQ_ZP_INTEGER, RRQ_SCALE_F32, k_stages, W_out, out_dtype, stream);
}

extern "C" int rrq_reconstruct_format(const uint32_t *codes, const void *scales,
                                      const float *zeros, int64_t rows, int64_t cols,
                                      int32_t group_size, int32_t n_stages, int32_t zero_point,
                                      int32_t scale_type, int32_t k_stages, void *W_out,
                                      int32_t out_dtype, hipStream_t stream)
{
    return reconstruct_common(codes, scales, zeros, rows, cols, group_size, n_stages, zero_point,
                              scale_type, k_stages, W_out, out_dtype, stream);
}

extern "C" int rrq_linear(const uint32_t *codes, const float *scales, const float *zeros,
                          int64_t rows, int64_t cols, int32_t group_size, int32_t n_stages,
                          int32_t k_stages, const uint16_t *X, int64_t n_tokens, float *Y,
                          hipStream_t stream)
{
    return linear_common(codes, scales, zeros, rows, cols, group_size, n_stages, RRQ_ZP_INTEGER,
                         RRQ_SCALE_F32, k_stages, X, n_tokens, Y, stream);
}

extern "C" int rrq_linear_format(const uint32_t *codes, const void *scales, const float *zeros,
                                 int64_t rows, int64_t cols, int32_t group_size, int32_t n_stages,
                                 int32_t zero_point, int32_t scale_type, int32_t k_stages,
                                 const uint16_t *X, int64_t n_tokens, float *Y, hipStream_t stream)
{
    return linear_common(codes, scales, zeros, rows, cols, group_size, n_stages, zero_point,
                         scale_type, k_stages, X, n_tokens, Y, stream);
}

extern "C" int rrq_package_bytes(int64_t rows, int64_t cols, int32_t group_size,
                                 int32_t n_stages, size_t *codes_bytes, size_t *scales_bytes)
{
    int64_t n = 0;
    const int st = check_common(rows, cols, group_size, n_stages, &n);
    if (st != RRQ_OK) return st;
    if (codes_bytes) *codes_bytes = (size_t)n_stages * (size_t)(n / 4);
    if (scales_bytes) *scales_bytes = (size_t)n_stages * (size_t)(n / group_size) * sizeof(float);
    return RRQ_OK;
}

extern "C" const char *rrq_status_string(int status)
{
    switch (status) {
    case RRQ_OK: return "success";
    case RRQ_ERR_NULL: return "a required pointer is NULL";
    case RRQ_ERR_ALIGN: return "a buffer is not aligned as required (16 bytes for W, codes, W_out and X; 4 for binary32 scales, zeros and Y; 2 for 16-bit scales)";
    case RRQ_ERR_SHAPE: return "bad shape: rows and cols must be >= 1, cols a multiple of group_size, rows*cols within range (and for rrq_linear rows, cols < 2^26, n_tokens >= 1)";
    case RRQ_ERR_GROUP: return "group_size must be 32, 64 or 128";
    case RRQ_ERR_STAGES: return "n_stages must be in 1..4 and k_stages in 1..n_stages";
    case RRQ_ERR_DTYPE: return "out_dtype must be RRQ_F32 or RRQ_BF16";
    case RRQ_ERR_HIP: return "the HIP runtime reported an error";
    case RRQ_ERR_FORMAT: return "zero_point must be an enum rrq_zero_point value and scale_type an enum rrq_scale_type value";
    default: return "unknown status";
    }
}

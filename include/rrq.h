/*
 * rrq.h - C ABI of librrq.so: Recurrent Residual Quantization (RRQ) package
 * construction and prefix reconstruction on AMD Instinct MI355X (gfx950).
 *
 * The method (paper: "Recurrent Residual Quantization: A Progressive
 * Multi-Precision Representation for LLMs"):
 *   - Eq. 1-3: a group of G weights shares a scale s and zero-point z;
 *     q = x/s + z, Q = R(q), and the stage leaves the residual
 *     r = x - (Q - z) s.
 *   - Eq. 4-7 and Algorithm 1: the base stage quantizes the weights (or an
 *     existing base checkpoint is loaded), each further stage quantizes the
 *     residual left by the stages before it; every stage stores its own
 *     codes, scales and zero-points.
 *   - Eq. 8 (restated as Eq. 18-19): the effective weight after t stages is
 *     the sum of the first t dequantized stages; Eq. 20: a linear layer on
 *     that weight is the sum of the stages' products.
 *   - Sec. 4.1: the main configuration is four calibration-free 2-bit RTN
 *     stages (2+2+2+2 bits) with group size 128, giving 2/4/6/8-bit prefixes.
 *
 * Arithmetic (the paper leaves it open; this library fixes it, and results
 * are bit-identical to that definition):
 *   residuals are IEEE binary32 and stay binary32 between stages;
 *   lo = min(+0, min r), hi = max(+0, max r) over the group;
 *   s = fl(fl(hi - lo) / 3); if s < 2^-126 (zero or subnormal) the group is
 *     degenerate for that stage: s = z = 0, all codes 0, residual unchanged;
 *   inv = fl(1 / s); z = RNE((0 - lo) * inv), an integer in {0,1,2,3};
 *   Q = clamp(RNE(r * inv + z), 0, 3);
 *     in both the product is exact (not rounded to binary32) and the value is
 *     rounded once to the nearest integer, ties to even;
 *   rhat = fl((Q - z) * s); next residual r <- fl(r - rhat);
 *   every other operation is one correctly rounded binary32 operation,
 *   nearest-even.
 *   Reconstruction after k stages: acc = rhat_0, acc = fl(acc + rhat_t) for
 *   t = 1..k-1 in stage order; binary32 output, or bfloat16 rounded to
 *   nearest-even.
 *
 * Layout. The weight matrix is row-major [rows][cols] (out x in); a group is G
 * consecutive elements of a row (along the input dimension), so groups never
 * span rows and any stack of matrices stored back to back with G | cols may be
 * passed as one call with rows = total rows. With N = rows * cols:
 *   codes  : uint32 [n_stages][N / 16]. Element e (flat row-major index) of
 *            stage k is bits 2*(e % 16) .. 2*(e % 16) + 1 of word
 *            codes[k * (N / 16) + e / 16].
 *   scales : float  [n_stages][N / G], scales[k * (N / G) + e / G].
 *   zeros  : float  [n_stages][N / G], same indexing; integer values 0..3,
 *            a zero zero-point is +0.0.
 *
 * Conventions for every call:
 *   - All buffers are device pointers (HIP device memory of the current
 *     device), allocated and owned by the caller. The library allocates
 *     nothing and keeps no pointer after it returns.
 *   - Work is enqueued on `stream` (0 = the null stream) and the call returns
 *     without waiting. Results are valid once the stream has reached that
 *     point; the caller keeps the buffers alive until then.
 *   - Arguments are checked before anything is enqueued. On an error the
 *     call returns a nonzero status and enqueues nothing. No exception ever
 *     crosses this interface.
 *   - Inputs must not overlap outputs, and outputs must not overlap each
 *     other.
 *   - The library holds no mutable state: calls may be made concurrently
 *     from several host threads (on different output buffers).
 */
#ifndef RRQ_H
#define RRQ_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every call. */
enum rrq_status {
    RRQ_OK = 0,
    RRQ_ERR_NULL = 1,   /* a required pointer is NULL */
    RRQ_ERR_ALIGN = 2,  /* a pointer is not aligned as documented */
    RRQ_ERR_SHAPE = 3,  /* rows or cols < 1, cols % group_size != 0, or rows*cols overflows */
    RRQ_ERR_GROUP = 4,  /* group_size not in {32, 64, 128} */
    RRQ_ERR_STAGES = 5, /* n_stages not in 1..RRQ_MAX_STAGES, or k_stages not in 1..n_stages */
    RRQ_ERR_DTYPE = 6,  /* out_dtype not one of enum rrq_dtype */
    RRQ_ERR_HIP = 7,    /* the HIP runtime reported an error while launching */
    RRQ_ERR_FORMAT = 8  /* zero_point or scale_type not one of the enums below */
};

/* Output element type of rrq_reconstruct. */
enum rrq_dtype {
    RRQ_F32 = 0,  /* IEEE binary32 */
    RRQ_BF16 = 1  /* bfloat16 bit patterns (uint16), rounded to nearest-even */
};

#define RRQ_MAX_STAGES 4

/*
 * Stage formats (the *_format calls). The paper's main configuration stores
 * 2-bit codes with per-group scales and zero-points (Eq. 1-3); its symmetric
 * configuration stores no zero-points and its package-size estimate assumes a
 * 16-bit scale per group (Sec. 4.1, Eq. 21, Table 14). Every stage of a
 * package has the same format. The calls without _format use
 * RRQ_ZP_INTEGER and RRQ_SCALE_F32, the arithmetic stated above.
 *
 * Zero-point kind:
 *   RRQ_ZP_INTEGER    z = RNE(|lo| inv) of the exact product, stored as float
 *                     (the default).
 *   RRQ_ZP_REAL       z = fl(|lo| inv) is kept real and stored; the code is
 *                     Q = clamp(RNE(fl(fl(r inv) + z)), 0, 3) (the sum is
 *                     rounded to binary32 first); dequantized values are
 *                     fl(fl(Q - z) s). The group's min and max land exactly
 *                     on codes 0 and 3.
 *   RRQ_ZP_SYMMETRIC  the range is widened to [-amax, amax], amax =
 *                     max(|lo|, hi), so s = fl(fl(2 amax) / 3), and z = 2
 *                     for every group (grid {-2s, -s, 0, s}); no zero-points
 *                     are stored (zeros may be NULL). A degenerate group gets
 *                     code 2 (value 0).
 * Scale storage:
 *   RRQ_SCALE_F32     float per group and stage (the default).
 *   RRQ_SCALE_F16     IEEE binary16 bit patterns (uint16_t), nearest-even.
 *   RRQ_SCALE_BF16    bfloat16 bit patterns (uint16_t), nearest-even.
 *   With a 16-bit type the scale fl(d / 3) is rounded to it first and the
 *   rounded value is the one that quantizes, dequantizes and is stored (a
 *   value that overflows the type is outside the precondition). A scale
 *   buffer then holds n_stages * rows*cols/G uint16_t, 2-byte aligned.
 */
enum rrq_zero_point {
    RRQ_ZP_INTEGER = 0,
    RRQ_ZP_REAL = 1,
    RRQ_ZP_SYMMETRIC = 2
};

enum rrq_scale_type {
    RRQ_SCALE_F32 = 0,
    RRQ_SCALE_F16 = 1,
    RRQ_SCALE_BF16 = 2
};

/*
 * rrq_construct - build the RRQ package of a bfloat16 weight matrix
 * (Algorithm 1 without a base checkpoint; Eq. 1-7; Sec. 4.1 configuration).
 *
 *   W          device, const uint16_t [rows][cols]: bfloat16 bit patterns.
 *              16-byte aligned. Precondition: every value is finite and every
 *              group's range hi - lo is finite in binary32, which holds whenever
 *              all |W| < 2^127. Inputs outside it (NaN, Inf, or a group holding
 *              values near +-3.4e38 of both signs) give unspecified codes,
 *              scales and zeros; the call still completes and touches no
 *              memory outside the documented buffers.
 *   rows, cols matrix shape; cols % group_size == 0.
 *   group_size G in {32, 64, 128}.
 *   n_stages   S in 1..4: the base stage plus S-1 residual stages (2S bits).
 *   codes      device, uint32 [S][rows*cols/16], 16-byte aligned (written).
 *   scales     device, float  [S][rows*cols/G], 4-byte aligned (written).
 *   zeros      device, float  [S][rows*cols/G], 4-byte aligned (written).
 *   stream     HIP stream the work is enqueued on.
 *
 * Returns RRQ_OK, or RRQ_ERR_NULL / _ALIGN / _SHAPE / _GROUP / _STAGES with
 * nothing enqueued, or RRQ_ERR_HIP if the kernel launch failed.
 */
int rrq_construct(const uint16_t *W, int64_t rows, int64_t cols, int32_t group_size,
                  int32_t n_stages, uint32_t *codes, float *scales, float *zeros,
                  hipStream_t stream);

/*
 * rrq_tensor - one weight tensor of rrq_construct_many: its bfloat16 input
 * and the device buffers of its own package, all as for rrq_construct.
 */
typedef struct rrq_tensor {
    const uint16_t *W;  /* device, [rows][cols] bfloat16 bit patterns, 16-byte aligned */
    uint32_t *codes;    /* device, uint32 [S][rows*cols/16], 16-byte aligned (written) */
    float *scales;      /* device, float [S][rows*cols/G], 4-byte aligned (written) */
    float *zeros;       /* device, float [S][rows*cols/G], 4-byte aligned (written) */
    int64_t rows, cols; /* shape, cols % G == 0 */
} rrq_tensor;

/*
 * rrq_construct_many - rrq_construct of several weight tensors, each into its
 * own package (Algorithm 1 without a base checkpoint, per tensor; the same
 * arithmetic, so every package is bit-identical to rrq_construct's of that
 * tensor). For a checkpoint stored tensor by tensor: the tensors' groups
 * share the GPU in one pass (one launch per 64 tensors) instead of one launch
 * each, whose start and end would otherwise leave most of the GPU idle on
 * small tensors.
 *
 *   tensors    host array of n_tensors descriptors (read during the call
 *              only); every descriptor as rrq_construct's arguments. The
 *              packages must not overlap each other or any W.
 *   n_tensors  >= 0 (0 enqueues nothing).
 *   group_size, n_stages  as rrq_construct, for every tensor.
 *   stream     HIP stream the work is enqueued on.
 *
 * Every descriptor is checked before anything is enqueued. Returns RRQ_OK,
 * RRQ_ERR_NULL (tensors NULL with n_tensors > 0, or a NULL buffer),
 * RRQ_ERR_ALIGN, RRQ_ERR_SHAPE (a bad shape, or n_tensors < 0), RRQ_ERR_GROUP,
 * RRQ_ERR_STAGES with nothing enqueued, or RRQ_ERR_HIP if a launch failed
 * (launches before it stay enqueued).
 */
int rrq_construct_many(const rrq_tensor *tensors, int32_t n_tensors, int32_t group_size,
                       int32_t n_stages, hipStream_t stream);

/*
 * rrq_construct_format - rrq_construct in a stage format (see enum
 * rrq_zero_point, enum rrq_scale_type). scales is float or uint16_t per group
 * and stage (4- or 2-byte aligned); zeros is written unless zero_point is
 * RRQ_ZP_SYMMETRIC (then it may be NULL). Returns as rrq_construct, or
 * RRQ_ERR_FORMAT for an unknown zero_point or scale_type.
 */
int rrq_construct_format(const uint16_t *W, int64_t rows, int64_t cols, int32_t group_size,
                         int32_t n_stages, int32_t zero_point, int32_t scale_type,
                         uint32_t *codes, void *scales, float *zeros, hipStream_t stream);

/*
 * rrq_construct_stats - rrq_construct_format plus the paper's outlier
 * diagnostic (Sec. 3) as a side output of the same pass: the Peak-to-Mean
 * Ratio of every group of W, its largest |w| over its mean |w|.
 *
 *   pmr    device, float [rows*cols/G], 4-byte aligned (written); required.
 *   other arguments as rrq_construct_format.
 *
 * Arithmetic (fixed; the paper states the ratio in real terms): K = max |w|;
 * S = fl(fl(p0 + p1) + fl(p2 + p3)) with p_i the binary32 sum, in index
 * order, of |w_j| over the group's elements j = i (mod 4); MAE = fl(S / G);
 * PMR = fl(K / MAE); a group of zeros gives 0. The tensor-level indicators of
 * the paper are the largest PMR over a tensor's groups and the mean / maximum
 * of that over tensors.
 */
int rrq_construct_stats(const uint16_t *W, int64_t rows, int64_t cols, int32_t group_size,
                        int32_t n_stages, int32_t zero_point, int32_t scale_type, uint32_t *codes,
                        void *scales, float *zeros, float *pmr, hipStream_t stream);

/*
 * rrq_group_pmr - the per-group Peak-to-Mean Ratio of W only (as in
 * rrq_construct_stats, without building a package): W as rrq_construct, pmr
 * device float [rows*cols/G] (written).
 */
int rrq_group_pmr(const uint16_t *W, int64_t rows, int64_t cols, int32_t group_size, float *pmr,
                  hipStream_t stream);

/*
 * rrq_construct_from_base - build the residual stages of an RRQ package on
 * an existing base checkpoint (Algorithm 1's first branch: the base stage's
 * codes, scales and zero-points are loaded, not computed; Eq. 4-7; the paper
 * presents this as the reuse of an existing low-bit checkpoint).
 *
 * On entry plane 0 of the package holds the base stage in this library's
 * layout: 2-bit codes Q_0 packed as above, and binary32 scales s_0 and
 * zero-points z_0 per group. Any finite s_0 and z_0 are accepted; z_0 need not
 * be an integer (a base from another quantizer may store a real zero-point).
 * Per element the base is dequantized as xhat_0 = fl(fl(Q_0 - z_0) * s_0)
 * (for an integer z_0 that is exactly the stage value of rrq_construct), the
 * residual R_0 = fl(W - xhat_0) is formed, and stages 1 .. n_stages - 1 are
 * the residual stages of rrq_construct applied to R_0, with the same
 * arithmetic. A base that equals rrq_construct's own stage 0 therefore
 * reproduces rrq_construct's package bit for bit.
 *
 *   W          as for rrq_construct. Precondition: every W and every
 *              R_0 = W - xhat_0 finite with a finite per-group range (holds
 *              when all |W| < 2^126 and all |xhat_0| < 2^126); otherwise the
 *              residual stages are unspecified (nothing outside the buffers
 *              is touched).
 *   rows, cols, group_size  as for rrq_construct.
 *   n_stages   S in 1..4, counting the base: planes 1 .. S-1 are written.
 *              S = 1 leaves the package as it is and enqueues nothing.
 *   codes      device, uint32 [S][rows*cols/16], 16-byte aligned: plane 0 read,
 *              planes 1 .. S-1 written.
 *   scales     device, float [S][rows*cols/G], 4-byte aligned: same planes.
 *   zeros      device, float [S][rows*cols/G], 4-byte aligned: same planes.
 *   stream     HIP stream the work is enqueued on.
 *
 * Returns RRQ_OK, or RRQ_ERR_NULL / _ALIGN / _SHAPE / _GROUP / _STAGES with
 * nothing enqueued, or RRQ_ERR_HIP if the kernel launch failed.
 */
int rrq_construct_from_base(const uint16_t *W, int64_t rows, int64_t cols, int32_t group_size,
                            int32_t n_stages, uint32_t *codes, float *scales, float *zeros,
                            hipStream_t stream);

/*
 * rrq_construct_from_base_format - rrq_construct_from_base in a stage format:
 * the base plane is read in that format (a 16-bit scale widened exactly; for
 * RRQ_ZP_SYMMETRIC z_0 = 2 and zeros may be NULL) and the residual stages
 * are built in it.
 */
int rrq_construct_from_base_format(const uint16_t *W, int64_t rows, int64_t cols,
                                   int32_t group_size, int32_t n_stages, int32_t zero_point,
                                   int32_t scale_type, uint32_t *codes, void *scales,
                                   float *zeros, hipStream_t stream);

/*
 * rrq_reconstruct - effective weight of the first k_stages stages of a
 * package (Eq. 8, Eq. 18-19): sum of the dequantized stages (Q - z) s,
 * binary32, in stage order (2 k_stages effective bits).
 *
 *   codes, scales, zeros  device, a package as written by rrq_construct for
 *              the same rows, cols, group_size and n_stages (read only; codes
 *              16-byte aligned, scales/zeros 4-byte aligned).
 *   rows, cols, group_size, n_stages  the package's shape (they define the
 *              per-stage plane strides); same rules as rrq_construct.
 *   k_stages   1..n_stages.
 *   W_out      device, [rows][cols] of out_dtype, 16-byte aligned (written).
 *   out_dtype  RRQ_F32 or RRQ_BF16.
 *   stream     HIP stream the work is enqueued on.
 *
 * Returns RRQ_OK, or an argument error with nothing enqueued, or RRQ_ERR_HIP.
 */
int rrq_reconstruct(const uint32_t *codes, const float *scales, const float *zeros,
                    int64_t rows, int64_t cols, int32_t group_size, int32_t n_stages,
                    int32_t k_stages, void *W_out, int32_t out_dtype, hipStream_t stream);

/*
 * rrq_reconstruct_format - rrq_reconstruct of a package in a stage format:
 * rhat = fl(fl(Q - z) s) with s the widened stored scale and z = 2 for
 * symmetric stages (zeros may then be NULL).
 */
int rrq_reconstruct_format(const uint32_t *codes, const void *scales, const float *zeros,
                           int64_t rows, int64_t cols, int32_t group_size, int32_t n_stages,
                           int32_t zero_point, int32_t scale_type, int32_t k_stages, void *W_out,
                           int32_t out_dtype, hipStream_t stream);

/*
 * rrq_linear - a linear layer on the prefix-k weight of a package, by the
 * stage decomposition of the prefill / decode product (Eq. 20; the prefix
 * weight of Eq. 19):
 *     Y[m][o] = sum_{t < k} sum_i X[m][i] (Q_t[o][i] - z_t) s_t ,
 * i.e. Y = X W~_(k)^T for the row-major [rows][cols] (out x in) weight, the
 * nn.Linear convention. The product is formed per group and stage as
 * s_t (sum_i X Q_t - z_t sum_i X) on the matrix cores.
 *
 *   codes, scales, zeros  device, a package (as rrq_reconstruct reads it).
 *   rows, cols, group_size, n_stages  the package's shape; same rules as
 *              rrq_construct, and rows, cols < 2^26, k_stages * rows * cols
 *              / 4 < 2^32 (the code planes read span less than 4 GiB).
 *   k_stages   1..n_stages (2 k_stages effective bits).
 *   X          device, bfloat16 bit patterns [n_tokens][cols], 16-byte
 *              aligned (read only).
 *   n_tokens   >= 1; the package is read once for up to 16 tokens (the
 *              decode form streams it for up to 4 tokens, and for 5 to 16
 *              on small packages of rows of 4096 inputs; the batch form for 5
 *              to 16 on packages of 3072 to 12288 rows or more of 2048 to
 *              4096 inputs, by stage and token count), more tokens 16
 *              per pass; from 128 tokens (groups of 128) tiles of 64 or
 *              128 tokens run as a matrix-core product with the 16-token
 *              tiles' accumulation order (the same results).
 *   Y          device, float [n_tokens][rows], 4-byte aligned (written).
 *   stream     HIP stream the work is enqueued on.
 *
 * Arithmetic: every product X * (4 + Q), X * 1 is exact in the matrix
 * cores; fp32 rounding enters in the accumulations only, in an order fixed
 * by rows, cols, group_size, k_stages and n_tokens (results are
 * deterministic; the same token may round differently in calls with another
 * n_tokens). With u = 2^-24, A = sum_{t, g} |s_t,g|
 * (11 + |z_t,g|) sum_{i in g} |X[m][i]|, p = groups per row and
 * n = k_stages * (min(p, 4 ceil(p / 16)) + 1),
 * |Y[m][o] - exact| <= 1.05 u A (group_size + 2 n + 24).
 *
 * Returns RRQ_OK, or RRQ_ERR_NULL / _ALIGN / _SHAPE / _GROUP / _STAGES with
 * nothing enqueued, or RRQ_ERR_HIP if the kernel launch failed.
 */
int rrq_linear(const uint32_t *codes, const float *scales, const float *zeros, int64_t rows,
               int64_t cols, int32_t group_size, int32_t n_stages, int32_t k_stages,
               const uint16_t *X, int64_t n_tokens, float *Y, hipStream_t stream);

/*
 * rrq_linear_format - rrq_linear on a package in a stage format (the exact
 * value uses the widened stored scales and z = 2 for symmetric stages; the
 * same error bound holds).
 */
int rrq_linear_format(const uint32_t *codes, const void *scales, const float *zeros,
                      int64_t rows, int64_t cols, int32_t group_size, int32_t n_stages,
                      int32_t zero_point, int32_t scale_type, int32_t k_stages,
                      const uint16_t *X, int64_t n_tokens, float *Y, hipStream_t stream);

/*
 * rrq_package_bytes - sizes the caller allocates for a package (host only,
 * no device work): codes_bytes = n_stages * rows*cols/4 and scales_bytes =
 * n_stages * (rows*cols/group_size) * 4; the zeros buffer has scales_bytes
 * too. Either output pointer may be NULL. Returns RRQ_OK or an argument
 * error (_SHAPE, _GROUP, _STAGES).
 */
int rrq_package_bytes(int64_t rows, int64_t cols, int32_t group_size, int32_t n_stages,
                      size_t *codes_bytes, size_t *scales_bytes);

/* rrq_status_string - static, NUL-terminated description of a status code. */
const char *rrq_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* RRQ_H */

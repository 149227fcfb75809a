/*
 * Plain scalar CPU oracle for RRQ construction and prefix reconstruction.
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library. It shares no source, header
 * or table with the HIP library, and the HIP library never calls it.
 *
 * It computes, group by group and element by element, the same fixed reading
 * of the paper as the numpy oracle (oracle/rrq_oracle.py), written a second
 * time as straight C so that large inputs finish in seconds:
 *   Eq. 1-3   per-group affine quantizer and its residual;
 *   Eq. 4-7   base stage on the weights, each later stage on the residual;
 *   Alg. 1    quantize / store / dequantize / subtract, without a base
 *             checkpoint and (second entry point) on a given base stage;
 *   Eq. 8     prefix reconstruction, also Eq. 18-19;
 *   Sec. 4.1  2-bit RTN stages, group size 128 (32 and 64 also accepted).
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off (no fast-math): every float
 * operation below is one IEEE binary32 operation rounded to nearest-even,
 * with no fused multiply-add.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_ERR_ARGS 1
#define ORACLE_ERR_NONFINITE 2
#define ORACLE_ERR_RANGE 3

static float bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Nearest bfloat16, ties to even (finite inputs). */
static uint16_t f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    uint32_t trunc = u >> 16;
    uint32_t rest = u & 0xFFFFu;
    if (rest > 0x8000u || (rest == 0x8000u && (trunc & 1u)))
        trunc += 1u;
    return (uint16_t)trunc;
}

/* Stage formats (zero-point kind, scale storage type). */
#define ZP_INT 0   /* z = RNE(fl(-lo inv)), integer */
#define ZP_REAL 1  /* z = fl(-lo inv), kept real */
#define ZP_SYM 2   /* symmetric: range [-amax, amax], z = 2^(bits-1), not stored */
#define SC_F32 0
#define SC_F16 1
#define SC_BF16 2

/* Nearest IEEE binary16, ties to even (finite input; overflow gives inf). */
static uint16_t f32_to_f16(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    const uint32_t sign = (u >> 16) & 0x8000u;
    const uint32_t a = u & 0x7FFFFFFFu;
    if (a >= 0x477FF000u) return (uint16_t)(sign | 0x7C00u);     /* >= 65520: inf */
    if (a <= 0x33000000u) return (uint16_t)sign;                 /* <= 2^-25: zero */
    const uint32_t e = a >> 23;
    const uint32_t m = (a & 0x7FFFFFu) | 0x800000u;
    if (e < 113) {                                                /* below 2^-14: subnormal */
        const uint32_t shift = 126 - e;                           /* 14 .. 24 */
        uint32_t q = m >> shift;
        const uint32_t rem = m & ((1u << shift) - 1u), half = 1u << (shift - 1);
        if (rem > half || (rem == half && (q & 1u))) q += 1u;
        return (uint16_t)(sign | q);
    }
    uint32_t q = ((e - 112) << 10) | ((a & 0x7FFFFFu) >> 13);
    const uint32_t rem = a & 0x1FFFu;
    if (rem > 0x1000u || (rem == 0x1000u && (q & 1u))) q += 1u;
    return (uint16_t)(sign | q);
}

static float f16_to_f32(uint16_t h)
{
    const uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
    const uint32_t e = (h >> 10) & 0x1Fu, m = h & 0x3FFu;
    float v;
    if (e == 0) v = (float)m * 0x1p-24f;
    else if (e == 31) v = m ? NAN : INFINITY;
    else v = ldexpf((float)(m | 0x400u), (int)e - 25);
    uint32_t u;
    memcpy(&u, &v, sizeof u);
    u |= sign;
    memcpy(&v, &u, sizeof v);
    return v;
}

/* The binary32 value of a scale stored in format sdt. */
static float round_scale(float s, int sdt)
{
    if (sdt == SC_F16) return f16_to_f32(f32_to_f16(s));
    if (sdt == SC_BF16) return bf16_to_f32(f32_to_bf16(s));
    return s;
}

/*
 * One min-max RTN stage of one group (Eq. 1-3) with 2^bits - 1 steps, in
 * stage format (zp, sdt): writes the codes Q[0..G), the scale (its binary32
 * value) and the zero-point, and replaces r[j] by r[j] - rhat[j] when
 * update_residual is set.
 */
static int rtn_stage_group(float *r, int G, int bits, int update_residual, int zp, int sdt,
                           uint8_t *Q, float *s_out, float *z_out)
{
    const int maxq = (1 << bits) - 1;
    const float zsym = (float)(1 << (bits - 1));
    float lo = 0.0f, hi = 0.0f;           /* zero is always in the range */
    for (int j = 0; j < G; ++j) {
        if (r[j] < lo) lo = r[j];
        if (r[j] > hi) hi = r[j];
    }
    if (zp == ZP_SYM) {                   /* symmetric range */
        const float amax = (0.0f - lo) > hi ? (0.0f - lo) : hi;
        lo = 0.0f - amax;
        hi = amax;
    }
    float d = hi - lo;
    if (!isfinite(d)) return ORACLE_ERR_RANGE;   /* precondition: finite range */
    float s = round_scale(d / (float)maxq, sdt); /* the stored scale is used */
    if (!isfinite(s)) return ORACLE_ERR_RANGE;
    if (!(s >= 0x1p-126f)) {              /* zero or subnormal: degenerate */
        const uint8_t qd = zp == ZP_SYM ? (uint8_t)zsym : 0;
        for (int j = 0; j < G; ++j) Q[j] = qd;
        *s_out = 0.0f;
        *z_out = zp == ZP_SYM ? zsym : 0.0f;
        return ORACLE_OK;                  /* residual unchanged */
    }
    float inv = 1.0f / s;
    float z;
    /* integer zero-point: RNE of the exact |lo| inv (exact in double); +0 */
    if (zp == ZP_INT) z = (float)rint((double)(0.0f - lo) * (double)inv) + 0.0f;
    else if (zp == ZP_REAL) z = (0.0f - lo) * inv + 0.0f;
    else z = zsym;
    for (int j = 0; j < G; ++j) {
        double q;
        if (zp == ZP_REAL) {
            float t = r[j] * inv;
            q = (double)rintf(t + z);      /* RNE of the rounded sum */
        } else {
            /* r inv + z with the product unrounded: exact in double wherever
             * its rounding to an integer is decided; rint ties to even. */
            q = rint((double)r[j] * (double)inv + (double)z);
        }
        if (q < 0.0) q = 0.0;
        if (q > (double)maxq) q = (double)maxq;
        Q[j] = (uint8_t)q;
        if (update_residual) {
            float qz = (float)Q[j] - z;    /* exact for an integer z */
            float rhat = qz * s;
            r[j] = r[j] - rhat;
        }
    }
    *s_out = s;
    *z_out = z;
    return ORACLE_OK;
}

/*
 * Construct the RRQ package of n binary32-widened bfloat16 weights W (flat,
 * row-major; groups are G consecutive elements). Outputs, all owned by the
 * caller: codes [S][n/16] uint32 (element e -> word e/16, bits 2(e%16)),
 * scales [S][n/G], zeros [S][n/G].
 */
int rrq_oracle_construct(const uint16_t *W, int64_t n, int32_t G, int32_t S,
                         uint32_t *codes, float *scales, float *zeros)
{
    if (!W || !codes || !scales || !zeros) return ORACLE_ERR_ARGS;
    if (G <= 0 || G > 1024 || G % 16 != 0 || n <= 0 || n % G != 0) return ORACLE_ERR_ARGS;
    if (S < 1 || S > 8) return ORACLE_ERR_ARGS;
    const int64_t n_groups = n / G;
    const int64_t words = n / 16;
    int bad = 0, bad_range = 0;

#pragma omp parallel for schedule(static) reduction(| : bad, bad_range)
    for (int64_t g = 0; g < n_groups; ++g) {
        float r[1024];
        uint8_t Q[1024];
        for (int j = 0; j < G; ++j) {
            r[j] = bf16_to_f32(W[g * G + j]);
            if (!isfinite(r[j])) bad = 1;
        }
        for (int k = 0; k < S; ++k) {
            float s = 0.0f, z = 0.0f;
            if (rtn_stage_group(r, G, 2, k + 1 < S, ZP_INT, SC_F32, Q, &s, &z) != ORACLE_OK)
                bad_range = 1;
            scales[(int64_t)k * n_groups + g] = s;
            zeros[(int64_t)k * n_groups + g] = z;
            for (int w = 0; w < G / 16; ++w) {
                uint32_t word = 0;
                for (int e = 0; e < 16; ++e)
                    word |= (uint32_t)Q[w * 16 + e] << (2 * e);
                codes[(int64_t)k * words + g * (G / 16) + w] = word;
            }
        }
    }
    return bad ? ORACLE_ERR_NONFINITE : bad_range ? ORACLE_ERR_RANGE : ORACLE_OK;
}

/*
 * Algorithm 1 with a base checkpoint: plane 0 of codes / scales / zeros holds
 * the base stage on entry (read only; any finite scale and zero-point, the
 * zero-point not necessarily an integer). Each group's base is dequantized,
 * xhat = fl(fl(Q - z) * s), the residual r = fl(W - xhat) is formed, and
 * planes 1 .. S-1 receive the residual stages exactly as in
 * rrq_oracle_construct.
 */
int rrq_oracle_construct_from_base(const uint16_t *W, int64_t n, int32_t G, int32_t S,
                                   uint32_t *codes, float *scales, float *zeros)
{
    if (!W || !codes || !scales || !zeros) return ORACLE_ERR_ARGS;
    if (G <= 0 || G > 1024 || G % 16 != 0 || n <= 0 || n % G != 0) return ORACLE_ERR_ARGS;
    if (S < 1 || S > 8) return ORACLE_ERR_ARGS;
    const int64_t n_groups = n / G;
    const int64_t words = n / 16;
    int bad = 0, bad_range = 0;

#pragma omp parallel for schedule(static) reduction(| : bad, bad_range)
    for (int64_t g = 0; g < n_groups; ++g) {
        float r[1024];
        uint8_t Q[1024];
        const float s0 = scales[g], z0 = zeros[g];
        for (int j = 0; j < G; ++j) {
            const float w = bf16_to_f32(W[g * G + j]);
            if (!isfinite(w)) bad = 1;
            const uint32_t word = codes[g * (G / 16) + j / 16];
            const float q0 = (float)((word >> (2 * (j % 16))) & 3u);
            const float base = (q0 - z0) * s0;     /* two roundings, no FMA */
            r[j] = w - base;
            if (!isfinite(r[j])) bad = 1;
        }
        for (int k = 1; k < S; ++k) {
            float s = 0.0f, z = 0.0f;
            if (rtn_stage_group(r, G, 2, k + 1 < S, ZP_INT, SC_F32, Q, &s, &z) != ORACLE_OK)
                bad_range = 1;
            scales[(int64_t)k * n_groups + g] = s;
            zeros[(int64_t)k * n_groups + g] = z;
            for (int w = 0; w < G / 16; ++w) {
                uint32_t word = 0;
                for (int e = 0; e < 16; ++e)
                    word |= (uint32_t)Q[w * 16 + e] << (2 * e);
                codes[(int64_t)k * words + g * (G / 16) + w] = word;
            }
        }
    }
    return bad ? ORACLE_ERR_NONFINITE : bad_range ? ORACLE_ERR_RANGE : ORACLE_OK;
}

/*
 * Construction in a stage format: zp in {0 integer zero-point, 1 real
 * zero-point, 2 symmetric}, sdt in {0 binary32, 1 binary16, 2 bfloat16
 * scales}. scales points to float [S][n/G] or uint16_t [S][n/G] (16-bit
 * patterns); zeros is float [S][n/G] and receives the zero-points (for
 * symmetric stages the implicit 2, which a package does not store).
 */
int rrq_oracle_construct_format(const uint16_t *W, int64_t n, int32_t G, int32_t S, int32_t zp,
                                int32_t sdt, uint32_t *codes, void *scales, float *zeros)
{
    if (!W || !codes || !scales || !zeros) return ORACLE_ERR_ARGS;
    if (G <= 0 || G > 1024 || G % 16 != 0 || n <= 0 || n % G != 0) return ORACLE_ERR_ARGS;
    if (S < 1 || S > 8 || zp < 0 || zp > 2 || sdt < 0 || sdt > 2) return ORACLE_ERR_ARGS;
    const int64_t n_groups = n / G;
    const int64_t words = n / 16;
    int bad = 0, bad_range = 0;

#pragma omp parallel for schedule(static) reduction(| : bad, bad_range)
    for (int64_t g = 0; g < n_groups; ++g) {
        float r[1024];
        uint8_t Q[1024];
        for (int j = 0; j < G; ++j) {
            r[j] = bf16_to_f32(W[g * G + j]);
            if (!isfinite(r[j])) bad = 1;
        }
        for (int k = 0; k < S; ++k) {
            float s = 0.0f, z = 0.0f;
            if (rtn_stage_group(r, G, 2, k + 1 < S, zp, sdt, Q, &s, &z) != ORACLE_OK)
                bad_range = 1;
            const int64_t gi = (int64_t)k * n_groups + g;
            if (sdt == SC_F32) ((float *)scales)[gi] = s;
            else if (sdt == SC_F16) ((uint16_t *)scales)[gi] = f32_to_f16(s);
            else ((uint16_t *)scales)[gi] = f32_to_bf16(s);
            zeros[gi] = z;
            for (int w = 0; w < G / 16; ++w) {
                uint32_t word = 0;
                for (int e = 0; e < 16; ++e)
                    word |= (uint32_t)Q[w * 16 + e] << (2 * e);
                codes[(int64_t)k * words + g * (G / 16) + w] = word;
            }
        }
    }
    return bad ? ORACLE_ERR_NONFINITE : bad_range ? ORACLE_ERR_RANGE : ORACLE_OK;
}

/* Prefix-k reconstruction of a package in a stage format (as above; zeros
 * is not read for symmetric stages). */
int rrq_oracle_reconstruct_format(const uint32_t *codes, const void *scales, const float *zeros,
                                  int64_t n, int32_t G, int32_t S, int32_t zp, int32_t sdt,
                                  int32_t k, int32_t out_bf16, void *out)
{
    if (!codes || !scales || !out || (zp != ZP_SYM && !zeros)) return ORACLE_ERR_ARGS;
    if (G <= 0 || G % 16 != 0 || n <= 0 || n % G != 0) return ORACLE_ERR_ARGS;
    if (S < 1 || k < 1 || k > S || zp < 0 || zp > 2 || sdt < 0 || sdt > 2) return ORACLE_ERR_ARGS;
    const int64_t n_groups = n / G;
    const int64_t words = n / 16;

#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n; ++e) {
        const int64_t g = e / G;
        float acc = 0.0f;
        for (int t = 0; t < k; ++t) {
            const int64_t gi = (int64_t)t * n_groups + g;
            uint32_t word = codes[(int64_t)t * words + e / 16];
            uint32_t q = (word >> (2 * (e % 16))) & 3u;
            float sc = sdt == SC_F32 ? ((const float *)scales)[gi]
                     : sdt == SC_F16 ? f16_to_f32(((const uint16_t *)scales)[gi])
                                     : bf16_to_f32(((const uint16_t *)scales)[gi]);
            float z = zp == ZP_SYM ? 2.0f : zeros[gi];
            float qz = (float)q - z;
            float rhat = qz * sc;
            acc = (t == 0) ? rhat : acc + rhat;
        }
        if (out_bf16)
            ((uint16_t *)out)[e] = f32_to_bf16(acc);
        else
            ((float *)out)[e] = acc;
    }
    return ORACLE_OK;
}

/*
 * Peak-to-Mean Ratio of every group of n bfloat16 weights (Sec. 3): K / MAE,
 * K = max |w|, MAE = fl(S / G) with S accumulated as four partial sums over
 * j = 0, 1, 2, 3 (mod 4), each in increasing j, combined as
 * fl(fl(p0 + p1) + fl(p2 + p3)); a group of zeros gives 0.
 */
int rrq_oracle_group_pmr(const uint16_t *W, int64_t n, int32_t G, float *pmr)
{
    if (!W || !pmr || G <= 0 || G % 4 != 0 || n <= 0 || n % G != 0) return ORACLE_ERR_ARGS;
    const int64_t n_groups = n / G;
#pragma omp parallel for schedule(static)
    for (int64_t g = 0; g < n_groups; ++g) {
        float p[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        float K = 0.0f;
        for (int j = 0; j < G; ++j) {
            const float a = fabsf(bf16_to_f32(W[g * G + j]));
            p[j % 4] = p[j % 4] + a;
            if (a > K) K = a;
        }
        const float S = (p[0] + p[1]) + (p[2] + p[3]);
        const float mae = S / (float)G;
        pmr[g] = S > 0.0f ? K / mae : 0.0f;
    }
    return ORACLE_OK;
}

/* Conversion helpers exported for the pins: binary32 -> binary16 bits. */
void rrq_oracle_f32_to_f16(const float *x, int64_t n, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = f32_to_f16(x[i]);
}

/*
 * Prefix-k reconstruction: out[e] = rhat_0[e] + rhat_1[e] + ... summed left
 * to right in binary32, with rhat_t = (Q_t - z_t) s_t. out_bf16 selects a
 * bfloat16 output (uint16 bit patterns, nearest-even) instead of binary32.
 */
int rrq_oracle_reconstruct(const uint32_t *codes, const float *scales,
                           const float *zeros, int64_t n, int32_t G, int32_t S,
                           int32_t k, int32_t out_bf16, void *out)
{
    if (!codes || !scales || !zeros || !out) return ORACLE_ERR_ARGS;
    if (G <= 0 || G % 16 != 0 || n <= 0 || n % G != 0) return ORACLE_ERR_ARGS;
    if (S < 1 || k < 1 || k > S) return ORACLE_ERR_ARGS;
    const int64_t n_groups = n / G;
    const int64_t words = n / 16;

#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n; ++e) {
        const int64_t g = e / G;
        float acc = 0.0f;
        for (int t = 0; t < k; ++t) {
            uint32_t word = codes[(int64_t)t * words + e / 16];
            uint32_t q = (word >> (2 * (e % 16))) & 3u;
            float qz = (float)q - zeros[(int64_t)t * n_groups + g];
            float rhat = qz * scales[(int64_t)t * n_groups + g];
            acc = (t == 0) ? rhat : acc + rhat;
        }
        if (out_bf16)
            ((uint16_t *)out)[e] = f32_to_bf16(acc);
        else
            ((float *)out)[e] = acc;
    }
    return ORACLE_OK;
}

/* Sets the number of OpenMP threads for later calls (n >= 1). */
void rrq_oracle_set_threads(int n)
{
    if (n >= 1) omp_set_num_threads(n);
}

/* Number of OpenMP threads a parallel region of this library uses. */
int rrq_oracle_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        n = omp_get_num_threads();
    }
    return n;
}

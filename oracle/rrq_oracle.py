"""Plain CPU oracle for Recurrent Residual Quantization (RRQ) construction and
prefix reconstruction.

TEST INFRASTRUCTURE. Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this module. The product path (the HIP library and
its Python binding) never imports, links or calls anything under ``oracle/``.

What it computes (paper, Sec. 3 "Recurrent Residual Quantization"):

* the per-group affine quantizer of Eq. 1-3: q = x/s + z, Q = R(q),
  residual r = x - (Q - z) s;
* the recursion of Eq. 4-7: a base stage on the weights, then each further
  stage quantizes the residual the stages before it left behind;
* Algorithm 1 without a base checkpoint: quantize, store codes / scales /
  zero-points, dequantize, subtract, repeated for every stage;
* Algorithm 1 with a base checkpoint: the base's codes, scales and zero-points
  are loaded and dequantized (a real-valued zero-point allowed), and only the
  residual stages are computed;
* the prefix reconstruction of Eq. 8 (restated as Eq. 18-19 in the
  prefill/decode appendix): the effective weight after t stages is the sum of
  the first t dequantized stages;
* the peak-to-mean ratio of Sec. 3 (``group_pmr``), the outlier diagnostic;
* the stage-sum product of Eq. 20: a linear layer on the prefix-t weight is the
  sum of the products of the activations with each stage (``linear``,
  evaluated in float64);
* the main configuration of Sec. 4.1: 2-bit RTN stages, 4 of them, group size
  128, calibration-free.

The paper leaves the floating-point details open; this oracle fixes them
(readings listed in the design notes, each one also stated at its step below):

* groups are G contiguous elements of the row-major (out x in) matrix, along
  the input dimension;
* residuals are carried in IEEE binary32 between stages;
* range: lo = min(+0, min r), hi = max(+0, max r) (zero is always on the grid);
* scale: s = fl(fl(hi - lo) / (2^b - 1)); a group whose s is zero or subnormal
  is degenerate: s = z = 0, all codes 0, residual passed through unchanged;
* inv = fl(1 / s); zero-point z = RNE((0 - lo) * inv) of the exact product,
  an integer stored as binary32;
* code: Q = clamp(RNE(r * inv + z), 0, 2^b - 1) of the exact value (the
  product is not rounded), ties to even;
* dequantized stage value rhat = fl((Q - z) * s); next residual
  r <- fl(r - rhat);
* reconstruction after k stages: acc = rhat_0, then acc = fl(acc + rhat_t) for
  t = 1 .. k-1 in stage order; output binary32, or bfloat16 rounded to
  nearest-even;
* codes are stored stage-planar, 16 two-bit codes per little-endian uint32,
  element e of the flat matrix in word e // 16 at bits 2 (e % 16) .. +1.

Inputs must be finite bfloat16 values whose per-group range hi - lo is finite
in binary32 (always so when every |x| < 2^127); the oracle raises otherwise.

Every step below is a separate numpy float32 operation (one IEEE rounding per
operation, no fused multiply-add). Where a step needs an exact value (r * inv
+ z, |lo| * inv), it is formed in float64, where it is exact; see
``_exact_round_sum``.
"""

from __future__ import annotations

import numpy as np

F32 = np.float32
SMALLEST_NORMAL_F32 = F32(2.0 ** -126)


# ---------------------------------------------------------------------------
# bfloat16 <-> binary32
# ---------------------------------------------------------------------------

def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to binary32 exactly: a bfloat16 is
    the upper half of the binary32 with the same value."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round binary32 values to the nearest bfloat16, ties to even.

    Written from the definition: the two bfloat16 neighbours of x are the
    truncation of x to its upper 16 bits and the next bfloat16 away from zero;
    pick the nearer one and on a tie the one whose last kept bit is 0. Inputs
    here are always finite.
    """
    x = np.asarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    trunc = b >> np.uint64(16)                 # toward zero
    rest = b & np.uint64(0xFFFF)               # dropped bits
    half = np.uint64(0x8000)
    odd = trunc & np.uint64(1)
    up = (rest > half) | ((rest == half) & (odd == np.uint64(1)))
    out = trunc + up.astype(np.uint64)         # carries into the exponent correctly
    return out.astype(np.uint16)


# ---------------------------------------------------------------------------
# One RTN stage on a batch of groups (Eq. 1-3)
# ---------------------------------------------------------------------------

def _exact_round_sum(r: np.ndarray, inv: np.ndarray, z: np.ndarray) -> np.ndarray:
    """RNE(r inv + z) of the exact value, for binary32 r and inv and a small
    integer z (the product is not rounded).

    In float64 the product r inv (two 24-bit significands) is exact. When
    |r inv| >= 1/8 its lowest bit is at or above 2^-51 and |r inv + z| < 8, so
    the sum is exact too; when |r inv| < 1/8 the sum lies within 1/8 of an
    integer, so the float64 rounding cannot move it across a half-integer. In
    both cases rounding the float64 sum to an integer, ties to even, gives the
    rounding of the exact value.
    """
    return np.rint(r.astype(np.float64) * inv.astype(np.float64) + z.astype(np.float64))


ZERO_POINTS = ("int", "real", "sym")
SCALE_DTYPES = ("f32", "f16", "bf16")


def round_scale(s: np.ndarray, scale_dtype: str) -> np.ndarray:
    """The binary32 value of a stage scale stored in ``scale_dtype``: itself,
    or the nearest (ties to even) binary16 / bfloat16 value, widened back."""
    s = np.asarray(s, dtype=np.float32)
    if scale_dtype == "f32":
        return s
    if scale_dtype == "f16":
        return s.astype(np.float16).astype(np.float32)
    if scale_dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(s))
    raise ValueError(scale_dtype)


def rtn_stage(r: np.ndarray, bits: int, zero_point: str = "int", scale_dtype: str = "f32"):
    """Quantize a batch of groups once with min-max RTN.

    ``r``: float32 array [n_groups, G] (the weights for the base stage, the
    residual for later stages). Returns (Q uint8 [n_groups, G], s float32
    [n_groups], z float32 [n_groups], rhat float32 [n_groups, G]).

    Eq. 1 (q = x/s + z with a scale and zero-point shared by the group),
    Eq. 2 (Q = R(q)) and Eq. 3 (dequantized value (Q - z) s).

    ``zero_point``: "int" (the default reading: z = RNE(-lo inv) and Q =
    RNE(r inv + z), each the single rounding of the exact value); "real"
    (z = fl(-lo inv) kept real, t = fl(r inv), Q = RNE(fl(t + z))); "sym"
    (symmetric stage: the range is widened to
    [-amax, amax], amax = max(-lo, hi), and z is fixed at 2^(b-1), not
    stored; a degenerate group gets the zero code Q = z).
    ``scale_dtype``: the scale is rounded to its storage type ("f16", "bf16")
    before it is used, and the rounded value quantizes and dequantizes.
    """
    assert r.dtype == np.float32 and r.ndim == 2
    if zero_point not in ZERO_POINTS or scale_dtype not in SCALE_DTYPES:
        raise ValueError("unknown stage format")
    maxq = (1 << bits) - 1
    zero = F32(0.0)

    # Range of the group, with zero included (reading: zero on the grid).
    lo = np.minimum(r.min(axis=1), zero)
    hi = np.maximum(r.max(axis=1), zero)
    lo = np.where(lo == zero, zero, lo)        # canonical +0
    hi = np.where(hi == zero, zero, hi)
    if zero_point == "sym":
        amax = np.maximum(zero - lo, hi)       # exact
        lo, hi = zero - amax, amax

    d = hi - lo                                # fl(hi - lo)
    if not np.all(np.isfinite(d)):
        raise ValueError("RRQ oracle: a group's range overflows binary32 (inputs need |x| < 2^127)")
    s = d / F32(maxq)                          # fl(d / maxq), IEEE division
    s = round_scale(s, scale_dtype)            # the stored scale is the one used
    if not np.all(np.isfinite(s)):
        raise ValueError("RRQ oracle: a stage scale overflows its storage type")
    degenerate = s < SMALLEST_NORMAL_F32       # zero or subnormal scale

    s_safe = np.where(degenerate, F32(1.0), s)
    inv = F32(1.0) / s_safe                    # fl(1 / s)
    if zero_point == "int":
        z = np.rint((zero - lo).astype(np.float64) * inv)   # RNE(|lo| inv), product exact
    elif zero_point == "real":
        z = (zero - lo) * inv                  # fl((0 - lo) * inv)
    else:
        z = np.full(lo.shape, F32(1 << (bits - 1)))
    z_deg = F32(1 << (bits - 1)) if zero_point == "sym" else zero
    z = (np.where(degenerate, z_deg, z) + zero).astype(np.float32)   # +0, not -0
    inv = np.where(degenerate, zero, inv)
    s = np.where(degenerate, zero, s)

    if zero_point == "real":
        t = r * inv[:, None]                   # fl(r * inv)
        q = np.rint(t + z[:, None])            # RNE(fl(t + z))
    else:
        q = _exact_round_sum(r, inv[:, None], z[:, None])   # RNE(r inv + z), one rounding
    Q = np.clip(q, 0, maxq)
    Q = np.where(degenerate[:, None], z_deg, Q).astype(np.uint8)

    qz = Q.astype(np.float32) - z[:, None]     # fl(Q - z) (exact for an integer z)
    rhat = qz * s[:, None]                     # fl((Q - z) * s)
    rhat = np.where(degenerate[:, None], zero, rhat)
    return Q, s.astype(np.float32), z.astype(np.float32), rhat.astype(np.float32)


# ---------------------------------------------------------------------------
# Packing of 2-bit codes
# ---------------------------------------------------------------------------

def pack_codes(Q: np.ndarray) -> np.ndarray:
    """Pack 2-bit codes [n] (n % 16 == 0) into uint32 words: element e goes to
    word e // 16, bits 2 (e % 16) and 2 (e % 16) + 1."""
    Q = np.asarray(Q, dtype=np.uint32).reshape(-1, 16)
    assert int(Q.max(initial=0)) <= 3
    shifts = (2 * np.arange(16, dtype=np.uint32))[None, :]
    return np.bitwise_or.reduce(Q << shifts, axis=1).astype(np.uint32)


def unpack_codes(words: np.ndarray) -> np.ndarray:
    """Inverse of ``pack_codes``."""
    words = np.asarray(words, dtype=np.uint32).reshape(-1, 1)
    shifts = (2 * np.arange(16, dtype=np.uint32))[None, :]
    return ((words >> shifts) & np.uint32(3)).astype(np.uint8).reshape(-1)


# ---------------------------------------------------------------------------
# Construction (Algorithm 1, no base checkpoint; Eq. 4-7)
# ---------------------------------------------------------------------------

def _check_shape(n_elems: int, group_size: int):
    if n_elems <= 0 or n_elems % group_size != 0 or n_elems % 16 != 0:
        raise ValueError("element count must be a positive multiple of the group size and of 16")


def construct_f32(x: np.ndarray, group_size: int, n_stages: int, bits: int = 2,
                  zero_point: str = "int", scale_dtype: str = "f32"):
    """Run the RRQ recursion on binary32 weights x (flat, row-major).

    Returns per-stage codes Q [S, n] (uint8), scales [S, n/G], zeros [S, n/G],
    the dequantized stage values rhat [S, n] and the final residual [n].
    Every stage uses the stage format (zero_point, scale_dtype) of
    ``rtn_stage``; scales are returned as their binary32 values.
    """
    x = np.ascontiguousarray(x, dtype=np.float32).reshape(-1)
    _check_shape(x.size, group_size)
    if not np.all(np.isfinite(x)):
        raise ValueError("RRQ oracle: inputs must be finite")
    n_groups = x.size // group_size
    r = x.reshape(n_groups, group_size).copy()
    Qs, ss, zs, rhats = [], [], [], []
    for k in range(n_stages):
        # Stage 0 quantizes the weights (base stage), stage k >= 1 the residual
        # left by stages 0..k-1 (Eq. 4-7; Algorithm 1's loop body).
        Q, s, z, rhat = rtn_stage(r, bits, zero_point, scale_dtype)
        Qs.append(Q.reshape(-1))
        ss.append(s)
        zs.append(z)
        rhats.append(rhat.reshape(-1))
        r = r - rhat                           # R_k = R_{k-1} - Rhat_k
    return (np.stack(Qs), np.stack(ss), np.stack(zs), np.stack(rhats),
            r.reshape(-1))


def store_scales(s: np.ndarray, scale_dtype: str) -> np.ndarray:
    """Scales as stored: float32, or float16 / bfloat16 bit patterns (uint16)."""
    s = np.asarray(s, dtype=np.float32)
    if scale_dtype == "f32":
        return s
    if scale_dtype == "f16":
        return s.astype(np.float16).view(np.uint16)
    return f32_to_bf16_bits(s)


def load_scales(stored: np.ndarray, scale_dtype: str) -> np.ndarray:
    """Binary32 values of stored scales (inverse of ``store_scales``)."""
    if scale_dtype == "f32":
        return np.asarray(stored, dtype=np.float32)
    u = np.asarray(stored, dtype=np.uint16)
    if scale_dtype == "f16":
        return u.view(np.float16).astype(np.float32)
    return bf16_bits_to_f32(u)


def construct(w_bits: np.ndarray, rows: int, cols: int, group_size: int,
              n_stages: int, zero_point: str = "int", scale_dtype: str = "f32"):
    """The package of the C-ABI call rrq_construct (default format) or
    rrq_construct_format: bfloat16 weights [rows, cols] (as uint16 bit
    patterns) -> codes [S, n/16] uint32, scales [S, n/G] (float32, or uint16
    bit patterns for 16-bit scales), zeros [S, n/G] float32 (for symmetric
    stages these hold the implicit zero-point 2, which is not stored)."""
    if cols % group_size != 0:
        raise ValueError("cols must be a multiple of the group size")
    w_bits = np.ascontiguousarray(w_bits, dtype=np.uint16).reshape(-1)
    assert w_bits.size == rows * cols
    x = bf16_bits_to_f32(w_bits)
    Q, s, z, _, _ = construct_f32(x, group_size, n_stages, bits=2, zero_point=zero_point,
                                  scale_dtype=scale_dtype)
    codes = np.stack([pack_codes(Q[k]) for k in range(n_stages)])
    return codes, store_scales(s, scale_dtype), z


# ---------------------------------------------------------------------------
# Construction on an existing base checkpoint (Algorithm 1, the branch that
# loads a base; Eq. 4-7)
# ---------------------------------------------------------------------------

def construct_from_base_f32(x: np.ndarray, base_Q: np.ndarray, base_s: np.ndarray,
                            base_z: np.ndarray, group_size: int, n_stages: int,
                            bits: int = 2):
    """The RRQ recursion when a base checkpoint is given (Algorithm 1's
    first branch): the base's codes, scales and zero-points are loaded, not
    computed, and dequantized with the same affine rule as every stage
    (Eq. 3): xhat_0 = fl(fl(Q_0 - z_0) * s_0). Then R_0 = fl(W - xhat_0)
    (Eq. 5) and residual stages 1 .. S-1 quantize it as in ``construct_f32``.
    The base's zero-point need not be an integer (a foreign quantizer may store
    a real one), so Q_0 - z_0 is rounded like any binary32 difference.

    ``x`` float32 [n]; ``base_Q`` uint8 codes [n]; ``base_s``, ``base_z``
    float32 [n/G]. Returns (Q [S, n], s [S, n/G], z [S, n/G], rhat [S, n],
    final residual [n]) with stage 0 = the base as given and rhat[0] = xhat_0.
    """
    x = np.ascontiguousarray(x, dtype=np.float32).reshape(-1)
    _check_shape(x.size, group_size)
    if not np.all(np.isfinite(x)):
        raise ValueError("RRQ oracle: inputs must be finite")
    n_groups = x.size // group_size
    Q0 = np.asarray(base_Q, dtype=np.uint8).reshape(n_groups, group_size)
    s0 = np.asarray(base_s, dtype=np.float32).reshape(n_groups)
    z0 = np.asarray(base_z, dtype=np.float32).reshape(n_groups)
    if int(Q0.max(initial=0)) > (1 << bits) - 1:
        raise ValueError("RRQ oracle: base codes out of range")

    # Load and dequantize the base (Algorithm 1, first branch; Eq. 3).
    qz0 = Q0.astype(np.float32) - z0[:, None]              # fl(Q_0 - z_0)
    xhat0 = qz0 * s0[:, None]                                # fl(. * s_0)
    r = x.reshape(n_groups, group_size) - xhat0             # R_0 = W - What_0
    if not np.all(np.isfinite(r)):
        raise ValueError("RRQ oracle: the base residual W - xhat_0 must be finite")

    Qs, ss, zs, rhats = [Q0.reshape(-1)], [s0], [z0], [xhat0.reshape(-1)]
    for k in range(1, n_stages):
        Q, s, z, rhat = rtn_stage(r, bits)                  # residual stage k
        Qs.append(Q.reshape(-1))
        ss.append(s)
        zs.append(z)
        rhats.append(rhat.reshape(-1))
        r = r - rhat                                         # R_k = R_{k-1} - Rhat_k
    return (np.stack(Qs), np.stack(ss), np.stack(zs), np.stack(rhats),
            r.reshape(-1))


def construct_from_base(w_bits: np.ndarray, rows: int, cols: int, base_codes: np.ndarray,
                        base_scales: np.ndarray, base_zeros: np.ndarray, group_size: int,
                        n_stages: int):
    """The package of the C-ABI call rrq_construct_from_base: bfloat16 weights
    [rows, cols] (uint16 bits) and a base stage (packed codes [n/16] uint32,
    scales and zeros [n/G] float32) -> codes [S, n/16], scales [S, n/G],
    zeros [S, n/G], whose plane 0 is the base as given."""
    if cols % group_size != 0:
        raise ValueError("cols must be a multiple of the group size")
    w_bits = np.ascontiguousarray(w_bits, dtype=np.uint16).reshape(-1)
    assert w_bits.size == rows * cols
    x = bf16_bits_to_f32(w_bits)
    base_Q = unpack_codes(np.asarray(base_codes, dtype=np.uint32).reshape(-1))
    Q, s, z, _, _ = construct_from_base_f32(x, base_Q, base_scales, base_zeros, group_size,
                                            n_stages, bits=2)
    codes = np.stack([pack_codes(Q[k]) for k in range(n_stages)])
    return codes, s, z


# ---------------------------------------------------------------------------
# Prefix reconstruction (Eq. 8, Eq. 18-19)
# ---------------------------------------------------------------------------

def dequant_stage(codes_k: np.ndarray, s_k: np.ndarray, z_k: np.ndarray,
                  group_size: int) -> np.ndarray:
    """rhat = fl(fl(Q - z) s) for one stage, from its codes and the binary32
    values of its scale and zero-point (Q - z is exact for an integer z)."""
    Q = unpack_codes(codes_k).reshape(-1, group_size).astype(np.float32)
    qz = Q - np.asarray(z_k, dtype=np.float32)[:, None]
    return (qz * np.asarray(s_k, dtype=np.float32)[:, None]).reshape(-1)


def _stage_zeros(zeros, k, n_groups, zero_point):
    if zero_point == "sym":
        return np.full(n_groups, F32(2.0))
    return np.asarray(zeros[k], dtype=np.float32)


def reconstruct_f32(codes, scales, zeros, group_size: int, k_stages: int,
                    zero_point: str = "int", scale_dtype: str = "f32"):
    """Effective weight after k stages: rhat_0 + rhat_1 + ... + rhat_{k-1},
    summed left to right in binary32. ``scales`` as stored (see
    ``store_scales``); for symmetric stages ``zeros`` is ignored (z = 2)."""
    codes = np.asarray(codes, dtype=np.uint32)
    if not 1 <= k_stages <= codes.shape[0]:
        raise ValueError("k_stages out of range")
    ng = codes.shape[1] * 16 // group_size
    sv = lambda k: load_scales(scales[k], scale_dtype)
    acc = dequant_stage(codes[0], sv(0), _stage_zeros(zeros, 0, ng, zero_point), group_size)
    for t in range(1, k_stages):
        acc = acc + dequant_stage(codes[t], sv(t), _stage_zeros(zeros, t, ng, zero_point),
                                  group_size)
    return acc.astype(np.float32)


def reconstruct(codes, scales, zeros, group_size: int, k_stages: int,
                out_dtype: str = "f32", zero_point: str = "int", scale_dtype: str = "f32"):
    """Prefix-k reconstruction as float32, or as bfloat16 bit patterns
    (uint16) rounded to nearest-even when out_dtype == "bf16"."""
    acc = reconstruct_f32(codes, scales, zeros, group_size, k_stages, zero_point, scale_dtype)
    if out_dtype == "f32":
        return acc
    if out_dtype == "bf16":
        return f32_to_bf16_bits(acc)
    raise ValueError(out_dtype)


# ---------------------------------------------------------------------------
# Outlier diagnostic: the peak-to-mean ratio of each group (Sec. 3)
# ---------------------------------------------------------------------------

def group_pmr(x: np.ndarray, group_size: int) -> np.ndarray:
    """Peak-to-Mean Ratio of every group (Sec. 3): K / MAE with K the largest
    |x| of the group and MAE the mean |x|.

    Fixed binary32 reading: S = sum |x| is accumulated as four partial sums
    p_i over the elements j = i (mod 4), each in increasing j from +0, then
    S = fl(fl(p0 + p1) + fl(p2 + p3)); MAE = fl(S / G); PMR = fl(K / MAE).
    A group of zeros has PMR 0. Returns float32 [n / G].
    """
    x = np.ascontiguousarray(x, dtype=np.float32).reshape(-1, group_size)
    a = np.abs(x)
    K = a.max(axis=1)
    p = [np.zeros(x.shape[0], dtype=np.float32) for _ in range(4)]
    for j in range(group_size):                       # each partial sum in index order
        p[j % 4] = p[j % 4] + a[:, j]
    S = (p[0] + p[1]) + (p[2] + p[3])
    mae = S / np.float32(group_size)
    with np.errstate(divide="ignore", invalid="ignore"):
        pmr = K / mae
    return np.where(S > 0, pmr, np.float32(0.0)).astype(np.float32)


# ---------------------------------------------------------------------------
# Stage-sum linear layer (the prefill / decode product of Eq. 20)
# ---------------------------------------------------------------------------

def stage_values_f64(codes_t: np.ndarray, s_t: np.ndarray, z_t: np.ndarray, rows: int,
                     cols: int, group_size: int, row_index=None) -> np.ndarray:
    """Exact values (Q - z) s of one stage as float64 [len(row_index), cols]
    (Q - z and its product with a binary32 s are exact in float64)."""
    words_per_row = cols // 16
    gpr = cols // group_size
    rows_sel = np.arange(rows) if row_index is None else np.asarray(row_index)
    w = np.asarray(codes_t, dtype=np.uint32).reshape(rows, words_per_row)[rows_sel]
    Q = unpack_codes(w.reshape(-1)).reshape(len(rows_sel), cols).astype(np.float64)
    s = np.asarray(s_t, dtype=np.float32).reshape(rows, gpr)[rows_sel].astype(np.float64)
    z = np.asarray(z_t, dtype=np.float32).reshape(rows, gpr)[rows_sel].astype(np.float64)
    return ((Q.reshape(len(rows_sel), gpr, group_size) - z[:, :, None]) * s[:, :, None]
            ).reshape(len(rows_sel), cols)


def linear(codes, scales, zeros, rows: int, cols: int, group_size: int, k_stages: int,
           x_bits: np.ndarray, row_index=None) -> np.ndarray:
    """Y = X W~_(k)^T by the stage decomposition of Eq. 20:
    Y[m, o] = sum_{t < k} sum_i X[m, i] (Q_t[o, i] - z_t) s_t, in exact real
    arithmetic up to float64 summation (every product is exact in float64).

    ``x_bits``: bfloat16 activations [M, cols] as uint16 bit patterns.
    Returns float64 [M, rows] (or [M, len(row_index)] for a subset of rows).
    """
    codes = np.asarray(codes, dtype=np.uint32)
    if not 1 <= k_stages <= codes.shape[0]:
        raise ValueError("k_stages out of range")
    x = bf16_bits_to_f32(np.asarray(x_bits, dtype=np.uint16)).astype(np.float64)
    x = x.reshape(-1, cols)
    y = None
    for t in range(k_stages):
        R = stage_values_f64(codes[t], scales[t], zeros[t], rows, cols, group_size, row_index)
        yt = x @ R.T                               # A Rhat_t of Eq. 20
        y = yt if y is None else y + yt            # sum over the prefix's stages
    return y


# ---------------------------------------------------------------------------
# Direct fixed-bit RTN (the comparison quantizer of Sec. 3.4 / Eq. 9-14)
# ---------------------------------------------------------------------------

def direct_rtn_dequant(x: np.ndarray, group_size: int, bits: int) -> np.ndarray:
    """Single-stage b-bit RTN of x with the same range/scale/zero-point rules,
    dequantized; the "direct B-bit quantization" that Sec. 3.4 compares RRQ
    with."""
    x = np.ascontiguousarray(x, dtype=np.float32).reshape(-1, group_size)
    _, _, _, rhat = rtn_stage(x, bits)
    return rhat.reshape(-1)

"""Pins of the stage formats: symmetric stages, real-valued zero-points and
16-bit scales (the paper's symmetric configuration and its 16-bit-scale size
estimate, Sec. 4.1, Eq. 21, Table 14; the real zero-point of the Table 2
toy).

What fixes the expected values, independent of the oracle's own code:
* hand-derived cases (tests/golden/variant_cases.json);
* brute force: every code is the nearest point of its stage's grid (the
  symmetric grid {-2s, -s, 0, s}, or the real-zero-point grid whose end
  points are the group's min and max);
* two independent writings of the binary16 rounding (numpy's conversion in
  the numpy oracle, a hand-written one in the C oracle) agree on every
  binary32 bit pattern of a wide sample, ties and subnormals included;
* identities: 16-bit scales that are exactly representable give the binary32
  package; the numpy and C oracles agree on every format.
"""

import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import rrq_oracle as o

HERE = os.path.dirname(os.path.abspath(__file__))
G = 32


def _hex32(h):
    return np.array([int(h, 16)], dtype=np.uint32).view(np.float32)[0]


def _cases():
    return json.load(open(os.path.join(HERE, "golden", "variant_cases.json")))["cases"]


def _group(case):
    x = np.full(G, case["pad"], dtype=np.float32)
    x[:len(case["x"])] = case["x"]
    return x


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
@pytest.mark.parametrize("impl", ["numpy", "c"])
def test_golden_variants(case, impl):
    x = _group(case)
    bits = (x.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(o.bf16_bits_to_f32(bits), x)
    zp, sd = case["zero_point"], case["scale_dtype"]
    S = 2 if "stage1" in case else 1
    if impl == "numpy":
        codes, s, z = o.construct(bits, 1, G, G, S, zp, sd)
    else:
        codes, s, z = oracle.c_construct_format(bits, G, S, zp, sd)
    for k in range(S):
        st = case[f"stage{k}"]
        Q = o.unpack_codes(codes[k])
        want = np.full(G, st["pad_code"])
        want[:len(st["codes"])] = st["codes"]
        assert np.array_equal(Q, want), (k, Q[:8])
        if "s16" in st:
            assert f"{int(np.asarray(s[k]).view(np.uint16)[0]):04X}" == st["s16"]
        else:
            assert f"{int(np.asarray(s[k]).view(np.uint32)[0]):08X}" == st["s"]
        assert f"{int(z[k].view(np.uint32)[0]):08X}" == st["z"]
    rhat0 = o.reconstruct(codes, s, z, G, 1, "f32", zp, sd)
    for i, h in enumerate(case["rhat0"]):
        assert rhat0[i].view(np.uint32) == int(h, 16), (i, rhat0[i])


def _groups(n_groups, seed, outliers=True):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((n_groups, G)) * 10.0 ** rng.uniform(-3, 1, (n_groups, 1))).astype(np.float32)
    if outliers:
        x = np.where(rng.random(x.shape) < 0.03, x * 25, x).astype(np.float32)
    return o.bf16_bits_to_f32(o.f32_to_bf16_bits(x))


@pytest.mark.parametrize("zp", ["sym", "real"])
def test_codes_are_nearest_on_the_stage_grid(zp):
    r = _groups(200, 3 if zp == "sym" else 4)
    Q, s, z, _ = o.rtn_stage(r, 2, zp)
    for g in range(r.shape[0]):
        if s[g] == 0:
            continue
        sg, zg = Fraction(float(s[g])), Fraction(float(z[g]))
        grid = [(q - zg) * sg for q in range(4)]
        for j in range(G):
            x = Fraction(float(r[g, j]))
            best = min(abs(x - v) for v in grid)
            assert abs(x - grid[Q[g, j]]) <= best + sg / 2 ** 19, (g, j)
        if zp == "sym":
            amax = max(abs(Fraction(float(v))) for v in r[g])
            assert float(zg) == 2.0
            assert abs(sg - 2 * amax / 3) <= sg / 2 ** 22           # s = 2 amax / 3
        else:
            j_lo, j_hi = int(np.argmin(r[g])), int(np.argmax(r[g]))
            if r[g, j_lo] < 0:
                assert Q[g, j_lo] == 0                               # min is an exact end point
            if r[g, j_hi] > 0:
                assert Q[g, j_hi] == 3
            lo = min(Fraction(0), min(Fraction(float(v)) for v in r[g]))
            assert abs(zg - (-lo) / sg) <= Fraction(1, 2 ** 20) * (1 + abs(zg))


def test_symmetric_residual_bound():
    """On the symmetric grid every element within [-2.5 s, 1.5 s] keeps a
    residual of at most s/2; elements beyond 1.5 s (clamped) at most amax/3."""
    r = _groups(300, 5)
    Q, s, z, rhat = o.rtn_stage(r, 2, "sym")
    res = (r.astype(np.float64) - rhat)
    amax = np.abs(r).max(axis=1).astype(np.float64)
    assert np.all(np.abs(res) <= np.maximum(s[:, None] * 0.5, amax[:, None] / 3) * (1 + 2.0 ** -20) + 1e-45)


def test_two_writings_of_binary16_rounding_agree():
    rng = np.random.default_rng(0)
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = [0x0000, 0x0FFF, 0x1000, 0x1001, 0x1FFF, 0x8000, 0x8001, 0x7FFF, 0xFFFF]
    pats = np.concatenate([hi | l for l in lows] + [rng.integers(0, 1 << 32, 1 << 18, dtype=np.uint64).astype(np.uint32)])
    x = pats.view(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) < 65504.0)]
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    got = oracle.c_f32_to_f16(x)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, [(hex(int(x[i].view(np.uint32))), hex(int(got[i])), hex(int(want[i]))) for i in bad[:5]]


@pytest.mark.parametrize("sd", ["f16", "bf16"])
def test_representable_16bit_scales_change_nothing(sd):
    """Groups whose stage-0 scale d/3 is a power of two: the 16-bit scale is
    exact, so the single-stage package equals the binary32 one."""
    rng = np.random.default_rng(9)
    n_groups = 64
    e = rng.integers(-10, 0, n_groups)
    x = np.zeros((n_groups, G), dtype=np.float32)
    x[:, 0] = -(2.0 ** e) * rng.integers(0, 3, n_groups)             # lo in {0, -s, -2s}
    x[:, 1] = 3 * 2.0 ** e + x[:, 0]                                  # hi - lo = 3 s
    x[:, 2:] = (rng.random((n_groups, G - 2)) * (x[:, 1:2] - x[:, 0:1]) + x[:, 0:1]).astype(np.float32)
    bits = o.f32_to_bf16_bits(x.reshape(-1))
    x = o.bf16_bits_to_f32(bits).reshape(n_groups, G)
    assert np.all(np.abs(x[:, 1] - x[:, 0] - 3 * 2.0 ** e) == 0)
    for zp in ("int", "real"):
        a = o.construct(bits, 1, bits.size, G, 1, zp, "f32")
        b = o.construct(bits, 1, bits.size, G, 1, zp, sd)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[2], b[2])
        assert np.array_equal(a[1], o.load_scales(b[1], sd))


@pytest.mark.parametrize("zp,sd", list(itertools.product(o.ZERO_POINTS, o.SCALE_DTYPES)))
def test_numpy_and_c_oracles_agree_on_every_format(zp, sd):
    rng = np.random.default_rng(len(zp) * 10 + len(sd))
    x = (rng.standard_normal(128 * 200) * 0.02).astype(np.float32)
    x = np.where(rng.random(x.size) < 1e-2, x * 20, x).astype(np.float32)
    bits = o.f32_to_bf16_bits(x)
    a = o.construct(bits, 1, bits.size, 128, 4, zp, sd)
    b = oracle.c_construct_format(bits, 128, 4, zp, sd)
    for p, q in zip(a, b):
        assert np.array_equal(np.asarray(p).view(np.uint8), np.asarray(q).view(np.uint8))
    for k in (1, 4):
        ra = o.reconstruct(a[0], a[1], a[2], 128, k, "bf16", zp, sd)
        rb = oracle.c_reconstruct_format(b[0], b[1], b[2], 128, k, zp, sd, "bf16")
        assert np.array_equal(ra, rb)


def test_default_format_is_the_frozen_reading():
    bits = o.f32_to_bf16_bits((np.random.default_rng(2).standard_normal(128 * 50) * 0.02).astype(np.float32))
    a = o.construct(bits, 1, bits.size, 128, 4)
    b = o.construct(bits, 1, bits.size, 128, 4, "int", "f32")
    c = oracle.c_construct(bits, 128, 4)
    for p, q, r in zip(a, b, c):
        assert np.array_equal(p, q) and np.array_equal(p, r)

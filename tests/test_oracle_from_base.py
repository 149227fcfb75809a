"""Pins of the oracle's construction on an existing base checkpoint
(Algorithm 1, the branch that loads a base; Eq. 3-7).

What fixes the expected values, independent of the oracle's own code:
* a hand-derived worked case with a real-valued base zero-point
  (tests/golden/from_base_cases.json);
* identities with the already pinned construction: a base that is the
  oracle's own first stage reproduces the full package; a base with zero
  scales leaves R_0 = W, so the residual stages are the stages of a direct
  package with one stage fewer;
* an exact base (W equal to its dequantized base) leaves nothing to quantize:
  every residual stage is degenerate;
* brute force: every residual stage's codes are nearest on its grid;
* the numpy and C writings agree bit for bit on random bases with real
  zero-points.
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


def _f(hexbits):
    return np.array([int(h, 16) for h in hexbits], dtype=np.uint32).view(np.float32)


def _weights(n, seed, outliers=True):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(n) * 0.02).astype(np.float32)
    if outliers:
        x = np.where(rng.random(n) < 1e-2, x * 20, x).astype(np.float32)
    return o.f32_to_bf16_bits(x)


def _random_base(n, G, seed, integer_zero=False):
    """A foreign base stage: random codes, positive scales of the weights'
    magnitude, zero-points real in [0, 3) (or integers 0..3)."""
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 2 ** 32, n // 16, dtype=np.uint64).astype(np.uint32)
    s = (0.02 * (0.5 + 4 * rng.random(n // G))).astype(np.float32)
    z = (rng.integers(0, 4, n // G) if integer_zero else 3 * rng.random(n // G)).astype(np.float32)
    return codes, s, z


def _golden():
    with open(os.path.join(HERE, "golden", "from_base_cases.json")) as fh:
        return json.load(fh)["cases"]


@pytest.mark.parametrize("case", _golden(), ids=lambda c: c["name"])
@pytest.mark.parametrize("impl", ["numpy", "c"])
def test_golden_from_base(case, impl):
    G, S = case["G"], case["S"]
    words = np.array([int(h, 16) for h in case["base_codes"]], dtype=np.uint32)
    s0, z0 = _f([case["base_scale"]]), _f([case["base_zero"]])
    Q0 = o.unpack_codes(words).astype(np.float64)
    xhat0 = (Q0 - float(z0[0])) * float(s0[0])         # exact here (hand-checked values)
    R0 = _f(case["residual"]).astype(np.float64)[(np.arange(G) // 4) % 4]
    x = (xhat0 + R0).astype(np.float32)
    assert np.array_equal(x.astype(np.float64), xhat0 + R0)   # W exact in binary32
    bits = (x.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(o.bf16_bits_to_f32(bits), x)        # and in bfloat16
    if impl == "numpy":
        codes, s, z = o.construct_from_base(bits, 1, G, words, s0, z0, G, S)
    else:
        codes, s, z = oracle.c_construct_from_base(bits, words, s0, z0, G, S)
    for k, st in enumerate(case["stages"]):
        assert [f"{w:08X}" for w in codes[k]] == st["codes"], k
        assert f"{s[k].view(np.uint32)[0]:08X}" == st["s"], k
        assert f"{z[k].view(np.uint32)[0]:08X}" == st["z"], k
    assert np.array_equal(o.reconstruct(codes, s, z, G, 1), xhat0.astype(np.float32))
    for k in range(2, S + 1):
        assert np.array_equal(o.reconstruct(codes, s, z, G, k), x)


@pytest.mark.parametrize("G", [32, 64, 128])
@pytest.mark.parametrize("S", [1, 2, 3, 4])
def test_own_first_stage_as_base_reproduces_package(G, S):
    """Loading the package's own first stage as the base (Algorithm 1's two
    branches meet): the result is the direct package."""
    bits = _weights(G * 96, 200 + G + S)
    want = o.construct(bits, 1, bits.size, G, S)
    base = o.construct(bits, 1, bits.size, G, 1)
    got = o.construct_from_base(bits, 1, bits.size, base[0][0], base[1][0], base[2][0], G, S)
    got_c = oracle.c_construct_from_base(bits, base[0][0], base[1][0], base[2][0], G, S)
    for a, b, c in zip(want, got, got_c):
        assert np.array_equal(a, b) and np.array_equal(a, c)


@pytest.mark.parametrize("G", [32, 128])
def test_zero_scale_base_leaves_weights_as_residual(G):
    """s_0 = 0: xhat_0 = 0 whatever the codes and zero-points, R_0 = W, and
    the residual stages are the stages of the direct package with S - 1
    stages."""
    n, S = G * 64, 4
    bits = _weights(n, 300 + G)
    codes0, _, z0 = _random_base(n, G, 301 + G)
    s0 = np.zeros(n // G, dtype=np.float32)
    got = o.construct_from_base(bits, 1, n, codes0, s0, z0, G, S)
    direct = o.construct(bits, 1, n, G, S - 1)
    for a, b in zip(got, direct):
        assert np.array_equal(a[1:], b)
    assert np.array_equal(got[0][0], codes0) and np.array_equal(got[2][0], z0)


def test_exact_base_leaves_degenerate_residual_stages():
    """W equal to its dequantized base: R_0 = 0, so every residual stage has
    s = z = 0 and zero codes, and every prefix reconstructs W."""
    G, n, S = 64, 64 * 32, 4
    rng = np.random.default_rng(5)
    Q0 = rng.integers(0, 4, n).astype(np.uint8)
    s0 = (2.0 ** rng.integers(-10, -2, n // G)).astype(np.float32)    # powers of two
    z0 = rng.integers(0, 4, n // G).astype(np.float32)
    x = ((Q0.reshape(-1, G) - z0[:, None]) * s0[:, None]).astype(np.float32).reshape(-1)
    bits = (x.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(o.bf16_bits_to_f32(bits), x)
    codes, s, z = o.construct_from_base(bits, 1, n, o.pack_codes(Q0), s0, z0, G, S)
    assert np.all(s[1:] == 0) and np.all(z[1:] == 0) and np.all(codes[1:] == 0)
    assert np.all(s[1:].view(np.uint32) == 0) and np.all(z[1:].view(np.uint32) == 0)
    for k in range(1, S + 1):
        assert np.array_equal(o.reconstruct(codes, s, z, G, k), x)


def _grid_error(r, Q, s, z):
    return sum(abs(Fraction(float(rj)) - (int(q) - Fraction(float(z))) * Fraction(float(s)))
               for rj, q in zip(r, Q))


def test_residual_stages_are_nearest_on_their_grids():
    """Brute force over every code vector of a few elements of each residual
    stage's group: the oracle's codes have the least distance to the grid
    (within the rounding of 1/s and r/s), on random real-zero-point bases."""
    G, n, S = 32, 32 * 6, 4
    for seed in range(6):
        bits = _weights(n, 400 + seed)
        codes0, s0, z0 = _random_base(n, G, 500 + seed)
        Q, s, z, rhat, _ = o.construct_from_base_f32(o.bf16_bits_to_f32(bits),
                                                     o.unpack_codes(codes0), s0, z0, G, S)
        r = o.bf16_bits_to_f32(bits).reshape(-1, G) - rhat[0].reshape(-1, G)
        for k in range(1, S):
            for g in range(n // G):
                if s[k][g] == 0:
                    continue
                idx = [0, 7, 19, 31]                   # 4^4 candidates per group
                rs, Qs = r[g, idx], Q[k].reshape(-1, G)[g, idx]
                mine = _grid_error(rs, Qs, s[k][g], z[k][g])
                best = min(_grid_error(rs, cand, s[k][g], z[k][g])
                           for cand in itertools.product(range(4), repeat=len(idx)))
                assert mine <= best + len(idx) * Fraction(float(s[k][g])) / 2 ** 20
                # each element individually nearest too
                for j in range(G):
                    e = abs(Fraction(float(r[g, j])) -
                            (int(Q[k].reshape(-1, G)[g, j]) - Fraction(float(z[k][g]))) * Fraction(float(s[k][g])))
                    assert e <= Fraction(float(s[k][g])) * (Fraction(1, 2) + Fraction(1, 2 ** 20)) or \
                        int(Q[k].reshape(-1, G)[g, j]) in (0, 3)
            r = r - rhat[k].reshape(-1, G)


@pytest.mark.parametrize("G,S,integer_zero", [(32, 4, False), (64, 3, False), (128, 4, False),
                                               (128, 2, True), (64, 1, False)])
def test_two_oracles_agree_on_random_bases(G, S, integer_zero):
    n = G * 512
    bits = _weights(n, 600 + G + S)
    base = _random_base(n, G, 700 + G + S, integer_zero)
    a = o.construct_from_base(bits, 1, n, *base, G, S)
    b = oracle.c_construct_from_base(bits, *base, G, S)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    assert np.array_equal(a[0][0], base[0])


def test_nonfinite_base_residual_rejected():
    G, n = 32, 64
    bits = _weights(n, 1)
    codes0 = np.full(n // 16, 0xFFFFFFFF, dtype=np.uint32)       # all codes 3
    s0 = np.full(n // G, 3e38, dtype=np.float32)
    z0 = np.zeros(n // G, dtype=np.float32)                       # 3 * 3e38 overflows
    with pytest.raises(ValueError):
        o.construct_from_base(bits, 1, n, codes0, s0, z0, G, 2)
    with pytest.raises(ValueError):
        oracle.c_construct_from_base(bits, codes0, s0, z0, G, 2)

"""Pins of the oracle's stage-sum product (Eq. 20): Y = X W~_(k)^T computed
as the sum over the prefix's stages of X Rhat_t^T.

What fixes the expected values, independent of ``linear``'s own code:
* hand-derived values on the hand-derived base-checkpoint package
  (tests/golden/linear_cases.json);
* brute force in exact rational arithmetic, element by element, on tiny
  packages;
* the pinned reconstruction: a one-hot X returns a column of W~_(k) exactly
  whenever the binary32 stage sum is exact, and for any X the product agrees
  with a float64 library matmul of the binary32 reconstruction within that
  reconstruction's rounding.
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import rrq_oracle as o

HERE = os.path.dirname(os.path.abspath(__file__))


def _golden_package():
    cases = json.load(open(os.path.join(HERE, "golden", "from_base_cases.json")))["cases"]
    case = cases[0]
    f = lambda h: np.array([int(h, 16)], dtype=np.uint32).view(np.float32)
    codes = np.array([[int(h, 16) for h in st["codes"]] for st in case["stages"]], dtype=np.uint32)
    s = np.stack([f(st["s"]) for st in case["stages"]])
    z = np.stack([f(st["z"]) for st in case["stages"]])
    return codes, s, z


def _x_named(name, n):
    if name == "ones":
        x = np.ones(n, dtype=np.float32)
    elif name == "alternating":
        x = np.where(np.arange(n) % 2 == 0, 1.0, -1.0).astype(np.float32)
    elif name.startswith("one_hot_"):
        x = np.zeros(n, dtype=np.float32)
        x[int(name.rsplit("_", 1)[1])] = 1.0
    else:
        raise KeyError(name)
    return o.f32_to_bf16_bits(x).reshape(1, n)


@pytest.mark.parametrize("case", json.load(open(os.path.join(HERE, "golden", "linear_cases.json")))["cases"],
                         ids=lambda c: c["name"])
def test_golden_linear(case):
    codes, s, z = _golden_package()
    x = _x_named(case["x"], 32)
    for k, want in case["y"].items():
        y = o.linear(codes, s, z, 1, 32, 32, int(k), x)
        assert y.shape == (1, 1) and y[0, 0] == want, (k, y[0, 0], want)


def _exact_package(rows, cols, G, S, seed):
    """A package whose stage values and their sums are exact in binary32:
    power-of-two scales, integer zero-points."""
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 2 ** 32, (S, rows * cols // 16), dtype=np.uint64).astype(np.uint32)
    s = (2.0 ** rng.integers(-8, -2, (S, rows * cols // G))).astype(np.float32)
    z = rng.integers(0, 4, (S, rows * cols // G)).astype(np.float32)
    return codes, s, z


def _brute(codes, s, z, rows, cols, G, k, x_bits):
    x = o.bf16_bits_to_f32(x_bits).reshape(-1, cols)
    M = x.shape[0]
    y = [[Fraction(0)] * rows for _ in range(M)]
    for t in range(k):
        for r in range(rows):
            for i in range(cols):
                e = r * cols + i
                q = (int(codes[t][e // 16]) >> (2 * (e % 16))) & 3
                g = e // G
                w = (q - Fraction(float(z[t][g]))) * Fraction(float(s[t][g]))
                for m in range(M):
                    y[m][r] += Fraction(float(x[m, i])) * w
    return y


@pytest.mark.parametrize("rows,cols,G,k,M", [(3, 64, 32, 2, 2), (2, 128, 64, 4, 3), (1, 128, 128, 3, 1)])
def test_bruteforce_rational(rows, cols, G, k, M):
    rng = np.random.default_rng(rows * 100 + cols + k)
    x = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    codes, s, z = o.construct(o.f32_to_bf16_bits(x), rows, cols, G, 4)
    xb = o.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    y = o.linear(codes, s, z, rows, cols, G, k, xb)
    ref = _brute(codes, s, z, rows, cols, G, k, xb)
    for m in range(M):
        for r in range(rows):
            assert abs(Fraction(float(y[m, r])) - ref[m][r]) <= abs(ref[m][r]) * Fraction(1, 2 ** 45) + Fraction(1, 2 ** 80)


def test_one_hot_returns_reconstruction_columns():
    rows, cols, G, S = 6, 256, 64, 4
    codes, s, z = _exact_package(rows, cols, G, S, 3)
    for k in range(1, S + 1):
        W = o.reconstruct(codes, s, z, G, k).reshape(rows, cols)
        for j in (0, 1, 63, 64, 200, 255):
            x = np.zeros((1, cols), dtype=np.float32)
            x[0, j] = 1.0
            y = o.linear(codes, s, z, rows, cols, G, k, o.f32_to_bf16_bits(x))
            assert np.array_equal(y[0], W[:, j].astype(np.float64)), (k, j)


@pytest.mark.parametrize("G", [32, 64, 128])
def test_agrees_with_library_matmul_of_reconstruction(G):
    rows, cols, M = 40, 512, 5
    rng = np.random.default_rng(G)
    w = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    w = np.where(rng.random(w.size) < 1e-2, w * 20, w).astype(np.float32)
    codes, s, z = o.construct(o.f32_to_bf16_bits(w), rows, cols, G, 4)
    xb = o.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    x = o.bf16_bits_to_f32(xb).reshape(M, cols).astype(np.float64)
    for k in range(1, 5):
        W = o.reconstruct(codes, s, z, G, k).reshape(rows, cols).astype(np.float64)
        y = o.linear(codes, s, z, rows, cols, G, k, xb)
        # W~ in binary32 is the stage sum rounded k - 1 times
        bound = (k * 2.0 ** -24) * (np.abs(x) @ np.abs(W).T) * 2 + 1e-30
        assert np.all(np.abs(y - x @ W.T) <= bound), k


def test_row_subset_matches_full():
    rows, cols, G = 10, 256, 128
    codes, s, z = _exact_package(rows, cols, G, 4, 9)
    xb = o.f32_to_bf16_bits(np.random.default_rng(1).standard_normal((2, cols)).astype(np.float32))
    full = o.linear(codes, s, z, rows, cols, G, 3, xb)
    sub = o.linear(codes, s, z, rows, cols, G, 3, xb, row_index=[9, 0, 4])
    assert np.array_equal(sub, full[:, [9, 0, 4]])

"""GPU parity of rrq_linear's decode form (up to 4 tokens, groups of 128,
cols a multiple of 4096 up to 16384; 2 to 4 stages at any row count, 1 stage
up to 1024 rows or from 12288 rows with up to 8192 cols; 5 to 8 tokens on
rows of 4096 inputs, up to 1024 rows at any stage count and from 3 stages up
to 2048 rows and from 4097 to 6144 rows; 9 to 16 tokens up to 1024 rows from
3 stages), through the C ABI,
against the oracle's Eq. 20 product in float64 on sampled output rows.

* exact: power-of-two scales, integer or dyadic zero-points and
  small-integer activations make every intermediate exactly representable,
  so the sampled outputs must equal the exact value bit for bit (this pins
  the kernel's row, group, stage, token and lane bookkeeping, partial last
  row tiles included);
* bounded: realistic packages built by the oracle, in every stage format,
  stay within the bound stated in include/rrq.h.
Packages come from the oracle or a seeded generator, never from the GPU.
"""

import math
import sys

import numpy as np
import pytest

import oracle
from oracle import rrq_oracle as npo

pytestmark = pytest.mark.gpu
U = 2.0 ** -24
G = 128


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _sample_rows(rows, seed):
    rng = np.random.default_rng(seed)
    idx = np.unique(np.concatenate([np.arange(min(8, rows)), np.arange(max(rows - 8, 0), rows),
                                    rng.choice(rows, min(256, rows), replace=False)]))
    return idx


def _run(gpu, codes, s, z, rows, cols, k, xb, zp=None, sd=None, s_raw=None):
    import torch
    M = xb.size // cols
    c = torch.from_numpy(codes.view(np.int32).copy()).cuda()
    sc = torch.from_numpy((s if s_raw is None else s_raw).copy()).cuda()
    ze = None if z is None else torch.from_numpy(z.copy()).cuda()
    X = torch.from_numpy(xb.view(np.int16).reshape(M, cols).copy()).cuda().view(torch.bfloat16)
    Y = torch.full((M, rows), float("nan"), dtype=torch.float32, device="cuda")
    if zp is None:
        gpu.rrq_linear(c, sc, ze, rows, cols, G, codes.shape[0], k, X, M, Y)
    else:
        gpu.rrq_linear_format(c, sc, ze, rows, cols, G, codes.shape[0], gpu.ZERO_POINTS[zp],
                              gpu.SCALE_TYPES[sd], k, X, M, Y)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


@pytest.mark.parametrize("rows,cols,M,k", [
    (6144, 4096, 1, 2), (6144, 4096, 4, 4), (6150, 8192, 3, 3), (6147, 12288, 2, 4),
    (8192, 16384, 1, 2), (24576, 4096, 4, 3),
    # few tiles (fewer workgroups than CUs), ragged last tile, small matrices
    (1, 4096, 1, 3), (5, 4096, 2, 4), (1023, 4096, 1, 4), (1021, 4096, 4, 2), (2047, 4096, 4, 2),
    (4096, 4096, 1, 3), (4099, 8192, 2, 4), (1024, 16384, 1, 3),
    # one stage
    (1000, 4096, 2, 1), (12290, 8192, 1, 1), (13, 12288, 4, 1),
    # rows of 12288 and 16384 inputs: 12 and 16 waves of 2 sets per workgroup
    (4096, 12288, 1, 4), (4099, 12288, 3, 3), (2050, 16384, 4, 4), (30, 16384, 2, 2),
    # 5 to 8 tokens: two quads of tokens (the second partly past the last)
    (1024, 4096, 5, 1), (1021, 4096, 8, 2), (3, 4096, 6, 4), (6144, 4096, 8, 4),
    (6000, 4096, 7, 3), (2048, 4096, 5, 3), (4099, 4096, 8, 3), (1999, 4096, 6, 4),
    # 9 to 16 tokens: four quads (the last partly past the last token)
    (1024, 4096, 16, 4), (1000, 4096, 12, 3), (3, 4096, 9, 4), (513, 4096, 13, 3),
])
def test_decode_form_exact(gpu, rows, cols, M, k):
    _log(f"decode exact rows={rows} cols={cols} M={M} k={k}")
    rng = np.random.default_rng(rows + cols + M + k)
    S = 4
    codes = rng.integers(0, 2 ** 32, (S, rows * cols // 16), dtype=np.uint64).astype(np.uint32)
    s = (2.0 ** rng.integers(-4, -1, (S, rows * cols // G))).astype(np.float32)
    z = rng.integers(0, 4, (S, rows * cols // G)).astype(np.float32)
    xb = npo.f32_to_bf16_bits(rng.integers(-4, 5, (M, cols)).astype(np.float32))
    y = _run(gpu, codes, s, z, rows, cols, k, xb)
    idx = _sample_rows(rows, k)
    ref = npo.linear(codes, s, z, rows, cols, G, k, xb, row_index=idx)
    assert np.all(np.abs(ref) < 2.0 ** 20)
    got = y[:, idx].astype(np.float64)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}"
    assert not np.any(np.isnan(y)), "unwritten outputs"


@pytest.mark.parametrize("zp,sd", [("int", "f32"), ("sym", "f16"), ("real", "f32"),
                                   ("int", "bf16")])
def test_decode_form_exact_formats(gpu, zp, sd):
    """Stage formats through the decode form: power-of-two scales stored as
    16-bit patterns where the format says so, dyadic real zero-points."""
    rows, cols, k = 6140, 4096, 4
    M = 3 if zp == "int" and sd == "f32" else 7
    _log(f"decode exact format {zp}/{sd} M={M}")
    rng = np.random.default_rng(77)
    S = 4
    codes = rng.integers(0, 2 ** 32, (S, rows * cols // 16), dtype=np.uint64).astype(np.uint32)
    s = (2.0 ** rng.integers(-4, -1, (S, rows * cols // G))).astype(np.float32)
    if zp == "sym":
        z = None
        zv = np.full_like(s, 2.0)
    elif zp == "real":
        z = (rng.integers(0, 13, s.shape) * 0.25).astype(np.float32)
        zv = z
    else:
        z = rng.integers(0, 4, s.shape).astype(np.float32)
        zv = z
    if sd == "f16":
        s_raw = s.astype(np.float16).view(np.uint16)
    elif sd == "bf16":
        s_raw = (s.view(np.uint32) >> 16).astype(np.uint16)
    else:
        s_raw = s
    xb = npo.f32_to_bf16_bits(rng.integers(-4, 5, (M, cols)).astype(np.float32))
    y = _run(gpu, codes, s, z, rows, cols, k, xb, zp=zp, sd=sd, s_raw=s_raw)
    idx = _sample_rows(rows, 5)
    ref = npo.linear(codes, s, zv, rows, cols, G, k, xb, row_index=idx)
    got = y[:, idx].astype(np.float64)
    assert np.array_equal(got, ref), np.max(np.abs(got - ref))


@pytest.mark.parametrize("zp,sd", [("sym", "f16"), ("real", "f32"), ("int", "bf16")])
def test_decode_form_exact_formats_four_quads(gpu, zp, sd):
    """Stage formats through the decode form's four quads of tokens (16
    tokens on 1000 rows of 4096 inputs, 4 and 3 stages)."""
    rows, cols, M = 1000, 4096, 16
    _log(f"decode exact format four quads {zp}/{sd}")
    rng = np.random.default_rng(78)
    S = 4
    codes = rng.integers(0, 2 ** 32, (S, rows * cols // 16), dtype=np.uint64).astype(np.uint32)
    s = (2.0 ** rng.integers(-4, -1, (S, rows * cols // G))).astype(np.float32)
    if zp == "sym":
        z, zv = None, np.full_like(s, 2.0)
    elif zp == "real":
        z = (rng.integers(0, 13, s.shape) * 0.25).astype(np.float32)
        zv = z
    else:
        z = rng.integers(0, 4, s.shape).astype(np.float32)
        zv = z
    s_raw = (s.astype(np.float16).view(np.uint16) if sd == "f16"
             else (s.view(np.uint32) >> 16).astype(np.uint16) if sd == "bf16" else s)
    xb = npo.f32_to_bf16_bits(rng.integers(-4, 5, (M, cols)).astype(np.float32))
    for k in (4, 3):
        y = _run(gpu, codes, s, z, rows, cols, k, xb, zp=zp, sd=sd, s_raw=s_raw)
        idx = _sample_rows(rows, 7)
        ref = npo.linear(codes, s, zv, rows, cols, G, k, xb, row_index=idx)
        got = y[:, idx].astype(np.float64)
        assert np.array_equal(got, ref), (k, np.max(np.abs(got - ref)))


@pytest.mark.parametrize("zp,sd", [("int", "f32"), ("sym", "f16"), ("real", "f32")])
@pytest.mark.parametrize("M", [4, 8])
def test_decode_form_realistic_within_bound(gpu, zp, sd, M):
    rows, cols = 6144, 4096
    rng = np.random.default_rng(9)
    w = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    w = np.where(rng.random(w.size) < 1e-3, w * 20, w).astype(np.float32)
    bits = npo.f32_to_bf16_bits(w)
    oc, os_, oz = oracle.c_construct_format(bits, G, 4, zp, sd)
    sv = npo.load_scales(os_, sd)
    zv = np.full_like(sv, 2.0) if zp == "sym" else oz
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    idx = _sample_rows(rows, 3)
    xa = np.abs(npo.bf16_bits_to_f32(xb).reshape(M, cols).astype(np.float64))
    T = xa.reshape(M, cols // G, G).sum(axis=2)
    for k in (2, 3, 4):
        y = _run(gpu, oc, sv, None if zp == "sym" else oz, rows, cols, k, xb, zp=zp, sd=sd,
                 s_raw=os_)
        ref = npo.linear(oc, sv, zv, rows, cols, G, k, xb, row_index=idx)
        A = sum(T @ (np.abs(sv[t].astype(np.float64)) * (11 + np.abs(zv[t].astype(np.float64))))
                .reshape(rows, cols // G)[idx].T for t in range(k))
        p = cols // G
        n = k * (min(p, 4 * math.ceil(p / 16)) + 1)
        tol = 1.05 * U * A * (G + 2 * n + 24) + 1e-300
        err = np.abs(y[:, idx].astype(np.float64) - ref)
        assert np.all(err <= tol), f"k={k}: {np.max(err / tol)}"
        _log(f"decode realistic {zp}/{sd} k={k}: max err / bound = {np.max(err / tol):.3g}")


@pytest.mark.parametrize("zp,sd", [("int", "f32"), ("sym", "f16")])
def test_decode_form_four_quads_realistic_within_bound(gpu, zp, sd):
    """Realistic packages through the four quads of tokens (16 tokens on 1000
    rows of 4096 inputs, 3 and 4 stages) stay within the stated bound."""
    rows, cols, M = 1000, 4096, 16
    rng = np.random.default_rng(19)
    w = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    w = np.where(rng.random(w.size) < 1e-3, w * 20, w).astype(np.float32)
    oc, os_, oz = oracle.c_construct_format(npo.f32_to_bf16_bits(w), G, 4, zp, sd)
    sv = npo.load_scales(os_, sd)
    zv = np.full_like(sv, 2.0) if zp == "sym" else oz
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    xa = np.abs(npo.bf16_bits_to_f32(xb).reshape(M, cols).astype(np.float64))
    T = xa.reshape(M, cols // G, G).sum(axis=2)
    for k in (3, 4):
        y = _run(gpu, oc, sv, None if zp == "sym" else oz, rows, cols, k, xb, zp=zp, sd=sd,
                 s_raw=os_)
        ref = npo.linear(oc, sv, zv, rows, cols, G, k, xb)
        A = sum(T @ (np.abs(sv[t].astype(np.float64)) * (11 + np.abs(zv[t].astype(np.float64))))
                .reshape(rows, cols // G).T for t in range(k))
        p = cols // G
        n = k * (min(p, 4 * math.ceil(p / 16)) + 1)
        tol = 1.05 * U * A * (G + 2 * n + 24) + 1e-300
        err = np.abs(y.astype(np.float64) - ref)
        assert np.all(err <= tol), f"k={k}: {np.max(err / tol)}"
        _log(f"decode four quads realistic {zp}/{sd} k={k}: max err / bound = {np.max(err / tol):.3g}")

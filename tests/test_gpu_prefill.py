"""GPU parity of rrq_linear's prefill form (groups of 128, at least 128 tokens),
through the C ABI:

* exact: power-of-two scales, integer or dyadic zero-points and
  small-integer activations make every intermediate exactly representable,
  so all outputs must equal the oracle's Eq. 20 product bit for bit (ragged
  token and row tiles, one to many groups per row, every stage count and
  format);
* same order: the prefill form accumulates in the general kernel's order, so
  on realistic packages its outputs equal, bit for bit, those of the same
  tokens sent 16 at a time (which the general kernel serves);
* bounded: realistic packages built by the oracle stay within the bound
  stated in include/rrq.h.
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


def _run(gpu, codes, s_raw, z, rows, cols, k, xb, zp="int", sd="f32"):
    import torch
    M = xb.size // cols
    c = torch.from_numpy(codes.view(np.int32).copy()).cuda()
    sc = torch.from_numpy(s_raw.copy()).cuda()
    ze = None if z is None else torch.from_numpy(z.copy()).cuda()
    X = torch.from_numpy(xb.view(np.int16).reshape(M, cols).copy()).cuda().view(torch.bfloat16)
    Y = torch.full((M, rows), float("nan"), dtype=torch.float32, device="cuda")
    gpu.rrq_linear_format(c, sc, ze, rows, cols, G, codes.shape[0], gpu.ZERO_POINTS[zp],
                          gpu.SCALE_TYPES[sd], k, X, M, Y)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


def _exact(rows, cols, M, seed):
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 2 ** 32, (4, rows * cols // 16), dtype=np.uint64).astype(np.uint32)
    s = (2.0 ** rng.integers(-4, -1, (4, rows * cols // G))).astype(np.float32)
    z = rng.integers(0, 4, (4, rows * cols // G)).astype(np.float32)
    xb = npo.f32_to_bf16_bits(rng.integers(-4, 5, (M, cols)).astype(np.float32))
    return codes, s, z, xb


@pytest.mark.parametrize("rows,cols,M", [
    (16, 128, 128), (5, 384, 140), (64, 1024, 192), (100, 4096, 129), (257, 2048, 130),
    (64, 12288, 200), (1, 4224, 161),
    # from 1024 tokens the 2-4 stage kernels raise their MFMA stretches' priority
    (70, 1024, 1100), (33, 2048, 1024),
])
@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_prefill_exact(gpu, rows, cols, M, k):
    _log(f"prefill exact rows={rows} cols={cols} M={M} k={k}")
    codes, s, z, xb = _exact(rows, cols, M, rows + cols + M)
    y = _run(gpu, codes, s, z, rows, cols, k, xb)
    ref = npo.linear(codes, s, z, rows, cols, G, k, xb)
    assert np.all(np.abs(ref) < 2.0 ** 20)
    bad = np.argwhere(y.astype(np.float64) != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}"


def _large_tiles(rows, M):
    """Whether rrq_linear takes the 128-row x 128-token tiles for this call:
    when they give at least 3/4 of the compute units a workgroup."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    return 4 * -(-rows // 128) * -(-M // 128) >= 3 * cus


# 128 x 128 tiles with ragged edges: 1990 rows leave the last row tile 70 rows
# (waves 0-3 full, wave 4 six rows, waves 5-7 none), 1500 tokens leave the
# last token tile 92 (its tiles 6 and 7 without tokens)
LARGE = [(1990, 1024, 1500), (2048, 1152, 1409)]


@pytest.mark.parametrize("rows,cols,M", LARGE)
@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_prefill_exact_large_tiles(gpu, rows, cols, M, k):
    assert _large_tiles(rows, M)
    _log(f"prefill exact, large tiles rows={rows} cols={cols} M={M} k={k}")
    codes, s, z, xb = _exact(rows, cols, M, rows + cols + M + k)
    y = _run(gpu, codes, s, z, rows, cols, k, xb)
    ref = npo.linear(codes, s, z, rows, cols, G, k, xb)
    assert np.all(np.abs(ref) < 2.0 ** 20)
    bad = np.argwhere(y.astype(np.float64) != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}"


def _wide_tiles(rows, M):
    """Whether rrq_linear takes waves of 32 rows at one stage (256 rows x
    128 tokens per workgroup): when they give every compute unit one."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    return -(-rows // 256) * -(-M // 128) >= cus


# one stage, 32-row waves with ragged edges: 3000 rows leave the last row tile
# 184 rows (waves 0-4 full, wave 5 24 rows: 8 in its second row tile, waves
# 6 and 7 none), 2700 tokens leave the last token tile 12
WIDE = (3000, 384, 2700)


@pytest.mark.parametrize("rows,M,k", [(2048, 1536, 1), (2048, 1536, 2), (2048, 1536, 4),
                                      (4096, 2048, 1)])
def test_prefill_exact_one_group_per_row(gpu, rows, M, k):
    """Rows of a single group on the 128 x 128 tiles and, at one stage with
    enough tiles, the 32-row waves: the group ring never holds a second
    group."""
    cols = 128
    assert _large_tiles(rows, M)
    _log(f"prefill exact, one group per row rows={rows} M={M} k={k}")
    codes, s, z, xb = _exact(rows, cols, M, rows + M + k)
    y = _run(gpu, codes, s, z, rows, cols, k, xb)
    ref = npo.linear(codes, s, z, rows, cols, G, k, xb)
    bad = np.argwhere(y.astype(np.float64) != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}"


@pytest.mark.parametrize("zp,sd", [("int", "f32"), ("sym", "f16"), ("real", "f32"), ("int", "bf16")])
def test_prefill_exact_wide_tiles(gpu, zp, sd):
    rows, cols, M = WIDE
    assert _wide_tiles(rows, M)
    _log(f"prefill exact, 32-row waves {zp}/{sd} rows={rows} cols={cols} M={M}")
    codes, s, z, xb = _exact(rows, cols, M, 31)
    if zp == "sym":
        zz, zv = None, np.full_like(s, 2.0)
    elif zp == "real":
        zz = (np.random.default_rng(6).integers(0, 13, s.shape) * 0.25).astype(np.float32)
        zv = zz
    else:
        zz = zv = z
    s_raw = (s.astype(np.float16).view(np.uint16) if sd == "f16"
             else (s.view(np.uint32) >> 16).astype(np.uint16) if sd == "bf16" else s)
    y = _run(gpu, codes, s_raw, zz, rows, cols, 1, xb, zp, sd)
    ref = npo.linear(codes, s, zv, rows, cols, G, 1, xb)
    bad = np.argwhere(y.astype(np.float64) != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}"


@pytest.mark.parametrize("rows,M", [(70, 148), (70, 1030), (1990, 1500)])
@pytest.mark.parametrize("zp,sd", [("sym", "f16"), ("real", "f32"), ("int", "bf16")])
def test_prefill_exact_formats(gpu, zp, sd, rows, M):
    cols, k = 2048, 3
    _log(f"prefill exact format {zp}/{sd} rows={rows} M={M}")
    codes, s, z, xb = _exact(rows, cols, M, 99)
    if zp == "sym":
        zz, zv = None, np.full_like(s, 2.0)
    elif zp == "real":
        zz = (np.random.default_rng(5).integers(0, 13, s.shape) * 0.25).astype(np.float32)
        zv = zz
    else:
        zz = zv = z
    s_raw = (s.astype(np.float16).view(np.uint16) if sd == "f16"
             else (s.view(np.uint32) >> 16).astype(np.uint16) if sd == "bf16" else s)
    y = _run(gpu, codes, s_raw, zz, rows, cols, k, xb, zp, sd)
    ref = npo.linear(codes, s, zv, rows, cols, G, k, xb)
    assert np.array_equal(y.astype(np.float64), ref)


def _realistic(rows, cols, seed, zp="int", sd="f32"):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    w = np.where(rng.random(w.size) < 1e-3, w * 20, w).astype(np.float32)
    oc, os_, oz = oracle.c_construct_format(npo.f32_to_bf16_bits(w), G, 4, zp, sd)
    return oc, os_, oz


@pytest.mark.parametrize("rows,cols,M,k", [(300, 4096, 160, 4), (64, 12288, 152, 2),
                                           (129, 1024, 250, 1), (100, 2048, 1056, 3),
                                           (1990, 1024, 1504, 4), (1990, 1024, 1504, 2),
                                           (3000, 384, 2720, 1)])
def test_prefill_equals_16_token_calls(gpu, rows, cols, M, k):
    """The prefill form and the general kernel's 16-token tiles accumulate
    every output in the same order: identical bits on a realistic package.
    The reference calls take 32 tokens at a time (the last one fewer but more
    than 16), a count that only the general kernel serves."""
    _log(f"prefill vs 16-token calls rows={rows} cols={cols} M={M} k={k}")
    oc, os_, oz = _realistic(rows, cols, rows + M)
    rng = np.random.default_rng(M)
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    y = _run(gpu, oc, os_, oz, rows, cols, k, xb)
    assert M % 32 == 0 or M % 32 > 16
    parts = [_run(gpu, oc, os_, oz, rows, cols, k, xb.reshape(M, cols)[m:m + 32].reshape(-1))
             for m in range(0, M, 32)]
    y16 = np.concatenate(parts, axis=0)
    assert np.array_equal(y.view(np.uint32), y16.view(np.uint32))


@pytest.mark.parametrize("zp,sd", [("int", "f32"), ("sym", "f16")])
def test_prefill_realistic_within_bound(gpu, zp, sd):
    rows, cols, M = 192, 4096, 144
    oc, os_, oz = _realistic(rows, cols, 7, zp, sd)
    sv = npo.load_scales(os_, sd)
    zv = np.full_like(sv, 2.0) if zp == "sym" else oz
    rng = np.random.default_rng(8)
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    xa = np.abs(npo.bf16_bits_to_f32(xb).reshape(M, cols).astype(np.float64))
    T = xa.reshape(M, cols // G, G).sum(axis=2)
    for k in (1, 4):
        y = _run(gpu, oc, os_, None if zp == "sym" else oz, rows, cols, k, xb, zp, sd)
        ref = npo.linear(oc, sv, zv, rows, cols, G, k, xb)
        A = sum(T @ (np.abs(sv[t].astype(np.float64)) * (11 + np.abs(zv[t].astype(np.float64))))
                .reshape(rows, cols // G).T for t in range(k))
        p = cols // G
        n = k * (min(p, 4 * math.ceil(p / 16)) + 1)
        tol = 1.05 * U * A * (G + 2 * n + 24) + 1e-300
        err = np.abs(y.astype(np.float64) - ref)
        assert np.all(err <= tol), f"k={k}: {np.max(err / tol)}"
        _log(f"prefill realistic {zp}/{sd} k={k}: max err / bound = {np.max(err / tol):.3g}")


@pytest.mark.parametrize("rows,cols,k", [(4096, 4096, 4), (4096, 4096, 1), (12288, 4096, 4),
                                          (12288, 4096, 1), (4096, 12288, 4), (4096, 12288, 1)])
def test_prefill_full_size_sampled(gpu, rows, cols, k):
    """The benchmark's prefill sizes (2048 tokens on the Qwen3-8B q/o,
    gate/up and down shapes at 1 and 4 stages, the launch configurations the
    bench times) on an exact package: sampled rows,
    every token, bit-exact."""
    M = 2048
    _log(f"prefill full size rows={rows} cols={cols} M={M} k={k}")
    codes, s, z, xb = _exact(rows, cols, M, rows + k)
    y = _run(gpu, codes, s, z, rows, cols, k, xb)
    rng = np.random.default_rng(k)
    idx = np.unique(np.concatenate([np.arange(16), np.arange(rows - 16, rows),
                                    rng.choice(rows, 48, replace=False)]))
    ref = npo.linear(codes, s, z, rows, cols, G, k, xb, row_index=idx)
    got = y[:, idx].astype(np.float64)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}"
    assert not np.any(np.isnan(y)), "unwritten outputs"


@pytest.mark.parametrize("rows,M,k", [(40, 130, 1), (40, 130, 4), (2048, 1536, 4)])
def test_prefill_widest_rows(gpu, rows, M, k):
    """Rows of 65536 inputs, the widest the prefill form takes (512 groups,
    quarters of 128): the small tile with ragged rows and tokens compared in
    full, and the large tile (16 x 12 tiles of 128) on sampled rows, every
    token; exact packages, bit-exact."""
    cols = 65536
    _log(f"prefill widest rows rows={rows} cols={cols} M={M} k={k}")
    codes, s, z, xb = _exact(rows, cols, M, rows + M + k)
    y = _run(gpu, codes, s, z, rows, cols, k, xb)
    if rows <= 64:
        idx = np.arange(rows)
    else:
        rng = np.random.default_rng(k)
        idx = np.unique(np.concatenate([np.arange(16), np.arange(rows - 16, rows),
                                        rng.choice(rows, 16, replace=False)]))
    ref = npo.linear(codes, s, z, rows, cols, G, k, xb, row_index=idx)
    assert np.all(np.abs(ref) < 2.0 ** 20)
    got = y[:, idx].astype(np.float64)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}"
    assert not np.any(np.isnan(y)), "unwritten outputs"

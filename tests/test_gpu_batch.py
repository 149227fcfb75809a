"""GPU parity of rrq_linear's batch form (groups of 128, 5 to 16 tokens, 2048
to 4096 cols, from 3072 to 12288 rows of 4096-input equivalents by stage and
token count), through the C ABI, against the oracle's Eq. 20 product in
float64:

* exact: power-of-two scales, integer or dyadic zero-points and
  small-integer activations make every intermediate exactly representable,
  so the outputs must equal the exact value bit for bit (ragged last row
  tiles, 16 to 32 groups per row, so waves with part of a set of groups or
  none, fewer tiles than workgroups and several per workgroup, token counts
  5 to 16, every stage count and format);
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


@pytest.mark.parametrize("rows,cols,M,k", [
    (12288, 4096, 16, 4), (12288, 4096, 5, 2), (6150, 4096, 13, 3), (10000, 2560, 16, 2),
    (12295, 2048, 7, 3), (24576, 4096, 16, 1), (24583, 3072, 11, 4),
    # the smallest packages the form takes, fewer tiles than workgroups
    (3072, 4096, 16, 4), (3100, 4096, 16, 4), (4099, 4096, 6, 2), (6147, 4096, 8, 1),
    # a wave with part of a set of 4 groups (25 and 17 groups per row)
    (9000, 3200, 9, 4), (12290, 2176, 12, 3),
])
def test_batch_exact(gpu, rows, cols, M, k):
    _log(f"batch exact rows={rows} cols={cols} M={M} k={k}")
    codes, s, z, xb = _exact(rows, cols, M, rows + cols + M)
    y = _run(gpu, codes, s, z, rows, cols, k, xb)
    if rows * cols > (1 << 22):
        rng = np.random.default_rng(rows)
        idx = np.unique(np.concatenate([np.arange(16), np.arange(rows - 16, rows),
                                        rng.choice(rows, 200, replace=False)]))
    else:
        idx = np.arange(rows)
    ref = npo.linear(codes, s, z, rows, cols, G, k, xb, row_index=idx)
    assert np.all(np.abs(ref) < 2.0 ** 20)
    got = y[:, idx].astype(np.float64)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}"
    assert not np.any(np.isnan(y)), "unwritten outputs"


@pytest.mark.parametrize("zp,sd", [("sym", "f16"), ("real", "f32"), ("int", "bf16")])
def test_batch_exact_formats(gpu, zp, sd):
    rows, cols, M, k = 6160, 4096, 11, 3
    _log(f"batch exact format {zp}/{sd}")
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
    y = _run(gpu, codes, s_raw, zz, rows, cols, k, xb, zp, sd)
    ref = npo.linear(codes, s, zv, rows, cols, G, k, xb)
    assert np.array_equal(y.astype(np.float64), ref)


@pytest.mark.parametrize("zp,sd", [("int", "f32"), ("sym", "f16"), ("real", "f32")])
def test_batch_realistic_within_bound(gpu, zp, sd):
    rows, cols, M = 12288, 2048, 8
    rng = np.random.default_rng(12)
    w = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    w = np.where(rng.random(w.size) < 1e-3, w * 20, w).astype(np.float32)
    oc, os_, oz = oracle.c_construct_format(npo.f32_to_bf16_bits(w), G, 4, zp, sd)
    sv = npo.load_scales(os_, sd)
    zv = np.full_like(sv, 2.0) if zp == "sym" else oz
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    xa = np.abs(npo.bf16_bits_to_f32(xb).reshape(M, cols).astype(np.float64))
    T = xa.reshape(M, cols // G, G).sum(axis=2)
    idx = np.unique(np.concatenate([np.arange(32), np.arange(rows - 32, rows),
                                    rng.choice(rows, 512, replace=False)]))
    for k in (1, 2, 4):
        y = _run(gpu, oc, os_, None if zp == "sym" else oz, rows, cols, k, xb, zp, sd)
        ref = npo.linear(oc, sv, zv, rows, cols, G, k, xb, row_index=idx)
        A = sum(T @ (np.abs(sv[t].astype(np.float64)) * (11 + np.abs(zv[t].astype(np.float64))))
                .reshape(rows, cols // G)[idx].T for t in range(k))
        p = cols // G
        n = k * (min(p, 4 * math.ceil(p / 16)) + 1)
        tol = 1.05 * U * A * (G + 2 * n + 24) + 1e-300
        err = np.abs(y[:, idx].astype(np.float64) - ref)
        assert np.all(err <= tol), f"k={k}: {np.max(err / tol)}"
        _log(f"batch realistic {zp}/{sd} k={k}: max err / bound = {np.max(err / tol):.3g}")

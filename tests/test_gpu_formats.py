"""GPU parity of the stage formats (symmetric stages, real-valued
zero-points, 16-bit scales) through the C ABI's *_format calls, against the
C oracle: construction bit-exact (codes, stored scale bits, zero-points),
reconstruction bit-exact, construction on a base in the same format, and the
linear layer within its stated bound."""

import itertools
import math
import sys

import numpy as np
import pytest

import oracle
from oracle import rrq_oracle as npo
from paper_2608_04048_amd import workloads as wl

pytestmark = pytest.mark.gpu
FORMATS = list(itertools.product(("int", "real", "sym"), ("f32", "f16", "bf16")))
U = 2.0 ** -24


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bits(seed, n, scale=0.02):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(n).astype(np.float32) * scale
    x = np.where(rng.random(n) < 1e-3, x * 20, x).astype(np.float32)
    return npo.f32_to_bf16_bits(x)


def _raw(t):
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
    return t.numpy().view(np.uint8).reshape(-1)


def _to_gpu(a):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    elif a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a.copy()).cuda()


def _check(rrq, bits, rows, cols, G, S, zp, sd, tag, ks=None):
    import torch
    _log(f"case {tag}: rows={rows} cols={cols} G={G} S={S} format={zp}/{sd}")
    W = torch.from_numpy(bits.view(np.int16).reshape(rows, cols)).cuda().view(torch.bfloat16)
    codes, scales, zeros = rrq.construct_format(W, G, S, zp, sd)
    torch.cuda.synchronize()
    oc, os_, oz = oracle.c_construct_format(bits, G, S, zp, sd)
    assert np.array_equal(_raw(codes), oc.view(np.uint8).reshape(-1)), f"{tag}: codes"
    assert np.array_equal(_raw(scales), os_.view(np.uint8).reshape(-1)), f"{tag}: scales"
    if zp != "sym":
        assert np.array_equal(_raw(zeros), oz.view(np.uint8).reshape(-1)), f"{tag}: zeros"
    else:
        assert zeros is None
    for k in (ks or range(1, S + 1)):
        for dt, tdt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
            got = rrq.reconstruct_format(codes, scales, zeros, rows, cols, G, k, zp, sd, tdt)
            torch.cuda.synchronize()
            want = oracle.c_reconstruct_format(oc, os_, oz, G, k, zp, sd, dt)
            assert np.array_equal(_raw(got), want.view(np.uint8)), f"{tag}: recon k={k} {dt}"
    return oc, os_, oz


@pytest.mark.parametrize("zp,sd", FORMATS)
@pytest.mark.parametrize("rows,cols,G", [(7, 192, 64), (13, 128 * 11, 128), (2, 32 * 129, 32),
                                         (300, 1024, 128)])
def test_construct_and_reconstruct(gpu, zp, sd, rows, cols, G):
    _check(gpu, _bits(rows + cols + G, rows * cols), rows, cols, G, 4, zp, sd, "shape")


@pytest.mark.parametrize("zp,sd", FORMATS)
def test_two_stages_and_tiny_weights(gpu, zp, sd):
    """Weights of ~1e-6: 16-bit scales become subnormal or underflow to zero
    (degenerate stages); two stages only."""
    bits = _bits(5, 64 * 1024, scale=2e-6)
    _check(gpu, bits, 64, 1024, 128, 2, zp, sd, "tiny")
    bits = _bits(6, 64 * 1024, scale=2e-8)
    _check(gpu, bits, 64, 1024, 64, 4, zp, sd, "tinier")


@pytest.mark.parametrize("zp", ["int", "real", "sym"])
def test_zero_and_constant_groups(gpu, zp):
    x = np.zeros((8, 128), dtype=np.float32)
    x[1] = 0.5
    x[2] = -3.0
    x[3, ::2] = 1.0
    x[4, 0] = -1e-30
    bits = npo.f32_to_bf16_bits(x.reshape(-1))
    _check(gpu, bits, 8, 128, 128, 4, zp, "f16", "special")
    _check(gpu, bits, 8, 128, 32, 4, zp, "f32", "special")


@pytest.mark.parametrize("zp,sd", FORMATS)
def test_from_base_in_format(gpu, zp, sd):
    """The oracle's own stage 0 in the format as the base: the GPU result is
    the oracle's direct package."""
    import torch
    rows, cols, G, S = 33, 1024, 128, 4
    bits = _bits(40, rows * cols)
    full = oracle.c_construct_format(bits, G, S, zp, sd)
    W = torch.from_numpy(bits.view(np.int16).reshape(rows, cols)).cuda().view(torch.bfloat16)
    codes = _to_gpu(np.concatenate([full[0][:1], np.zeros_like(full[0][1:])]))
    scales = _to_gpu(np.concatenate([full[1][:1], np.zeros_like(full[1][1:])]))
    zeros = None if zp == "sym" else _to_gpu(np.concatenate([full[2][:1], np.zeros_like(full[2][1:])]))
    gpu.rrq_construct_from_base_format(W, rows, cols, G, S, gpu.ZERO_POINTS[zp],
                                       gpu.SCALE_TYPES[sd], codes, scales, zeros)
    torch.cuda.synchronize()
    assert np.array_equal(_raw(codes), full[0].view(np.uint8).reshape(-1))
    assert np.array_equal(_raw(scales), full[1].view(np.uint8).reshape(-1))
    if zeros is not None:
        assert np.array_equal(_raw(zeros), full[2].view(np.uint8).reshape(-1))


@pytest.mark.parametrize("zp,sd", FORMATS)
def test_linear_in_format(gpu, zp, sd):
    import torch
    rows, cols, G, M = 96, 2048, 128, 5
    bits = _bits(50, rows * cols)
    oc, os_, oz = oracle.c_construct_format(bits, G, 4, zp, sd)
    sv = npo.load_scales(os_, sd)                      # binary32 values of the scales
    rng = np.random.default_rng(51)
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    X = torch.from_numpy(xb.view(np.int16).reshape(M, cols)).cuda().view(torch.bfloat16)
    Y = torch.empty((M, rows), dtype=torch.float32, device="cuda")
    xa = np.abs(npo.bf16_bits_to_f32(xb).reshape(M, cols).astype(np.float64))
    T = xa.reshape(M, cols // G, G).sum(axis=2)
    for k in (1, 2, 4):
        gpu.rrq_linear_format(_to_gpu(oc), _to_gpu(os_), None if zp == "sym" else _to_gpu(oz),
                              rows, cols, G, 4, gpu.ZERO_POINTS[zp], gpu.SCALE_TYPES[sd], k, X, M,
                              Y)
        torch.cuda.synchronize()
        ref = npo.linear(oc, sv, oz, rows, cols, G, k, xb)
        A = sum(T @ (np.abs(sv[t].astype(np.float64)) * (11 + np.abs(oz[t].astype(np.float64)))).reshape(rows, cols // G).T
                for t in range(k))
        p = cols // G
        n = k * (min(p, 4 * math.ceil(p / 16)) + 1)
        tol = 1.05 * U * A * (G + 2 * n + 24) + 1e-300
        err = np.abs(Y.cpu().numpy().astype(np.float64) - ref)
        assert np.all(err <= tol), f"k={k}: {np.max(err / tol)}"


@pytest.mark.parametrize("zp,sd", [("sym", "f16"), ("real", "f32"), ("int", "bf16")])
def test_qwen3_layer_full_in_format(gpu, zp, sd):
    """One Qwen3-8B-shaped layer as one flat call; the paper's symmetric
    configuration with 16-bit scales among them."""
    import torch
    w = wl.workload("qwen3_8b_layer")
    W = wl.materialize(w)
    bits = W.cpu().view(torch.int16).numpy().view(np.uint16)
    _check(gpu, bits, w.numel // 4096, 4096, 128, 4, zp, sd, "qwen3_8b_layer", ks=(2, 4))
    del W
    torch.cuda.empty_cache()

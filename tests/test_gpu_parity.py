"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Every comparison is bit-exact: codes, scales and zeros of the package; the
binary32 reconstruction (0 ulp); the bfloat16 reconstruction (0 ulp, the bar
allows 1). The oracle always starts from the same input bits as the GPU and
builds its own package; reconstruction is compared oracle-package vs
GPU-package, never fed from the GPU.
"""

import json
import os
import sys

import numpy as np
import pytest

import oracle
from oracle import rrq_oracle as npo
from paper_2608_04048_amd import workloads as wl

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _u32(t):
    """torch tensor -> numpy uint32 view of its bytes."""
    return t.detach().cpu().contiguous().numpy().view(np.uint32)


def _gpu_package(rrq, W, rows, cols, G, S):
    import torch
    codes, scales, zeros = rrq.construct(W.view(rows, cols), G, S)
    torch.cuda.synchronize()
    return codes, scales, zeros


def _check_case(rrq, w_bits_np, rows, cols, G, S, ks=None, tag=""):
    """Full parity of one matrix given as host bfloat16 bits."""
    import torch
    _log(f"case {tag}: rows={rows} cols={cols} G={G} S={S}")
    W = torch.from_numpy(w_bits_np.view(np.int16).reshape(rows, cols)).cuda().view(torch.bfloat16)
    codes, scales, zeros = _gpu_package(rrq, W, rows, cols, G, S)
    oc, os_, oz = oracle.c_construct(w_bits_np, G, S)
    assert np.array_equal(_u32(codes), oc), f"{tag}: codes differ at {np.argwhere(_u32(codes) != oc)[:5]}"
    assert np.array_equal(_u32(scales), os_.view(np.uint32)), f"{tag}: scales differ"
    assert np.array_equal(_u32(zeros), oz.view(np.uint32)), f"{tag}: zeros differ"
    for k in (ks or range(1, S + 1)):
        for dt, torch_dt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
            got = rrq.reconstruct(codes, scales, zeros, rows, cols, G, k, torch_dt)
            torch.cuda.synchronize()
            want = oracle.c_reconstruct(oc, os_, oz, G, k, dt)
            got_np = got.cpu().contiguous().view(torch.int32 if dt == "f32" else torch.int16).numpy()
            assert np.array_equal(got_np.reshape(-1).view(want.dtype), want), f"{tag}: recon k={k} {dt}"


def _random_bits(seed, n, scale=0.02, outliers=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(n).astype(np.float32) * scale
    if outliers:
        x = np.where(rng.random(n) < 1e-3, x * 20, x).astype(np.float32)
    return npo.f32_to_bf16_bits(x)


# ---------------------------------------------------------------------------
# Small and ragged shapes
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("rows,cols,G", [
    (1, 32, 32), (3, 96, 32), (7, 192, 64), (5, 640, 128), (1, 128 * 65, 128),
    (13, 128 * 11, 128), (64, 64 * 64, 64), (2, 32 * 129, 32), (1024, 1024, 128),
])
@pytest.mark.parametrize("S", [1, 2, 4])
def test_shapes_and_tails(gpu, rows, cols, G, S):
    bits = _random_bits(rows * 7919 + cols + G, rows * cols)
    _check_case(gpu, bits, rows, cols, G, S, tag=f"shape{rows}x{cols}")


@pytest.mark.parametrize("G", [32, 64, 128])
def test_three_stages(gpu, G):
    bits = _random_bits(33 + G, 37 * 1024)
    _check_case(gpu, bits, 37, 1024, G, 3, tag="S3")


def test_golden_cases_on_gpu(gpu):
    """The hand-derived cases, through the GPU."""
    cases = json.load(open(os.path.join(HERE, "golden", "hand_cases.json")))["construct"]
    for case in cases:
        x = np.array([int(h, 16) for h in case["x"]], dtype=np.uint32)
        bits = (x >> 16).astype(np.uint16)
        _check_case(gpu, bits, 1, bits.size, case["G"], 4, tag=case["name"])


def test_matrix_1024(gpu):
    import torch
    w = wl.workload("matrix_1024")
    W = wl.materialize(w)
    bits = W.cpu().view(torch.int16).numpy().view(np.uint16)
    _check_case(gpu, bits, 1024, 1024, 128, 4, tag="matrix_1024")


# ---------------------------------------------------------------------------
# Edge values
# ---------------------------------------------------------------------------

def test_constant_groups_every_bf16(gpu):
    b = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    f = npo.bf16_bits_to_f32(b)
    b = b[np.isfinite(f)]
    b = b[: (b.size // 4) * 4]
    bits = np.repeat(b, 32)
    _check_case(gpu, bits, bits.size // 128, 128, 32, 4, tag="constants")


def test_zeros_signed_zeros_subnormals_and_extremes(gpu):
    n = 128 * 64
    rng = np.random.default_rng(5)
    bits = np.zeros(n, dtype=np.uint16)
    bits[n // 8: n // 4] = 0x8000                                      # -0
    bits[n // 4: n // 2] = rng.integers(1, 0x80, n // 4).astype(np.uint16)       # subnormal +
    bits[n // 2: 5 * n // 8] = 0x8000 | rng.integers(1, 0x80, n // 8).astype(np.uint16)
    # extremes: largest magnitudes inside the precondition (|x| < 2^127) of
    # both signs, smallest normals
    bits[5 * n // 8: 3 * n // 4] = rng.choice([0x7E7F, 0xFE7F, 0x0080, 0x8080], n // 8)
    # one-signed groups may go up to the bfloat16 maximum
    bits[5 * n // 8: 5 * n // 8 + 128] = rng.choice([0x7F7F, 0x7F00, 0x0000], 128)
    tail = rng.integers(0, 65536, n // 4).astype(np.uint16)             # any value with
    tail = np.where(((tail >> 7) & 0xFF) >= 0xFE, 0, tail).astype(np.uint16)  # |x| < 2^127
    bits[3 * n // 4:] = tail
    for G in (32, 64, 128):
        _check_case(gpu, bits, n // 1024, 1024, G, 4, tag=f"edges_G{G}")


def test_clamp_paths(gpu):
    """Groups whose top element rounds to code 4 before the clamp: the
    hand case of the golden file repeated, mixed with ordinary groups so that
    clamped and unclamped groups share waves."""
    rng = np.random.default_rng(9)
    base = np.array([3, 0, 0.25, 1.25, 0.5, 1.5, 2.5, 1.75] + [0] * 24, dtype=np.float32)
    groups = []
    for i in range(64 * 9):
        if i % 5 == 0:
            groups.append(base * np.float32(2.0 ** rng.integers(-10, 10)))
        else:
            groups.append(rng.standard_normal(32).astype(np.float32))
    bits = npo.f32_to_bf16_bits(np.concatenate(groups))
    _check_case(gpu, bits, 64 * 9 // 4, 128, 32, 4, tag="clamp")
    # the same values as G=128 groups
    _check_case(gpu, bits, 64 * 9 // 4, 128, 128, 4, tag="clamp128")


# ---------------------------------------------------------------------------
# Workloads at full size
# ---------------------------------------------------------------------------

def test_qwen3_layer_full(gpu):
    """One Qwen3-8B-shaped layer (7 projections, 0.1% x20 outliers), every
    output compared, as one flat call."""
    import torch
    w = wl.workload("qwen3_8b_layer")
    W = wl.materialize(w)
    bits = W.cpu().view(torch.int16).numpy().view(np.uint16)
    _check_case(gpu, bits, w.numel // 4096, 4096, 128, 4, tag="qwen3_8b_layer")
    del W
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", wl.SWEEP)
def test_distribution_sweep(gpu, name):
    import torch
    w = wl.workload(name)
    W = wl.materialize(w)
    bits = W.cpu().view(torch.int16).numpy().view(np.uint16)
    _check_case(gpu, bits, 12288, 4096, w.group_size, 4, ks=(1, 4), tag=name)


def test_flat_call_equals_per_tensor_calls(gpu):
    """Groups never span rows, so a stack passed as one flat call gives the
    same package as one call per tensor."""
    import torch
    w = wl.workload("qwen3_8b_layer")
    W = wl.materialize(w)
    codes, scales, zeros = gpu.construct(W.view(-1, 4096), 128, 4)
    for t in w.tensors:
        c2, s2, z2 = gpu.construct(W[t.offset:t.offset + t.numel].view(t.rows, t.cols), 128, 4)
        torch.cuda.synchronize()
        a, b = t.offset // 16, (t.offset + t.numel) // 16
        assert torch.equal(codes[:, a:b], c2)
        a, b = t.offset // 128, (t.offset + t.numel) // 128
        assert torch.equal(scales[:, a:b], s2) and torch.equal(zeros[:, a:b], z2)
    again = gpu.construct(W.view(-1, 4096), 128, 4)
    torch.cuda.synchronize()
    assert all(torch.equal(x, y) for x, y in zip((codes, scales, zeros), again))


def _sampled_stack_check(gpu, name, n_sample=4096):
    """A full-size stack in one flat call (the benchmark's launch shape);
    outputs of sampled groups against the oracle run on those groups."""
    import torch
    w = wl.workload(name)
    G, S = w.group_size, w.n_stages
    _log(f"materialize {name}: {w.numel} elements")
    W = wl.materialize(w)
    rows = w.numel // 4096
    codes, scales, zeros = gpu.construct(W.view(rows, 4096), G, S)
    torch.cuda.synchronize()
    ng = w.n_groups
    rng = np.random.default_rng(17)
    idx = np.unique(np.concatenate([
        rng.integers(0, ng, n_sample), np.arange(64), np.arange(ng - 64, ng),
        [t.offset // G for t in w.tensors], [(t.offset + t.numel) // G - 1 for t in w.tensors]]))
    idx_t = torch.from_numpy(idx).cuda()
    wg = W.view(ng, G)[idx_t].cpu().view(torch.int16).numpy().view(np.uint16).reshape(-1)
    oc, os_, oz = oracle.c_construct(wg, G, S)
    gc = codes.view(S, ng, G // 16)[:, idx_t].cpu().numpy().view(np.uint32).reshape(S, -1)
    assert np.array_equal(gc, oc)
    assert np.array_equal(_u32(scales[:, idx_t]), os_.view(np.uint32))
    assert np.array_equal(_u32(zeros[:, idx_t]), oz.view(np.uint32))
    for k in w.recon_k:
        out = gpu.reconstruct(codes, scales, zeros, rows, 4096, G, k, torch.bfloat16)
        torch.cuda.synchronize()
        got = out.view(ng, G)[idx_t].cpu().view(torch.int16).numpy().view(np.uint16).reshape(-1)
        assert np.array_equal(got, oracle.c_reconstruct(oc, os_, oz, G, k, "bf16")), f"k={k}"
        del out
    del W, codes, scales, zeros
    torch.cuda.empty_cache()


def test_qwen3_8b_stack36_sampled(gpu):
    _sampled_stack_check(gpu, "qwen3_8b_stack36")


def test_dense32b_stack64_sampled(gpu):
    _sampled_stack_check(gpu, "dense32b_stack64")


# ---------------------------------------------------------------------------
# Reconstruction of given packages
# ---------------------------------------------------------------------------

def test_reconstruct_golden_packages(gpu):
    import torch
    cases = json.load(open(os.path.join(HERE, "golden", "hand_cases.json")))["reconstruct"]
    for case in cases:
        G = case["G"]
        codes = np.array([[int(h, 16) for h in row] for row in case["codes"]], dtype=np.uint32)
        sc = np.array([int(h, 16) for h in case["scales"]], dtype=np.uint32).view(np.float32).reshape(-1, 1)
        ze = np.array([int(h, 16) for h in case["zeros"]], dtype=np.uint32).view(np.float32).reshape(-1, 1)
        S = codes.shape[0]
        tc = torch.from_numpy(codes.view(np.int32)).cuda()
        ts, tz = torch.from_numpy(sc).cuda(), torch.from_numpy(ze).cuda()
        for k in range(1, S + 1):
            for dt, tdt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
                got = gpu.reconstruct(tc, ts, tz, 1, codes.shape[1] * 16, G, k, tdt)
                torch.cuda.synchronize()
                want = oracle.c_reconstruct(codes, sc, ze, G, k, dt)
                gb = got.cpu().view(torch.int32 if dt == "f32" else torch.int16).numpy().reshape(-1)
                assert np.array_equal(gb.view(want.dtype), want), (case["name"], k, dt)


def test_reconstruct_random_packages(gpu):
    """Packages drawn at random (any codes, integer zero-points, scales over
    many binades, some degenerate), not produced by construction."""
    import torch
    rng = np.random.default_rng(23)
    for G, S, rows, cols in ((32, 4, 9, 96), (64, 3, 5, 640), (128, 4, 33, 1280)):
        n = rows * cols
        codes = rng.integers(0, 2 ** 32, (S, n // 16), dtype=np.uint64).astype(np.uint32)
        sc = (2.0 ** rng.uniform(-30, 10, (S, n // G))).astype(np.float32)
        sc[:, ::7] = 0
        ze = rng.integers(0, 4, (S, n // G)).astype(np.float32)
        ze[sc == 0] = 0
        tc = torch.from_numpy(codes.view(np.int32)).cuda()
        ts, tz = torch.from_numpy(sc).cuda(), torch.from_numpy(ze).cuda()
        for k in range(1, S + 1):
            for dt, tdt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
                got = gpu.reconstruct(tc, ts, tz, rows, cols, G, k, tdt)
                torch.cuda.synchronize()
                want = oracle.c_reconstruct(codes, sc, ze, G, k, dt)
                gb = got.cpu().view(torch.int32 if dt == "f32" else torch.int16).numpy().reshape(-1)
                assert np.array_equal(gb.view(want.dtype), want), (G, S, k, dt)


def test_stream_argument(gpu):
    """Work is enqueued on the stream passed in."""
    import torch
    bits = _random_bits(77, 64 * 1024)
    W = torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16).view(64, 1024)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        codes, scales, zeros = gpu.construct(W, 128, 4)
    s.synchronize()
    oc, os_, oz = oracle.c_construct(bits, 128, 4)
    assert np.array_equal(_u32(codes), oc)

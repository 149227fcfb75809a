"""GPU parity of the stage-sum linear layer (rrq_linear, through the C ABI)
against the oracle's Eq. 20 product in float64.

Two bars:
* exact: on packages with power-of-two scales and integer zero-points and
  small-integer activations every intermediate of the kernel is exactly
  representable, so Y must equal the exact value bit for bit (this pins the
  indexing of every code, group, stage, row and token);
* bounded: on realistic packages (built by the oracle) and Gaussian
  activations, |Y - exact| stays within the bound stated in include/rrq.h.
Packages always come from the oracle or a seeded generator, never from the GPU.
"""

import math
import sys

import numpy as np
import pytest

import oracle
from oracle import rrq_oracle as npo
from paper_2608_04048_amd import workloads as wl

pytestmark = pytest.mark.gpu
U = 2.0 ** -24


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bound(codes, s, z, rows, cols, G, k, x_bits):
    """The bound of include/rrq.h for every output [M, rows]."""
    x = np.abs(npo.bf16_bits_to_f32(x_bits).reshape(-1, cols).astype(np.float64))
    T = x.reshape(x.shape[0], cols // G, G).sum(axis=2)                 # [M, gpr]
    A = np.zeros((x.shape[0], rows))
    for t in range(k):
        w = (np.abs(s[t].astype(np.float64)) * (11 + np.abs(z[t].astype(np.float64)))).reshape(rows, cols // G)
        A += T @ w.T
    p = cols // G
    n = k * (min(p, 4 * math.ceil(p / 16)) + 1)
    return 1.05 * U * A * (G + 2 * n + 24) + 1e-300


def _gpu_linear(rrq, codes, s, z, rows, cols, G, k, x_bits):
    import torch
    S = codes.shape[0]
    c = torch.from_numpy(codes.view(np.int32).copy()).cuda()
    sc = torch.from_numpy(s.copy()).cuda()
    ze = torch.from_numpy(z.copy()).cuda()
    X = torch.from_numpy(x_bits.view(np.int16).reshape(-1, cols).copy()).cuda().view(torch.bfloat16)
    Y = rrq.linear(X, c, sc, ze, rows, cols, G, k)
    torch.cuda.synchronize()
    assert Y.shape == (X.shape[0], rows) and S == c.shape[0]
    return Y.cpu().numpy()


def _exact_case(rows, cols, G, S, M, seed):
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 2 ** 32, (S, rows * cols // 16), dtype=np.uint64).astype(np.uint32)
    s = (2.0 ** rng.integers(-4, -1, (S, rows * cols // G))).astype(np.float32)
    z = rng.integers(0, 4, (S, rows * cols // G)).astype(np.float32)
    x = rng.integers(-4, 5, (M, cols)).astype(np.float32)
    return codes, s, z, npo.f32_to_bf16_bits(x)


@pytest.mark.parametrize("rows,cols,G,M", [
    (16, 128, 128, 1), (5, 256, 64, 3), (37, 1024, 128, 16), (64, 4096, 128, 1),
    (23, 96, 32, 17), (100, 2048, 32, 5), (8, 4096, 64, 33), (1, 32, 32, 2),
])
@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_exact_packages_bit_exact(gpu, rows, cols, G, M, k):
    _log(f"exact rows={rows} cols={cols} G={G} M={M} k={k}")
    codes, s, z, xb = _exact_case(rows, cols, G, 4, M, rows * 7 + cols + G + M)
    y = _gpu_linear(gpu, codes, s, z, rows, cols, G, k, xb)
    ref = npo.linear(codes, s, z, rows, cols, G, k, xb)
    assert np.all(np.abs(ref) < 2.0 ** 20)
    bad = np.argwhere(y.astype(np.float64) != ref)
    assert bad.size == 0, f"{len(bad)} outputs differ, first {bad[:3]}: {y[tuple(bad[0])]} vs {ref[tuple(bad[0])]}"


def _realistic(rows, cols, G, S, seed):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    w = np.where(rng.random(w.size) < 1e-3, w * 20, w).astype(np.float32)
    bits = npo.f32_to_bf16_bits(w)
    codes, s, z = oracle.c_construct(bits, G, S)
    return codes, s, z


@pytest.mark.parametrize("rows,cols,G,M", [(256, 4096, 128, 1), (300, 2048, 64, 16), (96, 1024, 32, 7),
                                          (1024, 4096, 128, 4)])
def test_realistic_packages_within_bound(gpu, rows, cols, G, M):
    codes, s, z = _realistic(rows, cols, G, 4, rows + cols + G)
    rng = np.random.default_rng(M)
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    worst = 0.0
    for k in range(1, 5):
        y = _gpu_linear(gpu, codes, s, z, rows, cols, G, k, xb)
        ref = npo.linear(codes, s, z, rows, cols, G, k, xb)
        tol = _bound(codes, s, z, rows, cols, G, k, xb)
        err = np.abs(y.astype(np.float64) - ref)
        assert np.all(err <= tol), f"k={k}: max err/tol {np.max(err / tol)}"
        worst = max(worst, float(np.max(err / tol)))
    _log(f"realistic rows={rows} cols={cols} G={G} M={M}: max err / bound = {worst:.3g}")


def test_foreign_base_package_within_bound(gpu):
    """A package on a foreign base (real-valued zero-points in stage 0)."""
    rows, cols, G, M = 128, 2048, 128, 3
    rng = np.random.default_rng(5)
    w = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    bits = npo.f32_to_bf16_bits(w)
    bc, bs, bz = wl.draw_base(rows * cols, G, 6, device="cpu")
    codes, s, z = oracle.c_construct_from_base(bits, bc.numpy().view(np.uint32), bs.numpy(),
                                               bz.numpy(), G, 4)
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    for k in range(1, 5):
        y = _gpu_linear(gpu, codes, s, z, rows, cols, G, k, xb)
        ref = npo.linear(codes, s, z, rows, cols, G, k, xb)
        assert np.all(np.abs(y - ref) <= _bound(codes, s, z, rows, cols, G, k, xb)), k


def test_prefix_stages_change_the_result(gpu):
    """Each further stage refines the product toward X W^T (the residual
    stages are not dropped): on realistic data the error to the unquantized
    product falls with k."""
    rows, cols, G, M = 256, 2048, 128, 8
    rng = np.random.default_rng(11)
    w = (rng.standard_normal(rows * cols) * 0.02).astype(np.float32)
    bits = npo.f32_to_bf16_bits(w)
    codes, s, z = oracle.c_construct(bits, G, 4)
    xb = npo.f32_to_bf16_bits(rng.standard_normal((M, cols)).astype(np.float32))
    full = npo.bf16_bits_to_f32(xb).reshape(M, cols).astype(np.float64) @ \
        npo.bf16_bits_to_f32(bits).reshape(rows, cols).astype(np.float64).T
    errs = [np.abs(_gpu_linear(gpu, codes, s, z, rows, cols, G, k, xb) - full).mean() for k in range(1, 5)]
    assert errs[0] > errs[1] > errs[2] > errs[3], errs


def test_qwen3_layer_every_projection(gpu):
    """Every projection of one Qwen3-8B-shaped layer (package built by the C
    oracle), decode (1 token) and a 16-token batch, every prefix, every
    output within the bound."""
    import torch
    w = wl.workload("qwen3_8b_layer")
    Wf = wl.materialize(w)
    rng = np.random.default_rng(3)
    for t in w.tensors:
        bits = Wf[t.offset:t.offset + t.numel].cpu().view(torch.int16).numpy().view(np.uint16)
        codes, s, z = oracle.c_construct(bits, 128, 4)
        for M in (1, 16):
            xb = npo.f32_to_bf16_bits(rng.standard_normal((M, t.cols)).astype(np.float32))
            ref = 0
            for k in range(1, 5):
                ref = ref + npo.linear(codes[k - 1:k], s[k - 1:k], z[k - 1:k], t.rows, t.cols, 128, 1, xb)
                y = _gpu_linear(gpu, codes, s, z, t.rows, t.cols, 128, k, xb)
                tol = _bound(codes, s, z, t.rows, t.cols, 128, k, xb)
                err = np.abs(y - ref)
                assert np.all(err <= tol), f"{t.name} M={M} k={k}: {np.max(err / tol)}"
        _log(f"{t.name}: ok")
    del Wf
    torch.cuda.empty_cache()


def test_graph_replay_matches_eager(gpu):
    """rrq_linear captured in a HIP graph: every replay (with eager work and
    synchronisations between them) gives the eager result bit for bit."""
    import torch
    rows, cols, G, S = 80, 512, 128, 4
    codes, s, z = _realistic(rows, cols, G, S, 77)
    rng = np.random.default_rng(5)
    xb = npo.f32_to_bf16_bits(rng.standard_normal((3, cols)).astype(np.float32))
    c_d = torch.from_numpy(codes.view(np.int32).copy()).cuda()
    s_d = torch.from_numpy(s.copy()).cuda()
    z_d = torch.from_numpy(z.copy()).cuda()
    X = torch.from_numpy(xb.view(np.int16).reshape(3, cols).copy()).cuda()
    Y_eager = torch.empty((3, rows), dtype=torch.float32, device="cuda")
    gpu.rrq_linear(c_d, s_d, z_d, rows, cols, G, S, 3, X, 3, Y_eager)
    torch.cuda.synchronize()
    Y = torch.full((3, rows), float("nan"), dtype=torch.float32, device="cuda")
    cs = torch.cuda.Stream()
    cs.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cs):
        gpu.rrq_linear(c_d, s_d, z_d, rows, cols, G, S, 3, X, 3, Y, cs)
    torch.cuda.current_stream().wait_stream(cs)
    for i in range(3):
        Y.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y, Y_eager), i
        # eager work between replays
        gpu.rrq_linear(c_d, s_d, z_d, rows, cols, G, S, 1 + i % 3, X, 2, Y_eager[:2])
        gpu.rrq_linear(c_d, s_d, z_d, rows, cols, G, S, 3, X, 3, Y_eager)
        torch.cuda.synchronize()

"""The C ABI's calls captured in HIP graphs, the way the benchmark replays
them: rrq_construct calls spread over several streams (forked from and
joined back to the capture stream) and rrq_linear calls of several forms,
each graph replayed several times with the program's own eager work and
synchronizations between the replays, every replay checked against the
eager calls' results bit for bit (the calls enqueue kernels only: no
memsets, allocations or host synchronization)."""

import sys

import numpy as np
import pytest

from oracle import rrq_oracle as npo

pytestmark = pytest.mark.gpu
G = 128


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bits(seed, n):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(n).astype(np.float32) * 0.02
    x = np.where(rng.random(n) < 1e-3, x * 20, x).astype(np.float32)
    return npo.f32_to_bf16_bits(x)


def test_construct_calls_on_streams_in_a_graph(gpu):
    """Per-tensor construction on 3 streams in one graph: after each of 4
    replays (buffers poisoned before each, an eager construct and a
    synchronization between them) every package equals the eager call's."""
    import torch
    _log("graph: construct calls on 3 streams")
    S = 4
    shapes = [(1024, 4096), (300, 1024), (4096, 1536), (17, 2048), (2048, 4096), (64, 128)]
    Ws = [torch.from_numpy(_bits(50 + i, r * c).view(np.int16)).cuda().view(torch.bfloat16)
          .view(r, c) for i, (r, c) in enumerate(shapes)]

    def alloc(r, c):
        n = r * c
        return (torch.empty((S, n // 16), dtype=torch.int32, device="cuda"),
                torch.empty((S, n // G), dtype=torch.float32, device="cuda"),
                torch.empty((S, n // G), dtype=torch.float32, device="cuda"))

    outs = [alloc(r, c) for r, c in shapes]
    ref = [gpu.construct(W, G, S) for W in Ws]
    torch.cuda.synchronize()

    cap = torch.cuda.Stream()
    side = [torch.cuda.Stream() for _ in range(3)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cap):
        fork = torch.cuda.Event()
        fork.record(cap)
        for sd in side:
            sd.wait_event(fork)
        for i, (W, (c, s, z)) in enumerate(zip(Ws, outs)):
            gpu.rrq_construct(W, W.shape[0], W.shape[1], G, S, c, s, z, side[i % 3])
        for sd in side:
            join = torch.cuda.Event()
            join.record(sd)
            cap.wait_event(join)
    for rep in range(4):
        for c, s, z in outs:
            c.fill_(-1)
            s.fill_(float("nan"))
            z.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, ((c, s, z), (rc, rs, rz)) in enumerate(zip(outs, ref)):
            assert torch.equal(c, rc) and torch.equal(s, rs) and torch.equal(z, rz), \
                f"replay {rep}, tensor {i}"
        # the program's own eager work between replays
        gpu.construct(Ws[rep % len(Ws)], G, S)
        torch.cuda.synchronize()
    del graph


@pytest.mark.parametrize("rows,cols,M,k", [
    (24576, 4096, 1, 4),     # decode form
    (4096, 12288, 1, 2),     # decode form, 12 waves of two sets
    (24576, 4096, 16, 3),    # batch form
    (4096, 12288, 16, 4),    # general kernel
    (4096, 4096, 256, 2),    # prefill form, 64 x 64 tiles
    (4096, 4096, 2048, 4),   # prefill form, 128 x 128 tiles
    (4096, 4096, 2048, 1),   # prefill form, waves of 32 rows
])
def test_linear_calls_in_a_graph(gpu, rows, cols, M, k):
    """rrq_linear on 3 packages captured in one graph: after each of 3
    replays (outputs poisoned before each, eager linear calls between them)
    every output equals the eager call's bit for bit."""
    import torch
    _log(f"graph: linear rows={rows} cols={cols} M={M} k={k}")
    S = 4
    rng = np.random.default_rng(rows + cols + M + k)
    pk = []
    for _ in range(3):
        c = torch.from_numpy(rng.integers(-2 ** 31, 2 ** 31, (S, rows * cols // 16),
                                          dtype=np.int64).astype(np.int32)).cuda()
        s = torch.from_numpy((2.0 ** rng.integers(-8, -3, (S, rows * cols // G)))
                             .astype(np.float32)).cuda()
        z = torch.from_numpy(rng.integers(0, 4, (S, rows * cols // G)).astype(np.float32)).cuda()
        X = torch.from_numpy(npo.f32_to_bf16_bits(rng.standard_normal((M, cols))
                                                   .astype(np.float32)).view(np.int16)
                             ).cuda().view(torch.bfloat16)
        pk.append((c, s, z, X))
    ref = []
    for c, s, z, X in pk:
        Y = torch.empty((M, rows), dtype=torch.float32, device="cuda")
        gpu.rrq_linear(c, s, z, rows, cols, G, S, k, X, M, Y)
        ref.append(Y)
    torch.cuda.synchronize()
    outs = [torch.empty((M, rows), dtype=torch.float32, device="cuda") for _ in pk]
    cap = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cap):
        for (c, s, z, X), Y in zip(pk, outs):
            gpu.rrq_linear(c, s, z, rows, cols, G, S, k, X, M, Y, cap)
    for rep in range(3):
        for Y in outs:
            Y.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (Y, R) in enumerate(zip(outs, ref)):
            assert torch.equal(Y, R), f"replay {rep}, package {i}"
        c, s, z, X = pk[rep]
        Ye = torch.empty((M, rows), dtype=torch.float32, device="cuda")
        gpu.rrq_linear(c, s, z, rows, cols, G, S, k, X, M, Ye)
        torch.cuda.synchronize()
    del graph

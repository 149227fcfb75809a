"""GPU parity of rrq_construct_many (several tensors, each into its own
package, in as few launches as the call takes) through the C ABI: every
package bit-identical to rrq_construct of that tensor alone, and to the CPU
oracle (Alg. 1, Eq. 1-7); lists of up to 252 tensors (several launches of 64),
ragged and tiny tensors among large ones, every group size, separate
allocations per tensor."""

import sys

import numpy as np
import pytest

import oracle
from oracle import rrq_oracle as npo
from paper_2608_04048_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bits(seed, n):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(n).astype(np.float32) * 0.02
    x = np.where(rng.random(n) < 1e-3, x * 20, x).astype(np.float32)
    return npo.f32_to_bf16_bits(x)


def _alloc(rows, cols, G, S):
    import torch
    n = rows * cols
    return (torch.full((S, n // 16), -1, dtype=torch.int32, device="cuda"),
            torch.full((S, n // G), float("nan"), dtype=torch.float32, device="cuda"),
            torch.full((S, n // G), float("nan"), dtype=torch.float32, device="cuda"))


def _run_many(gpu, shapes, G, S, seed, oracle_every=1):
    import torch
    Ws, outs = [], []
    for i, (rows, cols) in enumerate(shapes):
        Ws.append(torch.from_numpy(_bits(seed + i, rows * cols).view(np.int16))
                  .cuda().view(torch.bfloat16).view(rows, cols))
        outs.append(_alloc(rows, cols, G, S))
    gpu.rrq_construct_many([(W, W.shape[0], W.shape[1], *o) for W, o in zip(Ws, outs)], G, S)
    torch.cuda.synchronize()
    for i, (W, (c, s, z)) in enumerate(zip(Ws, outs)):
        c1, s1, z1 = gpu.construct(W, G, S)
        torch.cuda.synchronize()
        assert torch.equal(c, c1) and torch.equal(s, s1) and torch.equal(z, z1), f"tensor {i}"
        if i % oracle_every == 0:
            bits = W.view(-1).cpu().view(torch.int16).numpy().view(np.uint16)
            oc, os_, oz = oracle.c_construct(bits, G, S)
            assert np.array_equal(c.cpu().numpy().view(np.uint32), oc), f"tensor {i} codes"
            assert np.array_equal(s.cpu().numpy().view(np.uint32), os_.view(np.uint32))
            assert np.array_equal(z.cpu().numpy().view(np.uint32), oz.view(np.uint32))


@pytest.mark.parametrize("G", [32, 64, 128])
def test_mixed_shapes(gpu, G):
    """Tiny, ragged and medium tensors in one call (small total: groups split
    over lanes where the group size allows)."""
    _log(f"construct_many mixed G={G}")
    shapes = [(1, G), (3, 5 * G), (7, 11 * G), (1024, 1024), (33, 64 * G + 0), (1, 65 * G),
              (4096, 512), (5, G)]
    _run_many(gpu, shapes, G, 4, 100 + G)


@pytest.mark.parametrize("S", [1, 2, 3])
def test_stage_counts(gpu, S):
    _log(f"construct_many S={S}")
    _run_many(gpu, [(64, 1024), (7, 384), (300, 2048)], 128, S, 200 + S)


def test_more_than_one_launch(gpu):
    """70 tensors: one launch of 64, one of 6."""
    _log("construct_many 70 tensors")
    rng = np.random.default_rng(3)
    shapes = [(int(rng.integers(1, 40)), 128 * int(rng.integers(1, 24))) for _ in range(70)]
    _run_many(gpu, shapes, 128, 4, 300, oracle_every=7)


def test_layer_stack_one_call_equals_flat(gpu):
    """The 252 tensors of the 36-layer Qwen3-8B-shaped stack, each in its own
    package views of one flat buffer, in one call (4 launches of at most 64
    tensors, one lane per group): identical to the flat call over the stack."""
    import torch
    w = wl.workload("qwen3_8b_stack36")
    G, S, n = w.group_size, w.n_stages, w.numel
    _log(f"materialize {w.name}")
    W = wl.materialize(w)
    codes, scales, zeros = gpu.construct(W.view(-1, 4096), G, S)
    c2 = torch.full_like(codes, -1)
    s2 = torch.full_like(scales, float("nan"))
    z2 = torch.full_like(zeros, float("nan"))
    cf, sf, zf = c2.view(-1), s2.view(-1), z2.view(-1)
    tensors = []
    for t in w.tensors:
        # tensor t's own package: its S planes back to back at S * offset
        a, ag = S * t.offset // 16, S * t.offset // G
        tensors.append((W[t.offset:t.offset + t.numel], t.rows, t.cols,
                        cf[a:a + S * t.numel // 16], sf[ag:ag + S * t.numel // G],
                        zf[ag:ag + S * t.numel // G]))
    gpu.rrq_construct_many(tensors, G, S)
    torch.cuda.synchronize()
    for t in w.tensors:
        a, ag = S * t.offset // 16, S * t.offset // G
        pc = cf[a:a + S * t.numel // 16].view(S, -1)
        ps = sf[ag:ag + S * t.numel // G].view(S, -1)
        pz = zf[ag:ag + S * t.numel // G].view(S, -1)
        assert torch.equal(pc, codes[:, t.offset // 16:(t.offset + t.numel) // 16]), t.name
        assert torch.equal(ps, scales[:, t.offset // G:(t.offset + t.numel) // G]), t.name
        assert torch.equal(pz, zeros[:, t.offset // G:(t.offset + t.numel) // G]), t.name
    del W, codes, scales, zeros, c2, s2, z2
    torch.cuda.empty_cache()

"""GPU parity of construction on an existing base checkpoint
(rrq_construct_from_base, through the C ABI) against the CPU oracle.

Bit-exact everywhere: plane 0 (the base, read only) must come back
unchanged, planes 1 .. S-1 must equal the oracle's, and the package's
reconstructions (computed on the GPU from the GPU package) must equal the
oracle's reconstructions of the oracle package. Every base is a seeded
stand-in for a foreign checkpoint (random codes, real-valued zero-points) or
the oracle's own first stage; none comes from the GPU.
"""

import os
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


def _u32(t):
    return t.detach().cpu().contiguous().numpy().view(np.uint32)


def _random_bits(seed, n, scale=0.02):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(n).astype(np.float32) * scale
    x = np.where(rng.random(n) < 1e-3, x * 20, x).astype(np.float32)
    return npo.f32_to_bf16_bits(x)


def _cpu_base(n, G, seed):
    c, s, z = wl.draw_base(n, G, seed, device="cpu")
    return c.numpy().view(np.uint32).copy(), s.numpy().copy(), z.numpy().copy()


def _check(rrq, bits, rows, cols, G, S, base, tag, ks=None):
    """GPU package on `base` vs the C oracle's, then reconstructions."""
    import torch
    _log(f"case {tag}: rows={rows} cols={cols} G={G} S={S}")
    W = torch.from_numpy(bits.view(np.int16).reshape(rows, cols)).cuda().view(torch.bfloat16)
    bc = torch.from_numpy(base[0].view(np.int32)).cuda()
    bs = torch.from_numpy(base[1]).cuda()
    bz = torch.from_numpy(base[2]).cuda()
    codes, scales, zeros = rrq.construct_from_base(W, bc, bs, bz, G, S)
    torch.cuda.synchronize()
    oc, os_, oz = oracle.c_construct_from_base(bits, base[0], base[1], base[2], G, S)
    assert np.array_equal(_u32(codes[0]), base[0]), f"{tag}: base codes changed"
    assert np.array_equal(_u32(scales[0]), base[1].view(np.uint32)), f"{tag}: base scales changed"
    assert np.array_equal(_u32(zeros[0]), base[2].view(np.uint32)), f"{tag}: base zeros changed"
    gc = _u32(codes)
    assert np.array_equal(gc, oc), f"{tag}: codes differ at {np.argwhere(gc != oc)[:5]}"
    assert np.array_equal(_u32(scales), os_.view(np.uint32)), f"{tag}: scales differ"
    assert np.array_equal(_u32(zeros), oz.view(np.uint32)), f"{tag}: zeros differ"
    for k in (ks or range(1, S + 1)):
        for dt, torch_dt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
            got = rrq.reconstruct(codes, scales, zeros, rows, cols, G, k, torch_dt)
            torch.cuda.synchronize()
            want = oracle.c_reconstruct(oc, os_, oz, G, k, dt)
            got_np = got.cpu().contiguous().view(torch.int32 if dt == "f32" else torch.int16).numpy()
            assert np.array_equal(got_np.reshape(-1).view(want.dtype), want), f"{tag}: recon k={k} {dt}"


@pytest.mark.parametrize("rows,cols,G", [
    (1, 32, 32), (3, 96, 32), (7, 192, 64), (5, 640, 128), (1, 128 * 65, 128),
    (13, 128 * 11, 128), (64, 64 * 64, 64), (2, 32 * 129, 32), (300, 1024, 128),
])
@pytest.mark.parametrize("S", [2, 3, 4])
def test_foreign_base_shapes_and_tails(gpu, rows, cols, G, S):
    n = rows * cols
    bits = _random_bits(rows * 31 + cols + G, n)
    base = _cpu_base(n, G, rows * 17 + cols + S)
    _check(gpu, bits, rows, cols, G, S, base, tag=f"foreign{rows}x{cols}")


@pytest.mark.parametrize("G", [32, 64, 128])
def test_own_first_stage_as_base_gives_direct_package(gpu, G):
    """The oracle's own stage 0 as the base: the GPU result must be the
    oracle's direct package (Algorithm 1's two branches agree)."""
    import torch
    rows, cols, S = 97, 1024, 4
    bits = _random_bits(900 + G, rows * cols)
    bc, bs, bz = oracle.c_construct(bits, G, 1)
    _check(gpu, bits, rows, cols, G, S, (bc[0], bs[0], bz[0]), tag=f"own{G}")
    W = torch.from_numpy(bits.view(np.int16).reshape(rows, cols)).cuda().view(torch.bfloat16)
    codes, scales, zeros = gpu.construct_from_base(
        W, torch.from_numpy(bc[0].view(np.int32)).cuda(), torch.from_numpy(bs[0]).cuda(),
        torch.from_numpy(bz[0]).cuda(), G, S)
    torch.cuda.synchronize()
    dc, ds, dz = oracle.c_construct(bits, G, S)
    assert np.array_equal(_u32(codes), dc)
    assert np.array_equal(_u32(scales), ds.view(np.uint32))
    assert np.array_equal(_u32(zeros), dz.view(np.uint32))


def test_zero_scale_base_and_exact_base(gpu):
    """s_0 = 0 leaves R_0 = W (residual planes = a direct package with one
    stage fewer); an exactly representable base leaves R_0 = 0 (degenerate
    residual stages)."""
    G, rows, cols, S = 64, 33, 512, 4
    n = rows * cols
    bits = _random_bits(77, n)
    codes0, _, z0 = _cpu_base(n, G, 78)
    base = (codes0, np.zeros(n // G, dtype=np.float32), z0)
    _check(gpu, bits, rows, cols, G, S, base, tag="zero_scale")
    rng = np.random.default_rng(79)
    Q0 = rng.integers(0, 4, n).astype(np.uint8)
    s0 = (2.0 ** rng.integers(-10, -2, n // G)).astype(np.float32)
    z0 = rng.integers(0, 4, n // G).astype(np.float32)
    x = ((Q0.reshape(-1, G) - z0[:, None]) * s0[:, None]).astype(np.float32).reshape(-1)
    exact_bits = (x.view(np.uint32) >> 16).astype(np.uint16)
    _check(gpu, exact_bits, rows, cols, G, S, (npo.pack_codes(Q0), s0, z0), tag="exact_base")


def test_golden_from_base_on_gpu(gpu):
    import json
    here = os.path.dirname(os.path.abspath(__file__))
    cases = json.load(open(os.path.join(here, "golden", "from_base_cases.json")))["cases"]
    for case in cases:
        G, S = case["G"], case["S"]
        words = np.array([int(h, 16) for h in case["base_codes"]], dtype=np.uint32)
        f = lambda h: np.array([int(h, 16)], dtype=np.uint32).view(np.float32)
        s0, z0 = f(case["base_scale"]), f(case["base_zero"])
        Q0 = npo.unpack_codes(words).astype(np.float64)
        R0 = np.array([int(h, 16) for h in case["residual"]], dtype=np.uint32).view(np.float32)
        x = ((Q0 - float(z0[0])) * float(s0[0]) + R0.astype(np.float64)[(np.arange(G) // 4) % 4])
        bits = (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        _check(gpu, bits, 1, G, G, S, (words, s0, z0), tag=case["name"])


def test_single_stage_leaves_package_untouched(gpu):
    import torch
    G, rows, cols = 128, 4, 1024
    n = rows * cols
    W = torch.zeros((rows, cols), dtype=torch.bfloat16, device="cuda")
    codes = torch.full((1, n // 16), 12345, dtype=torch.int32, device="cuda")
    scales = torch.full((1, n // G), 0.5, dtype=torch.float32, device="cuda")
    zeros = torch.full((1, n // G), 1.5, dtype=torch.float32, device="cuda")
    gpu.rrq_construct_from_base(W, rows, cols, G, 1, codes, scales, zeros)
    torch.cuda.synchronize()
    assert bool((codes == 12345).all()) and bool((scales == 0.5).all()) and bool((zeros == 1.5).all())


def test_qwen3_layer_full_foreign_base(gpu):
    """One Qwen3-8B-shaped layer as one flat call on a seeded foreign base;
    every output compared."""
    import torch
    w = wl.workload("qwen3_8b_layer")
    W = wl.materialize(w)
    bc, bs, bz = wl.materialize_base(w)
    bits = W.cpu().view(torch.int16).numpy().view(np.uint16)
    base = (bc.cpu().numpy().view(np.uint32), bs.cpu().numpy(), bz.cpu().numpy())
    _check(gpu, bits, w.numel // 4096, 4096, 128, 4, base, tag="qwen3_8b_layer", ks=(1, 2, 4))
    del W, bc, bs, bz
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_qwen3_8b_stack36_full_foreign_base(gpu):
    """The 36-layer stack in one flat call (the benchmark's launch shape) on a
    seeded foreign base; every tensor's planes and its k = 2 and 4
    reconstructions (bf16) against the C oracle, element by element."""
    import torch
    w = wl.workload("qwen3_8b_stack36")
    G, S = w.group_size, w.n_stages
    _log(f"materialize {w.name}: {w.numel} elements")
    W = wl.materialize(w)
    bc, bs, bz = wl.materialize_base(w)
    ng = w.n_groups
    rows = w.numel // 4096
    codes = torch.empty((S, w.numel // 16), dtype=torch.int32, device="cuda")
    scales = torch.empty((S, ng), dtype=torch.float32, device="cuda")
    zeros = torch.empty((S, ng), dtype=torch.float32, device="cuda")
    codes[0].copy_(bc)
    scales[0].copy_(bs)
    zeros[0].copy_(bz)
    gpu.rrq_construct_from_base(W, rows, 4096, G, S, codes, scales, zeros)
    torch.cuda.synchronize()

    def same(got, want):
        want_t = torch.from_numpy(np.ascontiguousarray(want).view(
            np.int16 if want.dtype == np.uint16 else np.int32)).cuda()
        return torch.equal(got.contiguous().view(want_t.dtype).reshape(want_t.shape), want_t)

    outs = {k: gpu.reconstruct(codes, scales, zeros, rows, 4096, G, k, torch.bfloat16)
            for k in (2, 4)}
    torch.cuda.synchronize()
    for i, t in enumerate(w.tensors):
        a, b = t.offset, t.offset + t.numel
        bits = W[a:b].cpu().view(torch.int16).numpy().view(np.uint16)
        oc, os_, oz = oracle.c_construct_from_base(
            bits, bc[a // 16:b // 16].cpu().numpy().view(np.uint32),
            bs[a // G:b // G].cpu().numpy(), bz[a // G:b // G].cpu().numpy(), G, S)
        assert same(codes[:, a // 16:b // 16], oc), f"{t.name}: codes differ"
        assert same(scales[:, a // G:b // G], os_), f"{t.name}: scales differ"
        assert same(zeros[:, a // G:b // G], oz), f"{t.name}: zeros differ"
        for k, out in outs.items():
            want = oracle.c_reconstruct(oc, os_, oz, G, k, "bf16")
            assert same(out.view(-1)[a:b], want), f"{t.name}: reconstruction k={k} differs"
        if i % 28 == 27:
            _log(f"{w.name} from base: {i + 1}/{len(w.tensors)} tensors bit-exact")
    del W, bc, bs, bz, codes, scales, zeros, outs
    torch.cuda.empty_cache()

"""The HBM probes write exactly what include/hbm_probe.h states: the mixed
probe packs the first 80 bytes of every 128 bytes of src into dst, the
read-only probe XORs what it reads, the write-only probe fills, and the
construct-pattern probe stores XORs of each group's words in rrq_construct's
planes, and the reconstruct-pattern probe XORs of each chunk's loads; the
machine probes report clock ticks that behave as a timing must."""

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("src_bytes", [128, 16384 * 3 + 128 * 5, (1 << 24) + 128 * 7])
def test_probe_output(gpu, src_bytes):
    import torch

    from paper_2608_04048_amd import probe
    print(f"probe src_bytes={src_bytes}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(src_bytes)
    src = torch.randint(-2**31, 2**31 - 1, (src_bytes // 4,), dtype=torch.int32, device="cuda",
                        generator=g)
    dst = torch.full((src_bytes // 8 * 5 // 4 + 4,), -1, dtype=torch.int32, device="cuda")
    probe.hbm_probe_stream(src, src_bytes, dst)
    torch.cuda.synchronize()
    s = src.cpu().numpy().view(np.uint8).reshape(-1, 128)[:, :80].reshape(-1)
    d = dst.cpu().numpy().view(np.uint8)
    assert np.array_equal(d[:s.size], s)
    assert np.all(d[s.size:] == 0xFF)   # nothing written past the end


@pytest.mark.parametrize("nbytes", [16, 16384 * 3 + 16 * 5, (1 << 24) + 16 * 7])
def test_read_probe_xor(gpu, nbytes):
    import torch

    from paper_2608_04048_amd import probe
    print(f"read probe nbytes={nbytes}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(nbytes)
    src = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), dtype=torch.int32, device="cuda",
                        generator=g)
    out = torch.zeros(1, dtype=torch.int32, device="cuda")
    probe.hbm_probe_read(src, nbytes, out)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(src.cpu().numpy().view(np.uint32))
    assert out.cpu().numpy().view(np.uint32)[0] == want


@pytest.mark.parametrize("nbytes", [16, 16384 * 3 + 16 * 5, (1 << 24) + 16 * 7])
def test_write_probe_fill(gpu, nbytes):
    import torch

    from paper_2608_04048_amd import probe
    print(f"write probe nbytes={nbytes}", flush=True)
    dst = torch.full((nbytes // 4 + 4,), -1, dtype=torch.int32, device="cuda")
    probe.hbm_probe_write(dst, nbytes, 0x12345678)
    torch.cuda.synchronize()
    d = dst.cpu().numpy().view(np.uint32)
    assert np.all(d[:nbytes // 4] == 0x12345678)
    assert np.all(d[nbytes // 4:] == 0xFFFFFFFF)   # nothing written past the end


@pytest.mark.parametrize("G,n_groups,S,bpc", [
    (128, 64 * 3 + 5, 4, 0), (64, 1000, 3, 0), (32, 64 * 300 + 17, 4, 0),
    (128, 64 * 2048 + 3, 4, 0), (128, 64 * 700 + 9, 2, 1), (32, 64 * 40, 1, 32),
])
def test_construct_probe_output(gpu, G, n_groups, S, bpc):
    """The construct-pattern probe stores exactly what include/hbm_probe.h
    states, in rrq_construct's planes, and nothing past them."""
    import torch

    from paper_2608_04048_amd import probe
    print(f"construct probe G={G} n_groups={n_groups} S={S} blocks_per_cu={bpc}", flush=True)
    nw = n_groups * G // 2                      # 32-bit words of input
    g = torch.Generator(device="cuda").manual_seed(n_groups + G)
    src = torch.randint(-2**31, 2**31 - 1, (nw,), dtype=torch.int32, device="cuda", generator=g)
    wpg = G // 16
    codes = torch.full((S * n_groups * wpg + 8,), -1, dtype=torch.int32, device="cuda")
    scales = torch.full((S * n_groups + 8,), -1, dtype=torch.int32, device="cuda")
    zeros = torch.full((S * n_groups + 8,), -1, dtype=torch.int32, device="cuda")
    probe.hbm_probe_construct(src, n_groups, G, S, codes, scales, zeros, bpc)
    torch.cuda.synchronize()
    w = src.cpu().numpy().view(np.uint32).reshape(n_groups, G // 2)
    acc = np.bitwise_xor.reduce(w.reshape(n_groups, (G // 2) // wpg, wpg), axis=1)
    c = codes.cpu().numpy().view(np.uint32)
    sc = scales.cpu().numpy().view(np.uint32)
    ze = zeros.cpu().numpy().view(np.uint32)
    for k in range(S):
        kk = np.uint32(k)
        assert np.array_equal(c[k * n_groups * wpg:(k + 1) * n_groups * wpg],
                              (acc ^ kk).reshape(-1)), f"codes of stage {k}"
        assert np.array_equal(sc[k * n_groups:(k + 1) * n_groups], w[:, 0] ^ kk), f"scales {k}"
        assert np.array_equal(ze[k * n_groups:(k + 1) * n_groups], w[:, 1] ^ kk), f"zeros {k}"
    assert np.all(c[S * n_groups * wpg:] == 0xFFFFFFFF)
    assert np.all(sc[S * n_groups:] == 0xFFFFFFFF) and np.all(ze[S * n_groups:] == 0xFFFFFFFF)


@pytest.mark.parametrize("G,n_groups,k,bpc", [
    (128, 3, 1, 0), (128, 64 * 33 + 7, 2, 0), (64, 1001, 3, 0), (32, 64 * 200 + 3, 4, 0),
    (128, 64 * 2048 + 1, 4, 1), (64, 64 * 700, 2, 32),
])
def test_reconstruct_probe_output(gpu, G, n_groups, k, bpc):
    """The reconstruct-pattern probe stores exactly what include/hbm_probe.h
    states, and nothing past the output."""
    import torch

    from paper_2608_04048_amd import probe
    print(f"reconstruct probe G={G} n_groups={n_groups} k={k} blocks_per_cu={bpc}", flush=True)
    n = n_groups * G
    g = torch.Generator(device="cuda").manual_seed(n_groups * 7 + k)
    rnd = lambda m: torch.randint(-2**31, 2**31 - 1, (m,), dtype=torch.int32, device="cuda",
                                  generator=g)
    codes, scales, zeros = rnd(4 * n // 16), rnd(4 * n_groups), rnd(4 * n_groups)
    out = torch.full((n // 2 + 8,), -1, dtype=torch.int32, device="cuda")
    probe.hbm_probe_reconstruct(codes, scales, zeros, n_groups, G, k, out, bpc)
    torch.cuda.synchronize()
    c = codes.cpu().numpy().view(np.uint32).reshape(4, n // 16)
    s_ = scales.cpu().numpy().view(np.uint32).reshape(4, n_groups)
    z_ = zeros.cpu().numpy().view(np.uint32).reshape(4, n_groups)
    chunk = np.arange(n // 8)
    x = np.zeros(n // 8, dtype=np.uint32)
    for t in range(k):
        x ^= c[t][chunk // 2] ^ s_[t][chunk * 8 // G] ^ z_[t][chunk * 8 // G]
    want = np.stack([x, x + np.uint32(1), x + np.uint32(2), x + np.uint32(3)], axis=1).reshape(-1)
    o = out.cpu().numpy().view(np.uint32)
    assert np.array_equal(o[:n // 2], want)
    assert np.all(o[n // 2:] == 0xFFFFFFFF)


def test_machine_probes_report_ticks(gpu):
    """The issue and LDS probes run in bounds and report positive ticks per
    wave; a loop doing both the MFMAs and the FMAs takes at least as long as
    either alone (within timing noise), and more waves per SIMD never make a
    wave's own loop faster."""
    import torch

    from paper_2608_04048_amd import probe
    print("machine probes", flush=True)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    per = {}
    for wps in (1, 2):
        out = torch.full((cus * wps * 256,), float("nan"), dtype=torch.float32, device="cuda")
        ticks = torch.zeros(cus * wps * 4, dtype=torch.int64, device="cuda")
        for mode in (0, 1, 2):
            probe.hbm_probe_issue(mode, wps, 2000, out, ticks)
            torch.cuda.synchronize()
            t = ticks.cpu().numpy()
            assert np.all(t > 0)
            assert torch.isfinite(out).all()
            per[(wps, mode)] = t.mean()
        assert per[(wps, 2)] >= 0.9 * max(per[(wps, 0)], per[(wps, 1)])
    assert per[(2, 0)] >= 0.9 * per[(1, 0)]
    for wpc in (4, 8):
        out = torch.zeros(cus * wpc * 64, dtype=torch.int32, device="cuda")
        ticks = torch.zeros(cus * wpc, dtype=torch.int64, device="cuda")
        probe.hbm_probe_lds(wpc, 400, out, ticks)
        torch.cuda.synchronize()
        assert np.all(ticks.cpu().numpy() > 0)

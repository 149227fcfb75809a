"""The HBM streaming probe writes exactly what include/hbm_probe.h states:
the first 80 bytes of every 128 bytes of src, packed into dst."""

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

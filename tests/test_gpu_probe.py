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

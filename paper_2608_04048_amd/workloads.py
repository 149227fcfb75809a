"""Seeded synthetic bfloat16 weight stacks for tests and benchmarks.

No quantization arithmetic lives here: this module only draws random weights
with the shapes and value distributions of the models the paper quantizes
(Sec. 4.1, Appendix on package sizes) and lays them out back to back in one
flat bfloat16 buffer. Both the HIP path and the CPU oracle consume the bits it
produces.

Distributions (all with standard deviation 0.02, drawn in float32 and rounded
to bfloat16 nearest-even by torch):
  gauss     N(0, 0.02^2)
  outlier   gauss, and each element independently (probability 1e-3) scaled
            by 20: localized outliers, group peak-to-mean ratios in the
            range the paper reports for real checkpoints (Sec. 3, PMR)
  t3        Student-t with 3 degrees of freedom, scaled to std 0.02
  channel   gauss with 8 seeded input columns scaled by 50

Seeds: 2608 + 16 * layer + projection index.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import List, Tuple

BASE_SEED = 2608

# Linear projections of one decoder layer, (name, out, in).
QWEN3_8B_LAYER: List[Tuple[str, int, int]] = [
    ("q_proj", 4096, 4096), ("k_proj", 1024, 4096), ("v_proj", 1024, 4096),
    ("o_proj", 4096, 4096), ("gate_proj", 12288, 4096), ("up_proj", 12288, 4096),
    ("down_proj", 4096, 12288),
]
DENSE_32B_LAYER: List[Tuple[str, int, int]] = [
    ("q_proj", 5120, 5120), ("k_proj", 1024, 5120), ("v_proj", 1024, 5120),
    ("o_proj", 5120, 5120), ("gate_proj", 25600, 5120), ("up_proj", 25600, 5120),
    ("down_proj", 5120, 25600),
]


@dataclass(frozen=True)
class Tensor:
    name: str
    rows: int
    cols: int
    dist: str
    seed: int
    offset: int  # element offset in the flat buffer

    @property
    def numel(self) -> int:
        return self.rows * self.cols


@dataclass(frozen=True)
class Workload:
    name: str
    tensors: Tuple[Tensor, ...]
    group_size: int = 128
    n_stages: int = 4
    recon_k: Tuple[int, ...] = (1, 2, 3, 4)

    @property
    def numel(self) -> int:
        return sum(t.numel for t in self.tensors)

    @property
    def n_groups(self) -> int:
        return self.numel // self.group_size


def _stack(name, layer, n_layers, dist, G=128, S=4, recon_k=(1, 2, 3, 4)):
    tensors, off = [], 0
    for li in range(n_layers):
        for pi, (pname, rows, cols) in enumerate(layer):
            tensors.append(Tensor(f"layers.{li}.{pname}", rows, cols, dist,
                                  BASE_SEED + 16 * li + pi, off))
            off += rows * cols
    return Workload(name, tuple(tensors), G, S, recon_k)


def single(name, rows, cols, dist, G=128, S=4, seed=BASE_SEED, recon_k=(1, 2, 3, 4)):
    return Workload(name, (Tensor(name, rows, cols, dist, seed, 0),), G, S, recon_k)


def workload(name: str) -> Workload:
    """Named workloads (shapes of the paper's Qwen3-8B setup and a 32B-class
    dense model)."""
    if name == "matrix_1024":
        return single("matrix_1024", 1024, 1024, "gauss")
    if name == "qwen3_8b_layer":
        return _stack("qwen3_8b_layer", QWEN3_8B_LAYER, 1, "outlier")
    if name == "qwen3_8b_stack36":
        return _stack("qwen3_8b_stack36", QWEN3_8B_LAYER, 36, "outlier", recon_k=(2, 4))
    if name == "dense32b_stack64":
        return _stack("dense32b_stack64", DENSE_32B_LAYER, 64, "outlier", recon_k=(3,))
    if name.startswith("sweep_12288x4096_"):
        # sweep_12288x4096_<dist>_g<G>
        _, _, dist, g = name.split("_")
        return single(name, 12288, 4096, dist, G=int(g[1:]))
    raise KeyError(name)


SWEEP = [f"sweep_12288x4096_{d}_g{g}" for d in ("gauss", "t3", "channel") for g in (32, 64, 128)]
ALL = ["matrix_1024", "qwen3_8b_layer", "qwen3_8b_stack36", *SWEEP, "dense32b_stack64"]


def draw(t: Tensor, device="cuda"):
    """bfloat16 tensor [rows, cols] of one workload tensor."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(t.seed)
    shape = (t.rows, t.cols)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if t.dist == "gauss":
        x.mul_(0.02)
    elif t.dist == "outlier":
        x.mul_(0.02)
        mask = torch.rand(shape, generator=g, device=device) < 1e-3
        x[mask] *= 20.0
    elif t.dist == "t3":
        chi2 = torch.zeros(shape, device=device, dtype=torch.float32)
        for _ in range(3):
            chi2.add_(torch.randn(shape, generator=g, device=device, dtype=torch.float32).square_())
        # t3 = N / sqrt(chi2 / 3) has variance 3; scale to std 0.02
        x.div_(chi2.div_(3.0).sqrt_()).mul_(0.02 / 3.0 ** 0.5)
    elif t.dist == "channel":
        x.mul_(0.02)
        cols = torch.randperm(t.cols, generator=g, device=device)[:8]
        x[:, cols] *= 50.0
    else:
        raise ValueError(t.dist)
    return x.to(torch.bfloat16)


def materialize(w: Workload, device="cuda"):
    """One flat contiguous bfloat16 buffer holding every tensor of w."""
    import torch
    buf = torch.empty(w.numel, dtype=torch.bfloat16, device=device)
    for t in w.tensors:
        buf[t.offset:t.offset + t.numel].view(t.rows, t.cols).copy_(draw(t, device))
    return buf


BASE_CHECKPOINT_SEED_OFFSET = 7919


def draw_base(n: int, group_size: int, seed: int, device="cuda"):
    """A stand-in for a base checkpoint from another quantizer, for n weights
    in groups of group_size: uniformly random 2-bit codes (packed, 16 per
    uint32 word, returned as int32 [n/16]), per-group scales uniform in
    [0.01, 0.09] (the magnitude of 2-bit min-max scales of the weights above)
    and real-valued zero-points uniform in [0, 3) (float32 [n/G] each)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    codes = torch.randint(-2 ** 31, 2 ** 31, (n // 16,), generator=g, device=device,
                          dtype=torch.int64).to(torch.int32)
    scales = torch.rand(n // group_size, generator=g, device=device).mul_(0.08).add_(0.01)
    zeros = torch.rand(n // group_size, generator=g, device=device).mul_(3.0)
    return codes, scales, zeros


def materialize_base(w: Workload, device="cuda"):
    """Flat base-checkpoint buffers (codes, scales, zeros) for every tensor of
    w, laid out like the weights (tensor t's groups at t.offset / G)."""
    import torch
    G = w.group_size
    codes = torch.empty(w.numel // 16, dtype=torch.int32, device=device)
    scales = torch.empty(w.numel // G, dtype=torch.float32, device=device)
    zeros = torch.empty(w.numel // G, dtype=torch.float32, device=device)
    for t in w.tensors:
        c, s, z = draw_base(t.numel, G, t.seed + BASE_CHECKPOINT_SEED_OFFSET, device)
        codes[t.offset // 16:(t.offset + t.numel) // 16].copy_(c)
        scales[t.offset // G:(t.offset + t.numel) // G].copy_(s)
        zeros[t.offset // G:(t.offset + t.numel) // G].copy_(z)
    return codes, scales, zeros

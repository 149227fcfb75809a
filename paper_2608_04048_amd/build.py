"""Build librrq.so (the HIP kernels and the C ABI) and libhbm_probe.so (the
HBM streaming probe) in-tree for gfx950.

    python -m paper_2608_04048_amd.build          # compile, write the library
    python -m paper_2608_04048_amd.build --asm    # also keep the gfx950 assembly

The library lands next to this file (paper_2608_04048_amd/librrq.so), where
the Python binding loads it.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "librrq.so")
PROBE_LIB = os.path.join(PKG, "libhbm_probe.so")

ARCH = "gfx950"
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

# Device code: no contraction into FMA, no fast math, denormals kept (the
# HIP default), packed-FP32 instructions disabled.
DEVICE_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra"]
# Per-source device flags: the linear kernels keep their MFMA results in
# ordinary VGPRs (their accumulations are VALU work, so accumulator registers
# would only add copies).
SOURCE_FLAGS = {"rrq_linear": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
                "rrq_decode": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
                "rrq_batch": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
                "rrq_prefill": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build librrq.so)")


def _run(cmd):
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass does not know the packed-fp32 target feature and says
    # so; that line is expected and dropped.
    out = "\n".join(l for l in proc.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if proc.returncode != 0:
        raise RuntimeError(f"command failed ({proc.returncode}): {' '.join(cmd)}\n{out}")
    if out.strip():
        print(out)


def build(keep_asm: bool = False) -> str:
    """Compile every source and link librrq.so; returns the library path."""
    cc = hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    kern_objs = []
    for name in ("rrq_kernels", "rrq_linear", "rrq_decode", "rrq_batch", "rrq_prefill"):
        obj = os.path.join(BUILD_DIR, name + ".o")
        cmd = [cc, *DEVICE_FLAGS, *SOURCE_FLAGS.get(name, []), f"-I{INCLUDE}", f"-I{CSRC}", "-c",
               os.path.join(CSRC, name + ".hip"), "-o", obj]
        if keep_asm:
            cmd += ["-save-temps=obj"]
        _run(cmd)
        kern_objs.append(obj)
    api_obj = os.path.join(BUILD_DIR, "rrq_api.o")
    _run([cc, "-x", "c++", *HOST_FLAGS, "-D__HIP_PLATFORM_AMD__", f"-I{INCLUDE}", f"-I{CSRC}",
          f"-I{ROCM}/include",
          "-c", os.path.join(CSRC, "rrq_api.cpp"), "-o", api_obj])
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *kern_objs, api_obj, "-o", tmp])
    os.replace(tmp, LIB)
    build_probe()
    return LIB


def build_probe() -> str:
    """Compile libhbm_probe.so (the HBM streaming probe used by the benchmark)."""
    cc = hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    tmp = PROBE_LIB + ".tmp"
    _run([cc, *DEVICE_FLAGS, f"-I{INCLUDE}", "-shared",
          os.path.join(CSRC, "hbm_probe.hip"), "-o", tmp])
    os.replace(tmp, PROBE_LIB)
    return PROBE_LIB


if __name__ == "__main__":
    print(build(keep_asm="--asm" in sys.argv))

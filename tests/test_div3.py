"""The construct kernel computes a group's scale fl((hi - lo) / 3) without the
IEEE division sequence: q = fl(d fl(1/3)), rem = fma(-3, q, d),
s = fma(rem, fl(1/3), q). These are plain IEEE binary32 operations, so the
same arithmetic compiled for the host (hardware FMA, no contraction) shows
that the result equals IEEE d / 3 for every non-negative finite d; the GPU
parity tests then compare the kernel itself with the oracle."""

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_div3_exhaustive(tmp_path):
    exe = tmp_path / "div3"
    subprocess.run(["gcc", "-O2", "-std=c11", "-mfma", "-ffp-contract=off", "-fopenmp",
                    os.path.join(HERE, "csrc", "div3_exhaustive.c"), "-o", str(exe), "-lm"],
                   check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600)
    assert out.returncode == 0 and out.stdout.strip() == "0", out.stdout + out.stderr

"""RRQ oracle: plain CPU implementations of construction and reconstruction.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package. The product path
(``paper_2608_04048_amd``) never imports it.

Two independent writings of the same definition:
* ``rrq_oracle.py`` (numpy, vectorised over groups): the readable definition;
* ``rrq_oracle.c`` (plain scalar C, OpenMP over groups): the same steps for
  inputs too large for numpy, and the timed CPU baseline.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import rrq_oracle as np_oracle  # noqa: F401  (re-export)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rrq_oracle.c")
_LIB = os.path.join(_HERE, "librrq_oracle.so")

CFLAGS = ["-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
          "-fPIC", "-shared", "-Wall", "-Wextra"]

_lib = None


def build_c_oracle(force: bool = True) -> str:
    """Compile the C oracle into oracle/librrq_oracle.so with gcc."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build_c_oracle(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        lib.rrq_oracle_construct.argtypes = [P, ctypes.c_int64, ctypes.c_int32,
                                             ctypes.c_int32, P, P, P]
        lib.rrq_oracle_construct.restype = ctypes.c_int
        lib.rrq_oracle_construct_from_base.argtypes = [P, ctypes.c_int64, ctypes.c_int32,
                                                       ctypes.c_int32, P, P, P]
        lib.rrq_oracle_construct_from_base.restype = ctypes.c_int
        lib.rrq_oracle_construct_format.argtypes = [P, ctypes.c_int64, ctypes.c_int32,
                                                    ctypes.c_int32, ctypes.c_int32,
                                                    ctypes.c_int32, P, P, P]
        lib.rrq_oracle_construct_format.restype = ctypes.c_int
        lib.rrq_oracle_reconstruct_format.argtypes = [P, P, P, ctypes.c_int64, ctypes.c_int32,
                                                      ctypes.c_int32, ctypes.c_int32,
                                                      ctypes.c_int32, ctypes.c_int32,
                                                      ctypes.c_int32, P]
        lib.rrq_oracle_reconstruct_format.restype = ctypes.c_int
        lib.rrq_oracle_group_pmr.argtypes = [P, ctypes.c_int64, ctypes.c_int32, P]
        lib.rrq_oracle_group_pmr.restype = ctypes.c_int
        lib.rrq_oracle_f32_to_f16.argtypes = [P, ctypes.c_int64, P]
        lib.rrq_oracle_f32_to_f16.restype = None
        lib.rrq_oracle_reconstruct.argtypes = [P, P, P, ctypes.c_int64, ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_int32,
                                               ctypes.c_int32, P]
        lib.rrq_oracle_reconstruct.restype = ctypes.c_int
        lib.rrq_oracle_threads.argtypes = []
        lib.rrq_oracle_threads.restype = ctypes.c_int
        lib.rrq_oracle_set_threads.argtypes = [ctypes.c_int]
        lib.rrq_oracle_set_threads.restype = None
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


def c_construct(w_bits: np.ndarray, group_size: int, n_stages: int):
    """C oracle construction of flat bfloat16 bits -> (codes, scales, zeros)."""
    lib = _load()
    w = np.ascontiguousarray(w_bits, dtype=np.uint16).reshape(-1)
    n = w.size
    codes = np.empty((n_stages, n // 16), dtype=np.uint32)
    scales = np.empty((n_stages, n // group_size), dtype=np.float32)
    zeros = np.empty((n_stages, n // group_size), dtype=np.float32)
    rc = lib.rrq_oracle_construct(_ptr(w), n, group_size, n_stages,
                                  _ptr(codes), _ptr(scales), _ptr(zeros))
    if rc == 2:
        raise ValueError("RRQ oracle: inputs must be finite")
    if rc == 3:
        raise ValueError("RRQ oracle: a group's range overflows binary32 (inputs need |x| < 2^127)")
    if rc != 0:
        raise ValueError(f"RRQ oracle: bad arguments (status {rc})")
    return codes, scales, zeros


def c_construct_from_base(w_bits: np.ndarray, base_codes: np.ndarray, base_scales: np.ndarray,
                          base_zeros: np.ndarray, group_size: int, n_stages: int):
    """C oracle construction on a given base stage -> (codes, scales, zeros),
    plane 0 = the base as given."""
    lib = _load()
    w = np.ascontiguousarray(w_bits, dtype=np.uint16).reshape(-1)
    n = w.size
    codes = np.empty((n_stages, n // 16), dtype=np.uint32)
    scales = np.empty((n_stages, n // group_size), dtype=np.float32)
    zeros = np.empty((n_stages, n // group_size), dtype=np.float32)
    codes[0] = np.asarray(base_codes, dtype=np.uint32).reshape(-1)
    scales[0] = np.asarray(base_scales, dtype=np.float32).reshape(-1)
    zeros[0] = np.asarray(base_zeros, dtype=np.float32).reshape(-1)
    rc = lib.rrq_oracle_construct_from_base(_ptr(w), n, group_size, n_stages,
                                            _ptr(codes), _ptr(scales), _ptr(zeros))
    if rc == 2:
        raise ValueError("RRQ oracle: inputs and the base residual W - xhat_0 must be finite")
    if rc == 3:
        raise ValueError("RRQ oracle: a group's range overflows binary32")
    if rc != 0:
        raise ValueError(f"RRQ oracle: bad arguments (status {rc})")
    return codes, scales, zeros


def c_reconstruct(codes: np.ndarray, scales: np.ndarray, zeros: np.ndarray,
                  group_size: int, k_stages: int, out_dtype: str = "f32"):
    """C oracle prefix-k reconstruction -> float32 or bfloat16 bits (uint16)."""
    lib = _load()
    codes = np.ascontiguousarray(codes, dtype=np.uint32)
    scales = np.ascontiguousarray(scales, dtype=np.float32)
    zeros = np.ascontiguousarray(zeros, dtype=np.float32)
    S = codes.shape[0]
    n = codes.shape[1] * 16
    bf16 = out_dtype == "bf16"
    out = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
    rc = lib.rrq_oracle_reconstruct(_ptr(codes), _ptr(scales), _ptr(zeros), n,
                                    group_size, S, k_stages, int(bf16), _ptr(out))
    if rc != 0:
        raise ValueError(f"RRQ oracle: bad arguments (status {rc})")
    return out


def c_threads() -> int:
    """OpenMP threads the C oracle runs with."""
    return int(_load().rrq_oracle_threads())


def c_set_threads(n: int) -> None:
    """Run the C oracle's parallel regions on n OpenMP threads."""
    _load().rrq_oracle_set_threads(int(n))


ZP_CODES = {"int": 0, "real": 1, "sym": 2}
SCALE_CODES = {"f32": 0, "f16": 1, "bf16": 2}


def c_construct_format(w_bits: np.ndarray, group_size: int, n_stages: int, zero_point: str,
                       scale_dtype: str):
    """C oracle construction in a stage format -> (codes, scales as stored,
    zeros; for symmetric stages the zeros hold the implicit 2)."""
    lib = _load()
    w = np.ascontiguousarray(w_bits, dtype=np.uint16).reshape(-1)
    n = w.size
    codes = np.empty((n_stages, n // 16), dtype=np.uint32)
    scales = np.empty((n_stages, n // group_size),
                      dtype=np.float32 if scale_dtype == "f32" else np.uint16)
    zeros = np.empty((n_stages, n // group_size), dtype=np.float32)
    rc = lib.rrq_oracle_construct_format(_ptr(w), n, group_size, n_stages, ZP_CODES[zero_point],
                                         SCALE_CODES[scale_dtype], _ptr(codes), _ptr(scales),
                                         _ptr(zeros))
    if rc == 2:
        raise ValueError("RRQ oracle: inputs must be finite")
    if rc == 3:
        raise ValueError("RRQ oracle: a group's range or scale overflows its type")
    if rc != 0:
        raise ValueError(f"RRQ oracle: bad arguments (status {rc})")
    return codes, scales, zeros


def c_reconstruct_format(codes, scales, zeros, group_size: int, k_stages: int, zero_point: str,
                         scale_dtype: str, out_dtype: str = "f32"):
    lib = _load()
    codes = np.ascontiguousarray(codes, dtype=np.uint32)
    scales = np.ascontiguousarray(scales)
    zeros = np.ascontiguousarray(zeros, dtype=np.float32)
    S = codes.shape[0]
    n = codes.shape[1] * 16
    bf16 = out_dtype == "bf16"
    out = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
    rc = lib.rrq_oracle_reconstruct_format(_ptr(codes), _ptr(scales), _ptr(zeros), n,
                                           group_size, S, ZP_CODES[zero_point],
                                           SCALE_CODES[scale_dtype], k_stages, int(bf16),
                                           _ptr(out))
    if rc != 0:
        raise ValueError(f"RRQ oracle: bad arguments (status {rc})")
    return out


def c_f32_to_f16(x: np.ndarray) -> np.ndarray:
    """The C oracle's own binary32 -> binary16 rounding (bit patterns)."""
    x = np.ascontiguousarray(x, dtype=np.float32).reshape(-1)
    out = np.empty(x.size, dtype=np.uint16)
    _load().rrq_oracle_f32_to_f16(_ptr(x), x.size, _ptr(out))
    return out


def c_group_pmr(w_bits: np.ndarray, group_size: int) -> np.ndarray:
    """C oracle per-group peak-to-mean ratio of flat bfloat16 bits."""
    w = np.ascontiguousarray(w_bits, dtype=np.uint16).reshape(-1)
    out = np.empty(w.size // group_size, dtype=np.float32)
    rc = _load().rrq_oracle_group_pmr(_ptr(w), w.size, group_size, _ptr(out))
    if rc != 0:
        raise ValueError(f"RRQ oracle: bad arguments (status {rc})")
    return out

"""RRQ (Recurrent Residual Quantization) package construction and prefix
reconstruction on AMD Instinct MI355X.

Thin Python binding of librrq.so (include/rrq.h). The functions named like the
C ABI (``rrq_construct``, ``rrq_construct_many``, ``rrq_construct_from_base``, ``rrq_reconstruct``,
``rrq_linear``, their ``*_format`` twins, ``rrq_construct_stats``,
``rrq_group_pmr``, ``rrq_package_bytes``, ``rrq_status_string``) only marshal
arguments: tensors become device pointers,
the stream defaults to torch's current stream, and a nonzero status raises
``RRQError``. ``construct``, ``construct_from_base``, ``reconstruct`` and
``linear`` additionally allocate the output tensors with torch. Every computation runs in the HIP kernels; there is
no fallback, and a missing library raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librrq.so")

RRQ_OK = 0
RRQ_ERR_NULL = 1
RRQ_ERR_ALIGN = 2
RRQ_ERR_SHAPE = 3
RRQ_ERR_GROUP = 4
RRQ_ERR_STAGES = 5
RRQ_ERR_DTYPE = 6
RRQ_ERR_HIP = 7
RRQ_ERR_FORMAT = 8

RRQ_ZP_INTEGER = 0
RRQ_ZP_REAL = 1
RRQ_ZP_SYMMETRIC = 2
RRQ_SCALE_F32 = 0
RRQ_SCALE_F16 = 1
RRQ_SCALE_BF16 = 2
ZERO_POINTS = {"int": RRQ_ZP_INTEGER, "real": RRQ_ZP_REAL, "sym": RRQ_ZP_SYMMETRIC}
SCALE_TYPES = {"f32": RRQ_SCALE_F32, "f16": RRQ_SCALE_F16, "bf16": RRQ_SCALE_BF16}

RRQ_F32 = 0
RRQ_BF16 = 1

RRQ_MAX_STAGES = 4
GROUP_SIZES = (32, 64, 128)

_lib = None


class RRQError(RuntimeError):
    """A librrq call returned a nonzero status."""

    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {rrq_status_string(status)} (status {status})")


def load_library() -> ctypes.CDLL:
    """Load librrq.so (built by ``python -m paper_2608_04048_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2608_04048_amd.build`")
        # torch first: the library then binds to the HIP runtime torch has
        # loaded (torch ships its own copy; loading the library first would
        # bring a second runtime into the process, whose launches fail)
        import torch  # noqa: F401
        lib = ctypes.CDLL(LIB_PATH)
        P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.rrq_construct.argtypes = [P, I64, I64, I32, I32, P, P, P, P]
        lib.rrq_construct.restype = ctypes.c_int
        lib.rrq_construct_from_base.argtypes = [P, I64, I64, I32, I32, P, P, P, P]
        lib.rrq_construct_from_base.restype = ctypes.c_int
        lib.rrq_reconstruct.argtypes = [P, P, P, I64, I64, I32, I32, I32, P, I32, P]
        lib.rrq_reconstruct.restype = ctypes.c_int
        lib.rrq_linear.argtypes = [P, P, P, I64, I64, I32, I32, I32, P, I64, P, P]
        lib.rrq_linear.restype = ctypes.c_int
        lib.rrq_construct_stats.argtypes = [P, I64, I64, I32, I32, I32, I32, P, P, P, P, P]
        lib.rrq_construct_stats.restype = ctypes.c_int
        lib.rrq_construct_many.argtypes = [P, I32, I32, I32, P]
        lib.rrq_construct_many.restype = ctypes.c_int
        lib.rrq_group_pmr.argtypes = [P, I64, I64, I32, P, P]
        lib.rrq_group_pmr.restype = ctypes.c_int
        lib.rrq_construct_format.argtypes = [P, I64, I64, I32, I32, I32, I32, P, P, P, P]
        lib.rrq_construct_format.restype = ctypes.c_int
        lib.rrq_construct_from_base_format.argtypes = [P, I64, I64, I32, I32, I32, I32, P, P,
                                                       P, P]
        lib.rrq_construct_from_base_format.restype = ctypes.c_int
        lib.rrq_reconstruct_format.argtypes = [P, P, P, I64, I64, I32, I32, I32, I32, I32, P,
                                               I32, P]
        lib.rrq_reconstruct_format.restype = ctypes.c_int
        lib.rrq_linear_format.argtypes = [P, P, P, I64, I64, I32, I32, I32, I32, I32, P, I64,
                                          P, P]
        lib.rrq_linear_format.restype = ctypes.c_int
        lib.rrq_package_bytes.argtypes = [I64, I64, I32, I32, ctypes.POINTER(ctypes.c_size_t),
                                          ctypes.POINTER(ctypes.c_size_t)]
        lib.rrq_package_bytes.restype = ctypes.c_int
        lib.rrq_status_string.argtypes = [ctypes.c_int]
        lib.rrq_status_string.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def _ptr(x) -> Optional[int]:
    """Device pointer of a tensor (or a raw integer address, or None)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---------------------------------------------------------------------------
# C ABI, one to one
# ---------------------------------------------------------------------------

def rrq_status_string(status: int) -> str:
    return load_library().rrq_status_string(int(status)).decode()


def rrq_package_bytes(rows: int, cols: int, group_size: int, n_stages: int) -> Tuple[int, int]:
    """(codes_bytes, scales_bytes) of a package; the zeros buffer has scales_bytes."""
    cb, sb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    st = load_library().rrq_package_bytes(rows, cols, group_size, n_stages,
                                          ctypes.byref(cb), ctypes.byref(sb))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_package_bytes")
    return cb.value, sb.value


def rrq_construct(W, rows: int, cols: int, group_size: int, n_stages: int,
                  codes, scales, zeros, stream=None) -> None:
    """Enqueue package construction (see include/rrq.h)."""
    st = load_library().rrq_construct(_ptr(W), rows, cols, group_size, n_stages,
                                      _ptr(codes), _ptr(scales), _ptr(zeros), _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_construct")


def rrq_construct_from_base(W, rows: int, cols: int, group_size: int, n_stages: int,
                            codes, scales, zeros, stream=None) -> None:
    """Enqueue the residual stages on the base stage held in plane 0 of the
    package (see include/rrq.h)."""
    st = load_library().rrq_construct_from_base(_ptr(W), rows, cols, group_size, n_stages,
                                                _ptr(codes), _ptr(scales), _ptr(zeros),
                                                _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_construct_from_base")


def rrq_reconstruct(codes, scales, zeros, rows: int, cols: int, group_size: int,
                    n_stages: int, k_stages: int, W_out, out_dtype: int, stream=None) -> None:
    """Enqueue prefix-k reconstruction (see include/rrq.h)."""
    st = load_library().rrq_reconstruct(_ptr(codes), _ptr(scales), _ptr(zeros), rows, cols,
                                        group_size, n_stages, k_stages, _ptr(W_out),
                                        out_dtype, _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_reconstruct")


def rrq_linear(codes, scales, zeros, rows: int, cols: int, group_size: int, n_stages: int,
               k_stages: int, X, n_tokens: int, Y, stream=None) -> None:
    """Enqueue Y = X W~_(k)^T on a package (see include/rrq.h)."""
    st = load_library().rrq_linear(_ptr(codes), _ptr(scales), _ptr(zeros), rows, cols,
                                   group_size, n_stages, k_stages, _ptr(X), n_tokens, _ptr(Y),
                                   _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_linear")


class RrqTensor(ctypes.Structure):
    """One descriptor of rrq_construct_many (struct rrq_tensor of rrq.h)."""
    _fields_ = [("W", ctypes.c_void_p), ("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("zeros", ctypes.c_void_p), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64)]


def rrq_construct_many(tensors, group_size: int, n_stages: int, stream=None) -> None:
    """rrq_construct_many over a list of (W, rows, cols, codes, scales, zeros)
    tuples (device tensors or addresses): each tensor into its own package,
    in as few launches as the C ABI takes."""
    import numpy as np
    # struct rrq_tensor is four pointers and two int64: six 8-byte words
    desc = np.array([(_ptr(W) or 0, _ptr(codes) or 0, _ptr(scales) or 0, _ptr(zeros) or 0,
                      int(rows), int(cols))
                     for W, rows, cols, codes, scales, zeros in tensors],
                    dtype=np.uint64).reshape(-1, 6)
    assert ctypes.sizeof(RrqTensor) == 48
    st = load_library().rrq_construct_many(desc.ctypes.data if tensors else None, len(tensors),
                                           group_size, n_stages, _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_construct_many")


def rrq_construct_format(W, rows: int, cols: int, group_size: int, n_stages: int,
                         zero_point: int, scale_type: int, codes, scales, zeros,
                         stream=None) -> None:
    """Enqueue package construction in a stage format (see include/rrq.h)."""
    st = load_library().rrq_construct_format(_ptr(W), rows, cols, group_size, n_stages,
                                             zero_point, scale_type, _ptr(codes), _ptr(scales),
                                             _ptr(zeros), _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_construct_format")


def rrq_construct_stats(W, rows: int, cols: int, group_size: int, n_stages: int,
                        zero_point: int, scale_type: int, codes, scales, zeros, pmr,
                        stream=None) -> None:
    """Enqueue construction plus the per-group peak-to-mean ratios of W."""
    st = load_library().rrq_construct_stats(_ptr(W), rows, cols, group_size, n_stages,
                                            zero_point, scale_type, _ptr(codes), _ptr(scales),
                                            _ptr(zeros), _ptr(pmr), _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_construct_stats")


def rrq_group_pmr(W, rows: int, cols: int, group_size: int, pmr, stream=None) -> None:
    """Enqueue the per-group peak-to-mean ratios of W."""
    st = load_library().rrq_group_pmr(_ptr(W), rows, cols, group_size, _ptr(pmr), _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_group_pmr")


def rrq_construct_from_base_format(W, rows: int, cols: int, group_size: int, n_stages: int,
                                   zero_point: int, scale_type: int, codes, scales, zeros,
                                   stream=None) -> None:
    """Enqueue the residual stages on a base stage in a stage format."""
    st = load_library().rrq_construct_from_base_format(
        _ptr(W), rows, cols, group_size, n_stages, zero_point, scale_type, _ptr(codes),
        _ptr(scales), _ptr(zeros), _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_construct_from_base_format")


def rrq_reconstruct_format(codes, scales, zeros, rows: int, cols: int, group_size: int,
                           n_stages: int, zero_point: int, scale_type: int, k_stages: int,
                           W_out, out_dtype: int, stream=None) -> None:
    """Enqueue prefix-k reconstruction of a package in a stage format."""
    st = load_library().rrq_reconstruct_format(_ptr(codes), _ptr(scales), _ptr(zeros), rows,
                                               cols, group_size, n_stages, zero_point,
                                               scale_type, k_stages, _ptr(W_out), out_dtype,
                                               _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_reconstruct_format")


def rrq_linear_format(codes, scales, zeros, rows: int, cols: int, group_size: int,
                      n_stages: int, zero_point: int, scale_type: int, k_stages: int, X,
                      n_tokens: int, Y, stream=None) -> None:
    """Enqueue Y = X W~_(k)^T on a package in a stage format."""
    st = load_library().rrq_linear_format(_ptr(codes), _ptr(scales), _ptr(zeros), rows, cols,
                                          group_size, n_stages, zero_point, scale_type,
                                          k_stages, _ptr(X), n_tokens, _ptr(Y), _stream(stream))
    if st != RRQ_OK:
        raise RRQError(st, "rrq_linear_format")


# ---------------------------------------------------------------------------
# Tensor-level helpers (allocation + the calls above)
# ---------------------------------------------------------------------------

def _check_device_tensor(t, name, dtype):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU device, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")


def construct(W, group_size: int = 128, n_stages: int = 4, stream=None, out=None):
    """RRQ package of a bfloat16 matrix W [rows, cols] (cuda, contiguous).

    Returns (codes int32 [S, N/16] holding the uint32 words, scales float32
    [S, N/G], zeros float32 [S, N/G]). ``out`` may pass preallocated buffers.
    """
    import torch
    _check_device_tensor(W, "W", torch.bfloat16)
    rows, cols = (W.shape[0], W.shape[1]) if W.dim() == 2 else (1, W.numel())
    n = rows * cols
    if out is None:
        codes = torch.empty((n_stages, n // 16), dtype=torch.int32, device=W.device)
        scales = torch.empty((n_stages, n // group_size), dtype=torch.float32, device=W.device)
        zeros = torch.empty((n_stages, n // group_size), dtype=torch.float32, device=W.device)
    else:
        codes, scales, zeros = out
    rrq_construct(W, rows, cols, group_size, n_stages, codes, scales, zeros, stream)
    return codes, scales, zeros


def construct_from_base(W, base_codes, base_scales, base_zeros, group_size: int = 128,
                        n_stages: int = 4, stream=None):
    """RRQ package of a bfloat16 matrix W [rows, cols] on an existing base
    stage (base_codes int32 [N/16] holding uint32 words, base_scales and
    base_zeros float32 [N/G], all on W's device). Allocates the package,
    copies the base into plane 0 and builds planes 1 .. S-1 on the GPU.
    Returns (codes, scales, zeros) as ``construct`` does."""
    import torch
    _check_device_tensor(W, "W", torch.bfloat16)
    rows, cols = (W.shape[0], W.shape[1]) if W.dim() == 2 else (1, W.numel())
    n = rows * cols
    codes = torch.empty((n_stages, n // 16), dtype=torch.int32, device=W.device)
    scales = torch.empty((n_stages, n // group_size), dtype=torch.float32, device=W.device)
    zeros = torch.empty((n_stages, n // group_size), dtype=torch.float32, device=W.device)
    codes[0].copy_(base_codes.reshape(-1).view(torch.int32))
    scales[0].copy_(base_scales.reshape(-1))
    zeros[0].copy_(base_zeros.reshape(-1))
    rrq_construct_from_base(W, rows, cols, group_size, n_stages, codes, scales, zeros, stream)
    return codes, scales, zeros


def reconstruct(codes, scales, zeros, rows: int, cols: int, group_size: int, k_stages: int,
                out_dtype=None, stream=None, out=None):
    """Prefix-k effective weight [rows, cols] as float32 or bfloat16."""
    import torch
    out_dtype = torch.bfloat16 if out_dtype is None else out_dtype
    code = {torch.float32: RRQ_F32, torch.bfloat16: RRQ_BF16}[out_dtype]
    n_stages = codes.shape[0]
    if out is None:
        out = torch.empty((rows, cols), dtype=out_dtype, device=codes.device)
    rrq_reconstruct(codes, scales, zeros, rows, cols, group_size, n_stages, k_stages, out, code,
                    stream)
    return out


def linear(X, codes, scales, zeros, rows: int, cols: int, group_size: int, k_stages: int,
           stream=None, out=None):
    """Y = X W~_(k)^T (float32 [n_tokens, rows]) for bfloat16 X [n_tokens, cols]."""
    import torch
    _check_device_tensor(X, "X", torch.bfloat16)
    n_tokens = X.numel() // cols
    if out is None:
        out = torch.empty((n_tokens, rows), dtype=torch.float32, device=X.device)
    rrq_linear(codes, scales, zeros, rows, cols, group_size, codes.shape[0], k_stages, X,
               n_tokens, out, stream)
    return out


def construct_format(W, group_size: int = 128, n_stages: int = 4, zero_point: str = "int",
                     scale_type: str = "f32", stream=None):
    """Package of a bfloat16 matrix in a stage format ("int" / "real" / "sym"
    zero-points, "f32" / "f16" / "bf16" scales). Returns (codes int32,
    scales float32 or int16 holding 16-bit patterns, zeros float32 or None
    for symmetric stages)."""
    import torch
    _check_device_tensor(W, "W", torch.bfloat16)
    rows, cols = (W.shape[0], W.shape[1]) if W.dim() == 2 else (1, W.numel())
    n = rows * cols
    codes = torch.empty((n_stages, n // 16), dtype=torch.int32, device=W.device)
    scales = torch.empty((n_stages, n // group_size),
                         dtype=torch.float32 if scale_type == "f32" else torch.int16,
                         device=W.device)
    zeros = (None if zero_point == "sym" else
             torch.empty((n_stages, n // group_size), dtype=torch.float32, device=W.device))
    rrq_construct_format(W, rows, cols, group_size, n_stages, ZERO_POINTS[zero_point],
                         SCALE_TYPES[scale_type], codes, scales, zeros, stream)
    return codes, scales, zeros


def reconstruct_format(codes, scales, zeros, rows: int, cols: int, group_size: int,
                       k_stages: int, zero_point: str = "int", scale_type: str = "f32",
                       out_dtype=None, stream=None):
    """Prefix-k effective weight of a package in a stage format."""
    import torch
    out_dtype = torch.bfloat16 if out_dtype is None else out_dtype
    code = {torch.float32: RRQ_F32, torch.bfloat16: RRQ_BF16}[out_dtype]
    out = torch.empty((rows, cols), dtype=out_dtype, device=codes.device)
    rrq_reconstruct_format(codes, scales, zeros, rows, cols, group_size, codes.shape[0],
                           ZERO_POINTS[zero_point], SCALE_TYPES[scale_type], k_stages, out, code,
                           stream)
    return out


def group_pmr(W, group_size: int = 128, stream=None):
    """Per-group peak-to-mean ratios (float32 [N/G]) of a bfloat16 tensor."""
    import torch
    _check_device_tensor(W, "W", torch.bfloat16)
    rows, cols = (W.shape[0], W.shape[1]) if W.dim() == 2 else (1, W.numel())
    out = torch.empty(rows * cols // group_size, dtype=torch.float32, device=W.device)
    rrq_group_pmr(W, rows, cols, group_size, out, stream)
    return out

"""Binding of libhbm_probe.so (include/hbm_probe.h): streaming kernels used by
the benchmark as practical HBM ceilings: one with package construction's
read/write ratio (reads B bytes, writes 5B/8), a read-only and a write-only
one, two that replay package construction's and reconstruction's own loads
and stores, and two machine probes (matrix-core and vector instruction
issue, LDS reads) that report clock ticks per wave."""

from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhbm_probe.so")
_lib = None


def load_library() -> ctypes.CDLL:
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
        lib.hbm_probe_stream.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                         ctypes.c_void_p]
        lib.hbm_probe_stream.restype = ctypes.c_int
        lib.hbm_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                       ctypes.c_void_p]
        lib.hbm_probe_read.restype = ctypes.c_int
        lib.hbm_probe_write.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_uint32,
                                        ctypes.c_void_p]
        lib.hbm_probe_write.restype = ctypes.c_int
        lib.hbm_probe_construct.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                            ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
        lib.hbm_probe_construct.restype = ctypes.c_int
        lib.hbm_probe_reconstruct.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                              ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
        lib.hbm_probe_reconstruct.restype = ctypes.c_int
        lib.hbm_probe_issue.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                        ctypes.c_size_t, ctypes.c_void_p, ctypes.c_size_t,
                                        ctypes.c_void_p]
        lib.hbm_probe_issue.restype = ctypes.c_int
        lib.hbm_probe_lds.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t,
                                      ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        lib.hbm_probe_lds.restype = ctypes.c_int
        _lib = lib
    return _lib


def hbm_probe_stream(src, src_bytes: int, dst, stream=None) -> None:
    """Enqueue one probe pass over src (device tensor or address) into dst."""
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    sp = stream if isinstance(stream, int) else stream.cuda_stream
    ptr = lambda x: x if isinstance(x, int) else x.data_ptr()
    st = load_library().hbm_probe_stream(ptr(src), int(src_bytes), ptr(dst), sp)
    if st != 0:
        raise RuntimeError(f"hbm_probe_stream failed with status {st}")


def _sp(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return stream if isinstance(stream, int) else stream.cuda_stream


def _ptr(x):
    return x if isinstance(x, int) else x.data_ptr()


def hbm_probe_read(src, src_bytes: int, out, stream=None) -> None:
    """Enqueue one read-only pass over src; XORs the XOR of its words into out[0]."""
    st = load_library().hbm_probe_read(_ptr(src), int(src_bytes), _ptr(out), _sp(stream))
    if st != 0:
        raise RuntimeError(f"hbm_probe_read failed with status {st}")


def hbm_probe_write(dst, dst_bytes: int, value: int, stream=None) -> None:
    """Enqueue one write-only pass filling dst with the 32-bit value."""
    st = load_library().hbm_probe_write(_ptr(dst), int(dst_bytes), int(value) & 0xFFFFFFFF,
                                        _sp(stream))
    if st != 0:
        raise RuntimeError(f"hbm_probe_write failed with status {st}")


def hbm_probe_construct(W, n_groups: int, group_size: int, n_stages: int, codes, scales, zeros,
                        blocks_per_cu: int = 0, stream=None) -> None:
    """Enqueue one pass with construction's memory traffic (see
    include/hbm_probe.h for what it stores)."""
    st = load_library().hbm_probe_construct(_ptr(W), int(n_groups), int(group_size),
                                            int(n_stages), _ptr(codes), _ptr(scales),
                                            _ptr(zeros), int(blocks_per_cu), _sp(stream))
    if st != 0:
        raise RuntimeError(f"hbm_probe_construct failed with status {st}")


def hbm_probe_reconstruct(codes, scales, zeros, n_groups: int, group_size: int, k_stages: int,
                          out, blocks_per_cu: int = 0, stream=None) -> None:
    """Enqueue one pass with reconstruction's memory traffic, bfloat16 out
    (see include/hbm_probe.h for what it stores)."""
    st = load_library().hbm_probe_reconstruct(_ptr(codes), _ptr(scales), _ptr(zeros),
                                              int(n_groups), int(group_size), int(k_stages),
                                              _ptr(out), int(blocks_per_cu), _sp(stream))
    if st != 0:
        raise RuntimeError(f"hbm_probe_reconstruct failed with status {st}")


def hbm_probe_issue(mode: int, waves_per_simd: int, iters: int, out, ticks, stream=None) -> None:
    """Enqueue the issue probe (mode 0: MFMAs, 1: FMAs, 2: both); out holds
    CUs x waves_per_simd x 256 floats, ticks CUs x waves_per_simd x 4 int64."""
    st = load_library().hbm_probe_issue(int(mode), int(waves_per_simd), int(iters), _ptr(out),
                                        int(out.numel()), _ptr(ticks), int(ticks.numel()),
                                        _sp(stream))
    if st != 0:
        raise RuntimeError(f"hbm_probe_issue failed with status {st}")


def hbm_probe_lds(waves_per_cu: int, iters: int, out, ticks, stream=None) -> None:
    """Enqueue the LDS read probe; out holds CUs x waves_per_cu x 64 uint32,
    ticks CUs x waves_per_cu int64."""
    st = load_library().hbm_probe_lds(int(waves_per_cu), int(iters), _ptr(out), int(out.numel()),
                                      _ptr(ticks), int(ticks.numel()), _sp(stream))
    if st != 0:
        raise RuntimeError(f"hbm_probe_lds failed with status {st}")

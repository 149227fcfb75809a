"""The C ABI library: loads, exports every symbol include/rrq.h declares, sizes
packages, and rejects bad arguments with the documented status before doing
any device work. No GPU needed (nothing here reaches a kernel launch)."""

import ctypes
import os
import re

import pytest

import paper_2608_04048_amd as rrq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rrq.h")

FAKE = 0x10000          # aligned, never dereferenced: every case fails validation first
FAKE_MISALIGNED = 0x10004


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rrq_\w+)\s*\(", text)))


def _declared_enums():
    text = open(HEADER).read()
    return dict((k, int(v)) for k, v in re.findall(r"\b(RRQ_[A-Z0-9_]+)\s*=\s*(\d+)", text))


def test_library_exports_every_declared_function():
    lib = rrq.load_library()
    names = _declared_functions()
    assert names == ["rrq_construct", "rrq_construct_format", "rrq_construct_from_base",
                     "rrq_construct_from_base_format", "rrq_construct_many",
                     "rrq_construct_stats", "rrq_group_pmr",
                     "rrq_linear", "rrq_linear_format", "rrq_package_bytes", "rrq_reconstruct",
                     "rrq_reconstruct_format", "rrq_status_string"]
    for name in names:
        assert hasattr(lib, name), name
    out = os.popen(f"nm -D --defined-only {rrq.LIB_PATH}").read()
    exported = set(re.findall(r" T (rrq_\w+)", out))
    assert set(names) <= exported


def test_binding_constants_match_header():
    enums = _declared_enums()
    for name, value in enums.items():
        assert getattr(rrq, name) == value, name
    assert "RRQ_MAX_STAGES 4" in open(HEADER).read()


def test_package_bytes():
    assert rrq.rrq_package_bytes(1024, 1024, 128, 4) == (4 * 1024 * 1024 // 4, 4 * 8192 * 4)
    assert rrq.rrq_package_bytes(4096, 12288, 64, 3) == (3 * 4096 * 12288 // 4, 3 * 4096 * 192 * 4)
    assert rrq.rrq_package_bytes(1, 32, 32, 1) == (8, 4)
    # Qwen3-8B-shaped 36-layer stack as one flat call
    n = 36 * (2 * 4096 * 4096 + 2 * 1024 * 4096 + 3 * 12288 * 4096)
    assert rrq.rrq_package_bytes(n // 4096, 4096, 128, 4) == (n, 4 * (n // 128) * 4)


@pytest.mark.parametrize("args,status", [
    ((1024, 1000, 128, 4), rrq.RRQ_ERR_SHAPE),
    ((0, 1024, 128, 4), rrq.RRQ_ERR_SHAPE),
    ((1024, -128, 128, 4), rrq.RRQ_ERR_SHAPE),
    ((1 << 40, 1 << 40, 128, 4), rrq.RRQ_ERR_SHAPE),
    ((1024, 1024, 96, 4), rrq.RRQ_ERR_GROUP),
    ((1024, 1024, 256, 4), rrq.RRQ_ERR_GROUP),
    ((1024, 1024, 128, 0), rrq.RRQ_ERR_STAGES),
    ((1024, 1024, 128, 5), rrq.RRQ_ERR_STAGES),
])
def test_package_bytes_rejects(args, status):
    with pytest.raises(rrq.RRQError) as ei:
        rrq.rrq_package_bytes(*args)
    assert ei.value.status == status


def _construct_status(W=FAKE, rows=64, cols=128, G=128, S=4, codes=FAKE, scales=FAKE, zeros=FAKE):
    lib = rrq.load_library()
    return lib.rrq_construct(W, rows, cols, G, S, codes, scales, zeros, None)


def _reconstruct_status(codes=FAKE, scales=FAKE, zeros=FAKE, rows=64, cols=128, G=128, S=4, k=4,
                        out=FAKE, dt=rrq.RRQ_BF16):
    lib = rrq.load_library()
    return lib.rrq_reconstruct(codes, scales, zeros, rows, cols, G, S, k, out, dt, None)


@pytest.mark.parametrize("kw,status", [
    (dict(W=None), rrq.RRQ_ERR_NULL),
    (dict(codes=None), rrq.RRQ_ERR_NULL),
    (dict(scales=None), rrq.RRQ_ERR_NULL),
    (dict(zeros=None), rrq.RRQ_ERR_NULL),
    (dict(G=16), rrq.RRQ_ERR_GROUP),
    (dict(S=0), rrq.RRQ_ERR_STAGES),
    (dict(S=5), rrq.RRQ_ERR_STAGES),
    (dict(cols=100), rrq.RRQ_ERR_SHAPE),
    (dict(rows=0), rrq.RRQ_ERR_SHAPE),
    (dict(rows=1 << 62, cols=128), rrq.RRQ_ERR_SHAPE),
    (dict(W=FAKE + 8), rrq.RRQ_ERR_ALIGN),
    (dict(codes=FAKE_MISALIGNED), rrq.RRQ_ERR_ALIGN),
    (dict(scales=FAKE + 2), rrq.RRQ_ERR_ALIGN),
    (dict(zeros=FAKE + 1), rrq.RRQ_ERR_ALIGN),
])
def test_construct_rejects(kw, status):
    assert _construct_status(**kw) == status


def _from_base_status(W=FAKE, rows=64, cols=128, G=128, S=4, codes=FAKE, scales=FAKE, zeros=FAKE):
    lib = rrq.load_library()
    return lib.rrq_construct_from_base(W, rows, cols, G, S, codes, scales, zeros, None)


@pytest.mark.parametrize("kw,status", [
    (dict(W=None), rrq.RRQ_ERR_NULL),
    (dict(codes=None), rrq.RRQ_ERR_NULL),
    (dict(scales=None), rrq.RRQ_ERR_NULL),
    (dict(zeros=None), rrq.RRQ_ERR_NULL),
    (dict(G=16), rrq.RRQ_ERR_GROUP),
    (dict(S=0), rrq.RRQ_ERR_STAGES),
    (dict(S=5), rrq.RRQ_ERR_STAGES),
    (dict(cols=100), rrq.RRQ_ERR_SHAPE),
    (dict(rows=0), rrq.RRQ_ERR_SHAPE),
    (dict(rows=1 << 62, cols=128), rrq.RRQ_ERR_SHAPE),
    (dict(W=FAKE + 8), rrq.RRQ_ERR_ALIGN),
    (dict(codes=FAKE_MISALIGNED), rrq.RRQ_ERR_ALIGN),
    (dict(scales=FAKE + 2), rrq.RRQ_ERR_ALIGN),
    (dict(zeros=FAKE + 1), rrq.RRQ_ERR_ALIGN),
])
def test_construct_from_base_rejects(kw, status):
    assert _from_base_status(**kw) == status


def _many_status(tensors, n=None, G=128, S=4):
    arr = (rrq.RrqTensor * max(1, len(tensors)))()
    for i, t in enumerate(tensors):
        arr[i] = rrq.RrqTensor(*t)
    n = len(tensors) if n is None else n
    p = ctypes.cast(arr, ctypes.c_void_p) if tensors else None
    return rrq.load_library().rrq_construct_many(p, n, G, S, None)


GOOD = (FAKE, FAKE, FAKE, FAKE, 64, 128)


@pytest.mark.parametrize("bad,status", [
    ((0, FAKE, FAKE, FAKE, 64, 128), rrq.RRQ_ERR_NULL),
    ((FAKE, 0, FAKE, FAKE, 64, 128), rrq.RRQ_ERR_NULL),
    ((FAKE, FAKE, 0, FAKE, 64, 128), rrq.RRQ_ERR_NULL),
    ((FAKE, FAKE, FAKE, 0, 64, 128), rrq.RRQ_ERR_NULL),
    ((FAKE + 8, FAKE, FAKE, FAKE, 64, 128), rrq.RRQ_ERR_ALIGN),
    ((FAKE, FAKE + 4, FAKE, FAKE, 64, 128), rrq.RRQ_ERR_ALIGN),
    ((FAKE, FAKE, FAKE + 2, FAKE, 64, 128), rrq.RRQ_ERR_ALIGN),
    ((FAKE, FAKE, FAKE, FAKE + 1, 64, 128), rrq.RRQ_ERR_ALIGN),
    ((FAKE, FAKE, FAKE, FAKE, 0, 128), rrq.RRQ_ERR_SHAPE),
    ((FAKE, FAKE, FAKE, FAKE, 64, 100), rrq.RRQ_ERR_SHAPE),
])
def test_construct_many_rejects_any_bad_descriptor(bad, status):
    """Every descriptor is checked before anything is enqueued: a bad one
    anywhere in the list (here the last of 70, past the first launch's 64)
    fails the whole call (no GPU is touched by these checks)."""
    assert _many_status([GOOD] * 69 + [bad]) == status
    assert _many_status([bad]) == status


def test_construct_many_arguments():
    assert _many_status([], n=0) == rrq.RRQ_OK            # nothing to do, nothing enqueued
    assert rrq.load_library().rrq_construct_many(None, 3, 128, 4, None) == rrq.RRQ_ERR_NULL
    assert _many_status([GOOD], n=-1) == rrq.RRQ_ERR_SHAPE
    assert _many_status([GOOD], G=96) == rrq.RRQ_ERR_GROUP
    assert _many_status([GOOD], S=5) == rrq.RRQ_ERR_STAGES
    assert _many_status([GOOD], S=0) == rrq.RRQ_ERR_STAGES


def test_construct_from_base_single_stage_is_a_no_op():
    """n_stages = 1: the package is the base alone; the call succeeds after
    validation and enqueues nothing (the fake pointers are never touched and
    no device is needed)."""
    assert _from_base_status(S=1) == rrq.RRQ_OK
    assert _from_base_status(S=1, codes=FAKE_MISALIGNED) == rrq.RRQ_ERR_ALIGN


@pytest.mark.parametrize("kw,status", [
    (dict(codes=None), rrq.RRQ_ERR_NULL),
    (dict(out=None), rrq.RRQ_ERR_NULL),
    (dict(G=48), rrq.RRQ_ERR_GROUP),
    (dict(S=5, k=1), rrq.RRQ_ERR_STAGES),
    (dict(k=0), rrq.RRQ_ERR_STAGES),
    (dict(S=2, k=3), rrq.RRQ_ERR_STAGES),
    (dict(dt=2), rrq.RRQ_ERR_DTYPE),
    (dict(cols=130), rrq.RRQ_ERR_SHAPE),
    (dict(out=FAKE + 4), rrq.RRQ_ERR_ALIGN),
    (dict(codes=FAKE + 4), rrq.RRQ_ERR_ALIGN),
])
def test_reconstruct_rejects(kw, status):
    assert _reconstruct_status(**kw) == status


def test_status_strings():
    for st in range(9):
        s = rrq.rrq_status_string(st)
        assert isinstance(s, str) and s
    assert rrq.rrq_status_string(0) == "success"
    assert rrq.rrq_status_string(99) == "unknown status"


def test_binding_raises_on_error():
    with pytest.raises(rrq.RRQError) as ei:
        rrq.rrq_construct(FAKE, 64, 128, 128, 9, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == rrq.RRQ_ERR_STAGES


def test_product_does_not_import_oracle():
    """The HIP path and the oracle share no code: nothing in the package or
    its C++ sources refers to oracle/."""
    pkg = os.path.join(ROOT, "paper_2608_04048_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "rrq_oracle" not in text, f


PROBE_HEADER = os.path.join(ROOT, "include", "hbm_probe.h")


def test_probe_library_exports_declared_function():
    from paper_2608_04048_amd import probe
    text = re.sub(r"/\*.*?\*/", "", open(PROBE_HEADER).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(hbm_probe_\w+)\s*\(", text)))
    assert names == ["hbm_probe_construct", "hbm_probe_issue", "hbm_probe_lds",
                     "hbm_probe_read", "hbm_probe_reconstruct", "hbm_probe_stream",
                     "hbm_probe_write"]
    lib = probe.load_library()
    out = os.popen(f"nm -D --defined-only {probe.LIB_PATH}").read()
    for name in names:
        assert hasattr(lib, name)
        assert f" T {name}" in out


@pytest.mark.parametrize("src,nbytes,dst,status", [
    (0, 1024, FAKE, 1),
    (FAKE, 1024, 0, 1),
    (FAKE_MISALIGNED, 1024, FAKE, 2),
    (FAKE, 1024, FAKE_MISALIGNED, 2),
    (FAKE, 0, FAKE, 3),
    (FAKE, 1000, FAKE, 3),
])
def test_probe_rejects(src, nbytes, dst, status):
    from paper_2608_04048_amd import probe
    assert probe.load_library().hbm_probe_stream(src, nbytes, dst, None) == status


@pytest.mark.parametrize("src,nbytes,out,status", [
    (0, 1024, FAKE, 1),
    (FAKE, 1024, 0, 1),
    (FAKE + 8, 1024, FAKE, 2),
    (FAKE, 1024, FAKE + 2, 2),
    (FAKE, 0, FAKE, 3),
    (FAKE, 1000, FAKE, 3),
])
def test_read_probe_rejects(src, nbytes, out, status):
    from paper_2608_04048_amd import probe
    assert probe.load_library().hbm_probe_read(src, nbytes, out, None) == status


@pytest.mark.parametrize("dst,nbytes,status", [
    (0, 1024, 1), (FAKE + 8, 1024, 2), (FAKE, 0, 3), (FAKE, 1000, 3),
])
def test_write_probe_rejects(dst, nbytes, status):
    from paper_2608_04048_amd import probe
    assert probe.load_library().hbm_probe_write(dst, nbytes, 0, None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(W=0), 1), (dict(codes=0), 1), (dict(scales=0), 1), (dict(zeros=0), 1),
    (dict(W=FAKE + 8), 2), (dict(codes=FAKE + 4), 2), (dict(scales=FAKE + 2), 2),
    (dict(zeros=FAKE + 1), 2), (dict(G=16), 3), (dict(G=256), 3), (dict(n_groups=0), 3),
    (dict(S=0), 3), (dict(S=5), 3), (dict(bpc=-1), 3), (dict(bpc=33), 3),
])
def test_construct_probe_rejects(kw, status):
    """Argument errors are returned before anything is enqueued (no GPU is
    touched: these checks precede every HIP call)."""
    from paper_2608_04048_amd import probe
    a = dict(W=FAKE, n_groups=64, G=128, S=4, codes=FAKE, scales=FAKE, zeros=FAKE, bpc=0)
    a.update(kw)
    assert probe.load_library().hbm_probe_construct(
        a["W"], a["n_groups"], a["G"], a["S"], a["codes"], a["scales"], a["zeros"], a["bpc"],
        None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(codes=0), 1), (dict(scales=0), 1), (dict(zeros=0), 1), (dict(out=0), 1),
    (dict(codes=FAKE + 4), 2), (dict(out=FAKE + 8), 2), (dict(scales=FAKE + 2), 2),
    (dict(zeros=FAKE + 1), 2), (dict(G=16), 3), (dict(n_groups=0), 3), (dict(k=0), 3),
    (dict(k=5), 3), (dict(bpc=-1), 3), (dict(bpc=33), 3),
])
def test_reconstruct_probe_rejects(kw, status):
    from paper_2608_04048_amd import probe
    a = dict(codes=FAKE, scales=FAKE, zeros=FAKE, n_groups=64, G=128, k=2, out=FAKE, bpc=0)
    a.update(kw)
    assert probe.load_library().hbm_probe_reconstruct(
        a["codes"], a["scales"], a["zeros"], a["n_groups"], a["G"], a["k"], a["out"], a["bpc"],
        None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(out=None), 1), (dict(ticks=None), 1), (dict(mode=3), 3), (dict(mode=-1), 3),
    (dict(wps=0), 3), (dict(wps=5), 3), (dict(iters=0), 3),
])
def test_issue_probe_rejects(kw, status):
    from paper_2608_04048_amd import probe
    a = dict(mode=0, wps=1, iters=1, out=FAKE, ticks=FAKE)
    a.update(kw)
    assert probe.load_library().hbm_probe_issue(a["mode"], a["wps"], a["iters"], a["out"], 1 << 30,
                                                a["ticks"], 1 << 30, None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(out=None), 1), (dict(ticks=None), 1), (dict(wpc=6), 3), (dict(wpc=16), 3),
    (dict(iters=0), 3),
])
def test_lds_probe_rejects(kw, status):
    from paper_2608_04048_amd import probe
    a = dict(wpc=8, iters=1, out=FAKE, ticks=FAKE)
    a.update(kw)
    assert probe.load_library().hbm_probe_lds(a["wpc"], a["iters"], a["out"], 1 << 30, a["ticks"],
                                              1 << 30, None) == status


def _linear_status(codes=FAKE, scales=FAKE, zeros=FAKE, rows=64, cols=128, G=128, S=4, k=4,
                   X=FAKE, M=1, Y=FAKE):
    lib = rrq.load_library()
    return lib.rrq_linear(codes, scales, zeros, rows, cols, G, S, k, X, M, Y, None)


@pytest.mark.parametrize("kw,status", [
    (dict(codes=None), rrq.RRQ_ERR_NULL),
    (dict(X=None), rrq.RRQ_ERR_NULL),
    (dict(Y=None), rrq.RRQ_ERR_NULL),
    (dict(G=48), rrq.RRQ_ERR_GROUP),
    (dict(S=5, k=1), rrq.RRQ_ERR_STAGES),
    (dict(k=0), rrq.RRQ_ERR_STAGES),
    (dict(S=2, k=3), rrq.RRQ_ERR_STAGES),
    (dict(cols=130), rrq.RRQ_ERR_SHAPE),
    (dict(M=0), rrq.RRQ_ERR_SHAPE),
    (dict(rows=1 << 26), rrq.RRQ_ERR_SHAPE),
    (dict(cols=1 << 27), rrq.RRQ_ERR_SHAPE),
    # 4 stage planes of (2^17 x 2^17) / 4 bytes = 4 GiB of codes
    (dict(rows=1 << 17, cols=1 << 17, k=4), rrq.RRQ_ERR_SHAPE),
    (dict(X=FAKE + 8), rrq.RRQ_ERR_ALIGN),
    (dict(codes=FAKE + 4), rrq.RRQ_ERR_ALIGN),
    (dict(Y=FAKE + 2), rrq.RRQ_ERR_ALIGN),
])
def test_linear_rejects(kw, status):
    assert _linear_status(**kw) == status


def _fmt_status(fn, zp=0, sd=0, scales=FAKE, zeros=FAKE, **kw):
    lib = rrq.load_library()
    if fn == "construct":
        return lib.rrq_construct_format(FAKE, 64, 128, 128, 4, zp, sd, FAKE, scales, zeros, None)
    if fn == "from_base":
        return lib.rrq_construct_from_base_format(FAKE, 64, 128, 128, 4, zp, sd, FAKE, scales,
                                                  zeros, None)
    if fn == "reconstruct":
        return lib.rrq_reconstruct_format(FAKE, scales, zeros, 64, 128, 128, 4, zp, sd, 4, FAKE,
                                          rrq.RRQ_BF16, None)
    return lib.rrq_linear_format(FAKE, scales, zeros, 64, 128, 128, 4, zp, sd, 4, FAKE, 1, FAKE,
                                 None)


@pytest.mark.parametrize("fn", ["construct", "from_base", "reconstruct", "linear"])
@pytest.mark.parametrize("kw,status", [
    (dict(zp=3), rrq.RRQ_ERR_FORMAT),
    (dict(zp=-1), rrq.RRQ_ERR_FORMAT),
    (dict(sd=3), rrq.RRQ_ERR_FORMAT),
    (dict(scales=None), rrq.RRQ_ERR_NULL),
    (dict(zeros=None), rrq.RRQ_ERR_NULL),                      # zeros required unless symmetric
    (dict(sd=rrq.RRQ_SCALE_F32, scales=FAKE + 2), rrq.RRQ_ERR_ALIGN),
    (dict(sd=rrq.RRQ_SCALE_F16, scales=FAKE + 1), rrq.RRQ_ERR_ALIGN),
    (dict(zp=rrq.RRQ_ZP_REAL, zeros=FAKE + 2), rrq.RRQ_ERR_ALIGN),
])
def test_format_calls_reject(fn, kw, status):
    assert _fmt_status(fn, **kw) == status


def test_symmetric_allows_null_zeros_and_16bit_scales_at_2_bytes():
    """These argument checks pass (the S = 1 base call then enqueues nothing,
    so no device is needed to see it)."""
    lib = rrq.load_library()
    for sd in (rrq.RRQ_SCALE_F16, rrq.RRQ_SCALE_BF16):
        st = lib.rrq_construct_from_base_format(FAKE, 64, 128, 128, 1, rrq.RRQ_ZP_SYMMETRIC, sd,
                                                FAKE, FAKE + 2, None, None)
        assert st == rrq.RRQ_OK


def test_format_enums_match_header():
    text = open(HEADER).read()
    for name in ("RRQ_ZP_INTEGER", "RRQ_ZP_REAL", "RRQ_ZP_SYMMETRIC", "RRQ_SCALE_F32",
                 "RRQ_SCALE_F16", "RRQ_SCALE_BF16", "RRQ_ERR_FORMAT"):
        m = re.search(name + r"\s*=\s*(\d+)", text)
        assert m and int(m.group(1)) == getattr(rrq, name), name


@pytest.mark.parametrize("kw,status", [
    (dict(W=None), rrq.RRQ_ERR_NULL),
    (dict(pmr=None), rrq.RRQ_ERR_NULL),
    (dict(G=16), rrq.RRQ_ERR_GROUP),
    (dict(cols=100), rrq.RRQ_ERR_SHAPE),
    (dict(W=FAKE + 8), rrq.RRQ_ERR_ALIGN),
    (dict(pmr=FAKE + 2), rrq.RRQ_ERR_ALIGN),
])
def test_group_pmr_rejects(kw, status):
    a = dict(W=FAKE, rows=64, cols=128, G=128, pmr=FAKE)
    a.update(kw)
    assert rrq.load_library().rrq_group_pmr(a["W"], a["rows"], a["cols"], a["G"], a["pmr"], None) == status


def test_construct_stats_requires_pmr():
    lib = rrq.load_library()
    assert lib.rrq_construct_stats(FAKE, 64, 128, 128, 4, 0, 0, FAKE, FAKE, FAKE, None, None) == rrq.RRQ_ERR_NULL
    assert lib.rrq_construct_stats(FAKE, 64, 128, 128, 4, 0, 0, FAKE, FAKE, FAKE, FAKE + 2, None) == rrq.RRQ_ERR_ALIGN
    assert lib.rrq_construct_stats(FAKE, 64, 128, 128, 4, 5, 0, FAKE, FAKE, FAKE, FAKE, None) == rrq.RRQ_ERR_FORMAT

"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point declared in include/opattr.h, sizes its workspace, and
rejects bad arguments before enqueueing anything."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2609_11938_amd import opattr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "opattr.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(opattr.LIB_PATH):
        from paper_2609_11938_amd import build

        build.build()
    return opattr.library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(opattr_[a-z_]+)\s*\(", text)))


def test_header_declares_the_expected_calls():
    assert declared_functions() == sorted(opattr.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", opattr.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    exported = set(re.findall(r"\sT\s(opattr_\w+)", out))
    for f in declared_functions():
        assert f in exported, f
        assert hasattr(lib, f)


def test_struct_layouts_match_header():
    assert C.sizeof(opattr.opattr_kernels) == 64
    assert C.sizeof(opattr.opattr_profiled) == 48
    assert C.sizeof(opattr.opattr_ranges) == 40
    assert C.sizeof(opattr.opattr_dims) == 32
    assert C.sizeof(opattr.opattr_diag) == 64
    assert opattr.OP_ROW_DTYPE.itemsize == 192


def _structs(T=100, P=50, R=10, NN=8, NS=2, NOPS=4, flags=0):
    fake = C.c_void_p(0x1000)  # never dereferenced on the host
    k = opattr.opattr_kernels(T, fake, fake, fake, fake, fake, None, None)
    p = opattr.opattr_profiled(P, fake, fake, 20, 1, 0)
    r = opattr.opattr_ranges(R, fake, fake, fake, fake)
    d = opattr.opattr_dims(NN, NS, NOPS, 0, None, flags)
    return k, p, r, d


def test_workspace_size_is_pure_and_monotone(lib):
    sizes = []
    for T in (0, 1, 4096, 4097, 100_000):
        k, p, r, d = _structs(T=T)
        sizes.append(lib.opattr_workspace_bytes(C.byref(k), C.byref(p), C.byref(r), C.byref(d)))
    assert all(s > 0 for s in sizes)
    assert sizes == sorted(sizes)
    # hints drop the reordering buffers
    k, p, r, d = _structs(T=100_000, R=5_000)
    full = lib.opattr_workspace_bytes(C.byref(k), C.byref(p), C.byref(r), C.byref(d))
    d.flags = opattr.SEQ_DENSE | opattr.RANGES_NESTED
    hinted = lib.opattr_workspace_bytes(C.byref(k), C.byref(p), C.byref(r), C.byref(d))
    assert hinted < full
    assert lib.opattr_workspace_bytes(C.byref(k), C.byref(p), C.byref(r), None) == 0


def test_argument_errors_return_before_any_device_work(lib):
    k, p, r, d = _structs()
    fake = C.c_void_p(0x1000)
    ws = C.c_void_p(0x2000)
    INVALID, WORKSPACE = -1, -2
    # NULL diag / match
    assert lib.opattr_match(C.byref(k), C.byref(p), C.byref(d), 0, fake, None, None, ws,
                            C.c_size_t(1 << 40), None) == INVALID
    assert lib.opattr_match(C.byref(k), C.byref(p), C.byref(d), 0, None, None, fake, ws,
                            C.c_size_t(1 << 40), None) == INVALID
    # policy out of range
    assert lib.opattr_match(C.byref(k), C.byref(p), C.byref(d), 3, fake, None, fake, ws,
                            C.c_size_t(1 << 40), None) == INVALID
    # negative or too large sizes
    k.n = -1
    assert lib.opattr_enclose(C.byref(k), C.byref(r), C.byref(d), fake, None, fake, ws,
                              C.c_size_t(1 << 40), None) == INVALID
    k.n = 1 << 31
    assert lib.opattr_enclose(C.byref(k), C.byref(r), C.byref(d), fake, None, fake, ws,
                              C.c_size_t(1 << 40), None) == INVALID
    k.n = 100
    # too many names, unknown flag bits
    d.n_names = 1 << 20
    assert lib.opattr_match(C.byref(k), C.byref(p), C.byref(d), 0, fake, None, fake, ws,
                            C.c_size_t(1 << 40), None) == INVALID
    d.n_names = 8
    d.flags = 1 << 7
    assert lib.opattr_match(C.byref(k), C.byref(p), C.byref(d), 0, fake, None, fake, ws,
                            C.c_size_t(1 << 40), None) == INVALID
    d.flags = 0
    # missing range arrays
    r2 = opattr.opattr_ranges(10, fake, None, fake, fake)
    assert lib.opattr_enclose(C.byref(k), C.byref(r2), C.byref(d), fake, None, fake, ws,
                              C.c_size_t(1 << 40), None) == INVALID
    # aggregation kinds out of range
    bad_kind = (C.c_uint8 * 20)(*([3] + [0] * 19))
    assert lib.opattr_aggregate(C.byref(k), C.byref(p), fake, fake, C.byref(r), C.byref(d),
                                bad_kind, fake, fake, fake, ws, C.c_size_t(1 << 40),
                                None) == INVALID
    # undersized workspace
    need = lib.opattr_workspace_bytes(C.byref(k), C.byref(p), C.byref(r), C.byref(d))
    assert lib.opattr_attribute(C.byref(k), C.byref(p), C.byref(r), C.byref(d), 0, None, fake,
                                fake, None, None, fake, fake, fake, ws, C.c_size_t(need - 1),
                                None) == WORKSPACE
    # workspace off a 256-byte boundary
    assert lib.opattr_attribute(C.byref(k), C.byref(p), C.byref(r), C.byref(d), 0, None, fake,
                                fake, None, None, fake, fake, fake, C.c_void_p(0x2010),
                                C.c_size_t(need + 256), None) == WORKSPACE
    assert lib.opattr_diag_clear(None, None) == INVALID
    assert lib.opattr_read_diag(None, None, None) == INVALID


def test_strerror_names_every_status():
    for code in range(-10, 1):
        s = opattr.strerror(code)
        assert s and s != "unknown status"
    assert opattr.strerror(-99) == "unknown status"


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError, match="not built"):
        opattr.library(str(tmp_path / "missing.so"))


def test_to_device_rejects_bad_counters():
    tr = dict(counters=np.zeros((2, 20), np.float64))
    with pytest.raises(TypeError):
        opattr.to_device(tr, "cpu")

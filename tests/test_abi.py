"""The C-ABI library loads and exports exactly what include/cel.h declares
(CPU only: no compute call is made)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cel.h")
LIB = os.path.join(ROOT, "paper_2208_00184_amd", "libcel.so")


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(cel_[a-z_]+)\s*\(", src)))


def test_header_declares_the_five_entry_points():
    names = declared()
    for f in ("cel_topo_levels", "cel_blevel", "cel_cluster", "cel_place", "cel_makespan"):
        assert f in names
    assert "cel_last_error" in names and "cel_version" in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="libcel.so not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    for name in declared():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True).stdout
    exported = sorted(set(re.findall(r" T (cel_[a-z_]+)$", out, flags=re.M)))
    assert exported == declared()


@pytest.mark.skipif(not os.path.exists(LIB), reason="libcel.so not built")
def test_version_and_error_text():
    lib = ctypes.CDLL(LIB)
    lib.cel_version.restype = ctypes.c_int
    lib.cel_last_error.restype = ctypes.c_char_p
    assert lib.cel_version() >= 100
    assert isinstance(lib.cel_last_error(), bytes)


@pytest.mark.skipif(not os.path.exists(LIB), reason="libcel.so not built")
def test_host_side_argument_errors_without_gpu():
    """NULL graph / bad D are rejected before any HIP call."""
    lib = ctypes.CDLL(LIB)
    lib.cel_topo_levels.restype = ctypes.c_int
    n_levels = ctypes.c_int32(0)
    rc = lib.cel_topo_levels(None, None, None, None, ctypes.byref(n_levels), None)
    assert rc == -1
    lib.cel_last_error.restype = ctypes.c_char_p
    assert b"NULL" in lib.cel_last_error()


def test_binding_exports_match_header():
    from paper_2208_00184_amd import EXPORTS
    assert sorted(EXPORTS) == declared()

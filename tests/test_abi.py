"""The C-ABI library loads on a machine without a GPU and exports every entry
point that include/aladdin.h declares; the binding mirrors them by name.
No compute call is made here."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aladdin.h")
LIB = os.path.join(ROOT, "paper_2405_06856_amd", "libaladdin.so")


def declared_symbols():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ald_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2405_06856_amd import build
        build.build(verbose=False)
    return ctypes.CDLL(LIB)


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for name in ("ald_load_workers", "ald_place_stream", "ald_sweep_scenarios", "ald_create", "ald_destroy"):
        assert name in syms


def test_library_exports_every_declared_symbol(lib):
    missing = [s for s in declared_symbols() if not hasattr(lib, s)]
    assert not missing, missing


def test_binding_mirrors_the_header(lib):
    from paper_2405_06856_amd import aladdin
    assert set(aladdin.SYMBOLS) == set(declared_symbols())
    for s in declared_symbols():
        assert callable(getattr(aladdin, s))


def test_struct_layouts_match_the_header():
    from paper_2405_06856_amd import aladdin
    assert ctypes.sizeof(aladdin.Model) == 9 * 8 + 2 * 4
    assert ctypes.sizeof(aladdin.Scenario) == 16 + ctypes.sizeof(aladdin.Model)
    assert aladdin.DIAG_DTYPE.itemsize == 40


def test_error_strings_without_a_device(lib):
    lib.ald_strerror.restype = ctypes.c_char_p
    for code in (0, -1, -2, -3, -4, -5):
        assert lib.ald_strerror(code)
    # calls on a null handle fail cleanly instead of touching a device
    lib.ald_set_tile.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    assert lib.ald_set_tile(None, 128) == -1
    lib.ald_destroy.argtypes = [ctypes.c_void_p]
    assert lib.ald_destroy(None) == 0

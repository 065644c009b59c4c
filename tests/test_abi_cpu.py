"""C ABI checks that need no GPU: the library loads and exports every entry point that
include/acespec.h declares (no compute call is made here)."""
import ctypes
import os
import re

import paper_2609_02514_amd.acespec as A

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "acespec.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(acespec_[a-z_]+)\s*\(", src)))


def test_header_declares_the_bound_entry_points():
    assert declared_symbols() == sorted(A.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(A.LIB_PATH)
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_struct_layouts_match_the_header():
    # sizes of the plain structs as laid out by the C compiler on x86-64
    assert ctypes.sizeof(A.ModelDesc) == 40
    assert ctypes.sizeof(A.LayerWeights) == 48
    assert ctypes.sizeof(A.Weights) == 32
    assert ctypes.sizeof(A.KVCache) == 32
    assert ctypes.sizeof(A.Params) == 12
    assert ctypes.sizeof(A.Outputs) == 96


def test_last_error_starts_empty():
    assert A.acespec_last_error() == ""

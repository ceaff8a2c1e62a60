"""The C ABI library loads on a host without a GPU and exports every symbol
that include/nmspmm.h declares (no compute call is made here)."""
import ctypes
import os
import re

from paper_2607_12505_amd import nmspmm

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "nmspmm.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(nm_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_binding_names():
    assert declared_functions() == sorted(nmspmm.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(nmspmm.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings():
    for s in range(7):
        assert nmspmm.status_string(s)
    assert nmspmm.status_string(0) == "ok"
    assert nmspmm.status_string(99) == "unknown status"


def test_struct_sizes_match_header():
    # nm_desc: 8 int32 + 2 int64 + 2 int32 = 56 bytes; nm_plan: 6 int32
    assert ctypes.sizeof(nmspmm.NmDesc) == 56
    assert ctypes.sizeof(nmspmm.NmPlan) == 24

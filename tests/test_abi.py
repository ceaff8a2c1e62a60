"""The C ABI library loads on a host without a GPU and exports every symbol
that the headers under include/ declare (no GPU compute call is made here)."""
import ctypes
import glob
import os
import re

from paper_2607_12505_amd import nmsearch, nmspmm

HEADERS = sorted(glob.glob(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                                        "*.h")))


def declared_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(nm_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_header_declares_the_binding_names():
    assert len(HEADERS) == 2
    assert declared_functions() == sorted(nmspmm.EXPORTED + nmsearch.EXPORTED)


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
    # nm_outputs: 5 pointers; nm_search_params: 4 int32 + 1 uint64
    assert ctypes.sizeof(nmspmm.NmOutputs) == 40
    assert ctypes.sizeof(nmsearch.NmSearchParams) == 24

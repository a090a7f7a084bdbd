"""The C ABI library loads on the CPU host and exports every entry point the header
declares; host-only sizing functions follow their documented argument checks."""
import ctypes as C
import os
import re

import pytest

from paper_2403_04311_amd import alto

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "alto.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(alto_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("alto_route", "alto_aggregate", "alto_stream_step", "alto_pack_keys",
              "alto_workspace_bytes", "alto_stream_create", "alto_stream_pending"):
        assert n in names


def test_library_exports_every_declared_symbol():
    if not os.path.exists(alto.LIB_PATH):
        pytest.fail("libalto.so is not built (run __graft_entry__.build())")
    lib = C.CDLL(alto.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert set(alto.EXPORTS) <= set(declared_functions())


def test_workspace_sizing_host_checks():
    lib = alto.load()
    ok = alto.workspace_bytes((31, 2, 3, 4), 10000, 8, 3, "concat")
    assert ok > 0
    assert alto.workspace_bytes((31, 2, 3, 4), 10000, 8) > 0
    assert alto.workspace_bytes((40, 30), 100, 8) == 0            # wider than 63 bits
    assert alto.workspace_bytes((31, 2, 3, 4), -1, 8) == 0
    assert alto.workspace_bytes((31, 2, 3, 4), 100, 0) == 0
    assert alto.workspace_bytes((31, 2, 3, 4), 100, 8, 4, "concat") == 0   # La must be < depth
    L = alto.layout((31, 6, 12))
    A = alto.agg_struct(2, "concat")
    assert lib.alto_stream_state_bytes(C.byref(L), C.byref(A), 1 << 12, 1 << 14) > 0
    A.mask_level = 1
    assert lib.alto_stream_state_bytes(C.byref(L), C.byref(A), 1 << 12, 1 << 14) == 0
    # growing with the sizes it is given
    assert alto.workspace_bytes((31, 2, 3, 4), 1 << 20, 8, 3, "concat") > ok

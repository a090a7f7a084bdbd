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


def test_join_split_router_sizing_host_checks():
    lib = alto.load()
    L = alto.layout((31, 6, 12))
    assert lib.alto_join_workspace_bytes(C.byref(L), 1000) > 0
    assert lib.alto_join_workspace_bytes(C.byref(L), -1) == 0
    assert lib.alto_join_workspace_bytes(C.byref(L), 1 << 20) > lib.alto_join_workspace_bytes(C.byref(L), 1000)
    # split: the input layout gains a level, so at most 15 input levels
    assert lib.alto_split_workspace_bytes(C.byref(alto.layout((31, 18))), 1000) > 0
    assert lib.alto_split_workspace_bytes(C.byref(alto.layout((31, 18))), -1) == 0
    assert lib.alto_split_workspace_bytes(C.byref(alto.layout((2,) * 15)), 10) > 0
    assert lib.alto_split_workspace_bytes(C.byref(alto.layout((2,) * 16)), 10) == 0
    assert lib.alto_split_workspace_bytes(C.byref(alto.layout((40, 30))), 10) == 0   # wider than 63 bits
    # load-aware routing
    assert lib.alto_router_state_bytes(0) == 0
    assert 0 < lib.alto_router_state_bytes(1) < lib.alto_router_state_bytes(1 << 20)
    assert lib.alto_route_load_workspace_bytes(C.byref(L), 2, 1 << 16, 64) > 0
    for Lr, n, D in [(0, 100, 4), (4, 100, 4), (2, -1, 4), (2, 100, 0), (2, 100, 4097)]:
        assert lib.alto_route_load_workspace_bytes(C.byref(L), Lr, n, D) == 0, (Lr, n, D)
    h = C.c_void_p()
    # bad arguments are refused on the host, before anything is enqueued
    assert lib.alto_router_create(C.byref(L), 2, 4, 16, None, 0, None, C.byref(h)) == 1
    assert lib.alto_route_load(None, None, 0, None, None, None, None, None, None, None, 0, None) == 1
    assert lib.alto_read_probe(None, 16, None, None) == 1


# ---- host-side checks of the Python binding: tensors that would make a kernel read
# or write out of bounds are refused before anything reaches the library

def _err(fn, *a, **k):
    with pytest.raises(alto.AltoError) as e:
        fn(*a, **k)
    assert e.value.code == alto.E_ARG
    return str(e.value)


def test_binding_refuses_bad_tensors_for_aggregate():
    import torch
    bits = (6, 3, 2, 3, 5)
    n = 10
    keys = torch.zeros(n, dtype=torch.int64)
    fan = torch.ones((4, n), dtype=torch.int32)
    pf = torch.zeros((n, 8), dtype=torch.float32)
    p32 = torch.zeros(n, dtype=torch.int32)
    kw = dict(bits=bits, agg_level=4, op="mean", dim=8)
    assert "keys has dtype" in _err(alto.aggregate, keys.to(torch.int32), fan, payload_f32=pf, **kw)
    assert "fan is" in _err(alto.aggregate, keys, fan[:3], payload_f32=pf, **kw)            # too few levels
    assert "fan is" in _err(alto.aggregate, keys, fan[:, :5], payload_f32=pf, **kw)         # too few fragments
    assert "unit stride" in _err(alto.aggregate, keys, fan.t().contiguous().t(), payload_f32=pf, **kw)
    assert "payload_f32 holds" in _err(alto.aggregate, keys, fan, payload_f32=pf[:5], **kw)
    assert "rows hold" in _err(alto.aggregate, keys, fan, payload_f32=pf.reshape(n * 2, 4), **kw)
    assert "contiguous" in _err(alto.aggregate, keys, fan, payload_f32=pf.t(), **kw)
    assert "payload_f32 is required" in _err(alto.aggregate, keys, fan, **kw)
    assert "payload_i32 is required" in _err(alto.aggregate, keys, fan, bits=bits, agg_level=4, op="concat")
    out = alto.new_groups(n, 4, "mean", 8, device="cpu")
    out.mean = out.mean[:3]
    assert "out.mean holds" in _err(alto.aggregate, keys, fan, payload_f32=pf, out=out, **kw)
    out = alto.new_groups(n, 4, "concat", 1, cap_tokens=n, device="cpu")
    out.tok = out.tok[: n - 1]
    assert "out.tok holds" in _err(alto.aggregate, keys, fan, bits=bits, agg_level=4, op="concat",
                                   payload_i32=p32, out=out)
    assert "perm holds" in _err(alto.aggregate, keys, fan, payload_f32=pf, perm=torch.zeros(3, dtype=torch.int32),
                                **kw)
    assert "dest_offsets holds" in _err(alto.aggregate, keys, fan, payload_f32=pf, route_level=2, num_dest=8,
                                        dest_offsets=torch.zeros(8, dtype=torch.int64), **kw)
    # well-formed host tensors get as far as the device check
    assert "not on a GPU" in _err(alto.aggregate, keys, fan, payload_f32=pf, **kw)


def test_binding_refuses_bad_tensors_for_route_join_split_pack():
    import torch
    n = 16
    keys = torch.zeros(n, dtype=torch.int64)
    assert "keys has dtype" in _err(alto.route, keys.float(), (31, 6, 12), 2, 4)
    assert "perm holds" in _err(alto.route, keys, (31, 6, 12), 2, 4, perm=torch.zeros(2, dtype=torch.int32))
    assert "not on a GPU" in _err(alto.route, keys, (31, 6, 12), 2, 4)
    assert "match holds" in _err(alto.join, keys[:4], keys, (31, 6, 12), 2, match=torch.zeros(3, dtype=torch.int32))
    assert "not on a GPU" in _err(alto.join, keys[:4], keys, (31, 6, 12), 2)
    fan = torch.ones((2, n), dtype=torch.int32)
    tok = torch.zeros(n, dtype=torch.int32)
    assert "tokens holds" in _err(alto.split, keys, fan, tok[:3], (31, 6, 12), 0, 4, 4)
    assert "out_fan is" in _err(alto.split, keys, fan, tok, (31, 6, 12), 0, 4, 4,
                                out_fan=torch.zeros((2, n), dtype=torch.int32))
    assert "not on a GPU" in _err(alto.split, keys, fan, tok, (31, 6, 12), 0, 4, 4)
    path = torch.zeros((2, n), dtype=torch.int32)
    assert "path is" in _err(alto.pack_keys, path, (31, 6, 12))
    assert "not on a GPU" in _err(alto.pack_keys, torch.zeros((3, n), dtype=torch.int32), (31, 6, 12))


def test_noalloc_entry_point_refuses_inputs_larger_than_its_array():
    # refused on the host, before anything is enqueued or any device is touched
    bits = (3, 12, 12, 12, 12, 12)
    n = 1 << 21
    assert alto.workspace_bytes(bits, n, 256, 4, "mean", 128, 2) > alto.NOALLOC_SCRATCH_BYTES
    lib = alto.load()
    L, A = alto.layout(bits), alto.agg_struct(4, "mean", 128, 2)
    G = alto.Groups()
    rc = lib.alto_aggregate_noalloc(None, None, n, None, None, n, C.byref(L), C.byref(A), 4, 256,
                                    None, None, None, C.byref(G), None, None)
    assert rc == alto.E_ARG
    import torch
    small = 1000
    assert "more than the fixed" in _err(alto.aggregate_noalloc, torch.zeros(n, dtype=torch.int64),
                                         torch.ones((5, n), dtype=torch.int32), bits, 4, "mean", 128, 2, 4, 256,
                                         payload_f32=torch.zeros((n, 128)),
                                         perm=torch.zeros(n, dtype=torch.int32),
                                         dest_offsets=torch.zeros(257, dtype=torch.int64),
                                         dest=torch.zeros(n, dtype=torch.int32),
                                         out=alto.new_groups(small, 4, "mean", 128, cap_mask=small, device="cpu"),
                                         status=torch.zeros(1, dtype=torch.int32))

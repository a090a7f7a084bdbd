"""Python binding of libalto (argument marshalling only).

Every step of routing and aggregation runs in the HIP kernels of ``libalto.so``;
this module only converts torch tensors (device memory) and torch's current HIP
stream into the C ABI of ``include/alto.h``, and allocates output tensors for
convenience. It raises if the library is missing: there is no CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libalto.so")

OK, E_ARG, E_LAYOUT, E_DUPLICATE, E_FANOUT, E_LATE, E_CAPACITY, E_HIP = range(8)
CONCAT_I32, MEAN_F32 = 0, 1
RELEASE = {"complete": 0, "in_order": 1}
STATUS_NAMES = {0: "OK", 1: "ARG", 2: "LAYOUT", 3: "DUPLICATE", 4: "FANOUT", 5: "LATE",
                6: "CAPACITY", 7: "HIP"}

EXPORTS = ("alto_workspace_bytes", "alto_pack_keys", "alto_route", "alto_aggregate",
           "alto_stream_state_bytes", "alto_stream_create", "alto_stream_step",
           "alto_stream_pending", "alto_stream_destroy", "alto_join_workspace_bytes", "alto_join",
           "alto_split_workspace_bytes", "alto_split", "alto_router_state_bytes", "alto_router_create",
           "alto_router_destroy", "alto_route_load_workspace_bytes", "alto_route_load", "alto_profile_phases",
           "alto_read_probe", "alto_aggregate_noalloc", "alto_aggregate_dev", "alto_stream_step_dev",
           "alto_stream_step_overlap", "alto_aggregate_overlap")
NOALLOC_SCRATCH_BYTES = 128 << 20   # ALTO_NOALLOC_SCRATCH_BYTES of include/alto.h


class Layout(C.Structure):
    _fields_ = [("depth", C.c_int32), ("bits", C.c_uint8 * 16)]


class Agg(C.Structure):
    _fields_ = [("level", C.c_int32), ("op", C.c_int32), ("dim", C.c_int32),
                ("mask_level", C.c_int32), ("release", C.c_int32)]


class Groups(C.Structure):
    _fields_ = [("cap_groups", C.c_int64), ("cap_tokens", C.c_int64), ("cap_mask", C.c_int64),
                ("key", C.c_void_p), ("dest", C.c_void_p), ("count", C.c_void_p),
                ("first_i32", C.c_void_p), ("fan_up", C.c_void_p), ("tok_off", C.c_void_p),
                ("tok", C.c_void_p), ("mean", C.c_void_p), ("mask_key", C.c_void_p),
                ("mask", C.c_void_p), ("pend_key", C.c_void_p), ("pend_count", C.c_void_p),
                ("counts", C.c_void_p)]


_lib = None


class AltoError(RuntimeError):
    def __init__(self, code, what=""):
        super().__init__(f"alto error {STATUS_NAMES.get(code, code)}: {what}")
        self.code = code


def load():
    """Loads libalto.so (built in-tree by __graft_entry__.build())."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = C.CDLL(LIB_PATH)
    vp, i64, i32 = C.c_void_p, C.c_int64, C.c_int32
    lib.alto_workspace_bytes.restype = C.c_size_t
    lib.alto_workspace_bytes.argtypes = [C.POINTER(Layout), i64, i32, C.POINTER(Agg)]
    lib.alto_pack_keys.restype = C.c_int
    lib.alto_pack_keys.argtypes = [vp, i64, i64, C.POINTER(Layout), vp, vp, vp]
    lib.alto_route.restype = C.c_int
    lib.alto_route.argtypes = [vp, i64, C.POINTER(Layout), i32, i32, vp, vp, vp, vp, vp, C.c_size_t, vp]
    lib.alto_aggregate.restype = C.c_int
    lib.alto_aggregate.argtypes = [vp, vp, i64, vp, vp, i64, C.POINTER(Layout), C.POINTER(Agg), i32, i32,
                                   vp, vp, vp, C.POINTER(Groups), vp, vp, C.c_size_t, vp]
    lib.alto_aggregate_dev.restype = C.c_int
    lib.alto_aggregate_dev.argtypes = [vp, vp, i64, vp, vp, i64, vp, C.POINTER(Layout), C.POINTER(Agg), i32, i32,
                                       vp, vp, vp, C.POINTER(Groups), vp, vp, C.c_size_t, vp]
    lib.alto_aggregate_overlap.restype = C.c_int
    lib.alto_aggregate_overlap.argtypes = [vp, vp, i64, vp, vp, i64, C.POINTER(Layout), C.POINTER(Agg), i32, i32,
                                           vp, vp, vp, C.POINTER(Groups), vp, vp, C.c_size_t, vp, vp]
    lib.alto_stream_step_dev.restype = C.c_int
    lib.alto_stream_step_dev.argtypes = [vp, vp, vp, i64, vp, vp, i64, vp, vp, vp, vp, C.POINTER(Groups), vp,
                                         vp, C.c_size_t, vp]
    lib.alto_stream_step_overlap.restype = C.c_int
    lib.alto_stream_step_overlap.argtypes = [vp, vp, vp, i64, vp, vp, i64, vp, vp, vp, vp, C.POINTER(Groups), vp,
                                             vp, vp, C.c_size_t, vp, vp]
    lib.alto_aggregate_noalloc.restype = C.c_int
    lib.alto_aggregate_noalloc.argtypes = [vp, vp, i64, vp, vp, i64, C.POINTER(Layout), C.POINTER(Agg), i32, i32,
                                           vp, vp, vp, C.POINTER(Groups), vp, vp]
    lib.alto_stream_state_bytes.restype = C.c_size_t
    lib.alto_stream_state_bytes.argtypes = [C.POINTER(Layout), C.POINTER(Agg), i64, i64]
    lib.alto_stream_create.restype = C.c_int
    lib.alto_stream_create.argtypes = [C.POINTER(Layout), i32, i32, C.POINTER(Agg), i64, i64, vp,
                                       C.c_size_t, vp, C.POINTER(vp)]
    lib.alto_stream_step.restype = C.c_int
    lib.alto_stream_step.argtypes = [vp, vp, vp, i64, vp, vp, i64, vp, vp, vp, C.POINTER(Groups), vp,
                                     vp, C.c_size_t, vp]
    lib.alto_stream_pending.restype = C.c_int
    lib.alto_stream_pending.argtypes = [vp, C.POINTER(Groups), vp, vp]
    lib.alto_stream_destroy.restype = C.c_int
    lib.alto_stream_destroy.argtypes = [vp]
    lib.alto_join_workspace_bytes.restype = C.c_size_t
    lib.alto_join_workspace_bytes.argtypes = [C.POINTER(Layout), i64]
    lib.alto_join.restype = C.c_int
    lib.alto_join.argtypes = [vp, i64, vp, i64, C.POINTER(Layout), i32, vp, vp, vp, vp, vp, C.c_size_t, vp]
    lib.alto_router_state_bytes.restype = C.c_size_t
    lib.alto_router_state_bytes.argtypes = [i64]
    lib.alto_router_create.restype = C.c_int
    lib.alto_router_create.argtypes = [C.POINTER(Layout), i32, i32, i64, vp, C.c_size_t, vp, C.POINTER(C.c_void_p)]
    lib.alto_router_destroy.restype = C.c_int
    lib.alto_router_destroy.argtypes = [vp]
    lib.alto_route_load_workspace_bytes.restype = C.c_size_t
    lib.alto_route_load_workspace_bytes.argtypes = [C.POINTER(Layout), i32, i64, i32]
    lib.alto_route_load.restype = C.c_int
    lib.alto_route_load.argtypes = [vp, vp, i64, vp, vp, vp, vp, vp, vp, vp, C.c_size_t, vp]
    lib.alto_profile_phases.restype = C.c_int
    lib.alto_profile_phases.argtypes = [C.c_uint32]
    lib.alto_read_probe.restype = C.c_int
    lib.alto_read_probe.argtypes = [vp, i64, vp, vp]
    lib.alto_split_workspace_bytes.restype = C.c_size_t
    lib.alto_split_workspace_bytes.argtypes = [C.POINTER(Layout), i64]
    lib.alto_split.restype = C.c_int
    lib.alto_split.argtypes = [vp, vp, i64, vp, i64, C.POINTER(Layout), i32, i32, i32, vp, vp, i64, vp, vp, vp,
                               vp, vp, vp, C.c_size_t, vp]
    _lib = lib
    return lib


def layout(bits: Sequence[int]) -> Layout:
    l = Layout()
    l.depth = len(bits)
    for i, b in enumerate(bits):
        l.bits[i] = b
    return l


def agg_struct(level: int, op: str, dim: int = 1, mask_level: int = 0, release: str = "complete") -> Agg:
    a = Agg()
    a.level, a.op, a.dim, a.mask_level = level, (MEAN_F32 if op == "mean" else CONCAT_I32), dim, mask_level
    a.release = RELEASE[release]
    return a


def _p(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


_KEY_DTYPES = (torch.int64, torch.uint64) if hasattr(torch, "uint64") else (torch.int64,)


class _Args:
    """Host-side checks of the tensors handed to the C ABI: the kernels index them
    by the sizes given, so a tensor of the wrong type, device, layout or size is
    refused here (AltoError E_ARG) instead of being read or written out of bounds.
    Type, layout and size are checked before the device, so the checks also run on
    a host without a GPU."""

    def __init__(self, what: str):
        self.what = what
        self.dev = None
        self.tensors = []

    def fail(self, msg):
        raise AltoError(E_ARG, f"{self.what}: {msg}")

    def t(self, x, name, dtypes, numel=0, optional=False):
        """A flat buffer: one of ``dtypes``, contiguous, at least ``numel`` elements."""
        if x is None:
            if not optional:
                self.fail(f"{name} is required")
            return None
        if not isinstance(x, torch.Tensor):
            self.fail(f"{name} must be a torch tensor")
        dts = dtypes if isinstance(dtypes, tuple) else (dtypes,)
        if x.dtype not in dts:
            self.fail(f"{name} has dtype {x.dtype}, expected {' or '.join(str(d) for d in dts)}")
        if not x.is_contiguous():
            self.fail(f"{name} must be contiguous")
        if x.numel() < numel:
            self.fail(f"{name} holds {x.numel()} elements, needs {numel}")
        self.tensors.append((name, x))
        return x

    def rows(self, x, name, dtypes, nrows, ncols, optional=False):
        """A level-major [rows][ld] array (ld = stride(0) >= ncols, unit stride) with
        at least ``nrows`` rows; returns its leading dimension."""
        if x is None:
            if not optional:
                self.fail(f"{name} is required")
            return 0
        if not isinstance(x, torch.Tensor) or x.dim() != 2:
            self.fail(f"{name} must be a 2-D tensor [levels][n]")
        dts = dtypes if isinstance(dtypes, tuple) else (dtypes,)
        if x.dtype not in dts:
            self.fail(f"{name} has dtype {x.dtype}, expected {dts[0]}")
        if x.shape[1] > 1 and x.stride(1) != 1:
            self.fail(f"{name} must have unit stride along fragments")
        if x.shape[0] < nrows or x.shape[1] < ncols:
            self.fail(f"{name} is {tuple(x.shape)}, needs at least ({nrows}, {ncols})")
        ld = x.stride(0) if x.shape[0] > 1 else max(x.shape[1], 1)
        if ld < ncols:
            self.fail(f"{name} rows overlap (stride {ld} < {ncols})")
        self.tensors.append((name, x))
        return ld

    def payload(self, x, name, n, dim, optional=False):
        """float32 rows of ``dim`` values, row-major and contiguous, at least n rows."""
        if x is None:
            if not optional:
                self.fail(f"{name} is required")
            return None
        self.t(x, name, torch.float32, n * dim)
        if x.dim() >= 2 and x.shape[-1] != dim:
            self.fail(f"{name} rows hold {x.shape[-1]} values, dim is {dim}")
        return x

    def device(self):
        """Every tensor on one GPU; returns it."""
        for name, x in self.tensors:
            if x.device.type != "cuda":
                self.fail(f"{name} is on {x.device}, not on a GPU")
            if self.dev is None:
                self.dev = x.device
            elif x.device != self.dev:
                self.fail(f"{name} is on {x.device}, other arguments on {self.dev}")
        return self.dev


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _check(rc, what):
    if rc != OK:
        raise AltoError(rc, what)


def workspace_bytes(bits, n_max, num_dest, level=None, op="concat", dim=1, mask_level=0) -> int:
    lib = load()
    L = layout(bits)
    a = None if level is None else C.byref(agg_struct(level, op, dim, mask_level))
    return int(lib.alto_workspace_bytes(C.byref(L), int(n_max), int(num_dest), a))


def new_workspace(nbytes: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def new_status(device="cuda") -> torch.Tensor:
    return torch.zeros(1, dtype=torch.int32, device=device)


def pack_keys(path: torch.Tensor, bits, keys: Optional[torch.Tensor] = None, status=None, stream=None):
    """path: int32 [d][ld] (level-major, first n columns used)."""
    lib = load()
    a = _Args("alto_pack_keys")
    n = path.shape[1] if isinstance(path, torch.Tensor) and path.dim() == 2 else 0
    ld = a.rows(path, "path", torch.int32, len(bits), n)
    if keys is None:
        keys = torch.empty(n, dtype=torch.int64, device=path.device)
    if status is None:
        status = new_status(path.device)
    a.t(keys, "keys", _KEY_DTYPES, n)
    a.t(status, "status", torch.int32, 1)
    a.device()
    L = layout(bits)
    rc = lib.alto_pack_keys(_p(path), ld, n, C.byref(L), _p(keys), _p(status), _stream(stream))
    _check(rc, "alto_pack_keys")
    return keys, status


def route(keys, bits, route_level, num_dest, ws=None, perm=None, dest_offsets=None, dest=None,
          status=None, stream=None, with_dest=True):
    lib = load()
    a = _Args("alto_route")
    n = keys.shape[0]
    a.t(keys, "keys", _KEY_DTYPES, n)
    dev = keys.device
    if ws is None:
        ws = new_workspace(workspace_bytes(bits, n, num_dest), dev)
    if perm is None:
        perm = torch.empty(n, dtype=torch.int32, device=dev)
    if dest_offsets is None:
        dest_offsets = torch.empty(num_dest + 1, dtype=torch.int64, device=dev)
    if dest is None and with_dest:
        dest = torch.empty(n, dtype=torch.int32, device=dev)
    if status is None:
        status = new_status(dev)
    a.t(ws, "ws", torch.uint8)
    a.t(perm, "perm", torch.int32, n)
    a.t(dest_offsets, "dest_offsets", torch.int64, num_dest + 1)
    a.t(dest, "dest", torch.int32, n, optional=True)
    a.t(status, "status", torch.int32, 1)
    a.device()
    L = layout(bits)
    rc = lib.alto_route(_p(keys), n, C.byref(L), route_level, num_dest, _p(perm), _p(dest_offsets),
                        _p(dest), _p(status), _p(ws), _nbytes(ws), _stream(stream))
    _check(rc, "alto_route")
    return perm, dest_offsets, dest, status


@dataclass
class GroupTensors:
    key: torch.Tensor
    dest: torch.Tensor
    count: torch.Tensor
    first_i32: Optional[torch.Tensor]
    fan_up: torch.Tensor
    tok_off: Optional[torch.Tensor]
    tok: Optional[torch.Tensor]
    mean: Optional[torch.Tensor]
    mask_key: Optional[torch.Tensor]
    mask: Optional[torch.Tensor]
    pend_key: torch.Tensor
    pend_count: torch.Tensor
    counts: torch.Tensor
    cap_groups: int
    cap_tokens: int
    cap_mask: int

    def check(self, a: "_Args", op: str, agg_level: int, dim: int):
        """Every member large enough for the capacities it declares."""
        cg, ct, cm = self.cap_groups, self.cap_tokens, self.cap_mask
        if min(cg, ct, cm) < 0:
            a.fail("negative capacity")
        a.t(self.key, "out.key", _KEY_DTYPES, cg, optional=True)
        a.t(self.dest, "out.dest", torch.int32, cg, optional=True)
        a.t(self.count, "out.count", torch.int64, cg, optional=True)
        a.t(self.first_i32, "out.first_i32", torch.int32, cg, optional=True)
        a.t(self.fan_up, "out.fan_up", torch.int32, (agg_level - 1) * cg, optional=True)
        a.t(self.tok_off, "out.tok_off", torch.int64, cg + 1, optional=True)
        a.t(self.tok, "out.tok", torch.int32, ct, optional=True)
        if self.mean is not None:
            a.payload(self.mean, "out.mean", cg, dim)
        a.t(self.mask_key, "out.mask_key", _KEY_DTYPES, cm, optional=True)
        a.t(self.mask, "out.mask", torch.uint8, cm, optional=True)
        a.t(self.pend_key, "out.pend_key", _KEY_DTYPES, cg, optional=True)
        a.t(self.pend_count, "out.pend_count", torch.int64, cg, optional=True)
        a.t(self.counts, "out.counts", torch.int64, 4)

    def struct(self) -> Groups:
        g = Groups()
        g.cap_groups, g.cap_tokens, g.cap_mask = self.cap_groups, self.cap_tokens, self.cap_mask
        for name in ("key", "dest", "count", "first_i32", "fan_up", "tok_off", "tok", "mean",
                     "mask_key", "mask", "pend_key", "pend_count", "counts"):
            t = getattr(self, name)
            setattr(g, name, None if t is None else t.data_ptr())
        return g


def new_groups(cap_groups, agg_level, op, dim=1, cap_tokens=0, cap_mask=0, device="cuda",
               with_first=True) -> GroupTensors:
    cg = max(int(cap_groups), 0)
    e = lambda n, dt: torch.empty(max(n, 1), dtype=dt, device=device)
    return GroupTensors(
        key=e(cg, torch.int64), dest=e(cg, torch.int32), count=e(cg, torch.int64),
        first_i32=e(cg, torch.int32) if with_first else None,
        fan_up=e((agg_level - 1) * cg, torch.int32),
        tok_off=e(cg + 1, torch.int64) if op == "concat" else None,
        tok=e(cap_tokens, torch.int32) if op == "concat" else None,
        mean=torch.empty(max(cg, 1), dim, dtype=torch.float32, device=device) if op == "mean" else None,
        mask_key=e(cap_mask, torch.int64) if cap_mask else None,
        mask=e(cap_mask, torch.uint8) if cap_mask else None,
        pend_key=e(cg, torch.int64), pend_count=e(cg, torch.int64),
        counts=torch.zeros(4, dtype=torch.int64, device=device),
        cap_groups=cg, cap_tokens=int(cap_tokens), cap_mask=int(cap_mask))


def aggregate(keys, fan, bits, agg_level, op, dim=1, mask_level=0, route_level=0, num_dest=1,
              payload_i32=None, payload_f32=None, ws=None, perm=None, dest_offsets=None, dest=None,
              out: Optional[GroupTensors] = None, status=None, stream=None, n=None, n_dev=None,
              gather_stream=None):
    """Routes and aggregates one batch; returns (perm, dest_offsets, dest, groups, status).
    n_dev (int64 device tensor, optional): the count is read there on the device (n,
    or keys.shape[0], is then its bound: alto_aggregate_dev). gather_stream
    (optional): the payload gathers run there after the records
    (alto_aggregate_overlap; not with n_dev)."""
    lib = load()
    a = _Args("alto_aggregate")
    n = keys.shape[0] if n is None else n
    a.t(keys, "keys", _KEY_DTYPES, n)
    fan_ld = a.rows(fan, "fan", torch.int32, len(bits) - 1, n)
    a.t(payload_i32, "payload_i32", torch.int32, n, optional=op != "concat")
    a.payload(payload_f32, "payload_f32", n, dim, optional=op != "mean")
    dev = keys.device
    if ws is None:
        ws = new_workspace(workspace_bytes(bits, n, num_dest, agg_level, op, dim, mask_level), dev)
    if perm is None:
        perm = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
    if dest_offsets is None:
        dest_offsets = torch.empty(num_dest + 1, dtype=torch.int64, device=dev)
    if dest is None:
        dest = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
    if out is None:
        out = new_groups(n, agg_level, op, dim, cap_tokens=n if op == "concat" else 0,
                         cap_mask=n if mask_level else 0, device=dev,
                         with_first=payload_i32 is not None)
    if status is None:
        status = new_status(dev)
    a.t(ws, "ws", torch.uint8)
    a.t(perm, "perm", torch.int32, n, optional=True)
    a.t(dest_offsets, "dest_offsets", torch.int64, num_dest + 1, optional=True)
    a.t(dest, "dest", torch.int32, n, optional=True)
    out.check(a, op, agg_level, dim)
    a.t(status, "status", torch.int32, 1)
    a.t(n_dev, "n_dev", torch.int64, 1, optional=True)
    a.device()
    L = layout(bits)
    A = agg_struct(agg_level, op, dim, mask_level)
    G = out.struct()
    if gather_stream is not None:
        if n_dev is not None:
            a.fail("gather_stream with n_dev")
        rc = lib.alto_aggregate_overlap(_p(keys), _p(fan), fan_ld, _p(payload_i32), _p(payload_f32), n,
                                        C.byref(L), C.byref(A), route_level, num_dest, _p(perm), _p(dest_offsets),
                                        _p(dest), C.byref(G), _p(status), _p(ws), _nbytes(ws), _stream(stream),
                                        _stream(gather_stream))
    elif n_dev is None:
        rc = lib.alto_aggregate(_p(keys), _p(fan), fan_ld, _p(payload_i32), _p(payload_f32), n,
                                C.byref(L), C.byref(A), route_level, num_dest, _p(perm), _p(dest_offsets),
                                _p(dest), C.byref(G), _p(status), _p(ws), _nbytes(ws), _stream(stream))
    else:
        rc = lib.alto_aggregate_dev(_p(keys), _p(fan), fan_ld, _p(payload_i32), _p(payload_f32), n, _p(n_dev),
                                    C.byref(L), C.byref(A), route_level, num_dest, _p(perm), _p(dest_offsets),
                                    _p(dest), C.byref(G), _p(status), _p(ws), _nbytes(ws), _stream(stream))
    _check(rc, "alto_aggregate")
    return perm, dest_offsets, dest, out, status


def aggregate_noalloc(keys, fan, bits, agg_level, op, dim=1, mask_level=0, route_level=0, num_dest=1,
                      payload_i32=None, payload_f32=None, perm=None, dest_offsets=None, dest=None,
                      out: Optional[GroupTensors] = None, status=None, stream=None, n=None):
    """alto_aggregate_noalloc: as ``aggregate`` with every output given by the caller
    and no workspace (the library's own fixed device array serves as one; calls on
    one GPU must not overlap). Nothing is allocated here either: perm, dest_offsets,
    dest, out and status are required. Returns status."""
    lib = load()
    a = _Args("alto_aggregate_noalloc")
    n = keys.shape[0] if n is None else n
    a.t(keys, "keys", _KEY_DTYPES, n)
    fan_ld = a.rows(fan, "fan", torch.int32, len(bits) - 1, n)
    a.t(payload_i32, "payload_i32", torch.int32, n, optional=op != "concat")
    a.payload(payload_f32, "payload_f32", n, dim, optional=op != "mean")
    a.t(perm, "perm", torch.int32, n)
    a.t(dest_offsets, "dest_offsets", torch.int64, num_dest + 1)
    a.t(dest, "dest", torch.int32, n)
    if out is None:
        a.fail("out is required")
    out.check(a, op, agg_level, dim)
    a.t(status, "status", torch.int32, 1)
    need = workspace_bytes(bits, n, num_dest, agg_level, op, dim, mask_level)
    if need == 0 or need > NOALLOC_SCRATCH_BYTES:
        a.fail(f"needs {need} bytes of workspace, more than the fixed {NOALLOC_SCRATCH_BYTES}")
    a.device()
    L = layout(bits)
    A = agg_struct(agg_level, op, dim, mask_level)
    G = out.struct()
    rc = lib.alto_aggregate_noalloc(_p(keys), _p(fan), fan_ld, _p(payload_i32), _p(payload_f32), n, C.byref(L),
                                    C.byref(A), route_level, num_dest, _p(perm), _p(dest_offsets), _p(dest),
                                    C.byref(G), _p(status), _stream(stream))
    _check(rc, "alto_aggregate_noalloc")
    return status


class Stream:
    """Carried-state stream over caller-owned device memory."""

    def __init__(self, bits, route_level, num_dest, agg_level, op, dim=1, max_live_leaves=1 << 16,
                 max_groups=1 << 20, step_max=4096, device="cuda", stream=None, release="complete"):
        lib = load()
        self.lib = lib
        self.bits, self.Lr, self.D, self.La, self.op, self.dim = tuple(bits), route_level, num_dest, agg_level, op, dim
        self.L = layout(bits)
        self.A = agg_struct(agg_level, op, dim, 0, release)
        nbytes = lib.alto_stream_state_bytes(C.byref(self.L), C.byref(self.A), max_live_leaves, max_groups)
        if nbytes == 0:
            raise AltoError(E_ARG, "alto_stream_state_bytes")
        self.state = torch.empty(int(nbytes), dtype=torch.uint8, device=device)
        # a step merges up to max_live_leaves carried leaves with step_max new ones
        self.ws = new_workspace(lib.alto_workspace_bytes(C.byref(self.L), max_live_leaves + step_max,
                                                         num_dest, C.byref(self.A)), device)
        self.step_max = step_max
        self.max_live_leaves = max_live_leaves
        self.handle = C.c_void_p()
        rc = lib.alto_stream_create(C.byref(self.L), route_level, num_dest, C.byref(self.A),
                                    max_live_leaves, max_groups, _p(self.state), self.state.numel(),
                                    _stream(stream), C.byref(self.handle))
        _check(rc, "alto_stream_create")

    def step(self, keys, fan, payload_i32=None, payload_f32=None, out: Optional[GroupTensors] = None,
             perm=None, dest_offsets=None, dest=None, status=None, stream=None, n=None, n_dev=None,
             route_stream=None):
        """One step. n_dev (int64 device tensor, optional): the step's count is read
        there on the device, n (or keys.shape[0]) being its bound
        (alto_stream_step_dev): e.g. the previous stage's out.counts[0:1].
        route_stream (optional): the step's routing runs there and the rest on
        `stream` (alto_stream_step_overlap, with a second workspace of this handle),
        so that the next step's routing runs beside this step's merge and emission."""
        n = keys.shape[0] if n is None else n
        if n > self.step_max:
            raise AltoError(E_ARG, "step larger than step_max")
        a = _Args("alto_stream_step")
        a.t(keys, "keys", _KEY_DTYPES, n)
        fan_ld = a.rows(fan, "fan", torch.int32, len(self.bits) - 1, n)
        a.t(payload_i32, "payload_i32", torch.int32, n, optional=self.op != "concat")
        a.payload(payload_f32, "payload_f32", n, self.dim, optional=self.op != "mean")
        dev = keys.device
        if out is None:
            out = new_groups(n, self.La, self.op, self.dim,
                             cap_tokens=self.max_live_leaves + n if self.op == "concat" else 0,
                             device=dev, with_first=payload_i32 is not None)
        if status is None:
            status = new_status(dev)
        a.t(perm, "perm", torch.int32, n, optional=True)
        a.t(dest_offsets, "dest_offsets", torch.int64, self.D + 1, optional=True)
        a.t(dest, "dest", torch.int32, n, optional=True)
        out.check(a, self.op, self.La, self.dim)
        a.t(status, "status", torch.int32, 1)
        a.t(self.ws, "workspace", torch.uint8)
        a.t(n_dev, "n_dev", torch.int64, 1, optional=True)
        if a.device() != self.state.device:
            a.fail(f"arguments on {a.dev}, stream state on {self.state.device}")
        G = out.struct()
        if route_stream is not None:
            if getattr(self, "ws2", None) is None:
                self.ws2 = torch.empty_like(self.ws)
            rc = self.lib.alto_stream_step_overlap(self.handle, _p(keys), _p(fan), fan_ld, _p(payload_i32),
                                                   _p(payload_f32), n, _p(n_dev), _p(perm), _p(dest_offsets),
                                                   _p(dest), C.byref(G), _p(status), _p(self.ws), _p(self.ws2),
                                                   _nbytes(self.ws), _stream(route_stream), _stream(stream))
            _check(rc, "alto_stream_step_overlap")
            return out, status
        rc = self.lib.alto_stream_step_dev(self.handle, _p(keys), _p(fan), fan_ld, _p(payload_i32),
                                           _p(payload_f32), n, _p(n_dev), _p(perm), _p(dest_offsets), _p(dest),
                                           C.byref(G), _p(status), _p(self.ws), _nbytes(self.ws),
                                           _stream(stream))
        _check(rc, "alto_stream_step")
        return out, status

    def prepare(self, out: GroupTensors, status, perm=None, dest_offsets=None, dest=None, stream=None,
                route_stream=None) -> "PreparedStep":
        """The arguments that stay the same from step to step, checked once: returns
        a callable that takes only a step's inputs (keys, fan, payloads, n, n_dev)
        and calls the same entry point as step() (alto_stream_step_overlap with a
        route_stream, else alto_stream_step_dev). For callers that run many short
        steps, whose per-call argument checks would otherwise cost the host about as
        much as the step's launches. perm and dest must hold step_max elements;
        stream None is the current stream at this call. The
        tensors given here (and those of `out`) must stay allocated, in place and
        unresized while the returned object is used; prepare again after changing
        any of them."""
        return PreparedStep(self, out, status, perm, dest_offsets, dest, stream, route_stream)

    def pending(self, out: Optional[GroupTensors] = None, status=None, stream=None, cap=None):
        dev = self.state.device
        if out is None:
            out = new_groups(cap or self.max_live_leaves, self.La, self.op, self.dim, device=dev)
        if status is None:
            status = new_status(dev)
        a = _Args("alto_stream_pending")
        a.t(out.pend_key, "out.pend_key", _KEY_DTYPES, out.cap_groups, optional=True)
        a.t(out.pend_count, "out.pend_count", torch.int64, out.cap_groups, optional=True)
        a.t(out.counts, "out.counts", torch.int64, 4)
        a.t(status, "status", torch.int32, 1)
        if a.device() != self.state.device:
            a.fail(f"arguments on {a.dev}, stream state on {self.state.device}")
        G = out.struct()
        rc = self.lib.alto_stream_pending(self.handle, C.byref(G), _p(status), _stream(stream))
        _check(rc, "alto_stream_pending")
        return out, status

    def close(self):
        if self.handle:
            self.lib.alto_stream_destroy(self.handle)
            self.handle = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class LoadRouter:
    """Sticky least-loaded routing of flows (route-level prefixes) over
    caller-owned device memory; ``load`` (int64 [num_dest], device) holds the queue
    lengths: route() adds the fragments it sends, the caller subtracts what each
    destination has consumed."""

    def __init__(self, bits, route_level, num_dest, max_flows, n_max, device="cuda", stream=None):
        lib = load()
        self.lib = lib
        self.bits, self.Lr, self.D = tuple(bits), route_level, num_dest
        self.L = layout(bits)
        nbytes = lib.alto_router_state_bytes(max_flows)
        if nbytes == 0:
            raise AltoError(E_ARG, "alto_router_state_bytes")
        self.state = torch.empty(int(nbytes), dtype=torch.uint8, device=device)
        wsb = lib.alto_route_load_workspace_bytes(C.byref(self.L), route_level, n_max, num_dest)
        if wsb == 0:
            raise AltoError(E_ARG, "alto_route_load_workspace_bytes")
        self.ws = new_workspace(wsb, device)
        self.n_max = n_max
        self.max_flows = max_flows
        self.handle = C.c_void_p()
        self.reset(stream)

    def reset(self, stream=None):
        """(Re)creates the router on its state memory: every flow is forgotten."""
        self.close()
        rc = self.lib.alto_router_create(C.byref(self.L), self.Lr, self.D, self.max_flows, _p(self.state),
                                         self.state.numel(), _stream(stream), C.byref(self.handle))
        _check(rc, "alto_router_create")

    def route(self, keys, load, perm=None, dest_offsets=None, dest=None, counts=None, status=None, stream=None,
              n=None):
        """Returns (perm, dest_offsets, dest, counts, status); ``load`` is updated in place."""
        n = keys.shape[0] if n is None else n
        if n > self.n_max:
            raise AltoError(E_ARG, "batch larger than n_max")
        dev = keys.device
        m = max(n, 1)
        if perm is None:
            perm = torch.empty(m, dtype=torch.int32, device=dev)
        if dest_offsets is None:
            dest_offsets = torch.empty(self.D + 1, dtype=torch.int64, device=dev)
        if dest is None:
            dest = torch.empty(m, dtype=torch.int32, device=dev)
        if counts is None:
            counts = torch.zeros(2, dtype=torch.int64, device=dev)
        if status is None:
            status = new_status(dev)
        a = _Args("alto_route_load")
        a.t(keys, "keys", _KEY_DTYPES, n)
        a.t(load, "load", torch.int64, self.D)
        a.t(perm, "perm", torch.int32, n, optional=True)
        a.t(dest_offsets, "dest_offsets", torch.int64, self.D + 1, optional=True)
        a.t(dest, "dest", torch.int32, n, optional=True)
        a.t(counts, "counts", torch.int64, 2)
        a.t(status, "status", torch.int32, 1)
        if a.device() != self.state.device:
            a.fail(f"arguments on {a.dev}, router state on {self.state.device}")
        rc = self.lib.alto_route_load(self.handle, _p(keys), n, _p(load), _p(perm), _p(dest_offsets), _p(dest),
                                      _p(counts), _p(status), _p(self.ws), _nbytes(self.ws), _stream(stream))
        _check(rc, "alto_route_load")
        return perm, dest_offsets, dest, counts, status

    def close(self):
        if self.handle:
            self.lib.alto_router_destroy(self.handle)
            self.handle = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def join(left: torch.Tensor, right_keys: torch.Tensor, bits, level: int, match=None, hits=None, counts=None,
         status=None, ws=None, stream=None, n_left=None, n_right=None):
    """pcombine by ancestry: for every right fragment, the index of the left object
    whose prefix is the fragment's level-``level`` prefix (-1 if none); returns
    (match, hits, counts, status)."""
    lib = load()
    nl = left.shape[0] if n_left is None else n_left
    nr = right_keys.shape[0] if n_right is None else n_right
    dev = right_keys.device
    L = layout(bits)
    if ws is None:
        ws = new_workspace(lib.alto_join_workspace_bytes(C.byref(L), nl), dev)
    if match is None:
        match = torch.empty(max(nr, 1), dtype=torch.int32, device=dev)
    if hits is None:
        hits = torch.empty(max(nl, 1), dtype=torch.int32, device=dev)
    if counts is None:
        counts = torch.zeros(2, dtype=torch.int64, device=dev)
    if status is None:
        status = new_status(dev)
    a = _Args("alto_join")
    a.t(left, "left", _KEY_DTYPES, nl)
    a.t(right_keys, "right_keys", _KEY_DTYPES, nr)
    a.t(match, "match", torch.int32, nr)
    a.t(hits, "hits", torch.int32, nl, optional=True)
    a.t(counts, "counts", torch.int64, 2)
    a.t(status, "status", torch.int32, 1)
    a.t(ws, "ws", torch.uint8)
    a.device()
    rc = lib.alto_join(_p(left), nl, _p(right_keys), nr, C.byref(L), level, _p(match), _p(hits), _p(counts),
                       _p(status), _p(ws), _nbytes(ws), _stream(stream))
    _check(rc, "alto_join")
    return match, hits, counts, status


def split(keys: torch.Tensor, fan: torch.Tensor, tokens: torch.Tensor, bits, delim: int, seg_bits: int,
          tok_bits: int, out_keys=None, out_fan=None, out_tokens=None, out_idx=None, rest_idx=None, counts=None,
          status=None, ws=None, stream=None, n=None, want_rest=True):
    """split_text at a pmap entry: each complete parent's tokens cut at ``delim``
    into segments. Returns (out_keys, out_fan, out_tokens, out_idx, rest_idx,
    counts, status): rows 0..counts[0]-1 of the first four are the new fragments in
    new-key order (layout ``bits[:-1] + (seg_bits, tok_bits)``); rest_idx[:counts[2]]
    lists the input indices of the tokens of incomplete parents."""
    lib = load()
    n = keys.shape[0] if n is None else n
    dev = keys.device
    L = layout(bits)
    d = len(bits)
    m = max(n, 1)
    if ws is None:
        ws = new_workspace(lib.alto_split_workspace_bytes(C.byref(L), n), dev)
    if out_keys is None:
        out_keys = torch.empty(m, dtype=torch.int64, device=dev)
    if out_fan is None:
        out_fan = torch.empty((d, m), dtype=torch.int32, device=dev)
    if out_tokens is None:
        out_tokens = torch.empty(m, dtype=torch.int32, device=dev)
    if out_idx is None:
        out_idx = torch.empty(m, dtype=torch.int32, device=dev)
    if rest_idx is None and want_rest:
        rest_idx = torch.empty(m, dtype=torch.int32, device=dev)
    if counts is None:
        counts = torch.zeros(4, dtype=torch.int64, device=dev)
    if status is None:
        status = new_status(dev)
    a = _Args("alto_split")
    a.t(keys, "keys", _KEY_DTYPES, n)
    if isinstance(fan, torch.Tensor) and fan.dim() == 1 and d - 1 == 1:
        a.t(fan, "fan", torch.int32, n)
        fan_ld = m
    else:
        fan_ld = a.rows(fan, "fan", torch.int32, d - 1, n)
    a.t(tokens, "tokens", torch.int32, n)
    a.t(out_keys, "out_keys", _KEY_DTYPES, n)
    out_fan_ld = a.rows(out_fan, "out_fan", torch.int32, d, n)
    a.t(out_tokens, "out_tokens", torch.int32, n, optional=True)
    a.t(out_idx, "out_idx", torch.int32, n, optional=True)
    a.t(rest_idx, "rest_idx", torch.int32, n, optional=True)
    a.t(counts, "counts", torch.int64, 4)
    a.t(status, "status", torch.int32, 1)
    a.t(ws, "ws", torch.uint8)
    a.device()
    rc = lib.alto_split(_p(keys), _p(fan), fan_ld, _p(tokens), n,
                        C.byref(L), delim, seg_bits, tok_bits, _p(out_keys), _p(out_fan), out_fan_ld,
                        _p(out_tokens), _p(out_idx), _p(rest_idx) if rest_idx is not None else None,
                        _p(counts), _p(status), _p(ws), _nbytes(ws), _stream(stream))
    _check(rc, "alto_split")
    return out_keys, out_fan, out_tokens, out_idx, rest_idx, counts, status


class PreparedStep:
    """Stream.step with its fixed arguments checked and marshalled once (Stream.prepare)."""

    def __init__(self, s: Stream, out: GroupTensors, status, perm, dest_offsets, dest, stream, route_stream):
        a = _Args("alto_stream_step (prepared)")
        if out is None or status is None:
            a.fail("out and status are required")
        a.t(perm, "perm", torch.int32, s.step_max, optional=True)
        a.t(dest_offsets, "dest_offsets", torch.int64, s.D + 1, optional=True)
        a.t(dest, "dest", torch.int32, s.step_max, optional=True)
        out.check(a, s.op, s.La, s.dim)
        a.t(status, "status", torch.int32, 1)
        a.t(s.ws, "workspace", torch.uint8)
        if a.device() != s.state.device:
            a.fail(f"arguments on {a.dev}, stream state on {s.state.device}")
        if route_stream is not None and getattr(s, "ws2", None) is None:
            s.ws2 = torch.empty_like(s.ws)
        self.s, self.dev = s, s.state.device
        self.keep = (out, status, perm, dest_offsets, dest, stream, route_stream)   # alive while prepared
        self.G = out.struct()
        self.Gp = C.byref(self.G)
        self.fixed = (_p(perm), _p(dest_offsets), _p(dest))
        self.status = _p(status)
        self.ws, self.ws2 = _p(s.ws), _p(getattr(s, "ws2", None) if route_stream is not None else None)
        self.nbytes = _nbytes(s.ws)
        self.stream, self.route = _stream(stream), (_stream(route_stream) if route_stream is not None else None)
        self.out, self.status_t = out, status
        self.nrows = len(s.bits) - 1

    def __call__(self, keys, fan, payload_i32=None, payload_f32=None, n=None, n_dev=None):
        s = self.s
        n = keys.shape[0] if n is None else n
        if n > s.step_max:
            raise AltoError(E_ARG, "step larger than step_max")
        a = _Args("alto_stream_step (prepared)")
        a.t(keys, "keys", _KEY_DTYPES, n)
        fan_ld = a.rows(fan, "fan", torch.int32, self.nrows, n)
        a.t(payload_i32, "payload_i32", torch.int32, n, optional=s.op != "concat")
        a.payload(payload_f32, "payload_f32", n, s.dim, optional=s.op != "mean")
        a.t(n_dev, "n_dev", torch.int64, 1, optional=True)
        if a.device() != self.dev:
            a.fail(f"inputs on {a.dev}, prepared arguments on {self.dev}")
        perm, offs, dest = self.fixed
        if self.route is not None:
            rc = s.lib.alto_stream_step_overlap(s.handle, _p(keys), _p(fan), fan_ld, _p(payload_i32),
                                                _p(payload_f32), n, _p(n_dev), perm, offs, dest, self.Gp,
                                                self.status, self.ws, self.ws2, self.nbytes, self.route,
                                                self.stream)
            _check(rc, "alto_stream_step_overlap")
        else:
            rc = s.lib.alto_stream_step_dev(s.handle, _p(keys), _p(fan), fan_ld, _p(payload_i32), _p(payload_f32),
                                            n, _p(n_dev), perm, offs, dest, self.Gp, self.status, self.ws,
                                            self.nbytes, self.stream)
            _check(rc, "alto_stream_step")
        return self.out, self.status_t

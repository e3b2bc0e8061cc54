"""Python binding of libgts.so (ctypes).  Argument marshalling only: every
step of the simulation runs in the library's HIP kernels.  PyTorch provides
device memory and streams.

    from paper_2607_11262_amd import api
    g = api.upload(tile_graph)                # device image + handle
    res = api.simulate(g, hw_records)         # hw_records: uint32 [B, 32]
    res.cycles, res.makespan, res.status, res.digest   # torch tensors on the GPU

The library is loaded from the package directory; if it is missing the
first call raises (there is no CPU fallback).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgts.so")

GTS_OK = 0
ERRORS = {-1: "GTS_E_ARG", -2: "GTS_E_CYCLE", -3: "GTS_E_EDGE_ORDER", -4: "GTS_E_RANGE", -5: "GTS_E_HW",
          -6: "GTS_E_SCRATCH", -7: "GTS_E_HIP", -8: "GTS_E_DUP"}
SIM_OK, SIM_INFEASIBLE, SIM_OVERFLOW, SIM_DEADLOCK = 0, 1, 2, 3
OUT_NODES, OUT_DIGEST, NO_CONTENTION, ORDER_AT_FINISH = 1, 2, 4, 8

EXPORTS = ("gts_graph_validate", "gts_graph_device_bytes", "gts_graph_templates", "gts_graph_upload", "gts_graph_release", "gts_graph_sizes",
           "gts_scratch_bytes", "gts_simulate_batch", "gts_hwset_device_bytes", "gts_hwset_upload",
           "gts_hwset_release", "gts_simulate_hwset", "gts_simulate_hwset_noalloc", "gts_hw_validate", "gts_strerror", "gts_last_error")


class GtsError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        super().__init__(f"{where}: {ERRORS.get(code, code)}: {msg}")
        self.code = code


class _GraphHost(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_uint32), ("n_edges", ctypes.c_uint32), ("n_ctas", ctypes.c_uint32),
                ("n_kernels", ctypes.c_uint32), ("n_ops", ctypes.c_uint32),
                ("op_cls", ctypes.c_void_p), ("op_flags", ctypes.c_void_p), ("op_work", ctypes.c_void_p),
                ("op_warps", ctypes.c_void_p), ("node_op", ctypes.c_void_p), ("succ_ptr", ctypes.c_void_p),
                ("succ", ctypes.c_void_p), ("cta_node_begin", ctypes.c_void_p),
                ("kernel_cta_begin", ctypes.c_void_p), ("kernel_warps", ctypes.c_void_p),
                ("kernel_smem", ctypes.c_void_p), ("kernel_cluster", ctypes.c_void_p),
                ("node_tile", ctypes.c_void_p), ("node_addr", ctypes.c_void_p), ("op_rows", ctypes.c_void_p),
                ("op_pitch", ctypes.c_void_p)]


_lib = None


def lib():
    """The loaded libgts.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_11262_amd.build`")
        _lib = _bind(ctypes.CDLL(LIB_PATH))
    return _lib


def use_library(path: str):
    """Bind the calls to another build of the library at `path` (a CPU-only
    sanitizer build of the host side, for tests); returns it."""
    global _lib
    _lib = _bind(ctypes.CDLL(path))
    return _lib


def _bind(L):
    """Argument and return types of every exported call."""
    vp, u32, u64p = ctypes.c_void_p, ctypes.c_uint32, ctypes.POINTER(ctypes.c_uint64)
    L.gts_graph_validate.argtypes = [vp]
    L.gts_graph_device_bytes.argtypes = [vp, u64p]
    L.gts_graph_templates.argtypes = [vp] + [ctypes.POINTER(u32)] * 4
    L.gts_graph_upload.argtypes = [vp, vp, ctypes.c_uint64, vp, ctypes.POINTER(vp)]
    L.gts_graph_release.argtypes = [vp]
    L.gts_graph_sizes.argtypes = [vp] + [ctypes.POINTER(u32)] * 5
    L.gts_scratch_bytes.argtypes = [vp, u32, u32, u64p]
    L.gts_simulate_batch.argtypes = [vp, vp, u32, vp, vp, vp, vp, vp, ctypes.c_uint64, u32, vp]
    L.gts_hw_validate.argtypes = [vp]
    L.gts_hwset_device_bytes.argtypes = [u32, u64p]
    L.gts_hwset_upload.argtypes = [vp, u32, vp, ctypes.c_uint64, vp, ctypes.POINTER(vp)]
    L.gts_hwset_release.argtypes = [vp]
    L.gts_simulate_hwset.argtypes = [vp, vp, u32, u32, vp, vp, vp, vp, vp, ctypes.c_uint64, u32, vp]
    L.gts_simulate_hwset_noalloc.argtypes = [vp, vp, u32, u32, vp, vp, vp, vp, u32, vp]
    L.gts_strerror.argtypes = [ctypes.c_int]
    L.gts_strerror.restype = ctypes.c_char_p
    L.gts_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("gts_strerror", "gts_last_error"):
            getattr(L, name).restype = ctypes.c_int
    return L


def _check(rc: int, where: str):
    if rc != GTS_OK:
        raise GtsError(rc, where, lib().gts_last_error().decode())


def _host_struct(g):
    """ctypes view of a TileGraph (keeps the numpy arrays alive)."""
    arrs = dict(op_cls=np.ascontiguousarray(g.op_cls, np.uint8), op_flags=np.ascontiguousarray(g.op_flags, np.uint8),
                op_work=np.ascontiguousarray(g.op_work, np.uint32),
                op_warps=np.ascontiguousarray(g.op_warps, np.uint32),
                node_op=np.ascontiguousarray(g.node_op, np.uint16),
                succ_ptr=np.ascontiguousarray(g.succ_ptr, np.uint32), succ=np.ascontiguousarray(g.succ, np.uint32),
                cta_node_begin=np.ascontiguousarray(g.cta_node_begin, np.uint32),
                kernel_cta_begin=np.ascontiguousarray(g.kernel_cta_begin, np.uint32),
                kernel_warps=np.ascontiguousarray(g.kernel_warps, np.uint16),
                kernel_smem=np.ascontiguousarray(g.kernel_smem, np.uint32),
                kernel_cluster=np.ascontiguousarray(g.kernel_cluster, np.uint8),
                node_tile=(np.ascontiguousarray(g.node_tile, np.uint32) if g.node_tile is not None
                           else np.zeros(0, np.uint32)))
    for name, dt in (("node_addr", np.uint64), ("op_rows", np.uint32), ("op_pitch", np.uint32)):
        a = getattr(g, name, None)
        arrs[name] = np.ascontiguousarray(a, dt) if a is not None else np.zeros(0, dt)
    h = _GraphHost(n_nodes=arrs["node_op"].shape[0], n_edges=arrs["succ"].shape[0],
                   n_ctas=arrs["cta_node_begin"].shape[0] - 1, n_kernels=arrs["kernel_warps"].shape[0],
                   n_ops=arrs["op_cls"].shape[0],
                   **{k: (a.ctypes.data if a.size else None) for k, a in arrs.items()})
    return h, arrs


def validate(g) -> None:
    """Host-side validation through the library (no GPU needed)."""
    h, _keep = _host_struct(g)
    _check(lib().gts_graph_validate(ctypes.byref(h)), "gts_graph_validate")


def validate_code(g) -> int:
    h, _keep = _host_struct(g)
    return int(lib().gts_graph_validate(ctypes.byref(h)))


def device_bytes(g) -> int:
    h, _keep = _host_struct(g)
    n = ctypes.c_uint64(0)
    _check(lib().gts_graph_device_bytes(ctypes.byref(h), ctypes.byref(n)), "gts_graph_device_bytes")
    return int(n.value)


def templates(g) -> dict:
    """How the device image shares CTA structure (gts_graph_templates)."""
    h, _keep = _host_struct(g)
    out = [ctypes.c_uint32(0) for _ in range(4)]
    _check(lib().gts_graph_templates(ctypes.byref(h), *[ctypes.byref(x) for x in out]), "gts_graph_templates")
    keys = ("templated_kernels", "template_nodes", "expanded_nodes", "class_ops")
    return {k: int(x.value) for k, x in zip(keys, out)}


def hw_validate(rec) -> int:
    rec = np.ascontiguousarray(rec, np.uint32)
    return int(lib().gts_hw_validate(rec.ctypes.data))


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Graph:
    """An uploaded graph: the device image tensor and the library handle."""

    def __init__(self, image, handle, n_nodes, n_edges, n_ctas, n_kernels, n_ops, name=""):
        self.image, self.handle = image, handle
        self.n_nodes, self.n_edges, self.n_ctas, self.n_kernels, self.n_ops = n_nodes, n_edges, n_ctas, n_kernels, n_ops
        self.name = name

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.gts_graph_release(self.handle)
            self.handle = None


def upload(g, stream=None, device="cuda") -> Graph:
    import torch
    h, _keep = _host_struct(g)
    n = device_bytes(g)
    image = torch.empty(max(n, 1), dtype=torch.uint8, device=device)
    handle = ctypes.c_void_p()
    _check(lib().gts_graph_upload(ctypes.byref(h), ctypes.c_void_p(image.data_ptr()), n, _stream(stream),
                                  ctypes.byref(handle)), "gts_graph_upload")
    return Graph(image, handle, h.n_nodes, h.n_edges, h.n_ctas, h.n_kernels, h.n_ops, getattr(g, "name", ""))


def scratch_bytes(g: Graph, B: int, flags: int) -> int:
    n = ctypes.c_uint64(0)
    _check(lib().gts_scratch_bytes(g.handle, B, flags, ctypes.byref(n)), "gts_scratch_bytes")
    return int(n.value)


@dataclass
class Result:
    cycles: object      # torch.uint32-like int32 view [B, N, 2] or None
    makespan: object    # int64 copy-friendly tensor [B] (uint32 values)
    status: object      # int32 [B]
    digest: object      # int64 [B] (uint64 bit pattern) or None


def alloc_outputs(g: Graph, B: int, flags: int, device="cuda"):
    import torch
    cyc = torch.empty((B, g.n_nodes, 2), dtype=torch.int32, device=device) if flags & OUT_NODES else None
    mk = torch.empty(B, dtype=torch.int32, device=device)
    st = torch.empty(B, dtype=torch.int32, device=device)
    dg = torch.empty(B, dtype=torch.int64, device=device) if flags & OUT_DIGEST else None
    return cyc, mk, st, dg


def simulate_into(g: Graph, hw, flags, cyc, mk, st, dg, scratch, stream=None) -> None:
    """Enqueue one batch on `stream` writing into preallocated outputs."""
    hw = np.ascontiguousarray(hw, dtype=np.uint32).reshape(-1, 32)
    B = hw.shape[0]
    _check(lib().gts_simulate_batch(g.handle, hw.ctypes.data, B, ctypes.c_void_p(cyc.data_ptr() if cyc is not None else 0),
                                    ctypes.c_void_p(mk.data_ptr()), ctypes.c_void_p(st.data_ptr()),
                                    ctypes.c_void_p(dg.data_ptr() if dg is not None else 0),
                                    ctypes.c_void_p(scratch.data_ptr()), scratch.numel(), flags, _stream(stream)),
           "gts_simulate_batch")


def simulate(g: Graph, hw, flags: int = OUT_NODES | OUT_DIGEST, stream=None, scratch=None) -> Result:
    """Simulate g under every record of hw [B, 32] (uint32); returns device
    tensors (valid after `stream` synchronises).

    Scratch and outputs are allocated on the stream the kernels run on, so
    torch's caching allocator hands their blocks to a later allocation only
    after that stream's queued work (the simulation) has run, even when
    `stream` is not the current stream.  A caller-provided scratch tensor
    used on a side stream is marked with record_stream for the same reason."""
    import torch
    hw = np.ascontiguousarray(hw, dtype=np.uint32).reshape(-1, 32)
    B = hw.shape[0]
    need = scratch_bytes(g, B, flags)
    s = stream if stream is not None else torch.cuda.current_stream()
    with torch.cuda.stream(s):
        if scratch is None or scratch.numel() < need:
            scratch = torch.empty(max(need, 1), dtype=torch.uint8, device=g.image.device)
        elif stream is not None:
            scratch.record_stream(s)
        cyc, mk, st, dg = alloc_outputs(g, B, flags, g.image.device)
    simulate_into(g, hw, flags, cyc, mk, st, dg, scratch, s)
    return Result(cyc, mk, st, dg)


class HwSet:
    """Hardware records resident in device memory (gts_hwset_upload)."""

    def __init__(self, buf, handle, B):
        self.buf, self.handle, self.B = buf, handle, B

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.gts_hwset_release(self.handle)
            self.handle = None


def upload_hw(hw, stream=None, device="cuda") -> HwSet:
    import torch
    hw = np.ascontiguousarray(hw, dtype=np.uint32).reshape(-1, 32)
    B = hw.shape[0]
    n = ctypes.c_uint64(0)
    _check(lib().gts_hwset_device_bytes(B, ctypes.byref(n)), "gts_hwset_device_bytes")
    buf = torch.empty(max(int(n.value), 1), dtype=torch.uint8, device=device)
    handle = ctypes.c_void_p()
    _check(lib().gts_hwset_upload(hw.ctypes.data, B, ctypes.c_void_p(buf.data_ptr()), buf.numel(), _stream(stream),
                                  ctypes.byref(handle)), "gts_hwset_upload")
    return HwSet(buf, handle, B)


def simulate_hwset_into(g: Graph, hs: HwSet, first: int, B: int, flags, cyc, mk, st, dg, scratch, stream=None):
    """Enqueue records [first, first + B) of a resident set; outputs row b is
    record first + b (pass tensor views offset accordingly)."""
    _check(lib().gts_simulate_hwset(g.handle, hs.handle, first, B,
                                    ctypes.c_void_p(cyc.data_ptr() if cyc is not None else 0),
                                    ctypes.c_void_p(mk.data_ptr()), ctypes.c_void_p(st.data_ptr()),
                                    ctypes.c_void_p(dg.data_ptr() if dg is not None else 0),
                                    ctypes.c_void_p(scratch.data_ptr()), scratch.numel(), flags, _stream(stream)),
           "gts_simulate_hwset")


NOALLOC_SCRATCH_BYTES = 128 << 20  # GTS_NOALLOC_SCRATCH_BYTES


def simulate_hwset_noalloc(g: Graph, hs: HwSet, first: int, B: int, flags, cyc, mk, st, dg, stream=None):
    """As simulate_hwset_into, through gts_simulate_hwset_noalloc: the
    library's own per-GPU scratch array instead of a caller buffer (nothing is
    allocated; calls that overlap on one GPU race)."""
    _check(lib().gts_simulate_hwset_noalloc(g.handle, hs.handle, first, B,
                                            ctypes.c_void_p(cyc.data_ptr() if cyc is not None else 0),
                                            ctypes.c_void_p(mk.data_ptr()), ctypes.c_void_p(st.data_ptr()),
                                            ctypes.c_void_p(dg.data_ptr() if dg is not None else 0), flags,
                                            _stream(stream)),
           "gts_simulate_hwset_noalloc")


def to_numpy(res: Result):
    """Host copies with the unsigned dtypes of the ABI."""
    cyc = res.cycles.cpu().numpy().view(np.uint32) if res.cycles is not None else None
    mk = res.makespan.cpu().numpy().view(np.uint32)
    st = res.status.cpu().numpy()
    dg = res.digest.cpu().numpy().view(np.uint64) if res.digest is not None else None
    return cyc, mk, st, dg

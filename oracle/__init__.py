"""CPU oracle of the batched tile-graph simulation (ctypes wrapper).

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this module; the product path
(paper_2607_11262_amd.api / libgts.so) never does.

The C oracle (gts_oracle.c) simulates one (graph, hardware record) pair per
call of gtso_simulate; gts_oracle_simulate runs a batch of records, one after
another.  Graph arguments are read from any object with the TileGraph array
attributes (op_cls, op_flags, op_work, op_warps, node_op, succ_ptr, succ,
cta_node_begin, kernel_cta_begin, kernel_warps, kernel_smem); this module
does not import the product package.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gts_oracle.c")
_LIB = os.path.join(_HERE, "libgts_oracle.so")
_lib = None

STATUS_OK, STATUS_INFEASIBLE, STATUS_OVERFLOW, STATUS_DEADLOCK = 0, 1, 2, 3
F_NODES, F_DIGEST, F_NO_CONTENTION, F_ORDER_AT_FINISH = 1, 2, 4, 8


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain C, -O2)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def _open(path):
    lib = ctypes.CDLL(path)
    p = ctypes.c_void_p
    u32 = ctypes.c_uint32
    lib.gtso_simulate.argtypes = [u32, u32, u32, u32, u32] + [p] * 16 + [p, u32] + [p] * 5
    lib.gtso_simulate.restype = ctypes.c_int
    lib.gts_oracle_simulate.argtypes = [p, p, u32, p, p, p, p, u32]
    lib.gts_oracle_simulate.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        build()
        _lib = _open(_LIB)
    return _lib


def build_sanitized(path: str) -> str:
    """The oracle under AddressSanitizer and UBSan (gcc), for a process
    started with the sanitizer runtimes preloaded."""
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-o", path, _SRC])
    return path


def use_library(path: str) -> None:
    """Route every later call to the oracle built at `path` (sanitizer runs)."""
    global _lib
    _lib = _open(path)


def build_variant(source_text: str, path: str) -> None:
    """Compile an edited copy of the oracle source to `path` (used by the
    test that plants mistakes in the oracle to show the pins catch them)."""
    src = path + ".c"
    with open(src, "w") as f:
        f.write(source_text)
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-w", "-o", path, src])


def source_text() -> str:
    with open(_SRC) as f:
        return f.read()


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def _addr_arrays(g):
    """Tile addresses and per-op tile rows / row strides (transaction-level
    memory), or None each."""
    def opt(name, dt):
        a = getattr(g, name, None)
        return _c(a, dt) if a is not None else None
    return [opt("node_addr", np.uint64), opt("op_rows", np.uint32), opt("op_pitch", np.uint32)]


class OracleResult:
    __slots__ = ("cycles", "makespan", "status", "digest", "cta")

    def __init__(self, cycles, makespan, status, digest, cta):
        self.cycles, self.makespan, self.status, self.digest, self.cta = cycles, makespan, status, digest, cta


def simulate(g, hw, flags: int = 0, want_nodes: bool = True, want_cta: bool = False, lib_path=None) -> OracleResult:
    """One simulation of graph g under the 32-word hardware record hw
    (lib_path: an oracle variant built by build_variant, tests only)."""
    lib = _load() if lib_path is None else _open(lib_path)
    arrs = [_c(g.op_cls, np.uint8), _c(g.op_flags, np.uint8), _c(g.op_work, np.uint32), _c(g.op_warps, np.uint32),
            _c(g.node_op, np.uint16), _c(g.succ_ptr, np.uint32), _c(g.succ, np.uint32),
            _c(g.cta_node_begin, np.uint32), _c(g.kernel_cta_begin, np.uint32), _c(g.kernel_warps, np.uint16),
            _c(g.kernel_smem, np.uint32), _c(g.kernel_cluster, np.uint8),
            _c(g.node_tile, np.uint32) if g.node_tile is not None else None] + _addr_arrays(g)
    N = int(arrs[4].shape[0])
    C = int(arrs[7].shape[0]) - 1
    hw = _c(hw, np.uint32)
    assert hw.shape == (32,)
    cyc = np.zeros((N, 2), dtype=np.uint32) if want_nodes else None
    cta = np.zeros((max(C, 0), 2), dtype=np.uint32) if want_cta else None
    mk = np.zeros(1, dtype=np.uint32)
    st = np.zeros(1, dtype=np.int32)
    dg = np.zeros(1, dtype=np.uint64)
    rc = lib.gtso_simulate(N, int(arrs[6].shape[0]), C, int(arrs[9].shape[0]), int(arrs[0].shape[0]),
                           *[_ptr(a) for a in arrs], _ptr(hw), int(flags), _ptr(cyc), _ptr(mk), _ptr(st), _ptr(dg),
                           _ptr(cta))
    if rc != 0:
        raise RuntimeError(f"oracle failed rc={rc}")
    return OracleResult(cyc, int(mk[0]), int(st[0]), int(dg[0]), cta)


class _GraphHost(ctypes.Structure):
    """The batched call's graph struct (field order of the library's host
    graph, restated)."""
    _fields_ = [(n, ctypes.c_uint32) for n in ("n_nodes", "n_edges", "n_ctas", "n_kernels", "n_ops")] + \
               [(n, ctypes.c_void_p) for n in ("op_cls", "op_flags", "op_work", "op_warps", "node_op", "succ_ptr",
                                               "succ", "cta_node_begin", "kernel_cta_begin", "kernel_warps",
                                               "kernel_smem", "kernel_cluster", "node_tile", "node_addr",
                                               "op_rows", "op_pitch")]


def simulate_records(g, hws, flags: int = 0, want_nodes: bool = False):
    """All records of hws [B, 32] in one call of gts_oracle_simulate (one
    thread, record order).  Returns (makespan u32[B], status i32[B], digest
    u64[B], cycles [B][N][2] or None)."""
    lib = _load()
    arrs = [_c(g.op_cls, np.uint8), _c(g.op_flags, np.uint8), _c(g.op_work, np.uint32), _c(g.op_warps, np.uint32),
            _c(g.node_op, np.uint16), _c(g.succ_ptr, np.uint32), _c(g.succ, np.uint32),
            _c(g.cta_node_begin, np.uint32), _c(g.kernel_cta_begin, np.uint32), _c(g.kernel_warps, np.uint16),
            _c(g.kernel_smem, np.uint32), _c(g.kernel_cluster, np.uint8),
            _c(g.node_tile, np.uint32) if g.node_tile is not None else None] + _addr_arrays(g)
    h = _GraphHost(int(arrs[4].shape[0]), int(arrs[6].shape[0]), int(arrs[7].shape[0]) - 1, int(arrs[9].shape[0]),
                   int(arrs[0].shape[0]), *[(a.ctypes.data if a is not None and a.size else None) for a in arrs])
    hws = np.ascontiguousarray(hws, dtype=np.uint32).reshape(-1, 32)
    B = hws.shape[0]
    mk = np.zeros(B, dtype=np.uint32)
    st = np.zeros(B, dtype=np.int32)
    dg = np.zeros(B, dtype=np.uint64)
    cyc = np.zeros((B, h.n_nodes, 2), dtype=np.uint32) if want_nodes else None
    rc = lib.gts_oracle_simulate(ctypes.byref(h), _ptr(hws), B, _ptr(cyc), _ptr(mk), _ptr(st), _ptr(dg), int(flags))
    if rc != 0:
        raise RuntimeError(f"oracle failed rc={rc}")
    return mk, st, dg, cyc


def simulate_batch(g, hws, flags: int = 0, want_nodes: bool = False, threads: int = 1):
    """Simulations of g under each record of hws [B, 32]: runs of consecutive
    records through gts_oracle_simulate, distributed over `threads` host
    threads (the C call releases the GIL).  Returns (makespan u32[B], status
    i32[B], digest u64[B], cycles [B][N][2] or None)."""
    hws = np.ascontiguousarray(hws, dtype=np.uint32).reshape(-1, 32)
    B = hws.shape[0]
    if threads <= 1 or B <= 1:
        return simulate_records(g, hws, flags, want_nodes)
    step = max(1, B // (4 * threads))
    runs = [(i, min(B, i + step)) for i in range(0, B, step)]
    with ThreadPoolExecutor(max_workers=threads) as ex:
        res = list(ex.map(lambda r: simulate_records(g, hws[r[0]:r[1]], flags, want_nodes), runs))
    mk = np.concatenate([r[0] for r in res])
    st = np.concatenate([r[1] for r in res])
    dg = np.concatenate([r[2] for r in res])
    cyc = np.concatenate([r[3] for r in res]) if want_nodes else None
    return mk, st, dg, cyc

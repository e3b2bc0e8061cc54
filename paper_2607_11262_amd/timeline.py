"""Resource utilisation from a simulated timeline (GTSim Sec. 5.2 resources,
Sec. 7.1 Tensor Core utilisation of the pipelining case study).

A simulation reports each node's start and finish cycle.  A compute node of
class c that runs on k subpartition lanes keeps those k lanes of c's
pipelines busy from its start for its occupancy cycles (its latency overlaps
later work); a shared-memory node keeps the SM's shared-memory pipe busy,
and a global load or store keeps the SM's global-memory engine busy, for
their occupancies.  Occupancies follow from the hardware record: on k lanes
`max(1, ceil(work * 2^16 * n_subpart / (k * rate)))`, otherwise
`max(1, ceil(work * 2^16 / rate))`.

Utilisation of a resource = busy lane-cycles / (lanes of the machine x
makespan): every SM of the record contributes n_subpart lanes per compute
class and one shared-memory pipe and one engine.
"""
from __future__ import annotations

import numpy as np

from .gen import hw as H
from .gen.graph import ALU, GLOAD, GSTORE, SFU, SMEM, TENSOR

RESOURCES = ("tensor", "alu", "sfu", "smem", "gmem")
_RATE = {TENSOR: "rate_tensor", ALU: "rate_alu", SFU: "rate_sfu", SMEM: "rate_smem", GLOAD: "rate_gmem",
         GSTORE: "rate_gmem"}
_RES = {TENSOR: "tensor", ALU: "alu", SFU: "sfu", SMEM: "smem", GLOAD: "gmem", GSTORE: "gmem"}


def _cdiv(a, b):
    return -(-a // b)


def op_busy(g, rec):
    """Per op: (resource name or None, lanes k, occupancy in cycles)."""
    nsub = H.get(rec, "n_subpart")
    out = []
    for p in range(g.n_ops):
        cls, work, warps = int(g.op_cls[p]), int(g.op_work[p]), int(g.op_warps[p])
        if cls not in _RES:
            out.append((None, 0, 0))
            continue
        rate = H.get(rec, _RATE[cls])
        if cls in (TENSOR, ALU, SFU):
            k = len({w % nsub for w in range(32) if warps >> w & 1})
            occ = max(1, _cdiv(work * 65536 * nsub, k * rate))
        else:
            k = 1
            occ = max(1, _cdiv(work * 65536, rate))
        out.append((_RES[cls], k, occ))
    return out


def intervals(g, rec, cycles):
    """Busy intervals per resource: name -> (start, end, lanes) arrays."""
    cycles = np.asarray(cycles)
    busy = op_busy(g, rec)
    ops = np.asarray(g.node_op, dtype=np.int64)
    res = np.array([b[0] or "" for b in busy], dtype=object)[ops]
    k = np.array([b[1] for b in busy], dtype=np.int64)[ops]
    occ = np.array([b[2] for b in busy], dtype=np.int64)[ops]
    start = cycles[:, 0].astype(np.int64)
    out = {}
    for name in RESOURCES:
        m = res == name
        out[name] = (start[m], start[m] + occ[m], k[m])
    return out


def capacity(rec, name: str) -> int:
    """Lanes of one resource across the machine."""
    n_sm = H.get(rec, "n_sm")
    return n_sm * H.get(rec, "n_subpart") if name in ("tensor", "alu", "sfu") else n_sm


def utilization(g, rec, cycles, makespan=None) -> dict:
    """Fraction of each resource's lane-cycles that are busy over [0, makespan)."""
    cycles = np.asarray(cycles)
    if makespan is None:
        makespan = int(cycles[:, 1].max()) if cycles.size else 0
    out = {}
    for name, (a, b, k) in intervals(g, rec, cycles).items():
        busy = int(((b - a) * k).sum())
        out[name] = busy / (capacity(rec, name) * makespan) if makespan else 0.0
    return out


def profile(g, rec, cycles, bins: int = 64, makespan=None) -> dict:
    """Utilisation per resource in `bins` equal time slices of [0, makespan)."""
    cycles = np.asarray(cycles)
    if makespan is None:
        makespan = int(cycles[:, 1].max()) if cycles.size else 0
    edges = np.linspace(0, makespan, bins + 1)
    out = {}
    for name, (a, b, k) in intervals(g, rec, cycles).items():
        # busy lane-cycles per cycle as a step function, integrated per slice
        pts = np.concatenate([a, b])
        delta = np.concatenate([k, -k])
        order = np.argsort(pts, kind="stable")
        pts, level = pts[order], np.cumsum(delta[order])
        prim = np.concatenate([[0.0], np.cumsum(level[:-1] * np.diff(pts))]) if pts.size else np.zeros(0)

        def integral(x):  # busy lane-cycles in [0, x)
            if pts.size == 0:
                return np.zeros_like(x)
            i = np.searchsorted(pts, x, side="right") - 1
            base = np.where(i >= 0, prim[np.maximum(i, 0)], 0.0)
            return base + np.where(i >= 0, level[np.maximum(i, 0)] * (x - pts[np.maximum(i, 0)]), 0.0)

        tot = integral(edges)
        width = np.diff(edges)
        with np.errstate(invalid="ignore", divide="ignore"):
            out[name] = np.where(width > 0, np.diff(tot) / (capacity(rec, name) * width), 0.0)
    return out


def ready_cycles(g, cycles) -> np.ndarray:
    """Each node's ready cycle re-derived from its in-edges' releases (ORDER
    at the source's start + 1, DATA / SYNC at its finish); nodes without
    in-edges get their start (their CTA's launch is not part of a result)."""
    cycles = np.asarray(cycles).astype(np.int64)
    src = np.repeat(np.arange(g.n_nodes, dtype=np.int64), np.diff(g.succ_ptr.astype(np.int64)))
    dst = (g.succ & np.uint32((1 << 30) - 1)).astype(np.int64)
    kind = (g.succ >> np.uint32(30)).astype(np.int64)
    rel = np.where(kind == 1, cycles[src, 0] + 1, cycles[src, 1])
    ready = np.full(g.n_nodes, -1, dtype=np.int64)
    np.maximum.at(ready, dst, rel)
    return np.where(ready < 0, cycles[:, 0], ready)


def noc_residence(g, cycles) -> float:
    """Mean NoC residence of the REMOTE requests (Sec. 7.2): from the cycle a
    transfer is ready to its finish (queueing for the route, occupancy and
    traversal latency)."""
    from .gen.graph import REMOTE
    cycles = np.asarray(cycles)
    m = np.asarray(g.op_cls)[np.asarray(g.node_op)] == REMOTE
    if not m.any():
        return 0.0
    return float((cycles[m, 1].astype(np.int64) - ready_cycles(g, cycles)[m]).mean())

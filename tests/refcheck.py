"""Independent checks of simulation results (test helpers).

These re-state the timing rules in a different form from the event-driven
oracle, so that a slip in the oracle (a dropped latency, a wrong phase
order, a wrong lane, a wrong tie-break) shows up as a mismatch:

* ``verify_schedule`` takes a finished schedule (per-node start/finish and
  per-CTA SM/launch) and checks that it is the fixed point of the rules
  written as equations: every node's start equals max(ready, server
  availability) with each server's users taken in FIFO order of
  (ready cycle, node id), every finish equals start + the node's duration,
  every ready cycle equals the latest release over its in-edges (order edges
  at source start + 1, data/sync edges at source finish), and the CTA
  dispatch sequence re-simulated from the CTAs' retire cycles matches.
  Because each quantity depends only on strictly earlier ones the rules
  have exactly one fixed point, so passing means the schedule is the one
  the rules define.
* ``asap_bruteforce`` enumerates every path of a tiny DAG to get the
  uncontended (as-soon-as-possible) start of each node: the longest path
  with order edges weighing 1 and data/sync edges the source's duration.
* ``durations`` computes each op's occupancy / latency from the hardware
  record by the integer formulas (ceil division, Q16.16 rates).
"""
from __future__ import annotations

import json
import os

import numpy as np

from paper_2607_11262_amd.gen import hw as H
from collections import OrderedDict

from paper_2607_11262_amd.gen.graph import (ALU, DATA, GLOAD, GSTORE, LINE_BYTES, NO_TILE, ORDER, REMOTE, SFU,
                                             SMEM, SYNC, SYNC_EDGE, TENSOR, GraphBuilder, remote_flags)

MAXCYC = 0xFFFFFFFE
CLASS = {"TENSOR": TENSOR, "ALU": ALU, "SFU": SFU, "SMEM": SMEM, "GLOAD": GLOAD, "GSTORE": GSTORE, "SYNC": SYNC,
         "REMOTE": REMOTE}
KIND = {"D": DATA, "O": ORDER, "S": SYNC_EDGE}
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_schedules.json")


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


def durations(g, rec):
    """Per op: dict(kind, cls, lanes, occ, occ_m, lat, dram)."""
    nsub = H.get(rec, "n_subpart")
    rates = [H.get(rec, f) for f in ("rate_tensor", "rate_alu", "rate_sfu", "rate_smem", "rate_gmem", "rate_l2",
                                       "rate_dram")]
    lats = [H.get(rec, f) for f in ("lat_tensor", "lat_alu", "lat_sfu", "lat_smem", "lat_l2", "lat_dram",
                                      "lat_sync")]
    out = []
    for p in range(g.n_ops):
        cls, work, warps, miss = int(g.op_cls[p]), int(g.op_work[p]), int(g.op_warps[p]), int(g.op_flags[p]) & 1
        if cls in (TENSOR, ALU, SFU):
            lanes = sorted({w % nsub for w in range(32) if warps >> w & 1})
            occ = max(1, cdiv(work * 65536 * nsub, len(lanes) * rates[cls]))
            out.append(dict(kind="compute", cls=cls, lanes=lanes, occ=occ, lat=lats[cls]))
        elif cls == SMEM:
            out.append(dict(kind="smem", occ=max(1, cdiv(work * 65536, rates[3])), lat=lats[3]))
        elif cls == SYNC:
            out.append(dict(kind="sync", lat=max(1, lats[6])))
        elif cls == REMOTE:
            rate = H.get(rec, "noc_rate")
            out.append(dict(kind="remote", occ=max(1, cdiv(work * 65536, rate)) if rate else 1,
                            lat=H.get(rec, "noc_lat"), rank=int(g.op_flags[p]) >> 4))
        else:
            out.append(dict(kind="gmem", occ=max(1, cdiv(work * 65536, rates[4])),
                            occ_m=max(1, cdiv(work * 65536, rates[6] if miss else rates[5])),
                            lat=lats[5] if miss else lats[4], dram=bool(miss),
                            occ_l2=max(1, cdiv(work * 65536, rates[5])), occ_dram=max(1, cdiv(work * 65536, rates[6])),
                            lat_l2=lats[4], lat_dram=lats[5], lines=cdiv(work, LINE_BYTES)))
    return out


def node_duration(d) -> int:
    """Uncontended start-to-finish length of a node."""
    if d["kind"] in ("compute", "smem"):
        return d["occ"] + d["lat"]
    if d["kind"] == "sync":
        return d["lat"]
    return max(d["occ"], d["occ_m"]) + d["lat"]


def slots_per_kernel(g, rec):
    out = []
    for k in range(g.n_kernels):
        s = H.get(rec, "max_cta_per_sm")
        if int(g.kernel_smem[k]):
            s = min(s, H.get(rec, "smem_per_sm") // int(g.kernel_smem[k]))
        s = min(s, H.get(rec, "max_warps_per_sm") // int(g.kernel_warps[k]))
        out.append(s)
    return out


def verify_schedule(g, rec, flags, cycles, cta):
    """Raise AssertionError unless (cycles, cta) is the schedule the rules
    define for graph g on hardware record rec.  cycles [N,2], cta [C,2]."""
    N, C = g.n_nodes, g.n_ctas
    nocont = bool(flags & 4)
    order_fin = bool(flags & 8)
    dur = durations(g, rec)
    st = cycles[:, 0].astype(np.int64)
    fi = cycles[:, 1].astype(np.int64)
    node_cta = g.node_cta()
    cta_sm = cta[:, 0].astype(np.int64)
    launch = cta[:, 1].astype(np.int64)
    # ready cycle of every node from its in-edges' release cycles
    ready = launch[node_cta].copy()
    src, dst, kind = g.sources(), g.targets(), g.kinds()
    rel = np.where((kind == ORDER) & (not order_fin), st[src] + 1, fi[src])
    np.maximum.at(ready, dst, rel)
    ops = g.node_op.astype(np.int64)
    nsub = H.get(rec, "n_subpart")
    order = np.lexsort((np.arange(N), ready))  # FIFO (ready, id)
    lane_av, smem_av, eng_av, noc_av = {}, {}, {}, {}
    gstart = {}
    txn = tile_transactions(g)
    D, W = H.get(rec, "noc_nodes"), H.get(rec, "noc_width")
    for v in order:
        d = dur[ops[v]]
        sm = int(cta_sm[node_cta[v]])
        r = int(ready[v])
        if d["kind"] == "compute":
            # one pipeline per (SM, compute class, subpartition lane)
            s = r if nocont else max([r] + [lane_av.get((sm, d["cls"], l), 0) for l in d["lanes"]])
            for l in d["lanes"]:
                lane_av[(sm, d["cls"], l)] = s + d["occ"]
            assert st[v] == s and fi[v] == s + d["occ"] + d["lat"], f"compute node {v}: {st[v], fi[v]} != {s}"
        elif d["kind"] == "smem":
            s = r if nocont else max(r, smem_av.get(sm, 0))
            smem_av[sm] = s + d["occ"]
            assert st[v] == s and fi[v] == s + d["occ"] + d["lat"], f"smem node {v}"
        elif d["kind"] == "sync":
            assert st[v] == r and fi[v] == r + d["lat"], f"sync node {v}"
        elif d["kind"] == "remote":
            c = int(node_cta[v])
            target = cluster_first(g, c) + d["rank"]
            servers, hops = noc_route(sm, int(cta_sm[target]), D, W)
            s = r if nocont else max([r] + [noc_av.get(x, 0) for x in servers])
            for x in servers:
                noc_av[x] = s + d["occ"]
            assert st[v] == s and fi[v] == s + d["occ"] + d["lat"] * hops, f"remote node {v}: {st[v], fi[v]} != {s}"
        else:
            s = r if nocont else max(r, eng_av.get(sm, 0))
            if v in txn:  # transaction-level tile: the engine streams all its lines
                eng_av[sm] = s + max(1, cdiv(len(txn[v]) * LINE_BYTES * 65536, H.get(rec, "rate_gmem")))
            else:
                eng_av[sm] = s + d["occ"]
            assert st[v] == s, f"gmem node {v} start {st[v]} != {s}"
            gstart[v] = s
    # global L2 / DRAM servers in FIFO order of (arrival, id, transaction):
    # a node without an address arrives once, at its engine start; an
    # addressed node's transaction j when the engine starts injecting it.
    # With an L2 capacity, tracked tiles and addressed lines replay an
    # explicit LRU of 128-B lines.
    av = {False: 0, True: 0}
    cap = H.get(rec, "l2_lines")
    lines = OrderedDict()  # (tile, line) or ("addr", line) -> None, least recent first
    rg = H.get(rec, "rate_gmem")
    arrivals = []
    for v, s in gstart.items():
        if v in txn:
            arrivals += [(s + cdiv(j * LINE_BYTES * 65536, rg), v, j) for j in range(len(txn[v]))]
        else:
            arrivals.append((s, v, 0))
    tx_fin = {}
    for a, v, j in sorted(arrivals):
        d = dur[ops[v]]
        s = gstart[v]
        if v in txn:
            miss = bool(d["dram"])
            if cap:
                key = ("addr", txn[v][j])
                miss = key not in lines
                lines[key] = None
                lines.move_to_end(key)
                while len(lines) > cap:
                    lines.popitem(last=False)
            # the server's time in 2^-16 cycles: a line may take less than a cycle
            q = cdiv(LINE_BYTES << 32, H.get(rec, "rate_dram" if miss else "rate_l2"))
            m = a * 65536 if nocont else max(a * 65536, av[miss])
            av[miss] = m + q
            left = s + cdiv((j + 1) * LINE_BYTES * 65536, rg)
            f = max(left, cdiv(m + q, 65536)) + H.get(rec, "lat_dram" if miss else "lat_l2")
            tx_fin[v] = max(tx_fin.get(v, 0), f)
            if j == len(txn[v]) - 1:
                assert fi[v] == tx_fin[v], f"addressed node {v} finish {fi[v]} != {tx_fin[v]}"
            continue
        dram, occ_m, lat = d["dram"], d["occ_m"], d["lat"]
        tile = int(g.node_tile[v]) if g.node_tile is not None else NO_TILE
        if cap and tile != NO_TILE:
            hits = []
            for i in range(d["lines"]):
                key = (tile, i)
                hits.append(key in lines)
                lines[key] = None
                lines.move_to_end(key)
                while len(lines) > cap:
                    lines.popitem(last=False)
            assert all(hits) or not any(hits), f"node {v}: a whole-tile access hits all its lines or none"
            dram = not all(hits)
            occ_m, lat = (d["occ_dram"], d["lat_dram"]) if dram else (d["occ_l2"], d["lat_l2"])
        m = s if nocont else max(s, cdiv(av[dram], 65536))  # whole cycles, after any transaction
        av[dram] = (m + occ_m) * 65536
        assert fi[v] == max(s + d["occ"], m + occ_m) + lat, f"gmem node {v} finish"
    # CTA dispatch re-simulated from retire cycles
    exp_sm, exp_launch = dispatch_from_retires(g, rec, fi)
    assert np.array_equal(exp_sm, cta_sm), "CTA -> SM mapping"
    assert np.array_equal(exp_launch, launch), "CTA launch cycles"


def tile_transactions(g):
    """Per addressed load / store: the 128-B lines its tile covers, in the
    order its rows first reach them (a set of lines seen, rows in order)."""
    out = {}
    if getattr(g, "node_addr", None) is None:
        return out
    for v in np.flatnonzero(g.node_addr != np.uint64(0xFFFFFFFFFFFFFFFF)).tolist():
        p = int(g.node_op[v])
        R = int(g.op_rows[p]) if g.op_rows is not None else 1
        W = int(g.op_work[p]) // R
        P = int(g.op_pitch[p]) if g.op_pitch is not None else W
        a = int(g.node_addr[v])
        seen, order = set(), []
        for r in range(R):
            lo, hi = (a + r * P) // LINE_BYTES, (a + r * P + W - 1) // LINE_BYTES
            for line in range(lo, hi + 1):
                if line not in seen:
                    seen.add(line)
                    order.append(line)
        out[v] = order
    return out


def cluster_first(g, c: int) -> int:
    k = int(g.cta_kernel()[c])
    kb, cl = int(g.kernel_cta_begin[k]), int(g.kernel_cluster[k])
    return kb + (c - kb) // cl * cl


def noc_route(src_sm: int, dst_sm: int, D: int, W: int):
    """Servers a transfer between two SMs of one NoC domain holds, and the
    latency multiplier: a crossbar's injection and ejection ports (one
    traversal), or the mesh links of the dimension-order route, x first
    (one latency per hop)."""
    dom, a, b = src_sm // D, src_sm % D, dst_sm % D
    assert dst_sm // D == dom
    if W == 0:
        return [("in", dom, a), ("out", dom, b)], 1
    (x, y), (xb, yb) = (a % W, a // W), (b % W, b // W)
    links = []
    while x != xb:
        step = 1 if xb > x else -1
        links.append(("x", dom, x, y, step))
        x += step
    while y != yb:
        step = 1 if yb > y else -1
        links.append(("y", dom, x, y, step))
        y += step
    return links, len(links)


def cluster_placements(rec, cl: int):
    """Every placement of a cluster of cl CTAs, in the order dispatch tries
    them: lists of SMs by rank, domain by domain; strips of consecutive
    nodes, (compact mapping on a mesh) the most square bw x bh blocks that
    tile the mesh, row-major, or (strided mapping) ranks D / cl nodes apart."""
    D, W = H.get(rec, "noc_nodes"), H.get(rec, "noc_width")
    nsm = H.get(rec, "n_sm")
    shape = None
    if H.get(rec, "noc_map") == 1 and W:
        Hh = D // W
        fits = [bh for bh in range(1, cl + 1) if cl % bh == 0 and bh * bh <= cl and W % (cl // bh) == 0
                and Hh % bh == 0]
        shape = (cl // max(fits), max(fits)) if fits else None
    per_domain = []
    if shape:
        bw, bh = shape
        for by in range(D // W // bh):
            for bx in range(W // bw):
                per_domain.append([(by * bh + r // bw) * W + bx * bw + r % bw for r in range(cl)])
    elif H.get(rec, "noc_map") == 2:  # strided: ranks spread D / cl apart
        per_domain = [[j + r * (D // cl) for r in range(cl)] for j in range(D // cl)]
    else:
        per_domain = [[j * cl + r for r in range(cl)] for j in range(D // cl)]
    out = []
    for d in range(-(-nsm // D)):
        for nodes in per_domain:
            sms = [d * D + n for n in nodes]
            if all(s < nsm for s in sms):
                out.append(sms)
    return out


def dispatch_from_retires(g, rec, finish):
    """CTA (sm, launch) implied by each CTA's retire cycle (max finish of its
    nodes): in-order dispatch at t = 0 and at each retire cycle, to the SM
    with the most free slots (lowest id on ties), kernels in sequence."""
    C, K = g.n_ctas, g.n_kernels
    node_cta = g.node_cta()
    retire = np.zeros(C, dtype=np.int64)
    np.maximum.at(retire, node_cta, finish.astype(np.int64))
    cta_kernel = g.cta_kernel()
    slots = slots_per_kernel(g, rec)
    nsm = H.get(rec, "n_sm")
    kb = g.kernel_cta_begin.astype(np.int64)
    resident = [0] * nsm
    sm_of = np.full(C, -1, dtype=np.int64)
    launch = np.zeros(C, dtype=np.int64)
    kstart = {}
    nxt, retired = 0, 0
    pending = []  # (retire cycle, cta) of dispatched CTAs

    def dispatch(t):
        nonlocal nxt
        while nxt < C:
            k = int(cta_kernel[nxt])
            if retired < kb[k]:
                return
            cl = int(g.kernel_cluster[k])
            if cl > 1:  # a whole cluster on the first placement with room on each SM
                fit = [p for p in cluster_placements(rec, cl) if all(resident[s] < slots[k] for s in p)]
                if not fit:
                    return
                kstart.setdefault(k, t)
                la = t + H.get(rec, "cta_launch_lat") + (H.get(rec, "kernel_launch_lat") if kstart[k] == t else 0)
                for r, s in enumerate(fit[0]):
                    sm_of[nxt + r], launch[nxt + r] = s, la
                    resident[s] += 1
                    pending.append((int(retire[nxt + r]), nxt + r))
                nxt += cl
                continue
            free = [slots[k] - resident[m] for m in range(nsm)]
            best = max(range(nsm), key=lambda m: (free[m], -m))
            if free[best] <= 0:
                return
            kstart.setdefault(k, t)
            la = t + H.get(rec, "cta_launch_lat") + (H.get(rec, "kernel_launch_lat") if kstart[k] == t else 0)
            sm_of[nxt], launch[nxt] = best, la
            resident[best] += 1
            pending.append((int(retire[nxt]), nxt))
            nxt += 1

    dispatch(0)
    while pending:
        pending.sort()
        t = pending[0][0]
        while pending and pending[0][0] == t:
            _, c = pending.pop(0)
            resident[sm_of[c]] -= 1
            retired += 1
        dispatch(t)
    return sm_of, launch


def asap_bruteforce(g, rec, flags=0):
    """Uncontended starts by enumerating every path (tiny single-kernel graphs
    whose CTAs all launch in the first dispatch step)."""
    dur = durations(g, rec)
    ops = g.node_op.astype(np.int64)
    N = g.n_nodes
    launch0 = H.get(rec, "cta_launch_lat") + H.get(rec, "kernel_launch_lat")
    preds = [[] for _ in range(N)]
    for u, v, k in zip(g.sources(), g.targets(), g.kinds()):
        w = 1 if (k == ORDER and not (flags & 8)) else node_duration(dur[ops[u]])
        preds[int(v)].append((int(u), w))
    best = [None] * N

    def paths_to(v):  # all path weights ending at v, by explicit enumeration
        if not preds[v]:
            return [launch0]
        out = [launch0]
        for u, w in preds[v]:
            out += [x + w for x in paths_to(u)]
        return out

    for v in range(N):
        best[v] = max(paths_to(v))
    starts = np.array(best, dtype=np.int64)
    finishes = starts + np.array([node_duration(dur[ops[v]]) for v in range(N)], dtype=np.int64)
    return starts, finishes


def load_golden():
    with open(GOLDEN) as f:
        doc = json.load(f)
    cases = {c["name"]: c for c in doc["cases"]}
    out = []
    for c in doc["cases"]:
        src = cases[c["same_graph_as"]] if "same_graph_as" in c else c
        b = GraphBuilder()
        tiles = []
        for k in src["kernels"]:
            b.kernel(k["warps"], k["smem"], k.get("cluster", 1))
            for cta in k["ctas"]:
                b.cta()
                for cls, work, warps, extra, *tile in cta:
                    # fourth field: the L2-miss flag, or a REMOTE node's target rank;
                    # optional fifth: the tile a load / store touches, as an id or
                    # as {"addr", "rows", "pitch"} (transaction-level memory)
                    flags = remote_flags(extra) if cls == "REMOTE" else (1 if extra else 0)
                    if tile and isinstance(tile[0], dict):
                        t = tile[0]
                        b.node(CLASS[cls], work, warps, flags, addr=t["addr"], rows=t.get("rows", 1),
                               pitch=t.get("pitch", 0))
                        tiles.append(NO_TILE)
                    else:
                        b.node(CLASS[cls], work, warps, flags)
                        tiles.append(tile[0] if tile else NO_TILE)
        for u, v, kd in src["edges"]:
            b.edge(u, v, KIND[kd])
        g = b.build(c["name"])
        if any(t != NO_TILE for t in tiles):
            g.node_tile = np.array(tiles, dtype=np.uint32)
        rec = H.toy(**c["hw"])
        out.append((c, g, rec))
    return out

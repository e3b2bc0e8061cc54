"""Software-pipelining case study workloads (GTSim Sec. 4.2 pipeline
organisations, Sec. 7.1 case study, Table 4 tile-graph ablation).

A fused GEMM + SiLU persistent kernel: one thread block on one SM computes
`waves` output tiles (BM x BN, K = 1024 by default) one after another; the
four organisations differ only in which warp group runs which tile
operations and in the dependency edges between them:

* ``naive``       -- one warp group issues the TMA loads, the MMAs and the
                     epilogue of every tile in program order; the next
                     tile's loads follow the epilogue.
* ``cooperative`` -- warp-specialised: a producer warp issues every load;
                     two consumer warp groups split each tile by rows and
                     run its MMAs and epilogue together.
* ``pingpong``    -- warp-specialised: each tile is split into two
                     row-halves, one per consumer warp group, each with a
                     full mainloop of its own (B is loaded once per half,
                     the extra TMA traffic of this organisation); the two
                     groups' mainloops alternate, so one group's epilogue
                     overlaps the other's mainloop.
* ``threestage``  -- warp-specialised with a dedicated epilogue group: the
                     MMA group moves on to the next tile while the epilogue
                     group finishes the previous one (a DATA edge from the
                     last MMA of a tile to its epilogue; two accumulator
                     buffers).

Loads reuse `stages` shared-memory buffers: the load of pipeline step g waits
(SYNC) for the MMAs of step g - stages.  Each warp group's program order is
an ORDER chain.  Operands are FP8 (1 byte), the output FP16.  The first
tile's A panel misses L2 and later tiles hit it; B panels and stores miss.

The Table 4 ablation (no ORDER edges, no SYNC edges, DATA edges only) is
`gemm_silu(..., drop=kinds)`: the generator never adds edges of those kinds,
so a pair joined by both a dropped and a kept kind keeps the kept edge.
`without_edges` removes kinds from any built graph; there a pair whose edges
were merged into the strongest kind (DATA > SYNC > ORDER) goes entirely.
"""
from __future__ import annotations

import numpy as np

from . import hw as H
from .graph import (ALU, DATA, GLOAD, GSTORE, MISS, ORDER, SFU, SYNC_EDGE, TENSOR, GraphBuilder, TileGraph,
                    csr_from_edges)
from .rng import SplitMix64

ORGANIZATIONS = ("naive", "cooperative", "pingpong", "threestage")
TILES = ((128, 128, 64), (128, 256, 64), (256, 128, 64), (256, 256, 64), (256, 256, 128))
FP8, FP16 = 1, 2
WG0, WG1 = 0x00F, 0x0F0   # warp groups 0 (warps 0-3) and 1 (warps 4-7)
PRODUCER = 0x100          # warp 8


def gemm_silu(org: str, BM: int = 128, BN: int = 128, BK: int = 64, K: int = 1024, waves: int = 10,
              stages: int = 2, drop=()) -> TileGraph:
    """Persistent fused GEMM + SiLU on one CTA (see the module docstring);
    edges of the kinds in `drop` are left out."""
    if org not in ORGANIZATIONS:
        raise ValueError(f"organisation {org!r} not in {ORGANIZATIONS}")
    if K % BK or BM % 2:
        raise ValueError("K must be a multiple of BK and BM even")
    T = K // BK
    b = GraphBuilder(drop)
    warps = 4 if org == "naive" else 9
    b.kernel(warps, stages * (BM + BN) * BK * FP8)
    b.cta()
    order = {}     # warp group -> its nodes in program order
    mma_of = {}    # pipeline step -> MMA nodes that read its buffers
    step = [0]     # next pipeline step (buffer use) of the producer side

    def seq(group, v):
        order.setdefault(group, []).append(v)
        return v

    def load_step(group, rows_a, w, with_b=True):
        """TMA loads of one pipeline step: A (rows_a x BK) and B (BN x BK)."""
        g = step[0]
        step[0] += 1
        a = seq(group, b.node(GLOAD, rows_a * BK * FP8, group, MISS if w == 0 else 0))
        bb = seq(group, b.node(GLOAD, BN * BK * FP8, group, MISS)) if with_b else None
        for m in mma_of.get(g - stages, []):  # buffer reuse
            b.edge(m, a, SYNC_EDGE)
            if bb is not None:
                b.edge(m, bb, SYNC_EDGE)
        return g, a, bb

    def mma(group, rows, g, a, bb, prev):
        m = seq(group, b.node(TENSOR, 2 * rows * BN * BK, group))
        b.edge(a, m, DATA)
        b.edge(bb, m, DATA)
        if prev is not None:
            b.edge(prev, m, DATA)  # accumulator
        mma_of.setdefault(g, []).append(m)
        return m

    def epilogue(group, rows, last_mma):
        s = seq(group, b.node(SFU, rows * BN, group))        # sigmoid
        x = seq(group, b.node(ALU, rows * BN, group))        # x * sigmoid(x)
        st = seq(group, b.node(GSTORE, rows * BN * FP16, group, MISS))
        b.edge(last_mma, s, DATA)
        b.edge(s, x, DATA)
        b.edge(x, st, DATA)
        return st

    if org == "naive":
        for w in range(waves):
            pending = [load_step(WG0, BM, w) for _ in range(min(stages - 1, T))]
            prev = None
            for k in range(T):
                if k + stages - 1 < T:
                    pending.append(load_step(WG0, BM, w))
                g, a, bb = pending.pop(0)
                prev = mma(WG0, BM, g, a, bb, prev)
            epilogue(WG0, BM, prev)
    elif org == "cooperative":
        half = BM // 2
        for w in range(waves):
            prev = [None, None]
            for k in range(T):
                g, a, bb = load_step(PRODUCER, BM, w)
                prev = [mma(grp, half, g, a, bb, prev[i]) for i, grp in enumerate((WG0, WG1))]
            for i, grp in enumerate((WG0, WG1)):
                epilogue(grp, half, prev[i])
    elif org == "pingpong":
        half = BM // 2
        last_main = None  # last MMA of the previous half-tile mainloop (the other group)
        for w in range(waves):
            for i, grp in enumerate((WG0, WG1)):
                prev = None
                for k in range(T):
                    g, a, bb = load_step(PRODUCER, half, w)
                    prev = mma(grp, half, g, a, bb, prev)
                    if k == 0 and last_main is not None:
                        b.edge(last_main, prev, SYNC_EDGE)  # mainloops alternate between the groups
                last_main = prev
                epilogue(grp, half, prev)
    else:  # threestage
        stores = []
        for w in range(waves):
            prev = None
            for k in range(T):
                g, a, bb = load_step(PRODUCER, BM, w)
                prev = mma(WG0, BM, g, a, bb, prev)
                if k == 0 and w >= 2:
                    b.edge(stores[w - 2], prev, SYNC_EDGE)  # accumulator buffer w mod 2 is free again
            stores.append(epilogue(WG1, BM, prev))
    for nodes in order.values():
        for u, v in zip(nodes[:-1], nodes[1:]):
            b.edge(u, v, ORDER)
    names = {DATA: "data", ORDER: "order", SYNC_EDGE: "sync"}
    tag = "".join("_no_" + names[k] for k in sorted(set(int(k) for k in drop)))
    g = b.build(f"gemm_silu_{org}_{BM}x{BN}x{BK}_w{waves}{tag}")
    g.meta = dict(org=org, BM=BM, BN=BN, BK=BK, K=K, waves=waves, stages=stages, drop=tuple(sorted(drop)))
    return g


def without_edges(g: TileGraph, kinds) -> TileGraph:
    """The same graph with every edge of the given kinds removed."""
    kinds = set(int(k) for k in kinds)
    ptr = g.succ_ptr.astype(np.int64)
    src = np.repeat(np.arange(g.n_nodes, dtype=np.int64), np.diff(ptr))
    dst = (g.succ & np.uint32((1 << 30) - 1)).astype(np.int64)
    kind = (g.succ >> np.uint32(30)).astype(np.int64)
    keep = ~np.isin(kind, sorted(kinds))
    succ_ptr, succ = csr_from_edges(g.n_nodes, src[keep], dst[keep], kind[keep])
    names = {DATA: "data", ORDER: "order", SYNC_EDGE: "sync"}
    return TileGraph(op_cls=g.op_cls, op_flags=g.op_flags, op_work=g.op_work, op_warps=g.op_warps,
                     node_op=g.node_op, succ_ptr=succ_ptr, succ=succ, cta_node_begin=g.cta_node_begin,
                     kernel_cta_begin=g.kernel_cta_begin, kernel_warps=g.kernel_warps, kernel_smem=g.kernel_smem,
                     name=g.name + "_no_" + "_".join(names[k] for k in sorted(kinds)), meta=dict(g.meta),
                     kernel_cluster=g.kernel_cluster)


ABLATIONS = {"full": (), "no_order": (ORDER,), "no_sync": (SYNC_EDGE,), "data_only": (ORDER, SYNC_EDGE)}


def case_study_graphs():
    """(organisation, tile, ablation) for every case-study graph: four
    organisations x five tile shapes x the four Table 4 edge-class sets."""
    return [(org, tile, abl) for abl in ABLATIONS for tile in TILES for org in ORGANIZATIONS]


def case_study_graph(index: int) -> TileGraph:
    org, tile, abl = case_study_graphs()[index]
    return gemm_silu(org, *tile, drop=ABLATIONS[abl])


def sample_hopper_1sm(seed: int, B: int) -> np.ndarray:
    """Single-SM Hopper machines around Table 3's H100: tensor rate 0.5-4x
    (FP8 is 2x), DRAM 1.5-8 TB/s and TMA issue rate 50-200 B/cycle, each
    uniform."""
    rng = SplitMix64(seed, 11)
    out = np.zeros((B, H.NWORDS), dtype=np.uint32)
    for b in range(B):
        tp = rng.randint(500, 4000)
        mb = rng.randint(1_500_000, 8_000_000)
        tma = rng.randint(50, 200)
        out[b] = H.preset("H100", n_sm=1, tensor_permille=tp, dram_mb_s=mb, rate_gmem=tma * H.Q16)
    return out

"""Seeded random graphs that the windowed kernel accepts (test helper).

The windowed kernel takes a graph when every node without a successor in its
own CTA is a global load or store, every edge between CTAs leaves a load or
store and is a DATA or SYNC edge, out-degrees stay below 0xFFFF, no kernel
has clusters, every named tile (LRU L2) has fewer than 2^22 lines, and
byte addresses (transaction-level memory), if any, sit on every load and
store, each of at least one byte.  These graphs meet that and otherwise vary what
the kernel has to get right: 1-4 kernels of 1-32 warps, CTAs of a few to
several dozen nodes of every class (zero-work nodes included), all three
edge kinds inside a CTA, fan-outs beyond the three successors a node record
carries inline, and loads / stores with edges into later CTAs (of the same or
a later kernel), whose targets then have in-edges from several CTAs.

`window_eligible` states the host's rule directly, so a CPU test can check
the generator without the library's internals."""
import numpy as np

from paper_2607_11262_amd.gen.graph import (ALU, DATA, GLOAD, GSTORE, LINE_BYTES, MISS, NO_ADDR, NO_TILE, ORDER, SFU,
                                             SMEM, SYNC, SYNC_EDGE, TENSOR, GraphBuilder)
from paper_2607_11262_amd.gen import hw as H

MEM = (GLOAD, GSTORE)
# SM counts on both sides of the 64 / 128 / 192 / 256-SM boundaries where the
# windowed kernel changes how many SMs one lane carries
SM_COUNTS = (1, 2, 3, 63, 64, 65, 127, 128, 129, 191, 192, 193, 255, 256)


def windowed_graph(rng, n_kernels=(1, 4), ctas=(1, 12), nodes=(1, 40), cross_p=8):
    b = GraphBuilder()
    cta_nodes = []  # per CTA: (node ids, classes)
    nk = rng.randint(*n_kernels)
    for _k in range(nk):
        warps = rng.choice([1, 2, 4, 5, 8, 13, 32, rng.randint(1, 32)])
        b.kernel(warps, rng.choice([0, 0, 1024, 16 * 1024, 64 * 1024]))
        for _c in range(rng.randint(*ctas)):
            b.cta()
            n = rng.randint(*nodes)
            edges = set()
            kinds = {}
            for v in range(1, n):
                for u in sorted({rng.randint(0, v - 1) for _ in range(rng.randint(0, 3))}):
                    edges.add((u, v))
                    kinds[(u, v)] = rng.choice([DATA, DATA, ORDER, SYNC_EDGE])
            for _ in range(rng.randint(0, 2)):  # fan-outs beyond the inline three
                u = rng.randint(0, max(0, n - 5))
                for v in range(u + 1, min(n, u + rng.randint(4, 9))):
                    if (u, v) not in edges:
                        edges.add((u, v))
                        kinds[(u, v)] = rng.choice([DATA, SYNC_EDGE, ORDER])
            has_succ = {u for u, _ in edges}
            ids, classes = [], []
            for i in range(n):
                cls = rng.choice(list(MEM)) if i not in has_succ else rng.choice(
                    [TENSOR, ALU, SFU, SMEM, GLOAD, GLOAD, GSTORE, SYNC])
                if rng.randint(0, 7) == 0 or cls == SYNC:
                    work = 0
                elif cls in MEM or cls == SMEM:
                    work = rng.randint(1, 1 << 15)
                else:
                    work = rng.randint(1, 1 << 20)
                mask = 0
                while mask == 0:
                    mask = rng.randint(0, (1 << warps) - 1) if warps < 32 else rng.randint(1, 0xFFFFFFFF)
                flags = MISS if cls in MEM and rng.randint(0, 1) else 0
                ids.append(b.node(cls, work, mask, flags))
                classes.append(cls)
            for (u, v) in sorted(edges):
                b.edge(ids[u], ids[v], kinds[(u, v)])
            cta_nodes.append((ids, classes))
    # edges between CTAs: from a load / store into any node of a later CTA
    for ci, (ids, classes) in enumerate(cta_nodes):
        later = cta_nodes[ci + 1:]
        if not later:
            continue
        for u, cls in zip(ids, classes):
            if cls not in MEM or rng.randint(0, cross_p - 1) != 0:
                continue
            for _ in range(rng.randint(1, 3)):
                tids, _ = later[rng.randint(0, min(len(later), 4) - 1)]
                v = tids[rng.randint(0, len(tids) - 1)]
                b.edge(u, v, rng.choice([DATA, SYNC_EDGE]))  # duplicates merge at build
    return b.build("windowed_random")


def window_eligible(g) -> bool:
    """The windowed kernel's graph conditions, written out."""
    if g.n_nodes == 0 or np.any(np.asarray(g.kernel_cluster) > 1):
        return False
    cls = np.asarray(g.op_cls)[np.asarray(g.node_op, np.int64)]
    if getattr(g, "node_addr", None) is not None and np.any(np.asarray(g.node_addr) != NO_ADDR):
        mem = np.isin(cls, MEM)
        work = np.asarray(g.op_work, np.int64)[np.asarray(g.node_op, np.int64)]
        if np.any(mem & ((np.asarray(g.node_addr) == NO_ADDR) | (work == 0))):
            return False
    if g.node_tile is not None:
        named = np.asarray(g.node_tile) != NO_TILE
        work = np.asarray(g.op_work, np.int64)[np.asarray(g.node_op, np.int64)]
        if np.any(named & (-(-work // LINE_BYTES) >= 1 << 22)):
            return False
    if np.any(cls == 7):  # REMOTE
        return False
    cta = np.repeat(np.arange(len(g.cta_node_begin) - 1), np.diff(np.asarray(g.cta_node_begin, np.int64)))
    ptr = np.asarray(g.succ_ptr, np.int64)
    if np.any(np.diff(ptr) >= 0xFFFF):
        return False
    src = np.repeat(np.arange(g.n_nodes), np.diff(ptr))
    tgt = (np.asarray(g.succ, np.int64) & 0x3FFFFFFF)
    kind = np.asarray(g.succ, np.int64) >> 30
    cross = cta[src] != cta[tgt]
    if np.any(cross & ~np.isin(cls[src], MEM)) or np.any(cross & (kind == ORDER)):
        return False
    intra_succ = np.zeros(g.n_nodes, bool)
    intra_succ[src[~cross]] = True
    return bool(np.all(intra_succ | np.isin(cls, MEM)))


def windowed_machines(rng, B):
    """B random machines whose SM counts straddle the windowed kernel's
    lane boundaries, with up to eight subpartitions."""
    recs = []
    for _ in range(B):
        r = H.sample_random(rng, n_sm_max=256)
        r[H.FIELDS["n_sm"]] = rng.choice(SM_COUNTS) if rng.randint(0, 2) else rng.randint(1, 256)
        r[H.FIELDS["n_subpart"]] = rng.choice([1, 2, 3, 4, 8])
        r[H.FIELDS["max_cta_per_sm"]] = rng.randint(1, 8)
        r[H.FIELDS["max_warps_per_sm"]] = rng.randint(32, 64)
        r[H.FIELDS["smem_per_sm"]] = rng.randint(64, 228) * 1024
        recs.append(r)
    return np.stack(recs)

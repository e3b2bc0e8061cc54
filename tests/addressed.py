"""Seeded tile addresses for the loads and stores of a graph (test helper,
transaction-level memory): each memory op gets a random tile shape (rows
dividing its bytes, a row stride at least the row length, sometimes with
padding), each load / store a random byte address in a few-KiB window so
lines are shared and reused across nodes."""
import numpy as np

from paper_2607_11262_amd.gen.graph import GLOAD, GSTORE, NO_ADDR


def with_addresses(g, rng, tracked=0.85, window=16384):
    P = g.n_ops
    rows = np.ones(P, dtype=np.uint32)
    pitch = np.zeros(P, dtype=np.uint32)
    for p in range(P):
        work = int(g.op_work[p])
        if int(g.op_cls[p]) in (GLOAD, GSTORE) and work > 0:
            divisors = [d for d in (1, 2, 4, 8, 16, 32) if work % d == 0]
            rows[p] = rng.choice(divisors)
            W = work // int(rows[p])
            pitch[p] = W + rng.choice([0, 0, 16, 64, 128, 4 * W])
        else:
            pitch[p] = max(1, work)
    ops = g.node_op.astype(np.int64)
    mem = np.isin(g.op_cls, (GLOAD, GSTORE))[ops] & (g.op_work[ops] > 0)
    addr = np.full(g.n_nodes, NO_ADDR, dtype=np.uint64)
    for v in np.flatnonzero(mem).tolist():
        if rng.randint(0, 999) < tracked * 1000:
            addr[v] = rng.randint(0, window // 16) * 16 + rng.choice([0, 0, 0, 1 << 40])
    g.node_addr = addr
    g.op_rows = rows
    g.op_pitch = pitch
    g.node_tile = None
    return g

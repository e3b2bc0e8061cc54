"""Seeded graphs whose kernels replicate one random CTA graph (test helper).

Each kernel draws a random DAG of local nodes (out-degrees up to six, all
three edge kinds) and replicates it over its CTAs; every CTA picks, per node,
one of a few op variants (the same class, work and warps, with or without
the L2-miss flag), so the CTAs of a kernel fall into a handful of op
classes.  Nodes without a successor are stores, so the graphs meet the
windowed kernel's conditions.  Optionally one kernel gets a cross-CTA edge
(which rules out its template)."""
import numpy as np

from paper_2607_11262_amd.gen.graph import (ALU, DATA, GLOAD, GSTORE, ORDER, SFU, SYNC_EDGE, TENSOR, GraphBuilder)


def templated_graph(rng, n_kernels=3, n_local=(4, 40), n_ctas=(2, 40), cross_kernel=None):
    b = GraphBuilder()
    for k in range(n_kernels):
        n = rng.randint(*n_local)
        C = rng.randint(*n_ctas)
        edges = []
        for v in range(1, n):
            for u in sorted({rng.randint(0, v - 1) for _ in range(rng.randint(0, 3))}):
                edges.append((u, v, rng.choice([DATA, DATA, ORDER, SYNC_EDGE])))
        # a few wide fan-outs (more than the three inline successors)
        for _ in range(rng.randint(0, 2)):
            u = rng.randint(0, max(0, n - 6))
            for v in range(u + 1, min(n, u + 7)):
                if (u, v) not in {(a, c) for a, c, _ in edges}:
                    edges.append((u, v, DATA))
        has_succ = {u for u, _, _ in edges}
        cls = [GSTORE if i not in has_succ else rng.choice([TENSOR, ALU, SFU, GLOAD, GLOAD, GSTORE])
               for i in range(n)]
        work = [rng.randint(1, 1 << 14) for _ in range(n)]
        warps = [rng.choice([1, 2, 0xF, 0x3]) for _ in range(n)]
        n_class = rng.randint(1, 4)
        variants = [[rng.randint(0, 1) for _ in range(n)] for _ in range(n_class)]
        b.kernel(4, rng.choice([0, 1024, 8192]))
        for c in range(C):
            b.cta()
            var = variants[rng.randint(0, n_class - 1)]
            base = len(b.node_op)
            for i in range(n):
                flags = var[i] if cls[i] in (GLOAD, GSTORE) else 0
                b.node(cls[i], work[i] if not var[i] or cls[i] in (GLOAD, GSTORE) else work[i] + 1, warps[i], flags)
            for u, v, kind in edges:
                b.edge(base + u, base + v, kind)
            if cross_kernel == k and c == 1:
                # from a store of CTA 0 into a root of this CTA
                stores = [i for i in range(n) if cls[i] == GSTORE]
                b.edge(base - n + stores[0], base + 0, DATA)
    return b.build("templated")

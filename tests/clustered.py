"""Seeded random graphs with thread-block clusters and REMOTE nodes, and
random machines with an SM-cluster NoC (test helper).

Kernels have clusters of 1-8 CTAs; nodes draw every class, REMOTE nodes a
random target rank; edges join nodes of one cluster in either CTA order
(acyclic: an edge always goes from lower to higher in a random priority
order of the cluster's nodes)."""
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen.graph import (ALU, DATA, GLOAD, GSTORE, MISS, ORDER, REMOTE, SFU, SMEM, SYNC,
                                             SYNC_EDGE, TENSOR, GraphBuilder, remote_flags)

CLASSES = [TENSOR, ALU, SFU, SMEM, GLOAD, GSTORE, SYNC, REMOTE, REMOTE, REMOTE]


def clustered_graph(rng, n_kernels=(1, 3), clusters=(1, 4), nodes=(1, 8), cluster_sizes=(1, 2, 3, 4, 8)):
    b = GraphBuilder()
    for _ in range(rng.randint(*n_kernels)):
        cl = rng.choice(list(cluster_sizes))
        b.kernel(4, rng.choice([0, 1024, 16384]), cl)
        for _ in range(rng.randint(*clusters)):
            members = []
            for _ in range(cl):
                b.cta()
                for _ in range(rng.randint(*nodes)):
                    cls = rng.choice(CLASSES)
                    if cls == REMOTE:
                        flags = remote_flags(rng.randint(0, cl - 1))
                    elif cls in (GLOAD, GSTORE):
                        flags = MISS if rng.randint(0, 1) else 0
                    else:
                        flags = 0
                    members.append(b.node(cls, rng.randint(0, 1 << 13), rng.choice([1, 2, 3, 0xF]), flags))
            prio = list(range(len(members)))
            for i in range(len(prio) - 1, 0, -1):  # Fisher-Yates with the seeded stream
                j = rng.randint(0, i)
                prio[i], prio[j] = prio[j], prio[i]
            rank = {v: prio[i] for i, v in enumerate(members)}
            seen = set()
            for _ in range(rng.randint(0, 2 * len(members))):
                u, v = rng.choice(members), rng.choice(members)
                if u == v or (u, v) in seen or (v, u) in seen:
                    continue
                if rank[u] > rank[v]:
                    u, v = v, u
                seen.add((u, v))
                b.edge(u, v, rng.choice([DATA, DATA, ORDER, SYNC_EDGE]))
    return b.build("clustered")


def noc_machine(rng):
    """A random small machine with a crossbar or mesh NoC."""
    rec = H.sample_random(rng, n_sm_max=4)
    D = rng.choice([4, 8, 16])
    width = rng.choice([0, 2, 4]) if D % 4 == 0 else rng.choice([0, 2])
    rec[H.FIELDS["n_sm"]] = rng.randint(max(1, D // 2), 3 * D)
    rec[H.FIELDS["noc_nodes"]] = D
    rec[H.FIELDS["noc_width"]] = width
    rec[H.FIELDS["noc_rate"]] = rng.randint(H.Q16 // 2, 64 * H.Q16)
    rec[H.FIELDS["noc_lat"]] = rng.randint(0, 300)
    rec[H.FIELDS["noc_map"]] = rng.randint(0, 2)
    rec[H.FIELDS["max_warps_per_sm"]] = 64
    rec[H.FIELDS["smem_per_sm"]] = 64 * 1024
    return rec

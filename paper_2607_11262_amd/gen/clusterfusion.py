"""NoC-enabled fusion case study (GTSim Sec. 7.2): a fused attention block
for one decode step, one thread-block cluster per attention head, in the
manner of ClusterFusion.

Each CTA of a head's cluster (rank r of S) owns a 1/S slice of the hidden
dimension, of the head's QKV outputs and of the KV sequence:

  RMSNorm      load its x slice, sum of squares (ALU)      -> reduce #1
  QKV proj.    load the full x and its W_qkv rows, MMA       -> gather #2
  RoPE         rotate q and k (ALU)
  attention    per 64-token KV tile: load K, V; QK^T, softmax (SFU), PV
               local max                                     -> reduce #3
               rescale the local sum (ALU)                   -> reduce #4
               rescale the local output (ALU)                -> reduce #5
  O proj.      load its W_o columns, MMA, store its output slice

so the cluster communicates four reductions and one gather, as the paper
lists them.  Communication is either over the SM-cluster NoC (each CTA
writes its partial into every peer's shared memory with a REMOTE node, and
each CTA waits at a barrier for its peers' writes) or through DRAM (each CTA
stores its partial, every CTA waits for all stores, then loads its peers'
partials).  Both variants use the same clusters and placement.

FP16 activations and weights (2 B), FP32 partial statistics (4 B).
"""
from __future__ import annotations

from . import hw as H
from .graph import (ALU, DATA, GLOAD, GSTORE, MISS, ORDER, REMOTE, SFU, SYNC, SYNC_EDGE, TENSOR, GraphBuilder,
                    TileGraph, remote_flags)

FP16, FP32 = 2, 4
WG = 0xF       # one warp group issues everything of a CTA
KV_TILE = 64
CLUSTER_SIZES = (2, 4, 8, 16)
COMMS = ("noc", "dram")


def cluster_attention(cluster: int = 4, heads: int = 32, hidden: int = 4096, head_dim: int = 128,
                      kv_len: int = 4096, comm: str = "noc") -> TileGraph:
    S, d = int(cluster), int(head_dim)
    if comm not in COMMS:
        raise ValueError(f"comm {comm!r} not in {COMMS}")
    if hidden % S or (3 * d) % S or kv_len % (S * KV_TILE):
        raise ValueError("hidden, 3 * head_dim and kv_len / 64 must split evenly over the cluster")
    tiles = kv_len // (S * KV_TILE)
    b = GraphBuilder()
    b.kernel(4, 64 * 1024, S)
    for h in range(heads):
        # one head: per rank, named nodes in program order; edges by name
        nodes = [[] for _ in range(S)]   # (name, cls, work, flags, warps)
        edges = []                       # ((rank, name), (rank, name), kind)

        def node(r, name, cls, work, flags=0, warps=WG):
            nodes[r].append((name, cls, work, flags, warps))
            return (r, name)

        def edge(u, v, kind=DATA):
            edges.append((u, v, kind))

        def exchange(tag, src, dst, dst_cls, dst_work, nbytes):
            """All-to-all of each rank's `src` result; node `dst` runs once
            every peer's part has arrived."""
            if comm == "noc":
                for r in range(S):
                    for p in range(S):
                        if p != r:
                            w = node(r, f"{tag}_to{p}", REMOTE, nbytes, remote_flags(p), warps=1)
                            edge((r, src), w)
                            edge(w, (p, f"{tag}_bar"))
                    node(r, f"{tag}_bar", SYNC, 0)
                    edge((r, src), (r, f"{tag}_bar"))
                    node(r, dst, dst_cls, dst_work)
                    edge((r, f"{tag}_bar"), (r, dst))
            else:
                for r in range(S):
                    edge((r, src), node(r, f"{tag}_st", GSTORE, nbytes, MISS))
                    node(r, f"{tag}_bar", SYNC, 0)
                    for p in range(S):
                        edge((p, f"{tag}_st"), (r, f"{tag}_bar"))
                    for p in range(S):
                        if p != r:
                            ld = node(r, f"{tag}_ld{p}", GLOAD, nbytes, MISS)
                            edge((r, f"{tag}_bar"), ld)
                            edge(ld, (r, dst))
                    node(r, dst, dst_cls, dst_work)

        for r in range(S):
            # RMSNorm
            edge(node(r, "ld_x", GLOAD, hidden // S * FP16, MISS if h == 0 else 0), node(r, "sq", ALU, hidden // S))
        exchange("red1", "sq", "norm", ALU, S + hidden // S, FP32)
        for r in range(S):
            # QKV projection on the rank's 3d/S outputs
            qkv = (r, "qkv")
            for src in (node(r, "ld_w", GLOAD, 3 * d // S * hidden * FP16, MISS),
                        node(r, "ld_xf", GLOAD, hidden * FP16), (r, "norm")):
                edge(src, qkv)
            node(r, "qkv", TENSOR, 2 * (3 * d // S) * hidden)
        exchange("gat2", "qkv", "rope", ALU, 2 * d, 3 * d // S * FP16)
        for r in range(S):
            # attention over the rank's KV slice, two K / V buffers
            prev = (r, "rope")
            for t in range(tiles):
                k = node(r, f"ldk{t}", GLOAD, KV_TILE * d * FP16, MISS)
                v = node(r, f"ldv{t}", GLOAD, KV_TILE * d * FP16, MISS)
                qk = node(r, f"qk{t}", TENSOR, 2 * KV_TILE * d)
                sm = node(r, f"sm{t}", SFU, KV_TILE)
                pv = node(r, f"pv{t}", TENSOR, 2 * KV_TILE * d)
                for u, w in ((k, qk), (prev, qk), (qk, sm), (sm, pv), (v, pv)):
                    edge(u, w)
                if t >= 2:
                    edge((r, f"pv{t - 2}"), k, SYNC_EDGE)
                    edge((r, f"pv{t - 2}"), v, SYNC_EDGE)
                prev = pv
            node(r, "attn", ALU, KV_TILE)  # local max of the slice
            edge(prev, (r, "attn"))
        exchange("red3", "attn", "resc", ALU, S + KV_TILE, FP32)
        exchange("red4", "resc", "outs", ALU, d, FP32)
        exchange("red5", "outs", "comb", ALU, S * d, d * FP32)
        for r in range(S):
            # output projection on the rank's hidden/S columns
            wo = node(r, "ld_wo", GLOAD, d * (hidden // S) * FP16, MISS)
            op = node(r, "oproj", TENSOR, 2 * d * (hidden // S))
            edge((r, "comb"), op)
            edge(wo, op)
            edge(op, node(r, "st", GSTORE, hidden // S * FP16, MISS))
        # emit CTA by CTA; each CTA's program order is an ORDER chain
        ids = {}
        for r in range(S):
            b.cta()
            prev_id = None
            for name, cls, work, flags, warps in nodes[r]:
                v = b.node(cls, work, warps, flags)
                ids[(r, name)] = v
                if prev_id is not None:
                    b.edge(prev_id, v, ORDER)
                prev_id = v
        for u, v, kind in edges:
            b.edge(ids[u], ids[v], kind)
    g = b.build(f"cluster_attention_S{S}_{comm}")
    g.meta = dict(cluster=S, heads=heads, hidden=hidden, head_dim=d, kv_len=kv_len, comm=comm)
    return g


def _mesh_hops(W: int, D: int) -> float:
    pts = [(i % W, i // W) for i in range(D)]
    tot = sum(abs(a[0] - b[0]) + abs(a[1] - b[1]) for a in pts for b in pts if a != b)
    return tot / (D * (D - 1))


def noc_h100(topology: str = "crossbar", mapping: str = "strips", port_bytes: int = 32, latency: int = 180,
             **overrides):
    """Table 3's H100 with a 16-node SM-cluster NoC per domain: a crossbar
    (per-port bandwidth, one traversal latency), or a 4 x 4 mesh with the
    same total bandwidth (the 32 crossbar ports' bandwidth spread over the
    48 directed links) and the same average latency between distinct nodes
    (the crossbar latency divided by the mean hop count, 8/3)."""
    D = 16
    maps = {"strips": 0, "blocks": 1, "strided": 2}
    if topology == "crossbar":
        fields = dict(noc_nodes=D, noc_width=0, noc_rate=port_bytes * H.Q16, noc_lat=latency)
    elif topology == "mesh":
        links = 2 * (4 * 3 + 3 * 4)
        fields = dict(noc_nodes=D, noc_width=4, noc_rate=(2 * D * port_bytes * H.Q16) // links,
                      noc_lat=round(latency / _mesh_hops(4, D)))
    else:
        raise ValueError(topology)
    fields["noc_map"] = maps[mapping]
    fields.update(overrides)
    return H.preset("H100", **fields)


def sample_noc_machines(seed: int, B: int):
    """H100 machines with a 16-SM-domain NoC: crossbar or 4 x 4 mesh, any of
    the three mappings, port bandwidth 8-64 B/cycle and crossbar latency
    60-400 cycles (mesh at the equivalent per-hop latency), DRAM 1.5-8 TB/s,
    tensor rate 0.5-4x; each uniform."""
    import numpy as np
    from .rng import SplitMix64
    rng = SplitMix64(seed, 13)
    out = np.zeros((B, H.NWORDS), dtype=np.uint32)
    for b in range(B):
        topo = rng.choice(["crossbar", "mesh"])
        mapping = rng.choice(["strips", "blocks", "strided"])
        port = rng.randint(8, 64)
        lat = rng.randint(60, 400)
        mb = rng.randint(1_500_000, 8_000_000)
        tp = rng.randint(500, 4000)
        out[b] = noc_h100(topo, mapping, port, lat, dram_mb_s=mb, tensor_permille=tp)
    return out

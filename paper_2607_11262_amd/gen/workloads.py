"""Seeded synthetic tile-graph workloads.

The paper simulates TileLang / FlashAttention-family kernels built from its
frontend (Sec. 4.3) and validates them on A100/H100 (Sec. 6).  Neither the
kernels' sources nor measured cycles are used here: each generator encodes
only the tile-level structure the paper describes for the technique
(Sec. 4.2: fused stages linked by data edges, warp-specialised producer /
consumer roles, software-pipeline stages whose buffer reuse is an order
constraint), with tile shapes taken from the workload definitions below.

Every generator is deterministic given its arguments and seed.  Large
graphs are built by replicating one CTA template (all CTAs of a GEMM or
attention kernel are isomorphic up to which tiles miss in L2), so a 20 M
node graph is a handful of numpy operations.
"""
from __future__ import annotations

import numpy as np

from . import hw as hwmod
from .graph import (NO_ADDR, NO_TILE, ALU, DATA, GLOAD, GSTORE, MISS, ORDER, SFU, SYNC, SYNC_EDGE, TENSOR, GraphBuilder,
                    OpTable, TileGraph, csr_from_edges, empty_graph)
from .rng import SplitMix64

FP16 = 2
ALL4 = 0xF       # warp group: warps 0-3
PRODUCER = 0x10  # warp 4


# --------------------------------------------------------------------------
# CTA templates.  Each returns (roles, edges): roles[i] names local node i in
# issue/program order, edges are (u, v, kind) on local ids.
# --------------------------------------------------------------------------

def gemm_template(T: int, S: int, per_warp: bool):
    """Multistage (cp.async / TMA) GEMM mainloop, 4 warps, no warp
    specialisation.  Per k-step i: load A_i, load B_i (all warps), MMA_i
    (whole warp group, or one 32x32 quadrant per warp when per_warp), then
    one store of C.  S pipeline stages: the loads of step j reuse the shared
    buffer of step j-S, so they wait (SYNC) for MMA_{j-S}; program order of
    each warp is an ORDER chain (Sec. 4.2 software pipelining)."""
    roles, prog = [], [[] for _ in range(4)]
    idx = {}

    def add(role, warps):
        idx[role] = len(roles)
        roles.append(role)
        for w in warps:
            prog[w].append(idx[role])

    for j in range(min(S - 1, T)):
        add(("lA", j), range(4))
        add(("lB", j), range(4))
    for i in range(T):
        j = i + S - 1
        if j < T:
            add(("lA", j), range(4))
            add(("lB", j), range(4))
        if per_warp:
            for w in range(4):
                add(("mma", i, w), [w])
        else:
            add(("mma", i, -1), range(4))
    add(("st",), range(4))

    def mmas(i):
        return [idx[("mma", i, w)] for w in range(4)] if per_warp else [idx[("mma", i, -1)]]

    edges = []
    for i in range(T):
        for m in mmas(i):
            edges += [(idx[("lA", i)], m, DATA), (idx[("lB", i)], m, DATA)]
        if i > 0:
            edges += [(a, b, DATA) for a, b in zip(mmas(i - 1), mmas(i))]
        if i >= S:
            for m in mmas(i - S):
                edges += [(m, idx[("lA", i)], SYNC_EDGE), (m, idx[("lB", i)], SYNC_EDGE)]
    edges += [(m, idx[("st",)], DATA) for m in mmas(T - 1)]
    for seq in prog:
        edges += [(a, b, ORDER) for a, b in zip(seq[:-1], seq[1:])]
    return roles, edges


def attention_template(n_tiles: int, stages: int = 2):
    """Warp-specialised flash-attention CTA: producer warp 4 loads Q once and
    K_j, V_j per KV tile; consumer warp group 0-3 runs S_j = Q K_j^T (tensor),
    online softmax (SFU), O += P_j V_j (tensor), then stores O.  K/V buffers
    are `stages`-deep: loading K_j (V_j) waits for QK_{j-stages}
    (PV_{j-stages}) to finish (Sec. 4.2 warp specialisation + pipelining)."""
    roles = [("lQ",)]
    for j in range(n_tiles):
        roles += [("lK", j), ("lV", j), ("qk", j), ("sm", j), ("pv", j)]
    roles.append(("st",))
    idx = {r: i for i, r in enumerate(roles)}
    producer = [idx[("lQ",)]] + [idx[(k, j)] for j in range(n_tiles) for k in ("lK", "lV")]
    consumer = [idx[(k, j)] for j in range(n_tiles) for k in ("qk", "sm", "pv")] + [idx[("st",)]]
    e = [(idx[("lQ",)], idx[("qk", 0)], DATA)]
    for j in range(n_tiles):
        e += [(idx[("lK", j)], idx[("qk", j)], DATA), (idx[("qk", j)], idx[("sm", j)], DATA),
              (idx[("sm", j)], idx[("pv", j)], DATA), (idx[("lV", j)], idx[("pv", j)], DATA)]
        if j > 0:
            e += [(idx[("pv", j - 1)], idx[("pv", j)], DATA), (idx[("sm", j - 1)], idx[("sm", j)], DATA)]
        if j >= stages:
            e += [(idx[("qk", j - stages)], idx[("lK", j)], SYNC_EDGE),
                  (idx[("pv", j - stages)], idx[("lV", j)], SYNC_EDGE)]
    e.append((idx[("pv", n_tiles - 1)], idx[("st",)], DATA))
    for seq in (producer, consumer):
        e += [(a, b, ORDER) for a, b in zip(seq[:-1], seq[1:])]
    return roles, e


def chain_template(n: int):
    """Elementwise CTA: a DATA chain load -> compute ... -> store."""
    roles = [("c", i) for i in range(n)]
    return roles, [(i, i + 1, DATA) for i in range(n - 1)]


# --------------------------------------------------------------------------
# Assembly: kernels made of replicated templates
# --------------------------------------------------------------------------

class _Kernel:
    def __init__(self, warps: int, smem: int):
        self.warps, self.smem = warps, smem
        self.groups = []  # (template CSR ptr, succ, n_local, op matrix [count, n_local])

    def add(self, roles_edges, op_matrix: np.ndarray):
        roles, edges = roles_edges
        n_local = len(roles)
        op_matrix = np.asarray(op_matrix, dtype=np.uint16).reshape(-1, n_local)
        src = np.array([a for a, _, _ in edges], dtype=np.int64)
        dst = np.array([b for _, b, _ in edges], dtype=np.int64)
        kind = np.array([k for _, _, k in edges], dtype=np.int64)
        ptr, succ = csr_from_edges(n_local, src, dst, kind)
        self.groups.append((ptr, succ, n_local, op_matrix))


def _assemble(kernels, ops: OpTable, name: str, meta=None) -> TileGraph:
    node_op_parts, ptr_parts, succ_parts = [], [], []
    cta_sizes, kernel_ctas = [], []
    node_base, edge_base = 0, 0
    for k in kernels:
        nk = 0
        for ptr, succ, n_local, opm in k.groups:
            C = opm.shape[0]
            E = int(ptr[-1])
            node_off = (np.arange(C, dtype=np.uint64) * n_local + node_base).astype(np.uint32)
            edge_off = (np.arange(C, dtype=np.uint64) * E + edge_base).astype(np.uint64)
            ptr_parts.append((ptr[:-1].astype(np.uint64)[None, :] + edge_off[:, None]).ravel())
            succ_parts.append((succ[None, :] + node_off[:, None]).ravel())
            node_op_parts.append(opm.ravel())
            cta_sizes.append(np.full(C, n_local, dtype=np.int64))
            node_base += C * n_local
            edge_base += C * E
            nk += C
        kernel_ctas.append(nk)
    if edge_base >= 1 << 32 or node_base >= 1 << 30:
        raise ValueError("graph too large for the u32 CSR")
    succ_ptr = np.empty(node_base + 1, dtype=np.uint32)
    succ_ptr[:-1] = np.concatenate(ptr_parts) if ptr_parts else np.zeros(0, np.uint64)
    succ_ptr[-1] = edge_base
    cta_node_begin = np.zeros(sum(len(c) for c in cta_sizes) + 1, dtype=np.uint32)
    np.cumsum(np.concatenate(cta_sizes), out=cta_node_begin[1:])
    kernel_cta_begin = np.zeros(len(kernels) + 1, dtype=np.uint32)
    np.cumsum(kernel_ctas, out=kernel_cta_begin[1:])
    cls, flags, work, warps = ops.arrays()
    return TileGraph(op_cls=cls, op_flags=flags, op_work=work, op_warps=warps,
                     node_op=np.concatenate(node_op_parts).astype(np.uint16), succ_ptr=succ_ptr,
                     succ=np.concatenate(succ_parts).astype(np.uint32), cta_node_begin=cta_node_begin,
                     kernel_cta_begin=kernel_cta_begin,
                     kernel_warps=np.array([k.warps for k in kernels], dtype=np.uint16),
                     kernel_smem=np.array([k.smem for k in kernels], dtype=np.uint32), name=name,
                     meta=meta or {})


def _gemm_kernel(ops: OpTable, M, N, K, BM, BN, BK, S, per_warp, a_miss_first_touch, b_miss_first_touch,
                 elem=FP16):
    """A GEMM kernel as replicated CTA templates.  CTAs are rastered
    row-major over (M/BM, N/BN).  Static L2 model: the first CTA (in index
    order) touching an A row-panel or a B column-panel misses, later ones
    hit; C stores always go to DRAM."""
    assert M % BM == 0 and N % BN == 0 and K % BK == 0
    T = K // BK
    roles_edges = gemm_template(T, S, per_warp)
    roles = roles_edges[0]
    gm, gn = M // BM, N // BN
    ldA, ldB = BM * BK * elem, BN * BK * elem
    opA = (ops.get(GLOAD, ldA, ALL4, MISS), ops.get(GLOAD, ldA, ALL4))
    opB = (ops.get(GLOAD, ldB, ALL4, MISS), ops.get(GLOAD, ldB, ALL4))
    if per_warp:
        mma = [ops.get(TENSOR, 2 * (BM // 2) * (BN // 2) * BK, 1 << w) for w in range(4)]
    else:
        mma = [ops.get(TENSOR, 2 * BM * BN * BK, ALL4)]
    st = ops.get(GSTORE, BM * BN * elem, ALL4, MISS)
    base = np.zeros(len(roles), dtype=np.uint16)
    posA, posB = [], []
    for i, r in enumerate(roles):
        if r[0] == "lA":
            posA.append(i)
            base[i] = opA[1]
        elif r[0] == "lB":
            posB.append(i)
            base[i] = opB[1]
        elif r[0] == "mma":
            base[i] = mma[r[2]] if per_warp else mma[0]
        else:
            base[i] = st
    opm = np.tile(base, (gm * gn, 1))
    mi = np.arange(gm * gn) // gn
    ni = np.arange(gm * gn) % gn
    if a_miss_first_touch:
        opm[np.ix_(ni == 0, posA)] = opA[0]
    if b_miss_first_touch:
        opm[np.ix_(mi == 0, posB)] = opB[0]
    k = _Kernel(4, S * (BM + BN) * BK * elem)
    k.add(roles_edges, opm)
    return k


def gemm(M=1024, N=1024, K=1024, BM=128, BN=128, BK=32, S=2, per_warp=False, tiles=False) -> TileGraph:
    """Tiled GEMM C = A B in fp16 (the 1024^3 workload: 128x128x32 tiles, 2 stages).
    tiles: also name the tile every load / store touches (A block (m, k),
    B block (n, k), C block (m, n)), for the LRU L2 model."""
    ops = OpTable()
    k = _gemm_kernel(ops, M, N, K, BM, BN, BK, S, per_warp, True, True)
    g = _assemble([k], ops, f"gemm_{M}x{N}x{K}_{BM}x{BN}x{BK}_s{S}",
                  dict(M=M, N=N, K=K, BM=BM, BN=BN, BK=BK, S=S, per_warp=per_warp))
    if tiles:
        g.node_tile = gemm_tile_ids(M, N, K, BM, BN, BK, S, per_warp)
    return g


def gemm_addressed(M=1024, N=1024, K=1024, BM=128, BN=128, BK=32, S=2, per_warp=False, pad=0,
                   b_layout="kn", elem=FP16) -> TileGraph:
    """gemm(...) with transaction-level memory: every load and store carries
    the byte address of its tile in its tensor, and its op the tile's rows
    and row stride (Sec. 4.1 tile descriptor: storage, shape, layout,
    coordinates).  A is M x K row-major, C is M x N row-major, B is K x N
    row-major ("kn") or N x K row-major ("nk", i.e. column-major K x N);
    each leading dimension is padded by `pad` elements.  Tensors are placed
    one after another from address 0, each starting on a 4 KiB boundary.
    A tile (m, k) of A is BM rows of BK elements at A + (m*BM*lda + k*BK)*elem
    with stride lda*elem; a B tile is BK rows of BN elements ("kn") or BN
    rows of BK ("nk"); a C tile BM rows of BN."""
    g = gemm(M, N, K, BM, BN, BK, S, per_warp)
    lda, ldc = K + pad, N + pad
    ldb = (N if b_layout == "kn" else K) + pad
    A0 = 0
    B0 = -(-(M * lda * elem) // 4096) * 4096
    C0 = B0 + -(-((K if b_layout == "kn" else N) * ldb * elem) // 4096) * 4096
    T = K // BK
    gm, gn = M // BM, N // BN
    roles = gemm_template(T, S, per_warp)[0]
    kind = np.zeros(len(roles), dtype=np.int64)  # 1 A, 2 B, 3 C
    kstep = np.zeros(len(roles), dtype=np.int64)
    for i, r in enumerate(roles):
        if r[0] == "lA":
            kind[i], kstep[i] = 1, r[1]
        elif r[0] == "lB":
            kind[i], kstep[i] = 2, r[1]
        elif r[0] == "st":
            kind[i] = 3
    c = np.arange(gm * gn, dtype=np.int64)[:, None]
    mi, ni = c // gn, c % gn
    a_addr = A0 + (mi * BM * lda + kstep * BK) * elem
    if b_layout == "kn":
        b_addr = B0 + (kstep * BK * ldb + ni * BN) * elem
        b_rows, b_pitch = BK, ldb * elem
    else:
        b_addr = B0 + (ni * BN * ldb + kstep * BK) * elem
        b_rows, b_pitch = BN, ldb * elem
    c_addr = C0 + (mi * BM * ldc + ni * BN) * elem
    addr = np.where(kind == 1, a_addr, np.where(kind == 2, b_addr, np.where(kind == 3, c_addr, -1)))
    addr = addr.ravel()
    node_kind = np.tile(kind, gm * gn)
    # ops: one per (op, tensor) so each carries its tensor's tile shape
    shape = {1: (BM, lda * elem), 2: (b_rows, b_pitch), 3: (BM, ldc * elem)}
    ops = OpTable()
    for p in range(g.n_ops):
        ops.get(int(g.op_cls[p]), int(g.op_work[p]), int(g.op_warps[p]), int(g.op_flags[p]))
    new_op = g.node_op.astype(np.int64).copy()
    for t in (1, 2, 3):
        sel = node_kind == t
        for p in np.unique(new_op[sel]).tolist():
            rows, pitch = shape[t]
            q = ops.get(int(g.op_cls[p]), int(g.op_work[p]), int(g.op_warps[p]), int(g.op_flags[p]), rows, pitch)
            new_op[sel & (g.node_op == p)] = q
    cls, flags, work, warps = ops.arrays()
    rows, pitch = ops.shapes()
    g.op_cls, g.op_flags, g.op_work, g.op_warps = cls, flags, work, warps
    g.op_rows, g.op_pitch = rows, pitch
    g.node_op = new_op.astype(np.uint16)
    g.node_addr = np.where(addr >= 0, addr, 0).astype(np.uint64)
    g.node_addr[addr < 0] = np.uint64(NO_ADDR)
    g.name = g.name + f"_addr_{b_layout}_pad{pad}"
    g.meta.update(pad=pad, b_layout=b_layout)
    return g


def gemm_tile_ids(M, N, K, BM, BN, BK, S, per_warp=False) -> np.ndarray:
    """Tile id of every node of gemm(...): A blocks first (row-panel major),
    then B blocks, then C blocks; NO_TILE for MMA nodes."""
    T = K // BK
    gm, gn = M // BM, N // BN
    roles = gemm_template(T, S, per_warp)[0]
    local = np.full(len(roles), -1, dtype=np.int64)
    kind = np.zeros(len(roles), dtype=np.int64)  # 1 A, 2 B, 3 C
    for i, r in enumerate(roles):
        if r[0] == "lA":
            kind[i], local[i] = 1, r[1]
        elif r[0] == "lB":
            kind[i], local[i] = 2, r[1]
        elif r[0] == "st":
            kind[i] = 3
    c = np.arange(gm * gn, dtype=np.int64)[:, None]
    mi, ni = c // gn, c % gn
    ids = np.where(kind == 1, mi * T + local,
          np.where(kind == 2, gm * T + ni * T + local,
          np.where(kind == 3, gm * T + gn * T + mi * gn + ni, NO_TILE)))
    return ids.astype(np.uint32).ravel()


def _attention_kernel(ops: OpTable, batch, heads, kv_heads, seqlen, d, q_tile, kv_tile, causal,
                      q_hit=False, stages=2):
    """Flash-attention forward, one CTA per (batch, head, query block),
    head-major.  K/V tiles of a KV head miss L2 in the first CTA that
    reads them, hit afterwards; Q is read once (miss unless produced by the
    previous kernel); O stores go to DRAM."""
    nq = seqlen // q_tile
    group = heads // kv_heads
    lq = ops.get(GLOAD, q_tile * d * FP16, PRODUCER, 0 if q_hit else MISS)
    lkv = (ops.get(GLOAD, kv_tile * d * FP16, PRODUCER, MISS), ops.get(GLOAD, kv_tile * d * FP16, PRODUCER))
    qk = ops.get(TENSOR, 2 * q_tile * kv_tile * d, ALL4)
    sm = ops.get(SFU, q_tile * kv_tile, ALL4)
    pv = ops.get(TENSOR, 2 * q_tile * kv_tile * d, ALL4)
    st = ops.get(GSTORE, q_tile * d * FP16, ALL4, MISS)
    k = _Kernel(5, q_tile * d * FP16 + stages * 2 * kv_tile * d * FP16)
    templates = {}
    # first reader of each (batch, kv head, kv tile): min over (head in group, q block) in CTA order
    for b in range(batch):
        for h in range(heads):
            for qb in range(nq):
                n_tiles = (qb + 1) * q_tile // kv_tile if causal else seqlen // kv_tile
                if n_tiles not in templates:
                    templates[n_tiles] = attention_template(n_tiles, stages)
                roles = templates[n_tiles][0]
                row = np.zeros(len(roles), dtype=np.uint16)
                for i, r in enumerate(roles):
                    if r[0] == "lQ":
                        row[i] = lq
                    elif r[0] in ("lK", "lV"):
                        j = r[1]
                        if causal:
                            first = (h % group == 0) and (qb == j * kv_tile // q_tile)
                        else:
                            first = (h % group == 0) and qb == 0
                        row[i] = lkv[0] if first else lkv[1]
                    elif r[0] in ("qk", "pv"):
                        row[i] = qk if r[0] == "qk" else pv
                    elif r[0] == "sm":
                        row[i] = sm
                    else:
                        row[i] = st
                k.add(templates[n_tiles], row[None, :])
    return _coalesce(k)


def _coalesce(k: _Kernel) -> _Kernel:
    """Merge consecutive groups that share a template (same CSR)."""
    out = _Kernel(k.warps, k.smem)
    for g in k.groups:
        if out.groups:
            p = out.groups[-1]
            if p[2] == g[2] and p[0].shape == g[0].shape and np.array_equal(p[0], g[0]) and np.array_equal(p[1], g[1]):
                out.groups[-1] = (p[0], p[1], p[2], np.concatenate([p[3], g[3]]))
                continue
        out.groups.append(g)
    return out


def flash_attention(batch=8, heads=32, seqlen=4096, d=128, q_tile=128, kv_tile=64, causal=False) -> TileGraph:
    """FlashAttention-style forward, warp-specialised, non-causal (B8 H32 S4096 d128 by default)."""
    ops = OpTable()
    if not causal:
        # all CTAs share one template: build the op matrix vectorised
        nq = seqlen // q_tile
        n_tiles = seqlen // kv_tile
        roles_edges = attention_template(n_tiles)
        roles = roles_edges[0]
        lq = ops.get(GLOAD, q_tile * d * FP16, PRODUCER, MISS)
        lkv = (ops.get(GLOAD, kv_tile * d * FP16, PRODUCER, MISS), ops.get(GLOAD, kv_tile * d * FP16, PRODUCER))
        qk = ops.get(TENSOR, 2 * q_tile * kv_tile * d, ALL4)
        sm = ops.get(SFU, q_tile * kv_tile, ALL4)
        st = ops.get(GSTORE, q_tile * d * FP16, ALL4, MISS)
        base = np.zeros(len(roles), dtype=np.uint16)
        kvpos = []
        for i, r in enumerate(roles):
            base[i] = {"lQ": lq, "qk": qk, "pv": qk, "sm": sm, "st": st}.get(r[0], lkv[1])
            if r[0] in ("lK", "lV"):
                kvpos.append(i)
        C = batch * heads * nq
        opm = np.tile(base, (C, 1))
        first = (np.arange(C) % nq) == 0  # non-causal MHA: query block 0 reads every K/V tile first
        opm[np.ix_(first, kvpos)] = lkv[0]
        k = _Kernel(5, q_tile * d * FP16 + 2 * 2 * kv_tile * d * FP16)
        k.add(roles_edges, opm)
    else:
        k = _attention_kernel(ops, batch, heads, heads, seqlen, d, q_tile, kv_tile, True)
    return _assemble([k], ops, f"fa_fwd_b{batch}_h{heads}_s{seqlen}_d{d}" + ("_causal" if causal else ""),
                     dict(batch=batch, heads=heads, seqlen=seqlen, d=d, q_tile=q_tile, kv_tile=kv_tile,
                          causal=causal))


def splitkv_decode(batch=64, q_heads=32, kv_heads=8, d=128, kv_min=512, kv_max=32768, split=256,
                   kv_tile=64, seed=1004) -> TileGraph:
    """Split-KV decode attention (one query token per sequence; 64 sequences by default).
    One CTA per (sequence, KV head, split of `split` tokens) runs the
    warp-specialised attention pipeline over <= split/kv_tile KV tiles and
    stores a partial (fp32 O + log-sum-exp); one reduction CTA per
    (sequence, KV head) loads every partial (cross-CTA DATA edges), combines
    them on the CUDA cores and stores the output.  KV lengths are
    log-uniform per sequence, rounded up to whole KV tiles."""
    rng = SplitMix64(seed)
    lens = [-(-rng.loguniform_int(kv_min, kv_max) // kv_tile) * kv_tile for _ in range(batch)]
    group = q_heads // kv_heads
    ops = OpTable()
    lq = ops.get(GLOAD, group * d * FP16, PRODUCER, MISS)
    lkv = ops.get(GLOAD, kv_tile * d * FP16, PRODUCER, MISS)
    qk = ops.get(TENSOR, 2 * group * kv_tile * d, ALL4)
    sm = ops.get(SFU, group * kv_tile, ALL4)
    part_bytes = group * d * 4 + group * 4
    stp = ops.get(GSTORE, part_bytes, ALL4, MISS)
    ldp = ops.get(GLOAD, part_bytes, ALL4)
    st = ops.get(GSTORE, group * d * FP16, ALL4, MISS)
    b = GraphBuilder()
    b.ops = ops
    b.kernel(5, group * d * FP16 + 2 * 2 * kv_tile * d * FP16)
    stores = {}
    tiles_per_split = split // kv_tile
    for s in range(batch):
        n_tiles_total = lens[s] // kv_tile
        n_splits = -(-n_tiles_total // tiles_per_split)
        for h in range(kv_heads):
            for p in range(n_splits):
                nt = min(tiles_per_split, n_tiles_total - p * tiles_per_split)
                roles, edges = attention_template(nt)
                b.cta()
                ids = []
                for r in roles:
                    if r[0] == "lQ":
                        ids.append(_add(b, lq))
                    elif r[0] in ("lK", "lV"):
                        ids.append(_add(b, lkv))
                    elif r[0] in ("qk", "pv"):
                        ids.append(_add(b, qk))
                    elif r[0] == "sm":
                        ids.append(_add(b, sm))
                    else:
                        ids.append(_add(b, stp))
                for u, v, kd in edges:
                    b.edge(ids[u], ids[v], kd)
                stores[(s, h, p)] = ids[-1]
    for s in range(batch):
        n_splits = -(-(lens[s] // kv_tile) // tiles_per_split)
        comb = ops.get(ALU, n_splits * group * (d + 2) * 2, ALL4)
        for h in range(kv_heads):
            b.cta()
            loads = [_add(b, ldp) for _ in range(n_splits)]
            c = _add(b, comb)
            o = _add(b, st)
            for p, ld in enumerate(loads):
                b.edge(stores[(s, h, p)], ld, DATA)
                b.edge(ld, c, DATA)
                if p:
                    b.edge(loads[p - 1], ld, ORDER)
            b.edge(c, o, DATA)
    g = b.build(f"splitkv_decode_b{batch}")
    g.meta = dict(batch=batch, kv_lens=lens, split=split, q_heads=q_heads, kv_heads=kv_heads)
    return g


def _add(b: GraphBuilder, op: int) -> int:
    b.node_op.append(op)
    return len(b.node_op) - 1


def _elementwise_kernel(ops: OpTable, rows, row_tile, stages, in_hit):
    """One CTA per row_tile rows: load -> compute stages -> store (DATA
    chain).  stages: list of (class, work per CTA); loads/stores in bytes."""
    C = rows // row_tile
    roles_edges = chain_template(len(stages))
    row = []
    for i, (cls, work) in enumerate(stages):
        if cls == GLOAD:
            row.append(ops.get(GLOAD, work, ALL4, 0 if in_hit else MISS))
        elif cls == GSTORE:
            row.append(ops.get(GSTORE, work, ALL4, MISS))
        else:
            row.append(ops.get(cls, work, ALL4))
    k = _Kernel(4, 1024)
    k.add(roles_edges, np.tile(np.array(row, dtype=np.uint16), (C, 1)))
    return k


def decoder_layer(tokens=2048, hidden=4096, heads=32, kv_heads=8, ffn=14336, d=128, tile=64, bk=32,
                  stages=3, row_tile=16) -> TileGraph:
    """One Llama-like decoder layer in prefill (2048 tokens by default), nine kernels with
    implicit kernel boundaries: RMSNorm, QKV GEMM, RoPE, causal attention,
    O-projection, RMSNorm, fused gate+up GEMM, SwiGLU, down GEMM.  GEMMs use
    64x64x32 CTA tiles with one MMA node per warp quadrant (6 nodes per
    k-step).  Activations written by the previous kernel hit L2; weights miss
    on first touch."""
    ops = OpTable()
    qkv = hidden + 2 * kv_heads * d
    ks = []
    ks.append(_elementwise_kernel(ops, tokens, row_tile, [(GLOAD, row_tile * hidden * FP16),
                                                         (ALU, row_tile * hidden * 2), (ALU, row_tile * hidden * 3),
                                                         (GSTORE, row_tile * hidden * FP16)], in_hit=False))
    ks.append(_gemm_kernel(ops, tokens, qkv, hidden, tile, tile, bk, stages, True, False, True))
    rope_cols = hidden + kv_heads * d
    ks.append(_elementwise_kernel(ops, tokens, row_tile, [(GLOAD, row_tile * rope_cols * FP16),
                                                         (ALU, row_tile * rope_cols * 3),
                                                         (GSTORE, row_tile * rope_cols * FP16)], in_hit=True))
    ks.append(_attention_kernel(ops, 1, heads, kv_heads, tokens, d, 128, 64, True, q_hit=True))
    ks.append(_gemm_kernel(ops, tokens, hidden, hidden, tile, tile, bk, stages, True, False, True))
    ks.append(_elementwise_kernel(ops, tokens, row_tile, [(GLOAD, row_tile * hidden * FP16),
                                                         (ALU, row_tile * hidden * 2), (ALU, row_tile * hidden * 3),
                                                         (GSTORE, row_tile * hidden * FP16)], in_hit=True))
    ks.append(_gemm_kernel(ops, tokens, 2 * ffn, hidden, tile, tile, bk, stages, True, False, True))
    ks.append(_elementwise_kernel(ops, tokens, row_tile, [(GLOAD, row_tile * 2 * ffn * FP16),
                                                         (SFU, row_tile * ffn), (ALU, row_tile * ffn),
                                                         (GSTORE, row_tile * ffn * FP16)], in_hit=True))
    ks.append(_gemm_kernel(ops, tokens, hidden, ffn, tile, tile, bk, stages, True, False, True))
    return _assemble(ks, ops, f"decoder_layer_t{tokens}",
                     dict(tokens=tokens, hidden=hidden, heads=heads, kv_heads=kv_heads, ffn=ffn))


# --------------------------------------------------------------------------
# GEMM design sweep
# --------------------------------------------------------------------------

SWEEP_MNK = (1024, 2048, 4096, 8192)
SWEEP_BMN = (64, 128, 256)
SWEEP_BK = (32, 64)
SWEEP_STAGES = (2, 3, 4)


def sweep_params(seed=1002, n_graphs=64):
    """(M, N, K, BM, BN, BK, stages) tuples of the GEMM design sweep."""
    rng = SplitMix64(seed)
    out = []
    for _ in range(n_graphs):
        out.append((rng.choice(SWEEP_MNK), rng.choice(SWEEP_MNK), rng.choice(SWEEP_MNK), rng.choice(SWEEP_BMN),
                    rng.choice(SWEEP_BMN), rng.choice(SWEEP_BK), rng.choice(SWEEP_STAGES)))
    return out


def sweep_graph(params) -> TileGraph:
    M, N, K, BM, BN, BK, S = params
    return gemm(M, N, K, BM, BN, BK, S)


def sweep_nodes(params) -> int:
    M, N, K, BM, BN, BK, S = params
    return (M // BM) * (N // BN) * (3 * (K // BK) + 1)


# --------------------------------------------------------------------------
# The five workload configurations
# --------------------------------------------------------------------------

# The benchmark workloads by name: batch size, and the number n behind their
# seeds (graph seed 1000 + n, hardware seed 2000 + n).
WORKLOADS = {
    "gemm_1024_a100": dict(n=1, B=16),
    "gemm_design_sweep": dict(n=2, B=4096, graphs=64),
    "flash_attention_b8_h32_s4096": dict(n=3, B=256),
    "splitkv_decode_b64": dict(n=4, B=1024),
    "decoder_layer_prefill_2048": dict(n=5, B=64),
}


def workload_graph(name: str, index: int = 0) -> TileGraph:
    """Graph of a named workload (`index`: which GEMM of the design sweep)."""
    if name == "gemm_1024_a100":
        return gemm(1024, 1024, 1024, 128, 128, 32, 2)
    if name == "gemm_design_sweep":
        return sweep_graph(sweep_params()[index])
    if name == "flash_attention_b8_h32_s4096":
        return flash_attention()
    if name == "splitkv_decode_b64":
        return splitkv_decode(seed=1000 + WORKLOADS[name]["n"])
    if name == "decoder_layer_prefill_2048":
        return decoder_layer()
    raise KeyError(name)


def workload_hw(name: str, B: int | None = None, index: int = 0) -> np.ndarray:
    """Hardware records of a named workload: A100-based for the 1024^3 GEMM,
    H100-based sweeps otherwise (each design-sweep GEMM its own stream)."""
    B = WORKLOADS[name]["B"] if B is None else B
    seed = 2000 + WORKLOADS[name]["n"]
    if name == "gemm_1024_a100":
        return hwmod.sample_a100_sweep(seed, B)
    if name == "gemm_design_sweep":
        return hwmod.sample_h100_sweep(seed, B, stream=index + 1)
    return hwmod.sample_h100_sweep(seed, B)


# --------------------------------------------------------------------------
# Random DAGs for brute-force and cross-check tests
# --------------------------------------------------------------------------

def random_graph(rng: SplitMix64, n_nodes_max=12, n_kernels_max=2, ctas_max=3, edge_p=(1, 3),
                 cross_cta=True, classes=(TENSOR, ALU, SFU, 3, GLOAD, GSTORE, SYNC)) -> TileGraph:
    """A random valid tile graph: random kernels/CTAs, node classes, works,
    warp masks, and DAG edges of every kind (random topological order inside
    each CTA; cross-CTA edges only forward)."""
    b = GraphBuilder()
    nk = rng.randint(1, n_kernels_max)
    total = rng.randint(1, n_nodes_max)
    # distribute nodes over CTAs over kernels
    ctas = []
    for k in range(nk):
        warps = rng.randint(1, 8)
        smem = rng.randint(0, 3) * 8 * 1024
        for _ in range(rng.randint(1, ctas_max)):
            ctas.append((k, warps, smem))
    sizes = [1] * len(ctas)
    for _ in range(max(0, total - len(ctas))):
        sizes[rng.randint(0, len(ctas) - 1)] += 1
    cur_k = -1
    order_in_cta = []
    for (k, warps, smem), sz in zip(ctas, sizes):
        if k != cur_k:
            b.kernel(warps, smem)
            cur_k = k
        b.cta()
        ids = []
        for _ in range(sz):
            cls = rng.choice(list(classes))
            wm = 0
            while wm == 0:
                wm = rng.randint(0, (1 << warps) - 1)
            if cls in (TENSOR, ALU, SFU):
                work = rng.randint(0, 5000)
            elif cls == SYNC:
                work = 0
            else:
                work = rng.randint(0, 4096)
            flags = MISS if cls in (GLOAD, GSTORE) and rng.randint(0, 1) else 0
            ids.append(b.node(cls, work, wm, flags))
        # random topological order of this CTA's nodes
        perm = list(ids)
        for i in range(len(perm) - 1, 0, -1):
            j = rng.randint(0, i)
            perm[i], perm[j] = perm[j], perm[i]
        order_in_cta.append(perm)
    n = len(b.node_op)
    lo, hi = edge_p
    for ci, perm in enumerate(order_in_cta):
        for a in range(len(perm)):
            for bb in range(a + 1, len(perm)):
                if rng.randint(0, hi - 1) < lo:
                    b.edge(perm[a], perm[bb], rng.randint(0, 2))
        if cross_cta:
            for cj in range(ci + 1, len(order_in_cta)):
                for u in perm:
                    for v in order_in_cta[cj]:
                        if rng.randint(0, 6) == 0:
                            b.edge(u, v, rng.randint(0, 2))
    g = b.build("random")
    return g


__all__ = ["gemm", "flash_attention", "splitkv_decode", "decoder_layer", "sweep_params", "sweep_graph",
           "sweep_nodes", "workload_graph", "workload_hw", "random_graph", "WORKLOADS", "gemm_template",
           "attention_template", "empty_graph"]

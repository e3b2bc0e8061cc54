"""Tile-graph container and CSR construction (GTSim Sec. 4.1).

A tile graph is a DAG G = (V, E) of warp-level tile operations.  Each node
carries an execution group (a warp mask within its CTA), an operation
descriptor (resource class + work) and, reduced to what the timing model
reads, a tile descriptor (bytes / FLOPs and whether the access misses L2).
Edges are DATA (producer -> consumer), ORDER (program order of one warp) or
SYNC (cross-warp signal/wait, barrier, buffer reuse).  A kernel's CTAs may
form thread-block clusters (consecutive CTAs, dispatched together onto one
NoC domain); a REMOTE node moves bytes to another CTA of its cluster, whose
rank sits in the op flags (Sec. 5.2 DSMEM / SM-cluster NoC).  Global loads
and stores may name the tile they touch (``node_tile``), for the LRU L2 of
Sec. 5.2; the tile's 128-B lines are the access's cache lines.

Descriptors are dictionary-encoded: ``ops`` lists the distinct
(class, flags, work, warp_mask) tuples and every node stores an op index.
Nodes are numbered CTA-major and CTAs kernel-major, which is the layout the
C ABI expects (include/gts.h, gts_graph_host).
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

TENSOR, ALU, SFU, SMEM, GLOAD, GSTORE, SYNC, REMOTE = range(8)
CLASS_NAMES = ("TENSOR", "ALU", "SFU", "SMEM", "GLOAD", "GSTORE", "SYNC", "REMOTE")
COMPUTE_CLASSES = (TENSOR, ALU, SFU)
MISS = 1
RANK_SHIFT = 4      # REMOTE ops: target rank = flags >> RANK_SHIFT
MAX_CLUSTER = 16
NO_TILE = 0xFFFFFFFF
NO_ADDR = 0xFFFFFFFFFFFFFFFF
LINE_BYTES = 128
MAX_NODE_TXN = 1 << 21  # transactions one addressed node may have (bound: rows * (row bytes / 128 + 2))


def remote_flags(rank: int) -> int:
    return int(rank) << RANK_SHIFT

DATA, ORDER, SYNC_EDGE = 0, 1, 2
KIND_SHIFT = 30
TARGET_MASK = (1 << 30) - 1

# When one (u, v) pair is given with several kinds the strongest survives:
# DATA and SYNC both release at u's finish, which also satisfies ORDER.
_KIND_RANK = {DATA: 2, SYNC_EDGE: 1, ORDER: 0}


@dataclass
class TileGraph:
    op_cls: np.ndarray            # u8  [P]
    op_flags: np.ndarray          # u8  [P]
    op_work: np.ndarray           # u32 [P]
    op_warps: np.ndarray          # u32 [P]
    node_op: np.ndarray           # u16 [N]
    succ_ptr: np.ndarray          # u32 [N+1]
    succ: np.ndarray              # u32 [E]  target | kind << 30
    cta_node_begin: np.ndarray    # u32 [C+1]
    kernel_cta_begin: np.ndarray  # u32 [K+1]
    kernel_warps: np.ndarray      # u16 [K]
    kernel_smem: np.ndarray       # u32 [K]
    name: str = "graph"
    meta: dict = field(default_factory=dict)
    kernel_cluster: np.ndarray = None  # u8 [K] CTAs per cluster (None: all 1)
    node_tile: np.ndarray = None       # u32 [N] tile of a load / store, NO_TILE otherwise (None: no tiles)
    # transaction-level memory: byte address of a load / store's tile (NO_ADDR
    # otherwise; None: no addresses), and per op the tile's rows and row
    # stride in bytes (None: one row, stride = row bytes)
    node_addr: np.ndarray = None       # u64 [N]
    op_rows: np.ndarray = None         # u32 [P]
    op_pitch: np.ndarray = None        # u32 [P]

    def __post_init__(self):
        if self.kernel_cluster is None:
            self.kernel_cluster = np.ones(int(self.kernel_warps.shape[0]), dtype=np.uint8)
        self.kernel_cluster = np.asarray(self.kernel_cluster, dtype=np.uint8)
        if self.node_tile is not None:
            self.node_tile = np.asarray(self.node_tile, dtype=np.uint32)
        if self.node_addr is not None:
            self.node_addr = np.asarray(self.node_addr, dtype=np.uint64)
        if self.op_rows is not None:
            self.op_rows = np.asarray(self.op_rows, dtype=np.uint32)
        if self.op_pitch is not None:
            self.op_pitch = np.asarray(self.op_pitch, dtype=np.uint32)

    @property
    def n_nodes(self) -> int:
        return int(self.node_op.shape[0])

    @property
    def n_edges(self) -> int:
        return int(self.succ.shape[0])

    @property
    def n_ctas(self) -> int:
        return int(self.cta_node_begin.shape[0]) - 1

    @property
    def n_kernels(self) -> int:
        return int(self.kernel_warps.shape[0])

    @property
    def n_ops(self) -> int:
        return int(self.op_cls.shape[0])

    def targets(self) -> np.ndarray:
        return (self.succ & TARGET_MASK).astype(np.int64)

    def kinds(self) -> np.ndarray:
        return (self.succ >> KIND_SHIFT).astype(np.int64)

    def sources(self) -> np.ndarray:
        return np.repeat(np.arange(self.n_nodes, dtype=np.int64), np.diff(self.succ_ptr.astype(np.int64)))

    def node_cta(self) -> np.ndarray:
        return np.repeat(np.arange(self.n_ctas, dtype=np.int64), np.diff(self.cta_node_begin.astype(np.int64)))

    def cta_kernel(self) -> np.ndarray:
        return np.repeat(np.arange(self.n_kernels, dtype=np.int64), np.diff(self.kernel_cta_begin.astype(np.int64)))

    def indegree(self) -> np.ndarray:
        return np.bincount(self.targets(), minlength=self.n_nodes).astype(np.int64)

    def digest(self) -> str:
        """SHA-256 over every array: pins seed reproducibility of generators."""
        h = hashlib.sha256()
        for a in (self.op_cls, self.op_flags, self.op_work, self.op_warps, self.node_op, self.succ_ptr,
                  self.succ, self.cta_node_begin, self.kernel_cta_begin, self.kernel_warps, self.kernel_smem):
            h.update(np.ascontiguousarray(a).tobytes())
        if np.any(self.kernel_cluster != 1):
            h.update(np.ascontiguousarray(self.kernel_cluster).tobytes())
        if self.node_tile is not None:
            h.update(np.ascontiguousarray(self.node_tile).tobytes())
        return h.hexdigest()

    def arrays(self) -> dict:
        return dict(op_cls=self.op_cls, op_flags=self.op_flags, op_work=self.op_work, op_warps=self.op_warps,
                    node_op=self.node_op, succ_ptr=self.succ_ptr, succ=self.succ,
                    cta_node_begin=self.cta_node_begin, kernel_cta_begin=self.kernel_cta_begin,
                    kernel_warps=self.kernel_warps, kernel_smem=self.kernel_smem, kernel_cluster=self.kernel_cluster,
                    node_tile=self.node_tile, node_addr=self.node_addr, op_rows=self.op_rows, op_pitch=self.op_pitch)


class OpTable:
    """Dictionary of distinct (class, flags, work, warp_mask) tuples."""

    def __init__(self):
        self.index: dict = {}
        self.rows: list = []

    def get(self, cls: int, work: int, warps: int, flags: int = 0, rows: int = 1, pitch: int = 0) -> int:
        """Op id of the tuple; rows / pitch: the tile shape of an addressed
        load / store (pitch 0: rows packed, stride = row bytes)."""
        key = (int(cls), int(flags), int(work), int(warps), int(rows), int(pitch))
        if key not in self.index:
            self.index[key] = len(self.rows)
            self.rows.append(key)
        return self.index[key]

    def arrays(self):
        rows = self.rows or []
        cls = np.array([r[0] for r in rows], dtype=np.uint8)
        flags = np.array([r[1] for r in rows], dtype=np.uint8)
        work = np.array([r[2] for r in rows], dtype=np.uint32)
        warps = np.array([r[3] for r in rows], dtype=np.uint32)
        return cls, flags, work, warps

    def shapes(self):
        """(op_rows, op_pitch) arrays, or (None, None) when every op has the
        default shape (one row)."""
        if all(r[4] == 1 and r[5] == 0 for r in self.rows):
            return None, None
        nrows = np.array([r[4] for r in self.rows], dtype=np.uint32)
        pitch = np.array([r[5] if r[5] else r[2] // max(r[4], 1) for r in self.rows], dtype=np.uint32)
        return nrows, pitch


def csr_from_edges(n_nodes: int, src: np.ndarray, dst: np.ndarray, kind: np.ndarray):
    """Sorted, de-duplicated CSR.  Duplicate (u, v) pairs keep the strongest
    kind (DATA > SYNC > ORDER, all three release no earlier than ORDER)."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    kind = np.asarray(kind, dtype=np.int64)
    if src.size:
        rank = np.array([_KIND_RANK[k] for k in range(3)], dtype=np.int64)[kind]
        # sort by (src, dst, -rank) and keep the first of each (src, dst)
        order = np.lexsort((-rank, dst, src))
        src, dst, kind = src[order], dst[order], kind[order]
        keep = np.ones(src.size, dtype=bool)
        keep[1:] = (src[1:] != src[:-1]) | (dst[1:] != dst[:-1])
        src, dst, kind = src[keep], dst[keep], kind[keep]
    counts = np.bincount(src, minlength=n_nodes) if src.size else np.zeros(n_nodes, dtype=np.int64)
    succ_ptr = np.zeros(n_nodes + 1, dtype=np.uint32)
    np.cumsum(counts, out=succ_ptr[1:])
    succ = (dst.astype(np.uint32) | (kind.astype(np.uint32) << np.uint32(KIND_SHIFT))).astype(np.uint32)
    return succ_ptr, succ


class GraphBuilder:
    """Incremental builder for small hand-written graphs (tests, examples).

    Nodes must be added CTA by CTA and CTAs kernel by kernel.  Edges of the
    kinds in `drop` are ignored as they are added (the Table 4 ablation:
    a pair that also carries a kept kind keeps that edge)."""

    def __init__(self, drop=()):
        self.drop = frozenset(int(k) for k in drop)
        self.ops = OpTable()
        self.node_op: list = []
        self.node_addr: list = []
        self.cta_begin: list = [0]
        self.kernel_begin: list = [0]
        self.kernel_warps: list = []
        self.kernel_smem: list = []
        self.kernel_cluster: list = []
        self.src: list = []
        self.dst: list = []
        self.kind: list = []
        self._open_cta = False

    def kernel(self, warps: int, smem: int = 0, cluster: int = 1):
        self._close_cta()
        if self.kernel_warps:
            self.kernel_begin.append(len(self.cta_begin) - 1)
        self.kernel_warps.append(int(warps))
        self.kernel_smem.append(int(smem))
        self.kernel_cluster.append(int(cluster))
        return len(self.kernel_warps) - 1

    def cta(self):
        self._close_cta()
        self._open_cta = True
        return len(self.cta_begin) - 1

    def _close_cta(self):
        if self._open_cta:
            self.cta_begin.append(len(self.node_op))
            self._open_cta = False

    def node(self, cls: int, work: int = 0, warps: int = 1, flags: int = 0, addr: int | None = None,
             rows: int = 1, pitch: int = 0) -> int:
        """A node; addr (loads / stores): the byte address of its tile of
        `rows` rows of work / rows bytes, `pitch` bytes apart (0: packed)."""
        assert self._open_cta, "open a CTA first"
        self.node_op.append(self.ops.get(cls, work, warps, flags, rows, pitch))
        self.node_addr.append(NO_ADDR if addr is None else int(addr))
        return len(self.node_op) - 1

    def edge(self, u: int, v: int, kind: int = DATA):
        if int(kind) in self.drop:
            return
        self.src.append(int(u))
        self.dst.append(int(v))
        self.kind.append(int(kind))

    def build(self, name: str = "graph") -> TileGraph:
        self._close_cta()
        n_ctas = len(self.cta_begin) - 1
        kb = list(self.kernel_begin) + [n_ctas] if self.kernel_warps else [0]
        n = len(self.node_op)
        succ_ptr, succ = csr_from_edges(n, np.array(self.src, dtype=np.int64), np.array(self.dst, dtype=np.int64),
                                        np.array(self.kind, dtype=np.int64))
        cls, flags, work, warps = self.ops.arrays()
        return TileGraph(op_cls=cls, op_flags=flags, op_work=work, op_warps=warps,
                         node_op=np.array(self.node_op, dtype=np.uint16), succ_ptr=succ_ptr, succ=succ,
                         cta_node_begin=np.array(self.cta_begin, dtype=np.uint32),
                         kernel_cta_begin=np.array(kb, dtype=np.uint32),
                         kernel_warps=np.array(self.kernel_warps, dtype=np.uint16),
                         kernel_smem=np.array(self.kernel_smem, dtype=np.uint32), name=name,
                         kernel_cluster=np.array(self.kernel_cluster, dtype=np.uint8),
                         node_addr=(np.array(self.node_addr, dtype=np.uint64)
                                    if any(a != NO_ADDR for a in self.node_addr) else None),
                         op_rows=self.ops.shapes()[0], op_pitch=self.ops.shapes()[1])


def empty_graph() -> TileGraph:
    z32 = np.zeros(0, dtype=np.uint32)
    return TileGraph(op_cls=np.zeros(0, np.uint8), op_flags=np.zeros(0, np.uint8), op_work=z32, op_warps=z32,
                     node_op=np.zeros(0, np.uint16), succ_ptr=np.zeros(1, np.uint32), succ=z32,
                     cta_node_begin=np.zeros(1, np.uint32), kernel_cta_begin=np.zeros(1, np.uint32),
                     kernel_warps=np.zeros(0, np.uint16), kernel_smem=z32, name="empty")


class ValidationError(ValueError):
    pass


def validate(g: TileGraph) -> None:
    """Python statement of the graph validity rules of the C ABI (used to
    check generators without a GPU; the library re-checks on upload)."""
    N, C, K, P = g.n_nodes, g.n_ctas, g.n_kernels, g.n_ops
    if N == 0:
        if C or K:
            raise ValidationError("empty graph with CTAs or kernels")
        return
    cb = g.cta_node_begin.astype(np.int64)
    kb = g.kernel_cta_begin.astype(np.int64)
    if cb[0] != 0 or cb[-1] != N or np.any(np.diff(cb) <= 0):
        raise ValidationError("cta_node_begin must start at 0, end at N, every CTA non-empty")
    if kb[0] != 0 or kb[-1] != C or np.any(np.diff(kb) <= 0):
        raise ValidationError("kernel_cta_begin must start at 0, end at C, every kernel non-empty")
    if np.any(g.kernel_warps < 1) or np.any(g.kernel_warps > 32):
        raise ValidationError("kernel warps out of range")
    if np.any(g.node_op >= P):
        raise ValidationError("node op out of range")
    if np.any(g.op_cls > REMOTE):
        raise ValidationError("op class out of range")
    cl = g.kernel_cluster.astype(np.int64)
    if cl.shape[0] != K or np.any(cl < 1) or np.any(cl > MAX_CLUSTER) or np.any(np.diff(kb) % cl != 0):
        raise ValidationError("cluster sizes must be 1..16 and divide each kernel's CTA count")
    remote = g.op_cls == REMOTE
    if np.any(remote & ((g.op_flags & ((1 << RANK_SHIFT) - 1)) != 0)):
        raise ValidationError("REMOTE op with flags other than the rank")
    compute = np.isin(g.op_cls, COMPUTE_CLASSES)
    if np.any(compute & (g.op_warps == 0)):
        raise ValidationError("compute op with empty warp mask")
    node_cta = g.node_cta()
    node_kernel = g.cta_kernel()[node_cta]
    if g.node_tile is not None:
        tiles = g.node_tile.astype(np.int64)
        mem_node = np.isin(g.op_cls, (GLOAD, GSTORE))[g.node_op.astype(np.int64)]
        if tiles.shape[0] != N or np.any(~mem_node & (tiles != NO_TILE)):
            raise ValidationError("only loads and stores carry tile ids")
        has = tiles != NO_TILE
        lines = -(-g.op_work.astype(np.int64)[g.node_op.astype(np.int64)] // LINE_BYTES)
        if has.any():
            t, l = tiles[has], lines[has]
            first = {}
            for a, b in zip(t.tolist(), l.tolist()):
                if first.setdefault(a, b) != b:
                    raise ValidationError("a tile is accessed with different sizes")
    P = int(g.op_cls.shape[0])
    if g.op_rows is not None and (g.op_rows.shape[0] != P or np.any(g.op_rows == 0)):
        raise ValidationError("op rows must be given for every op and be at least 1")
    if g.op_pitch is not None and g.op_pitch.shape[0] != P:
        raise ValidationError("op pitch must be given for every op")
    if g.node_addr is not None:
        addr = g.node_addr.astype(np.uint64)
        ops_n = g.node_op.astype(np.int64)
        mem_node = np.isin(g.op_cls, (GLOAD, GSTORE))[ops_n]
        has = addr != np.uint64(NO_ADDR)
        if addr.shape[0] != N or np.any(~mem_node & has):
            raise ValidationError("only loads and stores carry tile addresses")
        if has.any() and g.node_tile is not None and np.any(g.node_tile != NO_TILE):
            raise ValidationError("a graph names its tiles by id or by address, not both")
        rows = (g.op_rows.astype(np.int64) if g.op_rows is not None else np.ones(P, np.int64))
        work = g.op_work.astype(np.int64)
        used = np.zeros(P, dtype=bool)
        used[ops_n[has]] = True
        for p in np.flatnonzero(used).tolist():
            R = int(rows[p])
            if work[p] == 0 or work[p] % R:
                raise ValidationError("an addressed tile's bytes must be a positive multiple of its rows")
            W = int(work[p]) // R
            pitch = int(g.op_pitch[p]) if g.op_pitch is not None else W
            if pitch < W:
                raise ValidationError("an addressed tile's row stride is below its row bytes")
            if R * (W // LINE_BYTES + 2) > MAX_NODE_TXN:
                raise ValidationError("an addressed tile has too many transactions")
        if has.any():
            pv = ops_n[has]
            R = rows[pv]
            W = work[pv] // R
            pitch = (g.op_pitch.astype(np.int64)[pv] if g.op_pitch is not None else W)
            span = (R - 1) * pitch + W  # bytes from the tile's first to its last byte + 1
            if np.any(addr[has] > np.uint64(NO_ADDR - 1) - span.astype(np.uint64)):
                raise ValidationError("an addressed tile wraps the address space")
    nrem = remote[g.node_op.astype(np.int64)]
    rank = (g.op_flags.astype(np.int64) >> RANK_SHIFT)[g.node_op.astype(np.int64)]
    if np.any(nrem & (rank >= cl[node_kernel])):
        raise ValidationError("REMOTE target rank outside the cluster")
    warps_lim = g.kernel_warps.astype(np.int64)[node_kernel]
    mask = g.op_warps.astype(np.int64)[g.node_op.astype(np.int64)]
    ncomp = compute[g.node_op.astype(np.int64)]
    if np.any(ncomp & ((mask >> warps_lim) != 0)):
        raise ValidationError("compute node uses a warp outside its CTA")
    src, dst, kind = g.sources(), g.targets(), g.kinds()
    if np.any(dst >= N) or np.any(kind > 2):
        raise ValidationError("edge target or kind out of range")
    if np.any(src == dst):
        raise ValidationError("self loop")
    # a cluster's CTAs are dispatched together: edges between them may go
    # either way
    ck = g.cta_kernel()
    cluster_id = kb[ck] + (np.arange(C) - kb[ck]) // cl[ck] * cl[ck]  # first CTA of the cluster
    back = node_cta[src] > node_cta[dst]
    if np.any(back & (cluster_id[node_cta[src]] != cluster_id[node_cta[dst]])):
        raise ValidationError("edge from a later CTA to an earlier one outside a cluster")
    if src.size:
        key = src * N + dst
        if np.unique(key).size != key.size:
            raise ValidationError("duplicate edge")
    indeg = np.bincount(dst, minlength=N)
    if np.any(indeg > 65535):
        raise ValidationError("in-degree above 65535")
    # Kahn's algorithm, vectorised by frontier
    deg = indeg.copy()
    frontier = np.flatnonzero(deg == 0)
    seen = 0
    ptr = g.succ_ptr.astype(np.int64)
    while frontier.size:
        seen += frontier.size
        starts, ends = ptr[frontier], ptr[frontier + 1]
        lens = ends - starts
        if lens.sum() == 0:
            break
        idx = np.repeat(starts - np.cumsum(lens) + lens, lens) + np.arange(lens.sum())
        tg = dst[idx]
        np.subtract.at(deg, tg, 1)
        cand = np.unique(tg)
        frontier = cand[deg[cand] == 0]
    if seen != N:
        raise ValidationError("graph has a cycle")

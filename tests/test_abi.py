"""The C ABI without a GPU: the library loads, exports every entry point the
header declares, and its host-side validation returns the documented codes."""
import os
import re

import numpy as np
import pytest

from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import workloads as W
from paper_2607_11262_amd.gen.graph import (ALU, DATA, GLOAD, ORDER, REMOTE, TENSOR, GraphBuilder, TileGraph,
                                             ValidationError, empty_graph, remote_flags, validate)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    txt = open(os.path.join(ROOT, "include", "gts.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*|int)\s*(gts_\w+)\s*\(", txt, re.M)))


def test_exports_match_header():
    names = header_functions()
    assert set(names) == set(api.EXPORTS)
    L = api.lib()
    for n in names:
        assert hasattr(L, n), n


def test_strerror():
    L = api.lib()
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8):
        assert L.gts_strerror(code)
    assert L.gts_strerror(-99) == b"unknown error"


def _two_nodes(edges, warps=0xF, kwarps=4):
    b = GraphBuilder()
    b.kernel(kwarps, 0)
    b.cta()
    b.node(TENSOR, 10, warps)
    b.node(ALU, 10, warps)
    for u, v, k in edges:
        b.edge(u, v, k)
    return b.build()


def _mutate(g, **kw):
    d = g.arrays()
    d.update(kw)
    return TileGraph(**d)


def test_valid_graphs():
    for g in (W.workload_graph("gemm_1024_a100"), W.splitkv_decode(batch=3, seed=1), empty_graph(),
              W.decoder_layer(tokens=128, hidden=256, heads=4, kv_heads=2, ffn=512, d=64)):
        assert api.validate_code(g) == 0
        assert api.device_bytes(g) > 0


def test_validation_codes():
    g = _two_nodes([(0, 1, DATA)])
    assert api.validate_code(g) == 0
    # cycle (two nodes pointing at each other)
    assert api.validate_code(_two_nodes([(0, 1, DATA), (1, 0, ORDER)])) == -2
    # self loop
    assert api.validate_code(_mutate(g, succ_ptr=np.array([0, 1, 1], np.uint32), succ=np.array([0], np.uint32))) == -2
    # duplicate edge
    assert api.validate_code(_mutate(g, succ_ptr=np.array([0, 2, 2], np.uint32),
                                     succ=np.array([1, 1 | (1 << 30)], np.uint32))) == -8
    # edge kind 3
    assert api.validate_code(_mutate(g, succ=np.array([1 | (3 << 30)], np.uint32))) == -4
    # target out of range
    assert api.validate_code(_mutate(g, succ=np.array([7], np.uint32))) == -4
    # op index out of range
    assert api.validate_code(_mutate(g, node_op=np.array([0, 5], np.uint16))) == -4
    # class out of range
    assert api.validate_code(_mutate(g, op_cls=np.array([9, 1], np.uint8))) == -4
    # compute op with empty warp mask
    assert api.validate_code(_mutate(g, op_warps=np.array([0, 1], np.uint32))) == -4
    # warp outside the CTA
    assert api.validate_code(_two_nodes([], warps=0x30, kwarps=4)) == -4
    # bad kernel warps
    assert api.validate_code(_mutate(g, kernel_warps=np.array([0], np.uint16))) == -4
    assert api.validate_code(_mutate(g, kernel_warps=np.array([33], np.uint16))) == -4
    # empty CTA / bad offsets
    assert api.validate_code(_mutate(g, cta_node_begin=np.array([0, 0, 2], np.uint32),
                                     kernel_cta_begin=np.array([0, 2], np.uint32))) == -4
    assert api.validate_code(_mutate(g, succ_ptr=np.array([0, 1, 0], np.uint32))) == -4
    # unknown op flag
    assert api.validate_code(_mutate(g, op_flags=np.array([2, 0], np.uint8))) == -4


def test_edge_order_code():
    b = GraphBuilder()
    b.kernel(4, 0)
    b.cta()
    a = b.node(GLOAD, 64, 1)
    b.cta()
    c = b.node(GLOAD, 64, 1)
    b.edge(c, a)  # from CTA 1 back to CTA 0
    assert api.validate_code(b.build()) == -3


def test_last_error_names_the_node():
    b = GraphBuilder()
    b.kernel(2, 0)
    b.cta()
    b.node(TENSOR, 1, 1)
    b.node(TENSOR, 1, 0b100)
    with pytest.raises(api.GtsError) as e:
        api.validate(b.build())
    assert "node 1" in str(e.value)


def test_hw_validation():
    assert api.hw_validate(H.preset("H100")) == 0
    assert api.hw_validate(H.toy()) == 0
    for field, val in (("n_sm", 0), ("n_sm", 1025), ("n_subpart", 0), ("n_subpart", 9), ("rate_dram", 0),
                       ("lat_l2", (1 << 30) + 1), ("cta_launch_lat", (1 << 31))):
        r = H.preset("H100")
        r[H.FIELDS[field]] = val
        assert api.hw_validate(r) == -5, field
    r = H.preset("H100")
    r[27] = 1  # reserved word
    assert api.hw_validate(r) == -5


def test_noc_hw_validation():
    noc = dict(noc_nodes=16, noc_width=4, noc_rate=8 * H.Q16, noc_lat=20, noc_map=1)
    assert api.hw_validate(H.preset("H100", **noc)) == 0
    assert api.hw_validate(H.preset("H100", **dict(noc, noc_width=0, noc_map=0))) == 0
    for field, val in (("noc_nodes", 65), ("noc_width", 3), ("noc_width", 32), ("noc_rate", 0),
                       ("noc_lat", (1 << 24) + 1), ("noc_map", 3)):
        assert api.hw_validate(H.preset("H100", **dict(noc, **{field: val}))) == -5, field
    # NoC fields without a NoC
    assert api.hw_validate(H.preset("H100", noc_width=4)) == -5


def _cluster_kernel(cl=2, n_ctas=4, back=None, rank=1, flags=0):
    b = GraphBuilder()
    b.kernel(4, 0, cl)
    ids = []
    for c in range(n_ctas):
        b.cta()
        ids.append((b.node(REMOTE, 256, 1, remote_flags(rank) | flags), b.node(ALU, 64, 1)))
    if back is not None:
        u, v = back
        b.edge(ids[u][0], ids[v][1])
    return b.build()


def test_cluster_validation_codes():
    cases = [
        (_cluster_kernel(), 0),
        (_cluster_kernel(back=(1, 0)), 0),             # back edge inside a cluster
        (_cluster_kernel(back=(3, 2)), 0),
        (_cluster_kernel(back=(2, 1)), -3),            # back edge between clusters
        (_cluster_kernel(cl=3, n_ctas=4), -4),         # clusters must divide the CTA count
        (_cluster_kernel(cl=17, n_ctas=17), -4),       # at most 16 CTAs per cluster
        (_cluster_kernel(rank=2), -4),                 # rank outside the cluster
        (_cluster_kernel(flags=1), -4),                # REMOTE ops carry only the rank
    ]
    for g, code in cases:
        assert api.validate_code(g) == code
        if code == 0:
            validate(g)
        else:
            with pytest.raises(ValidationError):
                validate(g)


def test_tile_validation_codes():
    g = W.gemm(512, 512, 256, 128, 128, 64, 2, tiles=True)
    assert api.validate_code(g) == 0
    validate(g)
    bad = g.node_tile.copy()
    mma = int(np.flatnonzero(g.op_cls[g.node_op] == TENSOR)[0])
    bad[mma] = 7  # a compute node naming a tile
    g2 = _mutate(g, node_tile=bad)
    assert api.validate_code(g2) == -4
    with pytest.raises(ValidationError):
        validate(g2)
    # one tile touched with two sizes: a C-block id on an A load
    loads = np.flatnonzero(g.op_cls[g.node_op] == GLOAD)
    bad = g.node_tile.copy()
    bad[loads[0]] = int(g.node_tile[-1])
    g3 = _mutate(g, node_tile=bad)
    assert api.validate_code(g3) == -4
    with pytest.raises(ValidationError):
        validate(g3)
    # line counts are 64-bit: work 0 and work 0xFFFFFFFF (0 and 2^25 lines)
    # on one tile is an inconsistency, not a wrapped match
    b = GraphBuilder()
    b.kernel(4, 0)
    b.cta()
    u = b.node(GLOAD, 0, 1)
    w = b.node(GLOAD, 0xFFFFFFFF, 1)
    b.edge(u, w, DATA)
    g4 = b.build()
    g4 = _mutate(g4, node_tile=np.array([5, 5], np.uint32))
    assert api.validate_code(g4) == -4
    with pytest.raises(ValidationError):
        validate(g4)
    assert api.validate_code(_mutate(g4, node_tile=np.array([5, 6], np.uint32))) == 0
    # tiles go to the device image; sharing is unaffected
    assert api.device_bytes(g) > api.device_bytes(_mutate(g, node_tile=None))
    assert api.templates(g)["templated_kernels"] == 1


def test_address_validation_codes():
    """Transaction-level tiles: the library and the Python statement of the
    rules agree on every case -- addresses only on loads / stores, never
    beside tile ids, rows dividing the bytes, a stride of at least a row, a
    bounded transaction count, no wrap past the address space."""
    from paper_2607_11262_amd.gen.graph import MAX_NODE_TXN, NO_ADDR
    g = W.gemm_addressed(256, 256, 256, 64, 64, 32, 2, pad=8)
    assert api.validate_code(g) == 0
    validate(g)
    # the device image holds each node's lines
    assert api.device_bytes(g) > api.device_bytes(_mutate(g, node_addr=None, op_rows=None, op_pitch=None))
    mma = int(np.flatnonzero(g.op_cls[g.node_op] == TENSOR)[0])
    load = int(np.flatnonzero(g.op_cls[g.node_op] == GLOAD)[0])
    lop = int(g.node_op[load])

    def check(g2):
        assert api.validate_code(g2) == -4
        with pytest.raises(ValidationError):
            validate(g2)

    bad = g.node_addr.copy()
    bad[mma] = 4096  # a compute node with an address
    check(_mutate(g, node_addr=bad))
    rows = g.op_rows.copy()
    rows[lop] = 0
    check(_mutate(g, op_rows=rows))
    rows = g.op_rows.copy()
    rows[lop] = 3  # does not divide the tile's bytes
    check(_mutate(g, op_rows=rows))
    pitch = g.op_pitch.copy()
    pitch[lop] = int(g.op_work[lop]) // int(g.op_rows[lop]) - 1  # rows overlap
    check(_mutate(g, op_pitch=pitch))
    bad = g.node_addr.copy()
    bad[load] = np.uint64(NO_ADDR - 100)  # wraps
    check(_mutate(g, node_addr=bad))
    tiles = np.full(g.n_nodes, 0xFFFFFFFF, np.uint32)
    tiles[load] = 3  # ids beside addresses
    check(_mutate(g, node_tile=tiles))
    # too many transactions on one tile
    b = GraphBuilder()
    b.kernel(4, 0)
    b.cta()
    b.node(GLOAD, 128 * MAX_NODE_TXN, 1, addr=0)
    check(b.build())
    b = GraphBuilder()
    b.kernel(4, 0)
    b.cta()
    b.node(GLOAD, 128 * (MAX_NODE_TXN - 2), 1, addr=0)
    g3 = b.build()
    assert api.validate_code(g3) == 0
    validate(g3)

"""Seeded tile ids for the loads and stores of a graph (test helper): each
memory node touches one of a few tiles of its own size (a tile is always
accessed whole, so its id is drawn among the tiles of that line count)."""
import numpy as np

from paper_2607_11262_amd.gen.graph import GLOAD, GSTORE, LINE_BYTES, NO_TILE


def with_tiles(g, rng, per_size=4, tracked=0.9):
    ops = g.node_op.astype(np.int64)
    mem = np.isin(g.op_cls, (GLOAD, GSTORE))[ops]
    lines = -(-g.op_work.astype(np.int64)[ops] // LINE_BYTES)
    tiles = np.full(g.n_nodes, NO_TILE, dtype=np.uint32)
    for v in np.flatnonzero(mem):
        if rng.randint(0, 999) < tracked * 1000:
            tiles[v] = int(lines[v]) * 64 + rng.randint(0, per_size - 1)
    g.node_tile = tiles
    return g

"""NoC-enabled fusion case study (Sec. 7.2) on the CPU: the cluster-fused
attention graphs, the crossbar / mesh machines, the NoC residence tool, and
the case study's findings under the oracle."""
import numpy as np
import pytest

import oracle
from paper_2607_11262_amd import api
from paper_2607_11262_amd import timeline as TL
from paper_2607_11262_amd.gen import clusterfusion as CF
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen.graph import (DATA, GLOAD, GSTORE, REMOTE, SYNC, GraphBuilder, remote_flags,
                                             validate)

HEADS = 8


@pytest.mark.parametrize("S", CF.CLUSTER_SIZES)
@pytest.mark.parametrize("comm", CF.COMMS)
def test_graphs(S, comm):
    g = CF.cluster_attention(S, heads=HEADS, comm=comm)
    validate(g)
    assert api.validate_code(g) == 0
    assert g.n_ctas == HEADS * S and int(g.kernel_cluster[0]) == S
    cls = g.op_cls[g.node_op]
    exchanges = 5  # four reductions and one gather
    if comm == "noc":
        assert int((cls == REMOTE).sum()) == HEADS * exchanges * S * (S - 1)
        # every REMOTE node targets another rank of its own cluster
        ranks = (g.op_flags[g.node_op] >> 4)[cls == REMOTE]
        own = (g.node_cta() % S)[cls == REMOTE]
        assert np.all(ranks != own)
    else:
        assert int((cls == REMOTE).sum()) == 0
        assert int((cls == SYNC).sum()) == HEADS * exchanges * S


def test_mesh_matches_crossbar_totals():
    x, m = CF.noc_h100("crossbar"), CF.noc_h100("mesh")
    # same total bandwidth: 32 crossbar ports vs 48 mesh links
    assert abs(48 * H.get(m, "noc_rate") - 32 * H.get(x, "noc_rate")) <= 48
    # same mean latency between distinct nodes of a 4 x 4 mesh (8/3 hops)
    assert CF._mesh_hops(4, 16) == pytest.approx(8 / 3)
    assert abs(H.get(m, "noc_lat") * 8 / 3 - H.get(x, "noc_lat")) <= 2
    assert api.hw_validate(x) == 0 and api.hw_validate(m) == 0


def test_noc_residence_hand_values():
    # toy machine, crossbar of 4 nodes, 16 B/cycle ports, latency 10; rank 0's
    # ALU (occ 4, latency 4, finish 8) feeds two 64-B transfers to rank 1:
    # the first holds the ports [8, 12) and finishes at 22, the second waits
    # for them: start 12, finish 26
    b = GraphBuilder()
    b.kernel(1, 1024, 2)
    b.cta()
    a = b.node(1, 64, 1)
    t1 = b.node(REMOTE, 64, 1, remote_flags(1))
    t2 = b.node(REMOTE, 64, 1, remote_flags(1))
    b.cta()
    b.node(1, 64, 1)
    b.edge(a, t1, DATA)
    b.edge(a, t2, DATA)
    g = b.build()
    rec = H.toy(n_sm=4, noc_nodes=4, noc_rate=16 * H.Q16, noc_lat=10)
    r = oracle.simulate(g, rec, 0)
    assert r.cycles[:3].tolist() == [[0, 8], [8, 22], [12, 26]]
    assert TL.ready_cycles(g, r.cycles)[1:3].tolist() == [8, 8]
    assert TL.noc_residence(g, r.cycles) == pytest.approx(((22 - 8) + (26 - 8)) / 2)


def _run(g, rec):
    r = oracle.simulate(g, rec, 0)
    assert r.status == 0
    return r


def test_noc_beats_dram():
    """Sec. 7.2 (1): exchanging through the NoC is faster than through DRAM,
    most for the largest clusters (the most traffic per exchange)."""
    rec = CF.noc_h100("crossbar")
    gain = {}
    for S in CF.CLUSTER_SIZES:
        noc = _run(CF.cluster_attention(S, heads=HEADS), rec).makespan
        dram = _run(CF.cluster_attention(S, heads=HEADS, comm="dram"), rec).makespan
        assert noc < dram, S
        gain[S] = dram / noc
    assert gain[16] == max(gain.values())


def test_topology_aware_mapping():
    """Sec. 7.2 (2): the crossbar's residence is uniform across cluster
    sizes; on the mesh a compact placement shortens residence against a
    topology-oblivious (strided) one, most for small clusters, and the two
    coincide once a cluster fills the mesh."""
    res = {}
    for S in CF.CLUSTER_SIZES:
        g = CF.cluster_attention(S, heads=HEADS)
        for key in (("crossbar", "strips"), ("mesh", "blocks"), ("mesh", "strided")):
            res[(S,) + key] = TL.noc_residence(g, _run(g, CF.noc_h100(*key)).cycles)
    xbar = [res[(S, "crossbar", "strips")] for S in CF.CLUSTER_SIZES]
    assert max(xbar) - min(xbar) < 0.05 * min(xbar)
    ratio = {S: res[(S, "mesh", "strided")] / res[(S, "mesh", "blocks")] for S in CF.CLUSTER_SIZES}
    assert all(ratio[S] > 1.1 for S in (2, 4, 8))
    assert ratio[16] == pytest.approx(1.0)
    assert ratio[2] == max(ratio.values())


def test_machine_sampler():
    recs = CF.sample_noc_machines(5, 64)
    assert all(api.hw_validate(r) == 0 for r in recs)
    assert {H.get(r, "noc_width") for r in recs} == {0, 4}
    assert {H.get(r, "noc_map") for r in recs} == {0, 1, 2}

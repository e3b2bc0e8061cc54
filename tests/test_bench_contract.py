"""bench.py pieces that need no GPU: the one-GPU guard, the algorithmic
bytes of a simulation, and the traffic record (HBM bytes per launch from a
committed counter summary, reported only while the kernel sources hash to
the recorded value)."""
import hashlib
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2607_11262_amd.gen.graph import DATA, GLOAD, GSTORE, GraphBuilder  # noqa: E402


def test_more_than_one_gpu_is_refused(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "4"])
    assert bench.main() == 2
    assert "one GPU" in capsys.readouterr().err


def test_algorithmic_bytes():
    """10 B per node and 4 B per edge of graph read, 16 B of per-simulation
    output, and 8 B per node more with per-node cycles."""
    b = GraphBuilder()
    b.kernel(4, 0)
    b.cta()
    a = b.node(GLOAD, 256, 1)
    s = b.node(GSTORE, 256, 1)
    b.edge(a, s, DATA)
    g = b.build("two")
    assert bench.alg_bytes_per_sim(g, False) == 10 * 2 + 4 * 1 + 16
    assert bench.alg_bytes_per_sim(g, True) == 10 * 2 + 4 * 1 + 16 + 8 * 2


def _record(tmp_path, sha, workload="gemm_design_sweep", outputs="digest"):
    p = tmp_path / "summary.md"
    p.write_text(f"text\n    traffic-record: workload={workload} outputs={outputs} sha256={sha} node_sims=1000 "
                 f"fetch_kib=1000 write_kib=3000 fetch_factor=2.0000 write_factor=1.0000\n")
    return str(tmp_path)


def test_traffic_record_read_while_sources_match(tmp_path):
    d = _record(tmp_path, bench.sources_hash())
    assert bench.recorded_traffic("gemm_design_sweep", "digest", d) == pytest.approx(
        (1000 * 1024 * 2.0 + 3000 * 1024 * 1.0) / 1000)


def test_traffic_record_ignored_for_other_sources_workloads_or_outputs(tmp_path):
    d = _record(tmp_path, "0" * 64)
    assert bench.recorded_traffic("gemm_design_sweep", "digest", d) is None
    d = _record(tmp_path, bench.sources_hash())
    assert bench.recorded_traffic("splitkv_decode_b64", "digest", d) is None
    assert bench.recorded_traffic("gemm_design_sweep", "nodes", d) is None
    assert bench.recorded_traffic("gemm_design_sweep", "digest", str(tmp_path / "missing")) is None


def test_workload_parts_cover_the_named_configs():
    """Every named workload and case study has its graphs and records; the
    sweep is 64 graphs x 4096 records, the others one graph each with the
    batch size of their configuration."""
    sizes = {"gemm_design_sweep": (64, 4096), "gemm_1024_a100": (1, 16)}
    for name, (n_graphs, B) in sizes.items():
        describe, make, n = bench.workload_parts(name)
        assert n == n_graphs
        g, hw = make(0)
        assert hw.shape == (B, 32) and g.n_nodes > 0


def test_cpu_leg_checks_every_launch_and_counts_mismatches():
    """The CPU leg with a stand-in plan whose 'GPU' outputs are the oracle's
    own: it samples every launch and finds no mismatch; a wrong makespan
    planted in one record and a wrong node cycle in every record are
    counted."""
    import numpy as np
    import torch

    import oracle
    from paper_2607_11262_amd.gen import hw as H
    from paper_2607_11262_amd.gen import workloads as W

    class FakePlan:
        pass

    g = W.gemm(256, 256, 256, 64, 64, 32, 2)
    hw = H.sample_h100_sweep(5, 12)
    mk, st, dg, cyc = oracle.simulate_records(g, hw, oracle.F_NODES | oracle.F_DIGEST, want_nodes=True)
    mk = mk.copy()
    cyc = cyc.copy()
    outs = (torch.from_numpy(cyc.view(np.int32)), torch.from_numpy(mk.view(np.int32)), torch.from_numpy(st),
            torch.from_numpy(dg.view(np.int64)))
    plan = FakePlan()
    plan.parts = [(None, None, outs, g, hw)]
    plan.launches = [(0, 0, 6), (0, 6, 6)]
    cpu, parity = bench.cpu_leg(plan, oracle.F_DIGEST, 1.0, True)
    assert parity["mismatches"] == 0 and parity["node_cycle_mismatches"] == 0
    assert parity["launches_sampled"] == 2 and parity["checked_sims"] == 12
    assert cpu["value"] > 0 and cpu["single_core"] > 0 and cpu["cores"] >= 1
    # plant a wrong makespan and a wrong node cycle in every record (stand-in GPU outputs)
    outs[1][3] += 1
    outs[0][:, 5, 1] += 1
    cpu, parity = bench.cpu_leg(plan, oracle.F_DIGEST, 1.0, True)
    assert parity["mismatches"] >= 1 and parity["node_cycle_mismatches"] >= 1

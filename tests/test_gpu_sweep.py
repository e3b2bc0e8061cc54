"""GPU parity of the GEMM design sweep in the bench's own launch shapes:
bench.py's plan (all 64 graphs x 4096 records, each graph's records in the
equal chunks its scratch budget allows -- graphs 6 and 50 take more than one
launch, at records first > 0 -- alternating over two streams) runs once, and
records drawn from every launch are checked against the oracle: at least 64
per graph (status, makespan, digest; 262,144 simulations run) and per-node
cycles on four records per graph."""
import sys

import numpy as np
import pytest

import bench
import oracle
from paper_2607_11262_amd import api

pytestmark = pytest.mark.gpu


def note(msg):
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def sweep_plan():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    streams = [torch.cuda.current_stream(), torch.cuda.Stream()]
    budget = int(220.0 * (1 << 30)) // 2  # bench.py's default budget over its two streams
    plan = bench.Plan(api, torch, "gemm_design_sweep", api.OUT_DIGEST, budget, streams, torch.device("cuda:0"))
    note(f"sweep plan: {len(plan.parts)} graphs, {len(plan.launches)} launches")
    plan.step(api, torch)
    torch.cuda.synchronize()
    yield plan, torch
    del plan
    torch.cuda.empty_cache()


def sample(plan, per_graph=64):
    """Per graph: records spread over each of its launches (seeded), at
    least `per_graph` in all."""
    rng = np.random.default_rng(11)
    out = {}
    for i, first, b in plan.launches:
        n_launch = sum(1 for j, _, _ in plan.launches if j == i)
        k = -(-per_graph // n_launch)
        out.setdefault(i, []).extend(int(first + r) for r in rng.choice(b, size=min(k, b), replace=False))
    return out


def test_sweep_launches_cover_chunked_graphs(sweep_plan):
    """The plan this test checks is the chunked one: some graph spans more
    than one launch, so launches with first > 0 run."""
    plan, _ = sweep_plan
    assert any(first > 0 for _, first, _ in plan.launches)
    assert len({i for i, _, _ in plan.launches}) == 64


def test_sweep_every_graph_against_oracle(sweep_plan):
    plan, torch = sweep_plan
    picks = sample(plan)
    total = 0
    for i in sorted(picks):
        dg, hs, (cyc, mk, st, dgst), g, hw = plan.parts[i]
        recs = sorted(picks[i])
        note(f"sweep graph {i} N={g.n_nodes}: {len(recs)} records, launches "
             f"{[(f, b) for j, f, b in plan.launches if j == i]}")
        gmk = mk.cpu().numpy().view(np.uint32)[recs]
        gst = st.cpu().numpy()[recs]
        gdg = dgst.cpu().numpy().view(np.uint64)[recs]
        omk, ost, odg, _ = oracle.simulate_batch(g, hw[recs], api.OUT_DIGEST, threads=16)
        bad = np.flatnonzero((gmk != omk) | (gst != ost) | (gdg != odg))
        assert bad.size == 0, f"graph {i}: records {[recs[j] for j in bad[:5]]} differ"
        total += len(recs)
    assert total >= 64 * 64


def test_sweep_node_cycles_four_per_graph(sweep_plan):
    """Four records of every graph (one in each launch where a graph has
    several) with per-node output, through the same chunked entry point
    (gts_simulate_hwset at the record's own offset), node by node against
    the oracle; their makespans and digests equal the plan's."""
    plan, torch = sweep_plan
    rng = np.random.default_rng(12)
    for i, part in enumerate(plan.parts):
        dg, hs, (cyc, mk, st, dgst), g, hw = part
        launches = [(f, b) for j, f, b in plan.launches if j == i]
        recs = sorted({int(f + rng.integers(b)) for f, b in launches} | set(int(x) for x in rng.choice(4096, 4, False)))[:4]
        flags = api.OUT_NODES | api.OUT_DIGEST
        streams = [torch.cuda.Stream() for _ in recs]  # the four records run side by side
        runs = []
        for r, s in zip(recs, streams):
            with torch.cuda.stream(s):
                scratch = torch.empty(api.scratch_bytes(dg, 1, flags), dtype=torch.uint8, device="cuda")
                out = api.alloc_outputs(dg, 1, flags)
            api.simulate_hwset_into(dg, hs, r, 1, flags, *out, scratch, s)
            runs.append((r, out, scratch))
        torch.cuda.synchronize()
        gmk = mk.cpu().numpy().view(np.uint32)
        gdg = dgst.cpu().numpy().view(np.uint64)
        for r, out, _ in runs:
            c, m, s_, d = (out[0].cpu().numpy().view(np.uint32)[0], int(out[1].cpu().numpy().view(np.uint32)[0]),
                           int(out[2].cpu().numpy()[0]), int(out[3].cpu().numpy().view(np.uint64)[0]))
            o = oracle.simulate(g, hw[r], flags)
            assert (s_, m, d) == (o.status, o.makespan, o.digest), f"graph {i} record {r}"
            assert m == int(gmk[r]) and d == int(gdg[r]), f"graph {i} record {r}: differs from the plan's launch"
            if o.status == 0:
                assert np.array_equal(c, o.cycles), f"graph {i} record {r}: node cycles differ"
        runs.clear()
        note(f"sweep graph {i}: node cycles of records {recs} match")

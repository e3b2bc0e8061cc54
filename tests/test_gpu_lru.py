"""GPU parity for the LRU L2 (Sec. 5.2 tile-derived accesses on a fully
associative LRU of 128-B lines): random graphs whose loads and stores name
tiles, on random machines with capacities from one line to all of them, and
tiled GEMMs on Table 3's H100 across L2 sizes, bit-exact against the
oracle (every node's start and finish, makespan, status, digest)."""
import numpy as np
import pytest

from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import workloads as W
from paper_2607_11262_amd.gen.rng import SplitMix64
from test_gpu_parity import ALL, compare, note, run_gpu
from tiled import with_tiles

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


@pytest.mark.parametrize("chunk", range(4))
def test_random_tiled_graphs(torch_cuda, chunk):
    for seed in range(chunk * 25, chunk * 25 + 25):
        rng = SplitMix64(seed, 41)
        g = with_tiles(W.random_graph(rng, n_nodes_max=rng.choice([20, 80, 300]), n_kernels_max=3, ctas_max=6),
                       rng, per_size=rng.choice([2, 8, 64]))
        B = rng.randint(1, 8)
        hws = []
        for _ in range(B):
            r = H.sample_random(rng, n_sm_max=rng.choice([1, 3, 70]))
            r[H.FIELDS["l2_lines"]] = rng.choice([0, 1, 4, 16, 64, 512, 1 << 20])
            hws.append(r)
        hws = np.stack(hws)
        flags = ALL | rng.choice([0, 0, 4, 8])
        note(f"tiled seed={seed} N={g.n_nodes} B={B} flags={flags}")
        compare(g, hws, flags, run_gpu(torch_cuda, g, hws, flags))


def test_tiled_gemm_capacities(torch_cuda):
    g = W.gemm(2048, 2048, 1024, 128, 128, 64, 3, tiles=True)
    hws = np.stack([H.preset("H100", n_sm=n, l2_lines=H.l2_lines(mib))
                    for n in (32, 132) for mib in (0, 0.25, 1, 4, 50)])
    note(f"tiled gemm N={g.n_nodes} B={hws.shape[0]}")
    compare(g, hws, ALL, run_gpu(torch_cuda, g, hws, ALL))


# ---- the windowed kernel's LRU decisions (memory batches of up to 256
# arrivals decided together in (cycle, id) order)

def _window_only(torch, g, hws, flags, monkeypatch):
    from test_gpu_windowed import run_window_only
    return run_window_only(torch, g, hws, flags, monkeypatch)


STATUS_RETRY = 0x52455452


def _check_ran(st, windows, what):
    assert not np.any(st == STATUS_RETRY), f"{what}: windowed kernel handed back sims {np.flatnonzero(st == STATUS_RETRY)}"
    feasible = st != api.SIM_INFEASIBLE
    assert np.all(windows[feasible] > 0), f"{what}: a feasible simulation did not run on the windowed kernel"
    return int(feasible.sum())


@pytest.mark.parametrize("chunk", range(6))
def test_window_lru_random(torch_cuda, chunk, monkeypatch):
    """150 random graphs the windowed kernel accepts, their loads / stores
    naming a few tiles of each size (so one memory batch repeats tiles), on
    machines of 1-256 SMs with L2s of one line to all of them: each
    simulation ran on the windowed kernel to the end, and every node's cycles
    equal the oracle's."""
    from windowed import window_eligible, windowed_graph, windowed_machines
    ran = 0
    for seed in range(chunk * 25, chunk * 25 + 25):
        rng = SplitMix64(seed, 93)
        g = with_tiles(windowed_graph(rng), rng, per_size=rng.choice([1, 2, 8, 64]), tracked=rng.choice([0.5, 0.9, 1.0]))
        assert window_eligible(g)
        B = rng.randint(1, 8)
        hws = windowed_machines(rng, B)
        for r in hws:
            r[H.FIELDS["l2_lines"]] = rng.choice([0, 1, 2, 8, 40, 256, 4096, 1 << 20])
        flags = ALL | rng.choice([0, api.NO_CONTENTION, api.ORDER_AT_FINISH])
        note(f"window lru seed={seed} N={g.n_nodes} B={B} l2={hws[:, H.FIELDS['l2_lines']].tolist()} flags={flags}")
        gpu, windows = _window_only(torch_cuda, g, hws, flags, monkeypatch)
        ran += _check_ran(gpu[2], windows, f"seed {seed}")
        compare(g, hws, flags, gpu)
    assert ran > 0


def _simultaneous_tiled_graph():
    """512 CTAs whose loads all arrive in the first cycles: memory batches of
    256 arrivals with the same tiles many times over."""
    from paper_2607_11262_amd.gen.graph import ALU, GLOAD, GSTORE, MISS, NO_TILE, GraphBuilder
    b = GraphBuilder()
    b.kernel(4, 0)
    tiles = {}
    for c in range(512):
        b.cta()
        la = b.node(GLOAD, 1024 * (c % 3 + 1), 0xF, MISS if c % 2 else 0)
        lb = b.node(GLOAD, 2048, 0xF, MISS)
        a = b.node(ALU, 4096, 0xF)
        st = b.node(GSTORE, 512, 0xF, MISS)
        tiles[la] = 100 * (c % 3) + c % 7  # one size per tile id
        tiles[lb] = 1000 + c % 11
        if c % 4:
            tiles[st] = 2000 + c % 13
        b.edge(la, a)
        b.edge(lb, a)
        b.edge(a, st)
    g = b.build("simultaneous_tiled")
    t = np.full(g.n_nodes, NO_TILE, dtype=np.uint32)
    for v, x in tiles.items():
        t[v] = x
    g.node_tile = t
    return g


@pytest.mark.parametrize("name", ["simultaneous", "gemm"])
def test_window_lru_batches(torch_cuda, name, monkeypatch):
    """Full batches of repeated tiles, and a tiled GEMM of the design sweep
    across L2 sizes, on the windowed kernel alone: no hand-back, and equal to
    the oracle node by node."""
    if name == "simultaneous":
        g = _simultaneous_tiled_graph()
        hws = np.stack([H.preset("H100", n_sm=n, l2_lines=l2) for n in (256, 129, 64)
                        for l2 in (1, 16, 64, 200, 1 << 20)])
    else:
        g = W.gemm(2048, 2048, 1024, 128, 128, 64, 3, tiles=True)
        hws = np.stack([H.preset("H100", n_sm=n, l2_lines=H.l2_lines(mib))
                        for n in (32, 132, 200) for mib in (0, 0.25, 1, 4, 50)])
    note(f"window lru {name} N={g.n_nodes} B={hws.shape[0]}")
    gpu, windows = _window_only(torch_cuda, g, hws, ALL, monkeypatch)
    _check_ran(gpu[2], windows, name)
    compare(g, hws, ALL, gpu)

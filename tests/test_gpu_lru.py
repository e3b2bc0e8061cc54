"""GPU parity for the LRU L2 (Sec. 5.2 tile-derived accesses on a fully
associative LRU of 128-B lines): random graphs whose loads and stores name
tiles, on random machines with capacities from one line to all of them, and
tiled GEMMs on Table 3's H100 across L2 sizes, bit-exact against the
oracle (every node's start and finish, makespan, status, digest)."""
import numpy as np
import pytest

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

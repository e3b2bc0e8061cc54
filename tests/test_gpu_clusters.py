"""GPU parity for thread-block clusters and the SM-cluster NoC (Sec. 5.2
DSMEM, Sec. 7.2): random clustered graphs with REMOTE nodes on random
crossbar / mesh machines, and the cluster-fused attention graphs under every
topology and mapping, bit-exact against the oracle (every node's start and
finish, makespan, status, digest)."""
import numpy as np
import pytest

from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import clusterfusion as CF
from paper_2607_11262_amd.gen.rng import SplitMix64
from clustered import clustered_graph, noc_machine
from test_gpu_parity import ALL, compare, note, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


@pytest.mark.parametrize("chunk", range(4))
def test_random_clustered_graphs(torch_cuda, chunk):
    for seed in range(chunk * 25, chunk * 25 + 25):
        rng = SplitMix64(seed, 31)
        g = clustered_graph(rng, nodes=(1, 12), clusters=(1, 6))
        B = rng.randint(1, 8)
        hws = np.stack([noc_machine(rng) for _ in range(B)])
        flags = ALL | rng.choice([0, 0, 4, 8])
        note(f"clustered seed={seed} N={g.n_nodes} C={g.n_ctas} B={B} flags={flags}")
        compare(g, hws, flags, run_gpu(torch_cuda, g, hws, flags))


@pytest.mark.parametrize("S", CF.CLUSTER_SIZES)
def test_cluster_attention(torch_cuda, S):
    hws = np.stack([CF.noc_h100(t, m) for t, m in (("crossbar", "strips"), ("mesh", "strips"), ("mesh", "blocks"),
                                                   ("mesh", "strided"))] + list(CF.sample_noc_machines(S, 4)))
    for comm in CF.COMMS:
        g = CF.cluster_attention(S, heads=8, kv_len=1024, comm=comm)
        note(f"cluster attention S={S} {comm} N={g.n_nodes} B={hws.shape[0]}")
        compare(g, hws, ALL, run_gpu(torch_cuda, g, hws, ALL))

"""GPU parity on the software-pipelining case-study graphs (Sec. 7.1) and
their Table 4 edge-class ablations: every node's (start, finish), makespan,
status and digest from the HIP path equal the oracle's, on single-SM Hopper
machines around Table 3's H100 (tensor rate, DRAM bandwidth and subpartition
count varied) and on random single-SM machines."""
import numpy as np
import pytest

from paper_2607_11262_amd import api
from paper_2607_11262_amd import timeline as TL
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import pipelining as PL
from paper_2607_11262_amd.gen.rng import SplitMix64
from test_gpu_parity import ALL, compare, note, run_gpu

pytestmark = pytest.mark.gpu


def machines(seed: int):
    recs = [H.preset("H100", n_sm=1, tensor_permille=tp, dram_mb_s=mb)
            for tp in (1000, 2000, 4000) for mb in (1_500_000, 3_100_000, 8_000_000)]
    recs.append(H.preset("H100", n_sm=1, tensor_permille=2000, n_subpart=2))
    recs.append(H.preset("H100", n_sm=4, tensor_permille=2000))
    rng = SplitMix64(seed, 7)
    for _ in range(3):
        r = H.sample_random(rng, n_sm_max=1)
        r[H.FIELDS["max_warps_per_sm"]] = 64
        r[H.FIELDS["smem_per_sm"]] = 256 * 1024
        recs.append(r)
    return np.stack(recs)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


@pytest.mark.parametrize("tile", PL.TILES)
def test_pipelining_parity(torch_cuda, tile):
    hws = machines(sum(tile))
    for name, kinds in PL.ABLATIONS.items():
        for org in PL.ORGANIZATIONS:
            g = PL.gemm_silu(org, *tile, drop=kinds)
            note(f"{g.name} N={g.n_nodes} B={hws.shape[0]}")
            compare(g, hws, ALL, run_gpu(torch_cuda, g, hws, ALL))


@pytest.mark.parametrize("name", list(PL.ABLATIONS))
def test_pipelining_general_kernel(torch_cuda, name, monkeypatch):
    monkeypatch.setenv("GTS_KERNEL", "general")
    hws = machines(3)
    for org in PL.ORGANIZATIONS:
        g = PL.gemm_silu(org, 128, 256, 64, waves=4, drop=PL.ABLATIONS[name])
        note(f"general kernel {g.name} N={g.n_nodes}")
        compare(g, hws, ALL, run_gpu(torch_cuda, g, hws, ALL))


def test_pipelining_case_study_on_gpu(torch_cuda):
    """The case study read off the GPU timelines: WS cooperative beats naive
    2-stage; WS ping-pong loses at (128,128,64) and wins at (256,256,128)."""
    rec = H.preset("H100", n_sm=1, tensor_permille=2000)[None, :]
    util = {}
    for tile in ((128, 128, 64), (256, 256, 128)):
        mk = {}
        for org in PL.ORGANIZATIONS:
            g = PL.gemm_silu(org, *tile)
            cyc, m, st, _ = run_gpu(torch_cuda, g, rec, ALL)
            assert st[0] == 0
            mk[org] = int(m[0])
            util[(tile, org)] = TL.utilization(g, rec[0], cyc[0])["tensor"]
            note(f"{tile} {org}: makespan {mk[org]} tensor {100 * util[(tile, org)]:.1f}%")
        assert mk["cooperative"] < mk["naive"]
        assert (mk["pingpong"] > mk["cooperative"]) == (tile == (128, 128, 64))
    assert util[((256, 256, 128), "pingpong")] > util[((256, 256, 128), "cooperative")]

"""GPU parity of transaction-level memory (tiles with byte addresses: each
expanded into its 128-B lines, streamed by the SM's engine, served one by
one by the L2 / DRAM servers with an LRU of lines): random graphs with
random tile shapes, strides and addresses, some memory nodes left without
an address, on random machines with and without an L2 capacity, and GEMMs
whose tiles sit in row-major or column-major tensors with and without
leading-dimension padding, every node's cycles bit-exact against the
oracle."""
import sys

import numpy as np
import pytest

import oracle
from addressed import with_addresses
from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import workloads as W
from paper_2607_11262_amd.gen.rng import SplitMix64

pytestmark = pytest.mark.gpu

ALL = api.OUT_NODES | api.OUT_DIGEST


def note(msg):
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def run_and_compare(torch, g, hws, flags):
    dg = api.upload(g)
    res = api.simulate(dg, hws, flags)
    torch.cuda.synchronize()
    cyc, mk, st, dgst = api.to_numpy(res)
    omk, ost, odg, ocyc = oracle.simulate_batch(g, hws, flags, want_nodes=True, threads=16)
    for b in range(hws.shape[0]):
        assert st[b] == ost[b], f"sim {b}: status {st[b]} != {ost[b]}"
        assert mk[b] == omk[b] and dgst[b] == odg[b], f"sim {b}: makespan {mk[b]} != {omk[b]}"
        if ost[b] == 0:
            diff = np.flatnonzero(np.any(cyc[b] != ocyc[b], axis=1))
            assert diff.size == 0, f"sim {b}: {diff.size} nodes differ, first {diff[:5]}"
    return mk, st


@pytest.mark.parametrize("chunk", range(4))
def test_random_addressed_graphs(torch_cuda, chunk):
    for seed in range(chunk * 25, chunk * 25 + 25):
        rng = SplitMix64(seed, 27)
        g = with_addresses(W.random_graph(rng, n_nodes_max=rng.choice([10, 40, 150]), n_kernels_max=2, ctas_max=5),
                           rng, tracked=rng.choice([0.5, 0.9, 1.0]))
        B = rng.randint(1, 6)
        hws = np.stack([H.sample_random(rng, n_sm_max=rng.choice([1, 4, 70])) for _ in range(B)])
        hws[:, H.FIELDS["l2_lines"]] = [rng.choice([0, 0, 1, 3, 16, 100, 4096]) for _ in range(B)]
        flags = ALL | rng.choice([0, 0, 4, 8])
        note(f"addressed random seed={seed} N={g.n_nodes} B={B} flags={flags}")
        run_and_compare(torch_cuda, g, hws, flags)


@pytest.mark.parametrize("variant", ["kn", "kn_pad8", "nk", "bk64"])
def test_addressed_gemm(torch_cuda, variant):
    kw = {"kn": dict(), "kn_pad8": dict(pad=8), "nk": dict(b_layout="nk"), "bk64": dict(BK=64)}[variant]
    BK = kw.pop("BK", 32)
    g = W.gemm_addressed(512, 512, 512, 128, 128, BK, 3, **kw)
    hws = H.sample_h100_sweep(60, 24)
    hws[:, H.FIELDS["l2_lines"]] = [0, 0, 0, 0] + [H.l2_lines(m) for m in (0.25, 1, 2, 4, 8, 16, 32, 64) * 2 + (50,) * 4]
    note(f"addressed gemm {variant} N={g.n_nodes}")
    mk, st = run_and_compare(torch_cuda, g, hws, ALL)
    assert (st == 0).sum() > 0

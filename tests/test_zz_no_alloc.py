"""gts_simulate_hwset_noalloc through the C ABI: its results equal
gts_simulate_hwset's (caller scratch) bit for bit on consecutive calls that
reuse the library's scratch array with smaller inputs, on the windowed and
the general kernel, and a batch larger than the array is refused before
anything is enqueued."""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import workloads as W

pytestmark = pytest.mark.gpu

ALL = api.OUT_NODES | api.OUT_DIGEST


def note(msg):
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def host(out):
    cyc, mk, st, dg = out
    return (cyc.cpu().numpy().view(np.uint32), mk.cpu().numpy().view(np.uint32), st.cpu().numpy(),
            dg.cpu().numpy().view(np.uint64))


def both(torch, g, hws, first, B):
    """The same records through the caller-scratch entry point and the
    no-allocation one, on the current stream; host copies of both."""
    dg = api.upload(g)
    hs = api.upload_hw(hws)
    scratch = torch.empty(api.scratch_bytes(dg, B, ALL), dtype=torch.uint8, device="cuda")
    ref = api.alloc_outputs(dg, B, ALL)
    api.simulate_hwset_into(dg, hs, first, B, ALL, *ref, scratch)
    out = api.alloc_outputs(dg, B, ALL)
    api.simulate_hwset_noalloc(dg, hs, first, B, ALL, *out)
    torch.cuda.synchronize()
    return host(ref), host(out)


def assert_same(ref, out):
    for a, b, name in zip(ref, out, ("cycles", "makespan", "status", "digest")):
        assert np.array_equal(a, b), f"{name} differs"


def test_noalloc_matches_caller_scratch():
    import torch
    assert torch.cuda.is_available()
    cases = [
        # (graph, records, first, B): each call smaller than the one before
        ("gemm 1024^3 (windowed kernel)", W.gemm(1024, 1024, 1024, 128, 128, 32, 2), H.sample_h100_sweep(11, 96), 16, 64),
        ("gemm 512^3 (windowed kernel)", W.gemm(512, 512, 512, 128, 128, 32, 2), H.sample_h100_sweep(12, 24), 3, 16),
        ("tiled gemm, LRU L2 (general kernel)", W.gemm(512, 512, 256, 64, 64, 32, 2, tiles=True),
         H.sample_h100_sweep(13, 8), 0, 8),
    ]
    for name, g, hws, first, B in cases:
        if "LRU" in name:
            hws = hws.copy()
            hws[:, 26] = np.arange(1, B + 1, dtype=np.uint32) * 2048  # L2 lines
        note(f"noalloc vs caller scratch: {name}, {g.n_nodes} nodes, records {first}..{first + B}")
        ref, out = both(torch, g, hws, first, B)
        assert_same(ref, out)
        assert (out[2] == api.SIM_OK).sum() > 0
        # and the first two simulations against the oracle
        for b in range(2):
            r = oracle.simulate(g, hws[first + b], ALL)
            assert out[2][b] == r.status and out[1][b] == r.makespan and out[3][b] == r.digest
            if r.status == 0:
                assert np.array_equal(out[0][b], r.cycles)


def test_noalloc_refuses_oversized_batch():
    import torch
    assert torch.cuda.is_available()
    g = W.gemm(1024, 1024, 1024, 128, 128, 32, 2)
    dg = api.upload(g)
    per_sim = api.scratch_bytes(dg, 2, 0) - api.scratch_bytes(dg, 1, 0)
    B = api.NOALLOC_SCRATCH_BYTES // per_sim + 1
    hws = H.sample_h100_sweep(14, B)
    hs = api.upload_hw(hws)
    out = api.alloc_outputs(dg, B, api.OUT_DIGEST)
    note(f"noalloc refuses {B} simulations of {per_sim} B each")
    with pytest.raises(api.GtsError) as e:
        api.simulate_hwset_noalloc(dg, hs, 0, B, api.OUT_DIGEST, *out)
    assert e.value.code == -6 and "no-allocation" in str(e.value)
    # the largest batch that fits still runs
    ok = B - 1
    api.simulate_hwset_noalloc(dg, hs, 0, ok, api.OUT_DIGEST, None, out[1][:ok], out[2][:ok], out[3][:ok])
    torch.cuda.synchronize()
    assert (out[2][:ok].cpu().numpy() == api.SIM_OK).all()

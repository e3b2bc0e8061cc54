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


# ---- the windowed kernel's transaction-level memory (lines streamed into the
# memory phase's batches, an LRU of lines decided per batch, servers in
# 2^-16 cycles)

STATUS_RETRY = 0x52455452


def _all_addressed(g, rng):
    """Every load / store of g gets at least one byte and an address."""
    from paper_2607_11262_amd.gen.graph import GLOAD, GSTORE
    work = np.asarray(g.op_work).copy()
    for p in range(g.n_ops):
        if int(g.op_cls[p]) in (GLOAD, GSTORE) and work[p] == 0:
            work[p] = rng.randint(1, 4096)
    g.op_work = work.astype(g.op_work.dtype)
    return with_addresses(g, rng, tracked=1.0)


def _window_only(torch, g, hws, flags, monkeypatch):
    from test_gpu_windowed import run_window_only
    return run_window_only(torch, g, hws, flags, monkeypatch)


def _compare(g, hws, flags, gpu):
    cyc, mk, st, dgst = gpu
    omk, ost, odg, ocyc = oracle.simulate_batch(g, hws, flags, want_nodes=True, threads=16)
    for b in range(hws.shape[0]):
        assert st[b] == ost[b], f"sim {b}: status {st[b]} != {ost[b]}"
        assert mk[b] == omk[b] and dgst[b] == odg[b], f"sim {b}: makespan {mk[b]} != {omk[b]}"
        if ost[b] == 0:
            diff = np.flatnonzero(np.any(cyc[b] != ocyc[b], axis=1))
            assert diff.size == 0, f"sim {b}: {diff.size} nodes differ, first {diff[:5]}"


@pytest.mark.parametrize("chunk", range(6))
def test_window_txn_random(torch_cuda, chunk, monkeypatch):
    """150 random graphs the windowed kernel accepts with every load / store
    addressed (random tile shapes, strides and overlapping addresses), on
    machines of 1-256 SMs whose engines move 1-256 B per cycle (above 128 B
    a node's last line and the next node's first can enter in one cycle),
    with L2s of 0 lines to 2^20: each simulation ran on the windowed kernel
    to the end, and every node's cycles equal the oracle's."""
    from windowed import window_eligible, windowed_graph, windowed_machines
    ran = 0
    for seed in range(chunk * 25, chunk * 25 + 25):
        rng = SplitMix64(seed, 97)
        g = _all_addressed(windowed_graph(rng), rng)
        assert window_eligible(g)
        B = rng.randint(1, 8)
        hws = windowed_machines(rng, B)
        for r in hws:
            r[H.FIELDS["l2_lines"]] = rng.choice([0, 0, 1, 3, 16, 100, 4096, 1 << 20])
        flags = ALL | rng.choice([0, 0, api.ORDER_AT_FINISH])
        note(f"window txn seed={seed} N={g.n_nodes} B={B} l2={hws[:, H.FIELDS['l2_lines']].tolist()} flags={flags}")
        gpu, windows = _window_only(torch_cuda, g, hws, flags, monkeypatch)
        st = gpu[2]
        assert not np.any(st == STATUS_RETRY), f"seed {seed}: handed back {np.flatnonzero(st == STATUS_RETRY)}"
        feasible = st != api.SIM_INFEASIBLE
        assert np.all(windows[feasible] > 0), f"seed {seed}: a feasible simulation did not run on the windowed kernel"
        ran += int(feasible.sum())
        _compare(g, hws, flags, gpu)
    assert ran > 0


@pytest.mark.parametrize("variant", ["kn", "kn_pad8", "nk", "bk64"])
def test_window_txn_gemm(torch_cuda, variant, monkeypatch):
    """The four GEMM layouts on the windowed kernel alone, L2s of 0.25-64
    MiB and static flags: no hand-back, equal to the oracle node by node."""
    kw = {"kn": dict(), "kn_pad8": dict(pad=8), "nk": dict(b_layout="nk"), "bk64": dict(BK=64)}[variant]
    BK = kw.pop("BK", 32)
    g = W.gemm_addressed(512, 512, 512, 128, 128, BK, 3, **kw)
    hws = H.sample_h100_sweep(61, 24)
    hws[:, H.FIELDS["l2_lines"]] = [0, 0, 0, 0] + [H.l2_lines(m) for m in (0.25, 1, 2, 4, 8, 16, 32, 64) * 2 + (50,) * 4]
    note(f"window txn gemm {variant} N={g.n_nodes}")
    gpu, windows = _window_only(torch_cuda, g, hws, ALL, monkeypatch)
    assert not np.any(gpu[2] == STATUS_RETRY)
    assert np.all(windows[gpu[2] == 0] > 0)
    _compare(g, hws, ALL, gpu)


def test_window_txn_hands_back(torch_cuda, monkeypatch):
    """An engine above 16 KiB per cycle (more of one node's lines in one
    cycle than a memory batch takes), and NO_CONTENTION (the lines of the
    nodes queued on an SM interleave), are handed to the general kernel,
    which then equals the oracle."""
    rng = SplitMix64(5, 98)
    from windowed import windowed_graph, windowed_machines
    g = _all_addressed(windowed_graph(rng), rng)
    hws = windowed_machines(rng, 4)
    hws[1, H.FIELDS["rate_gmem"]] = (1 << 30) + 1  # 16 KiB per cycle and a little more
    hws[3, H.FIELDS["rate_gmem"]] = 1 << 30        # 16 KiB per cycle: stays
    gpu, _ = _window_only(torch_cuda, g, hws, ALL, monkeypatch)
    assert gpu[2][1] == STATUS_RETRY and gpu[2][3] != STATUS_RETRY
    run_and_compare(torch_cuda, g, hws, ALL)
    gpu, _ = _window_only(torch_cuda, g, hws, ALL | api.NO_CONTENTION, monkeypatch)
    assert np.all(gpu[2] == STATUS_RETRY)
    run_and_compare(torch_cuda, g, hws, ALL | api.NO_CONTENTION)

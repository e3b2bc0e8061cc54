"""GPU parity of the windowed kernel on its own: random graphs it accepts,
shown to have run on it (not handed to the general kernel), bit-exact
against the oracle; the hand-back of a simulation that overflows its queues;
and simulations enqueued on a side stream."""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import workloads as W
from paper_2607_11262_amd.gen.rng import SplitMix64
from windowed import window_eligible, windowed_graph, windowed_machines

pytestmark = pytest.mark.gpu

ALL = api.OUT_NODES | api.OUT_DIGEST
STATUS_RETRY = 0x52455452  # the windowed kernel's internal hand-back marker
STATS_BYTES = 128          # per-simulation counter block at the end of each scratch slice


def note(msg):
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def run_window_only(torch, g, hws, flags, monkeypatch):
    """Records hws through gts_simulate_hwset with only the windowed kernel
    (GTS_KERNEL=window: no general-kernel pass).  Returns the outputs and
    the number of windows each simulation's counter block reports (0 where
    the windowed kernel did not run it)."""
    monkeypatch.setenv("GTS_KERNEL", "window")
    try:
        dg = api.upload(g)
        hs = api.upload_hw(hws)
        B = hws.shape[0]
        stride = api.scratch_bytes(dg, 2, flags) - api.scratch_bytes(dg, 1, flags)
        scratch = torch.zeros(api.scratch_bytes(dg, B, flags), dtype=torch.uint8, device="cuda")
        cyc, mk, st, dgst = api.alloc_outputs(dg, B, flags)
        api.simulate_hwset_into(dg, hs, 0, B, flags, cyc, mk, st, dgst, scratch)
        torch.cuda.synchronize()
        blk = scratch[:B * stride].view(B, stride)[:, stride - STATS_BYTES:].contiguous().view(torch.int64)
        windows = blk[:, 0].cpu().numpy()
    finally:
        monkeypatch.delenv("GTS_KERNEL")
    out = (cyc.cpu().numpy().view(np.uint32) if cyc is not None else None, mk.cpu().numpy().view(np.uint32),
           st.cpu().numpy(), dgst.cpu().numpy().view(np.uint64) if dgst is not None else None)
    return out, windows


def compare(g, hws, flags, gpu, threads=8):
    cyc, mk, st, dg = gpu
    want = bool(flags & api.OUT_NODES)
    omk, ost, odg, ocyc = oracle.simulate_batch(g, hws, flags, want_nodes=want, threads=threads)
    for b in range(hws.shape[0]):
        assert st[b] == ost[b], f"sim {b}: status {st[b]} != oracle {ost[b]}"
        assert mk[b] == omk[b], f"sim {b}: makespan {mk[b]} != oracle {omk[b]}"
        if flags & api.OUT_DIGEST:
            assert dg[b] == odg[b], f"sim {b}: digest differs"
        if want and ost[b] == 0:
            diff = np.flatnonzero(np.any(cyc[b] != ocyc[b], axis=1))
            assert diff.size == 0, f"sim {b}: {diff.size} nodes differ, first {diff[:5]}"


@pytest.mark.parametrize("chunk", range(8))
def test_window_random_graphs(torch_cuda, chunk, monkeypatch):
    """200 random graphs the windowed kernel accepts (memory sinks, edges
    between CTAs from loads / stores into shared nodes, 1-32 warps, 1-4
    kernels, fan-outs above three, zero-work nodes) on machines of 1-256 SMs
    crossing the 64 / 128 / 192-SM lane boundaries, under all four flag
    combinations: each simulation ran on the windowed kernel to the end, and
    every node's cycles equal the oracle's."""
    ran = 0
    for seed in range(chunk * 25, chunk * 25 + 25):
        rng = SplitMix64(seed, 88)
        g = windowed_graph(rng)
        assert window_eligible(g)
        B = rng.randint(1, 8)
        hws = windowed_machines(rng, B)
        flags = ALL | rng.choice([0, api.NO_CONTENTION, api.ORDER_AT_FINISH, api.NO_CONTENTION | api.ORDER_AT_FINISH])
        note(f"window random seed={seed} N={g.n_nodes} E={g.n_edges} B={B} n_sm={hws[:, 0].tolist()} flags={flags}")
        gpu, windows = run_window_only(torch_cuda, g, hws, flags, monkeypatch)
        st = gpu[2]
        assert not np.any(st == STATUS_RETRY), f"seed {seed}: windowed kernel handed back sims {np.flatnonzero(st == STATUS_RETRY)}"
        feasible = st != api.SIM_INFEASIBLE
        assert np.all(windows[feasible] > 0), f"seed {seed}: a feasible simulation did not run on the windowed kernel"
        ran += int(feasible.sum())
        compare(g, hws, flags, gpu)
    assert ran > 0


@pytest.mark.parametrize("waves", [1, 12])
def test_far_list_in_lds_and_in_scratch(torch_cuda, waves, monkeypatch):
    """Per-warp MMA GEMM CTAs (64x64x32 tiles, 3 stages, the decoder layer's
    GEMM shape) release five or eight successors per MMA node, so a lane's
    near list overflows and due entries wait at the front of its far list.
    The same records run with the LDS sized for one simulation per CU (the
    far lists nearly all in LDS) and for twelve (a few entries per lane in
    LDS, the rest in scratch): each simulation ran on the windowed kernel to
    the end, and every node's cycles equal the oracle's, both times."""
    monkeypatch.setenv("GTS_WINDOW_WAVES", str(waves))
    g = W.gemm(2048, 1024, 512, 64, 64, 32, 3, per_warp=True)
    assert window_eligible(g)
    hws = np.stack([H.preset("H100", n_sm=s, max_cta_per_sm=c)
                    for s, c in ((16, 8), (64, 4), (100, 2), (132, 2), (160, 4), (192, 3))])
    note(f"far list waves={waves} N={g.n_nodes} E={g.n_edges} B={hws.shape[0]}")
    gpu, windows = run_window_only(torch_cuda, g, hws, ALL, monkeypatch)
    st = gpu[2]
    assert not np.any(st == STATUS_RETRY), f"windowed kernel handed back sims {np.flatnonzero(st == STATUS_RETRY)}"
    assert np.all(windows > 0)
    compare(g, hws, ALL, gpu)


def _wide_roots_graph(n_loads=150):
    """Two CTAs of 150 independent loads feeding one store: more ready nodes
    on one SM than the windowed kernel's per-lane lists hold."""
    from paper_2607_11262_amd.gen.graph import GLOAD, GSTORE, MISS, GraphBuilder
    b = GraphBuilder()
    b.kernel(4, 0)
    for _ in range(2):
        b.cta()
        loads = [b.node(GLOAD, 256 * (i % 7 + 1), 1, MISS if i % 3 else 0) for i in range(n_loads)]
        st = b.node(GSTORE, 4096, 1, MISS)
        for ld in loads:
            b.edge(ld, st)
    return b.build("wide_roots")


def test_window_hands_back_overflow(torch_cuda, monkeypatch):
    """The wide-roots graph overflows the windowed kernel's ready lists on a
    one-SM machine: run alone, that kernel marks the simulation for the
    general kernel instead of finishing it."""
    g = _wide_roots_graph()
    hws = np.stack([H.preset("H100", n_sm=1, max_cta_per_sm=2)])
    gpu, _ = run_window_only(torch_cuda, g, hws, ALL, monkeypatch)
    assert gpu[2][0] == STATUS_RETRY
    # and through the normal path the general kernel finishes it exactly
    dg = api.upload(g)
    res = api.simulate(dg, hws, ALL)
    torch_cuda.cuda.synchronize()
    compare(g, hws, ALL, api.to_numpy(res))


def _simultaneous_loads_graph():
    from paper_2607_11262_amd.gen.graph import ALU, GLOAD, GSTORE, MISS, GraphBuilder
    b = GraphBuilder()
    b.kernel(4, 0)
    for c in range(512):
        b.cta()
        la = b.node(GLOAD, 1024 * (c % 3 + 1), 0xF, MISS if c % 2 else 0)
        lb = b.node(GLOAD, 2048, 0xF, MISS)
        a = b.node(ALU, 4096, 0xF)
        st = b.node(GSTORE, 512, 0xF, MISS)
        b.edge(la, a)
        b.edge(lb, a)
        b.edge(a, st)
    return b.build("simultaneous_loads")


@pytest.mark.parametrize("name", ["gemm_512", "fa_causal", "decode_small", "decoder_tiny", "simultaneous_loads"])
def test_window_only_finishes(torch_cuda, name, monkeypatch):
    """Workloads and the 512-arrival graph (more memory arrivals at one cycle
    than one window takes) finish on the windowed kernel alone, without a
    hand-back, and equal the oracle."""
    graphs = {
        "gemm_512": lambda: W.gemm(512, 512, 512, 128, 128, 32, 2),
        "fa_causal": lambda: W.flash_attention(1, 4, 1024, 128, 128, 64, causal=True),
        "decode_small": lambda: W.splitkv_decode(batch=6, kv_min=64, kv_max=4096, seed=9),
        "decoder_tiny": lambda: W.decoder_layer(tokens=256, hidden=512, heads=8, kv_heads=2, ffn=1024, d=64),
        "simultaneous_loads": _simultaneous_loads_graph,
    }
    g = graphs[name]()
    if name == "simultaneous_loads":
        hws = np.stack([H.preset("H100", n_sm=n) for n in (256, 255, 200, 129, 64)])
    else:
        hws = H.sample_h100_sweep(41, 16)
    note(f"window only {name} N={g.n_nodes}")
    gpu, windows = run_window_only(torch_cuda, g, hws, ALL, monkeypatch)
    assert not np.any(gpu[2] == STATUS_RETRY)
    assert np.all(windows[gpu[2] == 0] > 0)
    compare(g, hws, ALL, gpu)


def test_side_stream_lifetime(torch_cuda):
    """simulate() on a stream other than the current one: its scratch and
    outputs belong to that stream, so allocations made meanwhile on the
    current stream cannot take their memory while the kernels run."""
    torch = torch_cuda
    g = W.gemm(1024, 1024, 1024, 64, 64, 32, 3)
    hws = H.sample_h100_sweep(5, 64)
    dg = api.upload(g)
    side = torch.cuda.Stream()
    res = api.simulate(dg, hws, ALL, stream=side)
    # churn the current stream's allocator while the side stream runs
    junk = [torch.full((1 << 20,), i, dtype=torch.int64, device="cuda") for i in range(64)]
    del junk
    junk = [torch.full((1 << 22,), -1, dtype=torch.int64, device="cuda") for _ in range(16)]
    side.synchronize()
    torch.cuda.synchronize()
    compare(g, hws, ALL, api.to_numpy(res))
    del junk


def test_server_word_per_class(torch_cuda):
    """The one-server-word-per-class layout (every compute op holds every
    subpartition lane of every record of the batch): a GEMM on warp group
    0-3 takes it for records of at most four subpartitions; adding a record
    of eight turns it off for the whole batch.  Both batches give the same
    cycles for the shared records, equal to the oracle node by node."""
    g = W.gemm(1024, 1024, 512, 128, 128, 32, 3)
    base = H.sample_h100_sweep(77, 12)
    base[:, H.FIELDS["n_subpart"]] = [1, 2, 3, 4] * 3
    eight = H.preset("H100", n_sm=132)
    eight[H.FIELDS["n_subpart"]] = 8
    mixed = np.concatenate([base, eight[None, :]])
    dg = api.upload(g)
    a = api.to_numpy(api.simulate(dg, base, ALL))
    b = api.to_numpy(api.simulate(dg, mixed, ALL))
    torch_cuda.cuda.synchronize()
    n = base.shape[0]
    assert np.array_equal(a[0], b[0][:n]) and np.array_equal(a[1], b[1][:n]) and np.array_equal(a[3], b[3][:n])
    compare(g, mixed, ALL, b)

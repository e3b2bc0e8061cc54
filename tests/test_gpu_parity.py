"""GPU parity: the HIP path (through the C ABI) against the CPU oracle,
element by element, on the same seeded inputs.  Integer cycles, so the bar
is bit-exact: every (start, finish), makespan, status and digest."""
import sys

import numpy as np
import pytest

import oracle
import refcheck
from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import workloads as W
from paper_2607_11262_amd.gen.graph import empty_graph
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


def run_gpu(torch, g, hws, flags=ALL):
    dg = api.upload(g)
    res = api.simulate(dg, hws, flags)
    torch.cuda.synchronize()
    return api.to_numpy(res)


def compare(g, hws, flags, gpu, sims=None, nodes=True, threads=8):
    cyc, mk, st, dg = gpu
    B = hws.shape[0]
    sims = range(B) if sims is None else sims
    sims = list(sims)
    want = bool(nodes and (flags & api.OUT_NODES))
    omk, ost, odg, ocyc = oracle.simulate_batch(g, hws[sims], flags & ~api.OUT_NODES | (api.OUT_NODES if want else 0),
                                                want_nodes=want, threads=threads)
    for i, b in enumerate(sims):
        assert st[b] == ost[i], f"sim {b}: status {st[b]} != oracle {ost[i]}"
        assert mk[b] == omk[i], f"sim {b}: makespan {mk[b]} != oracle {omk[i]}"
        if flags & api.OUT_DIGEST:
            assert dg[b] == odg[i], f"sim {b}: digest differs"
        if want and ost[i] == 0:
            diff = np.flatnonzero(np.any(cyc[b] != ocyc[i], axis=1))
            assert diff.size == 0, f"sim {b}: {diff.size} nodes differ, first {diff[:5]}"


def test_golden_cases(torch_cuda):
    for case, g, rec in refcheck.load_golden():
        note(case["name"])
        gpu = run_gpu(torch_cuda, g, rec[None, :], ALL | case["flags"])
        cyc, mk, st, dg = gpu
        exp = case["expect"]
        assert st[0] == exp["status"] and mk[0] == exp["makespan"], case["name"]
        if "cycles" in exp:
            assert cyc[0].tolist() == exp["cycles"], case["name"]
        compare(g, rec[None, :], ALL | case["flags"], gpu)


@pytest.mark.parametrize("chunk", range(6))
def test_random_graphs(torch_cuda, chunk):
    for seed in range(chunk * 25, chunk * 25 + 25):
        rng = SplitMix64(seed, 21)
        g = W.random_graph(rng, n_nodes_max=rng.choice([5, 20, 80, 300]), n_kernels_max=3, ctas_max=6)
        B = rng.randint(1, 9)
        hws = np.stack([H.sample_random(rng, n_sm_max=rng.choice([1, 3, 70, 200])) for _ in range(B)])
        flags = ALL | rng.choice([0, 0, 4, 8, 12])
        note(f"random seed={seed} N={g.n_nodes} B={B} flags={flags}")
        compare(g, hws, flags, run_gpu(torch_cuda, g, hws, flags))


def _small_workloads():
    return [
        ("gemm_512", W.gemm(512, 512, 512, 128, 128, 32, 2)),
        ("gemm_perwarp", W.gemm(256, 256, 512, 64, 64, 32, 3, per_warp=True)),
        ("fa_small", W.flash_attention(1, 4, 1024, 128, 128, 64)),
        ("fa_causal", W.flash_attention(1, 4, 1024, 128, 128, 64, causal=True)),
        ("decode_small", W.splitkv_decode(batch=6, kv_min=64, kv_max=4096, seed=9)),
        ("decoder_tiny", W.decoder_layer(tokens=256, hidden=512, heads=8, kv_heads=2, ffn=1024, d=64)),
    ]


@pytest.mark.parametrize("name", [n for n, _ in _small_workloads()])
def test_small_workloads(torch_cuda, name):
    g = dict(_small_workloads())[name]
    hws = H.sample_h100_sweep(31, 24)
    for flags in (ALL, ALL | api.NO_CONTENTION):
        note(f"{name} N={g.n_nodes} flags={flags}")
        compare(g, hws, flags, run_gpu(torch_cuda, g, hws, flags))


def test_gemm_1024_full(torch_cuda):
    g = W.workload_graph("gemm_1024_a100")
    hws = W.workload_hw("gemm_1024_a100")
    note(f"gemm 1024 N={g.n_nodes} B={hws.shape[0]}")
    compare(g, hws, ALL, run_gpu(torch_cuda, g, hws, ALL))


def test_splitkv_decode_full(torch_cuda):
    g = W.workload_graph("splitkv_decode_b64")
    hws = W.workload_hw("splitkv_decode_b64")
    note(f"split-KV decode N={g.n_nodes} B={hws.shape[0]}")
    gpu = run_gpu(torch_cuda, g, hws, ALL)
    compare(g, hws, ALL, gpu, sims=range(0, 1024, 64), nodes=True)      # per node, 16 sampled sims
    compare(g, hws, ALL, gpu, sims=range(1, 1024, 8), nodes=False)      # makespan/digest/status


def test_gemm_design_sweep_sample(torch_cuda):
    ps = W.sweep_params()
    idx = sorted(range(64), key=lambda i: W.sweep_nodes(ps[i]))[:4]
    for i in idx:
        g = W.sweep_graph(ps[i])
        hws = W.workload_hw("gemm_design_sweep", B=256, index=i)
        note(f"design sweep graph {i} {ps[i]} N={g.n_nodes} B=256")
        gpu = run_gpu(torch_cuda, g, hws, ALL)
        compare(g, hws, ALL, gpu, sims=range(0, 256, 4), nodes=True)


def test_empty_graph_and_zero_batch(torch_cuda):
    g = empty_graph()
    hws = H.sample_h100_sweep(3, 4)
    cyc, mk, st, dg = run_gpu(torch_cuda, g, hws, ALL)
    assert st.tolist() == [0] * 4 and mk.tolist() == [0] * 4 and dg.tolist() == [0] * 4
    dgr = api.upload(W.workload_graph("gemm_1024_a100"))
    res = api.simulate(dgr, np.zeros((0, 32), np.uint32), ALL)
    torch_cuda.cuda.synchronize()
    assert res.makespan.numel() == 0


def test_determinism_permutation_split(torch_cuda):
    g = W.gemm(512, 256, 1024, 64, 128, 64, 4)
    hws = H.sample_h100_sweep(77, 40)
    note("determinism")
    a = run_gpu(torch_cuda, g, hws, ALL)
    b = run_gpu(torch_cuda, g, hws, ALL)
    perm = np.random.default_rng(5).permutation(40)
    c = run_gpu(torch_cuda, g, hws[perm], ALL)
    d1 = run_gpu(torch_cuda, g, hws[:13], ALL)
    d2 = run_gpu(torch_cuda, g, hws[13:], ALL)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    for x, y in zip(a, c):
        assert np.array_equal(x[perm], y)
    for x, y1, y2 in zip(a, d1, d2):
        assert np.array_equal(x, np.concatenate([y1, y2]))


def _wide_roots_graph(n_loads=150):
    """One CTA whose 150 independent loads are all ready at launch, feeding
    one store: more ready nodes on one SM than the windowed kernel queues,
    so the simulation is handed to the general kernel."""
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


def test_queue_overflow_falls_back(torch_cuda):
    g = _wide_roots_graph()
    hws = H.sample_h100_sweep(12, 6)
    note("wide roots fallback")
    compare(g, hws, ALL, run_gpu(torch_cuda, g, hws, ALL))


@pytest.mark.parametrize("name", ["gemm_512", "fa_causal", "decode_small", "decoder_tiny"])
def test_windowed_equals_general(torch_cuda, name, monkeypatch):
    """The same batch through the windowed kernel and through the general
    kernel gives identical results (both are also checked against the
    oracle above)."""
    g = dict(_small_workloads())[name]
    hws = H.sample_h100_sweep(41, 16)
    a = run_gpu(torch_cuda, g, hws, ALL)
    monkeypatch.setenv("GTS_KERNEL", "general")
    b = run_gpu(torch_cuda, g, hws, ALL)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_digest_only_mode_matches(torch_cuda):
    g = W.gemm(512, 512, 256, 128, 64, 32, 3)
    hws = H.sample_h100_sweep(8, 32)
    a = run_gpu(torch_cuda, g, hws, ALL)
    b = run_gpu(torch_cuda, g, hws, api.OUT_DIGEST)
    assert np.array_equal(a[1], b[1]) and np.array_equal(a[3], b[3]) and np.array_equal(a[2], b[2])


def test_gemm_design_sweep_bench_launch(torch_cuda):
    """The bench's launch shape: one sweep graph against its 4096 resident
    hardware records in one launch (digest outputs), sampled against the
    oracle; per-node cycles on two of the records."""
    ps = W.sweep_params()
    for gi in (0, 7):
        g = W.sweep_graph(ps[gi])
        hws = W.workload_hw("gemm_design_sweep", B=4096, index=gi)
        note(f"design sweep bench launch graph {gi} N={g.n_nodes} B=4096")
        dg = api.upload(g)
        hs = api.upload_hw(hws)
        flags = api.OUT_DIGEST
        scratch = torch_cuda.empty(api.scratch_bytes(dg, 4096, flags), dtype=torch_cuda.uint8, device="cuda")
        cyc, mk, st, dgst = api.alloc_outputs(dg, 4096, flags)
        api.simulate_hwset_into(dg, hs, 0, 4096, flags, None, mk, st, dgst, scratch)
        torch_cuda.cuda.synchronize()
        gpu = (None, mk.cpu().numpy().view(np.uint32), st.cpu().numpy(), dgst.cpu().numpy().view(np.uint64))
        compare(g, hws, flags, gpu, sims=list(range(0, 4096, 128)) + [4095], nodes=False)
        sub = hws[[1, 4094]]
        compare(g, sub, ALL, run_gpu(torch_cuda, g, sub, ALL))


def test_flash_attention_full(torch_cuda):
    """FlashAttention forward, 2.6M nodes, all 256 records in one launch:
    every record against the oracle (makespan, status, digest), per-node
    cycles on three."""
    g = W.workload_graph("flash_attention_b8_h32_s4096")
    hws = W.workload_hw("flash_attention_b8_h32_s4096")
    note(f"flash attention N={g.n_nodes} B={hws.shape[0]}")
    gpu = run_gpu(torch_cuda, g, hws, api.OUT_DIGEST)
    compare(g, hws, api.OUT_DIGEST, gpu, threads=16)
    sub = hws[[3, 128, 255]]
    compare(g, sub, ALL, run_gpu(torch_cuda, g, sub, ALL))


def test_splitkv_decode_digest_all(torch_cuda):
    """Split-KV decode: every one of the 1024 records, digest and makespan."""
    g = W.workload_graph("splitkv_decode_b64")
    hws = W.workload_hw("splitkv_decode_b64")
    note(f"split-KV decode N={g.n_nodes} B={hws.shape[0]} (all)")
    gpu = run_gpu(torch_cuda, g, hws, api.OUT_DIGEST)
    compare(g, hws, api.OUT_DIGEST, gpu, threads=16)


def test_decoder_layer_full(torch_cuda):
    """Decoder layer, 20.5M nodes over nine kernels, all 64 records in one
    launch, every record against the oracle; per-node cycles on two."""
    g = W.workload_graph("decoder_layer_prefill_2048")
    hws = W.workload_hw("decoder_layer_prefill_2048")
    note(f"decoder layer N={g.n_nodes} B={hws.shape[0]}")
    gpu = run_gpu(torch_cuda, g, hws, api.OUT_DIGEST)
    compare(g, hws, api.OUT_DIGEST, gpu, threads=16)
    sub = hws[[5, 63]]
    compare(g, sub, ALL, run_gpu(torch_cuda, g, sub, ALL))


@pytest.mark.parametrize("nsub", [1, 4])
def test_sm_count_boundaries(torch_cuda, nsub):
    """Machines at the SM counts where the windowed kernel changes how many
    SMs a lane carries (64, 128, 192, 256 SMs), past its 256-SM limit (the
    general kernel takes those), up to the record's 1024-SM maximum, in one
    batch and each alone: bit-exact against the oracle."""
    counts = [1, 63, 64, 65, 128, 129, 192, 255, 256, 257, 511, 1024]
    hws = np.stack([H.preset("H100", n_sm=n, n_subpart=nsub) for n in counts])
    graphs = (("gemm", W.gemm(2048, 2048, 512, 128, 128, 32, 3)),
              ("decoder_tiny", W.decoder_layer(tokens=256, hidden=512, heads=8, kv_heads=2, ffn=1024, d=64)))
    for name, g in graphs:
        note(f"{name} N={g.n_nodes} n_sub={nsub} n_sm={counts}")
        compare(g, hws, ALL, run_gpu(torch_cuda, g, hws))
        for i in (2, 8, 9, 11):  # alone: the launch picks its kernel from this record's SM count
            compare(g, hws[i:i + 1], ALL, run_gpu(torch_cuda, g, hws[i:i + 1]))


def test_largest_records(torch_cuda):
    """1024 SMs x 8 subpartitions (the record's maxima) on a graph that uses
    all three compute classes: the general kernel's per-SM servers then take
    108 KiB of LDS.  Either bit-exact against the oracle, or -- on a device
    whose workgroups hold less -- a GTS_E_HW error before any kernel runs."""
    g = W.decoder_layer(tokens=256, hidden=512, heads=8, kv_heads=2, ffn=1024, d=64)
    hws = np.stack([H.preset("H100", n_sm=1024, n_subpart=8), H.preset("H100", n_sm=1000, n_subpart=7)])
    note(f"decoder_tiny N={g.n_nodes} n_sm=1024/1000 n_sub=8/7")
    try:
        gpu = run_gpu(torch_cuda, g, hws)
    except api.GtsError as e:
        assert e.code == -5 and "LDS" in str(e), str(e)
        note(f"refused: {e}")
        return
    compare(g, hws, ALL, gpu)


def test_simultaneous_arrivals_split(torch_cuda):
    """Every SM's CTA starts with loads issued at one cycle: with 256 SMs
    that is up to 512 memory arrivals of a single cycle, more than one
    window of the windowed kernel takes, so the window boundary falls
    between the keys of one cycle.  Bit-exact against the oracle."""
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
    g = b.build("simultaneous_loads")
    hws = np.stack([H.preset("H100", n_sm=n) for n in (256, 255, 200, 129, 64)])
    note(f"simultaneous arrivals N={g.n_nodes}")
    compare(g, hws, ALL, run_gpu(torch_cuda, g, hws, ALL))

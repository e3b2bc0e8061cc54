"""GPU parity with template sharing (Sec. 6.4): graphs whose kernels replicate
one random CTA graph over many CTAs in a few op classes (with wide fan-outs,
all edge kinds, and a kernel with a cross-CTA edge that keeps expanded
records) run bit-exact against the oracle, and identically with sharing
turned off at upload."""
import numpy as np
import pytest

from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import workloads as W
from paper_2607_11262_amd.gen.rng import SplitMix64
from templated import templated_graph
from test_gpu_parity import ALL, compare, note

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _run(torch, g, hws, flags):
    res = api.simulate(api.upload(g), hws, flags)
    torch.cuda.synchronize()
    return api.to_numpy(res)


def _same(a, b):
    for x, y in zip(a, b):
        assert (x is None) == (y is None)
        if x is not None:
            assert np.array_equal(x, y)


@pytest.mark.parametrize("chunk", range(4))
def test_templated_random_graphs(torch_cuda, chunk, monkeypatch):
    for seed in range(chunk * 10, chunk * 10 + 10):
        rng = SplitMix64(seed, 90)
        g = templated_graph(rng, n_kernels=rng.randint(1, 4), n_ctas=(2, 60),
                            cross_kernel=rng.choice([None, None, 0, 1]))
        B = rng.randint(1, 6)
        hws = np.stack([H.sample_random(rng, n_sm_max=rng.choice([1, 4, 70, 200])) for _ in range(B)])
        flags = ALL | rng.choice([0, 0, 4, 8])
        note(f"templated seed={seed} N={g.n_nodes} K={g.n_kernels} {api.templates(g)} B={B} flags={flags}")
        on = _run(torch_cuda, g, hws, flags)
        compare(g, hws, flags, on)
        monkeypatch.setenv("GTS_TEMPLATES", "0")
        off = _run(torch_cuda, g, hws, flags)
        monkeypatch.delenv("GTS_TEMPLATES")
        _same(on, off)


def test_templated_workload_graphs_on_off(torch_cuda, monkeypatch):
    # GEMM (one template, 4 classes), flash attention, and the decoder layer
    # (8 of 9 kernels shared, attention expanded), on sweep machines
    hws = W.workload_hw("gemm_design_sweep", B=6, index=3)
    for name, g in (("gemm 2048x2048x1024", W.gemm(2048, 2048, 1024, 128, 128, 64, 3)),
                    ("attention", W.workload_graph("flash_attention_b8_h32_s4096")), ("decoder layer", W.workload_graph("decoder_layer_prefill_2048"))):
        note(f"{name} N={g.n_nodes} {api.templates(g)}")
        on = _run(torch_cuda, g, hws, api.OUT_DIGEST)
        monkeypatch.setenv("GTS_TEMPLATES", "0")
        off = _run(torch_cuda, g, hws, api.OUT_DIGEST)
        monkeypatch.delenv("GTS_TEMPLATES")
        _same(on, off)
        assert np.all(on[2] == 0)

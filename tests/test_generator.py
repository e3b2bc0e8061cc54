"""Seeded workload generators: structure, counts, validity, reproducibility."""
import numpy as np
import pytest

from paper_2607_11262_amd.gen import hw as H
from paper_2607_11262_amd.gen import workloads as W
from paper_2607_11262_amd.gen.graph import (GLOAD, GSTORE, MISS, TENSOR, ValidationError, GraphBuilder,
                                             empty_graph, validate)


def test_gemm_1024_counts():
    g = W.workload_graph("gemm_1024_a100")
    validate(g)
    assert g.n_nodes == 64 * (32 * 3 + 1) == 6208
    assert g.n_ctas == 64 and g.n_kernels == 1
    assert int(g.kernel_smem[0]) == 2 * (128 + 128) * 32 * 2
    # first-touch L2 misses: A panels in CTA column 0, B panels in CTA row 0
    cls = g.op_cls[g.node_op]
    miss = (g.op_flags[g.node_op] & MISS) != 0
    loads = cls == GLOAD
    assert int((loads & miss).sum()) == (8 + 8) * 32
    assert int((cls == GSTORE).sum()) == 64
    assert int((cls == TENSOR).sum()) == 64 * 32


def test_flash_attention_counts():
    g = W.workload_graph("flash_attention_b8_h32_s4096")
    assert g.n_ctas == 8 * 32 * 32
    assert g.n_nodes == 8192 * 322 == 2_637_824
    c = W.flash_attention(1, 2, 1024, 128, 128, 64)
    validate(c)
    assert c.n_nodes == 2 * 8 * (1 + 16 * 5 + 1)


def test_decoder_counts_formula():
    """Decoder-layer node count from the template formula (the full graph is
    generated in the GPU tests): GEMMs with 64x64x32 tiles and 6 nodes per
    k-step, causal attention with 2(i+1) KV tiles for query block i."""
    def gemm_nodes(M, N, K):
        return (M // 64) * (N // 64) * (6 * (K // 32) + 1)

    total = (gemm_nodes(2048, 6144, 4096) + gemm_nodes(2048, 4096, 4096) + gemm_nodes(2048, 28672, 4096)
             + gemm_nodes(2048, 4096, 14336))
    total += 32 * sum(1 + 5 * 2 * (i + 1) + 1 for i in range(16))
    total += 128 * (4 + 3 + 4 + 4)
    assert total == 20_515_200
    small = W.decoder_layer(tokens=128, hidden=256, heads=4, kv_heads=2, ffn=512, d=64)
    validate(small)
    assert small.n_kernels == 9


def test_splitkv_structure():
    g = W.splitkv_decode(batch=4, kv_min=64, kv_max=4096, seed=3)
    validate(g)
    lens = g.meta["kv_lens"]
    assert all(l % 64 == 0 and 64 <= l <= 4096 + 63 for l in lens)
    splits = sum(-(-(l // 64) // 4) for l in lens) * 8
    assert g.n_ctas == splits + 4 * 8
    # every reduction CTA receives one cross-CTA edge per split
    cta = g.node_cta()
    src, dst = g.sources(), g.targets()
    cross = cta[src] != cta[dst]
    assert int(cross.sum()) == splits


def test_sweep_params_and_sizes():
    ps = W.sweep_params()
    assert len(ps) == 64
    for M, N, K, BM, BN, BK, S in ps:
        assert M in W.SWEEP_MNK and N in W.SWEEP_MNK and K in W.SWEEP_MNK
        assert BM in W.SWEEP_BMN and BN in W.SWEEP_BMN and BK in W.SWEEP_BK and S in W.SWEEP_STAGES
    assert ps == W.sweep_params()
    small = min(ps, key=W.sweep_nodes)
    g = W.sweep_graph(small)
    validate(g)
    assert g.n_nodes == W.sweep_nodes(small)


def test_reproducible_digests():
    a = W.splitkv_decode(batch=5, seed=11)
    b = W.splitkv_decode(batch=5, seed=11)
    c = W.splitkv_decode(batch=5, seed=12)
    assert a.digest() == b.digest() != c.digest()
    assert W.workload_graph("gemm_1024_a100").digest() == W.workload_graph("gemm_1024_a100").digest()
    assert np.array_equal(W.workload_hw("flash_attention_b8_h32_s4096", B=8), W.workload_hw("flash_attention_b8_h32_s4096", B=8))
    assert not np.array_equal(W.workload_hw("gemm_design_sweep", B=8, index=0), W.workload_hw("gemm_design_sweep", B=8, index=1))


def test_hw_presets_table3():
    a = H.preset("A100")
    h = H.preset("H100")
    assert H.get(a, "n_sm") == 108 and H.get(h, "n_sm") == 132
    assert H.get(a, "rate_dram") == 65_396_561  # 1407 GB/s at 1410 MHz
    assert H.get(h, "rate_dram") == 102_606_868  # 3100 GB/s at 1980 MHz
    assert H.get(h, "rate_tensor") == 4096 << 16  # 2 x 2048 FMA/clk
    assert H.get(h, "rate_gmem") == 100 << 16 and H.get(a, "rate_gmem") == 128 << 16
    assert H.get(h, "lat_l2") == 380 and H.get(a, "lat_dram") == 250
    s = H.sample_h100_sweep(5, 100)
    assert s[:, 0].min() >= 64 and s[:, 0].max() <= 192


def test_validation_rejects():
    b = GraphBuilder()
    b.kernel(4, 0)
    b.cta()
    x = b.node(TENSOR, 10, 1)
    y = b.node(TENSOR, 10, 1)
    b.edge(x, y)
    b.edge(y, x)
    with pytest.raises(ValidationError):
        validate(b.build())
    b = GraphBuilder()
    b.kernel(2, 0)
    b.cta()
    b.node(TENSOR, 10, 0b100)  # warp 2 of a 2-warp CTA
    with pytest.raises(ValidationError):
        validate(b.build())
    validate(empty_graph())


def test_duplicate_edges_merge_to_strongest():
    b = GraphBuilder()
    b.kernel(1, 0)
    b.cta()
    x = b.node(TENSOR, 10, 1)
    y = b.node(TENSOR, 10, 1)
    b.edge(x, y, 1)
    b.edge(x, y, 0)
    g = b.build()
    assert g.n_edges == 1 and int(g.kinds()[0]) == 0

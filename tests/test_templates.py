"""Template sharing of isomorphic CTA graphs (Sec. 6.4), host side: which
kernels the upload shares, the class x slot op table and its limits, and the
opt-out.  Needs no GPU."""
import numpy as np
import pytest

from paper_2607_11262_amd import api
from paper_2607_11262_amd.gen import workloads as W
from paper_2607_11262_amd.gen.graph import DATA, GLOAD, GSTORE, TENSOR, GraphBuilder
from paper_2607_11262_amd.gen.rng import SplitMix64
from templated import templated_graph


def test_gemm_is_one_template():
    # 1024^3 GEMM, 128x128x32 tiles, 2 stages: 64 CTAs of 97 nodes; first-touch
    # CTAs use L2-miss loads, so the CTAs fall into 4 classes (A and B panel
    # first touched or not) over 4 op slots (load A, load B, MMA, store)
    g = W.gemm(1024, 1024, 1024, 128, 128, 32, 2)
    assert g.n_ctas == 64 and g.n_nodes == 64 * 97
    t = api.templates(g)
    assert t == {"templated_kernels": 1, "template_nodes": 97, "expanded_nodes": 0, "class_ops": 16}


def test_logical_to_physical_ratio():
    """Sec. 6.4 (graph construction): 88.58K physical nodes stand for 45.35M
    logical ones and 11.52K for 0.09M (92.16K).  Both ratios, 512 and 8, are
    the CTA counts of the square GEMMs 4096^3 and 512^3 with 128 x 256 CTA
    tiles (32 x 16 and 4 x 2 CTAs), the shapes of the paper's evaluated
    range: with one template per kernel, logical / physical nodes is the
    number of CTAs that share it."""
    assert round(45.35e6 / 88.58e3) == 512 and round(92.16e3 / 11.52e3) == 8
    big = W.gemm(4096, 4096, 4096, 128, 256, 64, 3)
    small = W.gemm(512, 512, 512, 128, 256, 64, 3)
    rb, rs = (g.n_nodes / api.templates(g)["template_nodes"] for g in (big, small))
    assert rb == 512 and rs == 8
    for g in (big, small):
        t = api.templates(g)
        assert t["templated_kernels"] == 1 and t["expanded_nodes"] == 0
    # and it grows with the GEMM the same way at other shapes
    assert W.gemm(8192, 8192, 1024, 128, 128, 32, 2).n_nodes / api.templates(
        W.gemm(8192, 8192, 1024, 128, 128, 32, 2))["template_nodes"] == 4096


def test_decoder_layer_kernels():
    g = W.workload_graph("decoder_layer_prefill_2048")
    t = api.templates(g)
    # the attention kernel (causal: CTAs of different lengths) stays expanded
    assert t["templated_kernels"] == g.n_kernels - 1
    assert t["class_ops"] <= 128
    assert t["template_nodes"] + t["expanded_nodes"] < g.n_nodes / 100


def expected_sharing(g, max_tops=128):
    """The sharing rule written out directly: a kernel with at least two CTAs
    of one node count, identical local successor lists (targets relative to
    the CTA, kinds) and no edge leaving or entering a CTA is shared, kernels
    in order, while its classes (distinct op vectors, at most 255) times its
    slots (distinct op columns across classes) fit in what is left of the
    table."""
    ptr = g.succ_ptr.astype(np.int64)
    tgt = (g.succ & 0x3FFFFFFF).astype(np.int64)
    kind = (g.succ >> 30).astype(np.int64)
    nb = g.cta_node_begin.astype(np.int64)
    src = np.repeat(np.arange(g.n_nodes), np.diff(ptr))
    cta_of = np.searchsorted(nb, np.arange(g.n_nodes), side="right") - 1
    used, nk, tnodes, expanded = 0, 0, 0, 0
    for k in range(g.n_kernels):
        c0, c1 = int(g.kernel_cta_begin[k]), int(g.kernel_cta_begin[k + 1])
        n = int(nb[c0 + 1] - nb[c0])
        ok = c1 - c0 >= 2 and all(int(nb[c + 1] - nb[c]) == n for c in range(c0, c1))
        shape, vecs = None, []
        for c in range(c0, c1 if ok else c0):
            local = []
            for i in range(n):
                u = int(nb[c]) + i
                local.append(tuple((int(t - nb[c]), int(kd))
                                   for t, kd in zip(tgt[ptr[u]:ptr[u + 1]], kind[ptr[u]:ptr[u + 1]])))
            if any(not (0 <= t < n) for row in local for t, _ in row):
                ok = False
            if shape is None:
                shape = local
            ok = ok and local == shape
            vecs.append(tuple(int(x) for x in g.node_op[nb[c]:nb[c] + n]))
        if ok:  # no edge from another CTA into the kernel's nodes
            into = (cta_of[tgt] != cta_of[src]) & (tgt >= nb[c0]) & (tgt < nb[c1])
            ok = not into.any()
        classes = list(dict.fromkeys(vecs))
        slots = len({tuple(v[i] for v in classes) for i in range(n)}) if ok else 0
        if ok and len(classes) <= 255 and used + len(classes) * slots <= max_tops:
            used += len(classes) * slots
            nk += 1
            tnodes += n
        else:
            expanded += int(nb[c1] - nb[c0])
    return {"templated_kernels": nk, "template_nodes": tnodes, "expanded_nodes": expanded, "class_ops": used}


def test_random_templated_graphs_match_the_rule():
    shared = 0
    for seed in range(40):
        rng = SplitMix64(seed, 78)
        g = templated_graph(rng, n_kernels=rng.randint(1, 4), cross_kernel=rng.choice([None, 0, 1]))
        api.validate(g)
        want = expected_sharing(g)
        assert api.templates(g) == want, seed
        shared += want["templated_kernels"]
    assert shared >= 20  # the draws do exercise sharing


def test_variable_cta_sizes_and_cross_cta_edges_are_not_shared():
    assert api.templates(W.workload_graph("splitkv_decode_b64"))["templated_kernels"] == 0  # split-KV decode
    for seed in range(10):
        rng = SplitMix64(seed, 77)
        g = templated_graph(rng, n_kernels=2, n_local=(4, 8), cross_kernel=1)
        t = api.templates(g)
        n1 = int(g.cta_node_begin[g.kernel_cta_begin[2]] - g.cta_node_begin[g.kernel_cta_begin[1]])
        assert t["expanded_nodes"] >= n1 and t == expected_sharing(g)


def _one_kernel(n_ctas, perturb=None, unique_ops=False):
    b = GraphBuilder()
    b.kernel(4, 0)
    for c in range(n_ctas):
        b.cta()
        w = 1000 + c if unique_ops else 1000
        a = b.node(GLOAD, w, 0xF)
        m = b.node(TENSOR, 4096, 0xF)
        s = b.node(GSTORE, 512, 0xF)
        b.edge(a, m, DATA)
        b.edge(m, s, DATA)
        if perturb == c:
            b.edge(a, s, DATA)
    return b.build("k")


def test_structure_must_match_exactly():
    assert api.templates(_one_kernel(8))["templated_kernels"] == 1
    assert api.templates(_one_kernel(8, perturb=5))["templated_kernels"] == 0
    assert api.templates(_one_kernel(1))["templated_kernels"] == 0  # nothing to share


def test_class_limits():
    # 100 classes x 3 slots = 300 table entries > 128
    assert api.templates(_one_kernel(100, unique_ops=True))["templated_kernels"] == 0
    t = api.templates(_one_kernel(40, unique_ops=True))  # 40 classes x 3 slots = 120 entries
    assert t["templated_kernels"] == 1 and t["class_ops"] == 120


def test_opt_out_and_image_size(monkeypatch):
    g = W.gemm(1024, 1024, 1024, 128, 128, 32, 2)
    on = api.device_bytes(g)
    monkeypatch.setenv("GTS_TEMPLATES", "0")
    assert api.templates(g)["templated_kernels"] == 0
    off = api.device_bytes(g)
    assert on > off  # the template sections come on top of the expanded records

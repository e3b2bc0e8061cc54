#!/usr/bin/env python3
"""Throughput of the batched tile-graph simulation on one MI355X.

Workload: the GEMM design sweep -- 64 seeded GEMM tile graphs (M, N, K in
{1,2,4,8}K; CTA tiles {64,128,256}^2 x {32,64}; 2-4 pipeline stages; 4 warps)
each simulated under 4096 seeded H100-based hardware configurations (SMs
64-192, DRAM 1.5-8 TB/s, shared memory 96-256 KiB, tensor rate 0.5-4x).
One step = one graph of the sweep against its 4096 configurations
(digest + makespan + status per simulation), step i using sweep graph i mod
64.  Graph images and hardware records are resident in HBM before timing.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Prints one JSON line: simulated tile-nodes per second (value), simulations
per second, the roofline of the simulation kernel (algorithmic bytes per
launch / mean launch time from HIP events, against 8 TB/s HBM) and the CPU
oracle timed on a bounded sample of the same workload on this host.

    python bench.py --workload pipelining

runs the software-pipelining case study instead (Sec. 7.1, Table 4): the
fused GEMM + SiLU persistent kernel in four pipeline organisations x five
tile shapes x four edge-class sets (80 graphs of 270-1020 nodes), each
simulated under 4096 seeded single-SM Hopper machines (tensor rate 0.5-4x,
DRAM 1.5-8 TB/s, TMA 50-200 B/cycle); its line adds the case-study table
(normalised performance and Tensor Core utilisation per organisation at
Table 3's H100 with FP8 rate), read off GPU timelines.

    python bench.py --workload noc

runs the NoC-enabled fusion case study (Sec. 7.2): the cluster-fused
attention block (32 heads, one cluster per head, clusters of 2-16 CTAs,
communication over the SM-cluster NoC or through DRAM; 8 graphs of
12K-61K nodes), each under 4096 seeded H100 machines with a 16-SM-domain
crossbar or 4 x 4 mesh NoC (any of three placements, port bandwidth 8-64
B/cycle, latency 60-400 cycles, DRAM 1.5-8 TB/s, tensor 0.5-4x); its line
adds the case-study table (NoC vs DRAM cycles and mean NoC residence per
topology and placement) read off GPU timelines.

    python bench.py --workload l2lru

runs eight GEMMs of the design sweep (the smallest of 40K-300K nodes) with
tile ids (the LRU L2 of Sec. 5.2), each under 4096 seeded H100 sweep
machines with an L2 of 4-64 MiB; its line adds the kernel cycles of one GEMM across L2 sizes
(static first-touch flags vs LRU) read off the GPU.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
B_PER_GRAPH = 4096


def alg_bytes_per_sim(g) -> int:
    """Bytes one simulation must read from the graph (16-byte node record per
    node, 4 bytes per edge) plus its 16 bytes of per-simulation output."""
    return 16 * g.n_nodes + 4 * g.n_edges + 16


PROFILE = os.path.join(ROOT, "profiles", "gts_sim_window_gemm_design_sweep.md")
KERNEL_SOURCES = ("gts_window.hip", "gts_common.h", "gts_dev.h")


def recorded_traffic(n_launch: int):
    """HBM bytes per launch of the simulation kernel, from the committed
    rocprofv3 counter summary (FETCH_SIZE and WRITE_SIZE summed over the
    timed launches, scaled by the same counters on a plain copy), or None
    when that summary was taken on other kernel sources or other launches."""
    try:
        text = open(PROFILE).read()
    except OSError:
        return None
    m = re.search(r"traffic-record: sha256=(\w+) launches=(\d+) fetch_kib=(\d+) write_kib=(\d+) "
                  r"fetch_factor=([\d.]+) write_factor=([\d.]+)", text)
    if not m:
        return None
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2607_11262_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    if m.group(1) != h.hexdigest() or int(m.group(2)) != n_launch:
        return None
    fetch = int(m.group(3)) * 1024 * float(m.group(5))
    write = int(m.group(4)) * 1024 * float(m.group(6))
    return (fetch + write) / n_launch


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", choices=("gemm_design_sweep", "pipelining", "noc", "l2lru"),
                    default="gemm_design_sweep")
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="bounded CPU-oracle sample length")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mem-budget-gb", type=float, default=220.0,
                    help="device scratch budget, split evenly over the streams")
    ap.add_argument("--graphs", type=str, default="", help="comma-separated sweep graph indices (default: step order)")
    ap.add_argument("--streams", type=int, default=2,
                    help="consecutive launches alternate over this many HIP streams, so one launch "
                         "overlaps the tail of the previous one")
    ap.add_argument("--launch-log", type=str, default="", help="write one JSON line per timed launch to this file")
    ap.add_argument("--host-io", action="store_true",
                    help="after the timed region, time the same steps through host buffers: hardware records "
                         "passed from host memory per call (gts_simulate_batch) and results copied back, then "
                         "also with each step's graph uploaded from host arrays")
    ap.add_argument("--phase-stats", action="store_true",
                    help="after the timed region, report the windowed kernel's per-phase counters per graph")
    ap.add_argument("--calibrate-copy-gib", type=float, default=0.0,
                    help="only run a plain device-to-device copy of this many GiB (HBM counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); simulations are independent, "
              "so a multi-GPU run would shard the batch across GPUs.", file=sys.stderr)
        return 2

    import torch

    from paper_2607_11262_amd import api
    from paper_2607_11262_amd.gen import clusterfusion as CF
    from paper_2607_11262_amd.gen import pipelining as PL
    from paper_2607_11262_amd.gen import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    if args.calibrate_copy_gib > 0:
        n = int(args.calibrate_copy_gib * (1 << 30))
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read": n, "bytes_written": n, "launches": 3}))
        return 0
    api.lib()  # fails loudly if libgts.so is missing
    dev = torch.device("cuda:0")
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(max(1, args.streams) - 1)]

    pipelining = args.workload == "pipelining"
    noc = args.workload == "noc"
    lru = args.workload == "l2lru"
    noc_graphs = [(S, comm) for S in CF.CLUSTER_SIZES for comm in CF.COMMS]
    if lru:
        all_params = W.sweep_params()
        lru_params = [q for q in sorted(all_params, key=W.sweep_nodes) if 40_000 <= W.sweep_nodes(q) <= 300_000][:8]
        n_graphs = len(lru_params)

        def make(gi):
            g = W.gemm(*lru_params[gi], tiles=True)
            hw = W.workload_hw("gemm_design_sweep", B=B_PER_GRAPH, index=gi)
            rng = np.random.default_rng(5000 + gi)
            hw[:, 26] = (rng.integers(4, 65, size=B_PER_GRAPH) * (1 << 20)) // 128  # L2 lines, 4-64 MiB
            return g, hw

        def describe(gi):
            return lru_params[gi]
    elif noc:
        n_graphs = len(noc_graphs)

        def make(gi):
            return CF.cluster_attention(noc_graphs[gi][0], comm=noc_graphs[gi][1]), CF.sample_noc_machines(gi, B_PER_GRAPH)

        def describe(gi):
            return noc_graphs[gi]
    elif pipelining:
        n_graphs = len(PL.case_study_graphs())

        def make(gi):
            return PL.case_study_graph(gi), PL.sample_hopper_1sm(gi, B_PER_GRAPH)

        def describe(gi):
            return PL.case_study_graphs()[gi]
    else:
        params = W.sweep_params()
        n_graphs = len(params)

        def make(gi):
            return W.sweep_graph(params[gi]), W.workload_hw("gemm_design_sweep", B=B_PER_GRAPH, index=gi)

        def describe(gi):
            return params[gi]
    if args.graphs:
        order = [int(x) for x in args.graphs.split(",")]
    else:
        order = list(range(n_graphs))
    step_graphs = [order[i % len(order)] for i in range(args.steps)]
    warm_graphs = [order[i % len(order)] for i in range(args.warmup)]
    needed = sorted(set(step_graphs) | set(warm_graphs))

    flags = api.OUT_DIGEST
    t_gen = time.time()
    prepared = {}
    host_graphs = {}
    budget = int(args.mem_budget_gb * (1 << 30)) // max(1, args.streams)
    max_scratch = 0
    for gi in needed:
        g, hw = make(gi)
        dg = api.upload(g)
        hs = api.upload_hw(hw)
        per_sim = api.scratch_bytes(dg, 1, flags) - api.scratch_bytes(dg, 0, flags)
        # launches of equal size (a short tail launch would cost a whole
        # simulation's latency for a few waves)
        most = max(1, min(B_PER_GRAPH, budget // max(per_sim, 1)))
        n_launch = -(-B_PER_GRAPH // most)
        chunk = -(-B_PER_GRAPH // n_launch)
        max_scratch = max(max_scratch, api.scratch_bytes(dg, chunk, flags))
        outs = api.alloc_outputs(dg, B_PER_GRAPH, flags, dev)
        prepared[gi] = (dg, hs, chunk, outs, g.n_nodes, alg_bytes_per_sim(g))
        host_graphs[gi] = (g, hw)
        print(f"[bench] graph {gi} {describe(gi)} N={g.n_nodes} E={g.n_edges} chunk={chunk}", file=sys.stderr,
              flush=True)
    t_gen = time.time() - t_gen
    # one scratch area per stream; each graph's outputs are its own
    scratches = [torch.empty(max_scratch, dtype=torch.uint8, device=dev) for _ in streams]
    launches = []  # (start event, end event, algorithmic bytes, node-sims)
    launch_info = []  # (graph, first record, records)

    n_launched = [0]

    def step(k, gi, record):
        dg, hs, chunk, (cyc, mk, st, dgst), n, abps = prepared[gi]
        for first in range(0, B_PER_GRAPH, chunk):
            # launches (not steps) alternate over the streams: the chunks of a
            # graph too large for one launch then run side by side
            stream, scratch = streams[n_launched[0] % len(streams)], scratches[n_launched[0] % len(streams)]
            n_launched[0] += 1
            b = min(chunk, B_PER_GRAPH - first)
            if record:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
            api.simulate_hwset_into(dg, hs, first, b, flags, None, mk[first:first + b], st[first:first + b],
                                    dgst[first:first + b], scratch, stream)
            if record:
                e1.record(stream)
                launches.append((e0, e1, abps * b, n * b))
                launch_info.append((gi, first, b))

    for k, gi in enumerate(warm_graphs):
        step(k, gi, False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k, gi in enumerate(step_graphs):
        step(k, gi, True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0

    # simulated nodes count only feasible simulations (an infeasible one
    # stops after the residency check); simulations/s counts all of them
    ok_per_graph = {gi: int((prepared[gi][3][2] == 0).sum().item()) for gi in set(step_graphs)}
    node_sims = sum(prepared[gi][4] * ok_per_graph[gi] for gi in step_graphs)
    sims = B_PER_GRAPH * len(step_graphs)
    durs = np.array([a.elapsed_time(b) * 1e-3 for a, b, _, _ in launches])
    if args.launch_log:
        with open(args.launch_log, "w") as f:
            for (gi, first, b), d in zip(launch_info, durs):
                f.write(json.dumps({"graph": gi, "first": first, "sims": b, "ms": float(d * 1e3)}) + "\n")
    abytes = np.array([x for _, _, x, _ in launches], dtype=np.float64)
    # dominant kernel: the simulation kernel (the only kernel in the step).
    # achieved: algorithmic bytes per launch / mean launch duration; with
    # launches overlapping on several streams the aggregate rate (all bytes
    # over the timed region) is higher and is reported beside it.
    achieved_gbs = float(abytes.sum() / durs.sum() / 1e9)
    aggregate_gbs = float(abytes.sum() / elapsed / 1e9)
    traffic = None if (pipelining or noc or lru) else recorded_traffic(len(launches))
    statuses = np.concatenate([prepared[gi][3][2].cpu().numpy() for gi in sorted(set(step_graphs))])

    host_io_rates = host_io(api, torch, prepared, host_graphs, scratches, streams, step_graphs, flags) \
        if args.host_io else None

    phases = None
    if args.phase_stats:
        if noc or lru:  # clustered and tiled graphs run on the general kernel, which keeps no such counters
            print("--phase-stats covers the windowed kernel only", file=sys.stderr)
        else:
            phases = phase_stats(api, torch, prepared, scratches[0], streams[0], sorted(set(step_graphs)), flags)

    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        # the oracle on a bounded sample of the same sweep: batches of
        # `threads` configurations, cycling through the timed graphs, each
        # result also checked against the GPU's
        import oracle
        threads = min(16, len(os.sched_getaffinity(0)))
        checked, bad, nodes_done = 0, 0, 0
        used = []
        c0 = time.perf_counter()
        k = 0
        while time.perf_counter() - c0 < args.cpu_seconds and (k // len(step_graphs) + 1) * threads <= B_PER_GRAPH:
            gi = step_graphs[k % len(step_graphs)]
            first = (k // len(step_graphs)) * threads
            k += 1
            g, hw = host_graphs[gi]
            idx = list(range(first, min(first + threads, B_PER_GRAPH)))
            mk_gpu = prepared[gi][3][1][idx].cpu().numpy().view(np.uint32)
            st_gpu = prepared[gi][3][2][idx].cpu().numpy()
            dg_gpu = prepared[gi][3][3][idx].cpu().numpy().view(np.uint64)
            omk, ost, odg, _ = oracle.simulate_batch(g, hw[idx], flags, want_nodes=False, threads=threads)
            checked += len(idx)
            bad += int(np.sum((omk != mk_gpu) | (ost != st_gpu) | (odg != dg_gpu)))
            nodes_done += g.n_nodes * int(np.sum(ost == 0))
            used.append(gi)
        csec = time.perf_counter() - c0
        cpu = {"value": nodes_done / csec, "unit": "simulated tile-nodes/s", "cores": threads, "kind": "oracle",
               "sample": f"{checked} simulations ({len(set(used))} sweep graphs, {threads} configurations each, "
                         f"cycling in step order), {threads} threads, {csec:.1f} s"}
        parity = {"checked_sims": checked, "mismatches": bad}

    out = {
        "metric": "simulated tile-nodes/sec (batched) + simulations/sec; % of HBM roofline",
        "value": node_sims / elapsed,
        "unit": "simulated tile-nodes/s",
        "n_gpus": 1,
        "steps": len(step_graphs),
        "warmup": len(warm_graphs),
        "ms_per_step": elapsed / len(step_graphs) * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": args.workload, "graphs": step_graphs, "sims_per_graph": B_PER_GRAPH,
                   "outputs": "makespan+status+digest", "parallelism": "one wavefront per simulation",
                   "streams": len(streams)},
        "simulations_per_s": sims / elapsed,
        "node_sims": node_sims,
        "infeasible_sims": int((statuses == 1).sum()),
        "roofline": {"bound": "hbm", "achieved": achieved_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved_gbs / HBM_PEAK_GBS, "traffic": traffic,
                     "traffic_over_algorithmic": (traffic / float(abytes.mean())) if traffic else None,
                     "kernel": "gts_sim_wave" if (noc or lru) else "gts_sim_window", "launches": len(launches),
                     "mean_launch_ms": float(durs.mean() * 1e3),
                     "streams": len(streams), "aggregate_gbs": aggregate_gbs,
                     "aggregate_frac": aggregate_gbs / HBM_PEAK_GBS},
        "cpu_baseline": cpu,
        "parity_sample": parity,
        "setup_s": t_gen,
    }
    if pipelining:
        out["case_study"] = case_study(api, torch, PL)
    if noc:
        out["case_study"] = noc_case_study(api, torch, CF)
    if lru:
        out["case_study"] = lru_case_study(api, torch, W)
    if phases is not None:
        out["phase_stats"] = phases
    if host_io_rates is not None:
        out["host_io"] = host_io_rates
    print(json.dumps(out))
    return 0


def host_io(api, torch, prepared, host_graphs, scratches, streams, step_graphs, flags):
    """The timed steps again, end to end from host memory (never the
    headline value): (a) each launch passes its hardware records from host
    memory (the C ABI copies them over PCIe into scratch) and each step's
    makespan / status / digest come back to pinned host memory; (b) as (a),
    with each step's graph also uploaded from its host arrays (validation and
    image construction on the CPU, then the copy)."""
    pinned = {gi: [torch.empty(prepared[gi][3][i].shape, dtype=prepared[gi][3][i].dtype, pin_memory=True)
                   for i in (1, 2, 3)] for gi in set(step_graphs)}
    rates = {}
    for mode in ("records", "records+graph"):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        nodes = 0
        keep = []  # uploaded images stay alive until every launch that reads them is done
        for k, gi in enumerate(step_graphs):
            stream, scratch = streams[k % len(streams)], scratches[k % len(streams)]
            dg, hs, chunk, (cyc, mk, st, dgst), n, _ = prepared[gi]
            g, hw = host_graphs[gi]
            if mode == "records+graph":
                dg = api.upload(g, stream)
                keep.append(dg)
            for first in range(0, B_PER_GRAPH, chunk):
                b = min(chunk, B_PER_GRAPH - first)
                api.simulate_into(dg, hw[first:first + b], flags, None, mk[first:first + b], st[first:first + b],
                                  dgst[first:first + b], scratch, stream)
            with torch.cuda.stream(stream):
                for dst, src in zip(pinned[gi], (mk, st, dgst)):
                    dst.copy_(src, non_blocking=True)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        keep.clear()
        for gi in set(step_graphs):
            nodes_ok = prepared[gi][4] * int((pinned[gi][1] == 0).sum().item())
            nodes += nodes_ok * step_graphs.count(gi)
        rates[mode] = {"value": nodes / dt, "unit": "simulated tile-nodes/s", "seconds": dt}
        print(f"[bench] host io {mode}: {nodes / dt:.4e} tile-nodes/s over {dt:.2f} s", file=sys.stderr, flush=True)
    return rates


PHASE_COLUMNS = ("windows", "local_steps", "local_nodes", "memory_arrivals", "retirements", "max_arrivals",
                 "clk_scan", "clk_retire", "clk_local", "clk_gather", "clk_memory")


def phase_stats(api, torch, prepared, scratch, stream, graphs, flags):
    """Where a windowed-kernel simulation spends its time: one untimed launch
    of each graph's first chunk, then the per-simulation counter block the
    kernel writes at the end of each simulation's scratch slice (windows,
    local steps, nodes issued by them, memory arrivals, retirements, the
    largest memory batch, and shader-clock ticks in the window scan,
    retirement, local, ring-gather and memory phases), averaged over the
    feasible simulations.  The clocks are read only in these launches
    (GTS_WINDOW_CLOCKS): each read waits for every outstanding scalar and LDS
    access, which the timed launches avoid."""
    rows = {}
    os.environ["GTS_WINDOW_CLOCKS"] = "1"  # the kernel reads its clock only when asked
    for gi in graphs:
        dg, hs, chunk, (cyc, mk, st, dgst), n, _ = prepared[gi]
        stride = api.scratch_bytes(dg, 2, flags) - api.scratch_bytes(dg, 1, flags)
        api.simulate_hwset_into(dg, hs, 0, chunk, flags, None, mk[:chunk], st[:chunk], dgst[:chunk], scratch, stream)
        torch.cuda.synchronize()
        blk = scratch[:chunk * stride].view(chunk, stride)[:, stride - 128:].contiguous().view(torch.int64)
        ok = (st[:chunk] == 0).cpu().numpy()
        if not ok.any():
            continue
        m = blk.cpu().numpy()[ok][:, :len(PHASE_COLUMNS)].astype(np.float64).mean(axis=0)
        row = {k: round(float(v), 1) for k, v in zip(PHASE_COLUMNS, m)}
        clk = m[6:11]
        row["nodes_per_local_step"] = round(float(m[2] / max(m[1], 1)), 2)
        row["arrivals_per_window"] = round(float(m[3] / max(m[0], 1)), 2)
        row["clk_share"] = {k[4:]: round(float(c / clk.sum()), 3) for k, c in zip(PHASE_COLUMNS[6:], clk)}
        row["clk_per_local_step"] = round(float(m[8] / max(m[1], 1)))
        row["clk_per_window_memory"] = round(float((m[9] + m[10]) / max(m[0], 1)))
        rows[str(gi)] = row
        print(f"[bench] phase stats graph {gi}: {json.dumps(row)}", file=sys.stderr, flush=True)
    os.environ.pop("GTS_WINDOW_CLOCKS", None)
    return rows


def lru_case_study(api, torch, W):
    """One GEMM (4096 x 4096 x 2048, 128 x 128 x 64 tiles, 3 stages) on
    Table 3's H100 across L2 sizes: kernel cycles under the static
    first-touch flags (0 MiB) and under the LRU L2."""
    from paper_2607_11262_amd.gen import hw as H
    g = W.gemm(4096, 4096, 2048, 128, 128, 64, 3, tiles=True)
    sizes = (0, 0.5, 2, 8, 32, 50)
    recs = np.stack([H.preset("H100", l2_lines=H.l2_lines(m)) for m in sizes])
    res = api.simulate(api.upload(g), recs, api.OUT_DIGEST)
    torch.cuda.synchronize()
    _, mk, st, _ = api.to_numpy(res)
    return {"graph": "gemm 4096x4096x2048 128x128x64 s3", "nodes": g.n_nodes,
            "cycles_by_l2_mib": {("static" if m == 0 else str(m)): int(c) for m, c in zip(sizes, mk)}}


def noc_case_study(api, torch, CF):
    """Sec. 7.2 table from GPU timelines on Table 3's H100 with a 16-node
    crossbar or a 4 x 4 mesh of the same total bandwidth and mean latency:
    per cluster size, kernel cycles with NoC and with DRAM communication,
    and the mean NoC residence of a request per topology and placement."""
    from paper_2607_11262_amd import timeline as TL
    topos = (("crossbar", "strips"), ("mesh", "strips"), ("mesh", "blocks"), ("mesh", "strided"))
    recs = np.stack([CF.noc_h100(t, m) for t, m in topos])
    table = {}
    for S in CF.CLUSTER_SIZES:
        row = {}
        for comm in CF.COMMS:
            g = CF.cluster_attention(S, comm=comm)
            res = api.simulate(api.upload(g), recs, api.OUT_NODES | api.OUT_DIGEST)
            torch.cuda.synchronize()
            cyc, mk, st, _ = api.to_numpy(res)
            for i, (t, m) in enumerate(topos):
                key = f"{t}-{m}"
                row.setdefault(key, {})[f"cycles_{comm}"] = int(mk[i])
                if comm == "noc":
                    row[key]["noc_residence"] = round(TL.noc_residence(g, cyc[i]), 1)
        for key in row:
            row[key]["noc_speedup_vs_dram"] = round(row[key]["cycles_dram"] / row[key]["cycles_noc"], 4)
        table[f"cluster{S}"] = row
    return table


def case_study(api, torch, PL):
    """Sec. 7.1 table from GPU timelines at Table 3's H100 (one SM, FP8
    tensor rate): per tile, each organisation's performance relative to naive
    2-stage and its Tensor Core utilisation (full tile graphs)."""
    from paper_2607_11262_amd import timeline as TL
    from paper_2607_11262_amd.gen import hw as H
    rec = H.preset("H100", n_sm=1, tensor_permille=2000)[None, :]
    table = {}
    for tile in PL.TILES:
        row = {}
        for org in PL.ORGANIZATIONS:
            g = PL.gemm_silu(org, *tile)
            res = api.simulate(api.upload(g), rec, api.OUT_NODES | api.OUT_DIGEST)
            torch.cuda.synchronize()
            cyc, mk, st, _ = api.to_numpy(res)
            row[org] = {"makespan": int(mk[0]), "tensor_util": round(TL.utilization(g, rec[0], cyc[0])["tensor"], 4)}
        for org in PL.ORGANIZATIONS:
            row[org]["perf_vs_naive"] = round(row["naive"]["makespan"] / row[org]["makespan"], 4)
        table["x".join(map(str, tile))] = row
    return table


if __name__ == "__main__":
    sys.exit(main())

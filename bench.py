#!/usr/bin/env python3
"""Throughput of the batched tile-graph simulation on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Default workload, `gemm_design_sweep`: 64 seeded GEMM tile graphs (M, N, K in
{1,2,4,8}K; CTA tiles {64,128,256}^2 x {32,64}; 2-4 pipeline stages; 4
warps), each simulated under its own 4096 seeded H100-based hardware
configurations (SMs 64-192, DRAM 1.5-8 TB/s, shared memory 96-256 KiB, tensor
rate 0.5-4x): 262,144 simulations.  One step = the whole sweep, digest +
makespan + status per simulation (per-node cycles for the whole sweep would
be about 0.6 TB).

The other named workloads, one step = every hardware record of the graph in
one launch, per-node (start, finish) cycles written for every simulation,
and the same steps timed again with digest outputs only:

    gemm_1024_a100                 GEMM 1024^3, 128x128x32, 2 stages, 6,208 nodes x 16 A100-based records
    flash_attention_b8_h32_s4096   flash attention fwd B8 H32 S4096 d128, 2,637,824 nodes x 256 records
    splitkv_decode_b64             split-KV decode, 64 sequences, 456,528 nodes x 1024 records
    decoder_layer_prefill_2048     Llama-like decoder layer, 20,515,200 nodes x 64 records

Graph images and hardware records are resident in HBM before timing.  The
line reports simulated tile-nodes per second (value), simulations per second,
the roofline of the simulation kernel (algorithmic bytes per step over the
step's wall time from HIP events, against 8 TB/s HBM; the per-launch figure
beside it) and the CPU oracle timed on a bounded sample of the same
simulations on this host's cores, each sampled result compared with the
GPU's.

Case studies (one step = every graph of the study, each under 4096 seeded
machines): `--workload pipelining` (Sec. 7.1, Table 4: fused GEMM + SiLU in
four pipeline organisations x five tiles x four edge sets), `--workload noc`
(Sec. 7.2: cluster-fused attention over an SM-cluster NoC), `--workload
l2lru` (eight sweep GEMMs with tile ids under an LRU L2 of 4-64 MiB),
`--workload txn` (Sec. 5.2 transaction-level memory: eight GEMMs whose tiles
carry addresses in row- or column-major tensors, with and without padding,
expanded into 128-B transactions under an LRU of lines of 4-64 MiB); each
line adds the study's table read off GPU timelines.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import statistics
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
B_STUDY = 4096
NAMED = ("gemm_design_sweep", "gemm_1024_a100", "flash_attention_b8_h32_s4096", "splitkv_decode_b64",
         "decoder_layer_prefill_2048")
STUDIES = ("pipelining", "noc", "l2lru", "txn")
KERNEL_SOURCES = ("gts_window.hip", "gts_sim.hip", "gts_common.h", "gts_dev.h")
PROFILES = os.path.join(ROOT, "profiles")


def alg_bytes_per_sim(g, out_nodes: bool) -> int:
    """Bytes one simulation must move: its graph read once -- per node the op
    id (2 B), warp mask (2 B), successor offset (4 B) and in-degree (2 B), 4 B
    per edge -- its makespan, status and digest (16 B), and with per-node
    output 8 B per node (start, finish)."""
    return 10 * g.n_nodes + 4 * g.n_edges + 16 + (8 * g.n_nodes if out_nodes else 0)


def sources_hash() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2607_11262_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


TRAFFIC_RE = re.compile(r"traffic-record: workload=(\S+) outputs=(\S+) sha256=(\w+) node_sims=(\d+) "
                        r"fetch_kib=(\d+) write_kib=(\d+) fetch_factor=([\d.]+) write_factor=([\d.]+)")


def recorded_traffic(workload: str, outputs: str, profiles=PROFILES):
    """HBM bytes per simulated node of the simulation kernels, from a
    committed rocprofv3 counter summary of this workload and output mode
    (FETCH_SIZE and WRITE_SIZE summed over the profiled dispatches, each
    scaled by what the same counter reads for a plain device copy, over the
    node-simulations of those dispatches); None when no summary was taken on
    the current kernel sources."""
    sha = sources_hash()
    try:
        names = sorted(os.listdir(profiles))
    except OSError:
        return None
    for name in names:
        if not name.endswith(".md"):
            continue
        with open(os.path.join(profiles, name)) as f:
            for m in TRAFFIC_RE.finditer(f.read()):
                if m.group(1) == workload and m.group(2) == outputs and m.group(3) == sha:
                    fetch = int(m.group(5)) * 1024 * float(m.group(7))
                    write = int(m.group(6)) * 1024 * float(m.group(8))
                    return (fetch + write) / int(m.group(4))
    return None


def cpu_model() -> str:
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def workload_parts(name, records=0):
    """(describe, make(i) -> (graph, hw records), count) of a workload's
    graphs; one step simulates every graph under all of its records
    (records: another record count per graph of the GEMM sweep)."""
    from paper_2607_11262_amd.gen import clusterfusion as CF
    from paper_2607_11262_amd.gen import pipelining as PL
    from paper_2607_11262_amd.gen import workloads as W
    if name == "gemm_design_sweep":
        params = W.sweep_params()
        return (lambda i: params[i],
                lambda i: (W.sweep_graph(params[i]), W.workload_hw(name, B=records or None, index=i)), len(params))
    if name in NAMED:
        return (lambda i: name, lambda i: (W.workload_graph(name), W.workload_hw(name)), 1)
    if name == "pipelining":
        return (lambda i: PL.case_study_graphs()[i],
                lambda i: (PL.case_study_graph(i), PL.sample_hopper_1sm(i, B_STUDY)), len(PL.case_study_graphs()))
    if name == "noc":
        graphs = [(S, comm) for S in CF.CLUSTER_SIZES for comm in CF.COMMS]
        return (lambda i: graphs[i],
                lambda i: (CF.cluster_attention(graphs[i][0], comm=graphs[i][1]), CF.sample_noc_machines(i, B_STUDY)),
                len(graphs))
    if name == "l2lru":
        ps = [q for q in sorted(W.sweep_params(), key=W.sweep_nodes) if 40_000 <= W.sweep_nodes(q) <= 300_000][:8]

        def make(i):
            hw = W.workload_hw("gemm_design_sweep", B=B_STUDY, index=i)
            rng = np.random.default_rng(5000 + i)
            hw[:, 26] = (rng.integers(4, 65, size=B_STUDY) * (1 << 20)) // 128  # L2 lines, 4-64 MiB
            return W.gemm(*ps[i], tiles=True), hw
        return (lambda i: ps[i], make, len(ps))
    if name == "txn":
        designs = [(M, N, K, BM, BN, BK, S, var) for (M, N, K, BM, BN, BK, S) in
                   ((512, 512, 1024, 128, 128, 32, 2), (1024, 512, 512, 128, 64, 32, 3),
                    (512, 1024, 512, 64, 128, 64, 2), (1024, 1024, 256, 128, 128, 64, 3))
                   for var in ("kn", "nk")]

        def make(i):
            M, N, K, BM, BN, BK, S, var = designs[i]
            hw = W.workload_hw("gemm_design_sweep", B=B_STUDY, index=i)
            rng = np.random.default_rng(6000 + i)
            hw[:, 26] = (rng.integers(4, 65, size=B_STUDY) * (1 << 20)) // 128  # L2 lines, 4-64 MiB
            return W.gemm_addressed(M, N, K, BM, BN, BK, S, b_layout=var, pad=8 * (i % 2)), hw
        return (lambda i: designs[i], make, len(designs))
    raise KeyError(name)


class Plan:
    """Every graph of the workload uploaded with its records, and the
    launches of one step: each graph's records in equal chunks that fit the
    per-stream scratch budget, consecutive launches alternating over the
    streams."""

    def __init__(self, api, torch, name, flags, budget, streams, dev, only=-1, records=0):
        describe, make, n = workload_parts(name, records)
        self.parts = []   # (graph handle, hw set, outputs, host graph, host hw)
        self.launches = []  # (part, first, count)
        self.flags = flags
        max_scratch = 0
        for i in (range(n) if only < 0 else [only]):
            g, hw = make(i)
            dg = api.upload(g)
            hs = api.upload_hw(hw)
            B = hw.shape[0]
            per_sim = api.scratch_bytes(dg, 2, flags) - api.scratch_bytes(dg, 1, flags)
            most = max(1, min(B, budget // max(per_sim, 1)))
            n_launch = -(-B // most)
            chunk = -(-B // n_launch)  # equal launches: a short tail launch costs a whole simulation's latency
            max_scratch = max(max_scratch, api.scratch_bytes(dg, chunk, flags))
            outs = api.alloc_outputs(dg, B, flags, dev)
            self.parts.append((dg, hs, outs, g, hw))
            for first in range(0, B, chunk):
                self.launches.append((len(self.parts) - 1, first, min(chunk, B - first)))
            print(f"[bench] graph {i} {describe(i)} N={g.n_nodes} E={g.n_edges} B={B} chunk={chunk}",
                  file=sys.stderr, flush=True)
        self.streams = streams
        self.scratches = [torch.empty(max(max_scratch, 1), dtype=torch.uint8, device=dev) for _ in streams]

    def step(self, api, torch, events=None, flags=None):
        """Enqueue one step; with `events`, append (start, end) HIP events
        around each launch on its stream."""
        flags = self.flags if flags is None else flags
        for k, (i, first, b) in enumerate(self.launches):
            dg, hs, (cyc, mk, st, dgst), _, _ = self.parts[i]
            s, scratch = self.streams[k % len(self.streams)], self.scratches[k % len(self.streams)]
            if events is not None:
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(s)
            api.simulate_hwset_into(dg, hs, first, b, flags, cyc[first:first + b] if cyc is not None else None,
                                    mk[first:first + b], st[first:first + b],
                                    dgst[first:first + b] if dgst is not None else None, scratch, s)
            if events is not None:
                e1.record(s)
                events.append((e0, e1))

    def timed(self, api, torch, steps, flags=None):
        """Run `steps` steps, each bracketed by HIP events on the first
        stream (the others wait for its start event, and it for their ends).
        Returns (per-step seconds, per-launch seconds, wall seconds)."""
        s0 = self.streams[0]
        step_ev, launch_ev = [], []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s0)
            for s in self.streams[1:]:
                s.wait_event(a)
            self.step(api, torch, launch_ev, flags)
            for s in self.streams[1:]:
                e = torch.cuda.Event()
                e.record(s)
                s0.wait_event(e)
            z.record(s0)
            step_ev.append((a, z))
        # every step is enqueued; wait for them one by one so that a long
        # region still reports progress (the host only waits: the GPU's
        # timing is unaffected)
        for k, (_, z) in enumerate(step_ev):
            z.synchronize()
            print(f"[bench] step {k + 1}/{steps} done at {time.perf_counter() - t0:.1f} s", file=sys.stderr,
                  flush=True)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return ([a.elapsed_time(z) * 1e-3 for a, z in step_ev], [a.elapsed_time(z) * 1e-3 for a, z in launch_ev],
                wall)

    def feasible(self):
        """Per graph: its feasible records (an infeasible simulation stops
        after the residency check and simulates no node)."""
        return [(p[2][2] == 0).cpu().numpy() for p in self.parts]

    def step_totals(self, out_nodes):
        ok = self.feasible()
        node_sims = sum(int(f.sum()) * p[3].n_nodes for f, p in zip(ok, self.parts))
        sims = sum(p[4].shape[0] for p in self.parts)
        abytes = sum(int(f.sum()) * (alg_bytes_per_sim(p[3], out_nodes) - 16) + 16 * p[4].shape[0]
                     for f, p in zip(ok, self.parts))
        return node_sims, sims, abytes, sum(int((~f).sum()) for f in ok)


def cpu_leg(plan, flags, seconds, out_nodes):
    """The oracle on this host: a single-thread rate first, then every core.
    Records are drawn in rounds that take a few records from each launch of
    the step (spread over the launch by a seeded permutation; about 50K
    simulated nodes per task, so small graphs are not timed as Python
    overhead), each result compared with the GPU's -- digest, makespan and
    status, and every node's cycles for the first records of each launch
    when per-node output is on.  A workload smaller than the budget is
    sampled again from its start (the rate counts the repeats; the parity
    count does not)."""
    import oracle
    from concurrent.futures import FIRST_COMPLETED, ThreadPoolExecutor, wait
    threads = len(os.sched_getaffinity(0))
    rng = np.random.default_rng(7)
    orders = [first + rng.permutation(b) for (_, first, b) in plan.launches]
    host_out = []
    for p in plan.parts:
        mk, st, dg = p[2][1:]
        host_out.append((mk.cpu().numpy().view(np.uint32), st.cpu().numpy(),
                         dg.cpu().numpy().view(np.uint64) if dg is not None else None))
    checked = bad = node_fail = 0
    nodes_checked_sims = 0
    unique = set()

    def one(task):
        i, recs, want = task
        g, hw = plan.parts[i][3], plan.parts[i][4]
        f = flags | (oracle.F_NODES if want else 0)
        return i, recs, want, oracle.simulate_records(g, hw[recs], f, want_nodes=want), g.n_nodes

    def check(res):
        nonlocal checked, bad, node_fail, nodes_checked_sims
        i, recs, want, (mk, st, dg, cyc), n = res
        gmk, gst, gdg = host_out[i]
        nodes = 0
        for k, r in enumerate(recs):
            checked += 1
            unique.add((i, r))
            wrong = st[k] != gst[r] or mk[k] != gmk[r] or (gdg is not None and dg[k] != gdg[r])
            bad += int(wrong)
            if want and st[k] == 0:
                gc = plan.parts[i][2][0][r].cpu().numpy().view(np.uint32)
                node_fail += int(not np.array_equal(gc, cyc[k]))
                nodes_checked_sims += 1
            nodes += n if st[k] == 0 else 0
        return nodes, len(recs)

    def tasks():
        pos = [0] * len(orders)
        while True:
            for j, o in enumerate(orders):
                i = plan.launches[j][0]
                take = max(1, 50_000 // max(1, plan.parts[i][3].n_nodes))
                if pos[j] >= len(o):
                    continue
                recs = [int(r) for r in o[pos[j]:pos[j] + take]]
                want = bool(out_nodes and pos[j] < 2)
                if want:
                    recs = recs[:2 - pos[j]]
                pos[j] += len(recs)
                yield i, recs, want
            if all(p >= len(o) for p, o in zip(pos, orders)):
                pos = [0] * len(orders)  # again from the start

    it = tasks()
    # single thread, about a sixth of the budget
    t1 = time.perf_counter()
    nodes1 = done1 = 0
    for task in it:
        n, c = check(one(task))
        nodes1 += n
        done1 += c
        if time.perf_counter() - t1 > seconds / 6:
            break
    sec1 = time.perf_counter() - t1
    # all cores: a sliding window of tasks in flight
    t2 = time.perf_counter()
    nodes_all = done_all = 0
    with ThreadPoolExecutor(max_workers=threads) as ex:
        live = {ex.submit(one, next(it)) for _ in range(2 * threads)}
        while live:
            done, live = wait(live, return_when=FIRST_COMPLETED)
            for fu in done:
                n, c = check(fu.result())
                nodes_all += n
                done_all += c
                if time.perf_counter() - t2 < seconds:
                    live.add(ex.submit(one, next(it)))
    sec_all = time.perf_counter() - t2
    launches_touched = len({j for j, (i, first, b) in enumerate(plan.launches)
                            if any(i == ui and first <= ur < first + b for ui, ur in unique)}) \
        if len(plan.launches) < 512 else None
    cpu = {"value": nodes_all / sec_all if sec_all > 0 else None, "unit": "simulated tile-nodes/s",
           "cores": threads, "kind": "oracle",
           "single_core": nodes1 / sec1 if sec1 > 0 else None,
           "cores_available": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count(), "cpu_model": cpu_model(),
           "sample": f"{done1} simulations on 1 thread ({sec1:.1f} s), then {done_all} on {threads} threads "
                     f"({sec_all:.1f} s), records drawn in rounds over every launch of the step"}
    parity = {"checked_sims": len(unique), "checks": checked, "mismatches": bad, "launches": len(plan.launches),
              "launches_sampled": launches_touched, "node_cycle_sims": nodes_checked_sims,
              "node_cycle_mismatches": node_fail}
    return cpu, parity


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", choices=NAMED + STUDIES, default="gemm_design_sweep")
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--digest-only", action="store_true",
                    help="named workloads other than the sweep: time digest outputs only (no per-node cycles)")
    ap.add_argument("--nodes-only", action="store_true",
                    help="named workloads other than the sweep: skip the second, digest-only timed region")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="bounded CPU-oracle sample length")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-case-study", action="store_true",
                    help="skip a study workload's case-study table (its launches would join a counter profile)")
    ap.add_argument("--mem-budget-gb", type=float, default=220.0,
                    help="device scratch budget, split evenly over the streams")
    ap.add_argument("--streams", type=int, default=2,
                    help="consecutive launches alternate over this many HIP streams, so one launch overlaps the "
                         "tail of the previous one")
    ap.add_argument("--launch-log", type=str, default="", help="write one JSON line per timed launch to this file")
    ap.add_argument("--host-io", action="store_true",
                    help="after the timed region, time the same steps through host buffers: hardware records "
                         "passed from host memory per call (gts_simulate_batch) and results copied back, then "
                         "also with each graph uploaded from its host arrays every step")
    ap.add_argument("--phase-stats", action="store_true",
                    help="after the timed region, report the windowed kernel's per-phase counters per graph")
    ap.add_argument("--only-graph", type=int, default=-1,
                    help="diagnostics: simulate only this graph of the workload (index into its graphs)")
    ap.add_argument("--records", type=int, default=0,
                    help="diagnostics: hardware records per graph of the GEMM sweep (default 4096)")
    ap.add_argument("--calibrate-copy-gib", type=float, default=0.0,
                    help="only run a plain device-to-device copy of this many GiB (HBM counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); simulations are independent, "
              "so a multi-GPU run would shard the batch across GPUs.", file=sys.stderr)
        return 2

    import torch

    from paper_2607_11262_amd import api

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

    name = args.workload
    sweep = name == "gemm_design_sweep"
    per_node = name in NAMED and not sweep and not args.digest_only
    flags = api.OUT_DIGEST | (api.OUT_NODES if per_node else 0)
    t_setup = time.time()
    budget = int(args.mem_budget_gb * (1 << 30)) // max(1, args.streams)
    plan = Plan(api, torch, name, flags, budget, streams, dev, only=args.only_graph, records=args.records)
    t_setup = time.time() - t_setup

    for k in range(args.warmup):
        plan.step(api, torch)
        torch.cuda.synchronize()
        print(f"[bench] warmup step {k + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    step_s, launch_s, wall = plan.timed(api, torch, args.steps)
    node_sims, sims, abytes, infeasible = plan.step_totals(per_node)
    K = args.steps
    if args.launch_log:
        with open(args.launch_log, "w") as f:
            for (i, first, b), d in zip(plan.launches * K, launch_s):
                f.write(json.dumps({"graph": i, "first": first, "sims": b, "ms": d * 1e3,
                                    "node_sims": int((plan.parts[i][2][2][first:first + b] == 0).sum().item())
                                    * plan.parts[i][3].n_nodes}) + "\n")
    mean_step = float(np.mean(step_s))
    achieved = abytes / mean_step / 1e9
    launches_per_step = len(plan.launches)
    mean_launch = float(np.mean(launch_s))
    outputs = "nodes" if per_node else "digest"
    traffic_per_node = recorded_traffic(name, outputs)
    traffic = traffic_per_node * node_sims if traffic_per_node else None

    digest_only = None
    if per_node and not args.nodes_only:
        # the same steps with digest outputs only (no per-node cycles written)
        for _ in range(args.warmup):
            plan.step(api, torch, flags=api.OUT_DIGEST)
        torch.cuda.synchronize()
        print("[bench] digest-only pass", file=sys.stderr, flush=True)
        d_step, d_launch, d_wall = plan.timed(api, torch, K, flags=api.OUT_DIGEST)
        nb = sum(int(f.sum()) * (alg_bytes_per_sim(p[3], False) - 16) + 16 * p[4].shape[0]
                 for f, p in zip(plan.feasible(), plan.parts))
        d_traffic = recorded_traffic(name, "digest")
        digest_only = {"value": node_sims * K / d_wall, "ms_per_step": float(np.mean(d_step)) * 1e3,
                       "median_ms_per_step": float(statistics.median(d_step)) * 1e3,
                       "achieved_gbs": nb / float(np.mean(d_step)) / 1e9,
                       "frac": nb / float(np.mean(d_step)) / 1e9 / HBM_PEAK_GBS,
                       "traffic": d_traffic * node_sims if d_traffic else None}
        # the per-node outputs of the last per-node step are what the CPU leg
        # checks: run it once more
        plan.step(api, torch)
        torch.cuda.synchronize()

    host_io_rates = host_io(api, torch, plan, K) if args.host_io else None

    phases = None
    if args.phase_stats:
        phases = phase_stats(api, torch, plan)

    cpu = parity = None
    if not args.no_cpu_baseline:
        cpu, parity = cpu_leg(plan, flags & ~api.OUT_NODES, args.cpu_seconds, per_node)
        cpu["value_unit_note"] = "simulated tile-nodes per second of the oracle (feasible simulations)"

    out = {
        "metric": "simulated tile-nodes/sec (batched) + simulations/sec; % of HBM roofline",
        "value": node_sims * K / wall,
        "unit": "simulated tile-nodes/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": wall / K * 1e3,
        "median_ms_per_step": float(statistics.median(step_s)) * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": name, "graphs": len(plan.parts),
                   "sims_per_step": sims,
                   "outputs": "per-node start/finish + makespan + status + digest" if per_node
                   else "makespan + status + digest",
                   "parallelism": "one wavefront per simulation", "streams": len(streams),
                   "launches_per_step": launches_per_step},
        "simulations_per_s": sims * K / wall,
        "node_sims_per_step": node_sims,
        "infeasible_sims_per_step": infeasible,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "traffic_over_algorithmic": (traffic / abytes) if traffic else None,
                     "traffic_per_node_sim": traffic_per_node,
                     "algorithmic_bytes_per_step": abytes,
                     "step_ms": mean_step * 1e3,
                     "kernel": {"noc": "gts_sim_wave", "txn": "gts_sim_window_txn",
                                "l2lru": "gts_sim_window_lru"}.get(name, "gts_sim_window"),
                     "launch_ms": mean_launch * 1e3,
                     "per_launch_gbs": abytes / launches_per_step / mean_launch / 1e9,
                     "note": "achieved = algorithmic bytes per step / mean step time (HIP events; launches of a "
                             "step overlap on the streams); per_launch_gbs = bytes per launch / mean launch time"},
        "cpu_baseline": cpu,
        "parity_sample": parity,
        "setup_s": t_setup,
    }
    if digest_only is not None:
        out["digest_only"] = digest_only
    if name == "pipelining" and not args.no_case_study:
        out["case_study"] = case_study(api, torch)
    if name == "noc" and not args.no_case_study:
        out["case_study"] = noc_case_study(api, torch)
    if name == "l2lru" and not args.no_case_study:
        out["case_study"] = lru_case_study(api, torch)
    if name == "txn":
        out["transactions_per_s"] = sum(int((p[2][2] == 0).sum().item()) * _transactions(p[3])
                                        for p in plan.parts) * K / wall
        if not args.no_case_study:
            out["case_study"] = txn_case_study(api, torch)
    if phases is not None:
        out["phase_stats"] = phases
    if host_io_rates is not None:
        out["host_io"] = host_io_rates
    print(json.dumps(out))
    return 0


def host_io(api, torch, plan, K):
    """The timed steps again, end to end from host memory (never the
    headline value): (a) each launch passes its hardware records from host
    memory (the C ABI copies them over PCIe into scratch) and each graph's
    makespan / status / digest come back to pinned host memory every step;
    (b) as (a), with every graph also uploaded from its host arrays every
    step (validation and image construction on the CPU, then the copy)."""
    pinned = [[torch.empty(x.shape, dtype=x.dtype, pin_memory=True) for x in p[2][1:] if x is not None]
              for p in plan.parts]
    node_sims = plan.step_totals(False)[0]
    rates = {}
    for mode in ("records", "records+graph"):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(K):
            keep = []  # uploaded images stay alive until every launch that reads them is done
            graphs = {}
            for k, (i, first, b) in enumerate(plan.launches):
                s, scratch = plan.streams[k % len(plan.streams)], plan.scratches[k % len(plan.streams)]
                dg, hs, (cyc, mk, st, dgst), g, hw = plan.parts[i]
                if mode == "records+graph":
                    if i not in graphs:
                        graphs[i] = api.upload(g, s)
                        keep.append(graphs[i])
                    dg = graphs[i]
                api.simulate_into(dg, hw[first:first + b], api.OUT_DIGEST, None, mk[first:first + b],
                                  st[first:first + b], dgst[first:first + b], scratch, s)
                if first + b == hw.shape[0]:  # the graph's last launch: its results to the host
                    with torch.cuda.stream(s):
                        for dst, src in zip(pinned[i], (mk, st, dgst)):
                            dst.copy_(src, non_blocking=True)
            torch.cuda.synchronize()
            keep.clear()
        dt = time.perf_counter() - t0
        rates[mode] = {"value": node_sims * K / dt, "unit": "simulated tile-nodes/s", "seconds": dt}
        print(f"[bench] host io {mode}: {node_sims * K / dt:.4e} tile-nodes/s over {dt:.2f} s", file=sys.stderr,
              flush=True)
    return rates


PHASE_COLUMNS = ("windows", "local_steps", "local_nodes", "memory_arrivals", "retirements", "max_arrivals",
                 "clk_scan", "clk_retire", "clk_local", "clk_gather", "clk_memory")


def phase_stats(api, torch, plan):
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
    scratch, stream = plan.scratches[0], plan.streams[0]
    seen = set()
    for (i, first, b) in plan.launches:
        if i in seen:
            continue
        seen.add(i)
        dg, hs, (cyc, mk, st, dgst), _, _ = plan.parts[i]
        flags = api.OUT_DIGEST
        stride = api.scratch_bytes(dg, 2, flags) - api.scratch_bytes(dg, 1, flags)
        api.simulate_hwset_into(dg, hs, 0, b, flags, None, mk[:b], st[:b], dgst[:b], scratch, stream)
        torch.cuda.synchronize()
        blk = scratch[:b * stride].view(b, stride)[:, stride - 128:].contiguous().view(torch.int64)
        ok = (st[:b] == 0).cpu().numpy()
        if not ok.any():
            continue
        m = blk.cpu().numpy()[ok][:, :len(PHASE_COLUMNS)].astype(np.float64).mean(axis=0)
        row = {k: round(float(v), 1) for k, v in zip(PHASE_COLUMNS, m)}
        clk = m[6:11]
        row["nodes_per_local_step"] = round(float(m[2] / max(m[1], 1)), 2)
        row["arrivals_per_window"] = round(float(m[3] / max(m[0], 1)), 2)
        row["clk_share"] = {k[4:]: round(float(c / max(clk.sum(), 1)), 3) for k, c in zip(PHASE_COLUMNS[6:], clk)}
        row["clk_per_local_step"] = round(float(m[8] / max(m[1], 1)))
        row["clk_per_window_memory"] = round(float((m[9] + m[10]) / max(m[0], 1)))
        rows[str(i)] = row
        print(f"[bench] phase stats graph {i}: {json.dumps(row)}", file=sys.stderr, flush=True)
    os.environ.pop("GTS_WINDOW_CLOCKS", None)
    return rows


def _transactions(g) -> int:
    """Transactions of one simulation of an addressed graph: its tiles'
    distinct 128-B lines (as the library expands them at upload)."""
    ops = g.node_op.astype(np.int64)
    has = g.node_addr != np.uint64(0xFFFFFFFFFFFFFFFF)
    total = 0
    for v in np.flatnonzero(has).tolist():
        p = ops[v]
        R = int(g.op_rows[p]) if g.op_rows is not None else 1
        W_ = int(g.op_work[p]) // R
        P = int(g.op_pitch[p]) if g.op_pitch is not None else W_
        a = int(g.node_addr[v])
        lines = set()
        for r in range(R):
            lines.update(range((a + r * P) // 128, (a + r * P + W_ - 1) // 128 + 1))
        total += len(lines)
    return total


def txn_case_study(api, torch):
    """Sec. 5.2's transaction-level memory on one GEMM (1024 x 1024 x 1024,
    128 x 128 x 32 tiles, 3 stages) at Table 3's H100 with its 50 MiB L2:
    kernel cycles under the whole-tile model (static first-touch flags, and
    the LRU of tiles) and with tiles expanded into 128-B transactions for
    row-major and column-major B, unpadded and with the leading dimensions
    padded by 8 elements (rows then straddle lines), and BK = 64 (128-B
    rows); transactions per simulation beside each."""
    from paper_2607_11262_amd.gen import hw as H
    from paper_2607_11262_amd.gen import workloads as W
    rec = H.preset("H100", l2_lines=H.l2_lines(H.L2_MIB["H100"]))
    static = H.preset("H100")
    cases = [("whole tiles, static flags", W.gemm(1024, 1024, 1024, 128, 128, 32, 3), static),
             ("whole tiles, LRU of tiles", W.gemm(1024, 1024, 1024, 128, 128, 32, 3, tiles=True), rec)]
    for var in ("kn", "nk"):
        for pad in (0, 8):
            cases.append((f"transactions, B {var}, pad {pad}",
                          W.gemm_addressed(1024, 1024, 1024, 128, 128, 32, 3, b_layout=var, pad=pad), rec))
    cases.append(("transactions, B kn, BK 64", W.gemm_addressed(1024, 1024, 1024, 128, 128, 64, 3), rec))
    out = {}
    for label, g, r in cases:
        res = api.simulate(api.upload(g), r[None, :], api.OUT_DIGEST)
        torch.cuda.synchronize()
        _, mk, st, _ = api.to_numpy(res)
        out[label] = {"cycles": int(mk[0]), "transactions": _transactions(g) if g.node_addr is not None else None}
    return out


def lru_case_study(api, torch):
    """One GEMM (4096 x 4096 x 2048, 128 x 128 x 64 tiles, 3 stages) on
    Table 3's H100 across L2 sizes: kernel cycles under the static
    first-touch flags (0 MiB) and under the LRU L2."""
    from paper_2607_11262_amd.gen import hw as H
    from paper_2607_11262_amd.gen import workloads as W
    g = W.gemm(4096, 4096, 2048, 128, 128, 64, 3, tiles=True)
    sizes = (0, 0.5, 2, 8, 32, 50)
    recs = np.stack([H.preset("H100", l2_lines=H.l2_lines(m)) for m in sizes])
    res = api.simulate(api.upload(g), recs, api.OUT_DIGEST)
    torch.cuda.synchronize()
    _, mk, st, _ = api.to_numpy(res)
    return {"graph": "gemm 4096x4096x2048 128x128x64 s3", "nodes": g.n_nodes,
            "cycles_by_l2_mib": {("static" if m == 0 else str(m)): int(c) for m, c in zip(sizes, mk)}}


def noc_case_study(api, torch):
    """Sec. 7.2 table from GPU timelines on Table 3's H100 with a 16-node
    crossbar or a 4 x 4 mesh of the same total bandwidth and mean latency:
    per cluster size, kernel cycles with NoC and with DRAM communication,
    and the mean NoC residence of a request per topology and placement."""
    from paper_2607_11262_amd import timeline as TL
    from paper_2607_11262_amd.gen import clusterfusion as CF
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


def case_study(api, torch):
    """Sec. 7.1 table from GPU timelines at Table 3's H100 (one SM, FP8
    tensor rate): per tile, each organisation's performance relative to naive
    2-stage and its Tensor Core utilisation (full tile graphs)."""
    from paper_2607_11262_amd import timeline as TL
    from paper_2607_11262_amd.gen import hw as H
    from paper_2607_11262_amd.gen import pipelining as PL
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

"""Benchmark: the full TAPS cost-table build on one MI355X.

One step = one pass of the whole hot path on the 96-layer GPT-style graph
(hidden 12288, 96 heads, seq 2048, batch 64, bf16) on a modeled cluster of
16 nodes x 8 devices (600 GB/s inside a node, 100 GB/s between nodes):
enumerate every strategy of every operator, compute the node (intra-op)
table and the edge (redistribution) table -- 599,136 strategies and
98,668,128 edge entries, left resident in HBM -- through one call of
taps_build_tables (sized on the host, queued without a synchronisation, so
consecutive steps overlap the host's work with the GPU's).  The graph
description is packed into the C structs once, outside the timed region.

Prints one JSON line.  `value` is edge entries per second of whole steps;
`roofline` relates the edge-table kernel (which dominates the step), timed
with HIP events the library records right around its launch on the same
stream, to MI355X's 8 TB/s HBM: each entry writes 36 bytes (t 8, vol 8,
intra 8, inter 8, meta 4).
`shared_tables` times the same build with identical edge tables computed once
(the paper searches one layer of a stack of identical layers) and checks the
result equal to the full evaluation;
`bandwidth_sweep` builds the tables at four inter-node bandwidths in
one pass (candidates costed once per entry, one selection and store per
point); `link_classes` builds them under three link classes (8-device nodes,
4-node groups, the groups above them); `value` and `roofline` always come from
the two-class full evaluation.
`roofline.traffic` is the edge kernel's HBM bytes per launch, from the
committed rocprofv3 counter summary (null once the kernel sources differ from
the ones the counters were taken with).  The kernel's binding limit is VALU
issue, not HBM: `roofline.valu` gives its wavefront VALU instructions per
launch (same counter summary) divided by the measured kernel time, against
the issue ceiling a calibration kernel of plain 32-bit integer VALU
instructions measures on this GPU (libtaps_calibrate.so).
`cpu_baseline` runs the CPU oracle over the whole graph on the host's cores
(one GPU's share of the host: 16), and single-threaded over its first layers.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
BYTES_PER_ENTRY = 36
# rocprofv3 counter summary of the edge kernel on the 96-layer workload: HBM bytes
# per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated) and a hash of the kernel
# sources they were taken with
COUNTERS = os.path.join(ROOT, "profiles", "edge_costs_gpt96L_16x8_counters.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2301_04285_amd", "csrc", f)
                  for f in ("taps_device.h", "taps_kernels.hip", "taps_internal.h")] + \
                 [os.path.join(ROOT, "paper_2301_04285_amd", "build.py")]   # the compile flags


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def counter_summary():
    """Figures of the edge kernel from the committed counter summary (HBM bytes
    per launch, VALU figures), or None when the kernel sources changed since the
    counters were taken."""
    import hashlib
    try:
        text = open(COUNTERS).read()
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines()
                  if ": " in line and line.split(": ", 1)[0].replace("_", "").isalnum()
                  and not line.startswith((" ", "|", "#", "*")))
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    if fields.get("kernel_sources_sha256", "").strip() != h.hexdigest():
        return None
    return fields


def measured_traffic(fields):
    return int(fields["traffic_bytes_per_launch"]) if fields else None


# calibration kinds of the fast class (taps_calibrate_valu_name): v_bitop3_b32,
# v_lshlrev_b16, v_lshrrev_b32, v_and_b32 -- the highest issue rates measured
FAST_KINDS = (2, 5, 7, 10)


def valu_ceiling() -> dict:
    """Issue rates (wavefront VALU instructions per second, whole GPU) of the
    calibration kernels: plain 32-bit adds and xors on vector operands,
    3-operand / bit-field operations (the slow class), and the fastest of the
    single-instruction fast-class kernels (the ceiling the edge kernel is
    measured against)."""
    import ctypes as C
    lib = C.CDLL(os.path.join(ROOT, "paper_2301_04285_amd", "libtaps_calibrate.so"))
    lib.taps_calibrate_valu.restype = C.c_int
    lib.taps_calibrate_valu.argtypes = [C.c_int, C.c_uint32, C.POINTER(C.c_float),
                                        C.POINTER(C.c_double), C.POINTER(C.c_uint32)]
    lib.taps_calibrate_valu_name.restype = C.c_char_p

    def rate(kind):
        ms, n, simds = C.c_float(), C.c_double(), C.c_uint32()
        rc = lib.taps_calibrate_valu(kind, 2000, C.byref(ms), C.byref(n), C.byref(simds))
        if rc != 0:
            raise RuntimeError(f"taps_calibrate_valu({kind}) failed: {rc}")
        r = n.value / (ms.value * 1e-3)
        return {"instr_per_s": r, "per_simd_per_cycle_at_2p4GHz": r / simds.value / 2.4e9,
                "ms": ms.value, "instructions": lib.taps_calibrate_valu_name(kind).decode()}

    rate(0)   # warm-up
    out = {"add_xor": rate(0), "bfe_lshl_or": rate(1)}
    out["fastest"] = max((rate(k) for k in FAST_KINDS), key=lambda r: r["instr_per_s"])
    return out


def valu_classes() -> int:
    """Issue rate of every instruction kind of the calibration library, relative
    to the first (v_add_u32 / v_xor_b32), as one JSON line per kind."""
    import ctypes as C
    import torch
    torch.cuda.init()
    lib = C.CDLL(os.path.join(ROOT, "paper_2301_04285_amd", "libtaps_calibrate.so"))
    lib.taps_calibrate_valu.restype = C.c_int
    lib.taps_calibrate_valu.argtypes = [C.c_int, C.c_uint32, C.POINTER(C.c_float),
                                        C.POINTER(C.c_double), C.POINTER(C.c_uint32)]
    lib.taps_calibrate_valu_name.restype = C.c_char_p
    base = None
    ms, n, simds = C.c_float(), C.c_double(), C.c_uint32()
    lib.taps_calibrate_valu(0, 2000, C.byref(ms), C.byref(n), C.byref(simds))   # warm-up
    for kind in range(lib.taps_calibrate_valu_kinds()):
        ms, n, simds = C.c_float(), C.c_double(), C.c_uint32()
        rc = lib.taps_calibrate_valu(kind, 2000, C.byref(ms), C.byref(n), C.byref(simds))
        if rc != 0:
            raise RuntimeError(f"taps_calibrate_valu({kind}) failed: {rc}")
        rate = n.value / (ms.value * 1e-3)
        base = base or rate
        print(json.dumps({"kind": kind, "instructions": lib.taps_calibrate_valu_name(kind).decode(),
                          "instr_per_s": rate, "cycles_per_instr_per_simd_at_2p4GHz":
                          simds.value * 2.4e9 / rate, "relative_rate": rate / base,
                          "ms": ms.value}), flush=True)
    return 0


def measured_valu(fields, kernel_ms: float, ceiling):
    """The edge kernel's VALU issue rate against the calibrated ceiling."""
    if not fields or "valu_instructions_per_launch" not in fields:
        return None
    instr = float(fields["valu_instructions_per_launch"])
    rate = instr / (kernel_ms * 1e-3)
    out = {"instructions_per_launch": instr,
           "instructions_per_64_entries": float(fields["valu_instructions_per_64_entries"]),
           "lane_utilisation": float(fields["valu_lane_utilisation"]),
           "achieved": rate, "unit": "wavefront VALU instructions/s",
           "source": os.path.relpath(COUNTERS, ROOT)}
    if ceiling:
        out["peak"] = ceiling["fastest"]["instr_per_s"]
        out["frac"] = rate / out["peak"]
        out["peak_source"] = ("calibration kernels: 8 independent chains of one instruction per "
                              "thread, 8 wavefronts per SIMD (libtaps_calibrate.so); the fastest "
                              "fast-class kernel, " + ceiling["fastest"]["instructions"])
        out["add_xor_peak"] = ceiling["add_xor"]["instr_per_s"]
        out["slow_class_peak"] = ceiling["bfe_lshl_or"]["instr_per_s"]
    return out


def cpu_info() -> dict:
    """The host CPU as lscpu reports it (model name, family / model / stepping,
    sockets, cores, threads, online CPUs, hypervisor), else /proc/cpuinfo's
    model name."""
    import subprocess
    keys = {"Model name": "model_name", "CPU family": "family", "Model": "model",
            "Stepping": "stepping", "Socket(s)": "sockets", "Core(s) per socket": "cores_per_socket",
            "Thread(s) per core": "threads_per_core", "CPU(s)": "online_cpus",
            "Hypervisor vendor": "hypervisor", "CPU max MHz": "max_mhz"}
    out = {}
    try:
        text = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for ln in text.splitlines():
            k, _, v = ln.partition(":")
            if k.strip() in keys and keys[k.strip()] not in out:
                out[keys[k.strip()]] = v.strip()
    except (OSError, subprocess.SubprocessError):
        pass
    if "model_name" not in out:
        try:
            with open("/proc/cpuinfo") as f:
                out["model_name"] = next((ln.split(":", 1)[1].strip() for ln in f
                                          if ln.startswith("model name")), "")
        except OSError:
            out["model_name"] = ""
    return out


def cpu_baseline(workload, cluster, layers: int) -> dict:
    """The oracle as it stands: every strategy, node table and edge table of the
    whole graph with its edge tables spread over the host's cores (`value`; each
    oracle call is one edge table, run from a thread pool, and releases the
    interpreter lock), and single-threaded over the graph's first `layers`
    transformer layers (`single_core`)."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import oracle as O

    g = workload.graph
    ops_per_layer = 14

    def run(keep, threads: int):
        edges = [e for e in g.edges if e.src in keep and e.dst in keep]
        t0 = time.perf_counter()
        strats = {k: O.enumerate_strategies(g.ops[k], cluster.devices) for k in sorted(keep)}
        for k in sorted(keep):
            O.node_table(g.ops[k], strats[k], cluster)

        def one(e):
            return O.edge_table(g.ops[e.src], strats[e.src], g.ops[e.dst], e.slot,
                                strats[e.dst], cluster).size

        if threads == 1:
            entries = sum(one(e) for e in edges)
        else:
            with ThreadPoolExecutor(threads) as pool:
                entries = sum(pool.map(one, edges))
        return entries, len(edges), time.perf_counter() - t0

    # one GPU's share of the machine's host is 16 cores, whatever the affinity mask
    # shows; host_cpus and affinity_cpus are reported beside it
    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    everything = set(range(len(g.ops)))
    entries, n_edges, dt = run(everything, cores)
    sample = set(range(min(len(g.ops), layers * ops_per_layer)))
    s_entries, s_edges, s_dt = run(sample, 1)
    return {"value": entries / dt, "unit": "edge entries/s", "cores": cores, "kind": "oracle",
            "cpu": cpu_info(), "host_cpus": os.cpu_count(),
            "affinity_cpus": len(os.sched_getaffinity(0)),
            "sample": f"the whole graph: {len(g.ops)} ops, {n_edges} edges, {entries} edge "
                      f"entries, enumeration + node + edge tables in {dt:.2f} s on {cores} "
                      f"threads",
            "seconds": dt,
            "single_core": {"value": s_entries / s_dt, "cores": 1, "seconds": s_dt,
                            "sample": f"first {layers} of 96 layers: {len(sample)} ops, {s_edges} "
                                      f"edges, {s_entries} edge entries",
                            "whole_graph_seconds_extrapolated": entries / (s_entries / s_dt)}}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5, help="workload 1..5 (default: 5, the largest)")
    ap.add_argument("--cpu-layers", type=int, default=2,
                    help="layers of the graph the single-threaded CPU oracle baseline covers; "
                         "the multi-threaded one covers the whole graph (0 = skip both)")
    ap.add_argument("--shared", type=int, default=1,
                    help="also time taps_edge_costs_shared (identical tables computed once) "
                         "and report it under shared_tables (0 = skip)")
    ap.add_argument("--sweep", type=int, default=4, choices=range(5),
                    help="also time taps_edge_costs_sweep at this many inter-node bandwidths "
                         "(the wide-MLP workload's 12.5-100 GB/s points, the benchmark's cluster "
                         "last) and report it under bandwidth_sweep (0 = skip)")
    ap.add_argument("--link-classes", type=int, default=1,
                    help="also time the build under the workload's hierarchy of link classes "
                         "(taps_node_costs_topology, taps_edge_costs_topology) and report it "
                         "under link_classes (0 = skip)")
    ap.add_argument("--valu-classes", action="store_true",
                    help="only time every instruction kind of libtaps_calibrate.so (issue rates "
                         "per class), print one JSON line per kind, then exit")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes (to scale HBM "
                         "traffic counters), then exit")
    args = ap.parse_args()
    if args.valu_classes:
        return valu_classes()
    if args.copy_calibration:
        import torch
        src = torch.ones(args.copy_calibration // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel() * 4, "launches": 3}))
        return 0
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the cost tables of one modeled cluster are built on a "
              f"single device (asked for --gpus {args.gpus}).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2301_04285_amd import taps, workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    w = W.config(args.config)
    cname, cl = w.clusters[0]
    g = taps.pack_graph(w.graph)
    log(f"[bench] {w.name}/{cname}: {g.n_ops} ops, {g.n_edges} edges")

    stream = torch.cuda.current_stream()
    tabs = taps.build_tables(g, cl, stream=stream)    # allocates the outputs once
    # the separate calls (enumerate, node, edge) give the same tables: checked below
    # for the shared-table and sweep legs, which run on them
    torch.cuda.synchronize()
    entries = int(tabs.edge_offsets[-1])
    strategies = int(tabs.op_offsets[-1])
    log(f"[bench] {strategies} strategies, {entries} edge entries")

    prepared = {}

    def step(ev=None, shared=False, edge_out=None, points=None, topology=None):
        if not points and topology is None:
            # one call, sized on the host, nothing synchronised (the headline build, and
            # the shared-table build into its own tables), its arguments packed once
            key = (shared, id(edge_out))
            if key not in prepared:
                target = tabs if edge_out is None else taps.Tables(
                    tabs.op_offsets, tabs.strategies, tabs.node, tabs.edge_offsets, edge_out)
                prepared[key] = taps.PreparedBuild(g, cl, target, shared=shared, stream=stream)
            if ev is not None:
                ev[0].record(stream)
                taps.taps_set_edge_kernel_events(ev[2], ev[3])
            prepared[key]()
            if ev is not None:
                ev[1].record(stream)
            return
        offs, strat = taps.taps_enumerate_strategies(g, cl, stream=stream, out=tabs.strategies)
        if topology is None:
            taps.taps_node_costs(g, cl, strat, offs, out=tabs.node, stream=stream)
        else:
            taps.taps_node_costs_topology(g, topology, strat, offs, out=tabs.node, stream=stream)
        if ev is not None:
            ev[0].record(stream)
            taps.taps_set_edge_kernel_events(ev[2], ev[3])
        if points:
            taps.taps_edge_costs_sweep(g, points, strat, offs, out=edge_out, stream=stream)
        elif topology is not None:
            taps.taps_edge_costs_topology(g, topology, strat, offs, out=edge_out, stream=stream)
        else:
            taps.taps_edge_costs(g, cl, strat, offs, out=edge_out or tabs.edge, stream=stream,
                                 shared=shared)
        if ev is not None:
            ev[1].record(stream)

    def timed(shared=False, edge_out=None, points=None, topology=None):
        for _ in range(args.warmup):
            step(shared=shared, edge_out=edge_out, points=points, topology=topology)
        torch.cuda.synchronize()
        # per step: the whole edge call, and the edge-table kernel alone (recorded by
        # the library on the same stream right around that launch)
        events = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(4))
                  for _ in range(args.steps)]
        for ev in events:
            for e in ev:
                e.record(stream)   # creates the event before the library records it again
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(args.steps):
            step(events[k], shared=shared, edge_out=edge_out, points=points, topology=topology)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        edge_ms = float(np.mean([ev[0].elapsed_time(ev[1]) for ev in events]))
        kernel_ms = float(np.mean([ev[2].elapsed_time(ev[3]) for ev in events]))
        return wall * 1e3 / args.steps, edge_ms, kernel_ms

    ms_per_step, build_gpu_ms, kernel_ms = timed()
    log(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step, build on the GPU "
        f"{build_gpu_ms:.3f} ms, edge kernel {kernel_ms:.3f} ms")

    bytes_per_launch = BYTES_PER_ENTRY * entries
    counters = counter_summary()
    ceiling = valu_ceiling()
    log(f"[bench] VALU ceiling: {ceiling['fastest']['instr_per_s']:.4g} instr/s "
        f"({ceiling['fastest']['instructions']}, "
        f"{ceiling['fastest']['per_simd_per_cycle_at_2p4GHz']:.3f} per SIMD per cycle), "
        f"add/xor {ceiling['add_xor']['instr_per_s']:.4g}, "
        f"slow class {ceiling['bfe_lshl_or']['instr_per_s']:.4g}")
    achieved = bytes_per_launch / (kernel_ms * 1e-3) / 1e9
    out = {
        "metric": "edge-cost entries/sec on 1 GPU (full cost-table build: enumerate + node + edge)",
        "value": entries / (ms_per_step * 1e-3),
        "unit": "edge entries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": f"{w.name}/{cname}", "edge_entries": entries,
                   "strategies": strategies, "ops": g.n_ops, "edges": g.n_edges,
                   "modeled_devices": cl.devices, "devices_per_node": cl.devices_per_node,
                   "bw_intra_GBps": cl.bw_intra / 1e9, "bw_inter_GBps": cl.bw_inter / 1e9},
        "build_ms": ms_per_step,
        "build_gpu_ms": build_gpu_ms,
        "edge_kernel_ms": kernel_ms,
        "edge_entries_per_s": entries / (kernel_ms * 1e-3),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": measured_traffic(counters) if args.config == 5 else None,
                     # the binding limit: VALU issue (rocprofv3 counters of the same
                     # kernel against the calibrated issue ceiling)
                     "limiter": "valu_issue",
                     "valu": measured_valu(counters, kernel_ms, ceiling)
                     if args.config == 5 else None},
    }
    if args.shared:
        # identical edge tables computed once (taps_edge_costs_shared), into a second
        # set of tables, checked equal to the full evaluation
        other = taps.alloc_table(entries, device="cuda")
        s_step, s_edge, s_kernel = timed(shared=True, edge_out=other)
        equal = all(torch.equal(tabs.edge[f][:entries], other[f][:entries])
                    for f in ("t", "vol", "intra", "inter", "meta"))
        log(f"[bench] shared tables: {s_step:.3f} ms/step, build on the GPU {s_edge:.3f} ms, "
            f"edge kernel {s_kernel:.3f} ms, equal to the full evaluation: {equal}")
        out["shared_tables"] = {
            "ms_per_step": s_step, "build_gpu_ms": s_edge, "edge_kernel_ms": s_kernel,
            "edge_entries_per_s": entries / (s_step * 1e-3),
            "hbm_write_frac": bytes_per_launch / (s_kernel * 1e-3) / 1e9 / HBM_PEAK_GBPS,
            "equal_to_full_evaluation": equal}
        prepared.clear()
        del other
    if args.sweep:
        # the same graph at several inter-node bandwidths in one pass
        # (taps_edge_costs_sweep); the point equal to the benchmark's cluster is
        # checked equal to the full evaluation above
        inter = [12.5e9, 25e9, 50e9, 100e9][-args.sweep:]
        points = [W.Cluster(cl.nodes, cl.devices_per_node, cl.bw_intra, int(b)) for b in inter]
        points[-1] = cl
        outs = [taps.alloc_table(entries, device="cuda") for _ in points]
        w_step, w_edge, w_kernel = timed(edge_out=outs, points=points)
        equal = all(torch.equal(tabs.edge[f][:entries], outs[-1][f][:entries])
                    for f in ("t", "vol", "intra", "inter", "meta"))
        k = len(points)
        log(f"[bench] bandwidth sweep, {k} points: {w_step:.3f} ms/step, edge call "
            f"{w_edge:.3f} ms, edge kernel {w_kernel:.3f} ms, last point equal to the full "
            f"evaluation: {equal}")
        out["bandwidth_sweep"] = {
            "inter_GBps": [p.bw_inter / 1e9 for p in points], "ms_per_step": w_step,
            "edge_call_ms": w_edge, "edge_kernel_ms": w_kernel,
            "edge_entries_per_s": k * entries / (w_step * 1e-3),
            "hbm_write_frac": k * bytes_per_launch / (w_kernel * 1e-3) / 1e9 / HBM_PEAK_GBPS,
            "equal_to_single_point": equal}
        del outs
    if args.link_classes and args.config in W.CONFIG_TOPOLOGIES:
        # the same build under a hierarchy of link classes (taps_*_costs_topology)
        topo = W.CONFIG_TOPOLOGIES[args.config]
        other = taps.alloc_table(entries, device="cuda")
        h_step, h_edge, h_kernel = timed(edge_out=other, topology=topo)
        log(f"[bench] link classes {topo.domains}: {h_step:.3f} ms/step, edge call {h_edge:.3f} ms, "
            f"edge kernel {h_kernel:.3f} ms")
        out["link_classes"] = {
            "domains": list(topo.domains), "bw_GBps": [b / 1e9 for b in topo.bw],
            "ms_per_step": h_step, "edge_call_ms": h_edge, "edge_kernel_ms": h_kernel,
            "edge_entries_per_s": entries / (h_step * 1e-3),
            "hbm_write_frac": bytes_per_launch / (h_kernel * 1e-3) / 1e9 / HBM_PEAK_GBPS}
        del other
    if args.cpu_layers > 0 and args.config == 5:
        log(f"[bench] CPU oracle baseline: the whole graph on the host's cores, "
            f"{args.cpu_layers} layers on one core")
        out["cpu_baseline"] = cpu_baseline(w, cl, args.cpu_layers)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

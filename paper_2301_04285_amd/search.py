"""Strategy search over the cost tables (Searching Strategies by ILP section, Eq. 15-19).

Host side, after the tables: the node table (one record per operator strategy) and the
edge table (one record per (producer strategy, consumer strategy) pair of every edge)
are read back once and turned into an integer program solved by HiGHS through
``scipy.optimize.milp``.

Formulation, read per original edge:

    variables   X[u, i] in {0, 1}     strategy i of operator u is chosen
                B[e, i, j] in [0, 1]  pair (i, j) of edge e = (u -> w) is chosen
    minimise    sum_u sum_i node[u][i] X[u, i] + sum_e sum_ij edge[e][i, j] B[e, i, j]
    subject to  sum_i X[u, i] = 1                 every operator           (Eq. 16)
                sum_j B[e, i, j] = X[u, i]        every edge, every i      (Eq. 17, out-degree)
                sum_i B[e, i, j] = X[w, j]        every edge, every j      (Eq. 17, in-degree)

The paper writes the degree constraints summed over all auxiliary edges of an auxiliary
vertex; the per-edge form implies them and keeps exactly one pair per original edge.
Once X is integral the pair variables are forced to 0 or 1, so they stay continuous.
The memory constraint (Eq. 18) needs a memory cost M_ij the paper does not define;
with ``memory`` and ``budget`` (per-strategy bytes per device from taps_memory_costs)
the chosen strategies must fit the budget, counted once per operator. Node costs enter once per operator (the paper folds the consumer's
intra-operator cost into the weight of each of its in-edges, which counts an operator
with several inputs several times and one with none never).

``compare`` runs the search twice on the same tables -- once on the topology-aware
time ``t`` (TAPS) and once on the communication volume ``vol`` (the volume-based
baseline of the Evaluation section) -- and prices both plans with ``t``.
"""
from __future__ import annotations

import time
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

__all__ = ["Plan", "solve", "plan_cost", "compare", "compare_mesh", "compare_topology",
           "host_tables"]


@dataclass
class Plan:
    choice: List[int]      # strategy index per operator
    objective: float       # cost of the plan in the field it was searched on
    solve_s: float         # HiGHS wall time
    n_binaries: int
    n_pairs: int


def host_tables(graph, tables, field: str):
    """Per-operator node cost vectors and per-edge (S_src, S_dst) cost matrices of one
    record field, as float64 numpy arrays, from `taps.Tables` (device tensors)."""
    offs = np.asarray(tables.op_offsets, dtype=np.int64)
    eoffs = np.asarray(tables.edge_offsets, dtype=np.int64)
    node_all = tables.node[field].cpu().numpy().astype(np.float64)
    edge_all = tables.edge[field].cpu().numpy().astype(np.float64)
    node = [node_all[offs[k]:offs[k + 1]] for k in range(len(graph.ops))]
    edge = []
    for x, e in enumerate(graph.edges):
        ns, nd = offs[e.src + 1] - offs[e.src], offs[e.dst + 1] - offs[e.dst]
        edge.append(edge_all[eoffs[x]:eoffs[x + 1]].reshape(ns, nd))
    return node, edge


def _cost_vector(node, edge, n_var, xoff, boff, scale):
    c = np.empty(n_var)
    for k in range(len(node)):
        c[xoff[k]:xoff[k + 1]] = node[k] / scale
    for x, m in enumerate(edge):
        c[boff[x]:boff[x + 1]] = m.ravel() / scale
    return c


def _scale(node, edge):
    return max([float(np.max(np.abs(v))) for v in node if v.size] +
               [float(np.max(np.abs(m))) for m in edge if m.size] + [1e-300])


def add_backward(graph, tables_edge, backward, offsets, field: str):
    """Per-edge (S_src, S_dst) matrices with each pair's backward cost added: the
    backward table of edge e is consumer-major (S_dst, S_src)."""
    offs = np.asarray(offsets, dtype=np.int64)
    b_all = backward[field].cpu().numpy().astype(np.float64)
    out, pos = [], 0
    for x, e in enumerate(graph.edges):
        ns, nd = offs[e.src + 1] - offs[e.src], offs[e.dst + 1] - offs[e.dst]
        out.append(tables_edge[x] + b_all[pos:pos + ns * nd].reshape(nd, ns).T)
        pos += ns * nd
    return out


def solve(graph, node: Sequence[np.ndarray], edge: Sequence[np.ndarray],
          time_limit: float = 600.0, within=None, maximise: bool = False,
          memory: Optional[Sequence[np.ndarray]] = None, budget: Optional[float] = None) -> Plan:
    """Cheapest plan: one strategy per operator minimising node plus edge costs.

    ``within=(node2, edge2, bound)`` keeps only plans whose cost in a second field is
    at most ``bound`` (a lexicographic second stage); ``maximise`` asks for the
    dearest such plan instead of the cheapest.  ``memory`` (per operator, the bytes
    per device of each strategy, as taps_memory_costs returns them) with ``budget``
    adds the device-memory constraint (Eq. 18): the chosen strategies' memory sums to
    at most ``budget`` bytes."""
    from scipy.optimize import LinearConstraint, milp
    from scipy.sparse import coo_matrix

    n_ops = len(graph.ops)
    sizes = np.array([len(v) for v in node], dtype=np.int64)
    if n_ops and sizes.min() == 0:
        raise ValueError(f"operator {int(np.argmin(sizes))} has no strategy")
    xoff = np.concatenate([[0], np.cumsum(sizes)])
    n_x = int(xoff[-1])
    pair_sizes = np.array([m.size for m in edge], dtype=np.int64)
    boff = n_x + np.concatenate([[0], np.cumsum(pair_sizes)])
    n_var = int(boff[-1])

    # costs scaled to O(1) for the solver; the plan is re-priced exactly below
    c = _cost_vector(node, edge, n_var, xoff, boff, _scale(node, edge))
    if maximise:
        c = -c

    rows, cols, vals = [], [], []
    row = 0
    # Eq. 16: one strategy per operator
    for k in range(n_ops):
        idx = np.arange(xoff[k], xoff[k + 1])
        rows.append(np.full(idx.size, row)); cols.append(idx); vals.append(np.ones(idx.size))
        row += 1
    n_eq1 = row
    # Eq. 17 per edge: row sums equal the producer's choice, column sums the consumer's
    for x, e in enumerate(graph.edges):
        ns, nd = edge[x].shape
        base = boff[x]
        ii, jj = np.meshgrid(np.arange(ns), np.arange(nd), indexing="ij")
        pair = (base + ii * nd + jj).ravel()
        rows.append(row + ii.ravel()); cols.append(pair); vals.append(np.ones(pair.size))
        rows.append(row + np.arange(ns)); cols.append(xoff[e.src] + np.arange(ns))
        vals.append(-np.ones(ns))
        row += ns
        rows.append(row + jj.ravel()); cols.append(pair); vals.append(np.ones(pair.size))
        rows.append(row + np.arange(nd)); cols.append(xoff[e.dst] + np.arange(nd))
        vals.append(-np.ones(nd))
        row += nd
    A = coo_matrix((np.concatenate(vals), (np.concatenate(rows), np.concatenate(cols))),
                   shape=(row, n_var)).tocsr()
    lb = np.zeros(row)
    lb[:n_eq1] = 1.0
    constraints = [LinearConstraint(A, lb, lb)]
    if within is not None:
        node2, edge2, bound = within
        s2 = _scale(node2, edge2)
        c2 = _cost_vector(node2, edge2, n_var, xoff, boff, s2)
        constraints.append(LinearConstraint(c2.reshape(1, -1), -np.inf, bound / s2))
    if memory is not None:
        if budget is None or budget <= 0:
            raise ValueError("a memory constraint needs a positive budget")
        mrow = np.zeros(n_var)
        for k in range(n_ops):
            mrow[xoff[k]:xoff[k + 1]] = np.asarray(memory[k], dtype=np.float64) / budget
        constraints.append(LinearConstraint(mrow.reshape(1, -1), -np.inf, 1.0))
    integrality = np.zeros(n_var)
    integrality[:n_x] = 1
    t0 = time.perf_counter()
    res = milp(c, constraints=constraints, integrality=integrality,
               bounds=(0.0, 1.0), options={"time_limit": time_limit, "mip_rel_gap": 1e-9})
    dt = time.perf_counter() - t0
    if res.x is None:
        raise RuntimeError(f"no plan found: {res.message}")
    choice = [int(np.argmax(res.x[xoff[k]:xoff[k + 1]])) for k in range(n_ops)]
    return Plan(choice, plan_cost(graph, node, edge, choice), dt, n_x, int(pair_sizes.sum()))


def plan_memory(memory: Sequence[np.ndarray], choice: Sequence[int]) -> int:
    """Bytes per device of the chosen strategies (the left side of Eq. 18)."""
    return sum(int(memory[k][c]) for k, c in enumerate(choice))


def plan_cost(graph, node: Sequence[np.ndarray], edge: Sequence[np.ndarray],
              choice: Sequence[int]) -> float:
    """Node cost of every chosen strategy plus edge cost of every chosen pair."""
    tot = sum(float(node[k][choice[k]]) for k in range(len(graph.ops)))
    tot += sum(float(edge[x][choice[e.src], choice[e.dst]]) for x, e in enumerate(graph.edges))
    return tot


def compare(graph, node_t, edge_t, node_vol, edge_vol, time_limit: float = 600.0,
            range_time_limit: float = 60.0, memory=None, budget=None) -> Dict:
    """TAPS (search on t) against the volume-based search (on vol), plans priced with
    the topology-aware time t.

    Many plans can share the smallest volume, and a volume-based search may return
    any of them, so the baseline is the range of t over the volume-optimal plans: the
    cheapest (most favourable to the baseline: the reduction against it is a lower
    bound) and the dearest.  Both come from a second solve restricted to plans whose
    volume equals the optimum.  When such a solve finds no plan within
    ``range_time_limit`` seconds, or returns one whose exact volume exceeds the
    optimum (solver tolerance), that end falls back to the plan of the plain volume
    search and ``range_exact`` says so.  ``memory`` and ``budget`` (see solve) bound
    every search by the device memory."""
    mem = dict(memory=memory, budget=budget)
    topo = solve(graph, node_t, edge_t, time_limit, **mem)
    vol = solve(graph, node_vol, edge_vol, time_limit, **mem)
    vmin = vol.objective
    ends, exact = {}, []
    for key, maximise in (("best", False), ("worst", True)):
        try:
            p = solve(graph, node_t, edge_t, range_time_limit,
                      within=(node_vol, edge_vol, vmin), maximise=maximise, **mem)
            ok = plan_cost(graph, node_vol, edge_vol, p.choice) <= vmin
        except RuntimeError:
            ok = False
        if not ok:
            p = vol
        ends[key] = p
        exact.append(ok)
    t_topo = plan_cost(graph, node_t, edge_t, topo.choice)
    t_best = plan_cost(graph, node_t, edge_t, ends["best"].choice)
    t_worst = plan_cost(graph, node_t, edge_t, ends["worst"].choice)
    red = lambda t: 1.0 - t_topo / t if t > 0 else 0.0
    out = {}
    if memory is not None:
        out["memory_bytes"] = [plan_memory(memory, p.choice)
                               for p in (topo, ends["best"], ends["worst"])]
    return {
        **out,
        "t_topology_plan_s": t_topo,
        "t_volume_plans_s": [t_best, t_worst],
        "reduction": [red(t_best), red(t_worst)],
        "range_exact": exact,
        "volume_optimal_plans_differ": ends["best"].choice != ends["worst"].choice,
        "topology_plan_is_volume_optimal": plan_cost(graph, node_vol, edge_vol,
                                                     topo.choice) <= vmin,
        "solve_s": [topo.solve_s, vol.solve_s],
        "binaries": topo.n_binaries,
        "pairs": topo.n_pairs,
        "topology_plan": topo.choice,
        "volume_plans": [ends["best"].choice, ends["worst"].choice],
    }


# ---------------------------------------------------------------------------
# The Evaluation section's comparison on the synthetic workloads: tables built
# by the library on the GPU, both searches on the host.
# ---------------------------------------------------------------------------

def compare_mesh(graph, cluster, mesh, time_limit: float = 600.0, device="cuda") -> Dict:
    """TAPS over every device matrix against TAPS restricted to the strategies a
    fixed device mesh expresses (each operator axis sharded over whole,
    consecutive mesh dimensions, as a mesh-based search would), both searched and
    priced with the topology-aware time t.  The restricted space is a subset, so
    its best plan is never cheaper."""
    import torch
    from . import taps
    out = {}
    for key, m in (("free", None), ("mesh", mesh)):
        tabs = taps.build_tables(graph, cluster, device=device, mesh=m)
        torch.cuda.synchronize()
        nt, et = host_tables(graph, tabs, "t")
        plan = solve(graph, nt, et, time_limit)
        out[key] = {"t_s": plan_cost(graph, nt, et, plan.choice), "binaries": plan.n_binaries,
                    "pairs": plan.n_pairs, "solve_s": plan.solve_s}
        del tabs
    out["mesh"] = {**out["mesh"], "dims": list(mesh)}
    out["mesh_over_free"] = out["mesh"]["t_s"] / out["free"]["t_s"] if out["free"]["t_s"] else 1.0
    return out


def compare_topology(graph, cluster, topology, time_limit: float = 600.0, device="cuda") -> Dict:
    """Searching with the link classes of ``topology`` against searching with the
    cluster's two classes and against the volume-based search, every plan priced
    with the topology's time."""
    import torch
    from . import taps
    h = taps.build_tables(graph, cluster, device=device, topology=topology)
    torch.cuda.synchronize()
    nh, eh = host_tables(graph, h, "t")
    del h
    two = taps.build_tables(graph, cluster, device=device)
    torch.cuda.synchronize()
    n2, e2 = host_tables(graph, two, "t")
    nv, ev = host_tables(graph, two, "vol")
    del two
    plans = {"classes": solve(graph, nh, eh, time_limit), "two_classes": solve(graph, n2, e2, time_limit),
             "volume": solve(graph, nv, ev, time_limit)}
    t = {k: plan_cost(graph, nh, eh, p.choice) for k, p in plans.items()}
    return {"domains": list(topology.domains), "bw_GBps": [b / 1e9 for b in topology.bw],
            "t_s": t, "reduction_vs_two_classes": 1.0 - t["classes"] / t["two_classes"],
            "reduction_vs_volume": 1.0 - t["classes"] / t["volume"],
            "solve_s": {k: p.solve_s for k, p in plans.items()}}


def experiment_workloads():
    """(name, graph, cluster) of every comparison: the five configurations (the
    transformer ones cut to one layer, as the paper searches one layer of a stack of
    identical layers), plus the paper's measured bandwidths (60 / 6 GB/s on two nodes
    of 8 devices)."""
    from . import workloads as W
    out = []
    for k in (1, 2, 3, 4, 5):
        w = W.config(k)
        g = W.leading_ops(w.graph, 14) if k in (3, 5) else w.graph
        tag = w.name + (" (one layer)" if k in (3, 5) else "")
        for cname, cl in w.clusters:
            out.append((f"{tag} / {cname}", g, cl, W.physical_mesh(k, cl)))
    paper = W.Cluster(2, 8, 60 * W.GB, 6 * W.GB)
    out.append(("gpt-4L-h1024-fp16 / 2x8 at 60/6 GB/s", W.config(2).graph, paper, (8, 2)))
    out.append(("mlp64-fp16 / 2x8 at 60/6 GB/s", W.config(4).graph, paper, (8, 2)))
    return out


def main() -> int:
    import argparse
    import json
    import sys

    ap = argparse.ArgumentParser(description="TAPS against volume-based search on the "
                                             "synthetic workloads (tables built on the GPU)")
    ap.add_argument("--only", default="", help="run the workloads whose name contains this")
    ap.add_argument("--time-limit", type=float, default=300.0, help="seconds per ILP")
    ap.add_argument("--range-time-limit", type=float, default=60.0,
                    help="seconds per solve of the volume-optimal range")
    ap.add_argument("--with-backward", action="store_true",
                    help="charge each edge in both directions (forward + backward tables)")
    ap.add_argument("--workload-json", default="",
                    help="search this workload (JSON written by workloads.workload_to_json, "
                         "e.g. `python -m paper_2301_04285_amd.workloads 2 w.json`) instead of "
                         "the built-in ones")
    ap.add_argument("--mesh-space", action="store_true",
                    help="instead: TAPS over every device matrix against TAPS over the strategies "
                         "of the workload's fixed physical mesh (taps_enumerate_strategies_mesh)")
    ap.add_argument("--link-classes", action="store_true",
                    help="instead: on the workloads with a three-level mesh, search with its link "
                         "classes against searching with two classes and by volume, all plans "
                         "priced with the link classes")
    ap.add_argument("--memory-budget-gb", type=float, default=0.0,
                    help="device-memory constraint (Eq. 18) in GB: the chosen strategies' weight "
                         "and output shards per device (taps_memory_costs) must fit (0 = none)")
    args = ap.parse_args()

    import torch
    from . import taps

    if not torch.cuda.is_available():
        print("the tables are built on a GPU", file=sys.stderr)
        return 1
    if args.workload_json:
        from . import workloads as W
        with open(args.workload_json) as f:
            w = W.workload_from_json(f.read())
        runs = [(f"{w.name} / {n}", w.graph, cl,
                 tuple(m for m in (cl.devices_per_node, cl.nodes) if m > 1))
                for n, cl in w.clusters]
    else:
        runs = experiment_workloads()
    for name, g, cl, mesh in runs:
        if args.only not in name:
            continue
        if args.mesh_space:
            r = compare_mesh(g, cl, mesh, args.time_limit)
            print(json.dumps({"workload": name, **r}), flush=True)
            continue
        if args.link_classes:
            from . import workloads as W
            topo = next((t for t in W.CONFIG_TOPOLOGIES.values() if t.devices == cl.devices and
                         t.domains[0] == cl.devices_per_node), None)
            if topo is None or len(mesh) < 3:
                continue
            topo = W.Topology(topo.domains, (cl.bw_intra, cl.bw_inter, cl.bw_inter // 4))
            r = compare_topology(g, cl, topo, args.time_limit)
            print(json.dumps({"workload": name, **r}), flush=True)
            continue
        tabs = taps.build_tables(g, cl)
        torch.cuda.synchronize()
        nt, et = host_tables(g, tabs, "t")
        nv, ev = host_tables(g, tabs, "vol")
        if args.with_backward:
            _, back = taps.taps_edge_costs(g, cl, tabs.strategies, tabs.op_offsets, backward=True)
            et = add_backward(g, et, back, tabs.op_offsets, "t")
            ev = add_backward(g, ev, back, tabs.op_offsets, "vol")
            del back
        mem = budget = None
        if args.memory_budget_gb > 0:
            m = taps.taps_memory_costs(g, tabs.strategies, tabs.op_offsets)
            flat = m.view(torch.int64).cpu().numpy()
            mem = [flat[int(tabs.op_offsets[k]):int(tabs.op_offsets[k + 1])] for k in range(len(g.ops))]
            budget = args.memory_budget_gb * 1e9
        r = compare(g, nt, et, nv, ev, args.time_limit, args.range_time_limit, mem, budget)
        r.pop("topology_plan")
        r.pop("volume_plans")
        print(json.dumps({"workload": name, "directions": "forward+backward" if
                          args.with_backward else "forward",
                          "memory_budget_gb": args.memory_budget_gb or None, **r}), flush=True)
    return 0


if __name__ == "__main__":
    raise SystemExit(main())

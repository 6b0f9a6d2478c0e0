"""Python binding of the C ABI in ``include/taps.h`` (ctypes).

Argument marshalling only: graph descriptions become the ABI's structs,
torch provides device memory and the current HIP stream, and every step of
the cost tables runs in ``libtaps.so``.  If the library is missing the calls
raise -- there is no other implementation to fall back to.
"""
from __future__ import annotations

import ctypes as C
import os
import re
from dataclasses import dataclass
from typing import Dict, List, Optional, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtaps.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "taps.h")

MAX_AXES = 8
MAX_RANK = 8
MAX_INPUTS = 4
MAX_WEIGHTS = 4

OK, ERR_ARG, ERR_TOPOLOGY, ERR_SHAPE, ERR_NO_STRATEGY, ERR_CAPACITY, ERR_DEVICE = range(7)


class TapsError(RuntimeError):
    def __init__(self, status: int, call: str, detail: str):
        self.status = status
        super().__init__(f"{call} failed: {status_str(status)}: {detail}")


class Cluster(C.Structure):
    _fields_ = [("nodes", C.c_uint32), ("devices_per_node", C.c_uint32),
                ("bw_intra", C.c_uint64), ("bw_inter", C.c_uint64)]


MAX_LEVELS = 8


class Mesh(C.Structure):
    _fields_ = [("n_dims", C.c_uint32), ("dims", C.c_uint32 * MAX_LEVELS)]


MAX_CLASSES = 4


class TopologyS(C.Structure):
    _fields_ = [("n_classes", C.c_uint32), ("domain", C.c_uint32 * MAX_CLASSES),
                ("bw", C.c_uint64 * MAX_CLASSES), ("bw_a2a", C.c_uint64)]


class Tensor(C.Structure):
    _fields_ = [("rank", C.c_uint8), ("axis", C.c_uint8 * MAX_RANK)]


class Op(C.Structure):
    _fields_ = [("n_axes", C.c_uint8), ("part_mask", C.c_uint8), ("dtype_bytes", C.c_uint8),
                ("n_in", C.c_uint8), ("n_w", C.c_uint8),
                ("axis_len", C.c_int64 * MAX_AXES),
                ("ins", Tensor * MAX_INPUTS), ("ws", Tensor * MAX_WEIGHTS), ("out", Tensor)]


class EdgeS(C.Structure):
    _fields_ = [("src_op", C.c_uint32), ("dst_op", C.c_uint32), ("dst_slot", C.c_uint32)]


class GraphS(C.Structure):
    _fields_ = [("n_ops", C.c_uint32), ("n_edges", C.c_uint32),
                ("ops", C.POINTER(Op)), ("edges", C.POINTER(EdgeS))]


class Table(C.Structure):
    _fields_ = [("t", C.c_void_p), ("vol", C.c_void_p), ("intra", C.c_void_p),
                ("inter", C.c_void_p), ("meta", C.c_void_p)]


STRATEGY_BYTES = 16   # sizeof(taps_strategy): log2_deg[8] uint8, pos[8] int8

_lib = None


def load():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2301_04285_amd.build`")
        L = C.CDLL(LIB_PATH)
        P = C.POINTER
        L.taps_enumerate_strategies.restype = C.c_int
        L.taps_enumerate_strategies.argtypes = [P(GraphS), P(Cluster), P(C.c_uint64), C.c_void_p,
                                                C.c_uint64, C.c_void_p]
        L.taps_enumerate_strategies_mesh.restype = C.c_int
        L.taps_enumerate_strategies_mesh.argtypes = [P(GraphS), P(Cluster), P(Mesh), P(C.c_uint64),
                                                     C.c_void_p, C.c_uint64, C.c_void_p]
        L.taps_node_costs_topology.restype = C.c_int
        L.taps_node_costs_topology.argtypes = [P(GraphS), P(TopologyS), C.c_void_p, P(C.c_uint64),
                                               Table, C.c_void_p]
        L.taps_edge_costs_topology.restype = C.c_int
        L.taps_edge_costs_topology.argtypes = [P(GraphS), P(TopologyS), C.c_void_p, P(C.c_uint64),
                                               P(C.c_uint64), Table, C.c_uint64, C.c_void_p]
        L.taps_build_tables.restype = C.c_int
        L.taps_build_tables.argtypes = [P(GraphS), P(Cluster), P(Mesh), P(C.c_uint64), C.c_void_p,
                                        C.c_uint64, Table, P(C.c_uint64), Table, C.c_uint64,
                                        C.c_uint32, C.c_void_p]
        L.taps_build_tables_noalloc.restype = C.c_int
        L.taps_build_tables_noalloc.argtypes = L.taps_build_tables.argtypes
        L.taps_node_costs.restype = C.c_int
        L.taps_node_costs.argtypes = [P(GraphS), P(Cluster), C.c_void_p, P(C.c_uint64), Table,
                                      C.c_void_p]
        L.taps_edge_costs.restype = C.c_int
        L.taps_edge_costs.argtypes = [P(GraphS), P(Cluster), C.c_void_p, P(C.c_uint64),
                                      P(C.c_uint64), Table, C.c_uint64, C.c_void_p]
        L.taps_edge_costs_shared.restype = C.c_int
        L.taps_edge_costs_shared.argtypes = L.taps_edge_costs.argtypes
        L.taps_edge_costs_backward.restype = C.c_int
        L.taps_edge_costs_backward.argtypes = L.taps_edge_costs.argtypes
        L.taps_edge_costs_sweep.restype = C.c_int
        L.taps_edge_costs_sweep.argtypes = [P(GraphS), P(Cluster), C.c_uint32, C.c_void_p,
                                            P(C.c_uint64), P(C.c_uint64), P(Table), C.c_uint64,
                                            C.c_void_p]
        L.taps_memory_costs.restype = C.c_int
        L.taps_memory_costs.argtypes = [P(GraphS), C.c_void_p, P(C.c_uint64), C.c_void_p,
                                        C.c_void_p]
        L.taps_set_edge_kernel_events.restype = C.c_int
        L.taps_set_edge_kernel_events.argtypes = [C.c_void_p, C.c_void_p]
        L.taps_set_long_segments_min.restype = C.c_uint64
        L.taps_set_long_segments_min.argtypes = [C.c_uint64]
        L.taps_status_str.restype = C.c_char_p
        L.taps_status_str.argtypes = [C.c_int]
        L.taps_last_error.restype = C.c_char_p
        L.taps_last_error.argtypes = []
        _lib = L
    return _lib


def declared_symbols() -> List[str]:
    """Entry points declared in include/taps.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:taps_status|const char \*|uint64_t)\s*(taps_\w+)\s*\(", text,
                                 flags=re.M)))


def status_str(status: int) -> str:
    return load().taps_status_str(status).decode()


def last_error() -> str:
    return load().taps_last_error().decode()


def _check(status: int, call: str) -> None:
    if status != OK:
        raise TapsError(status, call, last_error())


# ---------------------------------------------------------------------------
# marshalling
# ---------------------------------------------------------------------------

def _tensor(axes) -> Tensor:
    t = Tensor()
    t.rank = len(axes)
    for d, a in enumerate(axes):
        t.axis[d] = a
    return t


@dataclass
class PackedGraph:
    struct: GraphS
    ops: object
    edges: object
    n_ops: int
    n_edges: int
    edge_list: List[Tuple[int, int, int]]


def pack_graph(graph) -> PackedGraph:
    """``graph`` has ``ops`` (with axis_len, partitionable, dtype_bytes, ins,
    ws, out) and ``edges`` (with src, dst, slot), as ``workloads.Graph``."""
    n_ops, n_edges = len(graph.ops), len(graph.edges)
    ops = (Op * max(n_ops, 1))()
    for k, op in enumerate(graph.ops):
        o = ops[k]
        o.n_axes = len(op.axis_len)
        o.part_mask = sum(1 << a for a, p in enumerate(op.partitionable) if p)
        o.dtype_bytes = op.dtype_bytes
        o.n_in = len(op.ins)
        o.n_w = len(op.ws)
        for a, n in enumerate(op.axis_len):
            o.axis_len[a] = n
        for i, t in enumerate(op.ins):
            o.ins[i] = _tensor(t)
        for i, t in enumerate(op.ws):
            o.ws[i] = _tensor(t)
        o.out = _tensor(op.out)
    edges = (EdgeS * max(n_edges, 1))()
    for k, e in enumerate(graph.edges):
        edges[k].src_op, edges[k].dst_op, edges[k].dst_slot = e.src, e.dst, e.slot
    g = GraphS(n_ops, n_edges, C.cast(ops, C.POINTER(Op)) if n_ops else None,
               C.cast(edges, C.POINTER(EdgeS)) if n_edges else None)
    return PackedGraph(g, ops, edges, n_ops, n_edges,
                       [(e.src, e.dst, e.slot) for e in graph.edges])


def pack_cluster(cluster) -> Cluster:
    return Cluster(cluster.nodes, cluster.devices_per_node, cluster.bw_intra, cluster.bw_inter)


def _stream(stream) -> C.c_void_p:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _graph(graph) -> PackedGraph:
    return graph if isinstance(graph, PackedGraph) else pack_graph(graph)


def _u64_array(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_uint64))


# ---------------------------------------------------------------------------
# the three calls
# ---------------------------------------------------------------------------

def pack_mesh(mesh) -> Mesh:
    """A fixed device mesh, innermost dimension first."""
    dims = [int(m) for m in mesh]
    if len(dims) > MAX_LEVELS:
        raise ValueError(f"a mesh has at most {MAX_LEVELS} dimensions")
    return Mesh(len(dims), (C.c_uint32 * MAX_LEVELS)(*dims))


def taps_enumerate_strategies(graph, cluster, device="cuda", stream=None, size_only=False,
                              out=None, mesh=None):
    """(op_offsets as numpy uint64 [n_ops+1], strategies as a device uint8
    tensor [S, 16]: log2 degrees then device-map positions as int8).
    ``out``: a preallocated device uint8 tensor [capacity, 16] to fill in one
    call; otherwise a size query runs first.  ``mesh`` (sizes, innermost
    first): only the strategies a fixed device mesh expresses
    (taps_enumerate_strategies_mesh)."""
    import torch
    g = _graph(graph)
    cl = pack_cluster(cluster)
    offs = np.zeros(g.n_ops + 1, dtype=np.uint64)
    L = load()
    if mesh is None:
        name = "taps_enumerate_strategies"

        def call(ptr, cap):
            return L.taps_enumerate_strategies(C.byref(g.struct), C.byref(cl), _u64_array(offs),
                                               ptr, cap, _stream(stream))
    else:
        name = "taps_enumerate_strategies_mesh"
        ms = pack_mesh(mesh)

        def call(ptr, cap):
            return L.taps_enumerate_strategies_mesh(C.byref(g.struct), C.byref(cl), C.byref(ms),
                                                    _u64_array(offs), ptr, cap, _stream(stream))
    if out is None:
        _check(call(None, 0), name)
        if size_only:
            return offs, None
        out = torch.empty((max(int(offs[-1]), 1), STRATEGY_BYTES), dtype=torch.uint8,
                          device=device)
    _check(call(C.c_void_p(out.data_ptr()), int(out.shape[0])), name)
    return offs, out[:int(offs[-1])]


def alloc_table(n: int, device="cuda") -> Dict[str, "torch.Tensor"]:
    import torch
    n = max(int(n), 1)
    return {"t": torch.empty(n, dtype=torch.float64, device=device),
            "vol": torch.empty(n, dtype=torch.uint64, device=device),
            "intra": torch.empty(n, dtype=torch.uint64, device=device),
            "inter": torch.empty(n, dtype=torch.uint64, device=device),
            "meta": torch.empty(n, dtype=torch.uint32, device=device)}


def _table(tab) -> Table:
    if tab is None:
        return Table(None, None, None, None, None)
    return Table(*(C.c_void_p(tab[k].data_ptr()) for k in ("t", "vol", "intra", "inter", "meta")))


def taps_node_costs(graph, cluster, strategies, op_offsets, out=None, stream=None):
    """Node table (dict of device tensors, one record per strategy)."""
    g = _graph(graph)
    cl = pack_cluster(cluster)
    offs = np.ascontiguousarray(op_offsets, dtype=np.uint64)
    total = int(offs[-1])
    if out is None:
        out = alloc_table(total, device=strategies.device)
    st = load().taps_node_costs(C.byref(g.struct), C.byref(cl), C.c_void_p(strategies.data_ptr()),
                                _u64_array(offs), _table(out), _stream(stream))
    _check(st, "taps_node_costs")
    return {k: v[:total] for k, v in out.items()}


def pack_topology(topo) -> TopologyS:
    """workloads.Topology (block sizes and bandwidths per link class) -> the ABI struct."""
    if not 1 <= len(topo.domains) == len(topo.bw) <= MAX_CLASSES:
        raise ValueError(f"1 to {MAX_CLASSES} link classes, one bandwidth each")
    return TopologyS(len(topo.domains), (C.c_uint32 * MAX_CLASSES)(*topo.domains),
                     (C.c_uint64 * MAX_CLASSES)(*topo.bw), getattr(topo, "bw_a2a", 0))


def taps_node_costs_topology(graph, topology, strategies, op_offsets, out=None, stream=None):
    """Node table under a hierarchy of link classes (taps_node_costs_topology)."""
    g = _graph(graph)
    tp = pack_topology(topology)
    offs = np.ascontiguousarray(op_offsets, dtype=np.uint64)
    total = int(offs[-1])
    if out is None:
        out = alloc_table(total, device=strategies.device)
    st = load().taps_node_costs_topology(C.byref(g.struct), C.byref(tp),
                                         C.c_void_p(strategies.data_ptr()), _u64_array(offs),
                                         _table(out), _stream(stream))
    _check(st, "taps_node_costs_topology")
    return {k: v[:total] for k, v in out.items()}


def taps_edge_costs_topology(graph, topology, strategies, op_offsets, out=None, stream=None,
                             size_only=False):
    """Edge tables under a hierarchy of link classes (taps_edge_costs_topology):
    (edge_offsets, dict of device tensors or None for a size query)."""
    g = _graph(graph)
    tp = pack_topology(topology)
    offs = np.ascontiguousarray(op_offsets, dtype=np.uint64)
    eoffs = np.zeros(g.n_edges + 1, dtype=np.uint64)
    L = load()
    sptr = C.c_void_p(strategies.data_ptr()) if strategies is not None else None
    if out is None or size_only:
        st = L.taps_edge_costs_topology(C.byref(g.struct), C.byref(tp), sptr, _u64_array(offs),
                                        _u64_array(eoffs), _table(None), 0, _stream(stream))
        _check(st, "taps_edge_costs_topology")
        if size_only:
            return eoffs, None
        out = alloc_table(int(eoffs[-1]), device=strategies.device)
    cap = min(int(v.numel()) for v in out.values())
    st = L.taps_edge_costs_topology(C.byref(g.struct), C.byref(tp), sptr, _u64_array(offs),
                                    _u64_array(eoffs), _table(out), cap, _stream(stream))
    _check(st, "taps_edge_costs_topology")
    total = int(eoffs[-1])
    return eoffs, {k: v[:total] for k, v in out.items()}


def taps_edge_costs(graph, cluster, strategies, op_offsets, out=None, stream=None,
                    size_only=False, shared=False, backward=False):
    """(edge_offsets numpy uint64 [n_edges+1], edge table dict of device
    tensors or None for a size query).  ``shared``: taps_edge_costs_shared
    (identical tables computed once); ``backward``: taps_edge_costs_backward
    (the gradient's direction, tables consumer-major)."""
    if shared and backward:
        raise ValueError("shared tables are computed for the forward direction only")
    g = _graph(graph)
    cl = pack_cluster(cluster)
    offs = np.ascontiguousarray(op_offsets, dtype=np.uint64)
    eoffs = np.zeros(g.n_edges + 1, dtype=np.uint64)
    L = load()
    sptr = C.c_void_p(strategies.data_ptr()) if strategies is not None else None
    if out is None or size_only:   # size query first
        st = L.taps_edge_costs(C.byref(g.struct), C.byref(cl), sptr, _u64_array(offs),
                               _u64_array(eoffs), _table(None), 0, _stream(stream))
        _check(st, "taps_edge_costs")
        if size_only:
            return eoffs, None
        out = alloc_table(int(eoffs[-1]), device=strategies.device)
    cap = min(int(v.numel()) for v in out.values())
    name = ("taps_edge_costs_shared" if shared else
            "taps_edge_costs_backward" if backward else "taps_edge_costs")
    st = getattr(L, name)(C.byref(g.struct), C.byref(cl), sptr, _u64_array(offs),
                          _u64_array(eoffs), _table(out), cap, _stream(stream))
    _check(st, name)
    total = int(eoffs[-1])
    return eoffs, {k: v[:total] for k, v in out.items()}


def taps_memory_costs(graph, strategies, op_offsets, out=None, stream=None):
    """Per-device bytes of every strategy (device uint64 tensor, one per strategy)."""
    import torch
    g = _graph(graph)
    offs = np.ascontiguousarray(op_offsets, dtype=np.uint64)
    total = int(offs[-1])
    if out is None:
        out = torch.empty(max(total, 1), dtype=torch.uint64, device=strategies.device)
    if int(out.numel()) < total:
        raise ValueError(f"memory output holds {out.numel()} entries, {total} needed")
    st = load().taps_memory_costs(C.byref(g.struct),
                                  C.c_void_p(strategies.data_ptr()) if strategies is not None else None,
                                  _u64_array(offs), C.c_void_p(out.data_ptr()), _stream(stream))
    _check(st, "taps_memory_costs")
    return out[:total]


def taps_edge_costs_sweep(graph, clusters, strategies, op_offsets, out=None, stream=None,
                          size_only=False):
    """(edge_offsets numpy uint64 [n_edges+1], list of edge table dicts, one per
    cluster, or None for a size query).  The clusters differ only in their
    bandwidths; table k equals taps_edge_costs on clusters[k]."""
    g = _graph(graph)
    cls = list(clusters)
    arr = (Cluster * max(len(cls), 1))(*[pack_cluster(c) for c in cls])
    offs = np.ascontiguousarray(op_offsets, dtype=np.uint64)
    eoffs = np.zeros(g.n_edges + 1, dtype=np.uint64)
    L = load()
    sptr = C.c_void_p(strategies.data_ptr()) if strategies is not None else None
    if out is None or size_only:   # size query first
        st = L.taps_edge_costs_sweep(C.byref(g.struct), arr, len(cls), sptr, _u64_array(offs),
                                     _u64_array(eoffs), None, 0, _stream(stream))
        _check(st, "taps_edge_costs_sweep")
        if size_only:
            return eoffs, None
        out = [alloc_table(int(eoffs[-1]), device=strategies.device) for _ in cls]
    if len(out) != len(cls):
        raise ValueError(f"{len(out)} tables for {len(cls)} bandwidth points")
    cap = min(int(v.numel()) for o in out for v in o.values())
    tabs = (Table * len(out))(*[_table(o) for o in out])
    st = L.taps_edge_costs_sweep(C.byref(g.struct), arr, len(cls), sptr, _u64_array(offs),
                                 _u64_array(eoffs), tabs, cap, _stream(stream))
    _check(st, "taps_edge_costs_sweep")
    total = int(eoffs[-1])
    return eoffs, [{k: v[:total] for k, v in o.items()} for o in out]


def taps_set_long_segments_min(min_segments: int) -> int:
    """Single-table edge launches with at least ``min_segments`` row segments
    run long (eight-tile) segments, remainders last; returns the previous
    threshold.  The tables are the same either way."""
    return int(load().taps_set_long_segments_min(int(min_segments)))


def taps_set_edge_kernel_events(before, after) -> None:
    """Have this thread's next edge-table kernel recorded between two
    ``torch.cuda.Event``s (each recorded once already, so that it exists), or
    clear the setting with two Nones."""
    handles = []
    for ev in (before, after):
        h = 0 if ev is None else int(ev.cuda_event)
        if ev is not None and h == 0:
            raise ValueError("record the event once before passing it")
        handles.append(C.c_void_p(h) if h else None)
    _check(load().taps_set_edge_kernel_events(*handles), "taps_set_edge_kernel_events")


@dataclass
class Tables:
    op_offsets: np.ndarray
    strategies: "torch.Tensor"
    node: Dict[str, "torch.Tensor"]
    edge_offsets: np.ndarray
    edge: Dict[str, "torch.Tensor"]


TABLE_FIELDS = ("t", "vol", "intra", "inter", "meta")


def save_tables(path: str, tabs: Tables) -> None:
    """Write a table set to one .npz file (plain arrays, no pickled objects)."""
    arrays = {"op_offsets": np.asarray(tabs.op_offsets, dtype=np.uint64),
              "edge_offsets": np.asarray(tabs.edge_offsets, dtype=np.uint64),
              "strategies": tabs.strategies.cpu().numpy()}
    n_str, n_edge = int(tabs.op_offsets[-1]), int(tabs.edge_offsets[-1])
    for prefix, tab, n in (("node_", tabs.node, n_str), ("edge_", tabs.edge, n_edge)):
        for f in TABLE_FIELDS:
            v = tab[f][:n]
            arrays[prefix + f] = {8: lambda: v.view(_torch().int64).cpu().numpy().view(np.uint64),
                                  4: lambda: v.view(_torch().int32).cpu().numpy().view(np.uint32)}[
                v.element_size()]() if f != "t" else v.cpu().numpy()
    np.savez(path, **arrays)


def load_tables(path: str, device="cuda") -> Tables:
    """A table set written by save_tables, on `device`."""
    torch = _torch()
    with np.load(path, allow_pickle=False) as z:
        def dev(a):
            if a.dtype == np.uint64:
                return torch.from_numpy(a.view(np.int64).copy()).to(device).view(torch.uint64)
            if a.dtype == np.uint32:
                return torch.from_numpy(a.view(np.int32).copy()).to(device).view(torch.uint32)
            return torch.from_numpy(a.copy()).to(device)
        return Tables(z["op_offsets"].copy(), dev(z["strategies"]),
                      {f: dev(z["node_" + f]) for f in TABLE_FIELDS}, z["edge_offsets"].copy(),
                      {f: dev(z["edge_" + f]) for f in TABLE_FIELDS})


def _torch():
    import torch
    return torch


BUILD_SHARED = 1


def taps_build_tables(graph, cluster, mesh=None, out: Optional["Tables"] = None, device="cuda",
                      stream=None, size_only=False, shared=False):
    """The whole build in one call without a host synchronisation
    (taps_build_tables): a Tables, or (op_offsets, edge_offsets) for a size
    query.  ``out``: tables of an earlier build of the same graph to fill
    again; otherwise they are allocated after a size query.  ``shared``:
    identical edge tables computed once (TAPS_BUILD_SHARED)."""
    g = _graph(graph)
    cl = pack_cluster(cluster)
    ms = pack_mesh(mesh) if mesh is not None else None
    offs = np.zeros(g.n_ops + 1, dtype=np.uint64)
    eoffs = np.zeros(g.n_edges + 1, dtype=np.uint64)
    L = load()

    def call(strat, s_cap, node, edge, e_cap):
        return L.taps_build_tables(C.byref(g.struct), C.byref(cl), C.byref(ms) if ms else None,
                                   _u64_array(offs), strat, s_cap, _table(node), _u64_array(eoffs),
                                   _table(edge), e_cap, BUILD_SHARED if shared else 0,
                                   _stream(stream) if strat else None)
    if out is None:
        _check(call(None, 0, None, None, 0), "taps_build_tables")
        if size_only:
            return offs, eoffs
        import torch
        n_str, n_edge = int(offs[-1]), int(eoffs[-1])
        out = Tables(offs, torch.empty((max(n_str, 1), STRATEGY_BYTES), dtype=torch.uint8,
                                       device=device),
                     alloc_table(n_str, device), eoffs, alloc_table(n_edge, device))
    s_cap = min(int(out.strategies.shape[0]), *(int(v.numel()) for v in out.node.values()))
    e_cap = min(int(v.numel()) for v in out.edge.values())
    _check(call(C.c_void_p(out.strategies.data_ptr()), s_cap, out.node, out.edge, e_cap),
           "taps_build_tables")
    n_str, n_edge = int(offs[-1]), int(eoffs[-1])
    return Tables(offs, out.strategies[:n_str], {k: v[:n_str] for k, v in out.node.items()}, eoffs,
                  {k: v[:n_edge] for k, v in out.edge.items()})


def taps_build_tables_noalloc(graph, cluster, out: "Tables", mesh=None, stream=None,
                              shared=False) -> "Tables":
    """taps_build_tables_noalloc: the build of taps_build_tables into the caller's
    tables ``out`` (of a build of the same graph and cluster, or larger), with the
    library's device workspace in its fixed per-GPU array instead of allocations."""
    g = _graph(graph)
    cl = pack_cluster(cluster)
    ms = pack_mesh(mesh) if mesh is not None else None
    offs = np.zeros(g.n_ops + 1, dtype=np.uint64)
    eoffs = np.zeros(g.n_edges + 1, dtype=np.uint64)
    s_cap = min(int(out.strategies.shape[0]), *(int(v.numel()) for v in out.node.values()))
    e_cap = min(int(v.numel()) for v in out.edge.values())
    _check(load().taps_build_tables_noalloc(
        C.byref(g.struct), C.byref(cl), C.byref(ms) if ms else None, _u64_array(offs),
        C.c_void_p(out.strategies.data_ptr()), s_cap, _table(out.node), _u64_array(eoffs),
        _table(out.edge), e_cap, BUILD_SHARED if shared else 0, _stream(stream)),
        "taps_build_tables_noalloc")
    n_str, n_edge = int(offs[-1]), int(eoffs[-1])
    return Tables(offs, out.strategies[:n_str], {k: v[:n_str] for k, v in out.node.items()},
                  eoffs, {k: v[:n_edge] for k, v in out.edge.items()})


class PreparedBuild:
    """taps_build_tables with every argument packed once, for callers that
    rebuild the same tables repeatedly (a serving loop, a benchmark): each call
    only queues the build on the stream.  `out` (a Tables of a build of the same
    graph) receives the tables; it must stay alive while the object is used."""

    def __init__(self, graph, cluster, out: "Tables", mesh=None, shared=False, stream=None):
        self._g = _graph(graph)
        self._cl = pack_cluster(cluster)
        self._ms = pack_mesh(mesh) if mesh is not None else None
        self._offs = np.zeros(self._g.n_ops + 1, dtype=np.uint64)
        self._eoffs = np.zeros(self._g.n_edges + 1, dtype=np.uint64)
        self._out = out
        s_cap = min(int(out.strategies.shape[0]), *(int(v.numel()) for v in out.node.values()))
        e_cap = min(int(v.numel()) for v in out.edge.values())
        L = load()
        self._fn = L.taps_build_tables
        self._args = (C.byref(self._g.struct), C.byref(self._cl),
                      C.byref(self._ms) if self._ms else None, _u64_array(self._offs),
                      C.c_void_p(out.strategies.data_ptr()), s_cap, _table(out.node),
                      _u64_array(self._eoffs), _table(out.edge), e_cap,
                      BUILD_SHARED if shared else 0, _stream(stream))

    def __call__(self) -> None:
        st = self._fn(*self._args)
        if st != OK:
            _check(st, "taps_build_tables")


def build_tables(graph, cluster, device="cuda", stream=None, out: Optional[Tables] = None,
                 shared: bool = False, mesh=None, topology=None, fused: bool = True) -> Tables:
    """Enumeration, node table and edge table of one graph on one cluster.
    ``out``: tables of an earlier build of the same graph to fill again;
    ``shared``: identical edge tables computed once (taps_edge_costs_shared);
    ``mesh``: the strategy space of a fixed device mesh (sizes, innermost
    first) instead of every device matrix; ``topology``: the link classes of a
    workloads.Topology on the cluster's devices instead of its two.  Builds
    with two link classes go through the single call taps_build_tables unless
    ``fused`` is False (then the separate calls run)."""
    g = _graph(graph)
    if fused and topology is None:
        return taps_build_tables(g, cluster, mesh=mesh, out=out, device=device, stream=stream,
                                 shared=shared)
    offs, strat = taps_enumerate_strategies(g, cluster, device=device, stream=stream,
                                            out=out.strategies if out is not None else None,
                                            mesh=mesh)
    if topology is not None:
        if shared:
            raise ValueError("shared tables are built for two link classes only")
        node = taps_node_costs_topology(g, topology, strat, offs, stream=stream,
                                        out=out.node if out is not None else None)
        eoffs, edge = taps_edge_costs_topology(g, topology, strat, offs, stream=stream,
                                               out=out.edge if out is not None else None)
        return Tables(offs, strat, node, eoffs, edge)
    node = taps_node_costs(g, cluster, strat, offs, stream=stream,
                           out=out.node if out is not None else None)
    eoffs, edge = taps_edge_costs(g, cluster, strat, offs, stream=stream,
                                  out=out.edge if out is not None else None, shared=shared)
    return Tables(offs, strat, node, eoffs, edge)


def strategies_to_numpy(strategies) -> Tuple[np.ndarray, np.ndarray]:
    """(log2 degrees uint8 [S, 8], positions int8 [S, 8]) on the host."""
    a = strategies.cpu().numpy()
    return a[:, :MAX_AXES].copy(), a[:, MAX_AXES:].view(np.int8).copy()

"""The C-ABI library on the host: it loads, exports what include/taps.h
declares, validates its arguments before touching the GPU, and sizes tables
(no compute call here -- those need a GPU)."""
import ctypes as C
import subprocess

import numpy as np
import pytest

from paper_2301_04285_amd import taps as T
from paper_2301_04285_amd import workloads as W


@pytest.fixture(scope="module")
def lib():
    return T.load()


def test_exports_every_declared_symbol(lib):
    declared = T.declared_symbols()
    assert declared == sorted(["taps_build_tables", "taps_build_tables_noalloc",
                               "taps_enumerate_strategies", "taps_enumerate_strategies_mesh",
                               "taps_node_costs", "taps_edge_costs", "taps_node_costs_topology",
                               "taps_edge_costs_topology",
                               "taps_edge_costs_shared", "taps_edge_costs_backward",
                               "taps_edge_costs_sweep", "taps_memory_costs",
                               "taps_set_edge_kernel_events", "taps_set_long_segments_min",
                               "taps_status_str",
                               "taps_last_error"])
    out = subprocess.run(["nm", "-D", "--defined-only", T.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for name in declared:
        assert name in exported
        assert getattr(lib, name) is not None


def test_calibration_library_exports_its_header():
    """libtaps_calibrate.so (the benchmark's VALU issue ceiling) exports what
    include/taps_calibrate.h declares, and rejects bad arguments on the host."""
    import os
    import re
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    header = open(os.path.join(root, "include", "taps_calibrate.h")).read()
    declared = re.findall(r"^(?:int |const char \*)(taps_\w+)\(", header, flags=re.M)
    assert declared == ["taps_calibrate_valu_kinds", "taps_calibrate_valu_name",
                        "taps_calibrate_valu"]
    path = os.path.join(root, "paper_2301_04285_amd", "libtaps_calibrate.so")
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True,
                         check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    assert set(declared) <= exported
    cal = C.CDLL(path)
    cal.taps_calibrate_valu.restype = C.c_int
    cal.taps_calibrate_valu_name.restype = C.c_char_p
    kinds = cal.taps_calibrate_valu_kinds()
    assert kinds == 13
    names = [cal.taps_calibrate_valu_name(k).decode() for k in range(kinds)]
    assert names[0] == "v_add_u32 / v_xor_b32" and len(set(names)) == kinds
    assert cal.taps_calibrate_valu_name(kinds) is None and cal.taps_calibrate_valu_name(-1) is None
    ms, n, simds = C.c_float(), C.c_double(), C.c_uint32()
    assert cal.taps_calibrate_valu(kinds, 10, C.byref(ms), C.byref(n), C.byref(simds)) == 1
    assert cal.taps_calibrate_valu(-1, 10, C.byref(ms), C.byref(n), C.byref(simds)) == 1
    assert cal.taps_calibrate_valu(0, 0, C.byref(ms), C.byref(n), C.byref(simds)) == 1
    assert cal.taps_calibrate_valu(0, 10, None, C.byref(n), C.byref(simds)) == 1


def test_kernel_events_need_both_or_neither(lib):
    import ctypes as C
    assert lib.taps_set_edge_kernel_events(C.c_void_p(0x1000), None) == T.ERR_ARG
    assert "both" in T.last_error()
    assert lib.taps_set_edge_kernel_events(None, C.c_void_p(0x1000)) == T.ERR_ARG
    assert lib.taps_set_edge_kernel_events(None, None) == 0


def test_long_segment_threshold_setting(lib):
    # the launch-shape threshold: returns the previous value, default 32768
    prev = T.taps_set_long_segments_min(5)
    assert prev == 32768
    assert T.taps_set_long_segments_min(prev) == 5


def test_status_strings(lib):
    names = [T.status_str(s) for s in range(7)]
    assert names == ["TAPS_OK", "TAPS_ERR_ARG", "TAPS_ERR_TOPOLOGY", "TAPS_ERR_SHAPE",
                     "TAPS_ERR_NO_STRATEGY", "TAPS_ERR_CAPACITY", "TAPS_ERR_DEVICE"]


def _enum(lib, graph, cluster, offs=None):
    g = T.pack_graph(graph)
    cl = T.pack_cluster(cluster) if cluster is not None else None
    if offs is None:
        offs = np.zeros(len(graph.ops) + 1, np.uint64)
    return lib.taps_enumerate_strategies(C.byref(g.struct), C.byref(cl) if cl else None,
                                         T._u64_array(offs), None, 0, None)


@pytest.mark.parametrize("cluster,status", [
    (W.Cluster(3, 2, 10, 1), T.ERR_TOPOLOGY),
    (W.Cluster(2, 6, 10, 1), T.ERR_TOPOLOGY),
    (W.Cluster(0, 2, 10, 1), T.ERR_TOPOLOGY),
    (W.Cluster(64, 8, 10, 1), T.ERR_TOPOLOGY),     # 512 devices > 2^8
    (W.Cluster(2, 2, 0, 1), T.ERR_TOPOLOGY),
    (W.Cluster(2, 2, 10, 0), T.ERR_TOPOLOGY),
])
def test_cluster_validation(lib, cluster, status):
    assert _enum(lib, W.mlp2(), cluster) == status
    assert T.last_error() != ""


def test_null_arguments(lib):
    g = T.pack_graph(W.mlp2())
    cl = T.pack_cluster(W.Cluster(2, 2, 10, 1))
    offs = np.zeros(4, np.uint64)
    assert lib.taps_enumerate_strategies(None, C.byref(cl), T._u64_array(offs), None, 0, None) \
        == T.ERR_ARG
    assert lib.taps_enumerate_strategies(C.byref(g.struct), None, T._u64_array(offs), None, 0,
                                         None) == T.ERR_ARG
    assert lib.taps_enumerate_strategies(C.byref(g.struct), C.byref(cl), None, None, 0, None) \
        == T.ERR_ARG
    eo = np.zeros(3, np.uint64)
    good = np.array([0, 9, 13, 22], np.uint64)
    assert lib.taps_edge_costs(C.byref(g.struct), C.byref(cl), None, None, T._u64_array(eo),
                               T._table(None), 0, None) == T.ERR_ARG
    assert lib.taps_edge_costs(C.byref(g.struct), C.byref(cl), None, T._u64_array(good), None,
                               T._table(None), 0, None) == T.ERR_ARG
    assert lib.taps_node_costs(C.byref(g.struct), C.byref(cl), None, T._u64_array(good),
                               T.Table(1, 1, 1, 1, 1), None) == T.ERR_ARG


@pytest.mark.parametrize("mesh", [
    [4, 2],            # 8 devices on a 16-device cluster
    [8, 2, 2],         # 32 devices
    [3, 4, 4],         # not a power of two
    [1, 16],           # size 1
    [16, 0],
    [2] * 9,           # more dimensions than levels
])
def test_mesh_validation(lib, mesh):
    g = T.pack_graph(W.mlp2())
    cl = T.pack_cluster(W.Cluster(2, 8, 10, 1))
    offs = np.full(4, 7, np.uint64)
    m = T.Mesh(min(len(mesh), 8), (C.c_uint32 * 8)(*mesh[:8]))
    if len(mesh) > 8:
        m.n_dims = len(mesh)
    st = lib.taps_enumerate_strategies_mesh(C.byref(g.struct), C.byref(cl), C.byref(m),
                                            T._u64_array(offs), None, 0, None)
    assert st == T.ERR_TOPOLOGY and T.last_error() != ""
    assert (offs == 7).all()   # nothing written
    assert lib.taps_enumerate_strategies_mesh(C.byref(g.struct), C.byref(cl), None,
                                              T._u64_array(offs), None, 0, None) == T.ERR_ARG


@pytest.mark.parametrize("domains,bw", [
    ((8, 4, 16), (600, 100, 25)),          # not non-decreasing
    ((8, 24), (600, 100)),                 # not a power of two
    ((8, 512), (600, 100)),                # more than 256 devices
    ((8, 32, 128), (600, 0, 25)),          # a zero bandwidth
    ((8, 32, 128), (600, 100, 600000007)), # ratios too fine for exact keys
    ((), ()),                              # no class
    ((1, 2, 4, 8, 16), (5, 4, 3, 2, 1)),   # five classes
])
def test_topology_validation(lib, domains, bw):
    g = T.pack_graph(W.mlp2())
    n = len(domains)
    tp = T.TopologyS(n, (C.c_uint32 * 4)(*domains[:4]), (C.c_uint64 * 4)(*[b * W.GB for b in bw[:4]]),
                     0)
    offs = np.array([0, 9, 13, 22], np.uint64)
    eo = np.full(3, 5, np.uint64)
    assert lib.taps_edge_costs_topology(C.byref(g.struct), C.byref(tp), None, T._u64_array(offs),
                                        T._u64_array(eo), T._table(None), 0, None) == T.ERR_TOPOLOGY
    assert T.last_error() != "" and (eo == 5).all()
    assert lib.taps_node_costs_topology(C.byref(g.struct), C.byref(tp), None, T._u64_array(offs),
                                        T.Table(1, 1, 1, 1, 1), None) == T.ERR_TOPOLOGY
    assert lib.taps_edge_costs_topology(C.byref(g.struct), None, None, T._u64_array(offs),
                                        T._u64_array(eo), T._table(None), 0, None) == T.ERR_ARG


def _op(**kw):
    base = dict(name="x", kind="x", axis_names=("a", "b"), axis_len=(8, 8),
                partitionable=(True, True), dtype_bytes=2, ins=((0, 1),), ws=(), out=(0, 1))
    base.update(kw)
    return W.Op(**base)


@pytest.mark.parametrize("op", [
    _op(out=(0, 2)),                          # axis out of range
    _op(out=(0, 0)),                          # axis named twice
    _op(axis_len=(8, 0)),                     # zero length
    _op(dtype_bytes=0),
    _op(axis_len=(1 << 30, 1 << 30)),         # 2^61 bytes: volumes would not stay exact
])
def test_operator_validation(lib, op):
    g = W.Graph()
    object.__setattr__(op, "check", lambda: None)
    g.ops.append(op)
    assert _enum(lib, g, W.Cluster(2, 2, 10, 1)) == T.ERR_ARG


def _size_query(lib, graph, offs, cluster=W.Cluster(2, 2, 10, 1)):
    g = T.pack_graph(graph)
    cl = T.pack_cluster(cluster)
    eo = np.zeros(len(graph.edges) + 1, np.uint64)
    st = lib.taps_edge_costs(C.byref(g.struct), C.byref(cl), None,
                             T._u64_array(np.asarray(offs, np.uint64)), T._u64_array(eo),
                             T._table(None), 0, None)
    return st, eo


def test_edge_shape_mismatch(lib):
    g = W.mlp2()
    bad = W.Graph(list(g.ops), [W.Edge(0, 2, 0)])   # (64, 1024) into (64, 1024)? mm2.X is (64,1024)
    st, _ = _size_query(lib, bad, [0, 9, 13, 22])
    assert st == T.OK
    bad = W.Graph(list(g.ops), [W.Edge(2, 0, 0)])   # (64, 256) into mm1.X (64, 256): fine
    assert _size_query(lib, bad, [0, 9, 13, 22])[0] == T.OK
    bad = W.Graph(list(g.ops), [W.Edge(1, 0, 0)])   # (64, 1024) into (64, 256)
    assert _size_query(lib, bad, [0, 9, 13, 22])[0] == T.ERR_SHAPE
    bad = W.Graph(list(g.ops), [W.Edge(0, 1, 1)])   # gelu has one input
    assert _size_query(lib, bad, [0, 9, 13, 22])[0] == T.ERR_ARG
    bad = W.Graph(list(g.ops), [W.Edge(0, 5, 0)])
    assert _size_query(lib, bad, [0, 9, 13, 22])[0] == T.ERR_ARG


def test_edge_size_query_offsets(lib):
    g = W.gpt(2, 64, 4, 32, 4, 2)
    rng = np.random.default_rng(0)
    counts = rng.integers(1, 50, len(g.ops))
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.uint64)
    st, eo = _size_query(lib, g, offs)
    assert st == T.OK
    want = np.concatenate([[0], np.cumsum([counts[e.src] * counts[e.dst] for e in g.edges])])
    assert np.array_equal(eo, want.astype(np.uint64))
    assert len(g.edges) == 18 * 2 - 2


def test_offsets_must_increase(lib):
    st, _ = _size_query(lib, W.mlp2(), [0, 9, 9, 18])
    assert st == T.ERR_ARG
    st, _ = _size_query(lib, W.mlp2(), [1, 9, 13, 22])
    assert st == T.ERR_ARG


def test_capacity_and_partial_tables(lib):
    g = T.pack_graph(W.mlp2())
    cl = T.pack_cluster(W.Cluster(2, 2, 10, 1))
    offs = np.array([0, 9, 13, 22], np.uint64)
    eo = np.zeros(3, np.uint64)
    fake = T.Table(256, 256, 256, 256, 256)   # never dereferenced: the checks fail first
    partial = T.Table(256, None, 256, 256, 256)
    for fn in (lib.taps_edge_costs, lib.taps_edge_costs_shared, lib.taps_edge_costs_backward):
        assert fn(C.byref(g.struct), C.byref(cl), C.c_void_p(256), T._u64_array(offs),
                  T._u64_array(eo), fake, 71, None) == T.ERR_CAPACITY
        assert np.all(eo == 0)   # nothing written on error
        assert fn(C.byref(g.struct), C.byref(cl), C.c_void_p(256), T._u64_array(offs),
                  T._u64_array(eo), partial, 72, None) == T.ERR_ARG


def test_noalloc_rejects_a_build_beyond_its_workspace(lib):
    """taps_build_tables_noalloc refuses, on the host and before any HIP call, a
    build whose device workspace exceeds its fixed array (a 400-layer GPT on 128
    devices: its strategy descriptors alone take 40 MB, shared tables or not),
    and writes no offsets; its size query answers as taps_build_tables does."""
    g = T.pack_graph(W.gpt(400, 12288, 96, 2048, 64, 2))
    cl = T.pack_cluster(W.config(5).clusters[0][1])
    none = T.Table(None, None, None, None, None)
    offs = np.zeros(g.n_ops + 1, np.uint64)
    eo = np.zeros(g.n_edges + 1, np.uint64)
    assert lib.taps_build_tables_noalloc(C.byref(g.struct), C.byref(cl), None, T._u64_array(offs),
                                         None, 0, none, T._u64_array(eo), none, 0, 0, None) == 0
    offs2 = np.zeros_like(offs)
    eo2 = np.zeros_like(eo)
    assert lib.taps_build_tables(C.byref(g.struct), C.byref(cl), None, T._u64_array(offs2),
                                 None, 0, none, T._u64_array(eo2), none, 0, 0, None) == 0
    assert np.array_equal(offs, offs2) and np.array_equal(eo, eo2)
    fake = T.Table(256, 256, 256, 256, 256)   # never dereferenced: the check fails first
    offs3 = np.zeros_like(offs)
    eo3 = np.zeros_like(eo)
    for flags in (0, T.BUILD_SHARED):
        st = lib.taps_build_tables_noalloc(C.byref(g.struct), C.byref(cl), None,
                                           T._u64_array(offs3), C.c_void_p(256), int(offs[-1]),
                                           fake, T._u64_array(eo3), fake, int(eo[-1]), flags, None)
        assert st == T.ERR_CAPACITY
        assert "fixed workspace" in T.last_error()
        assert np.all(offs3 == 0) and np.all(eo3 == 0)   # nothing written on error


def test_shared_size_query_matches(lib):
    g = T.pack_graph(W.gpt(2, 64, 4, 32, 4, 2))
    cl = T.pack_cluster(W.Cluster(2, 2, 10, 1))
    counts = np.random.default_rng(1).integers(1, 50, g.n_ops)
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.uint64)
    a, b = np.zeros(g.n_edges + 1, np.uint64), np.zeros(g.n_edges + 1, np.uint64)
    none = T.Table(None, None, None, None, None)
    assert lib.taps_edge_costs(C.byref(g.struct), C.byref(cl), None, T._u64_array(offs),
                               T._u64_array(a), none, 0, None) == T.OK
    assert lib.taps_edge_costs_shared(C.byref(g.struct), C.byref(cl), None, T._u64_array(offs),
                                      T._u64_array(b), none, 0, None) == T.OK
    assert np.array_equal(a, b)


def _sweep(lib, clusters, n=None, tables=None, capacity=0, graph=None, offs=None):
    g = T.pack_graph(graph or W.mlp2())
    offs = np.asarray(offs if offs is not None else [0, 9, 13, 22], np.uint64)
    arr = (T.Cluster * max(len(clusters), 1))(*[T.pack_cluster(c) for c in clusters])
    eo = np.zeros(g.n_edges + 1, np.uint64)
    tabs = None if tables is None else (T.Table * len(tables))(*tables)
    st = lib.taps_edge_costs_sweep(C.byref(g.struct), arr, len(clusters) if n is None else n,
                                   C.c_void_p(256), T._u64_array(offs), T._u64_array(eo), tabs,
                                   capacity, None)
    return st, eo


def test_sweep_size_query_matches_single_point(lib):
    g = W.gpt(2, 64, 4, 32, 4, 2)
    counts = np.random.default_rng(2).integers(1, 50, len(g.ops))
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.uint64)
    pts = [W.Cluster(2, 2, 100 * W.GB, b * W.GB) for b in (12, 25, 50, 100)]
    st, eo = _sweep(lib, pts, graph=g, offs=offs)
    assert st == T.OK
    st1, eo1 = _size_query(lib, g, offs, pts[0])
    assert st1 == T.OK and np.array_equal(eo, eo1)
    none = T.Table(None, None, None, None, None)
    st, eo2 = _sweep(lib, pts, tables=[none] * 4, graph=g, offs=offs)
    assert st == T.OK and np.array_equal(eo2, eo1)


def test_sweep_argument_checks(lib):
    a, b = W.Cluster(2, 2, 10, 1), W.Cluster(2, 2, 20, 3)
    fake = T.Table(256, 256, 256, 256, 256)
    assert _sweep(lib, [a, b], n=0)[0] == T.ERR_ARG
    assert _sweep(lib, [a] * 9)[0] == T.ERR_ARG
    assert "bandwidth points" in T.last_error()
    st, eo = _sweep(lib, [a, W.Cluster(4, 1, 10, 1)], tables=[fake, fake], capacity=72)
    assert st == T.ERR_ARG and "point 1" in T.last_error() and np.all(eo == 0)
    assert _sweep(lib, [a, W.Cluster(2, 2, 0, 1)])[0] == T.ERR_TOPOLOGY
    none = T.Table(None, None, None, None, None)
    st, eo = _sweep(lib, [a, b], tables=[fake, none], capacity=72)
    assert st == T.ERR_ARG and np.all(eo == 0)
    st, eo = _sweep(lib, [a, b], tables=[fake, fake], capacity=71)
    assert st == T.ERR_CAPACITY and np.all(eo == 0)


def test_memory_costs_argument_checks(lib):
    g = T.pack_graph(W.mlp2())
    offs = np.array([0, 9, 13, 22], np.uint64)
    assert lib.taps_memory_costs(C.byref(g.struct), C.c_void_p(256), T._u64_array(offs), None,
                                 None) == T.ERR_ARG
    assert "memory" in T.last_error()
    assert lib.taps_memory_costs(C.byref(g.struct), None, T._u64_array(offs), C.c_void_p(256),
                                 None) == T.ERR_ARG
    assert lib.taps_memory_costs(C.byref(g.struct), C.c_void_p(256),
                                 T._u64_array(np.array([0, 9, 9, 18], np.uint64)),
                                 C.c_void_p(256), None) == T.ERR_ARG
    assert lib.taps_memory_costs(None, C.c_void_p(256), T._u64_array(offs), C.c_void_p(256),
                                 None) == T.ERR_ARG
    empty = T.pack_graph(W.Graph())   # no strategies: nothing to do, NULL buffers allowed
    assert lib.taps_memory_costs(C.byref(empty.struct), None, T._u64_array(np.zeros(1, np.uint64)),
                                 None, None) == T.OK


def test_device_errors_are_reported(lib):
    """Without a usable device every compute call returns TAPS_ERR_DEVICE
    (on a GPU machine this test is skipped)."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    g = T.pack_graph(W.mlp2())
    cl = T.pack_cluster(W.Cluster(2, 2, 10, 1))
    offs = np.zeros(4, np.uint64)
    # the size query is computed on the host; writing the strategies needs the device
    assert lib.taps_enumerate_strategies(C.byref(g.struct), C.byref(cl), T._u64_array(offs),
                                         None, 0, None) == T.OK
    assert list(offs) == [0, 9, 13, 22]
    assert lib.taps_enumerate_strategies(C.byref(g.struct), C.byref(cl), T._u64_array(offs),
                                         C.c_void_p(256), 22, None) == T.ERR_DEVICE
    assert "hip" in T.last_error().lower()


def test_build_size_query_counts_like_the_oracle(lib, oracle_lib):
    """taps_build_tables sizes every table on the host (an exact count of the
    enumeration filter, no GPU): its offsets equal the oracle's strategy counts
    and the row-major edge sizes, with and without a fixed mesh."""
    import random
    rng = random.Random(808)
    checked = 0
    for trial in range(60):
        g = W.random_graph(rng, rng.randint(1, 6), max_axes=6, max_rank=4, len_pow_range=(0, 9))
        n = rng.randint(0, 8)
        L = 1 << rng.randint(0, n)
        cl = W.Cluster((1 << n) // L, L, 600 * W.GB, 100 * W.GB)
        mesh = None
        if rng.random() < 0.5:
            mesh, left = [], n
            while left:
                e = rng.randint(1, min(3, left))
                mesh.append(1 << e)
                left -= e
        counts = [len(oracle_lib.enumerate_strategies(op, cl.devices) if mesh is None else
                      oracle_lib.enumerate_strategies_mesh(op, mesh)) for op in g.ops]
        try:
            offs, eoffs = T.taps_build_tables(g, cl, mesh=mesh, size_only=True)
        except T.TapsError as ex:
            assert ex.status == T.ERR_NO_STRATEGY and 0 in counts
            continue
        assert list(np.diff(offs)) == counts, (trial, mesh)
        assert list(np.diff(eoffs)) == [counts[e.src] * counts[e.dst] for e in g.edges]
        checked += 1
    # the workloads (every view and mesh)
    for k in W.ALL_CONFIGS:
        w = W.config(k)
        for _, cl in w.clusters:
            for mesh in (None, W.physical_mesh(k, cl)):
                offs, _ = T.taps_build_tables(w.graph, cl, mesh=mesh, size_only=True)
                got = np.diff(offs)
                for op_i in range(min(len(w.graph.ops), 20)):
                    op = w.graph.ops[op_i]
                    ref = (oracle_lib.enumerate_strategies(op, cl.devices) if mesh is None else
                           oracle_lib.enumerate_strategies_mesh(op, mesh))
                    assert got[op_i] == len(ref)
    assert checked > 30

"""GPU tables against the CPU oracle, through the C ABI.

Integers (vol, intra, inter, meta) must be identical; t within 1e-9
relative.  Small configurations are compared entry by entry in full; the
96-layer configuration (9.9e7 edge entries) is built in full on the GPU in
the same launch configuration the benchmark times and compared on seeded
samples the oracle computes one by one, plus properties checked over every
entry.
"""
import random
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2301_04285_amd import workloads as W

pytestmark = pytest.mark.gpu

RTOL = 1e-9


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def T():
    import torch
    from paper_2301_04285_amd import taps
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    taps.load()
    return taps


def _np(t):
    import torch
    if t.dtype == torch.uint64:
        return t.view(torch.int64).cpu().numpy().view(np.uint64)
    if t.dtype == torch.uint32:
        return t.view(torch.int32).cpu().numpy().view(np.uint32)
    return t.cpu().numpy()


def _signed(t):
    import torch
    return {torch.uint64: lambda: t.view(torch.int64),
            torch.uint32: lambda: t.view(torch.int32)}.get(t.dtype, lambda: t)()


def _host(tab):
    return {k: _np(v) for k, v in tab.items()}


def assert_records(got, ref, where=""):
    """got: dict of numpy arrays; ref: oracle RECORD_DTYPE array (same order)."""
    ref = ref.ravel()
    for f in ("vol", "intra", "inter", "meta"):
        bad = np.flatnonzero(got[f] != ref[f])
        assert bad.size == 0, (f"{where}: {f} differs at {bad[:5]}: "
                               f"gpu {got[f][bad[:5]]} oracle {ref[f][bad[:5]]}")
    denom = np.maximum(np.abs(ref["t"]), np.finfo(np.float64).tiny)
    rel = np.abs(got["t"] - ref["t"]) / denom
    bad = np.flatnonzero(rel > RTOL)
    assert bad.size == 0, f"{where}: t differs at {bad[:5]}: {got['t'][bad[:5]]} vs {ref['t'][bad[:5]]}"


def _oracle_strategies(op, cluster, mesh=None):
    if mesh is None:
        return O.enumerate_strategies(op, cluster.devices)
    return O.enumerate_strategies_mesh(op, mesh)


def check_strategies(T, graph, cluster, offs, strat, mesh=None):
    lg, pos = T.strategies_to_numpy(strat)
    for k, op in enumerate(graph.ops):
        ref = _oracle_strategies(op, cluster, mesh)
        a, b = int(offs[k]), int(offs[k + 1])
        assert b - a == len(ref), op.name
        deg = np.where(pos[a:b, :op.n_axes] >= 0, 1 << lg[a:b, :op.n_axes].astype(np.int64), 1)
        assert np.array_equal(deg, ref["degree"][:, :op.n_axes]), op.name
        assert np.array_equal(pos[a:b, :op.n_axes], ref["pos"][:, :op.n_axes]), op.name
        assert np.all(lg[a:b, op.n_axes:] == 0) and np.all(pos[a:b, op.n_axes:] == -1)
    return [_oracle_strategies(op, cluster, mesh) for op in graph.ops]


def full_check(T, graph, cluster, name, mesh=None):
    import torch
    say(f"[gpu] build {name}")
    tabs = T.build_tables(graph, cluster, mesh=mesh)
    torch.cuda.synchronize()
    say(f"[gpu] built {name}: {int(tabs.edge_offsets[-1])} edge entries")
    ref_strats = check_strategies(T, graph, cluster, tabs.op_offsets, tabs.strategies, mesh)
    node = _host(tabs.node)
    edge = _host(tabs.edge)
    for k, op in enumerate(graph.ops):
        a, b = int(tabs.op_offsets[k]), int(tabs.op_offsets[k + 1])
        ref = O.node_table(op, ref_strats[k], cluster)
        assert_records({f: v[a:b] for f, v in node.items()}, ref, f"{name} node {k} {op.name}")
    for x, e in enumerate(graph.edges):
        a, b = int(tabs.edge_offsets[x]), int(tabs.edge_offsets[x + 1])
        ref = O.edge_table(graph.ops[e.src], ref_strats[e.src], graph.ops[e.dst], e.slot,
                           ref_strats[e.dst], cluster)
        assert_records({f: v[a:b] for f, v in edge.items()}, ref, f"{name} edge {x}")
    return tabs


@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_full_tables_small_configs(T, cfg):
    w = W.config(cfg)
    for name, cl in w.clusters:
        full_check(T, w.graph, cl, f"{w.name}/{name}")


def test_full_tables_config3_both_views(T):
    w = W.config(3)
    for name, cl in w.clusters:
        full_check(T, w.graph, cl, f"{w.name}/{name}")


def test_long_segments_on_small_configs(T):
    """The long-segment launch shape (eight-tile row segments, each edge's
    full-length ones first, the rows' remainders last, longest first), which
    only launches of at least 32,768 segments take by default, forced on
    configurations 1-4 and random graphs and compared with the oracle in full."""
    prev = T.taps_set_long_segments_min(1)
    try:
        for cfg in (1, 2, 3, 4):
            w = W.config(cfg)
            for name, cl in w.clusters:
                full_check(T, w.graph, cl, f"long segments {w.name}/{name}")
        from paper_2301_04285_amd.taps import TapsError
        for k, (g, cl) in enumerate(_random_cases(7, 12)):
            try:
                full_check(T, g, cl, f"long segments random {k}")
            except TapsError as ex:
                assert ex.status == T.ERR_NO_STRATEGY
    finally:
        T.taps_set_long_segments_min(prev)


def test_largest_config_sampled(T):
    """The 96-layer GPT on 16 x 8 devices, built whole in HBM."""
    import torch
    w = W.config(5)
    name, cl = w.clusters[0]
    g = w.graph
    say(f"[gpu] build {w.name}/{name}")
    tabs = T.build_tables(g, cl)
    torch.cuda.synchronize()
    total = int(tabs.edge_offsets[-1])
    say(f"[gpu] built {total} edge entries")
    assert total == 98_668_128
    ref_strats = check_strategies(T, g, cl, tabs.op_offsets, tabs.strategies)
    # node tables in full
    node = _host(tabs.node)
    for k, op in enumerate(g.ops):
        a, b = int(tabs.op_offsets[k]), int(tabs.op_offsets[k + 1])
        assert_records({f: v[a:b] for f, v in node.items()},
                       O.node_table(op, ref_strats[k], cl), f"node {k}")
    # properties over every entry
    meta = tabs.edge["meta"].view(torch.int32)
    assert int((meta == -1).sum()) == 0, "an entry's sequence did not settle"
    assert int(((meta & 3) == 3).sum()) == 0
    vol = tabs.edge["vol"].view(torch.int64).double()
    t = tabs.edge["t"]
    assert bool((t >= vol / (cl.devices * cl.bw_intra) * (1 - 1e-12)).all())
    # seeded samples: every edge's first, last and a tile-boundary entry,
    # plus random entries of 64 random edges
    rng = random.Random(96)
    edge = tabs.edge
    deep = set(rng.sample(range(len(g.edges)), 64))
    picks = []
    for x, e in enumerate(g.edges):
        ns, nd = len(ref_strats[e.src]), len(ref_strats[e.dst])
        cand = {0, ns * nd - 1, min(ns * nd - 1, 255), min(ns * nd - 1, 256)}
        if x in deep:
            cand |= {rng.randrange(ns * nd) for _ in range(1500)}
        picks.append(sorted(cand))
    checked = 0
    for x, e in enumerate(g.edges):
        nd = len(ref_strats[e.dst])
        loc = np.array(picks[x], dtype=np.int64)
        glob = torch.from_numpy(loc + int(tabs.edge_offsets[x])).to(t.device)
        got = {f: _np(_signed(v).index_select(0, glob).view(v.dtype)) for f, v in edge.items()}
        ref = O.edge_entries(g.ops[e.src], ref_strats[e.src], g.ops[e.dst], e.slot,
                             ref_strats[e.dst], loc // nd, loc % nd, cl)
        assert_records(got, ref, f"edge {x}")
        checked += len(loc)
    say(f"[gpu] checked {checked} sampled entries")
    assert checked > 90_000


def test_largest_config_full_oracle(T):
    """Every one of the 96-layer GPT's 98,668,128 edge entries against the
    oracle, built by the benchmark's call (taps_build_tables: long row segments,
    the rows' remainders launched last).  The oracle's edge tables are computed
    by a pool of host threads (its calls release the interpreter lock) and each
    is compared with the GPU's slice as it arrives."""
    import os
    from concurrent.futures import ThreadPoolExecutor

    import torch
    w = W.config(5)
    name, cl = w.clusters[0]
    g = w.graph
    say(f"[gpu] build {w.name}/{name} for the full oracle comparison")
    tabs = T.build_tables(g, cl)
    torch.cuda.synchronize()
    total = int(tabs.edge_offsets[-1])
    assert total == 98_668_128
    edge = _host(tabs.edge)
    del tabs
    strats = [O.enumerate_strategies(op, cl.devices) for op in g.ops]
    eoff = [0]
    for e in g.edges:
        eoff.append(eoff[-1] + len(strats[e.src]) * len(strats[e.dst]))
    assert eoff[-1] == total

    def one(x):
        e = g.edges[x]
        ref = O.edge_table(g.ops[e.src], strats[e.src], g.ops[e.dst], e.slot, strats[e.dst], cl)
        a, b = eoff[x], eoff[x + 1]
        assert_records({f: v[a:b] for f, v in edge.items()}, ref, f"edge {x}")
        return b - a

    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    compared = 0
    with ThreadPoolExecutor(threads) as pool:
        for k, n in enumerate(pool.map(one, range(len(g.edges)))):
            compared += n
            if k % 200 == 199:
                say(f"[gpu] {k + 1} of {len(g.edges)} edges equal to the oracle ({compared} entries)")
    say(f"[gpu] all {compared} edge entries equal to the oracle ({threads} host threads)")
    assert compared == 98_668_128


def _entries(g, N):
    counts = [len(O.enumerate_strategies(op, N)) for op in g.ops]
    return sum(counts[e.src] * counts[e.dst] for e in g.edges)


def _random_cases(seed, count, max_entries=400_000):
    """Seeded random graphs on random meshes (N = 1..256), each small enough
    for the oracle to check in full."""
    rng = random.Random(seed)
    made = 0
    while made < count:
        g = W.random_graph(rng, rng.randint(2, 7), max_axes=6, max_rank=5, len_pow_range=(0, 9))
        n = rng.randint(0, 8)
        L = 1 << rng.randint(0, n)
        N = 1 << n
        if _entries(g, N) > max_entries:
            continue
        made += 1
        yield g, W.Cluster(N // L, L, rng.choice([600, 400, 200, 25]) * W.GB,
                           int(rng.choice([100, 50, 12.5, 6]) * W.GB))


def test_random_graphs_and_meshes(T):
    from paper_2301_04285_amd.taps import TapsError
    done = 0
    for k, (g, cl) in enumerate(_random_cases(2301, 40)):
        try:
            full_check(T, g, cl, f"random {k} N={cl.devices} L={cl.devices_per_node}")
        except TapsError as ex:
            assert ex.status == T.ERR_NO_STRATEGY
            assert any(len(O.enumerate_strategies(op, cl.devices)) == 0 for op in g.ops)
            continue
        done += 1
    assert done >= 20


def _within_tensor_limit(g):
    """Every tensor of g within the library's 2^40-byte bound."""
    for op in g.ops:
        for t in (op.out, *op.ins, *op.ws):
            size = op.dtype_bytes
            for a in t:
                size *= op.axis_len[a]
            if size > 1 << 40:
                return False
    return True


def test_high_rank_tensors(T):
    """Edges carrying tensors of rank 5 to 8 (the launches that cannot use the
    kernels compiled for rank 4 at most), beside edges of low rank in the same
    graph: the two-class tables entry by entry, the bandwidth sweep (with a
    point whose exact order needs 128-bit keys) and the link-class tables,
    against the oracle."""
    from paper_2301_04285_amd.taps import TapsError
    rng = random.Random(4285)
    done, top_rank = 0, 0
    while done < 10:
        g = W.random_graph(rng, rng.randint(2, 5), max_axes=8, max_rank=8, len_pow_range=(1, 6))
        n = rng.randint(1, 6)
        L = 1 << rng.randint(0, n)
        cl = W.Cluster((1 << n) // L, L, rng.choice([600, 200]) * W.GB,
                       rng.choice([100, 25]) * W.GB)
        rank = max((len(g.ops[e.src].out) for e in g.edges), default=0)
        if rank <= 4 or not _within_tensor_limit(g) or _entries(g, cl.devices) > 300_000:
            continue
        name = f"rank {rank} graph {done} N={cl.devices} L={cl.devices_per_node}"
        try:
            full_check(T, g, cl, name)
        except TapsError as ex:
            assert ex.status == T.ERR_NO_STRATEGY
            continue
        if done % 2 == 0:
            # the second point's reduced bandwidths exceed 2^32 (128-bit keys)
            sweep_check(T, g, [cl, W.Cluster(cl.nodes, cl.devices_per_node, (1 << 40) + 1, 3)],
                        name)
        else:
            domains = (cl.devices_per_node, cl.devices) if cl.nodes > 1 else (cl.devices,)
            bws = (cl.bw_intra, cl.bw_inter)[:len(domains)]
            _topology_check(T, g, cl, W.Topology(domains, bws), name)
        top_rank = max(top_rank, rank)
        done += 1
    assert top_rank == 8


def test_degenerate_clusters(T):
    g = W.gpt(1, 64, 4, 32, 4, 2)
    for cl in (W.Cluster(1, 1, 10, 1),        # one device: one whole strategy per op
               W.Cluster(16, 1, 300, 7),      # one device per node
               W.Cluster(1, 16, 300, 7)):     # a single node
        full_check(T, g, cl, f"gpt1 N={cl.devices} L={cl.devices_per_node}")
    # 256 devices, the largest mesh: batch x sequence must split 256 ways
    g = W.gpt(1, 64, 2, 128, 2, 2)
    for cl in (W.Cluster(2, 128, 300, 7), W.Cluster(32, 8, 300, 7), W.Cluster(256, 1, 300, 7)):
        full_check(T, g, cl, f"gpt1-s128 N={cl.devices} L={cl.devices_per_node}")


def _random_mesh(rng, n):
    dims, left = [], n
    while left:
        e = rng.randint(1, min(3, left))
        dims.append(1 << e)
        left -= e
    return dims


def test_fixed_mesh_spaces(T):
    """taps_enumerate_strategies_mesh and the tables over its strategies: the
    workloads on their meshes (the 4 x 4 x 8 and 2 x 4 x 8 meshes with the node's
    8 devices innermost), the 2 x 2 and 4 meshes of Table 3, and random graphs on
    random meshes."""
    cases = [(W.config(1).graph, W.config(1).clusters[0][1], [2, 2]),
             (W.config(1).graph, W.config(1).clusters[0][1], [4]),
             (W.config(2).graph, W.config(2).clusters[0][1], [8, 2]),
             (W.config(3).graph, W.config(3).clusters[0][1], [8, 4]),
             (W.config(3).graph, W.config(3).clusters[1][1], [16, 2]),
             (W.config(4).graph, W.config(4).clusters[0][1], [8, 4, 2]),
             (W.config(5).graph, W.config(5).clusters[0][1], [8, 4, 4])]
    for g, cl, mesh in cases:
        full_check(T, g, cl, f"{len(g.ops)} ops N={cl.devices} mesh={mesh}", mesh=mesh)
    rng = random.Random(4488)
    done = 0
    for k, (g, cl) in enumerate(_random_cases(4488, 16)):
        mesh = _random_mesh(rng, cl.devices.bit_length() - 1)
        try:
            full_check(T, g, cl, f"random {k} N={cl.devices} mesh={mesh}", mesh=mesh)
        except T.TapsError as ex:
            assert ex.status == T.ERR_NO_STRATEGY
            assert any(len(O.enumerate_strategies_mesh(op, mesh)) == 0 for op in g.ops)
            continue
        done += 1
    assert done >= 8


def _topology_check(T, graph, cluster, topo, name, sample=None):
    """Tables under link classes against the oracle: every entry, or `sample`
    seeded entries per edge."""
    import torch
    say(f"[gpu] build {name} under {topo}")
    tabs = T.build_tables(graph, cluster, topology=topo)
    torch.cuda.synchronize()
    strats = check_strategies(T, graph, cluster, tabs.op_offsets, tabs.strategies)
    node = _host(tabs.node)
    for k, op in enumerate(graph.ops):
        a, b = int(tabs.op_offsets[k]), int(tabs.op_offsets[k + 1])
        assert_records({f: v[a:b] for f, v in node.items()},
                       O.node_table_topo(op, strats[k], topo), f"{name} node {k}")
    rng = np.random.default_rng(99)
    for x, e in enumerate(graph.edges):
        a, b = int(tabs.edge_offsets[x]), int(tabs.edge_offsets[x + 1])
        src, dst = graph.ops[e.src], graph.ops[e.dst]
        if sample is None:
            got = {f: _np(v[a:b]) for f, v in tabs.edge.items()}
            ref = O.edge_table_topo(src, strats[e.src], dst, e.slot, strats[e.dst], topo)
        else:
            nd = len(strats[e.dst])
            loc = np.unique(np.concatenate([[0, b - a - 1], rng.integers(0, b - a, sample)]))
            glob = torch.from_numpy(loc + a).to(tabs.edge["t"].device)
            got = {f: _np(_signed(v).index_select(0, glob).view(v.dtype))
                   for f, v in tabs.edge.items()}
            ref = O.edge_entries_topo(src, strats[e.src], dst, e.slot, strats[e.dst], loc // nd,
                                      loc % nd, topo)
        assert_records(got, ref, f"{name} edge {x}")
    return tabs


def _random_topology(rng, n):
    k = rng.randint(1, 4)
    sizes = sorted(rng.randint(0, n) for _ in range(k - 1)) + [n]
    bw = [rng.choice([600, 400, 100, 50, 25, 12]) * W.GB for _ in range(k)]
    a2a = rng.choice([0, 0, 1200 * W.GB, 7 * 150 * W.GB, 50 * W.GB])
    return W.Topology(tuple(1 << e for e in sizes), tuple(bw), a2a)


def test_link_class_tables(T):
    """taps_node_costs_topology / taps_edge_costs_topology against the oracle: the
    three-class topologies of the wide MLP and (one layer, then the whole graph on
    samples) the 96-layer GPT, random graphs under random topologies, and the
    two-class topology, which must give exactly the tables of taps_edge_costs."""
    import torch
    for k in (4, 5):
        w = W.config(k)
        cl = w.clusters[0][1]
        g = w.graph if k == 4 else W.leading_ops(w.graph, 28)
        topo = W.CONFIG_TOPOLOGIES[k]
        _topology_check(T, g, cl, topo, f"{w.name}")
        # in-node AllToAlls over all seven links of an 8-device node
        _topology_check(T, g, cl, W.Topology(topo.domains, topo.bw, 7 * 150 * W.GB), f"{w.name}")
    w = W.config(5)
    _topology_check(T, w.graph, w.clusters[0][1], W.CONFIG_TOPOLOGIES[5], w.name, sample=40)
    rng = random.Random(5150)
    done = 0
    for k, (g, cl) in enumerate(_random_cases(5150, 24)):
        topo = _random_topology(rng, cl.devices.bit_length() - 1)
        try:
            _topology_check(T, g, cl, topo, f"random {k} N={cl.devices}")
        except T.TapsError as ex:
            assert ex.status in (T.ERR_NO_STRATEGY, T.ERR_TOPOLOGY)
            continue
        done += 1
    assert done >= 12
    for cfg in (1, 2, 4):
        w = W.config(cfg)
        cl = w.clusters[0][1]
        a = T.build_tables(w.graph, cl)
        b = T.build_tables(w.graph, cl, topology=W.Topology.of(cl))
        torch.cuda.synchronize()
        assert _same_tables(a.edge, b.edge) and _same_tables(a.node, b.node), w.name


def test_fused_build_equals_separate_calls(T):
    """taps_build_tables (host-sized, one call, no synchronisation) writes exactly
    what taps_enumerate_strategies(_mesh) + taps_node_costs + taps_edge_costs
    write, with and without TAPS_BUILD_SHARED: every configuration (both
    32-device views, every bandwidth), the workloads on their meshes, and random
    graphs on random meshes; a second build into the same tables, queued right
    behind the first, gives the same bits."""
    import torch
    cases = []
    for k in W.ALL_CONFIGS:
        w = W.config(k)
        for _, cl in w.clusters:
            cases.append((w.graph, cl, None))
        cases.append((w.graph, w.clusters[0][1], W.physical_mesh(k, w.clusters[0][1])))
    rng = random.Random(616)
    for g, cl in _random_cases(616, 16):
        cases.append((g, cl, _random_mesh(rng, cl.devices.bit_length() - 1) if rng.random() < 0.5
                      else None))
    for g, cl, mesh in cases:
        name = f"{len(g.ops)} ops N={cl.devices} L={cl.devices_per_node} mesh={mesh}"
        say(f"[gpu] fused build {name}")
        try:
            a = T.build_tables(g, cl, mesh=mesh, fused=False)
        except T.TapsError as ex:
            assert ex.status == T.ERR_NO_STRATEGY
            with pytest.raises(T.TapsError):
                T.build_tables(g, cl, mesh=mesh)
            continue
        b = T.build_tables(g, cl, mesh=mesh)
        T.build_tables(g, cl, mesh=mesh, out=b)   # queued behind the first
        c = T.build_tables(g, cl, mesh=mesh, shared=True)   # identical tables computed once
        torch.cuda.synchronize()
        assert list(a.op_offsets) == list(b.op_offsets) and list(a.edge_offsets) == list(b.edge_offsets)
        assert torch.equal(a.strategies, b.strategies), name
        assert _same_tables(a.node, b.node) and _same_tables(a.edge, b.edge), name
        assert _same_tables(a.edge, c.edge) and _same_tables(a.node, c.node), name


def test_prepared_build_repeats_the_build(T):
    """PreparedBuild (arguments packed once) fills the tables it was given with
    what taps_build_tables writes, full and shared, on every call: three calls in
    a row into cleared tables."""
    import torch
    for k in (2, 4):
        w = W.config(k)
        cl = w.clusters[-1][1]
        a = T.build_tables(w.graph, cl)
        for shared in (False, True):
            say(f"[gpu] prepared build {w.name} shared={shared}")
            b = T.taps_build_tables(w.graph, cl)
            run = T.PreparedBuild(w.graph, cl, b, shared=shared)
            for _ in range(3):
                for v in (*b.node.values(), *b.edge.values()):
                    _signed(v).fill_(-1)
                b.strategies.fill_(0)
                run()
                torch.cuda.synchronize()
                assert torch.equal(a.strategies, b.strategies), w.name
                assert _same_tables(a.node, b.node) and _same_tables(a.edge, b.edge), w.name


def test_concurrent_builds_streams_and_staging(T):
    """Single-call builds (full and shared) from 7 threads at once on 5 streams
    (two pairs of threads share a stream); one build on each of 20 streams in
    turn (more streams than the library keeps scratch blocks for); and 12
    builds queued on one stream behind a bounded spin kernel (more uploads in
    flight than there are staging buffers).  Every table equals the same build
    made alone."""
    import threading
    import torch
    cases = [(W.config(k).graph, W.config(k).clusters[0][1]) for k in (2, 3, 4)]
    refs = [T.build_tables(g, cl) for g, cl in cases]
    torch.cuda.synchronize()

    def same(c, got):
        ref = refs[c]
        return (list(got.op_offsets) == list(ref.op_offsets) and
                torch.equal(got.strategies, ref.strategies) and
                _same_tables(got.node, ref.node) and _same_tables(got.edge, ref.edge))

    streams = [torch.cuda.Stream() for _ in range(5)]
    results, errors = {}, []

    def work(t):
        try:
            s = streams[t % len(streams)]
            outs = []
            with torch.cuda.stream(s):
                for k in range(6):
                    c = (t + k) % len(cases)
                    outs.append((c, T.build_tables(*cases[c], stream=s, shared=k % 2 == 1)))
            s.synchronize()
            results[t] = outs
        except Exception as ex:   # reported below, in the test's thread
            errors.append(f"thread {t}: {ex!r}")

    say("[gpu] concurrent builds: 7 threads on 5 streams")
    threads = [threading.Thread(target=work, args=(t,)) for t in range(7)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=60)
    assert not errors, errors
    assert sorted(results) == list(range(7))
    for t, outs in results.items():
        for k, (c, got) in enumerate(outs):
            assert same(c, got), f"thread {t} build {k} (case {c})"

    say("[gpu] one build on each of 20 streams")
    outs = []
    for k in range(20):
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            outs.append((k % len(cases), s, T.build_tables(*cases[k % len(cases)], stream=s)))
    torch.cuda.synchronize()
    for k, (c, _, got) in enumerate(outs):
        assert same(c, got), f"stream {k} (case {c})"

    say("[gpu] 12 builds queued behind a spin kernel on one stream")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        torch.cuda._sleep(20_000_000)
        outs = [(k % len(cases), T.build_tables(*cases[k % len(cases)], stream=s))
                for k in range(12)]
    s.synchronize()
    for k, (c, got) in enumerate(outs):
        assert same(c, got), f"queued build {k} (case {c})"


def test_plan_larger_than_a_staging_buffer(T):
    """A 600-layer GPT on 2 devices: 8,400 operators and 10,798 edges, a plan of
    about 1.9 MB (more than a staging buffer holds at first, so one is replaced
    by a larger one, and the stream's scratch block grows), against the oracle;
    the shared-table build equals it, and a small build after it (on the grown
    buffers) still equals its own reference."""
    import torch
    g = W.gpt(600, 64, 2, 32, 2, 2)
    cl = W.Cluster(1, 2, 100 * W.GB, 10 * W.GB)
    small = W.config(2)
    ref_small = T.build_tables(small.graph, small.clusters[0][1])
    tabs = full_check(T, g, cl, "gpt 600 layers on 2 devices")
    shared = T.build_tables(g, cl, shared=True)
    again = T.build_tables(small.graph, small.clusters[0][1])
    torch.cuda.synchronize()
    assert _same_tables(tabs.edge, shared.edge) and _same_tables(tabs.node, shared.node)
    assert _same_tables(ref_small.edge, again.edge) and _same_tables(ref_small.node, again.node)


def test_fused_build_capacity_and_errors(T):
    """Capacity and argument errors are reported before any GPU work and leave the
    outputs untouched."""
    import torch
    w = W.config(2)
    cl = w.clusters[0][1]
    offs, eoffs = T.taps_build_tables(w.graph, cl, size_only=True)
    n_s, n_e = int(offs[-1]), int(eoffs[-1])
    for short_s, short_e in ((1, 0), (0, 1)):
        out = T.Tables(offs, torch.full((n_s - short_s, T.STRATEGY_BYTES), 7, dtype=torch.uint8,
                                        device="cuda"),
                       T.alloc_table(n_s - short_s), eoffs, T.alloc_table(n_e - short_e))
        for v in (*out.node.values(), *out.edge.values()):
            _signed(v).fill_(5)
        with pytest.raises(T.TapsError) as ex:
            T.taps_build_tables(w.graph, cl, out=out)
        assert ex.value.status == T.ERR_CAPACITY
        torch.cuda.synchronize()
        assert bool((out.strategies == 7).all())
        assert all(bool((_signed(v) == 5).all()) for v in (*out.node.values(), *out.edge.values()))


def test_link_class_degenerate_topologies(T):
    """Link classes at their edges: one class (every collective inside the one
    block), an innermost block of one device (every collective leaves it), block
    sizes repeated (empty classes), four classes on the largest mesh, and the
    in-node AllToAll bandwidth with one device per node (no in-node AllToAll)."""
    g = W.gpt(1, 64, 4, 32, 4, 2)
    cl16 = W.Cluster(2, 8, 600 * W.GB, 100 * W.GB)
    for topo in (W.Topology((16,), (300 * W.GB,)),
                 W.Topology((1, 16), (600 * W.GB, 100 * W.GB)),
                 W.Topology((2, 2, 8, 16), (600 * W.GB, 400 * W.GB, 100 * W.GB, 25 * W.GB)),
                 W.Topology((1, 4, 16), (600 * W.GB, 100 * W.GB, 50 * W.GB), 1200 * W.GB)):
        _topology_check(T, g, cl16, topo, f"gpt1 under {topo.domains}")
    g = W.gpt(1, 64, 2, 128, 2, 2)
    cl256 = W.Cluster(32, 8, 600 * W.GB, 100 * W.GB)
    _topology_check(T, g, cl256, W.Topology((8, 32, 128, 256), (600 * W.GB, 200 * W.GB, 50 * W.GB,
                                                                   25 * W.GB), 700 * W.GB),
                    "gpt1-s128 on 256 devices, four classes")
    one = W.Cluster(1, 1, 10, 1)
    _topology_check(T, W.gpt(1, 64, 4, 32, 4, 2), one, W.Topology((1,), (10,)), "one device")


def test_fused_build_degenerate(T):
    """The single-call build on one device, on 256 devices (batch x sequence split
    256 ways), on an empty graph and on operators without edges, against the
    oracle."""
    import torch
    full_check(T, W.gpt(1, 64, 4, 32, 4, 2), W.Cluster(1, 1, 10, 1), "fused one device")
    full_check(T, W.gpt(1, 64, 2, 128, 2, 2), W.Cluster(32, 8, 300, 7), "fused 256 devices")
    full_check(T, W.gpt(1, 64, 2, 128, 2, 2), W.Cluster(32, 8, 300, 7), "fused 256 devices on a mesh",
               mesh=[8, 4, 4, 2])
    tabs = T.build_tables(W.Graph(), W.Cluster(2, 2, 10, 1))
    torch.cuda.synchronize()
    assert list(tabs.op_offsets) == [0] and list(tabs.edge_offsets) == [0]
    g = W.Graph([W.matmul("a", 8, 8, 8, 2), W.matmul("b", 16, 8, 4, 4)], [])
    tabs = full_check(T, g, W.Cluster(2, 2, 10, 1), "fused, no edges")
    assert list(tabs.edge_offsets) == [0]


def test_empty_graph_and_no_edges(T):
    cl = W.Cluster(2, 2, 10, 1)
    tabs = T.build_tables(W.Graph(), cl)
    assert list(tabs.op_offsets) == [0] and list(tabs.edge_offsets) == [0]
    g = W.Graph([W.matmul("a", 8, 8, 8, 2)], [])
    tabs = full_check(T, g, cl, "one op")
    assert list(tabs.edge_offsets) == [0]


def test_capacity_error_on_device(T):
    import torch
    w = W.config(1)
    cl = w.clusters[0][1]
    offs, _ = T.taps_enumerate_strategies(w.graph, cl, size_only=True)
    small = torch.empty((int(offs[-1]) - 1, 16), dtype=torch.uint8, device="cuda")
    import ctypes as C
    g = T.pack_graph(w.graph)
    c = T.pack_cluster(cl)
    small.fill_(0xAB)
    st = T.load().taps_enumerate_strategies(C.byref(g.struct), C.byref(c), T._u64_array(offs),
                                            C.c_void_p(small.data_ptr()), int(offs[-1]) - 1, None)
    assert st == T.ERR_CAPACITY
    torch.cuda.synchronize()
    assert bool((small == 0xAB).all()), "nothing is written on a capacity error"


def test_no_strategy_error(T):
    import torch
    g = W.Graph([W.Op("odd", "x", ("a",), (3,), (True,), 2, ins=((0,),), ws=(), out=(0,))], [])
    with pytest.raises(T.TapsError) as ex:
        T.taps_enumerate_strategies(g, W.Cluster(2, 2, 10, 1))
    assert ex.value.status == T.ERR_NO_STRATEGY
    # with a caller buffer: nothing is written either
    ok = W.matmul("ok", 8, 8, 8, 2)
    g2 = W.Graph([ok, g.ops[0]], [])
    buf = torch.full((64, 16), 0xAB, dtype=torch.uint8, device="cuda")
    with pytest.raises(T.TapsError) as ex:
        T.taps_enumerate_strategies(g2, W.Cluster(2, 2, 10, 1), out=buf)
    assert ex.value.status == T.ERR_NO_STRATEGY
    torch.cuda.synchronize()
    assert bool((buf == 0xAB).all())


def test_shared_and_backward_on_empty_graphs(T):
    cl = W.Cluster(2, 2, 10, 1)
    for g in (W.Graph(), W.Graph([W.matmul("a", 8, 8, 8, 2)], [])):
        offs, strat = T.taps_enumerate_strategies(g, cl)
        for kw in ({"shared": True}, {"backward": True}):
            eoffs, tab = T.taps_edge_costs(g, cl, strat, offs, **kw)
            assert list(eoffs) == [0]


def test_repeatable_bitwise(T):
    import torch
    w = W.config(2)
    cl = w.clusters[0][1]
    a = T.build_tables(w.graph, cl)
    b = T.build_tables(w.graph, cl)
    torch.cuda.synchronize()
    for f in ("t", "vol", "intra", "inter", "meta"):
        assert np.array_equal(_np(a.edge[f]), _np(b.edge[f]))
        assert np.array_equal(_np(a.node[f]), _np(b.node[f]))


@pytest.mark.gpu
def test_edge_kernel_events(T):
    """The events given to taps_set_edge_kernel_events bracket the edge-table
    kernel inside the edge call, and are used once."""
    import torch
    w = W.config(2)
    cl = w.clusters[0][1]
    tabs = T.build_tables(w.graph, cl)
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev:
        e.record(stream)
    torch.cuda.synchronize()
    ev[0].record(stream)
    T.taps_set_edge_kernel_events(ev[2], ev[3])
    T.taps_edge_costs(w.graph, cl, tabs.strategies, tabs.op_offsets, out=tabs.edge, stream=stream)
    ev[1].record(stream)
    torch.cuda.synchronize()
    call_ms, kernel_ms = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
    assert 0.0 < kernel_ms <= call_ms
    # used once: a second call does not record them again (they stay before a
    # marker recorded ahead of it)
    mark = torch.cuda.Event(enable_timing=True)
    mark.record(stream)
    T.taps_edge_costs(w.graph, cl, tabs.strategies, tabs.op_offsets, out=tabs.edge, stream=stream)
    torch.cuda.synchronize()
    assert mark.elapsed_time(ev[3]) < 0 and mark.elapsed_time(ev[2]) < 0


@pytest.mark.gpu
def test_search_on_gpu_tables_matches_oracle_tables(T, oracle_lib):
    """The host search reaches the same optima on the library's tables as on the
    oracle's (configuration 1 and one GPT layer on 2 x 8 devices)."""
    import torch
    from paper_2301_04285_amd import search as S
    cases = [(W.config(1).graph, W.config(1).clusters[0][1]),
             (W.leading_ops(W.config(2).graph, 14), W.config(2).clusters[0][1])]
    for g, cl in cases:
        tabs = T.build_tables(g, cl)
        torch.cuda.synchronize()
        ref = oracle_lib.build_tables(g, cl)
        for f in ("t", "vol"):
            node, edge = S.host_tables(g, tabs, f)
            rnode = [np.asarray(v[f], np.float64) for v in ref.node]
            redge = [np.asarray(m[f], np.float64) for m in ref.edge]
            a, b = S.solve(g, node, edge), S.solve(g, rnode, redge)
            assert abs(a.objective - b.objective) <= 1e-9 * abs(b.objective)


def _same_tables(a, b):
    import torch
    return all(torch.equal(a[f], b[f]) for f in ("t", "vol", "intra", "inter", "meta"))


def oracle_check_edges(graph, cluster, tabs, name):
    """Every edge record of `tabs` (and its strategies) against the oracle."""
    strats = [O.enumerate_strategies(op, cluster.devices) for op in graph.ops]
    assert list(np.diff(tabs.op_offsets)) == [len(x) for x in strats], name
    edge = _host(tabs.edge)
    for x, e in enumerate(graph.edges):
        a, b = int(tabs.edge_offsets[x]), int(tabs.edge_offsets[x + 1])
        ref = O.edge_table(graph.ops[e.src], strats[e.src], graph.ops[e.dst], e.slot,
                           strats[e.dst], cluster)
        assert_records({f: v[a:b] for f, v in edge.items()}, ref, f"{name} edge {x}")
    return int(tabs.edge_offsets[-1])


def test_shared_tables_equal_full_evaluation(T):
    """taps_edge_costs_shared, and the single-call build with TAPS_BUILD_SHARED,
    write exactly the tables of taps_edge_costs, and every entry of both equals
    the oracle's."""
    import torch
    cases = [(W.config(2).graph, W.config(2).clusters[0][1]),
             (W.config(4).graph, W.config(4).clusters[0][1]),
             (W.gpt(3, 64, 2, 128, 2, 2), W.Cluster(2, 2, 200 * W.GB, 25 * W.GB))]
    rng = random.Random(77)
    for _ in range(6):
        g = W.random_graph(rng, rng.randint(2, 5), max_axes=4, max_rank=3, len_pow_range=(2, 7))
        # three disjoint copies of the graph, so that every edge repeats
        rep = W.Graph()
        for k in range(3):
            base = len(rep.ops)
            for op in g.ops:
                rep.ops.append(op)
            for e in g.edges:
                rep.connect(base + e.src, base + e.dst, e.slot)
        try:
            T.taps_enumerate_strategies(rep, W.Cluster(2, 4, 600 * W.GB, 50 * W.GB), size_only=True)
        except T.TapsError:
            continue
        cases.append((rep, W.Cluster(2, 4, 600 * W.GB, 50 * W.GB)))
    assert len(cases) >= 6
    checked = 0
    for k, (g, cl) in enumerate(cases):
        a = T.build_tables(g, cl)
        b = T.build_tables(g, cl, shared=True)                 # single call, shared
        c = T.build_tables(g, cl, shared=True, fused=False)    # taps_edge_costs_shared
        torch.cuda.synchronize()
        assert np.array_equal(a.edge_offsets, b.edge_offsets)
        assert np.array_equal(a.edge_offsets, c.edge_offsets)
        assert _same_tables(a.edge, b.edge)
        assert _same_tables(a.edge, c.edge)
        say(f"[gpu] shared tables case {k}: oracle comparison")
        checked += oracle_check_edges(g, cl, b, f"shared case {k} (single call)")
        checked += oracle_check_edges(g, cl, c, f"shared case {k} (separate calls)")
    say(f"[gpu] {checked} shared-table entries equal to the oracle")


@pytest.mark.gpu
def test_shared_tables_checks_the_strategies(T):
    """With caller strategies that differ between two identically described
    operators (one range reversed), sharing is refused for their edges and the
    tables still equal the full evaluation."""
    import torch
    w = W.config(2)
    cl = w.clusters[0][1]
    offs, strat = T.taps_enumerate_strategies(w.graph, cl)
    strat = strat.clone()
    k = 14 + 1   # layer 1's query projection, described like layer 0's
    a0, a1 = int(offs[k]), int(offs[k + 1])
    strat[a0:a1] = strat[a0:a1].flip(0)
    _, full = T.taps_edge_costs(w.graph, cl, strat, offs)
    _, shared = T.taps_edge_costs(w.graph, cl, strat, offs, shared=True)
    torch.cuda.synchronize()
    assert _same_tables(full, shared)


@pytest.mark.gpu
def test_shared_tables_largest_config(T):
    import torch
    w = W.config(5)
    cl = w.clusters[0][1]
    a = T.build_tables(w.graph, cl)
    b = T.build_tables(w.graph, cl, shared=True)
    torch.cuda.synchronize()
    assert int(b.edge_offsets[-1]) == 98668128
    assert _same_tables(a.edge, b.edge)
    del a, b
    torch.cuda.empty_cache()


def backward_check(T, graph, cluster, name, edges=None):
    """taps_edge_costs_backward against the oracle's backward tables, entry by entry."""
    import torch
    offs, strat = T.taps_enumerate_strategies(graph, cluster)
    eoffs, tab = T.taps_edge_costs(graph, cluster, strat, offs, backward=True)
    torch.cuda.synchronize()
    say(f"[gpu] backward {name}: {int(eoffs[-1])} entries")
    ref_strats = [O.enumerate_strategies(op, cluster.devices) for op in graph.ops]
    got = _host(tab)
    for x, e in enumerate(graph.edges):
        if edges is not None and x not in edges:
            continue
        a, b = int(eoffs[x]), int(eoffs[x + 1])
        ref = O.edge_table_reverse(graph.ops[e.src], ref_strats[e.src], graph.ops[e.dst], e.slot,
                                   ref_strats[e.dst], cluster)
        assert_records({f: v[a:b] for f, v in got.items()}, ref, f"{name} backward edge {x}")


@pytest.mark.gpu
def test_backward_tables(T):
    for cfg in (1, 2, 4):
        w = W.config(cfg)
        name, cl = w.clusters[0]
        backward_check(T, w.graph, cl, f"{w.name}/{name}")
    w = W.config(3)
    for name, cl in w.clusters:
        backward_check(T, W.leading_ops(w.graph, 28), cl, f"{w.name}/{name} (two layers)")
    rng = random.Random(4242)
    n = 0
    while n < 12:
        g = W.random_graph(rng, rng.randint(2, 6), max_axes=5, max_rank=4, len_pow_range=(1, 8))
        k = rng.randint(0, 7)
        N = 1 << k
        L = 1 << rng.randint(0, k)
        cl = W.Cluster(N // L, L, 600 * W.GB, rng.choice([12, 25, 100]) * W.GB)
        try:
            backward_check(T, g, cl, f"random {n}")
        except T.TapsError:
            continue
        n += 1


@pytest.mark.gpu
def test_backward_tables_largest_config_one_layer(T):
    w = W.config(5)
    name, cl = w.clusters[0]
    backward_check(T, W.leading_ops(w.graph, 14), cl, f"{w.name}/{name} (one layer)")


def sweep_check(T, graph, points, name, oracle=True):
    """taps_edge_costs_sweep: table k equals taps_edge_costs on points[k] bit
    for bit and, with `oracle`, the oracle's tables at that point."""
    import torch
    offs, strat = T.taps_enumerate_strategies(graph, points[0])
    eoffs, tabs = T.taps_edge_costs_sweep(graph, points, strat, offs)
    torch.cuda.synchronize()
    say(f"[gpu] sweep {name}: {len(points)} points, {int(eoffs[-1])} entries each")
    ref_strats = [O.enumerate_strategies(op, points[0].devices) for op in graph.ops] if oracle else None
    for k, cl in enumerate(points):
        e1, single = T.taps_edge_costs(graph, cl, strat, offs)
        torch.cuda.synchronize()
        assert np.array_equal(e1, eoffs)
        assert _same_tables(single, tabs[k]), f"{name} point {k}"
        if not oracle:
            continue
        got = _host(tabs[k])
        for x, e in enumerate(graph.edges):
            a, b = int(eoffs[x]), int(eoffs[x + 1])
            ref = O.edge_table(graph.ops[e.src], ref_strats[e.src], graph.ops[e.dst], e.slot,
                               ref_strats[e.dst], cl)
            assert_records({f: v[a:b] for f, v in got.items()}, ref, f"{name} point {k} edge {x}")
    return tabs


@pytest.mark.gpu
def test_sweep_tables(T):
    w = W.config(1)
    sweep_check(T, w.graph, [W.Cluster(2, 2, 200 * W.GB, 25 * W.GB),
                             W.Cluster(2, 2, 25 * W.GB, 200 * W.GB),
                             W.Cluster(2, 2, 100 * W.GB, 100 * W.GB)], w.name)
    w = W.config(4)   # the wide MLP at its inter-node bandwidth points
    sweep_check(T, w.graph, [cl for _, cl in w.clusters], w.name)
    w = W.config(2)
    sweep_check(T, w.graph, [W.Cluster(2, 8, 400 * W.GB, b * W.GB) for b in (50, 6, 400)], w.name)
    # one point: the single-table launch (row segments, not windows)
    sweep_check(T, w.graph, [W.Cluster(2, 8, 400 * W.GB, 50 * W.GB)], w.name + " one point")
    rng = random.Random(5151)
    n = 0
    while n < 10:
        g = W.random_graph(rng, rng.randint(2, 5), max_axes=5, max_rank=4, len_pow_range=(1, 8))
        k = rng.randint(0, 7)
        N = 1 << k
        L = 1 << rng.randint(0, k)
        # the last point has reduced bandwidths above 2^32 (the 128-bit order)
        pts = [W.Cluster(N // L, L, rng.choice([100, 200, 600]) * W.GB,
                         rng.choice([6, 12, 25, 100]) * W.GB) for _ in range(rng.randint(1, 7))]
        pts.append(W.Cluster(N // L, L, (1 << 40) + 1, 3))
        try:
            sweep_check(T, g, pts, f"random {n}")
        except T.TapsError:
            continue
        n += 1


@pytest.mark.gpu
def test_sweep_tables_largest_config(T):
    """The 96-layer GPT at four inter-node bandwidths: each table equals the
    single-point evaluation over all 98,668,128 entries."""
    import torch
    w = W.config(5)
    cl = w.clusters[0][1]
    pts = [W.Cluster(cl.nodes, cl.devices_per_node, cl.bw_intra, b * W.GB // 2)
           for b in (25, 50, 100, 200)]
    tabs = sweep_check(T, w.graph, pts, w.name, oracle=False)
    assert int(tabs[0]["t"].numel()) == 98668128
    del tabs
    torch.cuda.empty_cache()


@pytest.mark.gpu
def test_memory_costs(T):
    """taps_memory_costs against the oracle, every strategy of every operator."""
    import torch
    cases = [(W.config(c).graph, W.config(c).clusters[0][1]) for c in (1, 2, 3, 4, 5)]
    rng = random.Random(6161)
    while len(cases) < 13:
        g = W.random_graph(rng, rng.randint(1, 6), max_axes=6, max_rank=4, len_pow_range=(1, 9))
        k = rng.randint(0, 8)
        cl = W.Cluster(1 << rng.randint(0, k), 1, 10, 1)
        cl = W.Cluster(cl.nodes, (1 << k) // cl.nodes, 10, 1)
        try:
            T.taps_enumerate_strategies(g, cl, size_only=True)
        except T.TapsError:
            continue
        cases.append((g, cl))
    for g, cl in cases:
        offs, strat = T.taps_enumerate_strategies(g, cl)
        mem = _np(T.taps_memory_costs(g, strat, offs))
        torch.cuda.synchronize()
        for k, op in enumerate(g.ops):
            ref = O.memory_table(op, O.enumerate_strategies(op, cl.devices))
            a, b = int(offs[k]), int(offs[k + 1])
            assert np.array_equal(mem[a:b], ref), (k, op.name)

"""The oracle against explicit-device brute force on tiny meshes.

Checks, on seeded random problems with N <= 32 devices:
  * the inter-node group counts of AllReduce (Algorithm 2), AllGather and
    AllToAll (Algorithm 3, the AllToAll paragraph) against groups formed rank
    by rank;
  * that unification (Table 1) leaves every device holding the same elements;
  * that each candidate sequence (Table 2 / Algorithm 1) is a valid
    redistribution: explicit index ranges moved operator by operator end at
    the consumer's placement, with shard sizes and volumes (Eq. 9, Eq. 10)
    matching element counts;
  * that the bytes leaving a node (ring AllGather, peer-to-peer AllToAll,
    Eq. 14) equal ct x the link volume the oracle charges.
"""
import random
from fractions import Fraction
from math import prod

import numpy as np
import pytest

import bruteforce as BF
from paper_2301_04285_amd import workloads as W


def _random_matrix(rng, n):
    """A device matrix of 2^n devices with power-of-two axes (innermost first)."""
    D, left = [], n
    while left:
        e = rng.randint(1, left)
        D.append(1 << e)
        left -= e
    return D


def _random_map(rng, D, rank):
    axes = list(range(len(D)))
    rng.shuffle(axes)
    M = [-1] * rank
    for d in range(rank):
        if axes and rng.random() < 0.7:
            M[d] = axes.pop()
    return M


def _mesh_cases(seed, count):
    rng = random.Random(seed)
    for _ in range(count):
        n = rng.randint(1, 5)
        D = _random_matrix(rng, n)
        L = 1 << rng.randint(0, n)
        yield rng, D, L


def test_allreduce_ct_matches_explicit_groups(oracle_lib):
    n_cases = 0
    for rng, D, L in _mesh_cases(1, 1200):
        M = _random_map(rng, D, rng.randint(1, 4))
        if all(k in M for k in range(len(D))):
            continue  # nothing to reduce
        assert oracle_lib.allreduce_ct(D, M, L) == BF.allreduce_ct(D, M, L), (D, M, L)
        n_cases += 1
    assert n_cases > 200


def test_gather_ct_matches_explicit_groups(oracle_lib):
    for rng, D, L in _mesh_cases(7, 400):
        M = _random_map(rng, D, rng.randint(1, 4))
        used = [m for m in M if m >= 0]
        if not used:
            continue
        axis = rng.choice(used)
        assert oracle_lib.gather_ct(D, M, axis, L) == BF.gather_ct(D, M, axis, L), (D, M, axis, L)


def test_physical_reading_of_algorithm3_differs_from_literal(oracle_lib):
    """D = [2, 2, 2], two devices per node, gathering the outermost axis with
    the middle axis unused: the middle axis spans nodes, so its replicas cannot
    share results inside a node -- both devices of a node send (ct = 2)."""
    D, M, L = [2, 2, 2], [0, 2], 2
    assert BF.gather_ct(D, M, 2, L) == (2, 1)
    assert oracle_lib.gather_ct(D, M, 2, L) == (2, 1)


def test_single_node_and_one_device_per_node(oracle_lib):
    for rng, D, _ in _mesh_cases(11, 200):
        N = prod(D)
        M = _random_map(rng, D, rng.randint(1, 3))
        if any(k not in M for k in range(len(D))):
            assert oracle_lib.allreduce_ct(D, M, N) == 0
            assert oracle_lib.allreduce_ct(D, M, 1) == 1
        for a in (m for m in M if m >= 0):
            assert oracle_lib.gather_ct(D, M, a, N)[0] == 0
            assert oracle_lib.gather_ct(D, M, a, 1) == (1, 1)


# --- edges: unification, sequence validity, per-op volumes and node bytes ---

def _small_edges(seed, n_graphs=12):
    rng = random.Random(seed)
    for _ in range(n_graphs):
        g = W.random_graph(rng, rng.randint(3, 6), max_axes=4, max_rank=3,
                           len_pow_range=(0, 5))
        for e in g.edges:
            yield rng, g, e


def _check_edge_pair(oracle_lib, g, e, si, sj, cluster):
    src, dst = g.ops[e.src], g.ops[e.dst]
    N, L = cluster.devices, cluster.devices_per_node
    T = src.out
    shape = [src.axis_len[a] for a in T]
    beta = src.dtype_bytes
    # producer / consumer placement of the original tensor
    Dp = [0] * sum(1 for x in si["degree"] if x > 1)
    for a in range(src.n_axes):
        if si["degree"][a] > 1:
            Dp[si["pos"][a]] = int(si["degree"][a])
    Dc = [0] * sum(1 for x in sj["degree"] if x > 1)
    for a in range(dst.n_axes):
        if sj["degree"][a] > 1:
            Dc[sj["pos"][a]] = int(sj["degree"][a])
    Mp = [int(si["pos"][a]) if si["degree"][a] > 1 else -1 for a in T]
    Mc = [int(sj["pos"][a]) if sj["degree"][a] > 1 else -1 for a in dst.ins[e.slot]]
    held_p = BF.held_original(Dp, Mp, shape)
    held_c = BF.held_original(Dc, Mc, shape)
    costs = []
    for cand in range(4):
        u, ops, shard0 = oracle_lib.edge_detail(src, si, dst, e.slot, sj, cand, cluster)
        mesh = BF.Mesh(u.D, L)
        # unification leaves each device's elements where they were
        if cand == 0:
            assert prod(u.D) == N
            for r in range(N):
                rp = BF.initial_ranges(mesh, u.m_from, u.size, r)
                rc = BF.initial_ranges(mesh, u.m_to, u.size, r)
                assert BF.unified_to_original(u.orig, u.size, rp, len(shape)) == held_p[r]
                assert BF.unified_to_original(u.orig, u.size, rc, len(shape)) == held_c[r]
        sim = BF.Simulation(u.D, u.size, u.m_from, L)
        assert shard0 == sim.shard_elems() * beta * N
        assert len(ops) <= 2 * len(u.D)   # each device axis: gather+slice, or one AllToAll
        total_link = [0, 0]  # intra, inter (nb)
        for o in ops:
            shard_bytes = sim.shard_elems() * beta
            assert o.shard_nb == shard_bytes * N
            M_now = list(sim.M)
            p = u.D[o.axis]
            if o.kind == oracle_lib.SLICE:
                sim.slice(o.axis, o.to_dim)
                continue
            ct, k_in = BF.gather_ct(u.D, M_now, o.axis, L)
            assert (o.ct, o.k_in) == (ct, k_in)
            if o.kind == oracle_lib.ALLGATHER:
                assert o.volume_nb == (p - 1) * shard_bytes * N           # Eq. 9
                if ct:
                    node_bytes = BF.ring_allgather_node_bytes(u.D, M_now, o.axis, L, shard_bytes)
                    assert node_bytes * N == ct * o.link_nb
                sim.allgather(o.axis, o.from_dim)
            else:
                assert o.volume_nb * p == (p - 1) * shard_bytes * N       # Eq. 10
                if ct:
                    node_bytes = BF.alltoall_node_bytes(u.D, M_now, o.axis, L, shard_bytes)
                    assert node_bytes * N == ct * o.link_nb
                sim.alltoall(o.axis, o.from_dim, o.to_dim)
            if ct:
                total_link[1] += o.link_nb * ct
            else:
                assert o.link_nb == o.volume_nb
                total_link[0] += o.link_nb
        assert sim.matches(u.m_to), cand
        costs.append(total_link)
    return costs


@pytest.mark.parametrize("seed", [3, 5])
def test_candidate_sequences_are_valid_redistributions(oracle_lib, seed):
    checked = 0
    for rng, g, e in _small_edges(seed):
        src, dst = g.ops[e.src], g.ops[e.dst]
        n = rng.randint(1, 4)
        N = 1 << n
        L = 1 << rng.randint(0, n)
        cluster = W.Cluster(N // L, L, 7 * W.GB, 3 * W.GB)
        ss = oracle_lib.enumerate_strategies(src, N)
        sd = oracle_lib.enumerate_strategies(dst, N)
        if not len(ss) or not len(sd):
            continue
        pairs = [(rng.randrange(len(ss)), rng.randrange(len(sd))) for _ in range(6)]
        for i, j in pairs:
            costs = _check_edge_pair(oracle_lib, g, e, ss[i], sd[j], cluster)
            rec = oracle_lib.edge_cost(src, ss[i], dst, e.slot, sd[j], cluster)
            cand = rec[4] & 3
            assert [rec[2], rec[3]] == costs[cand]
            checked += 1
    assert checked > 40


def test_table2_replace_sequence_physically(oracle_lib):
    """Table 2's Algorithm-1 sequence moves real index ranges correctly on a
    16-device mesh with every d_i = 2."""
    D = [2, 2, 2, 2]
    sizes = [4, 4, 4, 4, 4]
    m_from, m_to = [-1, 1, 2, -1, 3], [1, -1, -1, 0, 3]
    for L in (1, 2, 4, 8, 16):
        for cand in range(4):
            sim = BF.Simulation(D, sizes, m_from, L)
            shard0 = sim.shard_elems() * 16
            ops, rec = oracle_lib.sequence_cost(D, m_from, m_to, cand, shard0, 16, L, 10, 1)
            for o in ops:
                ct = BF.gather_ct(D, list(sim.M), o.axis, L) if o.kind else None
                if ct is not None:
                    assert (o.ct, o.k_in) == ct
                {0: lambda: sim.slice(o.axis, o.to_dim),
                 1: lambda: sim.allgather(o.axis, o.from_dim),
                 2: lambda: sim.alltoall(o.axis, o.from_dim, o.to_dim)}[o.kind]()
            assert sim.matches(m_to)


def test_node_cost_against_explicit_groups(oracle_lib):
    rng = random.Random(17)
    checked = 0
    for _ in range(10):
        g = W.random_graph(rng, 4, max_axes=4, max_rank=3, len_pow_range=(0, 5))
        for op in g.ops:
            n = rng.randint(1, 5)
            N = 1 << n
            L = 1 << rng.randint(0, n)
            cl = W.Cluster(N // L, L, 9 * W.GB, 2 * W.GB)
            strats = oracle_lib.enumerate_strategies(op, N)
            for s in strats[: 12]:
                D = [0] * sum(1 for x in s["degree"] if x > 1)
                for a in range(op.n_axes):
                    if s["degree"][a] > 1:
                        D[s["pos"][a]] = int(s["degree"][a])
                vol = intra = inter = 0
                for t in (op.out, *op.ins, *op.ws):
                    M = [int(s["pos"][a]) if s["degree"][a] > 1 else -1 for a in t]
                    used = prod(D[m] for m in M if m >= 0)
                    gsz = N // used
                    if gsz == 1:
                        continue
                    mesh = BF.Mesh(D, L)
                    groups = mesh.groups_along([k for k in range(len(D)) if k not in M])
                    assert all(len(x) == gsz for x in groups)
                    elems = prod(op.axis_len[a] for a in t)
                    shard = elems * op.dtype_bytes // used
                    # ring AllReduce: each member sends 2(g-1) chunks of shard/g bytes
                    V = Fraction(2 * (gsz - 1) * shard, gsz)
                    assert (V * N).denominator == 1
                    V_nb = int(V * N)
                    ct = BF.allreduce_ct(D, M, L)
                    vol += V_nb
                    if ct:
                        inter += V_nb * ct
                    else:
                        intra += V_nb
                got = oracle_lib.node_cost(op, s, cl)
                assert got[1:4] == (vol, intra, inter)
                checked += 1
    assert checked > 50


# --- invariants on whole tables ---------------------------------------------

def _tables(oracle_lib, graph, cluster):
    return oracle_lib.build_tables(graph, cluster)


def test_one_node_tables_are_bandwidth_over_volume(oracle_lib):
    """One node: no collective leaves it, so every cost is volume / B_intra and
    the chosen sequence is the lowest-volume one (cf. the single-node
    comparison in the evaluation section)."""
    g = W.gpt(1, 64, 4, 32, 4, 2)
    cl = W.Cluster(1, 16, 300 * W.GB, 10 * W.GB)
    tab = _tables(oracle_lib, g, cl)
    for rec in [*tab.node, *tab.edge]:
        assert np.all(rec["inter"] == 0)
        assert np.all(rec["intra"] == rec["vol"])
        assert np.all(rec["meta"] >> 7 & 31 == 0)
        np.testing.assert_allclose(rec["t"], rec["vol"] / (16 * cl.bw_intra), rtol=1e-12)


def test_one_device_per_node_every_group_is_inter_node(oracle_lib):
    g = W.gpt(1, 64, 4, 32, 4, 2)
    cl = W.Cluster(16, 1, 300 * W.GB, 10 * W.GB)
    tab = _tables(oracle_lib, g, cl)
    for rec in [*tab.node, *tab.edge]:
        assert np.all(rec["intra"] == 0)
        assert np.all(rec["inter"] == rec["vol"])
        n_coll = rec["meta"] >> 2 & 31
        assert np.all(rec["meta"] >> 7 & 31 == n_coll)
        assert np.all(rec["meta"] >> 12 == n_coll)   # every ct is 1
        np.testing.assert_allclose(rec["t"], rec["vol"] / (16 * cl.bw_inter), rtol=1e-12)


def test_cost_monotone_in_inter_bandwidth_and_bounded(oracle_lib):
    g = W.mlp_stack(layers=4, batch=256)
    prev = None
    for bw in (100, 50, 25, 12.5):
        cl = W.Cluster(4, 4, 600 * W.GB, int(bw * W.GB))
        tab = _tables(oracle_lib, g, cl)
        for rec in [*tab.node, *tab.edge]:
            assert np.all(rec["t"] >= rec["vol"] / (16 * cl.bw_intra) * (1 - 1e-12))
        t = np.concatenate([r["t"].ravel() for r in [*tab.node, *tab.edge]])
        if prev is not None:
            assert np.all(t >= prev * (1 - 1e-12))
        prev = t


def test_naive_never_beats_remove(oracle_lib):
    """The naive sequence gathers a superset of what `remove` gathers, so it is
    never cheaper in either model; with ties to the lower index it is never
    the chosen candidate."""
    w = W.config(2)
    cl = w.clusters[0][1]
    tab = oracle_lib.build_tables(w.graph, cl, edges=range(0, 18))
    for rec in tab.edge[:18]:
        assert np.all(rec["meta"] & 3 != 3)


def test_tables_are_deterministic(oracle_lib):
    w = W.config(1)
    cl = w.clusters[0][1]
    a = oracle_lib.build_tables(w.graph, cl)
    b = oracle_lib.build_tables(w.graph, cl)
    for x, y in zip(a.edge + a.node, b.edge + b.node):
        assert x.tobytes() == y.tobytes()


# ---------------------------------------------------------------------------
# Backward direction: the gradient of an edge tensor moves from the consumer's
# map back to the producer's.
# ---------------------------------------------------------------------------

def _reversed_edge(src, dst, slot):
    """A virtual edge running the other way: the consumer, producing the tensor in
    its input map, feeds the producer, reading it in its output map."""
    import dataclasses
    a = dataclasses.replace(dst, out=dst.ins[slot], dtype_bytes=src.dtype_bytes)
    b = dataclasses.replace(src, ins=(src.out,))
    return a, b


@pytest.mark.parametrize("seed", range(6))
def test_reverse_table_equals_forward_table_of_the_reversed_edge(oracle_lib, seed):
    rng = random.Random(500 + seed)
    g = W.random_graph(rng, 3, max_axes=4, max_rank=3, len_pow_range=(2, 6))
    cl = W.Cluster(2, 4, 600 * W.GB, 50 * W.GB)
    strats = [oracle_lib.enumerate_strategies(op, cl.devices) for op in g.ops]
    for e in g.edges:
        if not len(strats[e.src]) or not len(strats[e.dst]):
            continue
        src, dst = g.ops[e.src], g.ops[e.dst]
        rev = oracle_lib.edge_table_reverse(src, strats[e.src], dst, e.slot, strats[e.dst], cl)
        a, b = _reversed_edge(src, dst, e.slot)
        fwd = oracle_lib.edge_table(a, strats[e.dst], b, 0, strats[e.src], cl)
        assert rev.shape == fwd.shape == (len(strats[e.dst]), len(strats[e.src]))
        for f in ("vol", "intra", "inter", "meta"):
            assert np.array_equal(rev[f], fwd[f])
        assert np.allclose(rev["t"], fwd["t"], rtol=1e-12, atol=0)


def test_reverse_table_of_a_self_similar_edge_is_the_forward_table(oracle_lib):
    """Between two alike element-wise operators the strategy lists and tensor maps
    coincide, so moving layout j to layout i costs the same in both tables."""
    op = W.elementwise("x", "gelu", ("b", "s", "h"), (64, 512, 1024), 1, 2)
    g = W.Graph()
    g.add(op)
    g.add(W.elementwise("y", "gelu", ("b", "s", "h"), (64, 512, 1024), 1, 2))
    g.connect(0, 1, 0)
    cl = W.Cluster(4, 4, 600 * W.GB, 50 * W.GB)
    s = oracle_lib.enumerate_strategies(g.ops[0], cl.devices)
    fwd = oracle_lib.edge_table(g.ops[0], s, g.ops[1], 0, s, cl)
    rev = oracle_lib.edge_table_reverse(g.ops[0], s, g.ops[1], 0, s, cl)
    assert fwd.shape == rev.shape and fwd.shape[0] > 10
    for f in ("t", "vol", "intra", "inter", "meta"):
        assert np.array_equal(fwd[f], rev[f])
    # and the direction matters elsewhere: a matmul output into a transposing consumer
    assert not np.array_equal(fwd["vol"], fwd["vol"].T) or fwd.shape[0] == 1


def test_reverse_tables_of_a_transformer_layer(oracle_lib):
    """Every edge of one GPT layer (16 edges, transposing and non-transposing maps)."""
    g = W.gpt(1, 64, 4, 128, 4, 2)
    cl = W.Cluster(2, 4, 600 * W.GB, 50 * W.GB)
    strats = [oracle_lib.enumerate_strategies(op, cl.devices) for op in g.ops]
    checked = 0
    for e in g.edges:
        src, dst = g.ops[e.src], g.ops[e.dst]
        rev = oracle_lib.edge_table_reverse(src, strats[e.src], dst, e.slot, strats[e.dst], cl)
        a, b = _reversed_edge(src, dst, e.slot)
        fwd = oracle_lib.edge_table(a, strats[e.dst], b, 0, strats[e.src], cl)
        for f in ("vol", "intra", "inter", "meta"):
            assert np.array_equal(rev[f], fwd[f])
        checked += rev.size
    assert len(g.edges) == 16 and checked > 10000

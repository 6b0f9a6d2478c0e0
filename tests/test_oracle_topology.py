"""Pins of the oracle's link-class hierarchies (an extension of the paper's two
classes, intra- and inter-node).

A topology has blocks of domains[0] <= domains[1] <= ... <= N consecutive
ranks; a collective belongs to the smallest block size that holds each of its
groups, and pays that class's bandwidth divided by the number of groups that
share the uplink of one block of the next smaller size (the paper's ct, with
"node" read as that block).  The pins build every group rank by rank (the
explicit-device brute force of bruteforce.py), decide the class from the
groups' ranks, count the shared uplinks and the bytes that leave a block, and
select the cheapest candidate with exact fractions; and check that the
domains (L, N) give the paper's two-class tables.
"""
import random
from fractions import Fraction
from math import prod

import numpy as np
import pytest

import bruteforce as BF
from paper_2301_04285_amd import workloads as W


def _random_topology(rng, n):
    """Non-decreasing block sizes (powers of two up to 2^n) and bandwidths, and
    half the time an in-block AllToAll bandwidth of its own."""
    k = rng.randint(1, 4)
    sizes = sorted(rng.randint(0, n) for _ in range(k - 1)) + [n]
    bw = [rng.choice([600, 400, 100, 50, 25, 12]) * W.GB for _ in range(k)]
    a2a = rng.choice([0, 0, 1200 * W.GB, 7 * 150 * W.GB, 50 * W.GB])
    return W.Topology(tuple(1 << e for e in sizes), tuple(bw), a2a)


def _matrix(s, n_axes):
    D = [0] * sum(1 for x in s["degree"][:n_axes] if x > 1)
    for a in range(n_axes):
        if s["degree"][a] > 1:
            D[s["pos"][a]] = int(s["degree"][a])
    return D


def _klass(groups, topo):
    """The smallest block size that holds every group, from the ranks."""
    for c, size in enumerate(topo.domains):
        if all(len({r // size for r in g}) == 1 for g in groups):
            return c
    raise AssertionError("the last domain holds every group")


def test_two_classes_are_the_paper_model(oracle_lib):
    rng = random.Random(31)
    for _ in range(12):
        g = W.random_graph(rng, 4, max_axes=4, max_rank=3, len_pow_range=(0, 6))
        n = rng.randint(0, 5)
        L = 1 << rng.randint(0, n)
        cl = W.Cluster((1 << n) // L, L, rng.choice([600, 25]) * W.GB,
                       int(rng.choice([100, 12.5, 7]) * W.GB))
        a = oracle_lib.build_tables(g, cl)
        b = oracle_lib.build_tables(g, cl, topology=W.Topology.of(cl))
        for x, y in zip(a.node + a.edge, b.node + b.edge):
            assert x.tobytes() == y.tobytes()


def test_node_costs_against_explicit_groups(oracle_lib):
    rng = random.Random(41)
    checked = 0
    for _ in range(12):
        g = W.random_graph(rng, 4, max_axes=4, max_rank=3, len_pow_range=(0, 5))
        for op in g.ops:
            n = rng.randint(1, 5)
            N = 1 << n
            topo = _random_topology(rng, n)
            for s in oracle_lib.enumerate_strategies(op, N)[:10]:
                D = _matrix(s, op.n_axes)
                vol = intra = inter = 0
                t = Fraction(0)
                for ten in (op.out, *op.ins, *op.ws):
                    M = [int(s["pos"][a]) if s["degree"][a] > 1 else -1 for a in ten]
                    used = prod(D[m] for m in M if m >= 0)
                    gsz = N // used
                    if gsz == 1:
                        continue
                    groups = BF.Mesh(D, N).groups_along([k for k in range(len(D)) if k not in M])
                    shard = prod(op.axis_len[a] for a in ten) * op.dtype_bytes // used
                    V_nb = 2 * (gsz - 1) * shard * N // gsz
                    c = _klass(groups, topo)
                    vol += V_nb
                    if c == 0:
                        intra += V_nb
                        t += Fraction(V_nb, N * topo.bw[0])
                    else:
                        ct = BF.allreduce_ct(D, M, topo.domains[c - 1])
                        assert ct > 0
                        inter += V_nb * ct
                        t += Fraction(V_nb * ct, N * topo.bw[c])
                got = oracle_lib.node_cost_topo(op, s, topo)
                assert got[1:4] == (vol, intra, inter)
                assert abs(got[0] - float(t)) <= 1e-12 * float(t) + 1e-300
                checked += 1
    assert checked > 60


def _candidate_costs(oracle_lib, g, e, si, sj, topo):
    """Per candidate: (exact seconds, vol, intra, inter, collectives, inter-class
    collectives, sum of ct), every collective's class and ct from explicit groups
    of the map just before it, and its block-leaving bytes counted edge by edge."""
    src, dst = g.ops[e.src], g.ops[e.dst]
    N = topo.devices
    cl = W.Cluster(1, N, 1, 1)   # only the sequences are read from here, not their costs
    beta = src.dtype_bytes
    out = []
    for cand in range(4):
        u, ops, shard0 = oracle_lib.edge_detail(src, si, dst, e.slot, sj, cand, cl)
        sim = BF.Simulation(u.D, u.size, u.m_from, N)
        mesh = BF.Mesh(u.D, N)
        t = Fraction(0)
        vol = intra = inter = n_coll = n_inter = sum_ct = 0
        for o in ops:
            shard_bytes = sim.shard_elems() * beta
            M_now = list(sim.M)
            p = u.D[o.axis]
            if o.kind == oracle_lib.SLICE:
                sim.slice(o.axis, o.to_dim)
                continue
            groups = mesh.groups_along([o.axis])
            c = _klass(groups, topo)
            n_coll += 1
            if o.kind == oracle_lib.ALLGATHER:
                V = (p - 1) * shard_bytes * N
                link = V
                if c:
                    ct, _ = BF.gather_ct(u.D, M_now, o.axis, topo.domains[c - 1])
                    out_bytes = BF.ring_allgather_node_bytes(u.D, M_now, o.axis,
                                                             topo.domains[c - 1], shard_bytes)
                    assert out_bytes * N == ct * link
                sim.allgather(o.axis, o.from_dim)
            else:
                V = (p - 1) * shard_bytes * N // p
                link = V
                if c:
                    ct, k = BF.gather_ct(u.D, M_now, o.axis, topo.domains[c - 1])
                    link = k * (p - k) * shard_bytes * N // p
                    out_bytes = BF.alltoall_node_bytes(u.D, M_now, o.axis, topo.domains[c - 1],
                                                       shard_bytes)
                    assert out_bytes * N == ct * link
                sim.alltoall(o.axis, o.from_dim, o.to_dim)
            vol += V
            if c == 0:
                intra += link
                a2a = o.kind == oracle_lib.ALLTOALL and topo.bw_a2a
                t += Fraction(link, N * (topo.bw_a2a if a2a else topo.bw[0]))
            else:
                inter += link * ct
                n_inter += 1
                sum_ct += ct
                t += Fraction(link * ct, N * topo.bw[c])
        assert sim.matches(u.m_to)
        out.append((t, vol, intra, inter, n_coll, n_inter, sum_ct))
    return out


@pytest.mark.parametrize("seed", [3, 8])
def test_edge_costs_against_explicit_groups(oracle_lib, seed):
    rng = random.Random(seed)
    checked = 0
    for _ in range(16):
        g = W.random_graph(rng, rng.randint(3, 5), max_axes=4, max_rank=3, len_pow_range=(0, 5))
        for e in g.edges:
            src, dst = g.ops[e.src], g.ops[e.dst]
            n = rng.randint(1, 4)
            N = 1 << n
            topo = _random_topology(rng, n)
            ss = oracle_lib.enumerate_strategies(src, N)
            sd = oracle_lib.enumerate_strategies(dst, N)
            if not len(ss) or not len(sd):
                continue
            for _ in range(5):
                i, j = rng.randrange(len(ss)), rng.randrange(len(sd))
                costs = _candidate_costs(oracle_lib, g, e, ss[i], sd[j], topo)
                best = min(range(4), key=lambda c: (costs[c][0], c))
                t, vol, intra, inter, n_coll, n_inter, sum_ct = costs[best]
                got = oracle_lib.edge_cost_topo(src, ss[i], dst, e.slot, sd[j], topo)
                assert got[4] & 3 == best
                assert got[1] == min(c[1] for c in costs)
                assert got[2:4] == (intra, inter)
                assert got[4] >> 2 == n_coll | (n_inter << 5) | (sum_ct << 10)
                assert abs(got[0] - float(t)) <= 1e-12 * float(t) + 1e-300
                checked += 1
    assert checked > 60


def test_one_block_is_volume_over_bandwidth(oracle_lib):
    """One block of all devices: nothing leaves it, t = vol / (N bw[0])."""
    g = W.gpt(1, 64, 4, 32, 4, 2)
    cl = W.Cluster(2, 8, 1, 1)
    tabs = oracle_lib.build_tables(g, cl, topology=W.Topology((16,), (300 * W.GB,)))
    for tab in tabs.node + tabs.edge:
        assert (tab["inter"] == 0).all()
        np.testing.assert_allclose(tab["t"], tab["intra"] / (16 * 300.0 * W.GB), rtol=1e-12)
        assert (tab["intra"] == tab["vol"]).all()


def test_cost_non_increasing_in_each_bandwidth(oracle_lib):
    g = W.gpt(1, 64, 4, 32, 4, 2)
    cl = W.Cluster(4, 4, 1, 1)
    base = W.Topology((4, 8, 16), (600 * W.GB, 100 * W.GB, 25 * W.GB))
    ref = oracle_lib.build_tables(g, cl, topology=base)
    for c in range(3):
        bw = list(base.bw)
        bw[c] *= 2
        faster = oracle_lib.build_tables(g, cl, topology=W.Topology(base.domains, tuple(bw)))
        for a, b in zip(ref.edge + ref.node, faster.edge + faster.node):
            assert (b["t"] <= a["t"] * (1 + 1e-12)).all()


def test_alltoall_bandwidth(oracle_lib):
    """An in-block AllToAll bandwidth equal to bw[0] changes nothing; a faster one
    lowers t exactly where the chosen sequence has an in-block AllToAll."""
    g = W.gpt(1, 64, 4, 32, 4, 2)
    cl = W.Cluster(4, 4, 1, 1)
    base = W.Topology((4, 8, 16), (600 * W.GB, 100 * W.GB, 25 * W.GB))
    same = W.Topology(base.domains, base.bw, base.bw[0])
    fast = W.Topology(base.domains, base.bw, 7 * base.bw[0])
    a = oracle_lib.build_tables(g, cl, topology=base)
    b = oracle_lib.build_tables(g, cl, topology=same)
    c = oracle_lib.build_tables(g, cl, topology=fast)
    lower = 0
    for x, y, z in zip(a.edge, b.edge, c.edge):
        assert x.tobytes() == y.tobytes()
        assert (z["t"] <= x["t"] * (1 + 1e-12)).all()
        lower += int((z["t"] < x["t"] * (1 - 1e-12)).sum())
    for x, z in zip(a.node, c.node):   # AllReduces are rings
        assert x.tobytes() == z.tobytes()
    assert lower > 0

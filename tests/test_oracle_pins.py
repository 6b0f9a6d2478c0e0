"""Pins of the CPU oracle to values and closed forms the paper prints.

Each test names the passage it follows.  The oracle is pinned here (and by
the explicit-device brute force in test_oracle_bruteforce.py) before any GPU
result is compared with it.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from conftest import golden_path, read_kv
from paper_2301_04285_amd import workloads as W


def _matmul(b=64, k=256, o=1024, dtype=4):
    return W.matmul("mm", b, k, o, dtype)


# --- GenerateStrategySet (Auxiliary Graph section, Table 3) -----------------

def test_table3_strategy_set(oracle_lib):
    rows = []
    with open(golden_path("table3_matmul_4_devices.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                p = line.split()
                rows.append((p[0], tuple(map(int, p[1:4])), tuple(map(int, p[4:7]))))
    s = oracle_lib.enumerate_strategies(_matmul(), 4)
    got = [(tuple(int(x) for x in r["degree"][:3]), tuple(int(x) for x in r["pos"][:3])) for r in s]
    assert got == [(deg, pos) for _, deg, pos in rows]


def _paper_count(p, n):
    """Number of strategies GenerateStrategySet makes for p partitionable axes
    on 2^n devices: sum_{i=1}^{min(p,n)} i! C(p,i) C(n-1,i-1)."""
    return sum(math.factorial(i) * math.comb(p, i) * math.comb(n - 1, i - 1)
               for i in range(1, min(p, n) + 1))


@pytest.mark.parametrize("p", [1, 2, 3, 4, 5, 6])
def test_strategy_count_formula(oracle_lib, p):
    for n in range(1, 8):
        op = W.Op("x", "x", tuple(f"a{a}" for a in range(p + 1)), (1 << 20,) * (p + 1),
                  (True,) * p + (False,), 2, ins=(tuple(range(p + 1)),), ws=(), out=(0,))
        got = len(oracle_lib.enumerate_strategies(op, 1 << n, filter_divisible=False))
        assert got == _paper_count(p, n), (p, n)


def test_strategy_divisibility_and_validity(oracle_lib):
    # an axis of length 2 can be split at most 2 ways; length 3 not at all
    op = W.Op("x", "x", ("a", "b", "c"), (2, 3, 1024), (True, True, True), 2,
              ins=((0, 1, 2),), ws=(), out=(0, 2))
    for n in range(1, 6):
        s = oracle_lib.enumerate_strategies(op, 1 << n)
        assert len(s) == len({(tuple(r["degree"]), tuple(r["pos"])) for r in s})
        for r in s:
            deg, pos = list(r["degree"][:3]), list(r["pos"][:3])
            assert deg[0] in (1, 2) and deg[1] == 1
            assert math.prod(deg) == 1 << n
            split = sorted(p for p in pos if p >= 0)
            assert split == list(range(len(split)))
            assert all((d > 1) == (p >= 0) for d, p in zip(deg, pos))


def test_single_device_has_one_whole_strategy(oracle_lib):
    g = W.mlp2()
    c = W.Cluster(1, 1, 100, 10)
    for op in g.ops:
        s = oracle_lib.enumerate_strategies(op, 1)
        assert len(s) == 1 and all(s[0]["degree"] == 1) and all(s[0]["pos"] == -1)
        assert oracle_lib.node_cost(op, s[0], c)[1:] == (0, 0, 0, 0)
    s0 = oracle_lib.enumerate_strategies(g.ops[0], 1)
    s1 = oracle_lib.enumerate_strategies(g.ops[1], 1)
    assert oracle_lib.edge_cost(g.ops[0], s0[0], g.ops[1], 0, s1[0], c) == (0.0, 0, 0, 0, 0)


def test_no_strategy_when_nothing_divides(oracle_lib):
    op = W.Op("x", "x", ("a",), (3,), (True,), 2, ins=((0,),), ws=(), out=(0,))
    assert len(oracle_lib.enumerate_strategies(op, 4)) == 0


# --- Intra-operator volume (Eq. 5-8) ----------------------------------------

@pytest.mark.parametrize("shape", [(64, 256, 1024), (1024, 2048, 512), (8, 4096, 4096)])
@pytest.mark.parametrize("n_dev", [2, 4, 8, 16, 64])
def test_eq8_matmul_volume(oracle_lib, shape, n_dev):
    """Eq. 8: Volume = 2((d-1) in out + (r-1) b out + (c-1) b in) / (d r c)
    per device (elements); the oracle's vol is in bytes x N."""
    b, k, o = shape
    op = _matmul(b, k, o, dtype=2)
    c = W.Cluster(1, n_dev, 100 * W.GB, 10 * W.GB)
    for s in oracle_lib.enumerate_strategies(op, n_dev):
        d, r, cc = (int(x) for x in s["degree"][:3])
        eq8 = Fraction(2 * ((d - 1) * k * o + (r - 1) * b * o + (cc - 1) * b * k), d * r * cc)
        vol = oracle_lib.node_cost(op, s, c)[1]
        assert Fraction(vol, n_dev * 2) == eq8


def test_eq5_to_7_each_allreduce(oracle_lib):
    """Eq. 5-7 separately: the Y, dW and E_X AllReduce volumes of MatMul."""
    b, k, o = 64, 256, 1024
    op = _matmul(b, k, o, dtype=4)
    for n_dev in (4, 8, 16):
        c = W.Cluster(1, n_dev, 100, 10)
        for s in oracle_lib.enumerate_strategies(op, n_dev):
            d, r, cc = (int(x) for x in s["degree"][:3])
            parts = [Fraction(2 * (r - 1) * b * o, d * r * cc),
                     Fraction(2 * (d - 1) * k * o, d * r * cc),
                     Fraction(2 * (cc - 1) * b * k, d * r * cc)]
            n_reduce = sum(1 for x in parts if x)
            meta = oracle_lib.node_cost(op, s, c)[4]
            assert (meta >> 2) & 31 == n_reduce


# --- Inter-node communication groups (Figure 2, Figure 3; Eq. 11) -----------

def test_figure2_inter_node_groups(oracle_lib):
    g = read_kv("figures_inter_node_groups.txt")
    L = int(g["fig2_devices_per_node"])
    D = [int(x) for x in g["fig2_device_matrix_inner_first"].split()]
    # AllReduce of a tensor that uses axes 1, 2 (reduced over axis 0) and of
    # one that uses axes 0, 1 (reduced over the outermost axis 2)
    assert oracle_lib.allreduce_ct(D, [1, 2], L) == int(g["fig2_inner_axis_ct"])
    ct = oracle_lib.allreduce_ct(D, [0, 1], L)
    assert ct == int(g["fig2_outer_axis_ct"])
    # the same groups as an AllGather along the outermost / innermost axis
    assert oracle_lib.gather_ct(D, [0, 1, 2], 2, L)[0] == int(g["fig2_outer_axis_ct"])
    assert oracle_lib.gather_ct(D, [0, 1, 2], 0, L)[0] == int(g["fig2_inner_axis_ct"])
    # Eq. 11: B_e = B_inter / ct
    assert int(g["fig2_link_bytes_per_s"]) // ct == int(g["fig2_effective_bytes_per_s"])
    # a 16-byte-per-device AllReduce over that axis costs V / B_e (Eq. 12)
    op = W.Op("x", "x", ("a", "b", "c"), (2, 4, 64), (True, True, True), 4,
              ins=(), ws=(), out=(1, 2))   # output lacks the outermost axis a
    s = np.zeros(1, dtype=oracle_lib.STRATEGY_DTYPE)
    s["degree"][0, :3] = (2, 4, 2)
    s["pos"][0, :3] = (2, 1, 0)
    s["degree"][0, 3:] = 1
    s["pos"][0, 3:] = -1
    c = W.Cluster(2, 8, 10 ** 12, int(g["fig2_link_bytes_per_s"]))
    t, vol, intra, inter, meta = oracle_lib.node_cost(op, s[0], c)
    per_device = Fraction(vol, 16)
    assert t == pytest.approx(float(per_device) / int(g["fig2_effective_bytes_per_s"]), rel=1e-12)
    assert intra == 0 and inter == vol * ct and meta >> 12 == ct


def test_figure3_weight_gradient_groups(oracle_lib):
    g = read_kv("figures_inter_node_groups.txt")
    L = int(g["fig3_devices_per_node"])
    degrees = (8, 2, 2)  # (d, r, c) on axes (b, in, out)
    for case in "abc":
        pos = [int(x) for x in g[f"fig3_{case}_positions"].split()]
        D = [0, 0, 0]
        for a, p in enumerate(pos):
            D[p] = degrees[a]
        M_dW = [pos[1], pos[2]]  # dW(in, out) keeps the in and out splits
        assert oracle_lib.allreduce_ct(D, M_dW, L) == int(g[f"fig3_{case}_ct"]), case


# --- Unification (Table 1) ---------------------------------------------------

def test_table1_unification(oracle_lib):
    g = read_kv("table1_unify.txt")
    ints = lambda k: [int(x) for x in g[k].split()]
    # the paper writes device matrices outermost first; the oracle stores D[0] innermost
    Dp = ints("producer_device_matrix")[::-1]
    Dc = ints("consumer_device_matrix")[::-1]
    shape = [int(g["s0"]), int(g["s1"])]
    u = oracle_lib.unify(16, Dp, ints("producer_map"), Dc, ints("consumer_map"), shape)
    assert u.D[::-1] == ints("unified_device_matrix")
    assert u.size == ints("unified_shape")
    assert u.m_from == ints("unified_producer_map")
    assert u.m_to == ints("unified_consumer_map")
    assert u.orig == [0, 0, 1, 1]


# --- Redistribution sequences (Table 2, Algorithm 1, Eq. 9, Eq. 10) ---------

def _table2():
    steps = {}
    kv = {}
    with open(golden_path("table2_redistribution.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line.startswith("step"):
                head, ops, vol = (x.strip() for x in line.split("|"))
                seq = []
                for o in ops.split(";"):
                    p = o.split()
                    seq.append((p[0], tuple(int(x) for x in p[1:])))
                steps[int(head.split()[1])] = (seq, vol)
            elif "=" in line:
                k, v = (x.strip() for x in line.split("=", 1))
                kv[k] = [int(x) for x in v.split()]
    return kv["m_from"], kv["m_to"], steps


_TABLE_STEP_OF_CANDIDATE = {3: 0, 2: 1, 1: 2, 0: 3}  # naive, remove, rearrange, replace


@pytest.mark.parametrize("dims", [(2, 2, 2, 2), (2, 4, 2, 8), (8, 2, 4, 2), (4, 4, 4, 2)])
def test_table2_sequences_and_volumes(oracle_lib, dims):
    m_from, m_to, steps = _table2()
    d0, d1, d2, d3 = dims
    D = [d0, d1, d2, d3]
    N = d0 * d1 * d2 * d3
    size_bytes = 1 << 20                 # Size(T) in bytes
    used = d1 * d2 * d3                  # M_from uses axes 1, 2, 3
    shard0_nb = size_bytes * N // used
    for cand, step in _TABLE_STEP_OF_CANDIDATE.items():
        ops, rec = oracle_lib.sequence_cost(D, m_from, m_to, cand, shard0_nb, N, N, 10, 1)
        want_seq, vol_expr = steps[step]
        got = []
        for o in ops:
            if o.kind == oracle_lib.SLICE:
                got.append(("S", (o.axis, o.to_dim)))
            elif o.kind == oracle_lib.ALLGATHER:
                got.append(("G", (o.axis, o.from_dim)))
            else:
                got.append(("A", (o.axis, o.from_dim, o.to_dim)))
        assert got == want_seq, (cand, got)
        frac = eval(vol_expr, {}, {"d0": Fraction(d0), "d1": Fraction(d1), "d2": Fraction(d2),
                                   "d3": Fraction(d3)})
        # rec volume is per-device bytes x N
        assert Fraction(rec[1], N) == frac * size_bytes, (cand, dims)

"""Pins of the oracle's fixed-mesh strategy spaces.

A fixed-mesh space is an extension of the paper (its device matrices are free,
Auxiliary Graph section): on a mesh [m_0 (innermost), ..., m_{k-1}] a strategy
may shard an operator axis only over whole, consecutive mesh dimensions.  The
pins are the paper's count formula with the number of levels replaced by the
number of mesh dimensions, Table 3's rows on the two 4-device meshes, a
brute-force construction from the definition, and the reduction to the
unrestricted space on a mesh of 2s.
"""
import itertools
import math
import random

import pytest

from conftest import golden_path
from paper_2301_04285_amd import workloads as W


def _table3_rows():
    rows = []
    with open(golden_path("table3_matmul_4_devices.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                p = line.split()
                rows.append((tuple(map(int, p[1:4])), tuple(map(int, p[4:7]))))
    return rows


def _key(r, n_axes):
    return (tuple(int(x) for x in r["degree"][:n_axes]), tuple(int(x) for x in r["pos"][:n_axes]))


def test_table3_on_both_4_device_meshes(oracle_lib):
    mm = W.matmul("mm", 64, 256, 1024, 4)
    rows = _table3_rows()
    # a 2 x 2 mesh has the two binary levels as its dimensions: all nine rows
    got = [_key(r, 3) for r in oracle_lib.enumerate_strategies_mesh(mm, [2, 2])]
    assert got == rows
    # a one-dimensional mesh of 4: only the rows that split one axis 4 ways (u1, u4, u9)
    got = [_key(r, 3) for r in oracle_lib.enumerate_strategies_mesh(mm, [4])]
    assert got == [rows[0], rows[3], rows[8]]


def _count(p, k):
    """The paper's GenerateStrategySet count with n levels replaced by k mesh
    dimensions: sum_{i=1}^{min(p,k)} i! C(p,i) C(k-1,i-1)."""
    if k == 0:
        return 1
    return sum(math.factorial(i) * math.comb(p, i) * math.comb(k - 1, i - 1)
               for i in range(1, min(p, k) + 1))


def _op(p, extra_whole=True):
    n = p + (1 if extra_whole else 0)
    return W.Op("x", "x", tuple(f"a{a}" for a in range(n)), (1 << 20,) * n,
                (True,) * p + (False,) * (n - p), 2, ins=(tuple(range(n)),), ws=(), out=(0,))


def _random_mesh(rng, max_levels=8):
    dims, levels = [], 0
    while True:
        e = rng.randint(1, 3)
        if levels + e > max_levels or (dims and rng.random() < 0.3):
            break
        dims.append(1 << e)
        levels += e
    return dims


@pytest.mark.parametrize("p", [1, 2, 3, 4, 5])
def test_count_formula_over_mesh_dimensions(oracle_lib, p):
    rng = random.Random(2301 + p)
    meshes = [[2], [8], [4, 2], [2, 4], [8, 4, 4], [8, 4, 2], [8, 16], [2, 2, 2, 2, 2],
              [4, 4, 4, 4]] + [_random_mesh(rng) for _ in range(12)]
    for mesh in meshes:
        got = oracle_lib.enumerate_strategies_mesh(_op(p), mesh, filter_divisible=False)
        assert len(got) == _count(p, len(mesh)), (p, mesh)


def _brute(op, mesh):
    """Every strategy on the mesh, built from the definition: an ordered choice of
    i distinct partitionable axes for device-matrix positions 0..i-1 and a
    composition of the mesh dimensions (innermost first) into i consecutive
    runs; the axis at position q gets the product of run q as its degree."""
    k = len(mesh)
    part = [a for a in range(op.n_axes) if op.partitionable[a]]
    out = set()
    if k == 0:
        return {((1,) * op.n_axes, (-1,) * op.n_axes)}
    for i in range(1, min(len(part), k) + 1):
        for cut in itertools.combinations(range(1, k), i - 1):
            bounds = (0,) + cut + (k,)
            degs = [math.prod(mesh[bounds[q]:bounds[q + 1]]) for q in range(i)]
            for axes in itertools.permutations(part, i):
                deg, pos = [1] * op.n_axes, [-1] * op.n_axes
                for q, a in enumerate(axes):
                    deg[a], pos[a] = degs[q], q
                out.add((tuple(deg), tuple(pos)))
    return out


def test_brute_force_from_the_definition(oracle_lib):
    rng = random.Random(7)
    for trial in range(40):
        p = rng.randint(1, 4)
        n_axes = p + rng.randint(0, 2)
        lens = tuple(rng.choice([1, 2, 3, 4, 6, 8, 12, 16, 64, 1024]) for _ in range(n_axes))
        partitionable = [True] * p + [False] * (n_axes - p)
        rng.shuffle(partitionable)
        op = W.Op("x", "x", tuple(f"a{a}" for a in range(n_axes)), lens, tuple(partitionable), 2,
                  ins=(tuple(range(n_axes)),), ws=(), out=(0,))
        mesh = _random_mesh(rng, 7)
        want = _brute(op, mesh)
        got = oracle_lib.enumerate_strategies_mesh(op, mesh, filter_divisible=False)
        keys = [_key(r, n_axes) for r in got]
        assert len(keys) == len(set(keys)) and set(keys) == want, (trial, mesh)
        # with the divisibility filter: exactly the dividing ones, in the same order
        kept = [k for k in keys if all(lens[a] % k[0][a] == 0 for a in range(n_axes))]
        got_f = oracle_lib.enumerate_strategies_mesh(op, mesh)
        assert [_key(r, n_axes) for r in got_f] == kept


def test_mesh_space_is_an_ordered_subset(oracle_lib):
    rng = random.Random(11)
    for trial in range(30):
        op = _op(rng.randint(1, 5), extra_whole=rng.random() < 0.5)
        mesh = _random_mesh(rng)
        n_dev = math.prod(mesh)
        full = [_key(r, op.n_axes) for r in oracle_lib.enumerate_strategies(op, n_dev)]
        sub = [_key(r, op.n_axes) for r in oracle_lib.enumerate_strategies_mesh(op, mesh)]
        it = iter(full)
        assert all(any(x == y for y in it) for x in sub), (trial, mesh)   # subsequence
        # a mesh of 2s is the unrestricted space
        assert [_key(r, op.n_axes) for r in
                oracle_lib.enumerate_strategies_mesh(op, [2] * (n_dev.bit_length() - 1))] == full


def test_one_device_mesh(oracle_lib):
    got = oracle_lib.enumerate_strategies_mesh(_op(3), [])
    assert len(got) == 1 and _key(got[0], 4) == ((1, 1, 1, 1), (-1, -1, -1, -1))

"""Explicit-device brute force for the topology model (test infrastructure).

Everything here works on named devices: a device matrix D (D[0] innermost)
gives every rank r < N = prod(D) its mixed-radix coordinates (axis 0
fastest), rank r sits on node r // L.  Collectives are formed as explicit
groups of ranks, the data a device holds is an explicit block (or index
range), and inter-node traffic is counted edge by edge.  None of it uses the
oracle's closed forms: it is the independent model the oracle is pinned to.
"""
from __future__ import annotations

from collections import defaultdict
from math import prod
from typing import Dict, FrozenSet, List, Sequence, Tuple


class Mesh:
    def __init__(self, D: Sequence[int], L: int):
        self.D = list(D)
        self.N = prod(self.D) if self.D else 1
        self.L = L
        self.coords: List[Tuple[int, ...]] = []
        for r in range(self.N):
            c, x = [], r
            for d in self.D:
                c.append(x % d)
                x //= d
            self.coords.append(tuple(c))

    def node(self, r: int) -> int:
        return r // self.L

    @property
    def nodes(self) -> List[int]:
        return sorted({self.node(r) for r in range(self.N)})

    def groups_along(self, axes: Sequence[int]) -> List[List[int]]:
        """Ranks that agree on every axis outside ``axes``."""
        axes = set(axes)
        by_key: Dict[Tuple[int, ...], List[int]] = defaultdict(list)
        for r, c in enumerate(self.coords):
            key = tuple(v for k, v in enumerate(c) if k not in axes)
            by_key[key].append(r)
        return list(by_key.values())

    def spans_nodes(self, group: Sequence[int]) -> bool:
        return len({self.node(r) for r in group}) > 1


def _per_node_equal(counts: Dict[int, int], nodes: Sequence[int]) -> int:
    vals = {counts.get(n, 0) for n in nodes}
    assert len(vals) == 1, f"nodes disagree: {counts}"
    return vals.pop()


def allreduce_ct(D: Sequence[int], M: Sequence[int], L: int) -> int:
    """Inter-node AllReduce groups touching one node, for a tensor with map M
    reduced over every axis M does not use.  0 when every group stays inside
    one node."""
    mesh = Mesh(D, L)
    unused = [k for k in range(len(D)) if k not in M]
    groups = mesh.groups_along(unused)
    counts: Dict[int, int] = defaultdict(int)
    for g in groups:
        if not mesh.spans_nodes(g):
            continue
        for n in {mesh.node(r) for r in g}:
            counts[n] += 1
    return _per_node_equal(counts, mesh.nodes)


def block(mesh: Mesh, M: Sequence[int], r: int) -> Tuple:
    """Which block of the (unified) tensor rank r holds: per dimension the
    coordinate of the axis that splits it, or None when it is whole."""
    c = mesh.coords[r]
    return tuple(c[m] if m >= 0 else None for m in M)


def gather_groups(mesh: Mesh, M: Sequence[int], axis: int):
    """Groups of a collective along ``axis`` with the data each one holds."""
    for g in mesh.groups_along([axis]):
        data: FrozenSet = frozenset(block(mesh, M, r) for r in g)
        yield g, data


def gather_ct(D: Sequence[int], M: Sequence[int], axis: int, L: int) -> Tuple[int, int]:
    """(ct, members per node) for an AllGather / AllToAll along ``axis``.
    Groups that hold exactly the same data inside one node are replicas: one of
    them crosses the node boundary and shares the result inside the node, so
    ct counts distinct data among the node's groups that leave the node."""
    mesh = Mesh(D, L)
    distinct: Dict[int, set] = defaultdict(set)
    k_in = set()
    for g, data in gather_groups(mesh, M, axis):
        per_node = defaultdict(int)
        for r in g:
            per_node[mesh.node(r)] += 1
        k_in.update(per_node.values())
        if len(per_node) > 1:
            for n in per_node:
                distinct[n].add(data)
    assert len(k_in) == 1
    ct = _per_node_equal({n: len(s) for n, s in distinct.items()}, mesh.nodes)
    return ct, k_in.pop()


def _distinct_crossing_groups(mesh: Mesh, M, axis, node):
    """One representative per distinct data among the groups at ``node`` that
    leave it."""
    seen = {}
    for g, data in gather_groups(mesh, M, axis):
        if mesh.spans_nodes(g) and any(mesh.node(r) == node for r in g):
            seen.setdefault(data, g)
    return list(seen.values())


def ring_allgather_node_bytes(D, M, axis: int, L: int, shard_bytes: int) -> int:
    """Bytes that leave one node for a ring AllGather along ``axis``: each
    member forwards p-1 shards to its ring successor (members ordered by their
    coordinate on the axis); count the ring edges leaving the node."""
    mesh = Mesh(D, L)
    p = D[axis]
    totals = {}
    for n in mesh.nodes:
        total = 0
        for g in _distinct_crossing_groups(mesh, M, axis, n):
            ring = sorted(g, key=lambda r: mesh.coords[r][axis])
            for q, r in enumerate(ring):
                nxt = ring[(q + 1) % len(ring)]
                if mesh.node(r) == n and mesh.node(nxt) != n:
                    total += (p - 1) * shard_bytes
        totals[n] = total
    return _per_node_equal(totals, mesh.nodes)


def alltoall_node_bytes(D, M, axis: int, L: int, shard_bytes: int) -> int:
    """Bytes that leave one node for a peer-to-peer AllToAll along ``axis``:
    every member sends shard/p to every other member."""
    mesh = Mesh(D, L)
    p = D[axis]
    assert shard_bytes % p == 0
    totals = {}
    for n in mesh.nodes:
        total = 0
        for g in _distinct_crossing_groups(mesh, M, axis, n):
            for r in g:
                if mesh.node(r) != n:
                    continue
                total += sum(shard_bytes // p for q in g if mesh.node(q) != n)
        totals[n] = total
    return _per_node_equal(totals, mesh.nodes)


# ---------------------------------------------------------------------------
# Physical placement of tensor elements
# ---------------------------------------------------------------------------

def chunk(size: int, parts: int, idx: int) -> Tuple[int, int]:
    assert size % parts == 0, (size, parts)
    w = size // parts
    return (idx * w, (idx + 1) * w)


def held_original(D: Sequence[int], M: Sequence[int], shape: Sequence[int], L: int = 1):
    """Per rank, per original dimension: the frozenset of indices it holds
    when dimension d is split by axis M[d] of D (or whole)."""
    mesh = Mesh(D, L)
    out = []
    for r in range(mesh.N):
        c = mesh.coords[r]
        dims = []
        for d, s in enumerate(shape):
            if M[d] >= 0:
                lo, hi = chunk(s, D[M[d]], c[M[d]])
                dims.append(frozenset(range(lo, hi)))
            else:
                dims.append(frozenset(range(s)))
        out.append(tuple(dims))
    return out


def unified_to_original(orig: Sequence[int], sizes: Sequence[int], ranges, rank: int):
    """Per original dimension, the index set covered by per-sub-dimension ranges
    (sub-dimensions of one original dimension combine outermost first)."""
    dims = []
    for d in range(rank):
        ks = [k for k in range(len(orig)) if orig[k] == d]
        idx = {0}
        for k in ks:
            lo, hi = ranges[k]
            idx = {i * sizes[k] + x for i in idx for x in range(lo, hi)}
        dims.append(frozenset(idx))
    return tuple(dims)


def initial_ranges(mesh: Mesh, M: Sequence[int], sizes: Sequence[int], r: int):
    c = mesh.coords[r]
    return [chunk(sizes[k], mesh.D[M[k]], c[M[k]]) if M[k] >= 0 else (0, sizes[k])
            for k in range(len(sizes))]


class Simulation:
    """Moves explicit index ranges through a redistribution sequence on a
    unified problem and checks every step."""

    def __init__(self, D, sizes, M_from, L):
        self.mesh = Mesh(D, L)
        self.sizes = list(sizes)
        self.M = list(M_from)
        self.ranges = [initial_ranges(self.mesh, self.M, self.sizes, r)
                       for r in range(self.mesh.N)]

    def shard_elems(self, r: int = 0) -> int:
        vals = {prod(hi - lo for lo, hi in self.ranges[q]) for q in range(self.mesh.N)}
        assert len(vals) == 1, "devices hold shards of different sizes"
        return vals.pop()

    def _group(self, r, axis):
        c = self.mesh.coords[r]
        return [q for q in range(self.mesh.N)
                if all(self.mesh.coords[q][k] == c[k] for k in range(len(c)) if k != axis)]

    def slice(self, axis, k):
        assert self.M[k] == -1, "slice of a dimension that is already split"
        assert axis not in self.M, "slice along an axis another dimension uses"
        p = self.mesh.D[axis]
        for r in range(self.mesh.N):
            assert self.ranges[r][k] == (0, self.sizes[k])
            self.ranges[r][k] = chunk(self.sizes[k], p, self.mesh.coords[r][axis])
        self.M[k] = axis

    def _gather_dim(self, axis, k):
        new = []
        for r in range(self.mesh.N):
            g = self._group(r, axis)
            others = {tuple(self.ranges[q][x] for x in range(len(self.sizes)) if x != k) for q in g}
            assert len(others) == 1, "gather group disagrees outside the gathered dimension"
            pieces = sorted(self.ranges[q][k] for q in g)
            for (a, b), (c, d) in zip(pieces, pieces[1:]):
                assert b == c, "gathered pieces are not contiguous"
            new.append((pieces[0][0], pieces[-1][1]))
        for r in range(self.mesh.N):
            self.ranges[r][k] = new[r]
            assert new[r] == (0, self.sizes[k])

    def allgather(self, axis, k):
        assert self.M[k] == axis
        self._gather_dim(axis, k)
        self.M[k] = -1

    def alltoall(self, axis, i, k):
        assert self.M[i] == axis and self.M[k] == -1
        self._gather_dim(axis, i)
        self.M[i] = -1
        p = self.mesh.D[axis]
        for r in range(self.mesh.N):
            assert self.ranges[r][k] == (0, self.sizes[k])
            self.ranges[r][k] = chunk(self.sizes[k], p, self.mesh.coords[r][axis])
        self.M[k] = axis

    def matches(self, M_to) -> bool:
        target = [initial_ranges(self.mesh, M_to, self.sizes, r) for r in range(self.mesh.N)]
        return self.ranges == target and self.M == list(M_to)

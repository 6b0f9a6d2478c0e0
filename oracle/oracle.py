"""ctypes front end of the C oracle (``taps_oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline call this module.  The library's GPU path neither imports nor links
it.  Nothing here computes costs; it marshals workload descriptions into the
oracle's own structs and returns numpy record arrays.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "taps_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

MAX_AXES = 8
MAX_RANK = 8
MAX_IN = 4
MAX_W = 4
MAX_DEV = 16
MAX_SUB = 48
MAX_SEQ = 96

SLICE, ALLGATHER, ALLTOALL = 0, 1, 2
CANDIDATES = ("replace", "rearrange", "remove", "naive")


class OrTensor(C.Structure):
    _fields_ = [("rank", C.c_int32), ("axis", C.c_int32 * MAX_RANK)]


class OrOp(C.Structure):
    _fields_ = [("n_axes", C.c_int32), ("part_mask", C.c_int32), ("dtype_bytes", C.c_int32),
                ("n_in", C.c_int32), ("n_w", C.c_int32), ("pad_", C.c_int32),
                ("axis_len", C.c_int64 * MAX_AXES),
                ("ins", OrTensor * MAX_IN), ("ws", OrTensor * MAX_W), ("out", OrTensor)]


class OrStrategy(C.Structure):
    _fields_ = [("degree", C.c_int32 * MAX_AXES), ("pos", C.c_int32 * MAX_AXES)]


class OrRecord(C.Structure):
    _fields_ = [("t", C.c_double), ("vol", C.c_uint64), ("intra", C.c_uint64),
                ("inter", C.c_uint64), ("meta", C.c_uint32), ("pad_", C.c_uint32)]


class OrRedop(C.Structure):
    _fields_ = [("kind", C.c_int32), ("axis", C.c_int32), ("from_dim", C.c_int32),
                ("to_dim", C.c_int32), ("ct", C.c_int32), ("k_in", C.c_int32),
                ("shard_nb", C.c_uint64), ("volume_nb", C.c_uint64), ("link_nb", C.c_uint64),
                ("cost", C.c_double)]


class OrUnified(C.Structure):
    _fields_ = [("h", C.c_int32), ("r", C.c_int32), ("D", C.c_int64 * MAX_DEV),
                ("orig", C.c_int32 * MAX_SUB), ("size", C.c_int64 * MAX_SUB),
                ("m_from", C.c_int32 * MAX_SUB), ("m_to", C.c_int32 * MAX_SUB)]


MAX_CLASSES = 4


class OrTopology(C.Structure):
    _fields_ = [("n_classes", C.c_int32), ("pad_", C.c_int32),
                ("domain", C.c_int64 * MAX_CLASSES), ("bw", C.c_uint64 * MAX_CLASSES),
                ("bw_a2a", C.c_uint64)]


def make_topology(topo) -> OrTopology:
    """workloads.Topology -> the oracle's struct."""
    assert 1 <= len(topo.domains) == len(topo.bw) <= MAX_CLASSES
    return OrTopology(len(topo.domains), 0, (C.c_int64 * MAX_CLASSES)(*topo.domains),
                      (C.c_uint64 * MAX_CLASSES)(*topo.bw), topo.bw_a2a)


RECORD_DTYPE = np.dtype([("t", "<f8"), ("vol", "<u8"), ("intra", "<u8"), ("inter", "<u8"),
                         ("meta", "<u4"), ("pad_", "<u4")])
assert RECORD_DTYPE.itemsize == C.sizeof(OrRecord)
STRATEGY_DTYPE = np.dtype([("degree", "<i4", (MAX_AXES,)), ("pos", "<i4", (MAX_AXES,))])
assert STRATEGY_DTYPE.itemsize == C.sizeof(OrStrategy)


def build(force: bool = False) -> str:
    """Compile the oracle with gcc into ``oracle/liboracle.so``."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                               "-o", tmp, SRC])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = C.CDLL(LIB)
        i64, u64, i32 = C.c_int64, C.c_uint64, C.c_int32
        P = C.POINTER
        L.or_enumerate.restype = i64
        L.or_enumerate.argtypes = [P(OrOp), i64, C.c_int, P(OrStrategy), i64]
        L.or_enumerate_mesh.restype = i64
        L.or_enumerate_mesh.argtypes = [P(OrOp), P(i64), C.c_int, C.c_int, P(OrStrategy), i64]
        L.or_node_cost_topo.restype = None
        L.or_node_cost_topo.argtypes = [P(OrOp), P(OrStrategy), i64, P(OrTopology), P(OrRecord)]
        L.or_node_table_topo.restype = i64
        L.or_node_table_topo.argtypes = [P(OrOp), P(OrStrategy), i64, i64, P(OrTopology),
                                         P(OrRecord)]
        L.or_edge_cost_topo.restype = C.c_int
        L.or_edge_cost_topo.argtypes = [P(OrOp), P(OrStrategy), P(OrOp), C.c_int, P(OrStrategy),
                                        i64, P(OrTopology), P(OrRecord)]
        L.or_edge_table_topo.restype = i64
        L.or_edge_table_topo.argtypes = [P(OrOp), P(OrStrategy), i64, P(OrOp), C.c_int,
                                         P(OrStrategy), i64, i64, P(OrTopology), P(OrRecord)]
        L.or_edge_entries_topo.restype = i64
        L.or_edge_entries_topo.argtypes = [P(OrOp), P(OrStrategy), P(OrOp), C.c_int,
                                           P(OrStrategy), P(i64), P(i64), i64, i64,
                                           P(OrTopology), P(OrRecord)]
        L.or_node_cost.restype = None
        L.or_node_cost.argtypes = [P(OrOp), P(OrStrategy), i64, i64, u64, u64, P(OrRecord)]
        L.or_node_table.restype = i64
        L.or_node_table.argtypes = [P(OrOp), P(OrStrategy), i64, i64, i64, u64, u64, P(OrRecord)]
        L.or_allreduce_ct.restype = i64
        L.or_allreduce_ct.argtypes = [P(i64), C.c_int, P(i32), C.c_int, i64]
        L.or_gather_ct.restype = i64
        L.or_gather_ct.argtypes = [P(i64), C.c_int, P(i32), C.c_int, C.c_int, i64, P(i64)]
        L.or_unify.restype = C.c_int
        L.or_unify.argtypes = [i64, P(i64), C.c_int, P(i32), P(i64), C.c_int, P(i32), C.c_int,
                               P(i64), P(OrUnified)]
        L.or_sequence_cost.restype = C.c_int
        L.or_sequence_cost.argtypes = [P(i64), C.c_int, P(i32), P(i32), C.c_int, C.c_int, u64,
                                       i64, i64, u64, u64, P(OrRedop), P(OrRecord)]
        L.or_edge_detail.restype = C.c_int
        L.or_edge_detail.argtypes = [P(OrOp), P(OrStrategy), P(OrOp), C.c_int, P(OrStrategy),
                                     i64, i64, u64, u64, C.c_int, P(OrUnified), P(OrRedop),
                                     P(u64)]
        L.or_edge_cost.restype = C.c_int
        L.or_edge_cost.argtypes = [P(OrOp), P(OrStrategy), P(OrOp), C.c_int, P(OrStrategy),
                                   i64, i64, u64, u64, P(OrRecord)]
        L.or_edge_cost_reverse.restype = C.c_int
        L.or_edge_cost_reverse.argtypes = L.or_edge_cost.argtypes
        L.or_edge_table_reverse.restype = i64
        L.or_edge_table_reverse.argtypes = [P(OrOp), P(OrStrategy), i64, P(OrOp), C.c_int,
                                            P(OrStrategy), i64, i64, i64, u64, u64, P(OrRecord)]
        L.or_edge_table.restype = i64
        L.or_edge_table.argtypes = [P(OrOp), P(OrStrategy), i64, P(OrOp), C.c_int,
                                    P(OrStrategy), i64, i64, i64, u64, u64, P(OrRecord)]
        L.or_edge_entries.restype = i64
        L.or_edge_entries.argtypes = [P(OrOp), P(OrStrategy), P(OrOp), C.c_int, P(OrStrategy),
                                      P(i64), P(i64), i64, i64, i64, u64, u64, P(OrRecord)]
        _lib = L
    return _lib


# ---------------------------------------------------------------------------
# marshalling
# ---------------------------------------------------------------------------

def _tensor(axes: Sequence[int]) -> OrTensor:
    t = OrTensor()
    t.rank = len(axes)
    for d, a in enumerate(axes):
        t.axis[d] = a
    return t


def make_op(op) -> OrOp:
    """``op`` is a ``workloads.Op`` (or anything with the same attributes)."""
    o = OrOp()
    o.n_axes = len(op.axis_len)
    o.part_mask = sum(1 << a for a, p in enumerate(op.partitionable) if p)
    o.dtype_bytes = op.dtype_bytes
    o.n_in = len(op.ins)
    o.n_w = len(op.ws)
    for a, n in enumerate(op.axis_len):
        o.axis_len[a] = n
    for k, t in enumerate(op.ins):
        o.ins[k] = _tensor(t)
    for k, t in enumerate(op.ws):
        o.ws[k] = _tensor(t)
    o.out = _tensor(op.out)
    return o


def _levels(n_devices: int) -> int:
    assert n_devices >= 1 and n_devices & (n_devices - 1) == 0
    return n_devices.bit_length() - 1


def enumerate_strategies(op, n_devices: int, filter_divisible: bool = True) -> np.ndarray:
    """GenerateStrategySet of one op: a STRATEGY_DTYPE array in canonical order."""
    o = make_op(op)
    L = lib()
    n = L.or_enumerate(C.byref(o), n_devices, int(filter_divisible), None, 0)
    assert n >= 0
    arr = np.zeros(n, dtype=STRATEGY_DTYPE)
    if n:
        got = L.or_enumerate(C.byref(o), n_devices, int(filter_divisible),
                             arr.ctypes.data_as(C.POINTER(OrStrategy)), n)
        assert got == n
    return arr


def enumerate_strategies_mesh(op, mesh: Sequence[int], filter_divisible: bool = True) -> np.ndarray:
    """The strategies of `enumerate_strategies` on prod(mesh) devices whose device
    matrix groups whole, consecutive dimensions of the fixed mesh `mesh`
    (innermost first), in the same order.  A fixed-mesh strategy space is an
    extension: the paper's device matrices are free."""
    o = make_op(op)
    L = lib()
    m = (C.c_int64 * max(1, len(mesh)))(*mesh)
    n = L.or_enumerate_mesh(C.byref(o), m, len(mesh), int(filter_divisible), None, 0)
    assert n >= 0
    arr = np.zeros(n, dtype=STRATEGY_DTYPE)
    if n:
        got = L.or_enumerate_mesh(C.byref(o), m, len(mesh), int(filter_divisible),
                                  arr.ctypes.data_as(C.POINTER(OrStrategy)), n)
        assert got == n
    return arr


def _sp(arr: np.ndarray):
    return arr.ctypes.data_as(C.POINTER(OrStrategy))


def _rp(arr: np.ndarray):
    return arr.ctypes.data_as(C.POINTER(OrRecord))


def node_table(op, strategies: np.ndarray, cluster) -> np.ndarray:
    o = make_op(op)
    out = np.zeros(len(strategies), dtype=RECORD_DTYPE)
    n = lib().or_node_table(C.byref(o), _sp(strategies), len(strategies), cluster.devices,
                            cluster.devices_per_node, cluster.bw_intra, cluster.bw_inter, _rp(out))
    assert n == len(strategies)
    return out


def memory_table(op, strategies: np.ndarray) -> np.ndarray:
    """Per-device bytes of each strategy (uint64): one shard of every weight
    and of the output.  Eq. 18 bounds the sum of the selected memory costs by
    the device memory but the paper does not define the cost itself; this is
    the reading used here.  A tensor dimension on op axis a is cut into
    degree[a] equal parts, so a shard has prod_d (len_d // degree_d) elements."""
    deg = strategies["degree"].astype(np.int64) if len(strategies) else np.ones((0, 8), np.int64)
    out = np.zeros(len(strategies), dtype=np.uint64)
    for t in (*op.ws, op.out):
        elems = np.ones(len(strategies), dtype=np.int64)
        for a in t:
            elems = elems * (op.axis_len[a] // deg[:, a])
        out += (elems * op.dtype_bytes).astype(np.uint64)
    return out


def edge_table(src_op, src_strats: np.ndarray, dst_op, slot: int, dst_strats: np.ndarray,
               cluster) -> np.ndarray:
    """Row-major (len(src_strats), len(dst_strats)) table of one edge."""
    a, b = make_op(src_op), make_op(dst_op)
    out = np.zeros(len(src_strats) * len(dst_strats), dtype=RECORD_DTYPE)
    n = lib().or_edge_table(C.byref(a), _sp(src_strats), len(src_strats), C.byref(b), slot,
                            _sp(dst_strats), len(dst_strats), cluster.devices,
                            cluster.devices_per_node, cluster.bw_intra, cluster.bw_inter, _rp(out))
    assert n == out.size, "oracle failed on this edge"
    return out.reshape(len(src_strats), len(dst_strats))


def edge_table_reverse(src_op, src_strats: np.ndarray, dst_op, slot: int, dst_strats: np.ndarray,
                       cluster) -> np.ndarray:
    """Backward table of one edge (the gradient from the consumer's map back to the
    producer's), consumer-major: shape (len(dst_strats), len(src_strats))."""
    a, b = make_op(src_op), make_op(dst_op)
    out = np.zeros(len(src_strats) * len(dst_strats), dtype=RECORD_DTYPE)
    n = lib().or_edge_table_reverse(C.byref(a), _sp(src_strats), len(src_strats), C.byref(b),
                                    slot, _sp(dst_strats), len(dst_strats), cluster.devices,
                                    cluster.devices_per_node, cluster.bw_intra, cluster.bw_inter,
                                    _rp(out))
    assert n == out.size, "oracle failed on this edge"
    return out.reshape(len(dst_strats), len(src_strats))


def edge_cost_reverse(src_op, si, dst_op, slot, sj, cluster):
    """Backward cost of one pair (the gradient from consumer strategy sj back to
    producer strategy si)."""
    a, b = make_op(src_op), make_op(dst_op)
    rec = OrRecord()
    s1 = np.ascontiguousarray(si, dtype=STRATEGY_DTYPE).reshape(1)
    s2 = np.ascontiguousarray(sj, dtype=STRATEGY_DTYPE).reshape(1)
    rc = lib().or_edge_cost_reverse(C.byref(a), _sp(s1), C.byref(b), slot, _sp(s2),
                                    cluster.devices, cluster.devices_per_node, cluster.bw_intra,
                                    cluster.bw_inter, C.byref(rec))
    assert rc == 0
    return (rec.t, rec.vol, rec.intra, rec.inter, rec.meta)


def edge_entries(src_op, src_strats, dst_op, slot, dst_strats, ii, jj, cluster) -> np.ndarray:
    a, b = make_op(src_op), make_op(dst_op)
    ii = np.ascontiguousarray(ii, dtype=np.int64)
    jj = np.ascontiguousarray(jj, dtype=np.int64)
    out = np.zeros(len(ii), dtype=RECORD_DTYPE)
    n = lib().or_edge_entries(C.byref(a), _sp(src_strats), C.byref(b), slot, _sp(dst_strats),
                              ii.ctypes.data_as(C.POINTER(C.c_int64)),
                              jj.ctypes.data_as(C.POINTER(C.c_int64)), len(ii), cluster.devices,
                              cluster.devices_per_node, cluster.bw_intra, cluster.bw_inter, _rp(out))
    assert n == len(ii)
    return out


def allreduce_ct(D: Sequence[int], M: Sequence[int], L: int) -> int:
    Da = (C.c_int64 * MAX_DEV)(*D)
    Ma = (C.c_int32 * MAX_SUB)(*M)
    return lib().or_allreduce_ct(Da, len(D), Ma, len(M), L)


def gather_ct(D: Sequence[int], M: Sequence[int], axis: int, L: int) -> Tuple[int, int]:
    """(ct, members of one group inside a node) of Algorithm 3."""
    Da = (C.c_int64 * MAX_DEV)(*D)
    Ma = (C.c_int32 * MAX_SUB)(*M)
    k = C.c_int64(0)
    ct = lib().or_gather_ct(Da, len(D), Ma, len(M), axis, L, C.byref(k))
    return ct, k.value


@dataclass
class Unified:
    D: List[int]
    orig: List[int]
    size: List[int]
    m_from: List[int]
    m_to: List[int]


def _unified(u: OrUnified) -> Unified:
    r = u.r
    return Unified(list(u.D[:u.h]), list(u.orig[:r]), list(u.size[:r]), list(u.m_from[:r]),
                   list(u.m_to[:r]))


def unify(N: int, Dp, Mp, Dc, Mc, shape) -> Unified:
    u = OrUnified()
    rc = lib().or_unify(N, (C.c_int64 * MAX_DEV)(*Dp), len(Dp), (C.c_int32 * MAX_RANK)(*Mp),
                        (C.c_int64 * MAX_DEV)(*Dc), len(Dc), (C.c_int32 * MAX_RANK)(*Mc),
                        len(shape), (C.c_int64 * MAX_RANK)(*shape), C.byref(u))
    assert rc == 0
    return _unified(u)


@dataclass
class RedOp:
    kind: int
    axis: int
    from_dim: int
    to_dim: int
    ct: int
    k_in: int
    shard_nb: int
    volume_nb: int
    link_nb: int
    cost: float

    def name(self) -> str:
        if self.kind == SLICE:
            return f"Slice({self.axis},{self.to_dim})"
        if self.kind == ALLGATHER:
            return f"AllGather({self.axis},{self.from_dim})"
        return f"AllToAll({self.axis},{self.from_dim}->{self.to_dim})"


def _ops(seq, n) -> List[RedOp]:
    return [RedOp(s.kind, s.axis, s.from_dim, s.to_dim, s.ct, s.k_in, s.shard_nb, s.volume_nb,
                  s.link_nb, s.cost) for s in seq[:n]]


def record_tuple(rec) -> Tuple[float, int, int, int, int]:
    return (float(rec["t"]), int(rec["vol"]), int(rec["intra"]), int(rec["inter"]),
            int(rec["meta"]))


def sequence_cost(D, m_from, m_to, cand: int, shard0_nb: int, N: int, L: int, bw_intra: int,
                  bw_inter: int):
    """Candidate ``cand`` on an already unified problem: (ops, record)."""
    seq = (OrRedop * MAX_SEQ)()
    rec = OrRecord()
    n = lib().or_sequence_cost((C.c_int64 * MAX_DEV)(*D), len(D), (C.c_int32 * MAX_SUB)(*m_from),
                               (C.c_int32 * MAX_SUB)(*m_to), len(m_from), cand, shard0_nb, N, L,
                               bw_intra, bw_inter, seq, C.byref(rec))
    assert n >= 0
    return _ops(seq, n), (rec.t, rec.vol, rec.intra, rec.inter, rec.meta)


def edge_detail(src_op, si, dst_op, slot, sj, cand: int, cluster):
    """(Unified problem, ops with costs, initial shard in nb) of one candidate."""
    a, b = make_op(src_op), make_op(dst_op)
    u = OrUnified()
    seq = (OrRedop * MAX_SEQ)()
    shard0 = C.c_uint64(0)
    s1 = np.ascontiguousarray(si, dtype=STRATEGY_DTYPE).reshape(1)
    s2 = np.ascontiguousarray(sj, dtype=STRATEGY_DTYPE).reshape(1)
    n = lib().or_edge_detail(C.byref(a), _sp(s1), C.byref(b), slot, _sp(s2), cluster.devices,
                             cluster.devices_per_node, cluster.bw_intra, cluster.bw_inter, cand,
                             C.byref(u), seq, C.byref(shard0))
    assert n >= 0
    return _unified(u), _ops(seq, n), shard0.value


def edge_cost(src_op, si, dst_op, slot, sj, cluster):
    a, b = make_op(src_op), make_op(dst_op)
    rec = OrRecord()
    s1 = np.ascontiguousarray(si, dtype=STRATEGY_DTYPE).reshape(1)
    s2 = np.ascontiguousarray(sj, dtype=STRATEGY_DTYPE).reshape(1)
    rc = lib().or_edge_cost(C.byref(a), _sp(s1), C.byref(b), slot, _sp(s2), cluster.devices,
                            cluster.devices_per_node, cluster.bw_intra, cluster.bw_inter,
                            C.byref(rec))
    assert rc == 0
    return (rec.t, rec.vol, rec.intra, rec.inter, rec.meta)


def node_cost(op, s, cluster):
    o = make_op(op)
    rec = OrRecord()
    s1 = np.ascontiguousarray(s, dtype=STRATEGY_DTYPE).reshape(1)
    lib().or_node_cost(C.byref(o), _sp(s1), cluster.devices, cluster.devices_per_node,
                       cluster.bw_intra, cluster.bw_inter, C.byref(rec))
    return (rec.t, rec.vol, rec.intra, rec.inter, rec.meta)


# ---------------------------------------------------------------------------
# several link classes (workloads.Topology)
# ---------------------------------------------------------------------------

def node_cost_topo(op, s, topo):
    o, t = make_op(op), make_topology(topo)
    rec = OrRecord()
    s1 = np.ascontiguousarray(s, dtype=STRATEGY_DTYPE).reshape(1)
    lib().or_node_cost_topo(C.byref(o), _sp(s1), topo.devices, C.byref(t), C.byref(rec))
    return (rec.t, rec.vol, rec.intra, rec.inter, rec.meta)


def node_table_topo(op, strategies: np.ndarray, topo) -> np.ndarray:
    o, t = make_op(op), make_topology(topo)
    out = np.zeros(len(strategies), dtype=RECORD_DTYPE)
    n = lib().or_node_table_topo(C.byref(o), _sp(strategies), len(strategies), topo.devices,
                                 C.byref(t), _rp(out))
    assert n == len(strategies)
    return out


def edge_cost_topo(src_op, si, dst_op, slot, sj, topo):
    a, b, t = make_op(src_op), make_op(dst_op), make_topology(topo)
    rec = OrRecord()
    s1 = np.ascontiguousarray(si, dtype=STRATEGY_DTYPE).reshape(1)
    s2 = np.ascontiguousarray(sj, dtype=STRATEGY_DTYPE).reshape(1)
    rc = lib().or_edge_cost_topo(C.byref(a), _sp(s1), C.byref(b), slot, _sp(s2), topo.devices,
                                 C.byref(t), C.byref(rec))
    assert rc == 0
    return (rec.t, rec.vol, rec.intra, rec.inter, rec.meta)


def edge_table_topo(src_op, src_strats: np.ndarray, dst_op, slot: int, dst_strats: np.ndarray,
                    topo) -> np.ndarray:
    a, b, t = make_op(src_op), make_op(dst_op), make_topology(topo)
    out = np.zeros(len(src_strats) * len(dst_strats), dtype=RECORD_DTYPE)
    n = lib().or_edge_table_topo(C.byref(a), _sp(src_strats), len(src_strats), C.byref(b), slot,
                                 _sp(dst_strats), len(dst_strats), topo.devices, C.byref(t),
                                 _rp(out))
    assert n == out.size, "oracle failed on this edge"
    return out.reshape(len(src_strats), len(dst_strats))


def edge_entries_topo(src_op, src_strats, dst_op, slot, dst_strats, ii, jj, topo) -> np.ndarray:
    a, b, t = make_op(src_op), make_op(dst_op), make_topology(topo)
    ii = np.ascontiguousarray(ii, dtype=np.int64)
    jj = np.ascontiguousarray(jj, dtype=np.int64)
    out = np.zeros(len(ii), dtype=RECORD_DTYPE)
    n = lib().or_edge_entries_topo(C.byref(a), _sp(src_strats), C.byref(b), slot, _sp(dst_strats),
                                   ii.ctypes.data_as(C.POINTER(C.c_int64)),
                                   jj.ctypes.data_as(C.POINTER(C.c_int64)), len(ii), topo.devices,
                                   C.byref(t), _rp(out))
    assert n == len(ii)
    return out


# ---------------------------------------------------------------------------
# whole graphs
# ---------------------------------------------------------------------------

@dataclass
class Tables:
    strategies: List[np.ndarray]   # per op
    node: List[np.ndarray]         # per op, RECORD_DTYPE
    edge: List[Optional[np.ndarray]]  # per edge, (S_src, S_dst) RECORD_DTYPE, or None if skipped


def build_tables(graph, cluster, edges: Optional[Sequence[int]] = None,
                 mesh: Optional[Sequence[int]] = None, topology=None) -> Tables:
    """Every table of ``graph`` on ``cluster`` (only the listed edges if given;
    over the strategies of the fixed mesh ``mesh`` if given; with the link
    classes of ``topology`` (a workloads.Topology of cluster.devices devices)
    in place of the cluster's two if given)."""
    strats = [enumerate_strategies(op, cluster.devices) if mesh is None
              else enumerate_strategies_mesh(op, mesh) for op in graph.ops]
    if topology is not None:
        assert topology.devices == cluster.devices
        node = [node_table_topo(op, s, topology) for op, s in zip(graph.ops, strats)]
        edge = []
        for k, e in enumerate(graph.edges):
            edge.append(edge_table_topo(graph.ops[e.src], strats[e.src], graph.ops[e.dst], e.slot,
                                        strats[e.dst], topology)
                        if edges is None or k in edges else None)
        return Tables(strats, node, edge)
    node = [node_table(op, s, cluster) for op, s in zip(graph.ops, strats)]
    want = set(range(len(graph.edges))) if edges is None else set(edges)
    edge = []
    for k, e in enumerate(graph.edges):
        if k in want:
            edge.append(edge_table(graph.ops[e.src], strats[e.src], graph.ops[e.dst], e.slot,
                                   strats[e.dst], cluster))
        else:
            edge.append(None)
    return Tables(strats, node, edge)
